"""kvc_chain on the GPU against the CPU oracle (same input states), and the chained pipelines end to end.

The oracle composes by materialising A1 B1 + A2 B2 and taking its truncated SVD (Eq. 6, Eq. 7); the GPU never forms
the T x d sum.  Compared: singular values, the product A B per unit, and caches materialised from the composed
states.  Truncation is tested only where it is well defined (a gap at r_out); lossless compositions always are.
"""
import numpy as np
import pytest
import torch

from oracle import kvc_oracle as O
from paper_2609_34060_amd import kvc, synth
from tests import helpers as Hp

pytestmark = pytest.mark.gpu

TOL_PROD = {"f32": 1e-4, "bf16": 1e-2}
TOL_SIGMA = 1e-4
TOL_CACHE = {"f32": 1e-5, "bf16": 1e-2}


def _orth(rng, n, k):
    q, r = np.linalg.qr(rng.standard_normal((n, k)))
    return q * np.sign(np.diag(r))


def _state(rng, L, H, d, T, r, dtype, scale=1.0, basis=None):
    """coef = U diag(s) with orthonormal U and s ~ scale * U[0.5, 2] (descending), basis orthonormal rows."""
    coef = np.zeros((L, 2, H, T, r))
    bas = np.zeros((L, 2, H, r, d))
    for idx in np.ndindex(L, 2, H):
        s = np.sort(rng.uniform(0.5, 2.0, r))[::-1] * scale * np.sqrt(T)
        coef[idx] = _orth(rng, T, r) * s
        bas[idx] = _orth(rng, d, r).T if basis is None else basis[idx]
    c = torch.from_numpy(coef).to(dtype)
    b = torch.from_numpy(bas).to(torch.float32)
    return kvc.State(c.cuda(), b.cuda(), torch.zeros(L, 2, H, r, device="cuda"))


def _chain_both(s1, s2, ro, layer_begin=0, layer_end=None):
    L, _, H, _, _ = s1.coef.shape
    d = s1.basis.shape[-1]
    T = max(s1.num_tokens, s2.num_tokens)
    out = kvc.State.empty(L, H, d, T, ro, s1.coef.dtype, "cuda")
    kvc.kvc_chain(s1, s2, out, layer_begin, layer_end)
    torch.cuda.synchronize()
    o1, o2 = Hp.oracle_state(s1.coef, s1.basis), Hp.oracle_state(s2.coef, s2.basis)
    ost, raw = O.chain(o1, o2, ro, layer_begin=layer_begin, layer_end=layer_end)
    return out, ost, raw


def _compare(out, raw, dtype, layers=None):
    coef, basis, sigma = raw
    gc = Hp.rows_f64(Hp.to_np_storage(out.coef), dtype)
    gb = out.basis.cpu().numpy().astype(np.float64)
    gs = out.sigma.cpu().numpy().astype(np.float64)
    L, _, H, T, r = gc.shape
    worst = 0.0
    for idx in np.ndindex(L, 2, H):
        if layers is not None and idx[0] not in layers:
            continue
        assert np.allclose(gb[idx] @ gb[idx].T, np.eye(r), atol=2e-6)
        e = O.max_relative_error(gc[idx] @ gb[idx], coef[idx] @ basis[idx])
        worst = max(worst, e)
        assert e <= TOL_PROD[dtype], (idx, e)
        es = np.max(np.abs(gs[idx] - sigma[idx])) / sigma[idx][0]
        assert es <= TOL_SIGMA, (idx, es)
    return worst


@pytest.mark.parametrize("dtype,r1,r2,ro,T1,T2", [
    (torch.bfloat16, 16, 16, 32, 700, 700),     # lossless
    (torch.bfloat16, 32, 32, 64, 1000, 800),    # lossless, shorter second state (zero rows)
    (torch.bfloat16, 32, 96, 128, 300, 300),    # lossless, capped at head_dim
    (torch.float32, 8, 8, 16, 256, 256),        # fp32 coefficients
])
def test_chain_lossless(dtype, r1, r2, ro, T1, T2):
    rng = np.random.default_rng(r1 * 1000 + r2 + T1)
    s1 = _state(rng, 2, 2, 128 if dtype == torch.bfloat16 else 64, T1, r1, dtype)
    s2 = _state(rng, 2, 2, 128 if dtype == torch.bfloat16 else 64, T2, r2, dtype)
    out, ost, raw = _chain_both(s1, s2, ro)
    w = _compare(out, raw, Hp.storage_name(dtype))
    # lossless: A_out B_out reproduces A1 B1 + A2 B2 itself
    dt = Hp.storage_name(dtype)
    o1, o2 = Hp.oracle_state(s1.coef, s1.basis), Hp.oracle_state(s2.coef, s2.basis)
    gc = Hp.rows_f64(Hp.to_np_storage(out.coef), dt)
    gb = out.basis.cpu().numpy().astype(np.float64)
    T = max(T1, T2)
    m = O.materialise(o1, 1, 1, 0, T) + O.materialise(o2, 1, 1, 0, T)
    assert O.max_relative_error(gc[1, 1, 0] @ gb[1, 1, 0], m) <= TOL_PROD[dt]
    print(f"lossless {dtype} {r1}+{r2}->{ro}: worst prod {w:.2e}")


# Shapes beyond the lossless cases above: head_dim 64 in bfloat16, ranks that are not multiples of 8, a rank sum
# between 64 and 128, float32 at head_dim 128, and a gap-truncated head_dim 64 chain.  Lossless cases (r_out at least
# r1 + r2, or the head dimension) also check A_out B_out against A1 B1 + A2 B2 of every unit.
@pytest.mark.parametrize("dtype,d,r1,r2,ro,T1,T2,scale2", [
    (torch.bfloat16, 64, 16, 8, 24, 500, 450, 1.0),     # head_dim 64, lossless
    (torch.bfloat16, 64, 40, 40, 64, 600, 600, 1.0),    # head_dim 64, capped at the head dimension
    (torch.bfloat16, 128, 10, 7, 17, 333, 333, 1.0),    # ranks off multiples of 8, lossless
    (torch.bfloat16, 128, 48, 40, 88, 400, 380, 1.0),   # rank sum 88, lossless
    (torch.float32, 128, 16, 16, 32, 256, 256, 1.0),    # float32 at head_dim 128, lossless
    (torch.bfloat16, 64, 12, 6, 12, 420, 420, 0.01),    # truncated at a gap (second state far below the first)
])
def test_chain_shapes(dtype, d, r1, r2, ro, T1, T2, scale2):
    rng = np.random.default_rng(d * 100000 + r1 * 1000 + r2)
    L, H = 2, 2
    s1 = _state(rng, L, H, d, T1, r1, dtype)
    s2 = _state(rng, L, H, d, T2, r2, dtype, scale=scale2)
    out, ost, raw = _chain_both(s1, s2, ro)
    dt = Hp.storage_name(dtype)
    w = _compare(out, raw, dt)
    if ro >= min(r1 + r2, d):
        o1, o2 = Hp.oracle_state(s1.coef, s1.basis), Hp.oracle_state(s2.coef, s2.basis)
        gc = Hp.rows_f64(Hp.to_np_storage(out.coef), dt)
        gb = out.basis.cpu().numpy().astype(np.float64)
        T = max(T1, T2)
        for layer in range(L):
            for kv_ in range(2):
                for h in range(H):
                    m = O.materialise(o1, layer, kv_, h, T) + O.materialise(o2, layer, kv_, h, T)
                    e = O.max_relative_error(gc[layer, kv_, h] @ gb[layer, kv_, h], m)
                    assert e <= TOL_PROD[dt], (layer, kv_, h, e)
    print(f"chain {dtype} d {d} {r1}+{r2}->{ro}: worst prod {w:.2e}")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_chain_truncated_with_gap(dtype):
    rng = np.random.default_rng(7)
    d = 128 if dtype == torch.bfloat16 else 64
    s1 = _state(rng, 2, 1, d, 900, 24, dtype)
    s2 = _state(rng, 2, 1, d, 900, 16, dtype, scale=0.01)   # well below the first state's spectrum
    out, ost, raw = _chain_both(s1, s2, 24)
    print("truncated worst prod", _compare(out, raw, Hp.storage_name(dtype)))


def test_chain_shared_subspace_is_exact_at_rank():
    """Both corrections in one rank-32 row space (the long-context recipe): composing to rank 32 loses nothing."""
    rng = np.random.default_rng(8)
    L, H, d, T, r = 1, 2, 128, 1200, 32
    basis = np.zeros((L, 2, H, r, d))
    for idx in np.ndindex(L, 2, H):
        basis[idx] = _orth(rng, d, r).T
    s1 = _state(rng, L, H, d, T, r, torch.bfloat16, basis=basis)
    s2 = _state(rng, L, H, d, T, r, torch.bfloat16, basis=basis)
    out, ost, raw = _chain_both(s1, s2, r)
    _compare(out, raw, "bf16")


def test_chain_layer_range_and_rank0_operand():
    rng = np.random.default_rng(9)
    s1 = _state(rng, 3, 1, 128, 500, 16, torch.bfloat16)
    s0 = kvc.State.empty(3, 1, 128, 500, 0, torch.bfloat16, "cuda")
    out, ost, raw = _chain_both(s1, s0, 16, 1, 3)
    _compare(out, raw, "bf16", layers=(1, 2))
    assert float(out.basis[0].abs().sum()) == 0.0          # layer 0 untouched


def _pipeline(w, ro_cap=None):
    """Fit every edge on ground-truth pairs, then M1 (apply each edge to the previous output) and M2 (compose the
    states and apply to the first agent's exact cache).  Returns per-agent worst errors vs the oracle."""
    pc = synth.build_paged(w, device="cuda", num_output_agents=2 * (w.num_agents - 1))
    L, H, d, T = len(pc.layers), w.num_kv_heads, w.head_dim, w.seq_tokens[0]
    sdt = synth.storage_dtype(w)
    dt = Hp.storage_name(sdt)
    cache = kvc.Cache(pc.k_pools, pc.v_pools)

    def tab(seq):
        return None if pc.tables is None else pc.tables[[pc.seqs[seq].table_row]]

    def batch(src, dst, st, ntok=T):
        return kvc.Batch([ntok], [pc.seqs[src].offset], [pc.seqs[dst].offset], [st], tab(src), tab(dst))

    gt = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size)
    A = w.num_agents
    # GPU: fit edges j-1 -> j on ground truth
    S = []
    for j in range(1, A):
        st = kvc.State.empty(L, H, d, T, w.rank, sdt, "cuda")
        kvc.kvc_fit_state(cache, batch((0, j - 1), (0, j), st))
        S.append(st)
    # M1: C_hat_j = apply(S_j, C_hat_{j-1}), C_hat_0 = C_0; outputs in slots 100 + (j - 1)
    prev = (0, 0)
    for j in range(1, A):
        kvc.kvc_apply(cache, batch(prev, (0, 100 + j - 1), S[j - 1]))
        prev = (0, 100 + j - 1)
    # M2: T_j = chain(T_{j-1}, S_j), C_hat_j = apply(T_j, C_0); outputs in slots 100 + A - 1 + (j - 1)
    Tst = S[0]
    for j in range(1, A):
        if j > 1:
            ro = min(Tst.rank + S[j - 1].rank, d) if ro_cap is None else min(ro_cap, Tst.rank + S[j - 1].rank, d)
            nxt = kvc.State.empty(L, H, d, T, ro, sdt, "cuda")
            kvc.kvc_chain(Tst, S[j - 1], nxt)
            Tst = nxt
        kvc.kvc_apply(cache, batch((0, 0), (0, 100 + A - 1 + j - 1), Tst))
    torch.cuda.synchronize()
    got = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size)

    # oracle pipeline on the same ground truth
    def oitem(src, dst, st=None):
        return O.Item(T, pc.seqs[src].offset, pc.seqs[dst].offset, Hp.table_np(tab(src), 0),
                      Hp.table_np(tab(dst), 0), st)

    OS = [O.fit(gt, [oitem((0, j - 1), (0, j))], w.rank)[0][0] for j in range(1, A)]
    ref = gt
    prev = (0, 0)
    for j in range(1, A):
        ref = O.apply(ref, [oitem(prev, (0, 100 + j - 1), OS[j - 1])])
        prev = (0, 100 + j - 1)
    OT = OS[0]
    for j in range(1, A):
        if j > 1:
            ro = min(OT.rank + OS[j - 1].rank, d) if ro_cap is None else min(ro_cap, OT.rank + OS[j - 1].rank, d)
            OT = O.chain(OT, OS[j - 1], ro)[0]
        ref = O.apply(ref, [oitem((0, 0), (0, 100 + A - 1 + j - 1), OT)])

    res = []
    for j in range(1, A):
        for slot, name in ((100 + j - 1, "M1"), (100 + A - 1 + j - 1, "M2")):
            it = oitem((0, 0), (0, slot))
            worst, approx = 0.0, 0.0
            for layer in range(L):
                for kv_ in range(2):
                    for h in range(H):
                        g = O.to_f64(O.read_rows(got, layer, kv_, h, it.dst_table, it.dst_offset, T), dt)
                        e = O.to_f64(O.read_rows(ref, layer, kv_, h, it.dst_table, it.dst_offset, T), dt)
                        truth = O.to_f64(O.read_rows(gt, layer, kv_, h, Hp.table_np(tab((0, j)), 0),
                                                     pc.seqs[(0, j)].offset, T), dt)
                        worst = max(worst, O.max_relative_error(g, e))
                        approx = max(approx, O.normalized_frobenius_error(g, truth))
            res.append((name, j, worst, approx))
    return res


def test_pipeline_llama_shapes_chained_m1_m2():
    w = synth.WORKLOADS["llama8b_4k"].with_(num_layers=2, num_kv_heads=2, seq_tokens=(1500,), num_agents=4)
    for name, j, worst, approx in _pipeline(w):
        print(f"{name} agent {j}: vs oracle {worst:.2e}, normalised Frobenius vs exact cache {approx:.2e}")
        assert worst <= TOL_CACHE["bf16"], (name, j, worst)


def test_pipeline_shared_subspace_truncated_chain():
    w = synth.WORKLOADS["llama8b_32k"].with_(num_layers=1, num_kv_heads=2, seq_tokens=(2048,), num_agents=4)
    for name, j, worst, approx in _pipeline(w, ro_cap=32):
        print(f"{name} agent {j}: vs oracle {worst:.2e}, normalised Frobenius vs exact cache {approx:.2e}")
        assert worst <= TOL_CACHE["bf16"], (name, j, worst)


def test_pipeline_tiny_fp32():
    for name, j, worst, approx in _pipeline(synth.WORKLOADS["tiny"].with_(num_agents=3)):
        print(f"{name} agent {j}: vs oracle {worst:.2e}, normalised Frobenius vs exact cache {approx:.2e}")
        assert worst <= TOL_CACHE["f32"], (name, j, worst)
