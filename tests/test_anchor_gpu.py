"""GPU parity of the anchor-pool path against the oracle: token-wise interpolation weights (Appendix A.3), the
anchored apply of Eq. 8 and the gate distances of Eq. 9.

Anchors are seeded synthetic low-rank states (Gaussian coefficients, orthonormal bases) with a different coefficient
scale per anchor, so that the distances, and with them the weights, differ between anchors.  The bar: weights and
gate distances to fp32 accuracy of the distance sums, corrected caches to the storage tolerance (1e-2 bf16, 1e-5
fp32), bit copies past the weighted rows.
"""
import numpy as np
import pytest
import torch

from oracle import kvc_oracle as O
from paper_2609_34060_amd import kvc, synth
from tests import helpers as Hp

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}


def _anchor_states(w, L, T, ranks, scales, key):
    H, d = w.num_kv_heads, w.head_dim
    sdt = synth.storage_dtype(w)
    out = []
    for v, (r, sc) in enumerate(zip(ranks, scales)):
        coef, basis, sigma = synth.random_state(L, H, d, T, r, sdt, "cuda", key, v, coef_scale=sc)
        out.append(kvc.State(coef.contiguous(), basis.contiguous(), sigma.contiguous()))
    return out


def _ostate(st):
    return Hp.oracle_state(st.coef, st.basis)


def _setup(name, layers, num_tokens=None, **over):
    w = synth.WORKLOADS[name].with_(num_layers=layers, **over)
    if num_tokens is not None:
        w = w.with_(seq_tokens=(num_tokens,))
    pc = synth.build_paged(w, device="cuda", num_output_agents=1)
    cache = kvc.Cache(pc.k_pools, pc.v_pools)
    T = w.seq_tokens[0]
    src, dst = pc.seqs[(0, 0)], pc.seqs[(0, 100)]
    tab = (lambda s: None) if pc.tables is None else (lambda s: pc.tables[[s.table_row]])
    return w, pc, cache, T, src, dst, tab


# Cases with at most ten 32-rank chunks fit every anchor's basis in LDS at once; those with more (the 6-anchor cases)
# take the one-anchor-at-a-time kernels.  The last two run at head_dim 64 (bf16), one of them with three KV heads.
@pytest.mark.parametrize("name,layers,ranks,Ts,over", [
    ("tiny", 2, [8, 4, 8], 200, {}),
    ("llama8b_4k", 2, [32] * 10, 4096, {}),
    ("llama8b_4k", 1, [16, 32, 48, 8, 40], 1531, {}),
    ("llama8b_4k", 1, [64, 48, 64, 40, 64, 56], 2050, {}),
    ("llama8b_4k", 1, [32, 16, 40], 900, {"head_dim": 64, "seq_tokens": (1000,)}),
    ("llama8b_4k", 1, [64, 48, 64, 40, 64, 56], 700, {"head_dim": 64, "num_kv_heads": 3, "seq_tokens": (800,)}),
    # block size 8: a 2048-token workgroup of the resident kernels spans 256 blocks, more than its register-held
    # table slice (128), so it reads its block ids from the table in memory
    ("llama8b_4k", 1, [32, 32, 16], 3000, {"block_size": 8, "seq_tokens": (3100,)}),
])
def test_anchor_weights_and_anchored_apply(name, layers, ranks, Ts, over):
    w, pc, cache, T, src, dst, tab = _setup(name, layers, num_tokens=None, **over)
    Ts = min(Ts, T)
    # base reconstructions of RMS 0.1 + 0.9 v: mean distances from about 0.8 upwards for unit-variance caches
    scales = [(0.1 + 0.9 * v) / np.sqrt(r / w.head_dim) for v, r in enumerate(ranks)]
    bases = _anchor_states(w, layers, T, ranks, scales, 3)
    deltas = _anchor_states(w, layers, T, ranks, [0.25 * np.sqrt(w.head_dim / r) for r in ranks], 4)
    anchors = kvc.Anchors(bases, Ts, layers)
    batch_w = kvc.Batch([T], [src.offset], [src.offset], [kvc.State.empty(layers, w.num_kv_heads, w.head_dim, 0, 0,
                                                                          synth.storage_dtype(w), "cuda")],
                        tab(src), tab(src))
    kvc.kvc_anchor_weights(cache, batch_w, anchors)
    batch_a = kvc.Batch([T], [src.offset], [dst.offset], batch_w.states, tab(src), tab(dst))
    kvc.kvc_apply_anchored(cache, batch_a, anchors.with_states(deltas))
    torch.cuda.synchronize()
    got_w = anchors.weights.cpu().numpy().astype(np.float64)

    cnp = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size)
    dt = cnp.dtype
    item = O.Item(T, src.offset, dst.offset, Hp.table_np(tab(src), 0), Hp.table_np(tab(dst), 0))
    dist = O.anchor_distances(cnp, item, [_ostate(b) for b in bases], Ts)
    ref_w = O.softmax_weights(dist)
    assert np.allclose(got_w.sum(axis=-1), 1.0, atol=1e-5)
    werr = np.max(np.abs(got_w - ref_w))
    spread = np.max(ref_w) - np.min(ref_w)
    print(f"{name}: weight err {werr:.2e} (weights span {np.min(ref_w):.3f}..{np.max(ref_w):.3f})")
    assert werr <= 2e-4, werr
    assert spread > 0.05  # the anchors are distinguishable, so the check has teeth

    ref = O.apply_anchored(cnp, item, [_ostate(d) for d in deltas], ref_w, Ts)
    gnp = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size)
    worst, teeth = 0.0, 0.0
    for layer in range(layers):
        for kv in range(2):
            for h in range(w.num_kv_heads):
                g = O.read_rows(gnp, layer, kv, h, item.dst_table, item.dst_offset, T)
                e = O.read_rows(ref, layer, kv, h, item.dst_table, item.dst_offset, T)
                s = O.read_rows(cnp, layer, kv, h, item.src_table, item.src_offset, T)
                worst = max(worst, O.max_relative_error(O.to_f64(g, dt), O.to_f64(e, dt)))
                teeth = max(teeth, O.max_relative_error(O.to_f64(s, dt), O.to_f64(e, dt)))
                assert np.array_equal(g[Ts:], s[Ts:])
    print(f"{name}: anchored apply err {worst:.2e} (uncorrected {teeth:.2e})")
    assert worst <= TOL[dt], worst
    assert teeth >= 10 * TOL[dt]


def test_anchored_apply_with_one_anchor_matches_kvc_apply():
    """V = 1: the weights are exactly 1 and the anchored apply is the single-state apply (one bf16 ulp of the value,
    plus fp32 summation-order noise near zero)."""
    w, pc, cache, T, src, dst, tab = _setup("llama8b_4k", 1, num_tokens=None)
    (delta,) = _anchor_states(w, 1, T, [32], [0.5], 5)
    st = kvc.State.empty(1, w.num_kv_heads, w.head_dim, 0, 0, torch.bfloat16, "cuda")
    anchors = kvc.Anchors([delta], T, 1)
    kvc.kvc_anchor_weights(cache, kvc.Batch([T], [src.offset], [src.offset], [st], tab(src), tab(src)), anchors)
    torch.cuda.synchronize()
    assert torch.all(anchors.weights == 1.0)
    kvc.kvc_apply_anchored(cache, kvc.Batch([T], [src.offset], [dst.offset], [st], tab(src), tab(dst)), anchors)
    torch.cuda.synchronize()
    got = [p.clone() for p in pc.k_pools + pc.v_pools]
    kvc.kvc_apply(cache, kvc.Batch([T], [src.offset], [dst.offset], [delta], tab(src), tab(dst)))
    torch.cuda.synchronize()
    for a, b in zip(got, pc.k_pools + pc.v_pools):
        a32, b32 = a.float(), b.float()
        ok = torch.isnan(b32) | ((a32 - b32).abs() <= b32.abs() * 2.0 ** -7 + 2.0 ** -16 * 8.0)
        assert bool(ok.all()), float((a32 - b32).abs().nan_to_num().max())


@pytest.mark.parametrize("name,layers,prefix,ranks,over", [("tiny", 2, 100, [8, 8, 8], {}),
                                                           ("llama8b_4k", 3, 1000, [32] * 4, {}),
                                                           ("llama8b_4k", 2, 4096, [32] * 4, {}),
                                                           # 3 layers x 4 chunks x 8 heads = 96 partials per anchor:
                                                           # the finishing sum takes two per lane for half the lanes
                                                           ("llama8b_4k", 3, 4096, [32] * 3, {}),
                                                           ("llama8b_4k", 1, 1500, [96, 96, 64, 96], {}),
                                                           ("llama8b_4k", 1, 700, [32, 32, 16],
                                                            {"head_dim": 64, "seq_tokens": (900,)}),
                                                           ("llama8b_4k", 1, 3000, [32, 32],
                                                            {"block_size": 8, "seq_tokens": (3100,)})])
def test_gate_distances_and_decision(name, layers, prefix, ranks, over):
    w, pc, cache, T, src, dst, tab = _setup(name, layers, num_tokens=None, **over)
    bases = _anchor_states(w, layers, T, ranks, [(0.1 + 0.9 * v) / np.sqrt(r / w.head_dim)
                                                 for v, r in enumerate(ranks)], 6)
    anchors = kvc.Anchors(bases, T, layers, weights=torch.empty(0, device="cuda"))
    st = kvc.State.empty(layers, w.num_kv_heads, w.head_dim, 0, 0, synth.storage_dtype(w), "cuda")
    batch = kvc.Batch([T], [src.offset], [src.offset], [st], tab(src), tab(src))
    dist = kvc.kvc_gate_distances(cache, batch, anchors, prefix)
    dist2 = kvc.kvc_gate_distances(cache, batch, anchors, prefix)
    torch.cuda.synchronize()
    assert torch.equal(dist, dist2)  # fixed summation order
    cnp = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size)
    item = O.Item(T, src.offset, src.offset, Hp.table_np(tab(src), 0), Hp.table_np(tab(src), 0))
    ref = O.gate_distances(cnp, item, [_ostate(b) for b in bases], prefix)
    got = dist.cpu().numpy().astype(np.float64)
    rel = np.max(np.abs(got - ref) / ref)
    print(f"{name}: gate distance rel err {rel:.2e}")
    assert rel <= 1e-4, (got, ref)
    for tau in (0.2, 0.5, 0.9, 1.0):
        acc, g, h = kvc.kvc_gate_decide(list(got), tau)
        og, oh, oacc = O.gate(got.astype(np.float64), tau)
        assert np.allclose(g, og, atol=1e-6) and abs(h - oh) <= 1e-6
        if abs(oh - tau) > 1e-6:
            assert acc == oacc
