"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each check is independent of the oracle's own formulas: hand-worked fixtures under tests/golden/, closed forms
(exact singular values of generated low-rank matrices, Eckart-Young), an independent library routine (LAPACK's
symmetric eigensolver instead of the oracle's SVD, torch's float32->bfloat16 cast), brute force with pure-Python
loops on tiny inputs, and invariants (rank-0 identity, permuted block tables).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import kvc_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _num(x):
    if isinstance(x, str):
        return -0.0 if x == "-0" else float(eval(x, {"sqrt": math.sqrt}))
    return float(x)


def _arr(rows):
    return np.array([[_num(v) for v in r] for r in rows], dtype=np.float64)


def _bf16_torch(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


# ------------------------------------------------------------------------------------------------ storage rounding

def test_bf16_decode_roundtrip_all_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = O.bf16_bits_to_f64(bits)
    ok = ~np.isnan(vals)
    assert np.array_equal(O.f64_to_bf16_bits(vals[ok]), bits[ok])
    assert np.all(np.isnan(O.bf16_bits_to_f64(O.f64_to_bf16_bits(vals[~ok]))))


def test_bf16_rounding_matches_torch_on_binary32_inputs():
    rng = np.random.default_rng(5)
    raw = rng.integers(0, 1 << 32, size=200000, dtype=np.uint64).astype(np.uint32)
    x32 = raw.view(np.float32)
    x32 = x32[np.isfinite(x32)]
    extra = np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38, 1e-40, -1e-40, 1.00390625, 1.01171875],
                     dtype=np.float32)
    x32 = np.concatenate([x32, extra, rng.standard_normal(100000).astype(np.float32)])
    assert np.array_equal(O.f64_to_bf16_bits(x32.astype(np.float64)), _bf16_torch(x32))


def test_bf16_rounding_is_single_rounding_from_binary64():
    # 1 + 2^-8 is the midpoint between bfloat16 1.0 (0x3F80) and 1 + 2^-7 (0x3F81).  A value just above it must go
    # up even though rounding it to binary32 first would land exactly on the midpoint and then tie to even.
    half = 2.0 ** -8
    cases = {
        1.0 + half + 2.0 ** -40: 0x3F81,
        1.0 + half - 2.0 ** -40: 0x3F80,
        1.0 + half: 0x3F80,                 # tie -> even
        1.0 + 3 * half: 0x3F82,             # tie -> even
        -(1.0 + half + 2.0 ** -40): 0xBF81,
        float("inf"): 0x7F80,
        -float("inf"): 0xFF80,
        -0.0: 0x8000,
        1e39: 0x7F80,                       # beyond the largest bfloat16
    }
    got = O.f64_to_bf16_bits(np.array(list(cases.keys())))
    assert [int(g) for g in got] == list(cases.values())
    nan_bits = O.f64_to_bf16_bits(np.array([float("nan")]))
    assert np.isnan(O.bf16_bits_to_f64(nan_bits))[0]


def test_f32_rounding_is_ieee():
    x = np.array([1.0 + 2.0 ** -24, 1.0 + 2.0 ** -24 + 2.0 ** -50, 1.0 + 3 * 2.0 ** -24])
    assert O.f64_to_f32(x).view(np.uint32).tolist() == [0x3F800000, 0x3F800001, 0x3F800002]


# ------------------------------------------------------------------------------------------------ apply

def _golden_cache(g, dtype):
    nb, bs, H, d = g["num_blocks"], g["block_size"], g["num_kv_heads"], g["head_dim"]
    pool = np.full((nb, bs, H, d), 99.0)
    src = _arr(g["src_rows"])
    for (blk, slot), row in zip(g["src_locations"], src):
        pool[blk, slot, 0] = row
    stored = O.to_storage(pool, dtype)
    return O.Cache(dtype, bs, [stored], [stored.copy()])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_apply_worked_example(dtype):
    g = _load("apply_worked_example.json")
    cache = _golden_cache(g, dtype)
    coef = _arr(g["coef"])
    basis = _arr(g["basis"])
    T, Ts = g["num_tokens"], g["state_tokens"]
    st = O.State(O.to_storage(coef[None, None, None].repeat(2, axis=1), dtype),
                 basis[None, None, None].repeat(2, axis=1).astype(np.float32), None, dtype)
    item = O.Item(T, g["src_offset"], g["dst_offset"], np.array(g["src_table"]), np.array(g["dst_table"]), st)
    assert st.num_tokens == Ts
    out = O.apply(cache, [item])
    exp = _arr(g["expected_rows"])
    for kv in range(2):
        for (blk, slot), row in zip(g["dst_locations"], exp):
            got = out.pool(0, kv)[blk, slot, 0]
            assert np.array_equal(O.to_f64(got, dtype), row)
            # signed zeros: the copied -0 stays -0; the corrected 0.5 + (-0.5) is +0
            assert np.array_equal(np.signbit(O.to_f64(got, dtype)), np.signbit(row))
        # the source rows are untouched
        for (blk, slot), row in zip(g["src_locations"], _arr(g["src_rows"])):
            assert np.array_equal(O.to_f64(out.pool(0, kv)[blk, slot, 0], dtype), row)


def _brute_apply_rows(src, coef, basis):
    """Pure-Python loops: out[t][j] = src[t][j] + sum_k coef[t][k] * basis[k][j] for covered rows."""
    out = [list(map(float, r)) for r in src]
    for t in range(len(coef)):
        for j in range(len(basis[0])):
            acc = float(src[t][j])
            for k in range(len(basis)):
                acc += float(coef[t][k]) * float(basis[k][j])
            out[t][j] = acc
    return np.array(out)


def test_apply_matches_brute_force_loops():
    rng = np.random.default_rng(3)
    T, Ts, r, d = 9, 7, 3, 5
    src = rng.standard_normal((T, d)).astype(np.float32)
    coef = rng.standard_normal((Ts, r))
    basis = rng.standard_normal((r, d))
    got = O.correct_rows(src, coef, basis, "f32")
    ref = _brute_apply_rows(src.astype(np.float64), coef, basis)
    assert np.allclose(got.astype(np.float64), ref, rtol=2 ** -23, atol=1e-12)
    assert np.array_equal(got[Ts:], src[Ts:])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_apply_rank0_and_zero_coverage_are_bit_copies(dtype):
    rng = np.random.default_rng(11)
    T, d = 37, 8
    vals = rng.standard_normal((T, d))
    vals[0, 0] = -0.0
    src = O.to_storage(vals, dtype)
    if dtype == "bf16":
        src[1, 1] = 0x7FC1       # a NaN payload survives a copy
    for coef, basis in [(np.zeros((T, 0)), np.zeros((0, d))), (np.zeros((0, 4)), rng.standard_normal((4, d)))]:
        out = O.correct_rows(src, coef, basis, dtype)
        assert out.tobytes() == src.tobytes()


def test_apply_through_permuted_tables_equals_contiguous():
    rng = np.random.default_rng(4)
    bs, H, d, T, r = 4, 2, 8, 13, 3
    nblk_seq = -(-T // bs)
    vals = rng.standard_normal((T, H, d))
    coef = rng.standard_normal((1, 2, H, T, r))
    basis = rng.standard_normal((1, 2, H, r, d)).astype(np.float32)
    st = O.State(coef.astype(np.float32), basis, None, "f32")

    # contiguous: src in blocks [0, nblk_seq), dst in [nblk_seq, 2 nblk_seq)
    pool = np.zeros((2 * nblk_seq, bs, H, d), dtype=np.float32)
    pool.reshape(-1, H, d)[:T] = vals
    c1 = O.Cache("f32", bs, [pool], [pool.copy()])
    o1 = O.apply(c1, [O.Item(T, 0, nblk_seq * bs, None, None, st)])
    ref = o1.k[0].reshape(-1, H, d)[nblk_seq * bs: nblk_seq * bs + T]

    # paged: the same rows behind a shuffled table, misaligned offsets on both sides
    nb = 3 * nblk_seq + 2
    perm = rng.permutation(nb)
    src_tab, dst_tab = perm[:nblk_seq + 1], perm[nblk_seq + 1: 2 * nblk_seq + 2]
    pool2 = np.zeros((nb, bs, H, d), dtype=np.float32)
    c2 = O.Cache("f32", bs, [pool2], [pool2.copy()])
    for kv in range(2):
        for h in range(H):
            O.write_rows(c2, 0, kv, h, src_tab, 3, vals[:, h].astype(np.float32))
    o2 = O.apply(c2, [O.Item(T, 3, 1, src_tab, dst_tab, st)])
    for h in range(H):
        got = O.read_rows(o2, 0, 0, h, dst_tab, 1, T)
        assert np.array_equal(got, ref[:, h])


# ------------------------------------------------------------------------------------------------ fit (Eq. 7)

def test_svd_worked_examples():
    g = _load("svd_worked_examples.json")
    for case in g["cases"]:
        z = _arr(case["z"])
        r = z.shape[1]
        a, b, s = O.truncated_svd(z, r)
        assert np.allclose(s, [_num(v) for v in case["sigma"]], atol=1e-14)
        assert np.allclose(a, _arr(case["A"]), atol=1e-14)
        assert np.allclose(b, _arr(case["B"]), atol=1e-14)
        a1, b1, _ = O.truncated_svd(z, 1)
        assert math.isclose(np.sum((z - a1 @ b1) ** 2), case["rank1_residual_sq"], rel_tol=1e-13)


def _lowrank(rng, T, d, r, s):
    u, _ = np.linalg.qr(rng.standard_normal((T, r)))
    v, _ = np.linalg.qr(rng.standard_normal((d, r)))
    return (u * s) @ v.T


@pytest.mark.parametrize("T,d,r", [(64, 16, 4), (40, 32, 8), (16, 16, 16)])
def test_fit_exact_rank_recovers_generator_singular_values(T, d, r):
    rng = np.random.default_rng(T * d + r)
    s = np.sort(rng.uniform(0.1, 1.0, r))[::-1]
    z = _lowrank(rng, T, d, r, s)
    a, b, sig = O.truncated_svd(z, r)
    assert np.allclose(sig, s, rtol=1e-12, atol=1e-13)
    assert np.allclose(a @ b, z, atol=1e-12)
    assert np.allclose(b @ b.T, np.eye(r), atol=1e-12)                # B = R_r^T has orthonormal rows
    assert np.allclose(a.T @ a, np.diag(sig ** 2), atol=1e-12)         # A = U_r Sigma_r


def test_fit_eckart_young_against_independent_eigensolver():
    rng = np.random.default_rng(8)
    T, d = 50, 12
    z = rng.standard_normal((T, d))
    lam = np.sort(np.linalg.eigvalsh(z.T @ z))[::-1]                    # LAPACK dsyevd, not the SVD
    for r in range(0, d + 1):
        a, b, s = O.truncated_svd(z, r)
        assert np.allclose(s, np.sqrt(lam[:r]), rtol=1e-10)
        resid = np.sum((z - a @ b) ** 2)
        assert math.isclose(resid, lam[r:].sum(), rel_tol=1e-9, abs_tol=1e-9)
        # the product equals the projection on the top-r eigenvectors of Z^T Z
        w, vecs = np.linalg.eigh(z.T @ z)
        top = vecs[:, np.argsort(w)[::-1][:r]]
        assert np.allclose(a @ b, z @ top @ top.T, atol=1e-9)


def _power_top_pair(z, iters=2000):
    """Pure-Python power iteration on Z^T Z for the leading singular triplet."""
    n, d = len(z), len(z[0])
    v = [1.0 / math.sqrt(d)] * d
    for _ in range(iters):
        zv = [sum(z[i][j] * v[j] for j in range(d)) for i in range(n)]
        w = [sum(z[i][j] * zv[i] for i in range(n)) for j in range(d)]
        nrm = math.sqrt(sum(x * x for x in w))
        v = [x / nrm for x in w]
    zv = [sum(z[i][j] * v[j] for j in range(d)) for i in range(n)]
    return math.sqrt(sum(x * x for x in zv)), v


def test_fit_top_triplet_matches_brute_force_power_iteration():
    rng = np.random.default_rng(9)
    z = rng.standard_normal((7, 4)) + np.outer(rng.standard_normal(7), [3.0, -1.0, 2.0, 0.5])
    s1, v1 = _power_top_pair(z.tolist())
    a, b, s = O.truncated_svd(z, 1)
    assert math.isclose(s[0], s1, rel_tol=1e-10)
    v1 = np.array(v1)
    v1 = v1 if v1[np.argmax(np.abs(v1))] > 0 else -v1                 # canonical sign
    assert np.allclose(b[0], v1, atol=1e-8)
    assert np.allclose(a[:, 0], z @ v1, atol=1e-7)


def test_fit_rank_above_data_rank_adds_zero_components():
    rng = np.random.default_rng(10)
    z = _lowrank(rng, 30, 10, 3, np.array([3.0, 2.0, 1.0]))
    a, b, s = O.truncated_svd(z, 6)
    assert np.allclose(s[3:], 0, atol=1e-12)
    assert np.allclose(a @ b, z, atol=1e-12)
    assert np.allclose(b @ b.T, np.eye(6), atol=1e-12)


def test_canonical_sign_convention():
    rng = np.random.default_rng(12)
    z = rng.standard_normal((20, 6))
    _, b, _ = O.truncated_svd(z, 6)
    for row in b:
        assert row[np.argmax(np.abs(row))] > 0
    # exact ties: the first tied index is made positive
    _, b, _ = O.truncated_svd(np.array([[2.0, 2.0], [1.0, -1.0]]), 2)
    assert b[0, 0] > 0 and b[1, 0] > 0


def _paired_cache(rng, dtype, T, H, d, L, bs, deviation):
    """A two-sequence contiguous cache: src rows, then dst rows = src + deviation(layer, kv, head)."""
    nb = 2 * (-(-T // bs))
    pools = {}
    for kv in range(2):
        pools[kv] = []
        for layer in range(L):
            pool = np.zeros((nb, bs, H, d))
            flat = pool.reshape(-1, H, d)
            src = rng.standard_normal((T, H, d))
            flat[:T] = src
            for h in range(H):
                flat[nb * bs // 2: nb * bs // 2 + T, h] = src[:, h] + deviation(layer, kv, h)
            pools[kv].append(O.to_storage(pool, dtype))
    return O.Cache(dtype, bs, pools[0], pools[1]), nb * bs // 2


def test_fit_reads_dst_minus_src_through_pages():
    rng = np.random.default_rng(13)
    T, H, d, L, bs, r = 24, 2, 8, 2, 4, 3
    devs = {}

    def deviation(layer, kv, h):
        devs[(layer, kv, h)] = _lowrank(rng, T, d, r, np.array([2.0, 1.0, 0.5]) * (1 + layer + kv + h))
        return devs[(layer, kv, h)]

    cache, dst_off = _paired_cache(rng, "f32", T, H, d, L, bs, deviation)
    states, raw = O.fit(cache, [O.Item(T, 0, dst_off, None, None)], r)
    coef, basis, sigma = raw[0]
    for (layer, kv, h), dv in devs.items():
        z = (O.read_rows(cache, layer, kv, h, None, dst_off, T).astype(np.float64)
             - O.read_rows(cache, layer, kv, h, None, 0, T).astype(np.float64))
        # float32 storage makes z rank 3 only up to rounding: compare with the projection of z on the top-3
        # eigenvectors of z^T z (an independent LAPACK routine), and with z itself at storage precision
        w, vecs = np.linalg.eigh(z.T @ z)
        top = vecs[:, np.argsort(w)[::-1][:r]]
        assert np.allclose(coef[layer, kv, h] @ basis[layer, kv, h], z @ top @ top.T, atol=1e-10)
        assert np.allclose(coef[layer, kv, h] @ basis[layer, kv, h], z, atol=1e-5)
        # the stored float32 deviation is the generated one up to float32 storage of both caches
        assert np.allclose(z, dv, atol=1e-5)
        assert np.allclose(sigma[layer, kv, h], np.array([2.0, 1.0, 0.5]) * (1 + layer + kv + h), rtol=1e-5)
    # base mode factorises the dst cache itself
    _, raw_base = O.fit(cache, [O.Item(T, 0, dst_off, None, None)], d, mode=O.MODE_BASE)
    cb, bb, _ = raw_base[0]
    assert np.allclose(cb[1, 0, 1] @ bb[1, 0, 1], O.read_rows(cache, 1, 0, 1, None, dst_off, T), atol=1e-12)


def test_fit_prefix_coverage_uses_only_leading_rows():
    rng = np.random.default_rng(14)
    T, H, d, L, bs = 20, 1, 6, 1, 4
    cache, dst_off = _paired_cache(rng, "f32", T, H, d, L, bs, lambda *a: rng.standard_normal((T, d)))
    states, raw = O.fit(cache, [O.Item(T, 0, dst_off, None, None)], 2, state_tokens=[11])
    z = (O.read_rows(cache, 0, 1, 0, None, dst_off, 11).astype(np.float64)
         - O.read_rows(cache, 0, 1, 0, None, 0, 11).astype(np.float64))
    a, b, s = O.truncated_svd(z, 2)
    assert states[0].num_tokens == 11
    assert np.allclose(raw[0][0][0, 1, 0] @ raw[0][1][0, 1, 0], a @ b, atol=1e-12)


# ------------------------------------------------------------------------------------------------ chain (Eq. 6)

def _state_from(a_list, b_list, dtype="f32"):
    """One-layer, one-head state whose K and V units carry the same factors."""
    a = np.asarray(a_list, dtype=np.float64)
    b = np.asarray(b_list, dtype=np.float64)
    coef = np.stack([a, a])[None, :, None]
    basis = np.stack([b, b])[None, :, None].astype(np.float32)
    return O.State(O.to_storage(coef, dtype), basis, None, dtype)


def test_chain_worked_example():
    g = _load("chain_worked_example.json")
    s1 = _state_from(g["first"]["A"], g["first"]["B"])
    s2 = _state_from(g["second"]["A"], g["second"]["B"])
    for key, r in (("rank2", 2), ("rank1", 1)):
        _, (coef, basis, sigma) = O.chain(s1, s2, r)
        assert np.allclose(sigma[0, 0, 0], g[key]["sigma"], atol=1e-14)
        assert np.allclose(coef[0, 0, 0], _arr(g[key]["A"]), atol=1e-14)
        assert np.allclose(basis[0, 0, 0], _arr(g[key]["B"]), atol=1e-14)


def test_chain_lossless_equals_sum_and_eq6_identity():
    rng = np.random.default_rng(15)
    T, d, r1, r2 = 40, 16, 3, 4
    d1 = _lowrank(rng, T, d, r1, np.array([3.0, 2.0, 1.0]))
    d2 = _lowrank(rng, T, d, r2, np.array([2.5, 1.5, 1.0, 0.5]))
    a1, b1, _ = O.truncated_svd(d1, r1)
    a2, b2, _ = O.truncated_svd(d2, r2)
    s1, s2 = _state_from(a1, b1), _state_from(a2, b2)
    # Eq. 6: the correction from agent i to agent k equals the sum of the two consecutive corrections
    _, (coef, basis, sigma) = O.chain(s1, s2, r1 + r2)
    c0 = rng.standard_normal((T, d))
    c1 = c0 + d1
    c2 = c1 + d2
    prod = coef[0, 0, 0] @ basis[0, 0, 0]
    assert np.allclose(prod, (a1 @ b1).astype(np.float32).astype(np.float64)
                       + (a2 @ b2).astype(np.float32).astype(np.float64), atol=1e-5)
    assert np.allclose(prod, c2 - c0, atol=1e-5)
    # and equals a direct fit of the non-chained deviation C2 - C0 (Eq. 6, chained == non-chained when exact)
    a02, b02, _ = O.truncated_svd(c2 - c0, r1 + r2)
    assert np.allclose(prod, a02 @ b02, atol=1e-5)


def test_chain_orthogonal_states_keep_union_of_singular_values():
    rng = np.random.default_rng(16)
    T, d = 30, 10
    u, _ = np.linalg.qr(rng.standard_normal((T, 5)))
    v, _ = np.linalg.qr(rng.standard_normal((d, 5)))
    s_a, s_b = np.array([5.0, 3.0, 1.0]), np.array([4.0, 2.0])
    a1, b1 = u[:, :3] * s_a, v[:, :3].T
    a2, b2 = u[:, 3:] * s_b, v[:, 3:].T
    s1, s2 = _state_from(a1, b1, "f32"), _state_from(a2, b2, "f32")
    for r_out in range(1, 6):
        _, (_, _, sigma) = O.chain(s1, s2, r_out)
        assert np.allclose(sigma[0, 0, 0], [5, 4, 3, 2, 1][:r_out], atol=1e-5)


def test_chain_shared_subspace_truncation_is_exact():
    # both corrections live in one rank-3 row space (the long-context workload's structure)
    rng = np.random.default_rng(17)
    T, d, r = 25, 9, 3
    v, _ = np.linalg.qr(rng.standard_normal((d, r)))
    w1, w2 = rng.standard_normal((T, r)), rng.standard_normal((T, r))
    s1, s2 = _state_from(w1, v.T), _state_from(w2, v.T)
    _, (coef, basis, sigma) = O.chain(s1, s2, r)
    ref = (w1.astype(np.float32).astype(np.float64) + w2.astype(np.float32).astype(np.float64)) \
        @ v.T.astype(np.float32).astype(np.float64)
    assert np.allclose(coef[0, 0, 0] @ basis[0, 0, 0], ref, atol=1e-10)


def test_chain_pads_shorter_state_with_zero_rows():
    rng = np.random.default_rng(18)
    d = 6
    a1, b1 = rng.standard_normal((10, 2)), np.linalg.qr(rng.standard_normal((d, 2)))[0].T
    a2, b2 = rng.standard_normal((14, 2)), np.linalg.qr(rng.standard_normal((d, 2)))[0].T
    s1, s2 = _state_from(a1, b1), _state_from(a2, b2)
    st, (coef, basis, _) = O.chain(s1, s2, 4)
    assert st.num_tokens == 14
    m = np.zeros((14, d))
    m[:10] += s1.coef_f64(0, 0, 0) @ s1.basis_f64(0, 0, 0)
    m += s2.coef_f64(0, 0, 0) @ s2.basis_f64(0, 0, 0)
    assert np.allclose(coef[0, 0, 0] @ basis[0, 0, 0], m, atol=1e-12)


# ------------------------------------------------------------------------------------------------ metrics

def test_memory_example_is_fifty_gib():
    g = _load("memory_example.json")
    got = O.full_dimensional_pool_bytes(g["num_anchors"], g["num_consumers"], g["num_layers"], g["num_kv_heads"],
                                        g["head_dim"], g["num_tokens"], g["elem_bytes"])
    assert got == g["expected_bytes"] == g["expected_gib"] * 2 ** 30


@pytest.mark.parametrize("dtype,coef_bytes", [("bf16", 2), ("f32", 4)])
def test_lowrank_state_bytes_counts_the_arrays_fit_returns(dtype, coef_bytes):
    """Section 3.3's O(N r (L + D)) state size, pinned to the storage numpy actually holds for the states the oracle's
    fit produces (coefficients in the cache dtype, float32 basis and sigma), not to a restated formula."""
    L, H, d, bs, T, r = 2, 3, 16, 8, 40, 5
    rng = np.random.default_rng(7)
    nb = 2 * (T // bs)
    pools = [[O.to_storage(rng.standard_normal((nb, bs, H, d)), dtype) for _ in range(L)] for _ in range(2)]
    cache = O.Cache(dtype, bs, pools[0], pools[1])
    states, _ = O.fit(cache, [O.Item(T, 0, T, None, None)], r)
    st = states[0]
    assert O.lowrank_state_bytes(L, H, d, T, r, coef_bytes) == st.coef.nbytes + st.basis.nbytes + st.sigma.nbytes
    assert O.lowrank_state_bytes(L, H, d, T, r, coef_bytes, with_sigma=False) == st.coef.nbytes + st.basis.nbytes
    # with r << min(T, d) the state is far smaller than the dense segment it replaces (Section 3.1 vs 3.3)
    assert O.lowrank_state_bytes(L, H, d, T, r, coef_bytes) < O.dense_segment_bytes(L, H, d, T, coef_bytes)


def test_effective_rank_and_error_metric():
    # energies 9, 4, 1, 0.25: 90 % of 14.25 needs the first two (13 / 14.25 = 0.912)
    assert O.effective_rank(np.array([3.0, 2.0, 1.0, 0.5])) == 2
    assert O.effective_rank(np.array([1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0])) == 9
    assert O.effective_rank(np.zeros(3)) == 0
    c = np.array([[3.0, 4.0]])
    assert math.isclose(O.normalized_frobenius_error(c + np.array([[0.0, 1.0]]), c), 0.2)
    assert math.isclose(O.max_relative_error(np.array([1.0, -2.5]), np.array([1.0, -2.0])), 0.25)


# ------------------------------------------------------------------------------------------------ anchors (Eq. 8-11)

def _anchor_setup(seed=21, T=12, H=2, d=6, L=2, bs=4):
    """A contiguous f32 cache with source rows at offset 0, and helpers that build per-unit states from functions
    of (layer, kv, head) -> (A, B)."""
    rng = np.random.default_rng(seed)
    nb = 2 * (-(-T // bs))
    pools = {kv: [O.to_storage(rng.standard_normal((nb, bs, H, d)).astype(np.float32).astype(np.float64), "f32")
                  for _ in range(L)] for kv in range(2)}
    cache = O.Cache("f32", bs, pools[0], pools[1])
    item = O.Item(T, 0, nb * bs // 2, None, None)

    def state(fn):
        coefs, bases = [], []
        for layer in range(L):
            ck, bk = [], []
            for kv in range(2):
                ch, bh = zip(*[fn(layer, kv, h) for h in range(H)])
                ck.append(np.stack(ch))
                bk.append(np.stack(bh))
            coefs.append(np.stack(ck))
            bases.append(np.stack(bk))
        coef = np.stack(coefs)
        return O.State(O.to_storage(coef, "f32"), np.stack(bases).astype(np.float32), None, "f32")

    def src(layer, kv, h):
        return O.read_rows(cache, layer, kv, h, None, 0, T).astype(np.float64)

    return rng, cache, item, state, src


def test_anchor_distances_and_weights_closed_form():
    """An anchor whose base reconstructs the source exactly has distance 0; one that reconstructs source + c has
    distance |c| (the mean of |c| over every feature of the row); the weights are then 1 / (1 + e^{-|c|/T}) and
    e^{-|c|/T} / (1 + e^{-|c|/T})."""
    _, cache, item, state, src = _anchor_setup()
    T, d, c = item.num_tokens, cache.head_dim, 0.5
    exact = state(lambda l, kv, h: (src(l, kv, h), np.eye(d)))
    shifted = state(lambda l, kv, h: (np.hstack([src(l, kv, h), np.full((T, 1), c)]),
                                      np.vstack([np.eye(d), np.ones((1, d))])))
    dist = O.anchor_distances(cache, item, [exact, shifted], T)
    assert np.allclose(dist[..., 0], 0.0, atol=1e-12)
    assert np.allclose(dist[..., 1], c, atol=1e-12)
    for temp in (1.0, 2.0):
        w = O.softmax_weights(dist, temp)
        e = math.exp(-c / temp)
        assert np.allclose(w[..., 0], 1.0 / (1.0 + e)) and np.allclose(w[..., 1], e / (1.0 + e))
    # one anchor: weight 1; swapping anchors swaps the weights
    assert np.array_equal(O.softmax_weights(dist[..., :1]), np.ones_like(dist[..., :1]))
    w_swapped = O.softmax_weights(O.anchor_distances(cache, item, [shifted, exact], T))
    assert np.allclose(w_swapped[..., ::-1], O.softmax_weights(dist))


def test_apply_anchored_reduces_to_single_state_apply():
    """V = 1 (w = 1), or V anchors carrying the same correction with any weights summing to 1, is the single-state
    apply; a zero correction weighted 1 - a plus a correction weighted a is the single apply of a times it."""
    rng, cache, item, state, src = _anchor_setup(seed=22)
    T, d, r, Ts = item.num_tokens, cache.head_dim, 3, 9
    delta = state(lambda l, kv, h: (rng.standard_normal((T, r)), np.linalg.qr(rng.standard_normal((d, r)))[0].T))
    single = O.apply(cache, [O.Item(T, 0, item.dst_offset, None, None,
                                    O.State(delta.coef[:, :, :, :Ts], delta.basis, None, "f32"))])
    nl = cache.num_layers
    got = O.apply_anchored(cache, item, [delta], np.ones((nl, 2, Ts, 1)), Ts)
    for pool_a, pool_b in zip(got.k + got.v, single.k + single.v):
        assert np.array_equal(pool_a, pool_b)
    w = rng.uniform(0.1, 1.0, (nl, 2, Ts, 3))
    w /= w.sum(axis=-1, keepdims=True)
    got3 = O.apply_anchored(cache, item, [delta, delta, delta], w, Ts)
    for pool_a, pool_b in zip(got3.k + got3.v, single.k + single.v):
        assert np.allclose(O.to_f64(pool_a, "f32"), O.to_f64(pool_b, "f32"), atol=2e-6)
    a = 0.25
    zero = O.State(np.zeros_like(delta.coef), delta.basis, None, "f32")
    scaled = O.State(O.to_storage(a * O.to_f64(delta.coef[:, :, :, :Ts], "f32"), "f32"), delta.basis, None, "f32")
    wz = np.stack([np.full((nl, 2, Ts), 1 - a), np.full((nl, 2, Ts), a)], axis=-1)
    got_z = O.apply_anchored(cache, item, [zero, delta], wz, Ts)
    single_a = O.apply(cache, [O.Item(T, 0, item.dst_offset, None, None, scaled)])
    for pool_a, pool_b in zip(got_z.k + got_z.v, single_a.k + single_a.v):
        assert np.array_equal(pool_a, pool_b)
    # rows past the weighted prefix are bit copies of the source
    rows = O.read_rows(got3, 1, 1, 1, None, item.dst_offset, T)
    assert np.array_equal(rows[Ts:], O.read_rows(cache, 1, 1, 1, None, 0, T)[Ts:])


def test_gate_distances_entropy_and_acceptance():
    _, cache, item, state, src = _anchor_setup(seed=23)
    T, H, d, L, c, k = item.num_tokens, cache.num_kv_heads, cache.head_dim, cache.num_layers, 0.5, 7
    exact = state(lambda l, kv, h: (src(l, kv, h), np.eye(d)))
    shifted = state(lambda l, kv, h: (np.hstack([src(l, kv, h), np.full((T, 1), c)]),
                                      np.vstack([np.eye(d), np.ones((1, d))])))
    dist = O.gate_distances(cache, item, [exact, shifted], k)
    # Eq. 9: sqrt of the sum over layers, heads, the k prefix rows and d features of c^2
    assert np.allclose(dist, [0.0, c * math.sqrt(L * H * k * d)], atol=1e-12)
    # Eq. 10-11 with two anchors: binary entropy of g_0 = 1 / (1 + e^{-d_1})
    g, h, _ = O.gate(dist, tau=1.0)
    p = 1.0 / (1.0 + math.exp(-dist[1]))
    assert np.allclose(g, [p, 1 - p])
    assert math.isclose(h, -(p * math.log2(p) + (1 - p) * math.log2(1 - p)))
    assert O.gate(dist, tau=h)[2] and not O.gate(dist, tau=h * 0.999)[2]
    # equal distances: uniform weights, entropy 1 (accepted only with tau >= 1); fewer than two anchors: dense
    g, h, acc = O.gate(np.array([3.0, 3.0, 3.0]), tau=0.99)
    assert np.allclose(g, 1 / 3) and math.isclose(h, 1.0) and not acc
    assert O.gate(np.array([0.0]), tau=1.0)[2] is False and O.gate(np.zeros(0), tau=1.0)[2] is False


def test_anchor_pool_evicts_least_used_of_five_oldest():
    """A scripted history worked out by hand from the rule (least frequently used among the five oldest, the older
    one on equal counts)."""
    pool = O.AnchorPool(6)
    for i in range(6):
        assert pool.insert(i, 10 + i) == (i, None)
    pool.record_use([0, 0, 1, 2, 3, 3, 3, 4])
    # five oldest: slots 0-4 with uses 2, 1, 1, 3, 1 -> slot 1 (oldest of the three with one use)
    assert pool.insert(6, 20) == (1, 1)
    # five oldest now slots 0, 2, 3, 4, 5 with uses 2, 1, 3, 1, 0 -> slot 5
    assert pool.insert(7, 30) == (5, 5)
    # five oldest now slots 0, 2, 3, 4, 1 (id 6, no use) with uses 2, 1, 3, 1, 0 -> slot 1
    assert pool.insert(8, 5) == (1, 6)
    # eligibility by stored length: ids 0, 2, 3, 4 have lengths 10, 12, 13, 14; id 7: 30; id 8: 5
    assert pool.eligible(12) == [2, 3, 4, 5] and pool.eligible(31) == [] and len(pool.eligible(0)) == 6


# ----------------------------------------------------------------------- rotary positional alignment (Appendix A.3)

def _llama_inv_freq(d, theta=500000.0):
    return theta ** (-np.arange(0, d, 2, dtype=np.float64) / d)


@pytest.mark.parametrize("style", ["half", "pairs"])
def test_rope_rotation_matches_complex_multiplication(style):
    """The rotation of each feature pair is multiplication of the complex number a + ib by e^{i theta}."""
    rng = np.random.default_rng(31)
    d, T = 16, 5
    rope = O.Rope(_llama_inv_freq(d, 10000.0), style)
    x = rng.standard_normal((T, d))
    pos = np.array([0, 3, 17, 4096, 32767])
    got = O.rope_rotate(x, pos, rope)
    if style == "half":
        z = x[:, : d // 2] + 1j * x[:, d // 2:]
    else:
        z = x[:, 0::2] + 1j * x[:, 1::2]
    w = z * np.exp(1j * np.outer(pos, rope.inv_freq))
    ref = np.hstack([w.real, w.imag]) if style == "half" else np.stack([w.real, w.imag], axis=-1).reshape(T, d)
    assert np.allclose(got, ref, rtol=0, atol=1e-12)


def test_rope_worked_example():
    """Hand-worked: d = 4, inv_freq (pi/2, pi), row (1, 2, 3, 4) at position 1.  Rotate-half pairs (1, 3) by pi/2 ->
    (-3, 1) and (2, 4) by pi -> (-2, -4); adjacent pairs (1, 2) by pi/2 -> (-2, 1) and (3, 4) by pi -> (-3, -4)."""
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    inv = np.array([math.pi / 2, math.pi])
    assert np.allclose(O.rope_rotate(x, 1, O.Rope(inv, "half")), [[-3.0, -2.0, 1.0, -4.0]], atol=1e-15)
    assert np.allclose(O.rope_rotate(x, 1, O.Rope(inv, "pairs")), [[-2.0, 1.0, -3.0, -4.0]], atol=1e-15)


def test_rope_group_and_relative_position_properties():
    rng = np.random.default_rng(32)
    d = 32
    rope = O.Rope(_llama_inv_freq(d), "half")
    q, k = rng.standard_normal((2, d))
    # R(a) R(b) = R(a + b), R(0) = I, norms preserved
    assert np.allclose(O.rope_rotate(O.rope_rotate(k, 700, rope), 1234, rope), O.rope_rotate(k, 1934, rope))
    assert np.array_equal(O.rope_rotate(k, 0, rope), k)
    assert math.isclose(np.linalg.norm(O.rope_rotate(k, 31000, rope)), np.linalg.norm(k))
    # attention logits depend only on the relative position: <R(p) q, R(p') k> = <R(p - p') q, k>
    lhs = O.rope_rotate(q, 9000, rope) @ O.rope_rotate(k, 8000, rope)
    assert math.isclose(lhs, O.rope_rotate(q, 1000, rope) @ k, rel_tol=1e-9)


def _rope_cache(rng, T, H, d, L, bs, dtype, rope):
    nb = 2 * (-(-T // bs))
    mk = lambda: [O.to_storage(rng.standard_normal((nb, bs, H, d)), dtype) for _ in range(L)]
    return O.Cache(dtype, bs, mk(), mk(), rope)


def test_apply_with_rope_reduces_to_plain_apply_and_rotates_keys_only():
    """At source and target position 0 the rotary apply is the plain apply (R(0) = I); values never rotate; keys
    with a rank-0 state are the source rotated by p_dst - p_src."""
    rng = np.random.default_rng(33)
    T, H, d, L, bs, r, Ts = 10, 2, 8, 2, 4, 3, 7
    rope = O.Rope(_llama_inv_freq(d, 10000.0), "half")
    cache = _rope_cache(rng, T, H, d, L, bs, "f32", rope)
    plain = O.Cache("f32", bs, cache.k, cache.v)
    coef = O.to_storage(rng.standard_normal((L, 2, H, Ts, r)), "f32")
    basis = np.linalg.qr(rng.standard_normal((L * 2 * H, d, r)))[0].transpose(0, 2, 1).reshape(L, 2, H, r, d)
    st = O.State(coef, basis.astype(np.float32), None, "f32")
    dst_off = cache.k[0].shape[0] * bs // 2
    a = O.apply(cache, [O.Item(T, 0, dst_off, None, None, st, 0, 0)])
    b = O.apply(plain, [O.Item(T, 0, dst_off, None, None, st)])
    for x, y in zip(a.k + a.v, b.k + b.v):
        assert np.array_equal(O.to_f64(x, "f32"), O.to_f64(y, "f32"))
    moved = O.apply(cache, [O.Item(T, 0, dst_off, None, None, st, 5, 4000)])
    for x, y in zip(moved.v, b.v):
        assert np.array_equal(x, y)
    zero = O.State(np.zeros((L, 2, H, 0, 0), np.float32), np.zeros((L, 2, H, 0, d), np.float32), None, "f32")
    shifted = O.apply(cache, [O.Item(T, 0, dst_off, None, None, zero, 5, 4000)])
    for layer in range(L):
        for h in range(H):
            src = O.to_f64(O.read_rows(cache, layer, 0, h, None, 0, T), "f32")
            got = O.to_f64(O.read_rows(shifted, layer, 0, h, None, dst_off, T), "f32")
            assert np.allclose(got, O.rope_rotate(src, 3995, rope), rtol=2e-7, atol=1e-7)


@pytest.mark.parametrize("style", ["half", "pairs"])
def test_fit_and_apply_with_rope_recover_canonical_deviation(style):
    """Canonical keys Kc_j = Kc_i + D (D of rank r) stored at different positions, K = R(p) Kc: the rotary fit
    returns D itself (Eq. 12 in canonical coordinates), a fit that ignores the positions does not, and applying the
    fitted state to K_i at p_i with target p_j reproduces K_j."""
    rng = np.random.default_rng(34)
    T, H, d, L, bs, r = 24, 2, 8, 1, 4, 2
    pi, pj = 37, 5000
    rope = O.Rope(_llama_inv_freq(d, 10000.0), style)
    nb = 2 * (-(-T // bs))
    kc = rng.standard_normal((nb * bs // 2, H, d))
    dev = np.stack([rng.standard_normal((T, r)) @ rng.standard_normal((r, d)) for _ in range(H)], axis=1)
    ki = O.rope_rotate(kc[:T], pi, rope)
    kj = O.rope_rotate(kc[:T] + dev, pj, rope)
    pool = np.zeros((nb * bs, H, d))
    pool[:T], pool[nb * bs // 2: nb * bs // 2 + T] = ki, kj
    k = [O.to_storage(pool.reshape(nb, bs, H, d), "f32")]
    v = [O.to_storage(rng.standard_normal((nb, bs, H, d)), "f32")]
    cache = O.Cache("f32", bs, k, v, rope)
    item = O.Item(T, 0, nb * bs // 2, None, None, None, pi, pj)
    states, raw = O.fit(cache, [item], r)
    for h in range(H):
        prod = raw[0][0][0, 0, h] @ raw[0][1][0, 0, h]
        assert np.allclose(prod, dev[:, h], atol=2e-5)
    _, wrong = O.fit(O.Cache("f32", bs, k, v, None), [item], r)
    assert max(np.max(np.abs(wrong[0][0][0, 0, h] @ wrong[0][1][0, 0, h] - dev[:, h])) for h in range(H)) > 0.1
    out = O.apply(cache, [O.Item(T, 0, nb * bs // 2, None, None, states[0], pi, pj)])
    got = O.to_f64(out.k[0], "f32").reshape(nb * bs, H, d)[nb * bs // 2: nb * bs // 2 + T]
    assert np.allclose(got, kj, atol=5e-5)


def test_anchor_distance_with_rope_uses_canonical_source_keys():
    """An anchor whose base reconstructs the canonical source keys exactly is at distance 0 for keys whatever the
    source position; the same anchor compared without re-alignment is not."""
    rng = np.random.default_rng(35)
    T, H, d, L, bs, ps = 8, 2, 6, 1, 4, 321
    rope = O.Rope(_llama_inv_freq(d, 10000.0), "half")
    cache = _rope_cache(rng, T, H, d, L, bs, "f32", rope)
    item = O.Item(T, 0, 0, None, None, None, ps, 0)
    coef = np.zeros((L, 2, H, T, d))
    for kv in range(2):
        for h in range(H):
            rows = O.to_f64(O.read_rows(cache, 0, kv, h, None, 0, T), "f32")
            coef[0, kv, h] = O.rope_rotate(rows, -ps, rope) if kv == 0 else rows
    exact = O.State(O.to_storage(coef, "f32"), np.broadcast_to(np.eye(d), (L, 2, H, d, d)).astype(np.float32),
                    None, "f32")
    dist = O.anchor_distances(cache, item, [exact], T)
    assert np.allclose(dist, 0.0, atol=1e-6)
    plain = O.anchor_distances(O.Cache("f32", bs, cache.k, cache.v), item, [exact], T)
    assert np.all(plain[:, 0] > 0.05) and np.allclose(plain[:, 1], 0.0, atol=1e-6)


# -------------------------------------------------------------- per-layer factorisation (Section 3.3, D = H d)

def _layer_cache(zs, bs=4):
    """A contiguous f32 cache whose layer-0 K and V rows of head h hold zs[h] (T x d); fitted in base mode."""
    H = len(zs)
    T, d = zs[0].shape
    nb = -(-T // bs)
    pool = np.zeros((nb * bs, H, d))
    for h in range(H):
        pool[:T, h] = zs[h]
    k = [O.to_storage(pool.reshape(nb, bs, H, d), "f32")]
    return O.Cache("f32", bs, k, [k[0].copy()]), O.Item(T, 0, 0, None, None)


def test_layer_fit_of_independent_heads_has_the_union_of_their_singular_values():
    """Head deviations with mutually orthogonal left factors: the per-layer SVD of [Z_0 ... Z_{H-1}] has exactly the
    heads' singular values, and rank sum(r_h) reproduces every head."""
    rng = np.random.default_rng(41)
    T, H, d, r = 40, 3, 8, 2
    u = np.linalg.qr(rng.standard_normal((T, H * r)))[0]
    s = [np.array([5.0, 1.5]), np.array([3.0, 0.5]), np.array([4.0, 2.5])]
    zs = [u[:, h * r:(h + 1) * r] * s[h] @ np.linalg.qr(rng.standard_normal((d, r)))[0].T for h in range(H)]
    cache, item = _layer_cache(zs)
    _, raw = O.fit(cache, [item], H * r, mode=O.MODE_BASE, grouping=O.GROUP_LAYER)
    coef, basis, sigma = raw[0]
    assert np.allclose(sigma[0, 0], np.sort(np.concatenate(s))[::-1], rtol=1e-6)
    assert np.allclose(coef[0, 0] @ basis[0, 0], np.hstack(zs), atol=1e-5)


def test_layer_fit_of_a_shared_left_factor_scales_singular_values_by_sqrt_heads():
    """Z_h = U diag(s) V_h^T with orthonormal V_h: [Z_0 ... Z_{H-1}] = U diag(s) [V_0^T ... V_{H-1}^T] and the
    right factor's rows have norm sqrt(H), so the per-layer singular values are sqrt(H) s and rank r is exact."""
    rng = np.random.default_rng(42)
    T, H, d, r = 30, 4, 8, 3
    s = np.array([4.0, 2.0, 1.0])
    u = np.linalg.qr(rng.standard_normal((T, r)))[0]
    zs = [u * s @ np.linalg.qr(rng.standard_normal((d, r)))[0].T for _ in range(H)]
    cache, item = _layer_cache(zs)
    states, raw = O.fit(cache, [item], r, mode=O.MODE_BASE, grouping=O.GROUP_LAYER)
    assert np.allclose(raw[0][2][0, 0], np.sqrt(H) * s, rtol=1e-6)
    st = states[0]
    for h in range(H):
        assert np.allclose(st.coef_f64(0, 0, h) @ st.basis_f64(0, 0, h), zs[h], atol=1e-5)


def test_layer_fit_eckart_young_against_independent_eigensolver():
    rng = np.random.default_rng(43)
    T, H, d, r = 50, 2, 8, 5
    zs = [rng.standard_normal((T, d)) for _ in range(H)]
    cache, item = _layer_cache(zs)
    _, raw = O.fit(cache, [item], r, mode=O.MODE_BASE, grouping=O.GROUP_LAYER)
    z = np.hstack([O.to_f64(O.read_rows(cache, 0, 0, h, None, 0, T), "f32") for h in range(H)])
    lam = np.linalg.eigvalsh(z.T @ z)[::-1]  # LAPACK's symmetric eigensolver, not the SVD
    res = np.linalg.norm(z - raw[0][0][0, 0] @ raw[0][1][0, 0]) ** 2
    assert math.isclose(res, lam[r:].sum(), rel_tol=1e-9)
    assert np.allclose(raw[0][2][0, 0] ** 2, lam[:r], rtol=1e-9)


def test_apply_with_a_layer_state_uses_each_heads_columns():
    """Brute force: head h of the corrected cache is C_src[h] + A B[:, h d : (h + 1) d], element by element."""
    rng = np.random.default_rng(44)
    T, H, d, r, bs = 6, 2, 4, 2, 4
    nb = 2 * (-(-T // bs))
    k = [O.to_storage(rng.standard_normal((nb, bs, H, d)), "f32")]
    v = [O.to_storage(rng.standard_normal((nb, bs, H, d)), "f32")]
    cache = O.Cache("f32", bs, k, v)
    coef = O.to_storage(rng.standard_normal((1, 2, T, r)), "f32")
    basis = rng.standard_normal((1, 2, r, H, d)).astype(np.float32)
    st = O.State(coef, basis, None, "f32", O.GROUP_LAYER)
    dst_off = nb * bs // 2
    out = O.apply(cache, [O.Item(T, 0, dst_off, None, None, st)])
    for kv, pools in ((0, out.k), (1, out.v)):
        for h in range(H):
            for t in range(T):
                for f in range(d):
                    acc = float(O.to_f64((k, v)[kv][0], "f32").reshape(nb * bs, H, d)[t, h, f])
                    for j in range(r):
                        acc += float(O.to_f64(coef[0, kv, t, j], "f32")) * float(basis[0, kv, j, h, f])
                    got = float(O.to_f64(pools[0], "f32").reshape(nb * bs, H, d)[dst_off + t, h, f])
                    assert math.isclose(got, acc, rel_tol=1e-6, abs_tol=1e-6)
