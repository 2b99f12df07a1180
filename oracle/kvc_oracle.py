"""CPU oracle for the low-rank KV-cache correction path of KVCMAS (test infrastructure only).

Only the tests, the smoke check of the package entry file and the cpu_baseline leg of the benchmark may import,
call or execute anything in this directory; the product path never does.  It shares no code with the GPU library:
it reads the same stored bytes and writes its own results.

Everything is plain float64 NumPy, written to be checked against the paper by eye:

  * apply     -- Eq. 4 with the source agent's materialised cache as the reference (Section 3.2, Eq. 6) and a
                 single state (Eq. 8 with V = 1, w = 1): C_hat_j = C_i + A B, rows past the state's coverage copied
                 (Appendix A.3, "Variable Segment Lengths").  One round-to-nearest-even to the storage dtype.
  * fit       -- Eq. 12 observed transition Z = C_j - Align(C_i) (in canonical coordinates for rotary keys) and the
                 rank-r truncated SVD of Eq. 7: A = U_r Sigma_r, B = R_r^T.  Also Z = C_j for a base cache
                 (Section 3.3, Z in {C, Delta}).
  * grouping  -- the factorisation unit: one (layer, K/V, KV head) with D = d, or one (layer, K/V) with all KV heads
                 side by side, D = H d (the paper's per-layer feature dimension, Section 3.3).
  * chain     -- Eq. 6: Delta_{k<-i} = Delta_{k<-j} + Delta_{j<-i}; the composed state is the rank-r truncated SVD
                 (Eq. 7) of the materialised sum A1 B1 + A2 B2.
  * anchors   -- Eq. 8 with V anchors and token-wise weights: interpolation weights from the mean absolute distance
                 of the source cache to each anchor's reconstructed base, softmax with T = 1, weighted sum of the
                 anchors' corrections (Appendix A.3, "Correction Weighting"); the reliability gate of Eq. 9-11 and
                 the anchor pool's insertion / least-frequently-used eviction rule (Appendix A.3).
  * rope      -- positional alignment of the key rows (Section 2.2, Appendix A.3 "Positional Alignment"): keys are
                 compared, fitted and corrected in canonical coordinates (segment token t at position t) and the
                 corrected keys are rotated to their target positions; values are never rotated.
  * metrics   -- normalised Frobenius error (Appendix A.1), effective rank at 90 % of the singular-value energy
                 (Section 3.1, Figure 2 caption), memory accounting O(VNLD) vs O(VNr(L+D)) (Sections 3.1, 3.3).

Readings of the paper taken here (all listed in the design notes): factorisation per (layer, K/V, KV head), or per
(layer, K/V) with the heads side by side;
Align = the rotary re-alignment of the keys (identity for a cache without rotary encoding, or at equal positions); canonical sign = largest-magnitude basis entry positive (lowest index on ties); the state's
coefficients are stored in the cache dtype, bases and singular values in float32.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np


# ------------------------------------------------------------------------------------------------------------------
# Storage conversions (bf16 is carried as uint16 bit patterns)
# ------------------------------------------------------------------------------------------------------------------

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (the top 16 bits of a binary32)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def _f64_to_f32_round_to_odd(x: np.ndarray) -> np.ndarray:
    """binary64 -> binary32 rounded to odd: truncate toward zero, then force the last bit to 1 if inexact.

    Rounding to odd with at least two extra bits followed by a round-to-nearest-even gives the correctly rounded
    result (Boldo and Melquiond, 'Emulation of FMA and correctly rounded sums: proved algorithms using rounding to
    odd', IEEE TC 2008); binary32 keeps 16 bits more than bfloat16."""
    x = np.asarray(x, dtype=np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        y = x.astype(np.float32)
    yd = y.astype(np.float64)
    finite = np.isfinite(x)
    # step toward zero where RNE went away from zero (including overflow to inf for finite x)
    away = finite & (np.abs(yd) > np.abs(x))
    y = np.where(away, np.nextafter(y, np.float32(0)), y)
    inexact = finite & (y.astype(np.float64) != x)
    bits = y.view(np.uint32) | np.where(inexact, np.uint32(1), np.uint32(0))
    return bits.view(np.float32)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round binary64 values once, to nearest-even, to bfloat16 bit patterns (NaN -> quiet NaN, sign kept)."""
    y = _f64_to_f32_round_to_odd(x)
    u = y.view(np.uint32).astype(np.uint64)
    nan = np.isnan(y)
    rounded = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    qnan = (u >> np.uint64(16)) | np.uint64(0x0040)
    return np.where(nan, qnan, rounded).astype(np.uint16)


def f64_to_f32(x: np.ndarray) -> np.ndarray:
    """Round binary64 once, to nearest-even, to binary32 (NumPy's cast is IEEE round-to-nearest-even)."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float64).astype(np.float32)


def to_f64(stored: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits_to_f64(stored) if dtype == "bf16" else np.asarray(stored, dtype=np.float32).astype(np.float64)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    return f64_to_bf16_bits(x) if dtype == "bf16" else f64_to_f32(x)


# ------------------------------------------------------------------------------------------------------------------
# Inputs in the oracle's own terms
# ------------------------------------------------------------------------------------------------------------------

@dataclasses.dataclass
class Rope:
    """Rotary position encoding of the key rows: feature pair i of a key at position p is rotated by the angle
    p * inv_freq[i].  style "half" pairs feature i with i + d/2 (the rotate-half layout of Llama and Qwen models),
    "pairs" pairs 2i with 2i + 1.  inv_freq: float64 [d/2]."""
    inv_freq: np.ndarray
    style: str = "half"

    def pair_index(self, d: int):
        """Feature indices (a, b) of the d/2 rotation pairs."""
        i = np.arange(d // 2)
        return (i, i + d // 2) if self.style == "half" else (2 * i, 2 * i + 1)


def rope_rotate(rows: np.ndarray, position, rope: Rope) -> np.ndarray:
    """Rotate key rows [..., d] to `position` (a scalar, or one position per row): every pair (a, b) becomes
    (a cos th - b sin th, a sin th + b cos th) with th = position * inv_freq[i].  float64 in and out."""
    rows = np.asarray(rows, dtype=np.float64)
    ia, ib = rope.pair_index(rows.shape[-1])
    pos = np.asarray(position, dtype=np.float64)
    theta = (pos[..., None] if pos.ndim else pos) * np.asarray(rope.inv_freq, dtype=np.float64)
    c, s = np.cos(theta), np.sin(theta)
    out = rows.copy()
    a, b = rows[..., ia], rows[..., ib]
    out[..., ia] = a * c - b * s
    out[..., ib] = a * s + b * c
    return out


@dataclasses.dataclass
class Cache:
    """Paged K/V pools: k[layer] and v[layer] are arrays [num_blocks, block_size, num_kv_heads, head_dim] holding
    float32 values or bfloat16 bit patterns (uint16).  `rope` set: the key rows carry rotary position encoding."""
    dtype: str
    block_size: int
    k: List[np.ndarray]
    v: List[np.ndarray]
    rope: Optional[Rope] = None

    def copy(self) -> "Cache":
        return Cache(self.dtype, self.block_size, [a.copy() for a in self.k], [a.copy() for a in self.v], self.rope)

    @property
    def num_layers(self) -> int:
        return len(self.k)

    @property
    def num_kv_heads(self) -> int:
        return self.k[0].shape[2]

    @property
    def head_dim(self) -> int:
        return self.k[0].shape[3]

    def pool(self, layer: int, kv: int) -> np.ndarray:
        return (self.k, self.v)[kv][layer]


GROUP_HEAD = 0   # one factorisation per (layer, K/V, KV head): Z is T x d
GROUP_LAYER = 1  # one per (layer, K/V): Z is T x (H d), every KV head's features side by side (Section 3.3, D)


@dataclasses.dataclass
class State:
    """Low-rank state of one sequence (Eq. 7).  Per KV head (GROUP_HEAD): coef = A (T x r) and basis = B (r x d) per
    (layer, K/V, head), coef [L, 2, H, T, r], basis [L, 2, H, r, d], sigma [L, 2, H, r].  Per layer (GROUP_LAYER): one
    factorisation of the layer's K (or V) rows with D = H d features, coef [L, 2, T, r], basis [L, 2, r, H, d]
    (row k of B is basis[l, kv, k].reshape(H d): head h's features are its columns h d .. h d + d - 1),
    sigma [L, 2, r].  coef in the coefficient dtype (float32 values or bf16 bits), basis and sigma float32."""
    coef: np.ndarray
    basis: np.ndarray
    sigma: Optional[np.ndarray]
    coef_dtype: str
    grouping: int = GROUP_HEAD

    @property
    def num_tokens(self) -> int:
        return self.coef.shape[-2]

    @property
    def rank(self) -> int:
        return self.coef.shape[-1]

    def coef_f64(self, layer: int, kv: int, head: int) -> np.ndarray:
        c = self.coef[layer, kv] if self.grouping == GROUP_LAYER else self.coef[layer, kv, head]
        return to_f64(c, self.coef_dtype)

    def basis_f64(self, layer: int, kv: int, head: int) -> np.ndarray:
        if self.grouping == GROUP_LAYER:
            return self.basis[layer, kv, :, head, :].astype(np.float64)
        return self.basis[layer, kv, head].astype(np.float64)


@dataclasses.dataclass
class Item:
    """One shared segment: rows t < num_tokens read from the src block sequence and written to / compared with the
    dst block sequence.  A table of None maps block index b to physical block b (contiguous rows).  With a rotary
    cache, segment token t sits at position src_position + t in the source agent's context and dst_position + t in
    the target's (canonical coordinates put it at t)."""
    num_tokens: int
    src_offset: int
    dst_offset: int
    src_table: Optional[np.ndarray]
    dst_table: Optional[np.ndarray]
    state: Optional[State] = None
    src_position: int = 0
    dst_position: int = 0


def to_canonical(rows_f64: np.ndarray, cache: "Cache", kv: int, position: int) -> np.ndarray:
    """Key rows of a segment starting at `position` in canonical coordinates (rotated back by `position`); values,
    and keys of a cache without rotary encoding, are returned as they are."""
    if kv == 1 or cache.rope is None:
        return rows_f64
    return rope_rotate(rows_f64, -position, cache.rope)


# ------------------------------------------------------------------------------------------------------------------
# Row addressing (the paged layout a serving engine keeps; Section 4.1 serves through vLLM)
# ------------------------------------------------------------------------------------------------------------------

def row_location(table: Optional[np.ndarray], offset: int, t: np.ndarray, block_size: int):
    """Token t of a block sequence lives at (block, slot): position p = offset + t, block = table[p // bs] (or
    p // bs without a table), slot = p % bs."""
    p = offset + np.asarray(t, dtype=np.int64)
    logical = p // block_size
    block = logical if table is None else np.asarray(table, dtype=np.int64)[logical]
    return block, p % block_size


def read_rows(cache: Cache, layer: int, kv: int, head: int, table, offset: int, num_tokens: int) -> np.ndarray:
    """Stored rows [num_tokens, head_dim] of one (layer, K/V, head) unit, as stored (no conversion)."""
    block, slot = row_location(table, offset, np.arange(num_tokens), cache.block_size)
    return cache.pool(layer, kv)[block, slot, head, :]


def write_rows(cache: Cache, layer: int, kv: int, head: int, table, offset: int, rows: np.ndarray) -> None:
    block, slot = row_location(table, offset, np.arange(rows.shape[0]), cache.block_size)
    cache.pool(layer, kv)[block, slot, head, :] = rows


# ------------------------------------------------------------------------------------------------------------------
# Eq. 7: rank-r truncated SVD with a canonical sign
# ------------------------------------------------------------------------------------------------------------------

def canonical_sign(u: np.ndarray, vt: np.ndarray):
    """Flip each singular pair so that the largest-magnitude entry of the basis row is positive.  Entries within a
    relative 2^-20 of the largest magnitude count as tied and the first of them decides, so that rounding noise
    does not pick the sign.  Singular vectors are unique only up to sign; a fixed convention makes factors
    readable and reproducible (comparisons use products, which do not depend on it)."""
    u = u.copy()
    vt = vt.copy()
    for k in range(vt.shape[0]):
        mag = np.abs(vt[k])
        j = int(np.argmax(mag >= mag.max() * (1.0 - 2.0 ** -20)))
        if vt[k, j] < 0:
            vt[k] = -vt[k]
            u[:, k] = -u[:, k]
    return u, vt


def truncated_svd(z: np.ndarray, rank: int):
    """Eq. 7: Z = U Sigma R^T ~ U_r Sigma_r R_r^T = A B with A = U_r Sigma_r (T x r) and B = R_r^T (r x d).

    Returns (A, B, sigma) in float64.  rank may not exceed min(T, d)."""
    z = np.asarray(z, dtype=np.float64)
    T, d = z.shape
    if rank > min(T, d):
        raise ValueError("rank exceeds min(T, d)")
    if rank == 0:
        return np.zeros((T, 0)), np.zeros((0, d)), np.zeros(0)
    u, s, vt = np.linalg.svd(z, full_matrices=False)      # s is descending
    u, vt = canonical_sign(u[:, :rank], vt[:rank])
    return u * s[:rank], vt, s[:rank].copy()


# ------------------------------------------------------------------------------------------------------------------
# apply: Eq. 4 / Eq. 8 (one state) with the source agent cache as reference, prefix coverage
# ------------------------------------------------------------------------------------------------------------------

def correct_rows(src: np.ndarray, coef: np.ndarray, basis: np.ndarray, dtype: str) -> np.ndarray:
    """C_hat = C_src + A B for the covered rows: one float64 evaluation, one rounding to the storage dtype.

    src: stored rows [T, d]; coef [Ts, r] float64 (Ts <= T); basis [r, d] float64.  Rows t >= Ts are copied bit for
    bit (the source cache is kept where no state covers the row).  A state of rank 0 or with Ts = 0 is a copy."""
    out = np.array(src, copy=True)
    Ts, r = coef.shape
    if Ts == 0 or r == 0:
        return out
    exact = to_f64(src[:Ts], dtype) + coef @ basis
    out[:Ts] = to_storage(exact, dtype)
    return out


def materialise_aligned(src: np.ndarray, corr: np.ndarray, dtype: str, rope: Rope, src_position: int,
                        dst_position: int) -> np.ndarray:
    """Key rows of a rotary cache (Appendix A.3, positional alignment): the source keys are taken to canonical
    coordinates, the canonical correction (float64, covering the first corr.shape[0] rows) is added there, and the
    result is rotated to the target positions, C_hat = R(p_dst) (R(-p_src) C_src + corr), one rounding.  Rows past
    the correction keep the re-aligned source R(p_dst) R(-p_src) C_src; at equal positions they are bit copies."""
    out = np.array(src, copy=True)
    canon = rope_rotate(to_f64(src, dtype), -src_position, rope)
    ts = corr.shape[0]
    canon[:ts] += corr
    n = out.shape[0] if src_position != dst_position else ts
    if n > 0:
        out[:n] = to_storage(rope_rotate(canon[:n], dst_position, rope), dtype)
    return out


def apply(cache: Cache, items: Sequence[Item], layer_begin: int = 0, layer_end: Optional[int] = None) -> Cache:
    """Materialise each item's target cache from its source rows and state; returns a new Cache (src untouched).
    Keys of a rotary cache are corrected in canonical coordinates and rotated to the item's target positions."""
    layer_end = cache.num_layers if layer_end is None else layer_end
    out = cache.copy()
    for it in items:
        st = it.state
        for layer in range(layer_begin, layer_end):
            for kv in range(2):
                for h in range(cache.num_kv_heads):
                    src = read_rows(cache, layer, kv, h, it.src_table, it.src_offset, it.num_tokens)
                    empty = st is None or st.rank == 0
                    if kv == 0 and cache.rope is not None:
                        corr = np.zeros((0, cache.head_dim)) if empty else \
                            st.coef_f64(layer, kv, h) @ st.basis_f64(layer, kv, h)
                        rows = materialise_aligned(src, corr, cache.dtype, cache.rope, it.src_position,
                                                   it.dst_position)
                    elif empty:
                        rows = src.copy()
                    else:
                        rows = correct_rows(src, st.coef_f64(layer, kv, h), st.basis_f64(layer, kv, h), cache.dtype)
                    write_rows(out, layer, kv, h, it.dst_table, it.dst_offset, rows)
    return out


# ------------------------------------------------------------------------------------------------------------------
# fit: Eq. 12 deviation, Eq. 7 factorisation
# ------------------------------------------------------------------------------------------------------------------

MODE_DELTA = 0   # Z = C_dst - C_src (observed transition, Eq. 12)
MODE_BASE = 1    # Z = C_dst (base cache of an anchor, Section 3.3)


def fit_unit(src: Optional[np.ndarray], dst: np.ndarray, dtype: str, rank: int):
    """(A, B, sigma) of one unit: Z = dst - src (or dst alone) in float64 from the stored values, then Eq. 7."""
    z = to_f64(dst, dtype)
    if src is not None:
        z = z - to_f64(src, dtype)
    return truncated_svd(z, rank)


def fit(cache: Cache, items: Sequence[Item], rank: int, coef_dtype: Optional[str] = None, mode: int = MODE_DELTA,
        layer_begin: int = 0, layer_end: Optional[int] = None, state_tokens: Optional[Sequence[int]] = None,
        grouping: int = GROUP_HEAD):
    """A state per item, fitted over its first state_tokens[i] rows (default: all rows).

    grouping GROUP_HEAD factorises every (layer, K/V, KV head) unit; GROUP_LAYER factorises each layer's K (or V)
    rows with all KV heads side by side, Z = [Z_0 ... Z_{H-1}] (T x H d), the paper's per-layer feature dimension.
    Layers outside [layer_begin, layer_end) are left zero.  Coefficients are rounded once to coef_dtype (default:
    the cache dtype), bases and singular values to float32.  Also returns the float64 factors (per unit, or per
    layer with the basis as [r, H d])."""
    layer_end = cache.num_layers if layer_end is None else layer_end
    coef_dtype = cache.dtype if coef_dtype is None else coef_dtype
    L, H, d = cache.num_layers, cache.num_kv_heads, cache.head_dim
    states, raw = [], []
    for i, it in enumerate(items):
        Ts = it.num_tokens if state_tokens is None else int(state_tokens[i])

        def deviation(layer, kv, h):
            # Eq. 12 in canonical coordinates: Z = R(-p_dst) C_dst - R(-p_src) C_src for rotary keys
            z = to_canonical(to_f64(read_rows(cache, layer, kv, h, it.dst_table, it.dst_offset, Ts), cache.dtype),
                             cache, kv, it.dst_position)
            if mode == MODE_DELTA:
                z = z - to_canonical(to_f64(read_rows(cache, layer, kv, h, it.src_table, it.src_offset, Ts),
                                            cache.dtype), cache, kv, it.src_position)
            return z

        if grouping == GROUP_LAYER:
            coef = np.zeros((L, 2, Ts, rank))
            basis = np.zeros((L, 2, rank, H * d))
            sigma = np.zeros((L, 2, rank))
            for layer in range(layer_begin, layer_end):
                for kv in range(2):
                    z = np.hstack([deviation(layer, kv, h) for h in range(H)])
                    coef[layer, kv], basis[layer, kv], sigma[layer, kv] = truncated_svd(z, rank)
            raw.append((coef, basis, sigma))
            states.append(State(to_storage(coef, coef_dtype), f64_to_f32(basis).reshape(L, 2, rank, H, d),
                                f64_to_f32(sigma), coef_dtype, GROUP_LAYER))
            continue
        coef = np.zeros((L, 2, H, Ts, rank))
        basis = np.zeros((L, 2, H, rank, d))
        sigma = np.zeros((L, 2, H, rank))
        for layer in range(layer_begin, layer_end):
            for kv in range(2):
                for h in range(H):
                    a, b, s = truncated_svd(deviation(layer, kv, h), rank)
                    coef[layer, kv, h] = a
                    basis[layer, kv, h] = b
                    sigma[layer, kv, h] = s
        raw.append((coef, basis, sigma))
        states.append(State(to_storage(coef, coef_dtype), f64_to_f32(basis), f64_to_f32(sigma), coef_dtype))
    return states, raw


# ------------------------------------------------------------------------------------------------------------------
# chain: Eq. 6 composition of two consecutive corrections, re-truncated by Eq. 7
# ------------------------------------------------------------------------------------------------------------------

def materialise(state: State, layer: int, kv: int, head: int, num_tokens: Optional[int] = None) -> np.ndarray:
    """A B of one unit in float64, zero-padded to num_tokens rows."""
    a = state.coef_f64(layer, kv, head)
    b = state.basis_f64(layer, kv, head)
    T = a.shape[0] if num_tokens is None else num_tokens
    m = np.zeros((T, b.shape[1]))
    m[:a.shape[0]] = a @ b
    return m


def chain(first: State, second: State, out_rank: int, coef_dtype: Optional[str] = None,
          layer_begin: int = 0, layer_end: Optional[int] = None):
    """State of Delta_{k<-i} from first = Delta_{j<-i} and second = Delta_{k<-j}: the rank-out_rank truncated SVD of
    A1 B1 + A2 B2 (rows beyond a state's coverage are zero).  Returns (State, float64 factors)."""
    L, _, H, _, _ = first.coef.shape
    d = first.basis.shape[-1]
    layer_end = L if layer_end is None else layer_end
    coef_dtype = first.coef_dtype if coef_dtype is None else coef_dtype
    T = max(first.num_tokens, second.num_tokens)
    coef = np.zeros((L, 2, H, T, out_rank))
    basis = np.zeros((L, 2, H, out_rank, d))
    sigma = np.zeros((L, 2, H, out_rank))
    for layer in range(layer_begin, layer_end):
        for kv in range(2):
            for h in range(H):
                m = materialise(first, layer, kv, h, T) + materialise(second, layer, kv, h, T)
                a, b, s = truncated_svd(m, out_rank)
                coef[layer, kv, h], basis[layer, kv, h], sigma[layer, kv, h] = a, b, s
    st = State(to_storage(coef, coef_dtype), f64_to_f32(basis), f64_to_f32(sigma), coef_dtype)
    return st, (coef, basis, sigma)


# ------------------------------------------------------------------------------------------------------------------
# Metrics and accounting
# ------------------------------------------------------------------------------------------------------------------

def normalized_frobenius_error(approx: np.ndarray, exact: np.ndarray) -> float:
    """||C_hat - C||_F / ||C||_F, the reuse-error measure of Appendix A.1."""
    exact = np.asarray(exact, dtype=np.float64)
    return float(np.linalg.norm(np.asarray(approx, dtype=np.float64) - exact) / np.linalg.norm(exact))


def max_relative_error(got: np.ndarray, ref: np.ndarray) -> float:
    """max |got - ref| / max |ref| (normalised infinity norm)."""
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    num = np.max(np.abs(np.asarray(got, dtype=np.float64) - ref)) if ref.size else 0.0
    return float(num / den) if den > 0 else float(num)


def effective_rank(sigma: np.ndarray, energy: float = 0.9) -> int:
    """Smallest k whose leading singular values keep `energy` of sum sigma^2 (Section 3.1, Figure 2 caption)."""
    e = np.asarray(sigma, dtype=np.float64) ** 2
    if e.sum() == 0:
        return 0
    c = np.cumsum(np.sort(e)[::-1]) / e.sum()
    return int(np.searchsorted(c, energy - 1e-15) + 1)


def dense_segment_bytes(num_layers: int, num_kv_heads: int, head_dim: int, num_tokens: int, elem_bytes: int) -> int:
    """Bytes of one full-dimensional K and V tensor set of a segment: L x {K,V} x T x D with D = H d."""
    return num_layers * 2 * num_tokens * num_kv_heads * head_dim * elem_bytes


def lowrank_state_bytes(num_layers: int, num_kv_heads: int, head_dim: int, num_tokens: int, rank: int,
                        coef_bytes: int, with_sigma: bool = True) -> int:
    """Bytes of a low-rank state: per unit A (T x r, coef dtype), B (r x d, float32) and sigma (r, float32)."""
    per_unit = num_tokens * rank * coef_bytes + rank * head_dim * 4 + (rank * 4 if with_sigma else 0)
    return num_layers * 2 * num_kv_heads * per_unit


def full_dimensional_pool_bytes(num_anchors: int, num_consumers: int, num_layers: int, num_kv_heads: int,
                                head_dim: int, num_tokens: int, elem_bytes: int) -> int:
    """O(V N L D) anchor memory of Section 3.1: each anchor keeps one base cache and one correction per consuming
    agent, all full-dimensional."""
    return num_anchors * (1 + num_consumers) * dense_segment_bytes(num_layers, num_kv_heads, head_dim, num_tokens,
                                                                   elem_bytes)


# ------------------------------------------------------------------------------------------------------------------
# Anchored correction: Eq. 8 with V anchors and token-wise weights (Appendix A.3)
# ------------------------------------------------------------------------------------------------------------------

def anchor_distances(cache: Cache, item: Item, bases: Sequence[State], num_tokens: int, layer_begin: int = 0,
                     layer_end: Optional[int] = None) -> np.ndarray:
    """Mean absolute distance of the source cache to each anchor's reconstructed base (Appendix A.3, correction
    weighting), per layer, K/V and token: d[l, kv, t, v] = mean over the layer's K (or V) row -- every KV head and
    feature, the paper's feature dimension D = H d -- of |C_src[t] - (A_v B_v)[t]|.  float64 [nl, 2, T, V]."""
    layer_end = cache.num_layers if layer_end is None else layer_end
    H, d = cache.num_kv_heads, cache.head_dim
    out = np.zeros((layer_end - layer_begin, 2, num_tokens, len(bases)))
    for li, layer in enumerate(range(layer_begin, layer_end)):
        for kv in range(2):
            for v, base in enumerate(bases):
                total = np.zeros(num_tokens)
                for h in range(H):
                    src = to_canonical(to_f64(read_rows(cache, layer, kv, h, item.src_table, item.src_offset,
                                                        num_tokens), cache.dtype), cache, kv, item.src_position)
                    recon = base.coef_f64(layer, kv, h)[:num_tokens] @ base.basis_f64(layer, kv, h)
                    total += np.abs(src - recon).sum(axis=1)
                out[li, kv, :, v] = total / (H * d)
    return out


def softmax_weights(distances: np.ndarray, temperature: float = 1.0) -> np.ndarray:
    """w_v = exp(-d_v / T) / sum_u exp(-d_u / T) over the last axis (Eq. 10 form, T = 1 in the paper); evaluated as
    exp(-(d_v - min_u d_u) / T) / sum, the same quantity without overflow."""
    e = np.exp(-(distances - distances.min(axis=-1, keepdims=True)) / temperature)
    return e / e.sum(axis=-1, keepdims=True)


def apply_anchored(cache: Cache, item: Item, deltas: Sequence[State], weights: np.ndarray, num_tokens: int,
                   layer_begin: int = 0, layer_end: Optional[int] = None) -> Cache:
    """Eq. 8 with token-wise weights: C_hat[t] = C_src[t] + sum_v w[l, kv, t, v] (A_v B_v)[t] for t < num_tokens,
    bit copy for num_tokens <= t < item.num_tokens; one rounding to the storage dtype.  Returns a new Cache."""
    layer_end = cache.num_layers if layer_end is None else layer_end
    out = cache.copy()
    for li, layer in enumerate(range(layer_begin, layer_end)):
        for kv in range(2):
            for h in range(cache.num_kv_heads):
                src = read_rows(cache, layer, kv, h, item.src_table, item.src_offset, item.num_tokens)
                corr = np.zeros((num_tokens, cache.head_dim))
                for v, delta in enumerate(deltas):
                    prod = delta.coef_f64(layer, kv, h)[:num_tokens] @ delta.basis_f64(layer, kv, h)
                    corr += weights[li, kv, :, v][:, None] * prod
                if kv == 0 and cache.rope is not None:
                    rows = materialise_aligned(src, corr, cache.dtype, cache.rope, item.src_position,
                                               item.dst_position)
                else:
                    rows = np.array(src, copy=True)
                    if num_tokens > 0:
                        rows[:num_tokens] = to_storage(to_f64(src[:num_tokens], cache.dtype) + corr, cache.dtype)
                write_rows(out, layer, kv, h, item.dst_table, item.dst_offset, rows)
    return out


# ------------------------------------------------------------------------------------------------------------------
# Reliability gate (Eq. 9-11) and anchor pool updates (Appendix A.3)
# ------------------------------------------------------------------------------------------------------------------

def gate_distances(cache: Cache, item: Item, bases: Sequence[State], prefix: int, layer_begin: int = 0,
                   layer_end: Optional[int] = None) -> np.ndarray:
    """Eq. 9: d_v = (sum over layers of ||V_src[:k] - V_v[:k]||_F^2)^(1/2), value states only, V_v the anchor's
    reconstructed base values (every KV head of the layer's value row).  float64 [V]."""
    layer_end = cache.num_layers if layer_end is None else layer_end
    sq = np.zeros(len(bases))
    for layer in range(layer_begin, layer_end):
        for v, base in enumerate(bases):
            for h in range(cache.num_kv_heads):
                src = to_f64(read_rows(cache, layer, 1, h, item.src_table, item.src_offset, prefix), cache.dtype)
                recon = base.coef_f64(layer, 1, h)[:prefix] @ base.basis_f64(layer, 1, h)
                sq[v] += np.sum((src - recon) ** 2)
    return np.sqrt(sq)


def gate(distances: np.ndarray, tau: float, temperature: float = 1.0):
    """Eq. 10-11: g = softmax(-d / T); normalised entropy H = -sum g log2 g / log2 |A|; the correction is accepted
    when |A| >= 2 and H <= tau (fewer than two compatible anchors mean dense prefill).  Returns (g, H, accept);
    with |A| < 2, H is reported as 1."""
    n = distances.shape[0]
    if n < 2:
        return np.ones(n), 1.0, False
    g = softmax_weights(distances, temperature)
    nz = g[g > 0]
    h = float(-(nz * np.log2(nz)).sum() / np.log2(n))
    return g, h, bool(h <= tau)


class AnchorPool:
    """Anchor bookkeeping of one shared-context slot (Appendix A.3, pool updates): at most `capacity` anchors, each
    with a stored length and a use count.  A new anchor (inserted after a dense prefill) takes a free slot; when the
    pool is full it replaces the least frequently used of the five oldest anchors (the oldest of them on equal
    counts).  Anchors eligible for a comparison prefix k are those whose stored length is at least k."""

    def __init__(self, capacity: int):
        self.capacity = capacity
        self.slots: List[Optional[dict]] = [None] * capacity
        self.clock = 0

    def insert(self, anchor_id: int, length: int) -> tuple:
        """Returns (slot, evicted anchor id or None)."""
        free = [i for i, e in enumerate(self.slots) if e is None]
        evicted = None
        if free:
            slot = free[0]
        else:
            oldest = sorted(range(self.capacity), key=lambda i: self.slots[i]["order"])[:5]
            slot = min(oldest, key=lambda i: (self.slots[i]["uses"], self.slots[i]["order"]))
            evicted = self.slots[slot]["id"]
        self.slots[slot] = {"id": anchor_id, "length": length, "uses": 0, "order": self.clock}
        self.clock += 1
        return slot, evicted

    def record_use(self, slots: Sequence[int]) -> None:
        for i in slots:
            self.slots[i]["uses"] += 1

    def eligible(self, prefix: int) -> List[int]:
        return [i for i, e in enumerate(self.slots) if e is not None and e["length"] >= prefix]
