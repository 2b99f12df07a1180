"""Seeded synthetic workloads for the low-rank KV-cache correction path.

This module only draws random inputs and lays them out in paged K/V pools.  It holds none of the correction
arithmetic (no deviation of one cache from another, no factorisation, no correction): the GPU library and the CPU
oracle both read what it produces, and neither is imported here.

Shapes follow the workloads the paper evaluates (Section 4.1): Llama-3.1-8B-shaped caches (32 layers, 8 KV heads,
head_dim 128), a LLaVA-OneVision-7B-shaped language model (28 layers, 4 KV heads, head_dim 128) whose shared context
mixes image and text tokens, shared contexts of 4K to 32K tokens (the serving sweeps of Section 4.3) and a concurrent
batch of requests with lengths spread over 1K-16K tokens.  No dataset is read: base caches are Gaussian and the
cross-agent deviations are built with a known low-rank structure (Section 3.1 observes effective rank below 32).

Per agent edge j the deviation D_j is added to the previous agent's cache (C_j = C_{j-1} + D_j) before rounding to
the storage dtype, so every edge's observed transition (Eq. 12 with identity alignment) is D_j plus storage rounding.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch


# ---------------------------------------------------------------------------------------------------------------
# Workload descriptions
# ---------------------------------------------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload.

    deviation modes:
      "exact"      D = U diag(s) V^T (U, V orthonormal, s ~ U[0.1, 1]) + N(0, noise^2), unscaled.
      "scaled"     as "exact" but multiplied by gamma = 0.25 * sqrt(T d / sum s^2), so that RMS(D) = 0.25.
      "shared"     D_j = W_j V^T with one orthonormal V (d x rank) per (layer, K/V, head) shared by every agent and
                   agent-specific W_j ~ N(0, coef_std^2).
      "vlm"        D = gamma [2 U_img ; U_txt] diag(s) V^T: image rows carry twice the singular values of text rows;
                   gamma gives the text rows RMS 0.25.
    """
    name: str
    num_layers: int
    num_kv_heads: int
    head_dim: int
    seq_tokens: Tuple[int, ...]          # shared tokens of each request
    num_agents: int
    rank: int
    dtype: str                           # "f32" or "bf16"
    block_size: int
    paged: bool                          # shuffled block tables (True) or contiguous rows (False)
    deviation: str
    noise_std: float = 0.0
    coef_std: float = 0.5
    image_tokens: int = 0
    seed: int = 0

    @property
    def num_requests(self) -> int:
        return len(self.seq_tokens)

    @property
    def units_per_layer(self) -> int:
        return 2 * self.num_kv_heads

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _serving_lengths(seed: int, n: int = 64, lo: int = 1024, hi: int = 16384) -> Tuple[int, ...]:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7])))
    return tuple(int(x) for x in rng.integers(lo, hi + 1, size=n))


WORKLOADS: Dict[str, Workload] = {
    # 2 layers, 4 KV heads, head_dim 64, 256 tokens, 2 agents, rank 8, fp32, contiguous rows.
    "tiny": Workload("tiny", 2, 4, 64, (256,), 2, 8, "f32", 16, False, "exact", noise_std=1e-3, seed=1001),
    # Llama-3-8B shapes, 4096 tokens, 4 agents chained, rank 16, bf16 paged.
    "llama8b_4k": Workload("llama8b_4k", 32, 8, 128, (4096,), 4, 16, "bf16", 16, True, "scaled",
                           noise_std=1e-2, seed=1002),
    # Llama-3-8B shapes, 32768 tokens, 8 agents chained, rank 32, shared subspace.
    "llama8b_32k": Workload("llama8b_32k", 32, 8, 128, (32768,), 8, 32, "bf16", 16, True, "shared",
                            coef_std=0.5, seed=1003),
    # Qwen2-7B-shaped language model of a VLM: 1280 image + 2048 text tokens, 6 agents, rank 32.
    "vlm": Workload("vlm", 28, 4, 128, (3328,), 6, 32, "bf16", 16, True, "vlm", image_tokens=1280, seed=1004),
    # 64 concurrent requests x 4 agents, lengths ~ U[1024, 16384], rank 64, one shared block pool.
    "serving": Workload("serving", 32, 8, 128, _serving_lengths(1005), 4, 64, "bf16", 16, True, "scaled",
                        noise_std=1e-2, seed=1005),
}


# ---------------------------------------------------------------------------------------------------------------
# Random pieces
# ---------------------------------------------------------------------------------------------------------------

def derive_seed(*keys: int) -> int:
    """A 63-bit seed from a tuple of integers (numpy SeedSequence hashing)."""
    return int(np.random.SeedSequence([int(k) for k in keys]).generate_state(1, np.uint64)[0]) & ((1 << 63) - 1)


def torch_generator(device, *keys: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(derive_seed(*keys))
    return g


def orthonormal_columns(x: torch.Tensor) -> torch.Tensor:
    """Orthonormalise the columns of x [..., n, k] (n >= k).

    On the CPU this is a float64 Householder QR with diag(R) > 0.  On a GPU the batch is orthonormalised twice by a
    Cholesky factor of x^T x computed on the host in float64 (CholeskyQR2); only plain float32 products run on the
    device."""
    if x.device.type == "cpu":
        q, r = torch.linalg.qr(x.to(torch.float64))
        sign = torch.sign(torch.diagonal(r, dim1=-2, dim2=-1))
        sign[sign == 0] = 1
        return (q * sign.unsqueeze(-2)).to(x.dtype)
    y = x.to(torch.float32)
    for _ in range(2):
        yt = y.transpose(-2, -1).contiguous()
        g = torch.matmul(yt, y).to("cpu", torch.float64)
        lower = torch.linalg.cholesky(g)
        rinv = torch.linalg.inv(lower.transpose(-2, -1))
        y = torch.matmul(y, rinv.to(y.device, torch.float32).contiguous())
    return y


def singular_profile(g: torch.Generator, batch: int, rank: int, device) -> torch.Tensor:
    """s ~ U[0.1, 1], sorted in descending order, [batch, rank] float64 on the CPU side of the generator."""
    s = torch.rand(batch, rank, generator=g, device=device, dtype=torch.float32).to(torch.float64) * 0.9 + 0.1
    return torch.sort(s, dim=-1, descending=True).values


def lowrank_factors(g: torch.Generator, batch: int, rows: int, cols: int, rank: int, device):
    """(U [batch, rows, rank], s [batch, rank], V [batch, cols, rank]) with orthonormal U and V."""
    u = orthonormal_columns(torch.randn(batch, rows, rank, generator=g, device=device))
    v = orthonormal_columns(torch.randn(batch, cols, rank, generator=g, device=device))
    s = singular_profile(g, batch, rank, device)
    return u, s, v


def deviation_batch(w: Workload, g: torch.Generator, batch: int, rows: int, device,
                    shared_v: Optional[torch.Tensor] = None, dtype=torch.float32) -> torch.Tensor:
    """Deviation D [batch, rows, d] for one agent edge of `batch` independent units (see Workload)."""
    d, r = w.head_dim, w.rank
    if w.deviation in ("exact", "scaled"):
        u, s, v = lowrank_factors(g, batch, rows, d, r, device)
        if w.deviation == "scaled":
            gamma = 0.25 * torch.sqrt(rows * d / (s * s).sum(-1, keepdim=True))
            s = s * gamma
        us = u.to(dtype) * s.to(device, dtype).unsqueeze(-2)
        dev = torch.matmul(us, v.to(dtype).transpose(-2, -1).contiguous())
    elif w.deviation == "shared":
        assert shared_v is not None
        coef = torch.randn(batch, rows, r, generator=g, device=device, dtype=torch.float32).to(dtype) * w.coef_std
        dev = torch.matmul(coef, shared_v.to(device, dtype).transpose(-2, -1).contiguous())
    elif w.deviation == "vlm":
        ni = min(w.image_tokens, rows)
        nt = rows - ni
        u_img = orthonormal_columns(torch.randn(batch, ni, r, generator=g, device=device)).to(dtype)
        u_txt = orthonormal_columns(torch.randn(batch, nt, r, generator=g, device=device)).to(dtype)
        v = orthonormal_columns(torch.randn(batch, d, r, generator=g, device=device)).to(dtype)
        s = singular_profile(g, batch, r, device)
        gamma = 0.25 * torch.sqrt(nt * d / (s * s).sum(-1, keepdim=True))
        s = (s * gamma).to(device, dtype).unsqueeze(-2)
        u = torch.cat([2.0 * u_img, u_txt], dim=-2)
        dev = torch.matmul(u * s, v.transpose(-2, -1).contiguous())
    else:
        raise ValueError(w.deviation)
    if w.noise_std > 0:
        dev = dev + w.noise_std * torch.randn(batch, rows, d, generator=g, device=device,
                                              dtype=torch.float32).to(dtype)
    return dev


# ---------------------------------------------------------------------------------------------------------------
# Paged pools
# ---------------------------------------------------------------------------------------------------------------

@dataclasses.dataclass
class Sequence_:
    request: int
    agent: int
    num_tokens: int
    offset: int          # row of token 0 inside the block sequence (table) or the pool (contiguous)
    table_row: int       # row in `tables` (paged) or -1


@dataclasses.dataclass
class PagedCaches:
    """Every sequence of a workload stored in one K pool and one V pool per layer.

    Pools are torch tensors [num_blocks, block_size, num_kv_heads, head_dim] (the layout one serving engine keeps
    per layer); `tables` is int32 [num_sequences, max_blocks] of physical block ids (paged) or None (contiguous)."""
    workload: Workload
    layers: List[int]
    k_pools: List[torch.Tensor]
    v_pools: List[torch.Tensor]
    tables: Optional[torch.Tensor]
    max_blocks: int
    num_blocks: int
    seqs: Dict[Tuple[int, int], Sequence_]      # (request, agent) -> sequence; agent -1 = output slot of agent j

    def seq(self, request: int, agent: int) -> Sequence_:
        return self.seqs[(request, agent)]


def storage_dtype(w: Workload) -> torch.dtype:
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def plan_blocks(w: Workload, num_output_agents: int, lead_slots: Sequence[int] = (), seed_extra: int = 0):
    """Assign blocks to every (request, agent) ground-truth sequence and to `num_output_agents` output sequences
    per request.  Returns (seqs, num_blocks, max_blocks, table np.int32 or None)."""
    bs = w.block_size
    names: List[Tuple[int, int]] = []
    for q in range(w.num_requests):
        for a in range(w.num_agents):
            names.append((q, a))
        for o in range(num_output_agents):
            names.append((q, 100 + o))
    lead = {}
    for i, nm in enumerate(names):
        lead[nm] = int(lead_slots[i % len(lead_slots)]) if lead_slots else 0
    need = {nm: -(-(lead[nm] + w.seq_tokens[nm[0]]) // bs) for nm in names}
    total = sum(need.values())
    max_blocks = max(need.values())
    seqs: Dict[Tuple[int, int], Sequence_] = {}
    if not w.paged:
        start = 0
        for nm in names:
            seqs[nm] = Sequence_(nm[0], nm[1], w.seq_tokens[nm[0]], start * bs + lead[nm], -1)
            start += need[nm]
        return seqs, total, max_blocks, None
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, 11, seed_extra])))
    perm = rng.permutation(total).astype(np.int32)
    table = np.full((len(names), max_blocks), -1, dtype=np.int32)
    pos = 0
    for row, nm in enumerate(names):
        table[row, :need[nm]] = perm[pos:pos + need[nm]]
        pos += need[nm]
        seqs[nm] = Sequence_(nm[0], nm[1], w.seq_tokens[nm[0]], lead[nm], row)
    return seqs, total, max_blocks, table


def _row_index(seq: Sequence_, table: Optional[np.ndarray], bs: int, t: np.ndarray):
    pos = seq.offset + t
    if table is None:
        return pos // bs, pos % bs
    return table[seq.table_row][pos // bs], pos % bs


def build_paged(w: Workload, device="cpu", layers: Optional[Sequence[int]] = None, num_output_agents: int = 0,
                lead_slots: Sequence[int] = (), fill_outputs: float = float("nan")) -> PagedCaches:
    """Generate every agent's cache of `w` (per layer, K and V, KV head) into paged pools on `device`.

    Agent 0 is N(0,1); agent j is agent j-1 plus one deviation (see Workload), all in float32, then rounded once to
    the storage dtype.  Output sequences are filled with `fill_outputs` so unwritten rows are visible."""
    layers = list(range(w.num_layers)) if layers is None else list(layers)
    seqs, nblk, max_blocks, table_np = plan_blocks(w, num_output_agents, lead_slots)
    H, d, bs = w.num_kv_heads, w.head_dim, w.block_size
    sdt = storage_dtype(w)
    k_pools, v_pools = [], []
    tables = None if table_np is None else torch.from_numpy(table_np).to(device)
    for layer in layers:
        pools = []
        for kv in range(2):
            pool = torch.full((nblk, bs, H, d), fill_outputs, dtype=sdt, device=device)
            for q in range(w.num_requests):
                T = w.seq_tokens[q]
                g = torch_generator(device, w.seed, layer, kv, q)
                cur = torch.randn(H, T, d, generator=g, device=device, dtype=torch.float32)
                shared_v = None
                if w.deviation == "shared":
                    shared_v = orthonormal_columns(torch.randn(H, d, w.rank, generator=g, device=device))
                t = np.arange(T)
                for a in range(w.num_agents):
                    if a > 0:
                        cur = cur + deviation_batch(w, g, H, T, device, shared_v=shared_v)
                    blk, slot = _row_index(seqs[(q, a)], table_np, bs, t)
                    bi = torch.from_numpy(np.asarray(blk, dtype=np.int64)).to(device)
                    si = torch.from_numpy(np.asarray(slot, dtype=np.int64)).to(device)
                    pool[bi, si] = cur.transpose(0, 1).to(sdt)
            pools.append(pool)
        k_pools.append(pools[0])
        v_pools.append(pools[1])
    return PagedCaches(w, layers, k_pools, v_pools, tables, max_blocks, nblk, seqs)


# ---------------------------------------------------------------------------------------------------------------
# Random low-rank states (for apply-only and chain parity with identical inputs)
# ---------------------------------------------------------------------------------------------------------------

def random_state(L: int, H: int, d: int, T: int, rank: int, coef_dtype: torch.dtype, device, *keys: int,
                 coef_scale: Optional[float] = None):
    """A state with orthonormal basis rows and Gaussian coefficients (default scale: RMS of A B equal to 0.25).

    Returns (coef [L, 2, H, T, rank] coef_dtype, basis [L, 2, H, rank, d] float32, sigma [L, 2, H, rank] float32);
    sigma is the column norm of coef (descriptive only)."""
    g = torch_generator(device, 77, L, H, d, T, rank, *keys)
    if coef_scale is None:
        coef_scale = 0.25 * math.sqrt(d / max(rank, 1))
    coef = (torch.randn(L, 2, H, T, rank, generator=g, device=device) * coef_scale).to(coef_dtype)
    if rank > 0:
        basis = orthonormal_columns(torch.randn(L * 2 * H, d, rank, generator=g, device=device))
        basis = basis.transpose(-2, -1).contiguous().reshape(L, 2, H, rank, d).to(torch.float32)
    else:
        basis = torch.zeros(L, 2, H, 0, d, device=device)
    sigma = coef.to(torch.float32).norm(dim=-2)
    return coef, basis, sigma
