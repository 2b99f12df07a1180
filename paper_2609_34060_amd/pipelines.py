"""Correction along an agent workflow (Section 3.2), as sequences of library calls.

  chained       the first agent's cache is exact (dense prefill); agent j's cache is materialised from the
                materialised cache of agent j - 1 with the correction Delta_{j<-j-1} fitted on the observed pair
                (Eq. 6 with the source agent cache as reference, applied edge by edge).
  non-chained   every agent's cache, the first one included, is materialised from one context-free reference cache
                with the correction Delta_{j<-ref} fitted against that reference.

Both use kvc_fit_state and kvc_apply only; the factorisation unit is a KV head or a whole layer (KVC_GROUP_HEAD or
KVC_GROUP_LAYER).  Sequences are given as (offset, table) pairs of one paged cache.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import torch

from . import kvc

Seq = Tuple[int, Optional[torch.Tensor]]  # (row offset, block-table row [1, max_blocks] or None)


def _empty_state(cache: kvc.Cache, T: int, rank: int, grouping: int) -> kvc.State:
    c = cache.c
    dt = torch.bfloat16 if c.dtype == kvc.KVC_BF16 else torch.float32
    dev = cache.k_pools[0].device
    if grouping == kvc.KVC_GROUP_LAYER:
        return kvc.State.empty_layer(c.num_layers, c.num_kv_heads, c.head_dim, T, rank, dt, dev)
    return kvc.State.empty(c.num_layers, c.num_kv_heads, c.head_dim, T, rank, dt, dev)


def fit(cache: kvc.Cache, src: Seq, dst: Seq, T: int, rank: int, grouping: int = kvc.KVC_GROUP_HEAD) -> kvc.State:
    """The rank-r state of the observed transition dst - src over T rows (Eq. 12, Eq. 7)."""
    st = _empty_state(cache, T, rank, grouping)
    kvc.kvc_fit_state(cache, kvc.Batch([T], [src[0]], [dst[0]], [st], src[1], dst[1]))
    return st


def apply(cache: kvc.Cache, src: Seq, out: Seq, T: int, state: kvc.State) -> None:
    """out = src + A B (one rounding); a rank-0 state copies the rows."""
    kvc.kvc_apply(cache, kvc.Batch([T], [src[0]], [out[0]], [state], src[1], out[1]))


def chained(cache: kvc.Cache, agents: Sequence[Seq], outs: Sequence[Seq], T: int, rank: int,
            grouping: int = kvc.KVC_GROUP_HEAD) -> None:
    """outs[0] = agents[0] (exact); outs[j] = outs[j - 1] + fit(agents[j - 1] -> agents[j])."""
    apply(cache, agents[0], outs[0], T, _empty_state(cache, 0, 0, kvc.KVC_GROUP_HEAD))
    for j in range(1, len(agents)):
        st = fit(cache, agents[j - 1], agents[j], T, rank, grouping)
        apply(cache, outs[j - 1], outs[j], T, st)


def non_chained(cache: kvc.Cache, reference: Seq, agents: Sequence[Seq], outs: Sequence[Seq], T: int, rank: int,
                grouping: int = kvc.KVC_GROUP_HEAD) -> None:
    """outs[j] = reference + fit(reference -> agents[j]) for every agent."""
    for j in range(len(agents)):
        st = fit(cache, reference, agents[j], T, rank, grouping)
        apply(cache, reference, outs[j], T, st)
