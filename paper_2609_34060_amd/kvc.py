"""Python binding of libkvc (ctypes): argument marshalling only.

The names mirror the C ABI in include/kvc.h: kvc_fit_state, kvc_apply, kvc_chain, the anchor-pool calls
(kvc_anchor_weights, kvc_apply_anchored, kvc_gate_distances, kvc_gate_decide, kvc_pool_*) and the size queries.  Every step
of the correction runs in the library's HIP kernels; torch only provides device memory and the stream.  Loading
fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvc.so")

KVC_OK, KVC_ERR_NULL_ARG, KVC_ERR_SHAPE, KVC_ERR_DTYPE, KVC_ERR_ALIGN = 0, 1, 2, 3, 4
KVC_ERR_ALIAS, KVC_ERR_WORKSPACE, KVC_ERR_UNSUPPORTED, KVC_ERR_HIP, KVC_ERR_TOO_LARGE = 5, 6, 7, 8, 9
KVC_NOALLOC_SCRATCH_BYTES = 2 << 20
KVC_F32, KVC_BF16 = 0, 1
KVC_FIT_DELTA, KVC_FIT_BASE = 0, 1
KVC_ROPE_NONE, KVC_ROPE_HALF, KVC_ROPE_PAIRS = 0, 1, 2
KVC_GROUP_HEAD, KVC_GROUP_LAYER = 0, 1
KVC_MAX_RANK = 128
KVC_MAX_ANCHORS = 16

EXPORTED = ["kvc_version", "kvc_status_str", "kvc_last_hip_error", "kvc_item_scratch_bytes", "kvc_state_bytes",
            "kvc_layer_state_bytes", "kvc_dense_bytes",
            "kvc_apply", "kvc_fit_workspace_bytes", "kvc_fit_state", "kvc_chain_workspace_bytes", "kvc_chain",
            "kvc_anchor_weights", "kvc_apply_anchored", "kvc_gate_workspace_bytes", "kvc_gate_distances",
            "kvc_gate_distances_noalloc",
            "kvc_gate_decide", "kvc_pool_create", "kvc_pool_destroy", "kvc_pool_insert", "kvc_pool_record_use",
            "kvc_pool_eligible", "kvc_pool_slot"]


class KvcError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_str(status)} (status {status})")
        self.status = status


class kvc_cache(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32), ("num_blocks", ctypes.c_int32),
                ("block_stride", ctypes.c_int64), ("token_stride", ctypes.c_int64), ("head_stride", ctypes.c_int64),
                ("k_layers", ctypes.POINTER(ctypes.c_void_p)), ("v_layers", ctypes.POINTER(ctypes.c_void_p)),
                ("rope_style", ctypes.c_int32), ("rope_reserved", ctypes.c_int32),
                ("rope_inv_freq", ctypes.POINTER(ctypes.c_double))]


class kvc_state(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("num_tokens", ctypes.c_int32), ("rank", ctypes.c_int32), ("coef_dtype", ctypes.c_int),
                ("grouping", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("coef", ctypes.c_void_p), ("basis", ctypes.c_void_p), ("sigma", ctypes.c_void_p)]


class kvc_item(ctypes.Structure):
    _fields_ = [("num_tokens", ctypes.c_int32), ("src_offset", ctypes.c_int32), ("dst_offset", ctypes.c_int32),
                ("src_position", ctypes.c_int32), ("dst_position", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("state", kvc_state)]


class kvc_batch(ctypes.Structure):
    _fields_ = [("num_items", ctypes.c_int32), ("max_blocks", ctypes.c_int32),
                ("items", ctypes.POINTER(kvc_item)), ("item_scratch", ctypes.c_void_p),
                ("src_tables", ctypes.c_void_p), ("dst_tables", ctypes.c_void_p)]


class kvc_anchors(ctypes.Structure):
    _fields_ = [("num_anchors", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("states", ctypes.POINTER(kvc_state)), ("weights", ctypes.c_void_p)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libkvc.so (built by build.py).  Raises if it is missing: there is no fallback path."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2609_34060_amd/build.py (hipcc, gfx950)")
    lib = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    lib.kvc_version.restype = i32
    lib.kvc_status_str.restype = ctypes.c_char_p
    lib.kvc_status_str.argtypes = [ctypes.c_int]
    lib.kvc_last_hip_error.restype = i32
    lib.kvc_item_scratch_bytes.restype = sz
    lib.kvc_item_scratch_bytes.argtypes = [i32]
    lib.kvc_state_bytes.restype = sz
    lib.kvc_state_bytes.argtypes = [i32, i32, i32, i32, i32, ctypes.c_int]
    lib.kvc_layer_state_bytes.restype = sz
    lib.kvc_layer_state_bytes.argtypes = [i32, i32, i32, i32, i32, ctypes.c_int]
    lib.kvc_dense_bytes.restype = sz
    lib.kvc_dense_bytes.argtypes = [i32, i32, i32, i32, ctypes.c_int]
    lib.kvc_apply.restype = ctypes.c_int
    lib.kvc_apply.argtypes = [ctypes.POINTER(kvc_cache), ctypes.POINTER(kvc_batch), i32, i32, vp]
    lib.kvc_fit_workspace_bytes.restype = sz
    lib.kvc_fit_workspace_bytes.argtypes = [ctypes.POINTER(kvc_cache), ctypes.POINTER(kvc_batch), i32, i32]
    lib.kvc_fit_state.restype = ctypes.c_int
    lib.kvc_fit_state.argtypes = [ctypes.POINTER(kvc_cache), ctypes.POINTER(kvc_batch), i32, i32, ctypes.c_int,
                                  vp, sz, vp]
    lib.kvc_chain_workspace_bytes.restype = sz
    lib.kvc_chain_workspace_bytes.argtypes = [ctypes.POINTER(kvc_state)] * 3 + [i32, i32]
    lib.kvc_chain.restype = ctypes.c_int
    lib.kvc_chain.argtypes = [ctypes.POINTER(kvc_state)] * 3 + [i32, i32, vp, sz, vp]
    pc, pb, pa = ctypes.POINTER(kvc_cache), ctypes.POINTER(kvc_batch), ctypes.POINTER(kvc_anchors)
    f32, i64 = ctypes.c_float, ctypes.c_int64
    lib.kvc_anchor_weights.restype = ctypes.c_int
    lib.kvc_anchor_weights.argtypes = [pc, pb, pa, i32, i32, f32, vp]
    lib.kvc_apply_anchored.restype = ctypes.c_int
    lib.kvc_apply_anchored.argtypes = [pc, pb, pa, i32, i32, vp]
    lib.kvc_gate_workspace_bytes.restype = sz
    lib.kvc_gate_workspace_bytes.argtypes = [pc, pa, i32, i32, i32]
    lib.kvc_gate_distances.restype = ctypes.c_int
    lib.kvc_gate_distances.argtypes = [pc, pb, pa, i32, i32, i32, vp, vp, sz, vp]
    lib.kvc_gate_distances_noalloc.restype = ctypes.c_int
    lib.kvc_gate_distances_noalloc.argtypes = [pc, pb, pa, i32, i32, i32, vp, vp]
    lib.kvc_gate_decide.restype = i32
    lib.kvc_gate_decide.argtypes = [ctypes.POINTER(f32), i32, f32, f32, ctypes.POINTER(f32), ctypes.POINTER(f32)]
    lib.kvc_pool_create.restype = vp
    lib.kvc_pool_create.argtypes = [i32]
    lib.kvc_pool_destroy.restype = None
    lib.kvc_pool_destroy.argtypes = [vp]
    lib.kvc_pool_insert.restype = i32
    lib.kvc_pool_insert.argtypes = [vp, i64, i32, ctypes.POINTER(i64)]
    lib.kvc_pool_record_use.restype = ctypes.c_int
    lib.kvc_pool_record_use.argtypes = [vp, ctypes.POINTER(i32), i32]
    lib.kvc_pool_eligible.restype = i32
    lib.kvc_pool_eligible.argtypes = [vp, i32, ctypes.POINTER(i32)]
    lib.kvc_pool_slot.restype = ctypes.c_int
    lib.kvc_pool_slot.argtypes = [vp, i32, ctypes.POINTER(i64), ctypes.POINTER(i32), ctypes.POINTER(i64)]
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().kvc_status_str(status).decode()


def _check(status: int, what: str) -> None:
    if status != KVC_OK:
        raise KvcError(status, what)


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return KVC_BF16
    if dt == torch.float32:
        return KVC_F32
    raise ValueError(f"unsupported dtype {dt}")


def _stream_handle(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# The library copies a batch's host items (pinned memory) into its device scratch on the call's stream, so the copy
# reads the host bytes only when the stream reaches it.  A Batch passed as a temporary would be freed on return and its
# pinned block handed to the next allocation before that; calls that use the item scratch therefore keep their batch
# alive until an event recorded after the call has completed.
_inflight: list = []


def _hold_until_done(stream, batch: "Batch") -> None:
    if batch._host is None:
        return
    ev = torch.cuda.Event()
    ev.record(torch.cuda.current_stream() if stream is None else stream)
    _inflight[:] = [x for x in _inflight if not x[0].query()]
    _inflight.append((ev, batch))


# ------------------------------------------------------------------------------------------------------------------
# Python-side holders (keep the tensors and ctypes arrays alive for the duration of a call)
# ------------------------------------------------------------------------------------------------------------------

class Cache:
    """kvc_cache over per-layer pools [num_blocks, block_size, num_kv_heads, head_dim] (or any strided view whose
    head_dim is contiguous).  rope_style / rope_inv_freq describe a rotary encoding of the key rows
    (KVC_ROPE_NONE: none)."""

    def __init__(self, k_pools: Sequence[torch.Tensor], v_pools: Sequence[torch.Tensor],
                 strides: Optional[Sequence[int]] = None, rope_style: int = 0,
                 rope_inv_freq: Optional[Sequence[float]] = None):
        assert len(k_pools) == len(v_pools) and len(k_pools) > 0
        p0 = k_pools[0]
        self.k_pools, self.v_pools = list(k_pools), list(v_pools)
        nb, bs, H, d = p0.shape
        if strides is None:
            strides = (p0.stride(0), p0.stride(1), p0.stride(2))
        n = len(k_pools)
        self._k = (ctypes.c_void_p * n)(*[p.data_ptr() for p in k_pools])
        self._v = (ctypes.c_void_p * n)(*[p.data_ptr() for p in v_pools])
        self._inv_freq = None
        if rope_inv_freq is not None:
            self._inv_freq = (ctypes.c_double * len(rope_inv_freq))(*[float(x) for x in rope_inv_freq])
        self.c = kvc_cache(_dtype_code(p0.dtype), n, H, d, bs, nb, strides[0], strides[1], strides[2],
                           ctypes.cast(self._k, ctypes.POINTER(ctypes.c_void_p)),
                           ctypes.cast(self._v, ctypes.POINTER(ctypes.c_void_p)), int(rope_style), 0,
                           None if self._inv_freq is None
                           else ctypes.cast(self._inv_freq, ctypes.POINTER(ctypes.c_double)))

    @property
    def num_layers(self):
        return self.c.num_layers


class State:
    """Low-rank state tensors.  Per KV head: coef [L, 2, H, T, r], basis [L, 2, H, r, d] float32, sigma [L, 2, H, r].
    Per layer (KVC_GROUP_LAYER, recognised by a 4-d coef): coef [L, 2, T, r], basis [L, 2, r, H, d] float32 (a row
    of H d features), sigma [L, 2, r]."""

    def __init__(self, coef: torch.Tensor, basis: torch.Tensor, sigma: Optional[torch.Tensor] = None):
        self.coef, self.basis, self.sigma = coef, basis, sigma
        if coef.dim() == 4:
            L, two, T, r = coef.shape
            assert two == 2 and basis.dim() == 5 and basis.shape[:3] == (L, 2, r)
            H, d, grouping = basis.shape[3], basis.shape[4], KVC_GROUP_LAYER
        else:
            L, two, H, T, r = coef.shape
            assert two == 2 and basis.shape[:4] == (L, 2, H, r)
            d, grouping = basis.shape[-1], KVC_GROUP_HEAD
        self.grouping = grouping
        self.s = kvc_state(L, H, d, T, r, _dtype_code(coef.dtype), grouping, 0,
                           coef.data_ptr() if coef.numel() else None,
                           basis.data_ptr() if basis.numel() else None,
                           sigma.data_ptr() if (sigma is not None and sigma.numel()) else None)

    @staticmethod
    def empty(L: int, H: int, d: int, T: int, rank: int, coef_dtype: torch.dtype, device) -> "State":
        return State(torch.zeros(L, 2, H, T, rank, dtype=coef_dtype, device=device),
                     torch.zeros(L, 2, H, rank, d, dtype=torch.float32, device=device),
                     torch.zeros(L, 2, H, rank, dtype=torch.float32, device=device))

    @staticmethod
    def empty_layer(L: int, H: int, d: int, T: int, rank: int, coef_dtype: torch.dtype, device) -> "State":
        """A per-layer state (one factorisation of each layer's K or V rows, D = H d)."""
        return State(torch.zeros(L, 2, T, rank, dtype=coef_dtype, device=device),
                     torch.zeros(L, 2, rank, H, d, dtype=torch.float32, device=device),
                     torch.zeros(L, 2, rank, dtype=torch.float32, device=device))

    @property
    def num_tokens(self) -> int:
        return self.s.num_tokens

    @property
    def rank(self) -> int:
        return self.s.rank


class Batch:
    """kvc_batch: host items, the device scratch the library copies them into, and the block tables (device int32
    [n, max_blocks] or None).  The host items sit in pinned memory when a GPU is present, so the library's copy runs
    asynchronously on the call's stream; a Batch is not modified after construction."""

    def __init__(self, num_tokens: Sequence[int], src_offsets: Sequence[int], dst_offsets: Sequence[int],
                 states: Sequence[State], src_tables: Optional[torch.Tensor] = None,
                 dst_tables: Optional[torch.Tensor] = None, device=None,
                 src_positions: Optional[Sequence[int]] = None, dst_positions: Optional[Sequence[int]] = None):
        n = len(num_tokens)
        self.states = list(states)
        nbytes = ctypes.sizeof(kvc_item) * max(n, 1)
        self._host = None
        if torch.cuda.is_available():
            self._host = torch.zeros(nbytes, dtype=torch.uint8, pin_memory=True)
            arr = (kvc_item * max(n, 1)).from_address(self._host.data_ptr())
        else:
            arr = (kvc_item * max(n, 1))()
        for i in range(n):
            arr[i].num_tokens = int(num_tokens[i])
            arr[i].src_offset = int(src_offsets[i])
            arr[i].dst_offset = int(dst_offsets[i])
            arr[i].src_position = 0 if src_positions is None else int(src_positions[i])
            arr[i].dst_position = 0 if dst_positions is None else int(dst_positions[i])
            arr[i].reserved = 0
            arr[i].state = states[i].s
        self._items = arr
        device = device if device is not None else (states[0].basis.device if n else "cuda")
        self.item_scratch = torch.empty(kvc_item_scratch_bytes(n), dtype=torch.uint8, device=device) if n else None
        self.src_tables = None if src_tables is None else src_tables.to(torch.int32).contiguous()
        self.dst_tables = None if dst_tables is None else dst_tables.to(torch.int32).contiguous()
        max_blocks = 0
        for t in (self.src_tables, self.dst_tables):
            if t is not None:
                assert t.shape[0] == n
                max_blocks = max(max_blocks, t.shape[1])
        if self.src_tables is not None and self.dst_tables is not None:
            assert self.src_tables.shape[1] == self.dst_tables.shape[1]
        self.b = kvc_batch(n, max_blocks, ctypes.cast(arr, ctypes.POINTER(kvc_item)),
                           self.item_scratch.data_ptr() if n else None,
                           None if self.src_tables is None else self.src_tables.data_ptr(),
                           None if self.dst_tables is None else self.dst_tables.data_ptr())


# ------------------------------------------------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ------------------------------------------------------------------------------------------------------------------

def kvc_version() -> int:
    return load().kvc_version()


def kvc_item_scratch_bytes(num_items: int) -> int:
    return load().kvc_item_scratch_bytes(num_items)


def kvc_state_bytes(L: int, H: int, d: int, T: int, rank: int, coef_dtype: int) -> int:
    return load().kvc_state_bytes(L, H, d, T, rank, coef_dtype)


def kvc_layer_state_bytes(L: int, H: int, d: int, T: int, rank: int, coef_dtype: int) -> int:
    return load().kvc_layer_state_bytes(L, H, d, T, rank, coef_dtype)


def kvc_dense_bytes(L: int, H: int, d: int, T: int, dtype: int) -> int:
    return load().kvc_dense_bytes(L, H, d, T, dtype)


def kvc_apply(cache: Cache, batch: Batch, layer_begin: int = 0, layer_end: Optional[int] = None,
              stream=None) -> None:
    layer_end = cache.num_layers if layer_end is None else layer_end
    st = load().kvc_apply(ctypes.byref(cache.c), ctypes.byref(batch.b), layer_begin, layer_end,
                          _stream_handle(stream))
    _check(st, "kvc_apply")
    _hold_until_done(stream, batch)


def kvc_fit_workspace_bytes(cache: Cache, batch: Batch, layer_begin: int = 0, layer_end: Optional[int] = None) -> int:
    layer_end = cache.num_layers if layer_end is None else layer_end
    return load().kvc_fit_workspace_bytes(ctypes.byref(cache.c), ctypes.byref(batch.b), layer_begin, layer_end)


def kvc_fit_state(cache: Cache, batch: Batch, layer_begin: int = 0, layer_end: Optional[int] = None,
                  mode: int = KVC_FIT_DELTA, workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    layer_end = cache.num_layers if layer_end is None else layer_end
    need = kvc_fit_workspace_bytes(cache, batch, layer_begin, layer_end)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=cache.k_pools[0].device)
    st = load().kvc_fit_state(ctypes.byref(cache.c), ctypes.byref(batch.b), layer_begin, layer_end, mode,
                              ctypes.c_void_p(workspace.data_ptr()), workspace.numel(), _stream_handle(stream))
    _check(st, "kvc_fit_state")
    _hold_until_done(stream, batch)


def kvc_chain_workspace_bytes(first: State, second: State, out: State, layer_begin: int = 0,
                              layer_end: Optional[int] = None) -> int:
    layer_end = first.s.num_layers if layer_end is None else layer_end
    return load().kvc_chain_workspace_bytes(ctypes.byref(first.s), ctypes.byref(second.s), ctypes.byref(out.s),
                                            layer_begin, layer_end)


def kvc_chain(first: State, second: State, out: State, layer_begin: int = 0, layer_end: Optional[int] = None,
              workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    layer_end = first.s.num_layers if layer_end is None else layer_end
    need = kvc_chain_workspace_bytes(first, second, out, layer_begin, layer_end)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=first.basis.device)
    st = load().kvc_chain(ctypes.byref(first.s), ctypes.byref(second.s), ctypes.byref(out.s), layer_begin,
                          layer_end, ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                          _stream_handle(stream))
    _check(st, "kvc_chain")


# ------------------------------------------------------------------------------------------------------------------
# Anchor pool (Section 3.3, Appendix A.3)
# ------------------------------------------------------------------------------------------------------------------

class Anchors:
    """kvc_anchors: the anchors' states (bases or delta corrections) and the weights tensor
    [layers, 2, num_tokens, V] float32 (allocated here when not given)."""

    def __init__(self, states: Sequence[State], num_tokens: int, num_layers: int,
                 weights: Optional[torch.Tensor] = None):
        self.states = list(states)
        V = len(self.states)
        self._arr = (kvc_state * max(V, 1))(*[st.s for st in self.states])
        if weights is None and V:
            weights = torch.empty(num_layers, 2, num_tokens, V, dtype=torch.float32,
                                  device=self.states[0].basis.device)
        self.weights = weights
        self.a = kvc_anchors(V, num_tokens, ctypes.cast(self._arr, ctypes.POINTER(kvc_state)),
                             None if weights is None or weights.numel() == 0 else weights.data_ptr())

    def with_states(self, states: Sequence[State]) -> "Anchors":
        """The same weights with other states (the delta corrections after the weights came from the bases)."""
        return Anchors(states, self.a.num_tokens, 0 if self.weights is None else self.weights.shape[0], self.weights)


def kvc_anchor_weights(cache: Cache, batch: Batch, anchors: Anchors, layer_begin: int = 0,
                       layer_end: Optional[int] = None, temperature: float = 1.0, stream=None) -> None:
    layer_end = cache.num_layers if layer_end is None else layer_end
    st = load().kvc_anchor_weights(ctypes.byref(cache.c), ctypes.byref(batch.b), ctypes.byref(anchors.a), layer_begin,
                                   layer_end, float(temperature), _stream_handle(stream))
    _check(st, "kvc_anchor_weights")


def kvc_apply_anchored(cache: Cache, batch: Batch, anchors: Anchors, layer_begin: int = 0,
                       layer_end: Optional[int] = None, stream=None) -> None:
    layer_end = cache.num_layers if layer_end is None else layer_end
    st = load().kvc_apply_anchored(ctypes.byref(cache.c), ctypes.byref(batch.b), ctypes.byref(anchors.a),
                                   layer_begin, layer_end, _stream_handle(stream))
    _check(st, "kvc_apply_anchored")


def kvc_gate_workspace_bytes(cache: Cache, anchors: Anchors, prefix: int, layer_begin: int = 0,
                             layer_end: Optional[int] = None) -> int:
    layer_end = cache.num_layers if layer_end is None else layer_end
    return load().kvc_gate_workspace_bytes(ctypes.byref(cache.c), ctypes.byref(anchors.a), prefix, layer_begin,
                                           layer_end)


def kvc_gate_distances(cache: Cache, batch: Batch, anchors: Anchors, prefix: int, layer_begin: int = 0,
                       layer_end: Optional[int] = None, distances: Optional[torch.Tensor] = None,
                       workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    layer_end = cache.num_layers if layer_end is None else layer_end
    dev = cache.k_pools[0].device
    if distances is None:
        distances = torch.empty(len(anchors.states), dtype=torch.float32, device=dev)
    need = kvc_gate_workspace_bytes(cache, anchors, prefix, layer_begin, layer_end)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = load().kvc_gate_distances(ctypes.byref(cache.c), ctypes.byref(batch.b), ctypes.byref(anchors.a), prefix,
                                   layer_begin, layer_end, ctypes.c_void_p(distances.data_ptr()),
                                   ctypes.c_void_p(workspace.data_ptr()), workspace.numel(), _stream_handle(stream))
    _check(st, "kvc_gate_distances")
    return distances


def kvc_gate_distances_noalloc(cache: Cache, batch: Batch, anchors: Anchors, prefix: int, layer_begin: int = 0,
                               layer_end: Optional[int] = None, distances: Optional[torch.Tensor] = None,
                               stream=None) -> torch.Tensor:
    """kvc_gate_distances with the library's static scratch instead of a workspace: `distances` (float32 [V], on the
    device) must be passed by a caller that cannot allocate; it is allocated here only when omitted."""
    layer_end = cache.num_layers if layer_end is None else layer_end
    if distances is None:
        distances = torch.empty(len(anchors.states), dtype=torch.float32, device=cache.k_pools[0].device)
    st = load().kvc_gate_distances_noalloc(ctypes.byref(cache.c), ctypes.byref(batch.b), ctypes.byref(anchors.a),
                                           prefix, layer_begin, layer_end, ctypes.c_void_p(distances.data_ptr()),
                                           _stream_handle(stream))
    _check(st, "kvc_gate_distances_noalloc")
    return distances


def kvc_gate_decide(distances: Sequence[float], tau: float, temperature: float = 1.0):
    """Returns (accept, gate weights, normalised entropy) of Eq. 10-11 for host distances."""
    n = len(distances)
    d = (ctypes.c_float * max(n, 1))(*[float(x) for x in distances])
    g = (ctypes.c_float * max(n, 1))()
    h = ctypes.c_float()
    acc = load().kvc_gate_decide(d, n, float(tau), float(temperature), g, ctypes.byref(h))
    return bool(acc), [g[i] for i in range(n)], h.value


class Pool:
    """kvc_pool_*: the anchor bookkeeping of one shared-context slot (host only)."""

    def __init__(self, capacity: int):
        self.p = load().kvc_pool_create(capacity)
        if not self.p:
            raise KvcError(KVC_ERR_SHAPE, "kvc_pool_create")
        self.capacity = capacity

    def __del__(self):
        if getattr(self, "p", None) and _lib is not None:
            _lib.kvc_pool_destroy(self.p)
            self.p = None

    def insert(self, anchor_id: int, length: int):
        ev = ctypes.c_int64()
        slot = load().kvc_pool_insert(self.p, anchor_id, length, ctypes.byref(ev))
        if slot < 0:
            raise KvcError(KVC_ERR_SHAPE, "kvc_pool_insert")
        return slot, (None if ev.value < 0 else ev.value)

    def record_use(self, slots: Sequence[int]) -> None:
        arr = (ctypes.c_int32 * max(len(slots), 1))(*slots)
        _check(load().kvc_pool_record_use(self.p, arr, len(slots)), "kvc_pool_record_use")

    def eligible(self, prefix: int) -> List[int]:
        arr = (ctypes.c_int32 * self.capacity)()
        n = load().kvc_pool_eligible(self.p, prefix, arr)
        return [arr[i] for i in range(n)]

    def slot(self, slot: int):
        aid, length, uses = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
        _check(load().kvc_pool_slot(self.p, slot, ctypes.byref(aid), ctypes.byref(length), ctypes.byref(uses)),
               "kvc_pool_slot")
        return aid.value, length.value, uses.value
