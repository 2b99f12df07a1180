"""The C ABI without a GPU: the library loads, exports every declared symbol, and rejects bad arguments on the host
before any launch (fake device addresses are never dereferenced: each case fails a host-side check)."""
import ctypes
import os
import re

import pytest

from oracle import kvc_oracle as O
from paper_2609_34060_amd import kvc

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "kvc.h")
FAKE = 0x7F0000001000        # a 4 KiB-aligned address that is only compared, never dereferenced


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvc_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = kvc.load()
    declared = _declared_functions()
    assert set(declared) == set(kvc.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.kvc_version() == 1


def test_status_strings():
    for st in range(10):
        assert kvc.status_str(st)
    assert kvc.status_str(0) == "ok"


def test_memory_accounting_matches_oracle_and_paper_example():
    for (L, H, d, T, r, dt, eb) in [(32, 8, 128, 32768, 32, kvc.KVC_BF16, 2), (2, 4, 64, 256, 8, kvc.KVC_F32, 4),
                                    (28, 4, 128, 3328, 0, kvc.KVC_BF16, 2)]:
        assert kvc.kvc_state_bytes(L, H, d, T, r, dt) == O.lowrank_state_bytes(L, H, d, T, r, eb)
        assert kvc.kvc_dense_bytes(L, H, d, T, dt) == O.dense_segment_bytes(L, H, d, T, eb)
    # per-layer state: per (layer, K/V) T r coefficients, r H d basis floats and r sigmas
    assert kvc.kvc_layer_state_bytes(32, 8, 128, 4096, 32, kvc.KVC_BF16) == 64 * (4096 * 32 * 2 + 32 * 1024 * 4 + 32 * 4)
    # Section 3.1: 20 anchors x (1 base + 4 corrections) of a 4K-token Llama-3.1-8B segment in BF16 = 50 GiB
    assert 20 * (1 + 4) * kvc.kvc_dense_bytes(32, 8, 128, 4096, kvc.KVC_BF16) == 50 * 2 ** 30


class Fixture:
    """A valid-looking bf16 cache/batch description made of fake device addresses."""

    def __init__(self, L=2, H=2, d=128, bs=16, nb=64, T=100, rank=16, n=1):
        self.ptrs_k = (ctypes.c_void_p * L)(*[FAKE + 0x100000 * i for i in range(L)])
        self.ptrs_v = (ctypes.c_void_p * L)(*[FAKE + 0x800000 + 0x100000 * i for i in range(L)])
        self.cache = kvc.kvc_cache(kvc.KVC_BF16, L, H, d, bs, nb, bs * H * d, H * d, d,
                                   ctypes.cast(self.ptrs_k, ctypes.POINTER(ctypes.c_void_p)),
                                   ctypes.cast(self.ptrs_v, ctypes.POINTER(ctypes.c_void_p)))
        self.items = (kvc.kvc_item * n)()
        for i in range(n):
            self.items[i].num_tokens = T
            self.items[i].src_offset = 0
            self.items[i].dst_offset = 512
            self.items[i].state = kvc.kvc_state(L, H, d, T, rank, kvc.KVC_BF16, kvc.KVC_GROUP_HEAD, 0,
                                                FAKE + 0x4000000, FAKE + 0x8000000, None)
        self.batch = kvc.kvc_batch(n, 0, ctypes.cast(self.items, ctypes.POINTER(kvc.kvc_item)), FAKE + 0xC000000,
                                   None, None)

    def apply(self, lb=0, le=None):
        le = self.cache.num_layers if le is None else le
        return kvc.load().kvc_apply(ctypes.byref(self.cache), ctypes.byref(self.batch), lb, le, None)


def _cases():
    def null_cache(f):
        return kvc.load().kvc_apply(None, ctypes.byref(f.batch), 0, 1, None), kvc.KVC_ERR_NULL_ARG

    def null_batch(f):
        return kvc.load().kvc_apply(ctypes.byref(f.cache), None, 0, 1, None), kvc.KVC_ERR_NULL_ARG

    def head_dim(f):
        f.cache.head_dim = 96
        return f.apply(), kvc.KVC_ERR_UNSUPPORTED

    def dtype(f):
        f.cache.dtype = 7
        return f.apply(), kvc.KVC_ERR_DTYPE

    def layer_range(f):
        return f.apply(1, 3), kvc.KVC_ERR_SHAPE

    def stride_align(f):
        f.cache.token_stride = 4          # 8 bytes
        return f.apply(), kvc.KVC_ERR_ALIGN

    def layer_ptr_align(f):
        f.ptrs_v[1] = FAKE + 8
        return f.apply(), kvc.KVC_ERR_ALIGN

    def null_layer(f):
        f.ptrs_k[0] = None
        return f.apply(), kvc.KVC_ERR_NULL_ARG

    def rank_gt_d(f):
        f.cache.head_dim = 64
        for i in range(f.batch.num_items):
            f.items[i].state.head_dim = 64
            f.items[i].state.rank = 65
        return f.apply(), kvc.KVC_ERR_SHAPE

    def rank_gt_max(f):
        f.items[0].state.rank = 129
        return f.apply(), kvc.KVC_ERR_SHAPE

    def state_tokens(f):
        f.items[0].state.num_tokens = f.items[0].num_tokens + 1
        return f.apply(), kvc.KVC_ERR_SHAPE

    def state_shape(f):
        f.items[0].state.num_kv_heads = 3
        return f.apply(), kvc.KVC_ERR_SHAPE

    def coef_dtype(f):
        f.items[0].state.coef_dtype = kvc.KVC_F32
        return f.apply(), kvc.KVC_ERR_DTYPE

    def coef_align(f):
        f.items[0].state.coef = FAKE + 2
        return f.apply(), kvc.KVC_ERR_ALIGN

    def null_coef(f):
        f.items[0].state.coef = None
        return f.apply(), kvc.KVC_ERR_NULL_ARG

    def beyond_pool(f):
        f.items[0].dst_offset = 64 * 16 - 10
        return f.apply(), kvc.KVC_ERR_SHAPE

    def beyond_table(f):
        f.batch.src_tables = FAKE
        f.batch.dst_tables = FAKE + 0x1000
        f.batch.max_blocks = 6             # 96 rows < 100
        return f.apply(), kvc.KVC_ERR_SHAPE

    def same_tables(f):
        f.items[0].dst_offset = 0
        f.batch.src_tables = FAKE
        f.batch.dst_tables = FAKE
        f.batch.max_blocks = 8
        return f.apply(), kvc.KVC_ERR_ALIAS

    def overlap_rows(f):
        f.items[0].dst_offset = 50
        return f.apply(), kvc.KVC_ERR_ALIAS

    def null_item_scratch(f):
        f.batch.item_scratch = None
        return f.apply(), kvc.KVC_ERR_NULL_ARG

    def item_scratch_align(f):
        f.batch.item_scratch = FAKE + 8
        return f.apply(), kvc.KVC_ERR_ALIGN

    def overlap_across_items(f):
        # item 1's destination rows [100, 200) are item 0's source rows [100, 200): a race inside one launch
        f.items[0].src_offset, f.items[0].dst_offset = 100, 300
        f.items[1].src_offset, f.items[1].dst_offset = 500, 100
        return f.apply(), kvc.KVC_ERR_ALIAS

    def overlap_destinations(f):
        f.items[0].src_offset, f.items[0].dst_offset = 0, 300
        f.items[1].src_offset, f.items[1].dst_offset = 120, 350
        return f.apply(), kvc.KVC_ERR_ALIAS

    def reserved(f):
        f.items[0].reserved = 1
        return f.apply(), kvc.KVC_ERR_SHAPE

    def negative_offset(f):
        f.items[0].src_offset = -1
        return f.apply(), kvc.KVC_ERR_SHAPE

    def negative_position(f):
        f.items[0].dst_position = -5
        return f.apply(), kvc.KVC_ERR_SHAPE

    def rope_style(f):
        f.cache.rope_style = 3
        return f.apply(), kvc.KVC_ERR_SHAPE

    def rope_reserved(f):
        f.cache.rope_reserved = 1
        return f.apply(), kvc.KVC_ERR_SHAPE

    def rope_null_freq(f):
        f.cache.rope_style = kvc.KVC_ROPE_HALF
        f.cache.rope_inv_freq = None
        return f.apply(), kvc.KVC_ERR_NULL_ARG

    def grouping_value(f):
        f.items[0].state.grouping = 2
        return f.apply(), kvc.KVC_ERR_SHAPE

    def state_reserved(f):
        f.items[0].state.reserved = 1
        return f.apply(), kvc.KVC_ERR_SHAPE

    def layer_rank_gt_max(f):
        f.items[0].state.grouping = kvc.KVC_GROUP_LAYER   # D = H d = 1024: the cap is KVC_MAX_RANK
        f.items[0].state.rank = 129
        return f.apply(), kvc.KVC_ERR_SHAPE

    def rope_nonfinite_freq(f):
        f.inv = (ctypes.c_double * 64)(*([1.0] * 63 + [float("inf")]))
        f.cache.rope_style = kvc.KVC_ROPE_PAIRS
        f.cache.rope_inv_freq = ctypes.cast(f.inv, ctypes.POINTER(ctypes.c_double))
        return f.apply(), kvc.KVC_ERR_SHAPE

    return [null_cache, null_batch, head_dim, dtype, layer_range, stride_align, layer_ptr_align, null_layer,
            rank_gt_d, rank_gt_max, state_tokens, state_shape, coef_dtype, coef_align, null_coef, beyond_pool,
            beyond_table, same_tables, overlap_rows, null_item_scratch, item_scratch_align, overlap_across_items,
            overlap_destinations, reserved, negative_offset, negative_position,
            rope_style, rope_reserved, rope_null_freq, rope_nonfinite_freq, grouping_value, state_reserved,
            layer_rank_gt_max]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c.__name__)
def test_apply_rejects_bad_arguments_before_launch(case):
    got, expected = case(Fixture(n=2) if case.__name__.startswith("overlap_") else Fixture())
    assert got == expected, (kvc.status_str(got), kvc.status_str(expected))


def test_apply_empty_batch_is_a_noop():
    f = Fixture()
    f.batch.num_items = 0
    assert f.apply() == kvc.KVC_OK
    f = Fixture()
    assert f.apply(1, 1) == kvc.KVC_OK           # an empty layer range is valid (nothing to launch)


class AnchorFixture(Fixture):
    """Fixture plus a valid-looking anchor set of V fake states (no kernel is ever launched by these cases)."""

    def __init__(self, V=3, Ts=80, **kw):
        super().__init__(**kw)
        L, H, d = self.cache.num_layers, self.cache.num_kv_heads, self.cache.head_dim
        self.states = (kvc.kvc_state * V)(*[kvc.kvc_state(L, H, d, 100, 16, kvc.KVC_BF16, kvc.KVC_GROUP_HEAD, 0,
                                                          FAKE + 0x10000000 * (v + 1),
                                                          FAKE + 0x10000000 * (v + 1) + 0x8000000, None)
                                            for v in range(V)])
        self.anchors = kvc.kvc_anchors(V, Ts, ctypes.cast(self.states, ctypes.POINTER(kvc.kvc_state)), FAKE + 0x300000)
        self.ws = (ctypes.c_uint8 * 0)()

    def weights(self, temperature=1.0, lb=0, le=None):
        le = self.cache.num_layers if le is None else le
        return kvc.load().kvc_anchor_weights(ctypes.byref(self.cache), ctypes.byref(self.batch),
                                             ctypes.byref(self.anchors), lb, le, temperature, None)

    def anchored(self):
        return kvc.load().kvc_apply_anchored(ctypes.byref(self.cache), ctypes.byref(self.batch),
                                             ctypes.byref(self.anchors), 0, self.cache.num_layers, None)

    def gate(self, prefix=50, ws=FAKE, ws_bytes=1 << 20, dist=FAKE + 0x200000):
        return kvc.load().kvc_gate_distances(ctypes.byref(self.cache), ctypes.byref(self.batch),
                                             ctypes.byref(self.anchors), prefix, 0, self.cache.num_layers, dist, ws,
                                             ws_bytes, None)


def _anchor_cases():
    def two_items(f):
        f.batch.num_items = 2
        return f.weights(), kvc.KVC_ERR_SHAPE

    def no_anchors(f):
        f.anchors.num_anchors = 0
        return f.anchored(), kvc.KVC_ERR_SHAPE

    def too_many_anchors(f):
        f.anchors.num_anchors = kvc.KVC_MAX_ANCHORS + 1
        return f.weights(), kvc.KVC_ERR_SHAPE

    def null_states(f):
        f.anchors.states = None
        return f.weights(), kvc.KVC_ERR_NULL_ARG

    def null_weights(f):
        f.anchors.weights = None
        return f.anchored(), kvc.KVC_ERR_NULL_ARG

    def weighted_beyond_item(f):
        f.anchors.num_tokens = 101
        return f.weights(), kvc.KVC_ERR_SHAPE

    def anchor_short(f):
        f.states[1].num_tokens = 70
        return f.anchored(), kvc.KVC_ERR_SHAPE

    def anchor_rank0(f):
        f.states[2].rank = 0
        return f.weights(), kvc.KVC_ERR_SHAPE

    def anchor_dtype(f):
        f.states[0].coef_dtype = kvc.KVC_F32
        return f.anchored(), kvc.KVC_ERR_DTYPE

    def anchor_shape(f):
        f.states[0].num_kv_heads = 5
        return f.weights(), kvc.KVC_ERR_SHAPE

    def bad_temperature(f):
        return f.weights(temperature=0.0), kvc.KVC_ERR_SHAPE

    def overlap(f):
        f.items[0].dst_offset = 30
        return f.anchored(), kvc.KVC_ERR_ALIAS

    def gate_prefix(f):
        return f.gate(prefix=81), kvc.KVC_ERR_SHAPE

    def gate_workspace(f):
        return f.gate(ws_bytes=16), kvc.KVC_ERR_WORKSPACE

    def gate_workspace_align(f):
        return f.gate(ws=FAKE + 8), kvc.KVC_ERR_WORKSPACE

    def gate_null_distances(f):
        return f.gate(dist=None), kvc.KVC_ERR_NULL_ARG

    def anchor_per_layer(f):
        f.states[1].grouping = kvc.KVC_GROUP_LAYER
        return f.weights(), kvc.KVC_ERR_UNSUPPORTED

    return [two_items, no_anchors, too_many_anchors, null_states, null_weights, weighted_beyond_item, anchor_short,
            anchor_rank0, anchor_dtype, anchor_shape, bad_temperature, overlap, gate_prefix, gate_workspace,
            gate_workspace_align, gate_null_distances, anchor_per_layer]


@pytest.mark.parametrize("case", _anchor_cases(), ids=lambda c: c.__name__)
def test_anchor_calls_reject_bad_arguments_before_launch(case):
    got, expected = case(AnchorFixture())
    assert got == expected, (kvc.status_str(got), kvc.status_str(expected))


def test_gate_workspace_query():
    f = AnchorFixture(V=4)
    H = f.cache.num_kv_heads
    need = kvc.load().kvc_gate_workspace_bytes(ctypes.byref(f.cache), ctypes.byref(f.anchors), 1200, 0, 2)
    # bf16: one float per (layer, chunk, KV head, anchor) with 512-token chunks (the larger count of the two bf16
    # kernels' 512 and 1024-token chunks), in 256-byte granules
    chunks = max(-(-1200 // 512), -(-1200 // 1024)) * H
    assert need == -(-(2 * chunks * 4 * 4) // 256) * 256


def test_per_layer_states_are_refused_where_unsupported():
    """Chain and anchors take per-head states; the per-layer fit takes D = H d <= 1024 with rank + 16 <= 128 (the
    Rayleigh-Ritz subspace), and rotary keys in a bf16 cache only with power-of-two blocks of at least 8."""
    lib = kvc.load()
    f = Fixture(T=300)
    L, H, d = f.cache.num_layers, f.cache.num_kv_heads, f.cache.head_dim

    def st(T, r, grouping):
        return kvc.kvc_state(L, H, d, T, r, kvc.KVC_BF16, grouping, 0, FAKE + 0x4000000, FAKE + 0x8000000, None)

    a, b, o = st(100, 8, kvc.KVC_GROUP_LAYER), st(100, 8, kvc.KVC_GROUP_HEAD), st(100, 8, kvc.KVC_GROUP_HEAD)
    assert lib.kvc_chain(ctypes.byref(a), ctypes.byref(b), ctypes.byref(o), 0, L, FAKE, 1 << 30,
                         None) == kvc.KVC_ERR_UNSUPPORTED

    def fit():
        return lib.kvc_fit_state(ctypes.byref(f.cache), ctypes.byref(f.batch), 0, L, kvc.KVC_FIT_DELTA, FAKE,
                                 1 << 40, None)

    def ws():
        return lib.kvc_fit_workspace_bytes(ctypes.byref(f.cache), ctypes.byref(f.batch), 0, L)

    f.items[0].state = st(300, 32, kvc.KVC_GROUP_LAYER)
    assert ws() > 0
    f.items[0].state = st(300, 120, kvc.KVC_GROUP_LAYER)   # rank + 16 > 128
    assert ws() == 0 and fit() == kvc.KVC_ERR_UNSUPPORTED
    f.items[0].state = st(300, 32, kvc.KVC_GROUP_LAYER)
    inv = (ctypes.c_double * 64)(*([1e-3] * 64))
    f.cache.rope_style = kvc.KVC_ROPE_HALF
    f.cache.rope_inv_freq = ctypes.cast(inv, ctypes.POINTER(ctypes.c_double))
    assert ws() > 0                    # rotary keys with a power-of-two block size of at least 8
    f.cache.block_size = 12            # bf16 rotary keys need the LDS Gram (power-of-two blocks of at least 8)
    f.cache.block_stride = 12 * H * d
    f.cache.num_blocks = 128
    assert ws() == 0 and fit() == kvc.KVC_ERR_UNSUPPORTED


def test_gate_noalloc_rejects_before_launch():
    """The allocation-free gate takes the same checks as kvc_gate_distances, and a call whose partial sums would not
    fit the static scratch is refused with KVC_ERR_TOO_LARGE before anything is enqueued."""
    lib = kvc.load()

    def call(f, prefix, dist=FAKE + 0x200000):
        return lib.kvc_gate_distances_noalloc(ctypes.byref(f.cache), ctypes.byref(f.batch), ctypes.byref(f.anchors),
                                              prefix, 0, f.cache.num_layers, dist, None)

    f = AnchorFixture()
    assert call(f, 81) == kvc.KVC_ERR_SHAPE
    assert call(f, 50, dist=None) == kvc.KVC_ERR_NULL_ARG
    f.states[0].num_kv_heads = 5
    assert call(f, 50) == kvc.KVC_ERR_SHAPE
    # 128 layers x 64 KV heads x 16 anchors: 4 partials of 4 bytes per (layer, head, anchor) fill 2 MiB exactly
    # (2048 tokens = four 512-token chunks), one more chunk does not fit
    f = AnchorFixture(V=16, Ts=4000, L=128, H=64, T=4096, nb=300)
    for v in range(16):
        f.states[v].num_tokens = 4096
    need = lib.kvc_gate_workspace_bytes(ctypes.byref(f.cache), ctypes.byref(f.anchors), 2048, 0, 128)
    assert need == kvc.KVC_NOALLOC_SCRATCH_BYTES
    assert lib.kvc_gate_workspace_bytes(ctypes.byref(f.cache), ctypes.byref(f.anchors), 2049, 0, 128) > need
    assert call(f, 2049) == kvc.KVC_ERR_TOO_LARGE
    assert "static scratch" in kvc.status_str(kvc.KVC_ERR_TOO_LARGE)
