"""Rotary positional alignment on the GPU against the oracle (Appendix A.3, "Positional Alignment").

Keys of a rotary cache are corrected in canonical coordinates and rotated to the target positions in the same pass
as the correction; rows past the state's coverage carry the re-aligned source (bit copies when source and target
positions agree); values are never rotated.  Inputs: the seeded workloads with a canonical random state and
inverse frequencies of the standard form theta^(-2i/d) (theta 10^4 and 5 x 10^5), both pair layouts, shifts of
either sign and the same position on both sides.  Bar: 1e-5 (float32) / 1e-2 (bfloat16) per slice as for
kvc_apply, bit-exact copies where the positions agree, values bit-identical to the plain apply.
"""
import numpy as np
import pytest
import torch

from oracle import kvc_oracle as O
from paper_2609_34060_amd import kvc, synth
from tests import helpers as Hp

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 1e-2}
HALF, PAIRS = kvc.KVC_ROPE_HALF, kvc.KVC_ROPE_PAIRS


def _case(name, layers):
    w = synth.WORKLOADS[name].with_(num_layers=layers)
    pc = synth.build_paged(w, device="cuda", num_output_agents=1)
    src, dst = pc.seqs[(0, 0)], pc.seqs[(0, 100)]
    tab = (lambda s: None) if pc.tables is None else (lambda s: pc.tables[[s.table_row]])
    return w, pc, src, dst, tab


@pytest.mark.parametrize("name,layers,style,theta,ps,pd,Ts,rank", [
    ("tiny", 2, HALF, 1e4, 0, 0, 200, 8),
    ("tiny", 2, PAIRS, 1e4, 37, 5000, 256, 8),
    ("tiny", 1, HALF, 5e5, 900, 12, 0, 0),
    ("llama8b_4k", 2, HALF, 5e5, 4096, 1000, 3001, 16),
    ("llama8b_4k", 1, PAIRS, 5e5, 100, 100, 1500, 32),
    ("llama8b_4k", 1, HALF, 1e4, 0, 32768, 4096, 48),
])
def test_apply_with_rope_matches_oracle(name, layers, style, theta, ps, pd, Ts, rank):
    w, pc, src, dst, tab = _case(name, layers)
    T, H, d = w.seq_tokens[0], w.num_kv_heads, w.head_dim
    inv = Hp.rope_inv_freq(d, theta)
    sdt = synth.storage_dtype(w)
    coef, basis, _ = synth.random_state(layers, H, d, Ts, rank, sdt, "cuda", 41, ps, pd)
    st = kvc.State(coef.contiguous(), basis.contiguous())
    before = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size, O.Rope(inv, Hp.ROPE_STYLE_NAME[style]))
    cache = kvc.Cache(pc.k_pools, pc.v_pools, rope_style=style, rope_inv_freq=inv)
    batch = kvc.Batch([T], [src.offset], [dst.offset], [st], tab(src), tab(dst), src_positions=[ps],
                      dst_positions=[pd])
    kvc.kvc_apply(cache, batch)
    torch.cuda.synchronize()
    got_k = [Hp.to_np_storage(p) for p in pc.k_pools]
    got_v = [Hp.to_np_storage(p) for p in pc.v_pools]
    # values: the plain apply, bit for bit
    kvc.kvc_apply(kvc.Cache(pc.k_pools, pc.v_pools), batch)
    torch.cuda.synchronize()
    for a, b in zip(got_v, pc.v_pools):
        assert np.array_equal(a, Hp.to_np_storage(b))
    item = O.Item(T, src.offset, dst.offset, Hp.table_np(tab(src), 0), Hp.table_np(tab(dst), 0),
                  Hp.oracle_state(coef, basis), ps, pd)
    ref = O.apply(before, [item])
    got = O.Cache(before.dtype, w.block_size, got_k, got_v, before.rope)
    dt = before.dtype
    worst, teeth = 0.0, 0.0
    for layer in range(layers):
        for h in range(H):
            g = O.read_rows(got, layer, 0, h, item.dst_table, item.dst_offset, T)
            e = O.read_rows(ref, layer, 0, h, item.dst_table, item.dst_offset, T)
            s = O.read_rows(before, layer, 0, h, item.src_table, item.src_offset, T)
            worst = max(worst, O.max_relative_error(O.to_f64(g, dt), O.to_f64(e, dt)))
            teeth = max(teeth, O.max_relative_error(O.to_f64(s, dt), O.to_f64(e, dt)))
            if ps == pd:
                assert np.array_equal(g[Ts:], s[Ts:])  # uncovered rows at equal positions: bit copies
    print(f"{name} style {style} ({ps}->{pd}): key err {worst:.2e} (source vs expected {teeth:.2e})")
    assert worst <= TOL[dt], worst
    if ps != pd or rank > 0:
        assert teeth >= 10 * TOL[dt]
