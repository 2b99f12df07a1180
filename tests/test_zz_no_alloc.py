"""kvc_gate_distances_noalloc (partial sums in the library's static device scratch) against kvc_gate_distances (a
caller workspace) and the oracle's Eq. 9 distances: two calls in a row on the same inputs, the second one smaller
than the first, so a result can not come from the previous call's scratch contents."""
import numpy as np
import pytest
import torch

from oracle import kvc_oracle as O
from paper_2609_34060_amd import kvc, synth
from tests import helpers as Hp

pytestmark = pytest.mark.gpu


def _case(name, layers, T, ranks, **over):
    w = synth.WORKLOADS[name].with_(num_layers=layers, seq_tokens=(T,), **over)
    pc = synth.build_paged(w, device="cuda", num_output_agents=1)
    sdt = synth.storage_dtype(w)
    bases = []
    for v, r in enumerate(ranks):
        scale = (0.1 + 0.9 * v) / np.sqrt(r / w.head_dim)
        c, b, _ = synth.random_state(layers, w.num_kv_heads, w.head_dim, T, r, sdt, "cuda", 8, v, coef_scale=scale)
        bases.append(kvc.State(c, b))
    src = pc.seqs[(0, 0)]
    tab = None if pc.tables is None else pc.tables[[src.table_row]]
    st = kvc.State.empty(layers, w.num_kv_heads, w.head_dim, 0, 0, sdt, "cuda")
    batch = kvc.Batch([T], [src.offset], [src.offset], [st], tab, tab)
    return w, pc, bases, batch, src, tab


def _oracle(w, pc, bases, src, tab, prefix, layer_end):
    cnp = Hp.oracle_cache(pc.k_pools, pc.v_pools, w.block_size)
    item = O.Item(w.seq_tokens[0], src.offset, src.offset, Hp.table_np(tab, 0), Hp.table_np(tab, 0))
    return O.gate_distances(cnp, item, [Hp.oracle_state(b.coef, b.basis) for b in bases], prefix, 0, layer_end)


@pytest.mark.parametrize("name,ranks,over", [("llama8b_4k", [32] * 6, {}),               # resident bases
                                             ("llama8b_4k", [64, 96, 64, 80, 64, 64], {}),  # one basis at a time
                                             ("tiny", [8, 4, 8, 6, 8, 2], {})])              # float32
def test_gate_noalloc_matches_workspace_call(name, ranks, over):
    w, pc, bases, batch, src, tab = _case(name, 3, 4096 if name != "tiny" else 256, ranks, **over)
    T = w.seq_tokens[0]
    cache = kvc.Cache(pc.k_pools, pc.v_pools)
    # first call: every layer, the whole segment, all anchors; second: one layer, a shorter prefix, fewer anchors
    calls = [(T, 3, len(ranks)), (T // 3 + 5, 1, 3)]
    for prefix, layers, V in calls:
        anchors = kvc.Anchors(bases[:V], T, layers, weights=torch.empty(0, device="cuda"))
        dist_ws = kvc.kvc_gate_distances(cache, batch, anchors, prefix, 0, layers)
        dist_na = torch.full((V,), float("nan"), dtype=torch.float32, device="cuda")
        kvc.kvc_gate_distances_noalloc(cache, batch, anchors, prefix, 0, layers, distances=dist_na)
        torch.cuda.synchronize()
        # same kernels and the same fixed summation order: the two entry points agree bit for bit
        assert torch.equal(dist_na, dist_ws), (dist_na, dist_ws)
        ref = _oracle(w, pc, bases[:V], src, tab, prefix, layers)
        got = dist_na.cpu().numpy().astype(np.float64)
        rel = np.max(np.abs(got - ref) / ref)
        print(f"{name}: prefix {prefix}, {layers} layers, {V} anchors: rel err vs oracle {rel:.2e}")
        assert rel <= 1e-4, (got, ref)
