#!/usr/bin/env python3
"""Benchmark of the online low-rank KV-cache correction path on one MI355X.

One step = one agent edge of the chained workflow over the whole cache (every layer, K and V, KV head):
  fit    S_j = truncated SVD of C_j - C_{j-1}            (kvc_fit_state: Gram, eigensolver, projection)
  chain  T_j = rank-r_out truncation of T_{j-1} + S_j     (kvc_chain)
  apply  C_hat_j = C_0 + T_j, paged gather/correct/scatter (kvc_apply)
Steps cycle over the edges of the workload; inputs are resident in HBM before the timed region.

Printed: one JSON line.  `value` is the corrected-KV throughput of kvc_apply in GB/s (algorithmic bytes: source and
destination rows, coefficients at their stored width, bases) measured with HIP events on the launch stream; fit
throughput is token*layers/s.  `roofline` is kvc_apply against the 8 TB/s HBM peak; `cpu_baseline` is the CPU
oracle timed on a bounded sample of the same workload on this host.  `copy_ceiling` gives, on the same GPU, the
rate of a pure bit copy through the same block tables (kvc_apply with a rank-0 state) and of hand-written copy
kernels (contiguous, read-only, write-only, paged whole blocks in several work orders, paged per-head rows).
`verify_last_apply` checks the output of the last timed apply against the oracle on a sampled layer and KV head;
`configs` times the apply on the 8B/4K, VLM (rotated data sets) and serving-batch shapes.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0


def _apply_bytes(L, H, d, T, r, elem=2, coef_elem=2):
    rows = L * 2 * H * T
    return rows * (2 * d * elem + r * coef_elem) + L * 2 * H * r * d * 4


def _fit_bytes(L, H, d, T, r, elem=2, coef_elem=2):
    # two streaming passes over src and dst rows, coefficients written once
    rows = L * 2 * H * T
    return rows * (2 * 2 * d * elem + r * coef_elem)


def _source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2609_34060_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _traffic(kernel_src_hash):
    """HBM bytes per apply launch from the committed rocprofv3 counter summary, if it was taken on this source."""
    path = os.path.join(ROOT, "profiles", "kvc_apply_llama8b_32k_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_src_hash:
        return None
    return rec.get("traffic_bytes_per_launch")


def _anchored_bytes(L, H, d, T, V, r, elem=2, coef_elem=2):
    # src and dst rows, every anchor's coefficient rows, the weights (read once per unit), the bases
    rows = L * 2 * H * T
    return rows * (2 * d * elem + V * r * coef_elem) + L * 2 * T * V * 4 * H + V * L * 2 * H * r * d * 4


def _weights_bytes(L, H, d, T, V, r, elem=2, coef_elem=2):
    # src rows, every anchor's base coefficient rows, the weights written, the bases
    rows = L * 2 * H * T
    return rows * (d * elem + V * r * coef_elem) + L * 2 * T * V * 4 + V * L * 2 * H * r * d * 4


def anchor_pool_measurement(args, kvc, synth, torch, rope=False):
    """The anchor-pool path of one transfer at the paper's anchor setting (V anchors of rank r on a shared segment):
    token-wise weights from the anchors' bases, the anchored apply of Eq. 8, and the gate distances of Eq. 9.  With
    rope the keys carry a rotary encoding (rotate-half, theta 5e5) and the segment sits at position 2048 in the source
    agent and 6144 in the target, so the weights compare canonical keys and the apply rotates every key row."""
    import numpy as np
    w = synth.WORKLOADS[args.anchor_workload].with_(num_agents=1)
    L, H, d, T, r, V = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0], w.rank, args.anchors
    r = args.anchor_rank
    pc = synth.build_paged(w, device="cuda", num_output_agents=1)
    if rope:
        inv = 500000.0 ** (-np.arange(0, d, 2, dtype=np.float64) / d)
        cache = kvc.Cache(pc.k_pools, pc.v_pools, rope_style=kvc.KVC_ROPE_HALF, rope_inv_freq=inv)
    else:
        cache = kvc.Cache(pc.k_pools, pc.v_pools)
    ps, pd = (2048, 6144) if rope else (0, 0)
    src, dst = pc.seqs[(0, 0)], pc.seqs[(0, 100)]
    tab = lambda s: pc.tables[[s.table_row]]
    sdt = torch.bfloat16

    def states(key, scale_of):
        out = []
        for v in range(V):
            c, b, sg = synth.random_state(L, H, d, T, r, sdt, "cuda", key, v, coef_scale=scale_of(v))
            out.append(kvc.State(c, b, sg))
        return out

    bases = states(11, lambda v: (0.1 + 0.9 * v) / (r / d) ** 0.5)
    deltas = states(12, lambda v: 0.25 * (d / r) ** 0.5)
    anchors = kvc.Anchors(bases, T, L)
    anchors_d = anchors.with_states(deltas)
    empty = kvc.State.empty(L, H, d, 0, 0, sdt, "cuda")
    bw = kvc.Batch([T], [src.offset], [src.offset], [empty], tab(src), tab(src), src_positions=[ps],
                   dst_positions=[ps])
    ba = kvc.Batch([T], [src.offset], [dst.offset], [empty], tab(src), tab(dst), src_positions=[ps],
                   dst_positions=[pd])
    prefix = T
    gws = torch.empty(max(1, kvc.kvc_gate_workspace_bytes(cache, anchors, prefix)), dtype=torch.uint8, device="cuda")
    dist = torch.empty(V, dtype=torch.float32, device="cuda")
    for _ in range(min(args.warmup, 10)):  # the GPU is warm from the main steps
        kvc.kvc_gate_distances(cache, bw, anchors, prefix, distances=dist, workspace=gws)
        kvc.kvc_anchor_weights(cache, bw, anchors)
        kvc.kvc_apply_anchored(cache, ba, anchors_d)
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for k in range(args.steps):
        ev[k][0].record()
        kvc.kvc_gate_distances(cache, bw, anchors, prefix, distances=dist, workspace=gws)
        ev[k][1].record()
        kvc.kvc_anchor_weights(cache, bw, anchors)
        ev[k][2].record()
        kvc.kvc_apply_anchored(cache, ba, anchors_d)
        ev[k][3].record()
    torch.cuda.synchronize()
    gate_ms = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    weights_ms = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    apply_ms = sum(e[2].elapsed_time(e[3]) for e in ev) / args.steps
    ab, wb = _anchored_bytes(L, H, d, T, V, r), _weights_bytes(L, H, d, T, V, r)
    del pc, cache, bases, deltas, anchors, anchors_d
    torch.cuda.empty_cache()
    where = (f"; rotary keys (rotate-half, theta 5e5), segment at position {ps} in the source and {pd} in the target"
             if rope else "")
    return {"workload": f"{w.name}: {L} layers x {H} KV heads x head_dim {d}, {T} shared tokens, {V} anchors of "
                        f"rank {r} (bf16 paged); gate prefix {prefix}{where}",
            "gate_ms": round(gate_ms, 4), "weights_ms": round(weights_ms, 4), "apply_anchored_ms": round(apply_ms, 4),
            "apply_anchored_gbps": round(ab / (apply_ms * 1e-3) / 1e9, 2),
            "apply_anchored_frac": round(ab / (apply_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "apply_anchored_bytes": ab,
            "weights_gbps": round(wb / (weights_ms * 1e-3) / 1e9, 2), "weights_bytes": wb}


def copy_ceiling(args, kvc, torch, cache, w, batch):
    """Copy ceilings on the same GPU, beside the apply: kvc_apply with a rank-0 state (every row a bit copy through
    the same block tables and the same kernel, no coefficients or bases: the paged per-head copy the apply is built
    on) and a contiguous device-to-device copy of the same number of row bytes."""
    L, H, d, T = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0]
    s0 = kvc.State.empty(L, H, d, T, 0, torch.bfloat16, "cuda")
    b0 = batch((0, 0), (0, 100), s0)
    row_bytes = L * 2 * H * T * d * 2  # read once and written once
    src = torch.empty(row_bytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    n = max(5, args.steps // 2)

    def timed(fn):
        for _ in range(2):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        ev[0].record()
        for i in range(n):
            fn()
            ev[i + 1].record()
        torch.cuda.synchronize()
        return sum(ev[i].elapsed_time(ev[i + 1]) for i in range(n)) / n

    paged_ms = timed(lambda: kvc.kvc_apply(cache, b0))
    contig_ms = timed(lambda: dst.copy_(src))
    del src, dst
    torch.cuda.empty_cache()
    pg, cg = 2 * row_bytes / (paged_ms * 1e-3) / 1e9, 2 * row_bytes / (contig_ms * 1e-3) / 1e9
    out = {"bytes": 2 * row_bytes,
           "paged_rank0_apply_ms": round(paged_ms, 4), "paged_rank0_apply_gbps": round(pg, 2),
           "paged_rank0_apply_frac": round(pg / HBM_PEAK_GBPS, 4),
           "torch_copy_ms": round(contig_ms, 4), "torch_copy_gbps": round(cg, 2),
           "torch_copy_frac": round(cg / HBM_PEAK_GBPS, 4)}
    # the hand-written copies of csrc/kvc_copybench.hip: 4 GiB read + 4 GiB written (read-only / write-only 4 GiB)
    from paper_2609_34060_amd import copybench
    out["kernels"] = copybench.ceilings("cuda", gib=4.0, reps=max(5, args.steps // 2))
    torch.cuda.empty_cache()
    return out


def rope_measurement(args, kvc, torch, pc, w, state, batch):
    """The same apply and fit with rotary keys (rotate-half pairs, theta 5 x 10^5 as in Llama-3.1): the segment moves
    from position 0 in the source agent to position 4096 in the target, so every key row is rotated in the pass."""
    import numpy as np
    L, H, d, T, r = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0], w.rank
    inv = 500000.0 ** (-np.arange(0, d, 2, dtype=np.float64) / d)
    cache = kvc.Cache(pc.k_pools, pc.v_pools, rope_style=kvc.KVC_ROPE_HALF, rope_inv_freq=inv)
    src, dst, prev = pc.seqs[(0, 0)], pc.seqs[(0, 100)], pc.seqs[(0, 1)]

    def positioned(a, b, st, pa, pb):
        return kvc.Batch([T], [a.offset], [b.offset], [st], pc.tables[[a.table_row]], pc.tables[[b.table_row]],
                         src_positions=[pa], dst_positions=[pb])

    ab = positioned(src, dst, state, 0, 4096)
    fs = kvc.State.empty(L, H, d, T, r, torch.bfloat16, "cuda")
    fb = positioned(src, prev, fs, 0, 4096)
    ws = torch.empty(kvc.kvc_fit_workspace_bytes(cache, fb), dtype=torch.uint8, device="cuda")

    def timed(fn):
        for _ in range(min(args.warmup, 10)):  # the GPU is warm from the main steps
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps)]
        for k in range(args.steps):
            ev[2 * k].record()
            fn()
            ev[2 * k + 1].record()
        torch.cuda.synchronize()
        return sum(ev[2 * k].elapsed_time(ev[2 * k + 1]) for k in range(args.steps)) / args.steps

    apply_ms = timed(lambda: kvc.kvc_apply(cache, ab))
    fit_ms = timed(lambda: kvc.kvc_fit_state(cache, fb, workspace=ws))
    gbps = _apply_bytes(L, H, d, T, r) / (apply_ms * 1e-3) / 1e9
    del ws, fs
    return {"workload": f"{w.name} with rotary keys (rotate-half, theta 5e5), segment moved from position 0 to 4096",
            "apply_ms": round(apply_ms, 4), "apply_gbps": round(gbps, 2),
            "apply_frac": round(gbps / HBM_PEAK_GBPS, 4), "fit_ms": round(fit_ms, 4),
            "fit_token_layers_per_s": round(T * L / (fit_ms * 1e-3), 1)}


def layer_fit_measurement(args, kvc, torch, pc, w):
    """The paper's per-layer factorisation (every KV head of a layer side by side, D = H d = 1024) of one 8B/32K edge
    at rank 32, and the apply of that state."""
    L, H, d, T = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0]
    r = 32
    cache = kvc.Cache(pc.k_pools, pc.v_pools)
    src, dst, out = pc.seqs[(0, 0)], pc.seqs[(0, 1)], pc.seqs[(0, 100)]
    st = kvc.State.empty_layer(L, H, d, T, r, torch.bfloat16, "cuda")
    fb = kvc.Batch([T], [src.offset], [dst.offset], [st], pc.tables[[src.table_row]], pc.tables[[dst.table_row]])
    ab = kvc.Batch([T], [src.offset], [out.offset], [st], pc.tables[[src.table_row]], pc.tables[[out.table_row]])
    ws = torch.empty(kvc.kvc_fit_workspace_bytes(cache, fb), dtype=torch.uint8, device="cuda")

    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * n)]
        for k in range(n):
            ev[2 * k].record()
            fn()
            ev[2 * k + 1].record()
        torch.cuda.synchronize()
        return sum(ev[2 * k].elapsed_time(ev[2 * k + 1]) for k in range(n)) / n

    fit_ms = timed(lambda: kvc.kvc_fit_state(cache, fb, workspace=ws), max(1, args.steps // 2))
    apply_ms = timed(lambda: kvc.kvc_apply(cache, ab), args.steps)
    # algorithmic bytes: rows read and written, per-layer coefficients (shared by the heads) and the bases
    apply_b = L * 2 * T * (H * d * 2 * 2 + r * 2) + L * 2 * r * H * d * 4
    ws_bytes = ws.numel()
    del ws, st
    return {"workload": f"{w.name}: per-layer factorisation (D = {H * d}) of one edge at rank {r}",
            "fit_ms": round(fit_ms, 3), "fit_token_layers_per_s": round(T * L / (fit_ms * 1e-3), 1),
            "apply_ms": round(apply_ms, 4), "apply_gbps": round(apply_b / (apply_ms * 1e-3) / 1e9, 2),
            "workspace_bytes": ws_bytes}


def chain_study(args, kvc, synth, torch):
    """Reuse error of chained and non-chained correction along a four-agent workflow (the paper's reuse-error
    figure): the generator's agent 0 stands for the context-free reference and agents 1-4 for A0 -> A3, one rank-16
    deviation per edge on the 8B/4K shapes; normalised Frobenius error per agent and per layer (all heads, K and V),
    per KV head and per layer factorisation."""
    import numpy as np
    from paper_2609_34060_amd import pipelines
    w = synth.WORKLOADS["llama8b_4k"].with_(num_agents=5)
    L, H, d, T, r = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0], w.rank
    res = {"workload": f"{w.name} with 5 agents (reference + A0..A3), rank {r} per edge, bf16 paged", "rank": r}
    for gname, grouping in (("head", kvc.KVC_GROUP_HEAD), ("layer", kvc.KVC_GROUP_LAYER)):
        for mode in ("chained", "non_chained"):
            pc = synth.build_paged(w, device="cuda", num_output_agents=4)
            cache = kvc.Cache(pc.k_pools, pc.v_pools)

            def seq(nm):
                s = pc.seqs[nm]
                return (s.offset, pc.tables[[s.table_row]])

            agents = [seq((0, a)) for a in range(5)]
            outs = [seq((0, 100 + j)) for j in range(4)]
            if mode == "chained":
                pipelines.chained(cache, agents[1:], outs, T, r, grouping)
            else:
                pipelines.non_chained(cache, agents[0], agents[1:], outs, T, r, grouping)
            torch.cuda.synchronize()
            per_agent, per_layer = [], np.zeros((4, L))
            for j in range(4):
                num = den = 0.0
                for layer, (kp, vp) in enumerate(zip(pc.k_pools, pc.v_pools)):
                    ln = ld = 0.0
                    for pool in (kp, vp):
                        def rows(nm):
                            s = pc.seqs[nm]
                            t = torch.arange(T, device="cuda") + s.offset
                            blk = pc.tables[s.table_row].long()[t // w.block_size]
                            return pool[blk, t % w.block_size].double()
                        g, e = rows((0, 100 + j)), rows((0, j + 1))
                        ln += float((g - e).square().sum())
                        ld += float(e.square().sum())
                    per_layer[j, layer] = (ln / ld) ** 0.5
                    num, den = num + ln, den + ld
                per_agent.append(round((num / den) ** 0.5, 5))
            res[f"{mode}_{gname}"] = {"per_agent": per_agent,
                                      "per_layer_mean_over_agents": [round(x, 5) for x in per_layer.mean(0)]}
            del pc, cache
            torch.cuda.empty_cache()
    return res


def _progress(msg):
    """One line on stderr as each measurement ends (the JSON line alone goes to stdout)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def _timed_calls(torch, fns, steps, warmup):
    """Mean, p10/p50/p90 milliseconds of fns[k % len(fns)]() over `steps` calls (HIP events on the current stream)."""
    import numpy as np
    for k in range(warmup):
        fns[k % len(fns)]()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    for k in range(steps):
        ev[k][0].record()
        fns[k % len(fns)]()
        ev[k][1].record()
    torch.cuda.synchronize()
    ms = [e[0].elapsed_time(e[1]) for e in ev]
    return sum(ms) / steps, [round(float(v), 4) for v in np.percentile(np.asarray(ms), [10, 50, 90])]


def secondary_apply(args, kvc, synth, torch, name, rotate):
    """kvc_apply alone on another configuration's shapes: one edge's state is fitted (untimed), then the apply is timed.
    With rotate > 1 that many independent data sets (caches, tables, states) are cycled, so that a working set smaller
    than the 256 MB MALL cannot stay cached between iterations."""
    w = synth.WORKLOADS[name].with_(num_agents=2)
    L, H, d, T, r = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0], w.rank
    sets, calls = [], []
    for s_ in range(rotate):
        pc = synth.build_paged(w.with_(seed=w.seed + 7919 * s_), device="cuda", num_output_agents=1)
        cache = kvc.Cache(pc.k_pools, pc.v_pools)
        st = kvc.State.empty(L, H, d, T, r, torch.bfloat16, "cuda")
        src, dst, out = pc.seqs[(0, 0)], pc.seqs[(0, 1)], pc.seqs[(0, 100)]
        tab = lambda q, pc=pc: pc.tables[[q.table_row]]
        kvc.kvc_fit_state(cache, kvc.Batch([T], [src.offset], [dst.offset], [st], tab(src), tab(dst)))
        ab = kvc.Batch([T], [src.offset], [out.offset], [st], tab(src), tab(out))
        sets.append((pc, cache, st, ab))
        calls.append(lambda cache=cache, ab=ab: kvc.kvc_apply(cache, ab))
    torch.cuda.synchronize()
    ms, q = _timed_calls(torch, calls, args.steps, min(args.warmup, 10))
    b = _apply_bytes(L, H, d, T, r)
    gbps = b / (ms * 1e-3) / 1e9
    del sets, calls
    torch.cuda.empty_cache()
    return {"workload": f"{w.name}: {L} layers x {H} KV heads x head_dim {d}, {T} shared tokens, rank {r}, bf16 paged "
                        f"(block {w.block_size}, shuffled table); {rotate} data set(s) rotated",
            "apply_ms": round(ms, 4), "apply_ms_p10_p50_p90": q, "apply_bytes": b, "apply_gbps": round(gbps, 2),
            "apply_frac": round(gbps / HBM_PEAK_GBPS, 4)}


def serving_measurement(args, kvc, synth, torch, window=2):
    """The concurrent serving batch: 64 requests (lengths ~ U[1024, 16384]) sharing one block pool, rank 64, one hop.
    The whole cache (32 layers, about 292 GB over four agents) does not fit in HBM, so a window of `window` layers is
    generated; per layer the batched fit of all 64 requests and one kvc_apply launch over all 64 requests are timed,
    and the full-model figures are the per-layer times x 32."""
    w = synth.WORKLOADS["serving"]
    full_layers = w.num_layers
    w = w.with_(num_layers=window, num_agents=2)
    H, d, r, Q = w.num_kv_heads, w.head_dim, w.rank, w.num_requests
    pc = synth.build_paged(w, device="cuda", num_output_agents=1)
    cache = kvc.Cache(pc.k_pools, pc.v_pools)
    rows = lambda seqs: pc.tables[[pc.seqs[s_].table_row for s_ in seqs]]
    src, dst, out = [(q, 0) for q in range(Q)], [(q, 1) for q in range(Q)], [(q, 100) for q in range(Q)]
    lens = list(w.seq_tokens)
    st = [kvc.State.empty(window, H, d, lens[q], r, torch.bfloat16, "cuda") for q in range(Q)]
    fb = kvc.Batch(lens, [pc.seqs[s_].offset for s_ in src], [pc.seqs[s_].offset for s_ in dst], st, rows(src),
                   rows(dst))
    ab = kvc.Batch(lens, [pc.seqs[s_].offset for s_ in src], [pc.seqs[s_].offset for s_ in out], st, rows(src),
                   rows(out))
    ws = torch.empty(kvc.kvc_fit_workspace_bytes(cache, fb, 0, 1), dtype=torch.uint8, device="cuda")
    fit_calls = [lambda l=l: kvc.kvc_fit_state(cache, fb, l, l + 1, workspace=ws) for l in range(window)]
    apply_calls = [lambda l=l: kvc.kvc_apply(cache, ab, l, l + 1) for l in range(window)]
    n = max(window, args.steps // 2)
    fit_ms, fq = _timed_calls(torch, fit_calls, n, window)
    apply_ms, aq = _timed_calls(torch, apply_calls, max(window, args.steps), window)
    tok = sum(lens)
    b = tok * 2 * H * (2 * d * 2 + r * 2) + Q * 2 * H * r * d * 4
    gbps = b / (apply_ms * 1e-3) / 1e9
    del ws, st, fb, ab, pc, cache
    torch.cuda.empty_cache()
    return {"workload": f"serving: {Q} requests (sum of lengths {tok}, ~U[1024, 16384]) x 8 KV heads x head_dim {d}, "
                        f"rank {r}, bf16 paged shared pool; one hop; {window} of {full_layers} layers generated",
            "apply_ms_per_layer_launch": round(apply_ms, 4), "apply_ms_p10_p50_p90": aq,
            "apply_bytes_per_launch": b, "apply_gbps": round(gbps, 2), "apply_frac": round(gbps / HBM_PEAK_GBPS, 4),
            "fit_ms_per_layer": round(fit_ms, 4), "fit_ms_p10_p50_p90": fq,
            "fit_token_layers_per_s": round(tok / (fit_ms * 1e-3), 1),
            "full_model_ms": {"fit": round(fit_ms * full_layers, 3), "apply": round(apply_ms * full_layers, 3)}}


def verify_last_apply(pc, w, edge, out_seq, layer, head):
    """The output of the last timed apply against the oracle on one sampled (layer, KV head): the oracle fits every
    edge 1 .. `edge` from the ground-truth caches, composes them as the benchmark does (T_1 = S_1, T_i = chain(T_{i-1},
    S_i) at the same rank) and applies the result to the first agent's rows."""
    import numpy as np
    import torch
    from oracle import kvc_oracle as O

    def np_storage(t):
        return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16).copy()

    t0 = time.perf_counter()
    k = np_storage(pc.k_pools[layer][:, :, head:head + 1, :])
    v = np_storage(pc.v_pools[layer][:, :, head:head + 1, :])
    cache = O.Cache("bf16", w.block_size, [k], [v])
    tabs = pc.tables.cpu().numpy().astype(np.int64)
    T, r = w.seq_tokens[0], w.rank

    def item(a, b, st=None):
        return O.Item(T, pc.seqs[a].offset, pc.seqs[b].offset, tabs[pc.seqs[a].table_row],
                      tabs[pc.seqs[b].table_row], st)

    comp = None
    for i in range(1, edge + 1):
        s_i = O.fit(cache, [item((0, i - 1), (0, i))], r)[0][0]
        comp = s_i if comp is None else O.chain(comp, s_i, r)[0]
    ref = O.apply(cache, [item((0, 0), out_seq, comp)])
    it = item((0, 0), out_seq)
    worst = teeth = 0.0
    for kv in range(2):
        g = O.to_f64(O.read_rows(cache, 0, kv, 0, it.dst_table, it.dst_offset, T), "bf16")
        e = O.to_f64(O.read_rows(ref, 0, kv, 0, it.dst_table, it.dst_offset, T), "bf16")
        s_ = O.to_f64(O.read_rows(cache, 0, kv, 0, it.src_table, it.src_offset, T), "bf16")
        worst = max(worst, O.max_relative_error(g, e))
        teeth = max(teeth, O.max_relative_error(s_, e))
    return {"layer": layer, "head": head, "edge": edge, "max_rel_err": float(f"{worst:.3e}"), "bar": 1e-2,
            "uncorrected_rel_err": float(f"{teeth:.3e}"), "ok": bool(worst <= 1e-2),
            "oracle_seconds": round(time.perf_counter() - t0, 2)}


def cpu_baseline(pc, w, sample_layers=(0, 1)):
    """The oracle as it stands on a bounded sample of the same workload: `sample_layers` (every K/V head) of the
    first two edges -- fit S_1 and S_2, compose T_2 = chain(S_1, S_2), apply T_2 to the first agent's cache."""
    import numpy as np
    import threadpoolctl
    import torch
    from oracle import kvc_oracle as O

    def np_storage(t):
        t = t.detach().to("cpu").contiguous()
        return t.view(torch.int16).numpy().view(np.uint16).copy() if t.dtype == torch.bfloat16 else t.numpy().copy()

    ls = list(sample_layers)
    cache = O.Cache("bf16", w.block_size, [np_storage(pc.k_pools[l]) for l in ls],
                    [np_storage(pc.v_pools[l]) for l in ls])
    tabs = pc.tables.cpu().numpy().astype(np.int64)
    T = w.seq_tokens[0]

    def item(src, dst, st=None):
        return O.Item(T, pc.seqs[src].offset, pc.seqs[dst].offset, tabs[pc.seqs[src].table_row],
                      tabs[pc.seqs[dst].table_row], st)

    threads = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] + [1])
    t0 = time.perf_counter()
    s1, _ = O.fit(cache, [item((0, 0), (0, 1))], w.rank)
    t1 = time.perf_counter()
    s2, _ = O.fit(cache, [item((0, 1), (0, 2))], w.rank)
    t2 = time.perf_counter()
    t_state, _ = O.chain(s1[0], s2[0], w.rank)
    t3 = time.perf_counter()
    O.apply(cache, [item((0, 0), (0, 101), t_state)])
    t4 = time.perf_counter()
    nl = len(ls)
    apply_gbps = _apply_bytes(nl, w.num_kv_heads, w.head_dim, T, w.rank) / (t4 - t3) / 1e9
    fit_s = (t2 - t0) / 2
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": round(apply_gbps, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
        "host_cpus": os.cpu_count(), "cpu_model": model,
        "cores_note": "cores = BLAS threads the oracle's linear algebra used; host_cpus = os.cpu_count()",
        "sample": f"layers {ls} of {w.num_layers} (all K/V heads), edges 1-2: fit {fit_s:.2f} s per edge, "
                  f"chain {t3 - t2:.2f} s, apply {t4 - t3:.2f} s (value = apply GB/s on the sample)",
        "fit_token_layers_per_s": round(T * nl / fit_s, 1),
        "seconds": round(t4 - t0, 2),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama8b_32k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--anchor-workload", default="llama8b_4k",
                    help="shapes of the anchor-pool measurement (the paper's 4K-token pool example)")
    ap.add_argument("--anchors", type=int, default=10, help="anchors per shared slot (the paper's default V)")
    ap.add_argument("--anchor-rank", type=int, default=32)
    ap.add_argument("--no-anchor-pool", action="store_true")
    ap.add_argument("--no-rope", action="store_true", help="skip the rotary re-alignment measurement")
    ap.add_argument("--no-layer-fit", action="store_true", help="skip the per-layer factorisation measurement")
    ap.add_argument("--no-chain-study", action="store_true", help="skip the chained / non-chained error study")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the apply timings on the 8B/4K, VLM and serving-batch shapes")
    ap.add_argument("--no-verify", action="store_true",
                    help="skip the oracle check of the last timed apply's output on a sampled layer and head")
    ap.add_argument("--no-copy-ceiling", action="store_true",
                    help="skip the same-GPU copy ceilings (rank-0 apply through the tables, contiguous copy)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="before the steps, run one elementwise kernel that reads BYTES and writes BYTES (dst = -src "
                         "in float32), a plain copy of known size, so that HBM counters of a profiling run can be "
                         "scaled")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the correction path has no cross-GPU step to measure (asked for "
              f"{args.gpus}).", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2609_34060_amd import kvc, synth

    kvc.load()
    dev = "cuda"
    w = synth.WORKLOADS[args.workload]
    assert w.num_requests == 1 and w.dtype == "bf16", "single-request bf16 workloads only"
    L, H, d, T, r = w.num_layers, w.num_kv_heads, w.head_dim, w.seq_tokens[0], w.rank
    A = w.num_agents
    t_gen = time.perf_counter()
    pc = synth.build_paged(w, device=dev, num_output_agents=A - 1)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    cache = kvc.Cache(pc.k_pools, pc.v_pools)

    def tab(seq):
        return pc.tables[[pc.seqs[seq].table_row]]

    def batch(src, dst, st):
        return kvc.Batch([T], [pc.seqs[src].offset], [pc.seqs[dst].offset], [st], tab(src), tab(dst))

    # per-edge fit states, two alternating composed states
    S = [kvc.State.empty(L, H, d, T, r, torch.bfloat16, dev) for _ in range(A - 1)]
    Tc = [kvc.State.empty(L, H, d, T, r, torch.bfloat16, dev) for _ in range(2)]
    fit_batches = [batch((0, j - 1), (0, j), S[j - 1]) for j in range(1, A)]
    ws_fit = torch.empty(kvc.kvc_fit_workspace_bytes(cache, fit_batches[0]), dtype=torch.uint8, device=dev)
    ws_chain = torch.empty(max(1, kvc.kvc_chain_workspace_bytes(S[0], S[1], Tc[0])), dtype=torch.uint8, device=dev)
    apply_batches = {(j, k): batch((0, 0), (0, 100 + j - 1), Tc[k]) for j in range(1, A) for k in range(2)}
    # T_1 = S_1 (set-up, untimed)
    kvc.kvc_fit_state(cache, fit_batches[0], workspace=ws_fit)
    torch.cuda.synchronize()
    if args.copy_calibration > 0:
        a_src = torch.ones(args.copy_calibration // 4, dtype=torch.float32, device=dev)
        a_dst = torch.empty_like(a_src)
        torch.neg(a_src, out=a_dst)
        torch.cuda.synchronize()
        del a_src, a_dst

    # edge j maps C_{j-1} to C_j (S[j - 1]); edges 2 .. A-1 compose with the previous edge's state
    edges = list(range(2, A))
    assert edges, "the benchmark chains at least three agents"

    def step(k, ev):
        j = edges[k % len(edges)]
        cur, prev = Tc[k % 2], (S[0] if j == 2 else Tc[(k + 1) % 2])
        ev[0].record()
        kvc.kvc_fit_state(cache, fit_batches[j - 1], workspace=ws_fit)
        ev[1].record()
        kvc.kvc_chain(prev, S[j - 1], cur, workspace=ws_chain)
        ev[2].record()
        kvc.kvc_apply(cache, apply_batches[(j, k % 2)])
        ev[3].record()

    for k in range(args.warmup):
        step(k, [torch.cuda.Event(enable_timing=True) for _ in range(4)])
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(args.warmup + k, evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    _progress(f"{args.steps} timed steps done")
    fit_all = [e[0].elapsed_time(e[1]) for e in evs]
    chain_all = [e[1].elapsed_time(e[2]) for e in evs]
    apply_all = [e[2].elapsed_time(e[3]) for e in evs]
    fit_ms, chain_ms, apply_ms = (sum(x) / args.steps for x in (fit_all, chain_all, apply_all))

    def pct(x):
        q = np.percentile(np.asarray(x), [10, 50, 90])
        return [round(float(v), 4) for v in q]

    apply_b = _apply_bytes(L, H, d, T, r)
    apply_gbps = apply_b / (apply_ms * 1e-3) / 1e9
    fit_tl = T * L / (fit_ms * 1e-3)
    src_hash = _source_hash("kvc_apply.hip", "kvc_device.h")
    traffic = _traffic(src_hash)
    out = {
        "metric": "corrected KV GB/s & % HBM peak (kvc_apply); fit tokens*layers/s",
        "value": round(apply_gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {L} layers x {H} KV heads x head_dim {d}, {T} shared tokens, {A} agents "
                               f"chained, rank {r}, bf16 paged (block {w.block_size}, shuffled table), "
                               f"step = fit + chain + apply of one edge",
                   "layers": L, "kv_heads": H, "head_dim": d, "shared_tokens": T, "agents": A, "rank": r,
                   "block_size": w.block_size},
        "pct_hbm_peak": round(100.0 * apply_gbps / HBM_PEAK_GBPS, 2),
        "apply_ms": round(apply_ms, 4),
        "fit_ms": round(fit_ms, 4),
        "chain_ms": round(chain_ms, 4),
        "ms_p10_p50_p90": {"apply": pct(apply_all), "fit": pct(fit_all), "chain": pct(chain_all)},
        "fit_token_layers_per_s": round(fit_tl, 1),
        "fit_gbps_two_pass": round(_fit_bytes(L, H, d, T, r) / (fit_ms * 1e-3) / 1e9, 2),
        "roofline": {"bound": "hbm", "achieved": round(apply_gbps, 2), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(apply_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else round(traffic / (apply_ms * 1e-3) / 1e9, 2),
                     "kernel": "apply_bf16_mfma", "algorithmic_bytes_per_launch": apply_b,
                     "traffic_bytes_per_launch": traffic},
        "generation_s": round(t_gen, 2),
        "source_hash": src_hash,
    }
    last_edge = edges[(args.warmup + args.steps - 1) % len(edges)]
    if not args.no_verify:
        out["verify_last_apply"] = verify_last_apply(pc, w, last_edge, (0, 100 + last_edge - 1), L - 1, H // 2)
        _progress("verify_last_apply done")
    if not args.no_copy_ceiling:
        out["copy_ceiling"] = copy_ceiling(args, kvc, torch, cache, w, batch)
        _progress("copy_ceiling done")
        cc = out["copy_ceiling"]["kernels"]
        blocks = {k_: v_["gbps"] for k_, v_ in cc.items() if k_.startswith("paged_blocks")}
        out["copy_ceiling"]["apply_vs_paged_block_copy_logical"] = round(apply_gbps / cc["paged_blocks_logical_x1"]["gbps"], 4)
        out["copy_ceiling"]["apply_vs_best_paged_block_copy"] = round(apply_gbps / max(blocks.values()), 4)
        out["copy_ceiling"]["apply_vs_best_contiguous_copy"] = round(
            apply_gbps / max(cc["contiguous_xcd"]["gbps"], cc["contiguous_chunked"]["gbps"]), 4)
    if not args.no_rope:
        out["rope"] = rope_measurement(args, kvc, torch, pc, w, Tc[0], batch)
        _progress("rope done")
    if not args.no_layer_fit:
        out["layer_fit"] = layer_fit_measurement(args, kvc, torch, pc, w)
        _progress("layer_fit done")
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(pc, w)
        _progress("cpu_baseline done")
    if not args.no_anchor_pool:
        del cache, S, Tc, fit_batches, apply_batches, ws_fit, ws_chain, pc
        torch.cuda.empty_cache()
        out["anchor_pool"] = anchor_pool_measurement(args, kvc, synth, torch)
        _progress("anchor_pool done")
        if not args.no_rope:
            out["anchor_pool_rope"] = anchor_pool_measurement(args, kvc, synth, torch, rope=True)
            _progress("anchor_pool_rope done")
    if not args.no_chain_study:
        out["chain_study"] = chain_study(args, kvc, synth, torch)
        _progress("chain_study done")
    if not args.no_configs:
        out["configs"] = {}
        out["configs"]["llama8b_4k"] = secondary_apply(args, kvc, synth, torch, "llama8b_4k", 1)
        _progress("configs.llama8b_4k done")
        out["configs"]["vlm"] = secondary_apply(args, kvc, synth, torch, "vlm", 3)
        _progress("configs.vlm done")
        out["configs"]["serving"] = serving_measurement(args, kvc, synth, torch)
        _progress("configs.serving done")
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
