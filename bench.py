"""Benchmark of the DGE eviction step on one MI355X.

One step = one pass of the whole hot path over one layer's synthetic input:
dge_score -> dge_select_topb (max-pool + top-(B-w)) -> dge_compact.  Default
workload: one Llama-3-8B-shaped layer (32 query / 8 KV heads, d 128, batch 1,
L 4096, window 32 + k 2 draft rows, B 512, pool 7, bf16).

Inputs are resident in HBM before timing.  They are rotated over ``--sets``
distinct device copies (default 48, ~0.8 GB in total) so that no step finds its
K/V in the 256 MB Infinity Cache from an earlier step.  Steps are captured in
HIP graphs (8 steps per graph) so the timed region measures the GPU, not Python
launch overhead; the graphs are checked against the eager result first.

Prints ONE JSON line (metric, value, roofline of the dominant kernel, CPU
oracle baseline).  Progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
WORKLOAD_TEXT = {
    "c1": "c1: tiny fp32 layer, 4q/2kv heads, d=64, L=512, window 8 + k=2, B=64, max-pool 5",
    "c2": "c2: one Llama-3-8B-shaped layer, 32q/8kv heads, d=128, batch 1, L=4096, "
          "window 32 + k=2 draft rows, B=512, max-pool 7",
    "c3": "c3: 32 Llama-3-8B-shaped layers, 32q/8kv heads, d=128, batch 1, L=16384, "
          "window 32 + k=2, PyramidKV-style budgets 2048 -> 256, max-pool 7",
    "c4": "c4: 32 Llama-3-8B-shaped layers, 32q/8kv heads, d=128, ragged batch of 8 with "
          "L_b in [16384, 32768], window 32 + k=2, B=2048, max-pool 7",
    "c5": "c5: H2O on one Llama-3-8B-shaped layer, 32q/8kv heads, d=128, L=8192 + k=2, "
          "all 8194 rows scored, 512 heavy + 512 recent",
}
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 matrix peak
GRAPH_STEPS = 8


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def graph_steps(steps: int, sets: int) -> int:
    """Steps per captured graph: the largest of GRAPH_STEPS, 4, 2, 1 that divides both the
    requested step count (so exactly that many are timed) and the number of buffer sets."""
    for g in (GRAPH_STEPS, 4, 2, 1):
        if steps % g == 0 and sets % g == 0:
            return g
    return 1


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="c4",
                   help="c1..c5 (default c4, the largest single-GPU configuration: 32 layers, "
                        "a ragged batch of 8 sequences of 16K-32K tokens)")
    p.add_argument("--sets", type=int, default=48)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--copy-cal", action="store_true",
                   help="only run a plain 256 MiB device-to-device copy 8 times (the reference "
                        "for scaling FETCH_SIZE / WRITE_SIZE counters to bytes)")
    p.add_argument("--lse", action="store_true",
                   help="score with the scoring rows' log-sum-exp supplied (dge_score_lse); the "
                        "LSE is prepared outside the timed region, as an attention forward would")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--repeat-kv", action="store_true",
                   help="the prototype's layout: every KV head repeated to the G query heads of its "
                        "group, scored and selected per query head (no group mean); one layer")
    p.add_argument("--streams", type=int, default=1,
                   help="single-layer workloads: run independent steps (different buffer sets, "
                        "i.e. different requests' layers) on this many streams at once; reported "
                        "on its own line, the default bench keeps one stream")
    p.add_argument("--rope", action="store_true",
                   help="only time dge_rope on the workload's keys (every cached row of every KV "
                        "head), HIP events per call; one JSON line with its HBM rate")
    p.add_argument("--project", action="store_true",
                   help="only time dge_project_rope (query/key capture from the layer input) at "
                        "Llama-3-8B shapes: the scoring rows' q and k projections (HBM-bound on the "
                        "weights) and every row of an 8194-row layer (matrix cores); one JSON line")
    p.add_argument("--attend", action="store_true",
                   help="the checks after the path on one layer of the workload: attention of the "
                        "scoring rows over the compacted cache (dge_cache_attention) and the "
                        "evicted mass / matching loss (dge_evicted_mass)")
    p.add_argument("--compact-cmp", action="store_true",
                   help="only time dge_compact (out of place) against dge_compact_inplace on one "
                        "layer of the workload, the cache restored outside the timed events")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(f"bench.py: runs on one GPU; --gpus {args.gpus} is not supported (every step "
              "is independent per KV head and sequence: tensor- or batch-parallel sharding "
              "needs no exchange)", file=sys.stderr)
        sys.exit(2)
    import torch
    import dge_inputs as di
    import paper_2609_33334_amd as dge

    if args.copy_cal:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(8):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel(), "copies": 8}), flush=True)
        return

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = "cuda:0"
    if args.project:
        return bench_project(args, dev)
    wl = di.WORKLOADS[args.workload]
    log(f"[bench] workload {wl.name}: generating inputs")
    x = di.make_layer(wl, with_v=True)
    if args.compact_cmp:
        return bench_compact_cmp(args, wl, x, dev)
    if args.rope:
        return bench_rope(args, wl, x, dev)
    if args.attend:
        return bench_attend(args, wl, x, dev)
    if args.repeat_kv:
        return bench_repeat_kv(args, wl, x, dev)
    if args.streams > 1:
        return bench_streams(args, wl, x, dev)
    if wl.h2o:
        return bench_h2o(args, wl, x, dev)
    is_bf16 = wl.dtype == "bf16"
    elt = 2 if is_bf16 else 4

    def dev_t(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits))
        if is_bf16:
            t = t.view(torch.int16).view(torch.bfloat16)
        return t.to(dev)

    geom = dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                        wl.cached_lens, dtype=dge.DGE_BF16 if is_bf16 else dge.DGE_F32, device=dev)
    q0, k0, v0 = dev_t(x.q_bits), dev_t(x.k_bits), dev_t(x.v_bits)
    n_tail = wl.window + wl.k_draft
    L_layers = wl.n_layers
    budgets = [wl.budget_of_layer(l) for l in range(L_layers)]
    # one step = every layer once; single-layer workloads rotate over --sets copies so that
    # no step finds its inputs in the Infinity Cache, multi-layer ones are large enough
    # (each layer gets its own copy of the generated layer's tensors)
    S = max(1, args.sets) if L_layers == 1 else 1
    # A multi-layer cache is held layer-major ([layer][KV head][row][d], queries likewise):
    # the layers' KV heads are then consecutive heads of one geometry, and a single
    # dge_score call scores every layer (each layer keeps its own copy of the tensors).
    Hq, Hkv = wl.n_q_heads, wl.n_kv_heads
    geom_all = geom if L_layers == 1 else dge.Geometry(
        Hq * L_layers, Hkv * L_layers, wl.head_dim, wl.window, wl.k_draft, wl.cached_lens,
        dtype=geom.dtype, device=dev)
    ws_score = torch.empty(dge.workspace_size(geom_all, dge.OP_SCORE), dtype=torch.uint8, device=dev)
    ws_sel = torch.empty(dge.workspace_size(geom, dge.OP_SELECT), dtype=torch.uint8, device=dev)
    sets = []     # sets[set] = (q_all, k_all, v_all, raw_all, per-layer [(q, k, v, out, budget)])
    nr = wl.window + wl.k_draft
    for i in range(S):
        if L_layers == 1:
            q_all, k_all, v_all = q0.clone(), k0.clone(), v0.clone()
        else:
            # every layer its own inputs: layer 0 is the seeded host layer the oracle checks,
            # the others are drawn per layer (planted workloads on the host with their own
            # seeds, unplanted ones on the device)
            q_all = torch.empty(Hq * L_layers, geom.batch * nr, wl.head_dim, dtype=q0.dtype, device=dev)
            k_all = torch.empty(Hkv * L_layers, geom.total_rows, wl.head_dim, dtype=k0.dtype, device=dev)
            v_all = torch.empty_like(k_all)
            for l in range(L_layers):
                if l == 0:
                    ql, kl, vl = q0, k0, v0
                elif wl.plant == "none":
                    ql, kl, vl = di.device_layer(wl, l, dev)
                else:
                    xl = di.make_layer(wl, layer=l)
                    ql, kl, vl = dev_t(xl.q_bits), dev_t(xl.k_bits), dev_t(xl.v_bits)
                q_all[l * Hq:(l + 1) * Hq] = ql
                k_all[l * Hkv:(l + 1) * Hkv] = kl
                v_all[l * Hkv:(l + 1) * Hkv] = vl
                del ql, kl, vl
            log(f"[bench] {L_layers} layers generated")
        raw_all = torch.empty(Hkv * L_layers, geom.total_rows, dtype=torch.float32, device=dev)
        # outputs packed layer after layer (the layout of dge_select_compact_layers)
        nb = geom.batch * Hkv
        n_sels = [B - wl.window for B in budgets]
        flat = dict(idx=torch.empty(max(4, nb * sum(n_sels)), dtype=torch.int32, device=dev),
                    n_kept=torch.zeros(max(4, L_layers * geom.batch), dtype=torch.int32, device=dev),
                    k=torch.empty(nb * sum(x + n_tail for x in n_sels), wl.head_dim,
                                  dtype=k0.dtype, device=dev),
                    v=torch.empty(nb * sum(x + n_tail for x in n_sels), wl.head_dim,
                                  dtype=k0.dtype, device=dev))
        row = []
        io = ro = 0
        for l in range(L_layers):
            n_sel = n_sels[l]
            rows = nb * (n_sel + n_tail)
            shape = (geom.batch, Hkv, n_sel + n_tail, wl.head_dim)
            out = dict(raw=raw_all[l * Hkv:(l + 1) * Hkv],
                       idx=flat["idx"][io:io + nb * n_sel].view(geom.batch, Hkv, n_sel),
                       n_kept=flat["n_kept"][l * geom.batch:(l + 1) * geom.batch],
                       k=flat["k"][ro:ro + rows].view(shape), v=flat["v"][ro:ro + rows].view(shape))
            io += nb * n_sel
            ro += rows
            row.append((q_all[l * Hq:(l + 1) * Hq], k_all[l * Hkv:(l + 1) * Hkv],
                        v_all[l * Hkv:(l + 1) * Hkv], out, budgets[l]))
        sets.append((q_all, k_all, v_all, raw_all, row, flat))
    torch.cuda.synchronize()
    row_lse = None
    if args.lse:
        # natural-log softmax normaliser of each scoring row over keys j <= p (fp32, torch),
        # per layer and sequence; rows in the order of q: [layer * H_q][batch * n_rows]
        G = wl.group
        q_all0, k_all0 = sets[0][0], sets[0][1]
        row_lse = torch.empty(Hq * L_layers, geom.batch * nr, dtype=torch.float32, device=dev)
        for l in range(L_layers):
            for b, N in enumerate(wl.cached_lens):
                off = int(wl.kv_offsets[b])
                qq = q_all0[l * Hq:(l + 1) * Hq, b * nr:(b + 1) * nr].float()
                kk = k_all0[l * Hkv:(l + 1) * Hkv, off:off + N].float().repeat_interleave(G, dim=0)
                xx = torch.matmul(qq, kk.transpose(1, 2).contiguous()) / (wl.head_dim ** 0.5)
                pos = torch.arange(N - nr, N, device=dev)
                xx = xx.masked_fill(torch.arange(N, device=dev)[None, None, :] > pos[None, :, None],
                                    float("-inf"))
                row_lse[l * Hq:(l + 1) * Hq, b * nr:(b + 1) * nr] = torch.logsumexp(xx, dim=2)
                del xx, kk, qq

    def score_call(i):
        q_all, k_all, _, raw_all, _, _ = sets[i % S]
        if row_lse is not None:
            dge.score_lse(geom_all, dge.ROWS_WINDOW_DRAFT, q_all, k_all, row_lse, raw=raw_all)
        else:
            dge.score(geom_all, dge.ROWS_WINDOW_DRAFT, q_all, k_all, raw=raw_all, ws=ws_score)

    def step(i):
        score_call(i)
        _, k_all, v_all, raw_all, row, flat = sets[i % S]
        if L_layers == 1:
            q, k, v, out, B = row[0]
            dge.select_compact(geom, out["raw"], wl.pool, n_tail, B - wl.window, k, v,
                               idx=out["idx"], n_kept=out["n_kept"], k_out=out["k"],
                               v_out=out["v"], ws=ws_sel)
        else:   # every layer, each with its own budget, in one launch
            dge.select_compact_layers(geom, raw_all, wl.pool, n_tail,
                                      [B - wl.window for B in budgets], k_all, v_all,
                                      idx=flat["idx"], n_kept=flat["n_kept"], k_out=flat["k"],
                                      v_out=flat["v"], ws=ws_sel)

    def score_only(i):
        score_call(i)

    # eager warmup and reference result
    for i in range(max(args.warmup, S)):
        step(i)
    torch.cuda.synchronize()
    # set 0's outputs: the scores of every layer and the packed selections / caches
    outs0 = dict(sets[0][5], raw=sets[0][3])
    ref = {kk: vv.clone() for kk, vv in outs0.items()}

    # HIP graphs of gsteps consecutive steps, covering every buffer set; gsteps divides
    # --steps, so exactly the requested number of steps is timed
    gsteps = graph_steps(args.steps, S) if L_layers == 1 else 1
    stream = torch.cuda.Stream()
    graphs, sgraphs = [], []
    n_graphs = max(1, S // gsteps)
    with torch.cuda.stream(stream):
        for gi in range(n_graphs):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                for j in range(gsteps):
                    step(gi * gsteps + j)
            graphs.append(g)
            sg = torch.cuda.CUDAGraph()
            with torch.cuda.graph(sg, stream=stream):
                for j in range(gsteps):
                    score_only(gi * gsteps + j)
            sgraphs.append(sg)
    torch.cuda.synchronize()
    # graph replays must reproduce the eager result (set 0 is in graph 0)
    for kk in ref:
        outs0[kk].zero_()
    torch.cuda.synchronize()
    graphs[0].replay()
    torch.cuda.synchronize()
    for kk in ref:
        assert torch.equal(outs0[kk], ref[kk]), f"graph replay differs from eager ({kk})"

    K = args.steps
    n_rep = K // gsteps
    for r in range(min(n_rep, 2 * n_graphs)):
        graphs[r % n_graphs].replay()
    torch.cuda.synchronize()
    log(f"[bench] timing {K} steps ({n_rep} graph replays of {gsteps} steps, {S} buffer sets, "
        f"{L_layers} layers per step)")
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for r in range(n_rep):
        graphs[r % n_graphs].replay()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    ms_per_step = gpu_ms / K
    # dominant kernel (dge_score) timed the same way, on the same stream
    es0 = torch.cuda.Event(enable_timing=True)
    es1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    es0.record()
    for r in range(n_rep):
        sgraphs[r % n_graphs].replay()
    es1.record()
    torch.cuda.synchronize()
    score_us = es0.elapsed_time(es1) * 1e3 / K      # one dge_score launch per step
    log(f"[bench] {ms_per_step * 1e3:.2f} us/step (event), wall {wall * 1e6 / K:.2f} us/step; "
        f"dge_score {score_us:.2f} us/call ({L_layers} layers per call)")
    # the median over individually timed graph replays (at least 20), after the timed region
    per = []
    for r in range(max(20, min(n_rep, 64))):
        a0 = torch.cuda.Event(enable_timing=True)
        a1 = torch.cuda.Event(enable_timing=True)
        a0.record()
        graphs[r % n_graphs].replay()
        a1.record()
        torch.cuda.synchronize()
        per.append(a0.elapsed_time(a1) / gsteps)
    ms_median = float(np.median(per))

    L = sum(wl.prompt_lens)
    units = L * wl.n_kv_heads * L_layers          # prefix tokens x KV heads per step
    value = units / (ms_per_step * 1e-3)
    # algorithmic bytes of one dge_score call: K once + the scoring queries
    n_rows = wl.window + wl.k_draft
    score_bytes = (wl.n_kv_heads * geom.total_rows * wl.head_dim * elt
                   + wl.n_q_heads * wl.batch * n_rows * wl.head_dim * elt)   # per layer
    achieved = score_bytes * L_layers / (score_us * 1e-6) / 1e9
    roofline = {"kernel": ("dge_score_lse (colsum launch)" if args.lse else
                           "dge_score (stats + reduce + colsum launches)"), "bound": "hbm",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(wl.name, args.lse, L_layers),
                "bytes_per_launch": int(score_bytes * L_layers), "us_per_launch": round(score_us, 3),
                "layers_per_launch": L_layers}
    # whole step against its own algorithmic bytes (score + compaction + indices)
    step_bytes = 0
    for B in budgets:
        n_sel = B - wl.window
        step_bytes += score_bytes + 4 * wl.n_kv_heads * wl.batch * (n_sel + n_tail) * wl.head_dim * elt \
            + 4 * wl.n_kv_heads * wl.batch * n_sel
    step_frac = step_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, x, args.cpu_seconds)
    line = {
        "metric": "prefix tokens x KV heads scored+compacted per second (DGE eviction step)",
        "value": round(value, 1), "unit": "token*kvhead/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 6),
        "ms_per_step_median": round(ms_median, 6), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if is_bf16 else "f32",
        "data": ("synthetic (seeded Gaussian Q/K/V"
                 + {"spans": " with planted spans", "scale_rows": " with planted x4 keys"}.get(wl.plant, "")
                 + (", every layer its own draw" if L_layers > 1 else "") + "; no model weights)"),
        "config": {"workload": WORKLOAD_TEXT.get(wl.name, wl.name),
                   "global_batch": wl.batch, "seq_len": L, "layers": L_layers,
                   "parallelism": "single GPU",
                   "step": (("dge_score_lse (row LSE supplied)" if args.lse else "dge_score")
                            + (" over all layers (layer-major cache) -> dge_select_compact_layers"
                               " (every layer's pool, top-(B_l-w), gather in one launch)"
                               if L_layers > 1 else
                               " -> dge_select_compact (pool, top-(B-w), gather)")),
                   "step_hbm_frac": round(step_frac, 4), "buffer_sets": S},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def bench_repeat_kv(args, wl, x, dev):
    """The eviction step on the repeated-KV layout the paper's prototype uses (App.
    "Complexity and overheads"): K and V copied to all H_q query heads, dge_score with one
    query head per cache head (no group mean), dge_select_compact per query head.  Same
    timing method as the main path (HIP graphs over rotating buffer sets); `value` counts
    prefix tokens x cache heads (H_q here).  Prints one JSON line."""
    import torch
    import paper_2609_33334_amd as dge

    def dev_t(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits))
        return t.view(torch.int16).view(torch.bfloat16).to(dev)

    G = wl.n_q_heads // wl.n_kv_heads
    H = wl.n_q_heads
    g1 = dge.Geometry(H, H, wl.head_dim, wl.window, wl.k_draft, wl.cached_lens, device=dev)
    q0 = dev_t(x.q_bits)
    k0 = dev_t(np.repeat(x.k_bits, G, axis=0))
    v0 = dev_t(np.repeat(x.v_bits, G, axis=0))
    n_tail = wl.window + wl.k_draft
    n_sel = wl.budget_of_layer(0) - wl.window
    S = max(1, args.sets) if wl.n_layers == 1 else 1
    ws_score = torch.empty(dge.workspace_size(g1, dge.OP_SCORE), dtype=torch.uint8, device=dev)
    ws_sel = torch.empty(dge.workspace_size(g1, dge.OP_SELECT), dtype=torch.uint8, device=dev)
    sets = []
    for _ in range(S):
        out = dict(raw=torch.empty(H, g1.total_rows, dtype=torch.float32, device=dev),
                   idx=torch.empty(g1.batch, H, n_sel, dtype=torch.int32, device=dev),
                   n_kept=torch.zeros(max(4, g1.batch), dtype=torch.int32, device=dev),
                   k=torch.empty(g1.batch, H, n_sel + n_tail, wl.head_dim, dtype=k0.dtype, device=dev),
                   v=torch.empty(g1.batch, H, n_sel + n_tail, wl.head_dim, dtype=k0.dtype, device=dev))
        sets.append((q0.clone(), k0.clone(), v0.clone(), out))

    def step(i):
        q, k, v, out = sets[i % S]
        dge.score(g1, dge.ROWS_WINDOW_DRAFT, q, k, raw=out["raw"], ws=ws_score)
        dge.select_compact(g1, out["raw"], wl.pool, n_tail, n_sel, k, v, idx=out["idx"],
                           n_kept=out["n_kept"], k_out=out["k"], v_out=out["v"], ws=ws_sel)

    for i in range(max(args.warmup, S)):
        step(i)
    torch.cuda.synchronize()
    gsteps = graph_steps(args.steps, S)
    stream = torch.cuda.Stream()
    graphs = []
    with torch.cuda.stream(stream):
        for gi in range(max(1, S // gsteps)):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=stream):
                for j in range(gsteps):
                    step(gi * gsteps + j)
            graphs.append(gr)
    torch.cuda.synchronize()
    n_rep = args.steps // gsteps
    K = n_rep * gsteps
    for r in range(min(n_rep, 2 * len(graphs))):
        graphs[r % len(graphs)].replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for r in range(n_rep):
        graphs[r % len(graphs)].replay()
    e1.record()
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / K
    L = sum(wl.prompt_lens)
    kv_native = 2 * wl.n_kv_heads * g1.total_rows * wl.head_dim * 2
    print(json.dumps({
        "metric": "prefix tokens x cache heads scored+compacted per second (repeated-KV layout)",
        "value": round(L * H / (ms_per_step * 1e-3), 1), "unit": "token*head/s",
        "ms_per_step": round(ms_per_step, 6), "steps": K, "warmup": args.warmup,
        "workload": WORKLOAD_TEXT.get(wl.name, wl.name),
        "layout": f"K/V repeated x{G} to {H} cache heads, per-query-head scores and top-(B-w)",
        "kv_bytes_per_layer": {"repeated": kv_native * G, "native_gqa": kv_native}}), flush=True)


def bench_streams(args, wl, x, dev):
    """Throughput of independent eviction steps of a single-layer workload in flight together:
    step j of a graph runs on stream j % n (its own workspaces), the streams forked from and
    joined back to the timed stream, so the latency-bound launches of different steps
    overlap.  Prints one JSON line (not the default bench line)."""
    import torch
    import paper_2609_33334_amd as dge

    if wl.n_layers != 1 or wl.h2o:
        print("bench.py: --streams is for the single-layer eviction workloads", file=sys.stderr)
        sys.exit(2)
    n = args.streams

    def dev_t(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits))
        if wl.dtype == "bf16":
            t = t.view(torch.int16).view(torch.bfloat16)
        return t.to(dev)

    geom = dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                        wl.cached_lens, dtype=dge.DGE_BF16 if wl.dtype == "bf16" else dge.DGE_F32,
                        device=dev)
    q0, k0, v0 = dev_t(x.q_bits), dev_t(x.k_bits), dev_t(x.v_bits)
    n_tail = wl.window + wl.k_draft
    n_sel = wl.budget_of_layer(0) - wl.window
    S = max(n, args.sets)
    ws = [(torch.empty(dge.workspace_size(geom, dge.OP_SCORE), dtype=torch.uint8, device=dev),
           torch.empty(dge.workspace_size(geom, dge.OP_SELECT), dtype=torch.uint8, device=dev))
          for _ in range(n)]
    sets = []
    for _ in range(S):
        out = dict(raw=torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32, device=dev),
                   idx=torch.empty(geom.batch, geom.n_kv_heads, n_sel, dtype=torch.int32, device=dev),
                   n_kept=torch.zeros(max(4, geom.batch), dtype=torch.int32, device=dev),
                   k=torch.empty(geom.batch, geom.n_kv_heads, n_sel + n_tail, wl.head_dim,
                                 dtype=k0.dtype, device=dev),
                   v=torch.empty(geom.batch, geom.n_kv_heads, n_sel + n_tail, wl.head_dim,
                                 dtype=k0.dtype, device=dev))
        sets.append((q0.clone(), k0.clone(), v0.clone(), out))

    def step(i, c):
        q, k, v, out = sets[i % S]
        dge.score(geom, dge.ROWS_WINDOW_DRAFT, q, k, raw=out["raw"], ws=ws[c][0])
        dge.select_compact(geom, out["raw"], wl.pool, n_tail, n_sel, k, v, idx=out["idx"],
                           n_kept=out["n_kept"], k_out=out["k"], v_out=out["v"], ws=ws[c][1])

    for i in range(max(args.warmup, S)):
        step(i, 0)
    torch.cuda.synchronize()
    ref = {kk: vv.clone() for kk, vv in sets[n - 1][3].items()}
    gsteps = GRAPH_STEPS * n
    main_s = torch.cuda.Stream()
    side = [torch.cuda.Stream() for _ in range(n - 1)]
    graphs = []
    with torch.cuda.stream(main_s):
        for gi in range(max(1, S // gsteps)):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=main_s):
                for sd in side:
                    sd.wait_stream(main_s)
                for j in range(gsteps):
                    c = j % n
                    with torch.cuda.stream(main_s if c == 0 else side[c - 1]):
                        step(gi * gsteps + j, c)
                for sd in side:
                    main_s.wait_stream(sd)
            graphs.append(gr)
    torch.cuda.synchronize()
    for kk in ref:
        sets[n - 1][3][kk].zero_()
    torch.cuda.synchronize()
    graphs[0].replay()
    torch.cuda.synchronize()
    for kk in ref:
        assert torch.equal(sets[n - 1][3][kk], ref[kk]), f"graph replay differs from eager ({kk})"
    n_rep = max(1, (args.steps + gsteps - 1) // gsteps)
    K = n_rep * gsteps
    for r in range(min(n_rep, 2 * len(graphs))):
        graphs[r % len(graphs)].replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(main_s):
        e0.record()
        for r in range(n_rep):
            graphs[r % len(graphs)].replay()
        e1.record()
    torch.cuda.synchronize()
    ms_per_step = e0.elapsed_time(e1) / K
    L = sum(wl.prompt_lens)
    print(json.dumps({
        "metric": "prefix tokens x KV heads scored+compacted per second (DGE eviction step)",
        "value": round(L * wl.n_kv_heads / (ms_per_step * 1e-3), 1), "unit": "token*kvhead/s",
        "ms_per_step": round(ms_per_step, 6), "steps": K, "warmup": args.warmup,
        "concurrent_steps": n, "workload": WORKLOAD_TEXT.get(wl.name, wl.name),
        "step": "dge_score -> dge_select_compact; independent steps on separate streams"}),
        flush=True)


def bench_rope(args, wl, x, dev):
    """dge_rope over every cached key row of one layer (the K the scoring reads), in place,
    each call bracketed by HIP events (median of the repetitions).  Elementwise: the
    roofline is one read and one write of K."""
    import torch
    import paper_2609_33334_amd as dge

    k = torch.from_numpy(np.ascontiguousarray(x.k_bits)).view(torch.int16).view(torch.bfloat16).to(dev)
    T = k.shape[1]
    pos = torch.arange(T, dtype=torch.int32, device=dev)
    for _ in range(3):
        dge.rope(k, pos)
    torch.cuda.synchronize()
    reps = max(20, min(args.steps, 200))
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dge.rope(k, pos)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e3)
    us = float(np.median(ts))
    nbytes = 2 * k.numel() * 2
    print(json.dumps({"kernel": "dge_rope (keys of one layer, in place)", "workload": wl.name,
                      "rows": int(k.shape[0] * T), "bytes": nbytes, "us_per_call": round(us, 3),
                      "GBps": round(nbytes / us / 1e3, 1),
                      "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4), "reps": reps}),
          flush=True)


def bench_attend(args, wl, x, dev):
    """The two checks that follow the path, on one layer of the workload, after its scoring
    (dge_score_with_lse) and selection + compaction (dge_select_compact): attention of the
    window and draft rows over the compacted cache (dge_cache_attention: output and
    log-partition, the continuation check of Eq. 1) and their evicted mass, missed mass and
    matching loss (dge_evicted_mass, K only).  Back-to-back calls between HIP events on the
    launching stream (median of five groups).  Algorithmic bytes: the compacted K (and V for
    the attention) once, the query rows, the outputs.  Prints one JSON line."""
    import torch
    import paper_2609_33334_amd as dge
    is_bf16 = wl.dtype == "bf16"
    elt = 2 if is_bf16 else 4

    def dev_t(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits))
        if is_bf16:
            t = t.view(torch.int16).view(torch.bfloat16)
        return t.to(dev)

    g = dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                     wl.cached_lens, dtype=dge.DGE_BF16 if is_bf16 else dge.DGE_F32, device=dev)
    q, k, v = dev_t(x.q_bits), dev_t(x.k_bits), dev_t(x.v_bits)
    n_tail = wl.window + wl.k_draft
    n_sel = wl.budget_of_layer(0) - wl.window
    raw, row_lse = dge.score_with_lse(g, dge.ROWS_WINDOW_DRAFT, q, k)
    idx, nk, kc, vc = dge.select_compact(g, raw, wl.pool, n_tail, n_sel, k, v)
    out, lse = dge.cache_attention(g, q, n_tail, n_tail, kc, vc, n_sel, n_tail, nk)
    rho, beta, lm = dge.evicted_mass(g, q, n_tail, n_tail, kc, n_sel, n_tail, nk, row_lse)
    torch.cuda.synchronize()
    reps = max(20, min(args.steps, 200))
    stream = torch.cuda.current_stream()
    rows = wl.batch * n_tail
    kc_bytes = wl.batch * wl.n_kv_heads * (n_sel + n_tail) * wl.head_dim * elt
    q_bytes = wl.n_q_heads * rows * wl.head_dim * elt
    cases = {
        "cache_attention": (lambda: dge.cache_attention(g, q, n_tail, n_tail, kc, vc, n_sel, n_tail, nk,
                                                        out=out, lse=lse),
                            2 * kc_bytes + q_bytes + wl.n_q_heads * rows * (wl.head_dim + 1) * 4),
        "evicted_mass": (lambda: dge.evicted_mass(g, q, n_tail, n_tail, kc, n_sel, n_tail, nk, row_lse,
                                                  rho=rho, beta=beta, l_match=lm),
                         kc_bytes + q_bytes + 2 * wl.n_q_heads * rows * 4 + 2 * wl.batch * wl.n_kv_heads * 4),
    }
    res = {}
    for name, (call, nbytes) in cases.items():
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                call()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3 / reps)
        us = float(np.median(ts))
        gbs = nbytes / us / 1e3
        res[name] = {"us_per_call": round(us, 3), "bytes": int(nbytes),
                     "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                                  "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4)}}
        log(f"[bench] {name} {wl.name}: {us:.2f} us, {gbs:.0f} GB/s")
    print(json.dumps({"kernel": "dge_cache_attention / dge_evicted_mass over one compacted layer",
                      "workload": wl.name, "query_rows": rows, "retained_rows_per_head": n_sel + n_tail,
                      "reps": reps, "cases": res}), flush=True)


def bench_project(args, dev):
    """dge_project_rope at Llama-3-8B shapes (hidden 4096, 32 query / 8 KV heads of 128): the
    34 scoring rows (window 32 + k 2) through W_q and W_k, bound by streaming the weights
    from HBM, and all 8194 rows of a layer through W_q (H2O's prompt queries), bound by the
    matrix cores.  Synthetic bf16 inputs (x ~ N(0,1), W ~ N(0, 1/hidden)), weights rotated
    over enough copies that no call finds them in the Infinity Cache; HIP events around
    back-to-back calls on the launching stream (median of five groups).  Prints one JSON
    line."""
    import torch
    import paper_2609_33334_amd as dge
    hidden, d = 4096, 128
    gen = torch.Generator(device=dev)
    gen.manual_seed(2609)
    reps = max(20, min(args.steps, 200))
    res = {}
    for name, rows, heads, n_sets in (("q_scoring_rows", 34, 32, 16), ("k_scoring_rows", 34, 8, 48),
                                      ("fused_qk_scoring_rows", 34, 40, 16),
                                      ("q_all_rows_8194", 8194, 32, 4)):
        x = torch.randn(rows, hidden, generator=gen, device=dev).to(torch.bfloat16)
        ws = [(torch.randn(heads * d, hidden, generator=gen, device=dev) / hidden ** 0.5).to(torch.bfloat16)
              for _ in range(n_sets)]
        pos = torch.arange(26507, 26507 + rows, dtype=torch.int32, device=dev)
        out = torch.empty(heads, rows, d, dtype=torch.bfloat16, device=dev)
        need = dge.project_rope_workspace(rows, hidden, heads, d)
        wsp = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
        for i in range(2 * n_sets):
            dge.project_rope(x, ws[i % n_sets], pos, heads, d, out=out, ws=wsp)
        torch.cuda.synchronize()
        # back-to-back calls between two HIP events on the launching stream: the average
        # launch duration (a lone event pair would add the launch latency to every call)
        stream = torch.cuda.current_stream()
        ts = []
        for _ in range(5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for i in range(reps):
                dge.project_rope(x, ws[i % n_sets], pos, heads, d, out=out, ws=wsp)
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e3 / reps)
        us = float(np.median(ts))
        nbytes = heads * d * hidden * 2 + rows * hidden * 2 + heads * rows * d * 2 + rows * 4
        flops = 2 * rows * heads * d * hidden
        gbs = nbytes / us / 1e3
        tfs = flops / us / 1e6
        entry = {"rows": rows, "heads": heads, "us_per_call": round(us, 3), "bytes": nbytes,
                 "flops": flops, "GBps": round(gbs, 1), "TFLOPs": round(tfs, 1)}
        if rows < 1000:
            entry["roofline"] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                                 "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4)}
        else:
            entry["roofline"] = {"bound": "mfma", "achieved": round(tfs, 1),
                                 "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                                 "frac": round(tfs / MFMA_BF16_PEAK_TFS, 4)}
        res[name] = entry
        log(f"[bench] project_rope {name}: {us:.2f} us, {gbs:.0f} GB/s, {tfs:.0f} TFLOP/s")
        del ws, x, out
    print(json.dumps({"kernel": "dge_project_rope (RoPE(x W^T), hidden 4096, head_dim 128, bf16)",
                      "reps": reps, "cases": res}), flush=True)


def bench_compact_cmp(args, wl, x, dev):
    """Compaction of one layer (Alg. 1 step C) into a separate buffer (dge_compact) and as an
    edit of the cache itself (dge_compact_inplace), from the same selection.  Each call is
    bracketed by HIP events on the stream it runs on; the in-place call's cache is restored
    by a device copy before the first event.  Prints one JSON line."""
    import torch
    import paper_2609_33334_amd as dge

    def dev_t(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits))
        return t.view(torch.int16).view(torch.bfloat16).to(dev)

    geom = dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                        wl.cached_lens, device=dev)
    q, k, v = dev_t(x.q_bits), dev_t(x.k_bits), dev_t(x.v_bits)
    n_tail = wl.window + wl.k_draft
    n_sel = wl.budget_of_layer(0) - wl.window
    raw = dge.score(geom, dge.ROWS_WINDOW_DRAFT, q, k)
    idx, nk = dge.select_topb(geom, raw, wl.pool, n_tail, n_sel)
    k_out, v_out = dge.compact(geom, idx, nk, n_sel, n_tail, k, v)
    kw, vw = k.clone(), v.clone()
    torch.cuda.synchronize()
    reps = max(1, min(args.steps, 200))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    t_out, t_in = [], []
    for _ in range(reps):
        ev[0].record()
        dge.compact(geom, idx, nk, n_sel, n_tail, k, v, k_out=k_out, v_out=v_out)
        ev[1].record()
        kw.copy_(k)
        vw.copy_(v)
        ev[2].record()
        dge.compact_inplace(geom, idx, nk, n_sel, n_tail, kw, vw)
        ev[3].record()
        torch.cuda.synchronize()
        t_out.append(ev[0].elapsed_time(ev[1]) * 1e3)
        t_in.append(ev[2].elapsed_time(ev[3]) * 1e3)
    nk_h = nk.cpu().numpy()
    rows = int(sum(int(nk_h[b]) + n_tail for b in range(wl.batch))) * wl.n_kv_heads
    moved = 2 * 2 * rows * wl.head_dim * 2        # K and V, read + write, bf16
    med_out, med_in = float(np.median(t_out)), float(np.median(t_in))
    print(json.dumps({"workload": wl.name, "compacted_rows": rows, "bytes_moved": moved,
                      "dge_compact_us": round(med_out, 3), "dge_compact_inplace_us": round(med_in, 3),
                      "compact_GBps": round(moved / med_out / 1e3, 1),
                      "inplace_GBps": round(moved / med_in / 1e3, 1), "reps": reps}), flush=True)


def bench_h2o(args, wl, x, dev):
    """H2O step on one layer (Sec. 6 baselines; App. H2O complexity): accumulated attention
    of every cached row (dge_h2o_colsum, row LSE computed in the library unless --lse),
    then the top-(B - n_recent) heavy rows plus the n_recent most recent ones
    (dge_select_compact with pool 1).  The dominant kernel is MFMA-bound."""
    import torch
    import paper_2609_33334_amd as dge

    def dev_t(bits):
        t = torch.from_numpy(np.ascontiguousarray(bits))
        return t.view(torch.int16).view(torch.bfloat16).to(dev)

    geom = dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                        wl.cached_lens, dtype=dge.DGE_BF16, device=dev)
    qa0, k0, v0 = dev_t(x.q_all_bits), dev_t(x.k_bits), dev_t(x.v_bits)
    n_tail, n_sel = wl.n_recent, wl.budget - wl.n_recent
    lse = None
    if args.lse:   # natural-log LSE of every cached row, prepared outside the timed region
        N = wl.cached_lens[0]
        rows = []
        for hq in range(wl.n_q_heads):
            qq = qa0[hq].float()
            kk = k0[hq // wl.group].float()
            xx = (qq @ kk.t()) / (wl.head_dim ** 0.5)
            xx = xx.masked_fill(torch.ones(N, N, device=dev, dtype=torch.bool).triu(1), float("-inf"))
            rows.append(torch.logsumexp(xx, dim=1))
            del xx
        lse = torch.stack(rows).contiguous()
    S = 4
    ws_h2o = torch.empty(dge.workspace_size(geom, dge.OP_H2O), dtype=torch.uint8, device=dev)
    ws_sel = torch.empty(dge.workspace_size(geom, dge.OP_SELECT), dtype=torch.uint8, device=dev)
    sets = []
    for _ in range(S):
        out = dict(col=torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32, device=dev),
                   idx=torch.empty(1, geom.n_kv_heads, n_sel, dtype=torch.int32, device=dev),
                   n_kept=torch.zeros(4, dtype=torch.int32, device=dev),
                   k=torch.empty(1, geom.n_kv_heads, n_sel + n_tail, wl.head_dim, dtype=k0.dtype, device=dev),
                   v=torch.empty(1, geom.n_kv_heads, n_sel + n_tail, wl.head_dim, dtype=k0.dtype, device=dev))
        sets.append((qa0.clone(), k0.clone(), v0.clone(), out))

    def h2o_only(i):
        qa, k, v, out = sets[i % S]
        dge.h2o_colsum(geom, qa, k, lse=lse, colsum=out["col"], ws=ws_h2o)

    def step(i):
        qa, k, v, out = sets[i % S]
        h2o_only(i)
        dge.select_compact(geom, out["col"], 1, n_tail, n_sel, k, v, idx=out["idx"],
                           n_kept=out["n_kept"], k_out=out["k"], v_out=out["v"], ws=ws_sel)

    for i in range(max(args.warmup, S)):
        step(i)
    torch.cuda.synchronize()
    ref = {kk: vv.clone() for kk, vv in sets[0][3].items()}
    stream = torch.cuda.Stream()
    gs = graph_steps(args.steps, S)      # steps per graph, dividing --steps
    with torch.cuda.stream(stream):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for j in range(gs):
                step(j)
        sg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(sg, stream=stream):
            for j in range(gs):
                h2o_only(j)
    torch.cuda.synchronize()
    for kk in ref:
        sets[0][3][kk].zero_()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    for kk in ref:
        assert torch.equal(sets[0][3][kk], ref[kk]), f"graph replay differs from eager ({kk})"
    n_rep = max(1, args.steps // gs)
    K = n_rep * gs
    g.replay()
    torch.cuda.synchronize()

    def timed(graph):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(n_rep):
            graph.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    log(f"[bench] timing {K} H2O steps ({n_rep} replays of {gs})")
    ms_per_step = timed(g)
    h2o_ms = timed(sg)
    N = wl.cached_lens[0]
    passes = 1 if lse is not None else 2       # the LSE pass repeats QK^T
    flops = passes * (N * (N + 1) // 2) * 2 * wl.head_dim * wl.n_q_heads
    achieved = flops / (h2o_ms * 1e-3) / 1e12
    log(f"[bench] {ms_per_step * 1e3:.1f} us/step; dge_h2o_colsum {h2o_ms * 1e3:.1f} us/call, "
        f"{achieved:.0f} TFLOP/s executed")
    units = N * wl.n_kv_heads
    roofline = {"kernel": "dge_h2o_colsum (" + ("LSE supplied" if lse is not None else
                                                "row LSE computed in the library") + ")",
                "bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFS,
                "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFS, 4),
                "traffic": None, "flops_per_launch": flops, "us_per_launch": round(h2o_ms * 1e3, 3)}
    cpu = None if args.no_cpu_baseline else cpu_baseline_h2o(wl, x, args.cpu_seconds)
    line = {
        "metric": "cached tokens x KV heads scored+compacted per second (H2O eviction step)",
        "value": round(units / (ms_per_step * 1e-3), 1), "unit": "token*kvhead/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian Q/K/V; no model weights)",
        "config": {"workload": WORKLOAD_TEXT[wl.name], "global_batch": 1, "seq_len": N,
                   "layers": 1, "parallelism": "single GPU",
                   "step": "dge_h2o_colsum -> dge_select_compact (512 heavy + 512 recent)",
                   "buffer_sets": S},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def cpu_baseline_h2o(wl, x, seconds):
    """The float64 oracle's H2O colsum on a bounded sample: the query heads of the first
    KV head (one GQA group), scaled to all 8 KV heads."""
    import oracle
    from threadpoolctl import threadpool_limits
    cores = cpu_threads()
    G = wl.group
    q = x.q_all[:G]
    k = x.k[:1]
    with threadpool_limits(limits=cores):
        t0 = time.perf_counter()
        oracle.h2o_colsum(q, k, wl.kv_offsets, G, 1)
        el = time.perf_counter() - t0
    N = wl.cached_lens[0]
    rate = N / el                      # one KV head of N tokens in el seconds
    log(f"[bench] cpu oracle: one GQA group of H2O colsum in {el:.1f}s -> {rate:.3g} token*kvhead/s")
    return {"value": round(rate, 1), "unit": "token*kvhead/s", "cores": cores, "kind": "oracle",
            "sample": f"H2O colsum of one KV head's GQA group ({G} query heads x {N} rows) in "
                      f"float64 numpy, {el:.1f} s; select/compact not included"}


SCORE_SOURCES = ("paper_2609_33334_amd/csrc/score.hip", "paper_2609_33334_amd/csrc/dge_device.hpp")


def score_source_hash() -> str:
    """sha256 of the score kernels' code with comments and whitespace removed."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in SCORE_SOURCES:
        with open(os.path.join(ROOT, f)) as fh:
            code = fh.read()
        code = re.sub(r"/\*.*?\*/", "", code, flags=re.S)
        code = re.sub(r"//[^\n]*", "", code)
        h.update(re.sub(r"\s+", "", code).encode())
    return h.hexdigest()


def measured_traffic(workload: str, lse: bool, layers_per_call: int):
    """HBM bytes per dge_score call from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary, or None when there is none, it was taken with another number of layers per
    call, or the score kernels changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"score_traffic_{workload}{'_lse' if lse else ''}.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != score_source_hash():
        return None
    if rec.get("layers_per_call", 1) != layers_per_call:
        return None
    return rec.get("hbm_bytes_per_call")


def cpu_threads() -> int:
    """Host threads the oracle may use: this process's CPU affinity, capped by
    OMP_NUM_THREADS when that is set (the GPU host's share of cores)."""
    n = len(os.sched_getaffinity(0))
    try:
        cap = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        cap = 0
    return min(n, cap) if cap > 0 else n


def _oracle_sample(wl, x):
    """The bounded sample of a workload the CPU oracle is timed on, as a list of
    (workload, layer inputs) and its description: whole layers for c1/c2, four distinct
    layers for c3, sequence 0 of layers 0 and 1 for c4 (same seeds as in the full batch)."""
    import dge_inputs as di
    if wl.n_layers == 1:
        return [(wl, x)], f"one {wl.name} layer"
    if wl.batch == 1:
        return ([(wl, x)] + [(wl, di.make_layer(wl, layer=l)) for l in (1, 2, 3)],
                f"layers 0-3 of {wl.name}")
    w1 = di.small_variant(wl.name, [wl.prompt_lens[0]], name=f"{wl.name}_seq0")
    return ([(w1, di.make_layer(w1, layer=l)) for l in (0, 1)],
            f"sequence 0 (L={wl.prompt_lens[0]}) of layers 0 and 1 of {wl.name}")


def _time_oracle(sample, seconds):
    import oracle
    reps = units = 0
    t0 = time.perf_counter()
    while True:
        w, xl = sample[reps % len(sample)]
        oracle.evict_layer(xl.q, xl.k, xl.v, w.kv_offsets, w.n_q_heads, w.n_kv_heads, w.window,
                           w.k_draft, w.budget_of_layer(xl.layer), w.pool)
        reps += 1
        units += sum(w.prompt_lens) * w.n_kv_heads
        el = time.perf_counter() - t0
        if el >= seconds and reps >= len(sample):
            return reps, units, el


def cpu_baseline(wl, x, seconds):
    """The float64 oracle, untuned, on this host's cores, timed on a bounded sample of the
    workload (score, pool, select, compact of each sampled layer); the rate is per prefix
    token x KV head, and the whole step's time is extrapolated from it."""
    from threadpoolctl import threadpool_limits
    threads = cpu_threads()
    sample, what = _oracle_sample(wl, x)
    with threadpool_limits(limits=threads):
        reps, units, el = _time_oracle(sample, seconds)
    rate = units / el
    step_units = sum(wl.prompt_lens) * wl.n_kv_heads * wl.n_layers
    log(f"[bench] cpu oracle ({threads} threads): {reps} layer passes over {what} in {el:.1f}s "
        f"-> {rate:.3g} token*kvhead/s")
    one = None
    with threadpool_limits(limits=1):
        r1, u1, e1 = _time_oracle(sample, seconds / 3)
    one = round(u1 / e1, 1)
    log(f"[bench] cpu oracle, one thread: {r1} layer passes in {e1:.1f}s -> {one:.3g} token*kvhead/s")
    return {"value": round(rate, 1), "unit": "token*kvhead/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} passes over {what} (score, pool, select, compact; float64 numpy), "
                      f"{el:.1f} s; the full step's {step_units} token*kvheads would take "
                      f"{step_units / rate:.0f} s (extrapolated)",
            "affinity_cpus": len(os.sched_getaffinity(0)), "value_one_core": one}


if __name__ == "__main__":
    main()
