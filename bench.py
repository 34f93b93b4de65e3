#!/usr/bin/env python3
"""Throughput of the fractal KV-archive hot path on one MI355X.

One step is one pass of the whole path over one batch of synthetic K/V:
residual-VQ assignment of every archived head vector with the fixed-span
encode of the resulting symbol streams fused into the same kernel, bulk decode
of every span, and a batch of random O(1) lookups.  The separate assignment and
encode kernels are timed too (their rooflines are reported beside the fused
one).  Inputs are resident in device memory before the timed region.

Prints one JSON line.  `value` is archived tokens per second over the whole
step (a token is one position across all layers, heads and K/V); per-phase
rates, the dominant kernel's roofline fraction and the CPU oracle's rate on the
same workload are reported beside it.  `other_workloads` gives the GPT-2-shaped
and hybrid workloads' step rate and, per group, the fused kernel against the
matrix peak and HBM and the bulk decode against HBM.  The step is captured once as a HIP graph
and replayed (no host launch overhead in the timed region); each kernel's
average duration comes from a graph of back-to-back launches of that kernel.
`reference_rates` gives what a library fp16 GEMM and a streaming elementwise
kernel reach on the same device, and each roofline entry its achieved rate as
a fraction of that (`frac_of_reference`) beside the datasheet fraction; it also
gives the rate of the library's matrix-core loop (the assignment's instruction
back to back from registers), and the matrix-bound entries their fraction of
it (`frac_of_mfma_loop`).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP16_MFMA_TFLOPS = 2500.0   # MI355X dense fp16 matrix peak
PEAK_HBM_GBS = 8000.0            # MI355X HBM3E bandwidth
METRIC = "archived tokens/s (RVQ assign + CGR encode) and decoded symbols/s, 1 MI355X"


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_07144_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "rvq_assign_encode": ("rvq_kernels.hip", "fkv_hip_common.h", "fkv_internal.h"),
    "rvq_assign": ("rvq_kernels.hip", "fkv_hip_common.h", "fkv_internal.h"),
    "cgr_encode": ("cgr_kernels.hip", "cgr_device.h", "fkv_hip_common.h", "fkv_internal.h"),
    "cgr_decode": ("cgr_kernels.hip", "cgr_device.h", "fkv_hip_common.h", "fkv_internal.h"),
    "span_lookup": ("cgr_kernels.hip", "cgr_device.h", "fkv_hip_common.h", "fkv_internal.h"),
}


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None when absent or
    taken on a different version of the kernel's source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(workload, {}).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != source_hash(*KERNEL_SOURCES[kernel]):
        return None
    return rec.get("bytes_per_launch")


def build_workload(name: str, n_lookups: int):
    import torch
    from paper_2607_07144_amd import fkv, workloads

    cfg = workloads.CONFIGS[name]
    groups = []
    for gi, g in enumerate(cfg.groups):
        if name == "long_gqa":
            x, books, sb = workloads.make_group_torch(cfg, gi)
            host = None
        else:
            xh, bh, sbh = workloads.make_group_numpy(cfg, gi)
            x, books, sb = (torch.from_numpy(a).cuda() for a in (xh, bh, sbh))
            host = (xh, bh, sbh)
        ns = x.shape[0]
        codec = fkv.Codec(g.N, g.r_scale)
        n_sym = cfg.T_arch * g.S
        n_spans = codec.n_spans(n_sym)
        rng = np.random.default_rng(cfg.seed + 17 * gi)
        qs = rng.integers(0, ns, size=n_lookups).astype(np.int32)
        qt = rng.integers(0, cfg.T_arch, size=n_lookups).astype(np.int32)
        groups.append(dict(
            g=g, codec=codec, x=x, books=books, sb=sb, host=host, ns=ns, n_sym=n_sym, n_spans=n_spans,
            sym=torch.empty((ns, n_sym), dtype=torch.uint8, device="cuda"),
            pts=torch.empty((ns, n_spans, 2), dtype=torch.float64, device="cuda"),
            dec=torch.empty((ns, n_sym), dtype=torch.uint8, device="cuda"),
            qs=torch.from_numpy(qs).cuda(), qt=torch.from_numpy(qt).cuda(), qs_h=qs, qt_h=qt,
            out=torch.empty((n_lookups, g.S), dtype=torch.uint8, device="cuda"),
        ))
    return cfg, groups


def run_kernel(fkv, cfg, groups, name):
    """One launch of one step kernel for every group, on the current stream."""
    for gr in groups:
        if name == "rvq_assign_encode":
            fkv.fkv_rvq_assign_encode(gr["codec"], gr["x"], gr["books"], gr["sb"], cfg.t_begin, cfg.t_end,
                                      symbols=gr["sym"], points=gr["pts"])
        elif name == "rvq_assign":
            fkv.fkv_rvq_assign(gr["x"], gr["books"], gr["sb"], cfg.t_begin, cfg.t_end, symbols=gr["sym"])
        elif name == "cgr_encode":
            fkv.fkv_cgr_encode_spans(gr["codec"], gr["sym"], points=gr["pts"])
        elif name == "cgr_decode":
            fkv.fkv_cgr_decode_spans(gr["codec"], gr["pts"], gr["n_sym"], symbols=gr["dec"])
        else:
            fkv.fkv_span_lookup(gr["codec"], gr["pts"], gr["n_sym"], gr["g"].S, gr["qs"], gr["qt"],
                                out=gr["out"])


STEP = ("rvq_assign_encode", "cgr_decode", "span_lookup")


def run_step(fkv, cfg, groups):
    """One pass of the whole path per group: assignment and span encode in one call (the fused kernel,
    or from 2^23 head vectors on the assignment kernel and then the encode kernel), bulk decode, random
    lookups."""
    for gr in groups:
        for name in STEP:
            run_kernel(fkv, cfg, [gr], name)


def algorithmic(cfg, groups):
    """Algorithmic FLOPs / bytes per launch of each kernel, summed over groups."""
    a = {"rvq_assign": {"flops": 0, "bytes": 0}, "cgr_encode": {"bytes": 0}, "cgr_decode": {"bytes": 0},
         "span_lookup": {"bytes": 0}, "symbols": 0, "lookups": 0, "head_vectors": 0}
    for gr in groups:
        g, ns, d = gr["g"], gr["ns"], cfg.d
        nb = gr["books"].shape[0]
        a["rvq_assign"]["flops"] += ns * cfg.T_arch * g.S * 2 * g.K * d
        a["rvq_assign"]["bytes"] += ns * cfg.T_arch * d * 2 + nb * g.S * g.K * d * 2 + ns * cfg.T_arch * g.S
        codec_bytes = ns * gr["n_sym"] + ns * gr["n_spans"] * 16
        a.setdefault("rvq_assign_encode", {"flops": 0, "bytes": 0})
        a["rvq_assign_encode"]["flops"] += ns * cfg.T_arch * g.S * 2 * g.K * d
        a["rvq_assign_encode"]["bytes"] += (ns * cfg.T_arch * d * 2 + nb * g.S * g.K * d * 2 + ns * gr["n_sym"] +
                                            ns * gr["n_spans"] * 16)
        a["cgr_encode"]["bytes"] += codec_bytes
        a["cgr_decode"]["bytes"] += codec_bytes
        L = gr["codec"].L
        qt = gr["qt_h"].astype(np.int64) * g.S
        spans_touched = (qt + g.S - 1) // L - qt // L + 1
        a["span_lookup"]["bytes"] += int(gr["qs_h"].size * (8 + g.S) + 16 * spans_touched.sum())
        a["symbols"] += ns * gr["n_sym"]
        a["lookups"] += gr["qs_h"].size
        a["head_vectors"] += ns * cfg.T_arch
    return a


SETTLE_S = 0.2   # --settle-s


def time_graph(fn, reps: int, replays: int, stream, settle_s: float | None = None):
    """Average duration of one fn() call: a graph of `reps` back-to-back calls, replayed and
    bracketed by events on the stream the replays run on.  Before timing, the graph is replayed
    for at least `settle_s` seconds, so that the call is timed in its own steady state: after a
    phase at the board's power limit (the assignment) the shader clock takes a while to recover,
    and a kernel timed right after it would carry that phase's clock."""
    import torch

    if settle_s is None:
        settle_s = SETTLE_S
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for _ in range(reps):
            fn()
    t0 = time.perf_counter()
    g.replay()
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < settle_s:
        g.replay()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3 / (reps * replays)


def other_workloads(fkv, side, names, n_lookups: int, steps: int, warmup: int, cpu: bool):
    """The GPT-2-shaped and hybrid workloads measured the same way as the headline one, per group:
    the fused assignment + encode launch against the matrix peak and against HBM (the hybrid
    value group is HBM-bound), bulk decode against HBM, and the whole step as archived tokens/s.
    With `cpu`, the oracle is timed and checks the GPU on the GPT-2 shape in full and on the first
    64 streams of each hybrid group."""
    import torch

    out = {}
    for name in names:
        cfg, groups = build_workload(name, n_lookups)
        with torch.cuda.stream(side):
            for _ in range(max(1, warmup)):
                run_step(fkv, cfg, groups)
        torch.cuda.synchronize()
        step_s = time_graph(lambda: run_step(fkv, cfg, groups), 1, max(1, steps), side)
        per_group = []
        for gr in groups:
            g, ns, d = gr["g"], gr["ns"], cfg.d
            nb = gr["books"].shape[0]
            flops = ns * cfg.T_arch * g.S * 2 * g.K * d
            fused_bytes = (ns * cfg.T_arch * d * 2 + nb * g.S * g.K * d * 2 + ns * gr["n_sym"] +
                           ns * gr["n_spans"] * 16)
            codec_bytes = ns * gr["n_sym"] + ns * gr["n_spans"] * 16
            t_f = time_graph(lambda: run_kernel(fkv, cfg, [gr], "rvq_assign_encode"), 10, max(1, steps // 4), side)
            t_d = time_graph(lambda: run_kernel(fkv, cfg, [gr], "cgr_decode"), 10, max(1, steps // 4), side)
            per_group.append({
                "kinds": list(g.kinds), "S": g.S, "K": g.K, "N": g.N, "L": gr["codec"].L, "streams": ns,
                "rvq_assign_encode": {"avg_launch_us": round(t_f * 1e6, 2),
                                      "tflops": round(flops / t_f / 1e12, 2),
                                      "mfma_frac": round(flops / t_f / 1e12 / PEAK_FP16_MFMA_TFLOPS, 4),
                                      "gbs": round(fused_bytes / t_f / 1e9, 1),
                                      "hbm_frac": round(fused_bytes / t_f / 1e9 / PEAK_HBM_GBS, 4)},
                "cgr_decode": {"avg_launch_us": round(t_d * 1e6, 2), "gbs": round(codec_bytes / t_d / 1e9, 1),
                               "hbm_frac": round(codec_bytes / t_d / 1e9 / PEAK_HBM_GBS, 4)},
            })
        out[name] = {"description": cfg.description, "archived_tokens_per_s": round(cfg.batch * cfg.T_arch / step_s, 1),
                     "ms_per_step": round(step_s * 1e3, 5), "groups": per_group}
        if cpu:
            out[name]["cpu_oracle"] = cpu_baseline(cfg, groups, max(gr["ns"] for gr in groups) if name == "gpt2" else 64,
                                                   cfg.T_arch, 8, 384)
        del groups
        torch.cuda.empty_cache()
    return out


def next_rows(fkv, cfg, groups, side, replays: int, cpu: bool = False):
    """Measurements of the rows beyond the step: rehydration of the step's lookup queries, one
    decoding step's archive update (the position leaving the recent window is assigned on every
    stream and its symbols appended) and one Lloyd iteration of codebook training.  With `cpu`, the
    oracle is timed on a bounded sample of each and checks the GPU's results there."""
    import torch

    res = {"rehydrate": {"queries": 0, "bytes": 0, "s": 0.0}, "evict_append": {"s": 0.0, "bytes": 0}}
    with torch.cuda.stream(side):
        for gr in groups:
            g = gr["g"]
            nq = gr["qs"].numel()
            out = torch.empty((nq, cfg.d), dtype=torch.float16, device="cuda")
            t = time_graph(lambda: fkv.fkv_rehydrate(gr["codec"], gr["pts"], gr["n_sym"], g.S, gr["books"],
                                                     gr["sb"], gr["qs"], gr["qt"], out=out), 10, replays, side)
            L = gr["codec"].L
            qt = gr["qt_h"].astype(np.int64) * g.S
            spans = int(((qt + g.S - 1) // L - qt // L + 1).sum())
            res["rehydrate"]["queries"] += nq
            res["rehydrate"]["bytes"] += nq * (8 + g.S * cfg.d * 2 + cfg.d * 2) + 16 * spans
            res["rehydrate"]["s"] += t
            # one eviction: token t_end - 1 of every stream, appended after the archived symbols; the
            # assignment takes the streams of each book together (one block per book's streams)
            ns = gr["ns"]
            n_old = gr["n_sym"] - g.S
            pts = gr["pts"].clone()
            sym1 = torch.empty((ns, g.S), dtype=torch.uint8, device="cuda")
            grp = torch.from_numpy(fkv.book_groups(gr["sb"].cpu().numpy())).cuda()

            def step():
                fkv.fkv_rvq_assign_groups(gr["x"], gr["books"], gr["sb"], grp, cfg.t_end - 1, cfg.t_end,
                                          symbols=sym1)
                fkv.fkv_cgr_append(gr["codec"], pts, n_old, sym1)

            res["evict_append"]["s"] += time_graph(step, 10, replays, side)
            res["evict_append"]["bytes"] += ns * (cfg.d * 2 + g.S) + gr["books"].numel() * 2 + ns * 32
            res["evict_append"]["groups"] = res["evict_append"].get("groups", 0) + int(grp.shape[0])
            res["evict_append"]["group_size"] = int(grp.shape[1])
            # one Lloyd iteration of codebook training over every stage (assign, accumulate, update)
            bk = gr["books"].clone()
            nb, S, K = bk.shape[0], bk.shape[1], bk.shape[2]
            symk = torch.empty_like(gr["sym"])
            sums = torch.zeros((nb, K, cfg.d), dtype=torch.int64, device="cuda")
            counts = torch.zeros((nb, K), dtype=torch.int32, device="cuda")

            def lloyd():
                for stage in range(S):
                    # the update of `stage` uses the assignment of stages 0..stage only
                    fkv.fkv_rvq_assign(gr["x"], bk, gr["sb"], cfg.t_begin, cfg.t_end, symbols=symk,
                                       n_stages=stage + 1)
                    fkv.fkv_kmeans_step(gr["x"], bk, gr["sb"], cfg.t_begin, cfg.t_end, symk, stage, sums=sums,
                                        counts=counts)

            res.setdefault("kmeans", {"s": 0.0, "books": 0})
            res["kmeans"]["s"] += time_graph(lloyd, 2, replays, side)
            res["kmeans"]["books"] += nb
    rh, ev = res["rehydrate"], res["evict_append"]
    ach = rh["bytes"] / rh["s"] / 1e9
    cpu_res = next_rows_oracle(fkv, cfg, groups[0]) if cpu else None
    return {
        "cpu_oracle": cpu_res,
        "rehydrate": {"queries": rh["queries"], "avg_launch_us": round(rh["s"] / len(groups) * 1e6, 2),
                      "queries_per_s": round(rh["queries"] / rh["s"], 1),
                      "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                   "frac": round(ach / PEAK_HBM_GBS, 4)}},
        "evict_append": {"us_per_decoding_step": round(ev["s"] * 1e6, 2),
                         "positions_per_s": round(1.0 / ev["s"], 1),
                         "streams": sum(gr["ns"] for gr in groups),
                         "assignment": "grouped by book: %d groups of %d streams" % (ev["groups"], ev["group_size"])},
        "kmeans": {"ms_per_lloyd_iteration": round(res["kmeans"]["s"] * 1e3, 4),
                   "books": res["kmeans"]["books"],
                   "note": "every stage s: assignment of stages 0..s, cluster sums, centroid update"},
    }


def next_rows_oracle(fkv, cfg, gr):
    """The oracle on this host for the rows beyond the step, each on a bounded sample of the first
    group and scaled to the whole workload, and as checker of the GPU's results on that sample:
    rehydration of the step's queries (outputs rounded once to binary16, statuses), the eviction
    step on 64 streams (teacher-forced assignment, appended points bit for bit against a fresh GPU
    append), and a stage-0 Lloyd update on the streams of the first 16 books over their first 1536
    archived tokens (new codewords bit for bit against the GPU's update of the same sample)."""
    import torch
    import oracle

    g = gr["g"]
    S, L, ns, n_sym = g.S, gr["codec"].L, gr["ns"], gr["n_sym"]
    threads = oracle.default_threads()
    oc = oracle.Codec(g.N, g.r_scale)
    books_h = gr["books"].cpu().numpy()
    sb_h = gr["sb"].cpu().numpy()
    pts_h = gr["pts"].cpu().numpy()
    out = {"cores": threads, "cpu_model": cpu_model(), "kind": "oracle"}

    # rehydration of the step's queries
    nq = gr["qs"].numel()
    gout = fkv.fkv_rehydrate(gr["codec"], gr["pts"], n_sym, S, gr["books"], gr["sb"], gr["qs"], gr["qt"])
    t0 = time.perf_counter()
    want, wst, _ = oracle.rehydrate(oc, pts_h, n_sym, S, books_h, sb_h, gr["qs_h"].astype(np.uint32),
                                    gr["qt_h"].astype(np.uint32), threads=threads)
    t1 = time.perf_counter()
    out["rehydrate"] = {"queries": nq, "queries_per_s": round(nq / (t1 - t0), 1),
                        "output_mismatches": int((want.astype(np.float16).view(np.uint16) !=
                                                  gout.cpu().numpy().view(np.uint16)).any(axis=1).sum()),
                        "status_nonzero": int((wst != 0).sum())}

    # the eviction step on the first 64 streams: assignment of token t_end - 1, then append
    n_s = min(64, ns)
    n_old = n_sym - S
    sym1 = torch.empty((ns, S), dtype=torch.uint8, device="cuda")
    grp = torch.from_numpy(fkv.book_groups(sb_h)).cuda()
    fkv.fkv_rvq_assign_groups(gr["x"], gr["books"], gr["sb"], grp, cfg.t_end - 1, cfg.t_end, symbols=sym1)
    pts2 = gr["pts"].clone()
    fkv.fkv_cgr_append(gr["codec"], pts2, n_old, sym1)
    sym1_h = sym1.cpu().numpy()
    x1 = gr["x"][:n_s, cfg.t_end - 1:cfg.t_end].cpu().numpy()
    t0 = time.perf_counter()
    ra = oracle.rvq_assign(x1, books_h, sb_h[:n_s], 0, 1, force=sym1_h[:n_s], want_residual=False,
                           want_gaps=False, threads=threads)
    opts = oracle.append(oc, pts_h[:n_s], n_old, ra["symbols"], threads=threads)
    t1 = time.perf_counter()
    out["evict_append"] = {"streams": n_s, "us_per_decoding_step": round((t1 - t0) / n_s * ns * 1e6, 1),
                           "hard_mismatches": ra["n_hard"], "teacher_forced": ra["n_forced"],
                           "point_mismatches": int((opts.view(np.uint64) !=
                                                    pts2[:n_s].cpu().numpy().view(np.uint64)).any(axis=2).sum())}

    # a stage-0 Lloyd update on the streams of the first 16 books, first 1536 archived tokens
    nb_s = min(16, int(books_h.shape[0]))
    sel = np.nonzero(sb_h < nb_s)[0]
    te = min(cfg.t_end, cfg.t_begin + 1536)
    bk_s = gr["books"][:nb_s].clone()
    symk = torch.empty((ns, (te - cfg.t_begin) * S), dtype=torch.uint8, device="cuda")
    nbad = torch.zeros(1, dtype=torch.int32, device="cuda")   # the other streams' books are not in the sample
    fkv.fkv_rvq_assign(gr["x"], bk_s, gr["sb"], cfg.t_begin, te, symbols=symk, n_bad=nbad, n_stages=1)
    fkv.fkv_kmeans_step(gr["x"], bk_s, gr["sb"], cfg.t_begin, te, symk, 0)
    xs = gr["x"][torch.from_numpy(sel).cuda(), :te].cpu().numpy()
    syms = symk.cpu().numpy()[sel]
    t0 = time.perf_counter()
    new, _, counts = oracle.kmeans_update(xs, books_h[:nb_s], sb_h[sel], cfg.t_begin, te, syms, 0)
    t1 = time.perf_counter()
    tok = len(sel) * (te - cfg.t_begin)
    out["kmeans_stage0_update"] = {
        "sample": "%d streams (books 0..%d) x first %d archived tokens" % (len(sel), nb_s - 1, te - cfg.t_begin),
        "ms_per_stage_update_whole_workload": round((t1 - t0) / tok * ns * (cfg.t_end - cfg.t_begin) * 1e3, 1),
        "codeword_mismatches": int((new[:, 0].view(np.uint16) != bk_s[:, 0].cpu().numpy().view(np.uint16))
                                   .any(axis=2).sum()),
        "members": int(counts.sum())}
    return out


def read_stress(fkv, side, replays: int, cpu: bool = False):
    """Read side at HBM scale: the 144-stream x 131,072-token archive (2 symbols per token, N = 256).
    Bulk decode rotates over 4 copies of the points so that consecutive launches do not hit the
    memory-side cache; 2^20 random lookups, beside a library gather of the same queries' points (the
    random-transaction bound); the per-position retrieval index (build and one suffix scan of 16
    bytes per position)."""
    import torch
    from paper_2607_07144_amd import workloads

    c = workloads.READ_STRESS
    sym_h, qs_h, qt_h = workloads.read_stress_inputs()
    codec = fkv.Codec(c["N"])
    ns, n_sym = sym_h.shape
    sym = torch.from_numpy(sym_h).cuda()
    pts = fkv.fkv_cgr_encode_spans(codec, sym)
    copies = [pts] + [pts.clone() for _ in range(3)]
    dec = torch.empty_like(sym)
    qs, qt = torch.from_numpy(qs_h.astype(np.int32)).cuda(), torch.from_numpy(qt_h.astype(np.int32)).cuda()
    out = torch.empty((qs.numel(), c["S"]), dtype=torch.uint8, device="cuda")
    traj = torch.empty((ns, n_sym, 2), dtype=torch.float64, device="cuda")
    query = sym[5, 1000:1003].contiguous()
    hits = torch.empty((1 << 16, 2), dtype=torch.int32, device="cuda")
    nh = torch.zeros(1, dtype=torch.int32, device="cuda")
    rot = [0]

    def decode():
        fkv.fkv_cgr_decode_spans(codec, copies[rot[0] % 4], n_sym, symbols=dec)
        rot[0] += 1

    with torch.cuda.stream(side):
        t_dec = time_graph(decode, 8, replays, side)
        rot[0] = 0

        def lookup():
            fkv.fkv_span_lookup(codec, copies[rot[0] % 4], n_sym, c["S"], qs, qt, out=out)
            rot[0] += 1

        t_lk = time_graph(lookup, 8, replays, side)
        t_tr = time_graph(lambda: fkv.fkv_trajectory(codec, sym, traj=traj), 2, replays, side)
        t_sc = time_graph(lambda: fkv.fkv_suffix_search(codec, traj, query, max_hits=1 << 16, hits=hits,
                                                        n_hits=nh), 4, replays, side)
        t_ga = gather_reference(copies, qs_h, qt_h, c["S"], L=codec.L, stream=side)
    lk_err = int((out != sym.view(ns, -1, c["S"])[qs.long(), qt.long()]).any(dim=1).sum().item())
    nf = torch.zeros(1, dtype=torch.int32, device="cuda")
    fkv.fkv_cgr_decode_spans(codec, pts, n_sym, symbols=dec, n_failed=nf)
    dec_err = int((dec != sym).sum().item())
    n_pos = ns * n_sym
    dec_bytes = n_pos + pts.numel() * 8
    L = codec.L
    a = qt_h.astype(np.int64) * c["S"]
    lk_bytes = int(qs_h.size * (8 + c["S"]) + 16 * ((a + c["S"] - 1) // L - a // L + 1).sum())
    hbm = lambda b, t: {"bound": "hbm", "achieved": round(b / t / 1e9, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(b / t / 1e9 / PEAK_HBM_GBS, 4)}
    cpu_res = None
    if cpu:
        # the oracle on this host: encode and bulk decode of the first 16 streams, and the first
        # 65,536 queries, each scaled to the whole archive / all queries; and as checker of the
        # GPU's points, decoded symbols and lookups there
        import oracle

        threads = oracle.default_threads()
        oc = oracle.Codec(c["N"])
        n_s = 16
        t0 = time.perf_counter()
        opts = oracle.encode(oc, sym_h[:n_s], threads=threads)
        t1 = time.perf_counter()
        odec, _, onf, _ = oracle.decode(oc, opts, n_sym, threads=threads)
        t2 = time.perf_counter()
        nq = 1 << 16
        oq = qs_h[:nq].astype(np.uint32), qt_h[:nq].astype(np.uint32)
        lpts = pts.cpu().numpy()
        t3 = time.perf_counter()
        lout, lst, _ = oracle.lookup(oc, lpts, n_sym, c["S"], oq[0], oq[1], threads=threads)
        t4 = time.perf_counter()
        gpts = pts[:n_s].cpu().numpy()
        # the retrieval index of the first 16 streams and one suffix scan over it (hits within those streams)
        t5 = time.perf_counter()
        otraj = oracle.trajectory(oc, sym_h[:n_s], codec.L, threads=threads)
        t6 = time.perf_counter()
        oh, onh, _ = oracle.suffix_search(oc, otraj, query.cpu().numpy(), verify=True, max_hits=1 << 16)
        t7 = time.perf_counter()
        # a fresh GPU scan (the timed replays accumulate into one hit counter)
        gh_t, gnh, _ = fkv.fkv_suffix_search(codec, traj, query, max_hits=1 << 16)
        gh = gh_t[:int(gnh.item())].cpu().numpy()
        gh = gh[gh[:, 0] < n_s]
        cpu_res = {"cores": threads, "cpu_model": cpu_model(), "kind": "oracle",
                   "sample": "encode, bulk decode, index build and one suffix scan of the first %d of %d streams, "
                             "lookups of the first %d of %d queries, scaled to the whole archive"
                             % (n_s, ns, nq, qs_h.size),
                   "index_positions_per_s": round(n_s * n_sym / (t6 - t5), 1),
                   "suffix_scan_positions_per_s": round(n_s * n_sym / (t7 - t6), 1),
                   "encode_symbols_per_s": round(n_s * n_sym / (t1 - t0), 1),
                   "decode_symbols_per_s": round(n_s * n_sym / (t2 - t1), 1),
                   "lookups_per_s": round(nq / (t4 - t3), 1),
                   "checks": {"point_mismatches": int((opts.view(np.uint64) != gpts.view(np.uint64)).any(axis=2).sum()),
                              "oracle_decode_failed_spans": int(onf),
                              "decode_symbol_mismatches": int((odec != dec[:n_s].cpu().numpy()).sum()),
                              "lookup_mismatches": int((lout != out[:nq].cpu().numpy()).any(axis=1).sum()),
                              "lookup_status_nonzero": int((lst != 0).sum()),
                              "index_mismatches": int((otraj.view(np.uint64) !=
                                                       traj[:n_s].cpu().numpy().view(np.uint64)).any(axis=2).sum()),
                              "suffix_hits": int(onh),
                              "suffix_hit_set_equal": sorted(map(tuple, oh.astype(np.int64).tolist())) ==
                                                      sorted(map(tuple, gh.astype(np.int64).tolist()))}}
    return {
        "archive": "%d streams x %d symbols, N=%d, L=%d" % (ns, n_sym, c["N"], L),
        "cpu_oracle": cpu_res,
        "bulk_decode": {"avg_launch_us": round(t_dec * 1e6, 2), "symbols_per_s": round(n_pos / t_dec, 1),
                        "roofline": hbm(dec_bytes, t_dec), "rotation": 4, "decode_failed_spans": int(nf.item()),
                        "roundtrip_symbol_errors": dec_err},
        "lookup": {"queries": int(qs_h.size), "avg_launch_us": round(t_lk * 1e6, 2),
                   "lookups_per_s": round(qs_h.size / t_lk, 1), "roofline": hbm(lk_bytes, t_lk),
                   "rotation": 4, "lookup_errors": lk_err,
                   "gather_reference": {"op": "torch.index_select of the queries' 16-byte points as complex128 "
                                              "(same archive, same 4-copy rotation)",
                                        "avg_launch_us": round(t_ga * 1e6, 2),
                                        "gathers_per_s": round(qs_h.size / t_ga, 1)},
                   "frac_of_reference": round(t_ga / t_lk, 4)},
        "index_build": {"avg_launch_us": round(t_tr * 1e6, 2), "positions_per_s": round(n_pos / t_tr, 1),
                        "roofline": hbm(n_pos * 17, t_tr)},
        "suffix_scan": {"avg_launch_us": round(t_sc * 1e6, 2), "positions_per_s": round(n_pos / t_sc, 1),
                        "query_len": 3, "roofline": hbm(n_pos * 16, t_sc)},
    }


def gather_reference(copies, qs_h, qt_h, S: int, L: int, stream, reps: int = 8, replays: int = 5):
    """The random-transaction bound of the lookups: a library gather (torch.index_select) of the
    same queries' 16-byte points from the same archive, with no decoding, rotating over the same
    copies as the lookups (so that neither is served from the memory-side cache).  Each query of
    this archive touches one span, so lookups/s and gathers/s compare one to one.  Timed eagerly:
    `reps` back-to-back gathers between events on `stream`, best of `replays`."""
    import torch

    n_spans = copies[0].shape[1]
    rows = qs_h.astype(np.int64) * n_spans + (qt_h.astype(np.int64) * S) // L
    # one complex128 element per point, so that each gathered element is one 16-byte load
    flats = [p.reshape(-1, 2).view(torch.complex128).reshape(-1) for p in copies]
    idx = torch.from_numpy(rows).to(flats[0].device)
    dst = torch.empty(idx.numel(), dtype=flats[0].dtype, device=flats[0].device)
    best = float("inf")
    with torch.cuda.stream(stream):
        torch.index_select(flats[0], 0, idx, out=dst)
        for _ in range(replays):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for k in range(reps):
                torch.index_select(flats[k % len(flats)], 0, idx, out=dst)
            e1.record(stream)
            e1.synchronize()
            best = min(best, e0.elapsed_time(e1) / 1e3 / reps)
    return best


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _span_prefix(T_arch: int, S: int, L: int, want: int) -> int:
    """The largest token count <= want whose symbols fill whole spans (all tokens if want >= T_arch)."""
    if want >= T_arch:
        return T_arch
    n = want
    while n > 0 and (n * S) % L:
        n -= 1
    return max(n, 1)


def cpu_baseline(cfg, groups, max_streams: int, max_tokens: int, st_streams: int, st_tokens: int):
    """The CPU oracle on a bounded sample of the same step, timed on this host, and the oracle as
    checker of the GPU's outputs on that sample.

    Sample: the first `max_streams` streams of each group (the first layer's streams: streams are
    ordered layer-major) on their first `max_tokens` archived tokens (a whole number of spans).
    The all-cores leg runs the full step there (RVQ, encode, decode, and the step's lookups that
    fall in the sample) with OpenMP over streams; the single-thread leg runs RVQ, encode and decode
    on `st_streams` x `st_tokens` of the same sample.  Both are scaled per stream-token (lookups
    per query) to the whole workload.  As checker, the all-cores leg takes the GPU's symbols as
    teacher (near-ties within 1e-5 relative are accepted and counted per stage; any other
    difference is a hard mismatch) and compares the GPU's points, decoded symbols and lookups bit
    for bit."""
    import torch
    import oracle

    threads = oracle.default_threads()
    t_all = t_one = 0.0
    sample, check = [], []
    for gi, gr in enumerate(groups):
        g, L = gr["g"], gr["codec"].L
        ns = min(gr["ns"], max_streams)
        nt = _span_prefix(cfg.T_arch, g.S, L, max_tokens)
        n_sym = nt * g.S
        xh = gr["x"][:ns, :cfg.t_begin + nt].cpu().numpy() if gr["host"] is None else gr["host"][0][:ns, :cfg.t_begin + nt]
        bh = gr["books"].cpu().numpy()
        sbh = gr["sb"][:ns].cpu().numpy()
        gsym = gr["sym"][:ns, :n_sym].cpu().numpy()
        gpts = gr["pts"][:ns, :(n_sym + L - 1) // L].cpu().numpy()
        gdec = gr["dec"][:ns, :n_sym].cpu().numpy()
        keep = (gr["qs_h"] < ns) & (gr["qt_h"] < nt)
        qs, qt = gr["qs_h"][keep].astype(np.uint32), gr["qt_h"][keep].astype(np.uint32)
        gout = gr["out"].cpu().numpy()[keep]
        oc = oracle.Codec(g.N, g.r_scale)

        t0 = time.perf_counter()
        o = oracle.rvq_assign(xh, bh, sbh, cfg.t_begin, cfg.t_begin + nt, force=gsym, force_tol=1e-5,
                              want_residual=False, want_gaps=True, threads=threads)
        pts = oracle.encode(oc, o["symbols"], threads=threads)
        dsym, _, nfail, _ = oracle.decode(oc, pts, n_sym, threads=threads)
        t1 = time.perf_counter()
        lout, _, _ = oracle.lookup(oc, pts, n_sym, g.S, qs, qt, threads=threads)
        t2 = time.perf_counter()
        scale_tok = gr["ns"] * cfg.T_arch / (ns * nt)
        t_all += (t1 - t0) * scale_tok + (t2 - t1) * gr["qs_h"].size / max(1, int(keep.sum()))

        sn, stt = min(ns, st_streams), _span_prefix(cfg.T_arch, g.S, L, st_tokens)
        t0 = time.perf_counter()
        o1 = oracle.rvq_assign(xh[:sn, :cfg.t_begin + stt], bh, sbh[:sn], cfg.t_begin, cfg.t_begin + stt,
                               want_residual=False, want_gaps=False, threads=1)
        p1 = oracle.encode(oc, o1["symbols"], threads=1)
        oracle.decode(oc, p1, stt * g.S, threads=1)
        t_one += (time.perf_counter() - t0) * gr["ns"] * cfg.T_arch / (sn * stt)

        gaps = o["gaps"].reshape(ns, nt, g.S)
        check.append({
            "group": gi, "streams": ns, "tokens_per_stream": nt,
            "assignments_per_stage": ns * nt,
            "near_ties_per_stage": [int((gaps[:, :, st] < 1e-5).sum()) for st in range(g.S)],
            "teacher_forced": o["n_forced"], "hard_mismatches": o["n_hard"],
            "symbols_equal": bool(np.array_equal(o["symbols"], gsym)),
            "point_mismatches": int((pts.view(np.uint64) != gpts.view(np.uint64)).any(axis=2).sum()),
            "oracle_decode_failed_spans": int(nfail),
            "decode_symbol_mismatches": int((dsym != gdec).sum()),
            "lookups_checked": int(keep.sum()), "lookup_mismatches": int((lout != gout).any(axis=1).sum()),
        })
        sample.append("%d/%d streams x first %d/%d archived tokens" % (ns, gr["ns"], nt, cfg.T_arch))
    tokens = cfg.batch * cfg.T_arch
    return {"value": tokens / t_all, "unit": "archived tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "single_thread": {"value": tokens / t_one, "cores": 1,
                              "sample": "RVQ, encode and decode on the first %d streams x first %d archived "
                                        "tokens of each group, scaled per stream-token" % (st_streams, st_tokens)},
            "sample": "%s of %s (full step on the sample: RVQ, encode, decode and the step's lookups that fall "
                      "in it), time scaled per stream-token (lookups per query) to the whole workload"
                      % ("; ".join(sample), cfg.name),
            "checks": check}


def gpu_checks(fkv, cfg, groups):
    """Whole-workload checks on the GPU after the timed region: decode failures counted by the
    kernel's own counter, round-trip symbol errors (decoded vs assigned) and lookup errors
    (looked-up vs assigned), per group."""
    import torch

    out = []
    for gr in groups:
        nf = torch.zeros(1, dtype=torch.int32, device="cuda")
        fkv.fkv_cgr_decode_spans(gr["codec"], gr["pts"], gr["n_sym"], symbols=gr["dec"], n_failed=nf)
        fkv.fkv_span_lookup(gr["codec"], gr["pts"], gr["n_sym"], gr["g"].S, gr["qs"], gr["qt"], out=gr["out"])
        S = gr["g"].S
        sym = gr["sym"].view(gr["ns"], -1, S)
        want = sym[gr["qs"].long(), gr["qt"].long()]
        out.append({"decode_failed_spans": int(nf.item()),
                    "roundtrip_symbol_errors": int((gr["dec"] != gr["sym"]).sum().item()),
                    "lookup_errors": int((gr["out"] != want).any(dim=1).sum().item()),
                    "spans": gr["ns"] * gr["n_spans"], "lookups": int(gr["qs"].numel())})
    return out


def reference_rates(torch, fkv=None):
    """What plain kernels reach on this device, as context for the roofline
    fractions: a dense fp16 GEMM (8192 x 8192 x 8192 through torch.matmul), a
    streaming elementwise kernel (torch.add over 1 GiB of fp32: 1 GiB read,
    1 GiB written) and, when the library is given, its matrix-core loop (the
    assignment's v_mfma_f32_32x32x16_f16 issued back to back from registers by
    two waves per SIMD, no memory traffic): the practical ceiling of that
    instruction under the board's power limit.  Best of a few repetitions,
    events on the current stream."""
    def best_ms(f, reps=5):
        f()
        torch.cuda.synchronize()
        best = float("inf")
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            f()
            e1.record()
            torch.cuda.synchronize()
            best = min(best, e0.elapsed_time(e1))
        return best

    n = 8192
    a = torch.randn((n, n), device="cuda", dtype=torch.float16)
    b = torch.randn((n, n), device="cuda", dtype=torch.float16)
    c = torch.empty((n, n), device="cuda", dtype=torch.float16)
    gemm_ms = best_ms(lambda: torch.matmul(a, b, out=c))
    del a, b, c
    x = torch.ones(1 << 28, device="cuda", dtype=torch.float32)
    y = torch.empty_like(x)
    add_ms = best_ms(lambda: torch.add(x, 1.0, out=y))
    del x, y
    torch.cuda.empty_cache()
    res = {"fp16_gemm_tflops": round(2.0 * n ** 3 / (gemm_ms / 1e3) / 1e12, 1),
           "fp16_gemm": "torch.matmul 8192^3, fp16 in and out",
           "stream_gbs": round(2.0 * (1 << 30) / (add_ms / 1e3) / 1e9, 1),
           "stream": "torch.add over 1 GiB fp32 (read + write)"}
    if fkv is not None:
        out = torch.empty(1, dtype=torch.float32, device="cuda")
        blocks, iters = 512, 20000
        flops = fkv.fkv_diag_mfma_loop(blocks, iters, out=out)[1]
        const_ms = best_ms(lambda: fkv.fkv_diag_mfma_loop(blocks, iters, out=out))
        if float(out.item()) != 64.0 * iters:
            raise RuntimeError("matrix-core loop returned %r, expected %r" % (float(out.item()), 64.0 * iters))
        loop_ms = best_ms(lambda: fkv.fkv_diag_mfma_loop(blocks, iters, out=out, random_operands=True))
        res["mfma_loop_tflops"] = round(flops / (loop_ms / 1e3) / 1e12, 1)
        res["mfma_loop"] = ("fkv_diag_mfma_loop: v_mfma_f32_32x32x16_f16 from registers, %d blocks x 4 waves x "
                            "4 chains x %d, two pseudo-random operand sets alternating per lane" % (blocks, iters))
        res["mfma_loop_constant_operands_tflops"] = round(flops / (const_ms / 1e3) / 1e12, 1)
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long_gqa",
                    choices=["gpt2", "tiny", "gpt2_hybrid_b16", "long_gqa"])
    ap.add_argument("--lookups", type=int, default=1 << 16)
    ap.add_argument("--cpu-streams", type=int, default=64,
                    help="streams per group the CPU oracle baseline runs on (the first layer's)")
    ap.add_argument("--cpu-tokens", type=int, default=1536,
                    help="archived tokens per sampled stream for the CPU oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-read-stress", action="store_true",
                    help="skip the read-side measurements on the 144 x 131,072-token archive")
    ap.add_argument("--no-next-rows", action="store_true",
                    help="skip rehydrate, eviction and k-means (the rows beyond the step)")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip the GPT-2-shaped and hybrid workloads measured beside the headline one")
    ap.add_argument("--no-reference-rates", action="store_true",
                    help="skip the library GEMM and streaming-kernel reference rates")
    ap.add_argument("--settle-s", type=float, default=0.2,
                    help="seconds each timing graph is replayed before it is timed (0: no settle period; "
                         "counter passes, which need few dispatches, use 0)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one streaming elementwise kernel (torch.neg) that reads and writes "
                         "this many MiB before the step: a kernel of known traffic for scaling HBM "
                         "byte counters")
    args = ap.parse_args()
    global SETTLE_S
    SETTLE_S = args.settle_s
    if args.gpus != 1:
        print("bench.py measures the path on one GPU; it has no multi-GPU mode (the streams are "
              "independent and would shard across GPUs with no exchange)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_07144_amd import fkv

    torch.cuda.set_device(0)
    if args.copy_probe_mib > 0:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    cfg, groups = build_workload(args.workload, args.lookups)
    names = ["rvq_assign_encode", "rvq_assign", "cgr_encode", "cgr_decode", "span_lookup"]
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        for _ in range(max(1, args.warmup)):
            run_step(fkv, cfg, groups)
    torch.cuda.synchronize()

    # The step is captured once as a HIP graph (the four launches of each group)
    # and replayed, so host launch overhead stays out of the timed region.
    step_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(step_graph, stream=side):
        run_step(fkv, cfg, groups)
    for _ in range(args.warmup):
        step_graph.replay()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        step_graph.replay()
    stop.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / args.steps

    # Average duration of each kernel: a graph of `reps` back-to-back launches of
    # that kernel alone, replayed for at least 0.2 s (the kernel's own steady
    # state; see time_graph), then replayed and bracketed by events on the
    # launch stream.
    reps = 10
    phase_ms = {}
    for n in names:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for _ in range(reps):
                run_kernel(fkv, cfg, groups, n)
        t_settle = time.perf_counter()
        g.replay()
        torch.cuda.synchronize()
        while time.perf_counter() - t_settle < SETTLE_S:
            g.replay()
            torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()  # replay() launches on the current stream
        for _ in range(max(1, args.steps // 4)):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        phase_ms[n] = e0.elapsed_time(e1) / (reps * max(1, args.steps // 4))

    extra = {} if args.no_next_rows else next_rows(fkv, cfg, groups, side, max(1, args.steps // 4),
                                                   not args.no_cpu_baseline)
    if not args.no_read_stress:
        extra["read_stress"] = read_stress(fkv, side, max(1, args.steps // 4), not args.no_cpu_baseline)
    others_res = None
    if not args.no_other_workloads:
        others = [n for n in ("gpt2", "gpt2_hybrid_b16") if n != cfg.name]
        others_res = other_workloads(fkv, side, others, args.lookups, args.steps, args.warmup,
                                     not args.no_cpu_baseline)
    alg = algorithmic(cfg, groups)
    tokens = cfg.batch * cfg.T_arch
    launches = len(groups)
    rooflines = {}
    for n in names:
        t = phase_ms[n] / 1e3 / launches  # average duration of one launch
        if n in ("rvq_assign", "rvq_assign_encode"):
            ach = alg[n]["flops"] / launches / t / 1e12
            rooflines[n] = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_FP16_MFMA_TFLOPS,
                            "unit": "TFLOP/s", "frac": round(ach / PEAK_FP16_MFMA_TFLOPS, 4)}
        else:
            ach = alg[n]["bytes"] / launches / t / 1e9
            rooflines[n] = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": round(ach / PEAK_HBM_GBS, 4)}
        rooflines[n]["traffic"] = measured_traffic(n, cfg.name)
        rooflines[n]["avg_launch_us"] = round(t * 1e6, 2)
    # the assignment + encode call is one kernel only in its fused form; in the two-kernel form the
    # dominant kernel is the assignment itself
    fused_form = all(fkv.fkv_rvq_assign_encode_fused(gr["x"], gr["books"], cfg.t_begin, cfg.t_end, symbols=gr["sym"])
                     for gr in groups)
    rooflines["rvq_assign_encode"]["form"] = ("fused kernel" if fused_form else
                                              "assignment kernel, then span encode kernel")
    if not fused_form:
        rooflines["rvq_assign_encode"]["traffic"] = None
    dominant = max((n for n in names if fused_form or n != "rvq_assign_encode"), key=lambda n: phase_ms[n])
    roof = dict(rooflines[dominant])
    roof["kernel"] = dominant

    line = {
        "metric": METRIC,
        "value": round(tokens / (ms_step / 1e3), 1),
        "unit": "archived tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 (RVQ matrix cores, fp32 accumulate) / f64 (span codec)",
        "data": "synthetic",
        "config": {"workload": cfg.name, "description": cfg.description, "layers": cfg.layers,
                   "heads": cfg.heads, "head_dim": cfg.d, "tokens": cfg.T, "batch": cfg.batch,
                   "archived_tokens": cfg.T_arch,
                   "groups": [{"kinds": list(gr["g"].kinds), "S": gr["g"].S, "K": gr["g"].K, "N": gr["g"].N,
                               "L": gr["codec"].L, "streams": gr["ns"]} for gr in groups],
                   "lookups_per_step": alg["lookups"]},
        "phases_ms": {n: round(v, 5) for n, v in phase_ms.items()},
        "write_tokens_per_s": round(tokens / (phase_ms["rvq_assign_encode"] / 1e3), 1),
        "head_vectors_per_s": round(alg["head_vectors"] / (phase_ms["rvq_assign"] / 1e3), 1),
        "decoded_symbols_per_s": round(alg["symbols"] / (phase_ms["cgr_decode"] / 1e3), 1),
        "lookups_per_s": round(alg["lookups"] / (phase_ms["span_lookup"] / 1e3), 1),
        "roofline": roof,
        "rooflines": rooflines,
        "next_rows": extra,
        "other_workloads": others_res,
        "reference_rates": None,
        "cpu_baseline": None,
    }
    if not args.no_reference_rates:
        ref = reference_rates(torch, fkv)
        line["reference_rates"] = ref
        # each kernel's achieved rate as a fraction of what the library kernel
        # of the same kind reaches here, and matrix-bound ones also as a
        # fraction of the matrix-core loop
        for n, r in rooflines.items():
            r["frac_of_reference"] = round(r["achieved"] / (ref["fp16_gemm_tflops"] if r["bound"] == "mfma"
                                                            else ref["stream_gbs"]), 4)
            if r["bound"] == "mfma":
                r["frac_of_mfma_loop"] = round(r["achieved"] / ref["mfma_loop_tflops"], 4)
        roof["frac_of_reference"] = rooflines[dominant]["frac_of_reference"]
        if "frac_of_mfma_loop" in rooflines[dominant]:
            roof["frac_of_mfma_loop"] = rooflines[dominant]["frac_of_mfma_loop"]
    line["gpu_checks"] = gpu_checks(fkv, cfg, groups)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, groups, args.cpu_streams, args.cpu_tokens, 8, 384)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
