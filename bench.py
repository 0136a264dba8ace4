"""Benchmark of the TReVS pruning hot path on one MI355X.

One step = stage 1 (trevs_prellm_prune) + stage 2 (trevs_inllm_prune) over one
batch of synthetic inputs already resident in HBM.  Prints ONE JSON line with
the throughput in visual tokens per second (B*N input visual tokens carried
through both stages per step), the roofline record of the dominant kernel
(the textual-relevance stream of stage 1, timed live with HIP events on the
launch stream), and the CPU oracle's rate on a bounded sample of the same
workload."""

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}  # dense matrix-core peaks of the compute type
METRIC = "visual tokens scored+pruned/sec (both stages) at 1 MI355X; % of HBM roofline"
ANALYSIS_METRIC = ("analysis samples/sec (text sensitivity of every head for two questions, "
                   "Eq. 1, + Spearman of s^v and s^t in the top-K1 saliency set) at 1 MI355X")


def algorithmic_bytes(w, text_len, softmax="visual"):
    """Bytes the method must move per step (every input read once, every
    output written once) and per launch of the relevance kernel.  The causal
    softmax domain also reads each text row's non-visual keys (prefix and
    text rows of K)."""
    e = w.elem_bytes
    B = w.B
    m_bar = float(np.mean(text_len))
    rel = B * (e * (w.H_v * w.N + w.N * w.d + m_bar * w.d) + 8 * w.N)
    stage1 = B * e * (w.H_v * w.N + w.N * w.d + m_bar * w.d + 2 * w.K1 * w.d) + 4 * B * w.K1
    So = w.S - w.K1 + w.K2
    stage2 = (B * e * (m_bar * w.H_q * w.d_h + w.K1 * w.H_kv * w.d_h)
              + B * (2 * So * w.D * e + 4 * So * w.H_kv * w.d_h * e + 2 * w.n_pos * So * 8 + 4 * w.K2))
    if softmax == "causal":
        stage2 += B * e * (w.P + m_bar) * w.H_kv * w.d_h
    return dict(relevance=rel, stage1=stage1, stage2=stage2, total=stage1 + stage2)


def counter_traffic(workload):
    """HBM bytes per relevance launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, each scaled by what the counter reads
    for a plain copy of known size), or None when that summary is missing or
    was taken from other kernel sources than the ones built now."""
    path = os.path.join(ROOT, "profiles", f"hbm_counters_{workload}.md")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path).read().splitlines():
        k, sep, v = line.partition(": ")
        if sep and k in ("source_sha256", "hbm_bytes_per_launch"):
            vals[k] = v.strip()
    h = hashlib.sha256()
    for f in ("stage1.hip", "common.hpp", "kernels.hpp"):
        with open(os.path.join(ROOT, "paper_2609_37581_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if vals.get("source_sha256") != h.hexdigest() or "hbm_bytes_per_launch" not in vals:
        return None
    return float(vals["hbm_bytes_per_launch"])


def cpu_info():
    """Host CPU model, the cores this process may run on, and the BLAS
    library's thread count (the threads the oracle's matrix products use)."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        blas = affinity
    return model, affinity, blas


def cpu_baseline(w, s1, s2, budget_s, ratio_mode="weights", k_div=0, softmax="visual"):
    """The CPU oracle as it stands, on single samples of the same workload,
    repeated until about budget_s seconds of work."""
    import oracle
    model, affinity, threads = cpu_info()
    t0 = time.perf_counter()
    n = 0
    while True:
        b = n % w.B
        oracle.prellm(s1["cls_logits"][b:b + 1], s1["vis_feats"][b:b + 1], s1["text_emb"][b:b + 1],
                      s1["text_len"][b:b + 1], w.dtype, n_seg=w.n_seg, k_keep=w.K1, rho=w.rho,
                      ratio_mode=ratio_mode, k_div=k_div)
        oracle.inllm(s2["q"][b:b + 1], s2["k"][b:b + 1], s2["v"][b:b + 1], s2["hidden"][b:b + 1],
                     s2["pos"][:, b:b + 1], s2["text_len"][b:b + 1], w.dtype, P=w.P, K1=w.K1,
                     n_keep=w.n_keep, k_keep=w.K2, scale=1.0 / math.sqrt(w.d_h), softmax=softmax)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return {"value": n * w.N / el, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} single samples (B=1) of {w.name}, both stages, float64 NumPy, "
                      f"{el:.1f} s",
            "cpu_model": model, "affinity_cores": affinity, "blas_threads": int(threads),
            "latency_ms_per_sample": el / n * 1e3}


def profile_flops(w, text_len):
    """Matrix flops of one profile launch (one question): the logits of the
    valid text rows of every query head against the K1 visual keys."""
    return 2.0 * float(np.sum(text_len)) * w.H_q * w.K1 * w.d_h


def cpu_baseline_analysis(w, si, sv, st, budget_s):
    """The CPU oracle on single samples of the analysis workload."""
    import oracle
    t0 = time.perf_counter()
    n = 0
    while True:
        b = n % w.B
        oracle.sensitivity(si["q0"][b:b + 1], si["k"][b:b + 1], si["q1"][b:b + 1], si["k"][b:b + 1],
                           si["text_len0"][b:b + 1], si["text_len1"][b:b + 1], w.dtype, P=w.P,
                           K1=w.K1, scale=1.0 / math.sqrt(w.d_h))
        oracle.topk_saliency_spearman(sv[b].astype(np.float64), st[b].astype(np.float64), w.K1)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    model, affinity, threads = cpu_info()
    return {"value": n / el, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} single samples (B=1) of the analysis on {w.name}, float64 NumPy, {el:.1f} s",
            "cpu_model": model, "affinity_cores": affinity, "blas_threads": int(threads)}


def run_analysis(args, w):
    """One step = trevs_text_sensitivity (two questions at the stage-2 shape)
    + trevs_topk_spearman (top-K1 of the stage-1 scores), inputs in HBM."""
    import torch

    from paper_2609_37581_amd import trevs
    from synthetic import sensitivity_inputs, stage1_inputs

    dev = torch.device("cuda:0")
    print(f"[bench] generating the analysis inputs of {w.name}", file=sys.stderr, flush=True)
    si = sensitivity_inputs(w)
    s1 = stage1_inputs(w)

    def to_dev(a):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return (t.view(torch.bfloat16) if t.dtype == torch.uint16 else t).to(dev)

    q0, q1, k = to_dev(si["q0"]), to_dev(si["q1"]), to_dev(si["k"])
    tl0, tl1 = to_dev(si["text_len0"]), to_dev(si["text_len1"])
    sens = trevs.TextSensitivity(q0, k, q1, k, tl0, tl1, P=w.P, K_in=w.K1)
    # s^v and s^t from the library's stage 1 (outside the timed region)
    pre = trevs.Prellm(to_dev(s1["cls_logits"]), to_dev(s1["vis_feats"]), to_dev(s1["text_emb"]),
                       to_dev(s1["text_len"]), k_keep=w.K1, n_seg=w.n_seg, want_scores=True)
    pre()
    spear = trevs.TopkSpearman(pre.sal, pre.rel, w.K1)
    stream = torch.cuda.current_stream()
    nk = 2 * trevs.SENSITIVITY_NUM_KERNELS
    per = nk + 2
    ev = trevs.HipEvents(args.steps * per)

    def step(i=None, all_events=False):
        if i is None:
            sens(stream)
            spear(stream)
            return
        base = i * per
        if all_events:
            sens(stream, events=ev.handles[base:base + nk])
        else:
            # profile launches of both questions only (slots 4,5 and 10,11)
            e = [None] * nk
            for j in (4, 5, 10, 11):
                e[j] = ev.handles[base + j]
            sens(stream, events=e)
        if all_events:
            ev.record(base + nk, stream)
        spear(stream)
        if all_events:
            ev.record(base + nk + 1, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        step(i)
    stop.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = start.elapsed_time(stop) / args.steps
    prof_ms = [sum(ev.elapsed_ms(i * per + a, i * per + a + 1) for i in range(args.steps)) / args.steps
               for a in (4, 10)]
    nb_steps = min(args.steps, 20)
    for i in range(nb_steps):
        step(i, all_events=True)
    torch.cuda.synchronize()
    names = list(trevs.SENSITIVITY_KERNELS) + ["topk_spearman"]
    kern_ms = {n: 0.0 for n in names}
    for i in range(nb_steps):
        for j, n in enumerate(names):
            kern_ms[n] += ev.elapsed_ms(i * per + 2 * j, i * per + 2 * j + 1) / nb_steps
    ev.close()

    flops = [profile_flops(w, si["text_len0"]), profile_flops(w, si["text_len1"])]
    achieved = (flops[0] + flops[1]) / ((prof_ms[0] + prof_ms[1]) * 1e-3) / 1e12
    peak = MFMA_PEAK_TFLOPS[w.dtype]
    result = {
        "metric": ANALYSIS_METRIC,
        "value": w.B / (ms_step * 1e-3),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name}-analysis", "B": w.B, "N": w.N, "K1": w.K1,
                   "T_max": w.T_max, "H_q": w.H_q, "H_kv": w.H_kv, "d_head": w.d_h},
        "roofline": {"bound": "mfma", "kernel": "analysis.profile", "achieved": achieved,
                     "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak, "traffic": None,
                     "flops_per_launch": flops},
        "profile_us": [m * 1e3 for m in prof_ms],
        "kernels_us_separate_pass": {n: round(v * 1e3, 3) for n, v in kern_ms.items()},
        "wall_s": t_wall,
    }
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline_analysis(w, si, pre.sal.cpu().numpy(),
                                                       pre.rel.cpu().numpy(), args.cpu_seconds)
    print(json.dumps(result), flush=True)


def stage_latency(pre, inl, stream, n, trevs):
    """Per-step and per-stage latencies (ms) from a separate pass of n steps
    with a HIP event before stage 1, between the stages and after stage 2 on
    the launch stream."""
    ev = trevs.HipEvents(3 * n)
    for i in range(n):
        ev.record(3 * i, stream)
        pre(stream)
        ev.record(3 * i + 1, stream)
        inl(stream)
        ev.record(3 * i + 2, stream)
    stream.synchronize()
    t1 = np.array([ev.elapsed_ms(3 * i, 3 * i + 1) for i in range(n)])
    t2 = np.array([ev.elapsed_ms(3 * i + 1, 3 * i + 2) for i in range(n)])
    ev.close()
    return t1, t2


def graph_step_ms(pre, inl, steps, warmup):
    """Both stages captured once into a HIP graph (torch.cuda.CUDAGraph over
    the library's launches; the path records no memset) and replayed: the
    same kernels with the per-launch host work removed."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        pre(side)
        inl(side)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pre()
        inl()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def plain_step_ms(pre, inl, stream, steps, warmup):
    """ms per step of both stages, no events inside the timed region."""
    import torch
    for _ in range(warmup):
        pre(stream)
        inl(stream)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        pre(stream)
        inl(stream)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def layer_row_stats(q, k, w, causal=True):
    """What the layer's own attention pass would hand over per text row
    (input preparation, outside the timed region): the log-sum-exp of the
    row's logits over its softmax domain and the sum and sum of squares of
    the attention over the visual columns, from plain float32 torch ops."""
    import torch
    G = w.H_q // w.H_kv
    t0 = w.P + w.K1
    out = torch.empty((w.B, w.H_q, w.T_max, 3), dtype=torch.float32, device=q.device)
    keys = torch.arange(w.S, device=q.device)
    if causal:
        allowed = keys[None, :] <= (t0 + torch.arange(w.T_max, device=q.device))[:, None]
    else:
        allowed = ((keys >= w.P) & (keys < t0))[None, :].expand(w.T_max, -1)
    for b in range(w.B):
        for g in range(w.H_kv):
            qt = q[b, t0:t0 + w.T_max, g * G:(g + 1) * G].float().permute(1, 0, 2).contiguous()
            kk = k[b, :, g].float().t().contiguous()
            x = (qt @ kk) / math.sqrt(w.d_h)
            x = x.masked_fill(~allowed[None], float("-inf"))
            lse = torch.logsumexp(x, dim=-1)
            A = torch.exp(x[..., w.P:t0] - lse[..., None])
            out[b, g * G:(g + 1) * G] = torch.stack([lse, A.sum(-1), (A * A).sum(-1)], dim=-1)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--k-div", type=int, default=0,
                    help="farthest-point diversity tokens K_d within K1 (default 0: all pivots)")
    ap.add_argument("--ratio-mode", default="weights", choices=["weights", "budget"],
                    help="textual ratio as Eq. (7) branch weights (default) or as a budget split")
    ap.add_argument("--softmax", default="visual", choices=["visual", "causal"],
                    help="stage-2 softmax over the visual keys (default) or each text row's "
                         "whole causal row")
    ap.add_argument("--settle", type=float, default=0.1,
                    help="seconds of untimed steps before the warm-up steps (steady GPU clocks)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the latency, graph-replay and other-softmax passes (profiling runs)")
    ap.add_argument("--analysis", action="store_true",
                    help="time the Sec. 3 diagnostics (text sensitivity + Spearman) instead")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the pruning path "
              "shards by sample across GPUs with no exchange, so run one process per GPU.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_37581_amd import trevs
    from synthetic import DEFAULT_BENCH_WORKLOAD, WORKLOADS, stage1_inputs, stage2_inputs

    w = WORKLOADS[args.workload or DEFAULT_BENCH_WORKLOAD]
    if args.analysis:
        run_analysis(args, w)
        return
    dev = torch.device("cuda:0")
    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    s1 = stage1_inputs(w)
    s2 = stage2_inputs(w)

    def to_dev(a):
        t = torch.from_numpy(np.ascontiguousarray(a))
        return (t.view(torch.bfloat16) if t.dtype == torch.uint16 else t).to(dev)

    cls, Z, T = to_dev(s1["cls_logits"]), to_dev(s1["vis_feats"]), to_dev(s1["text_emb"])
    tl = to_dev(s1["text_len"])
    q, k, v, hid, pos = (to_dev(s2[x]) for x in ("q", "k", "v", "hidden", "pos"))
    tl2 = to_dev(s2["text_len"])
    pre = trevs.Prellm(cls, Z, T, tl, k_keep=w.K1, n_seg=w.n_seg, textual_ratio=w.rho,
                       ratio_mode=args.ratio_mode, k_div=args.k_div)
    inl = trevs.Inllm(q, k, v, hid, pos, tl2, P=w.P, K_in=w.K1, n_keep_heads=w.n_keep,
                      k_keep=w.K2, softmax=args.softmax)
    stream = torch.cuda.current_stream()
    n1, n2 = 2 * trevs.PRELLM_NUM_KERNELS, 2 * trevs.INLLM_NUM_KERNELS
    ev = trevs.HipEvents(args.steps * (n1 + n2))

    def step(i=None, all_events=False):
        if i is None:
            pre(stream)
            inl(stream)
        elif not all_events:
            # the timed steps record events around the relevance kernel only
            # (recording around every kernel costs tens of microseconds a step)
            e = [None] * n1
            e[2], e[3] = ev.handles[i * (n1 + n2) + 2], ev.handles[i * (n1 + n2) + 3]
            pre(stream, events=e)
            inl(stream)
        else:
            base = i * (n1 + n2)
            pre(stream, events=ev.handles[base:base + n1])
            inl(stream, events=ev.handles[base + n1:base + n1 + n2])

    # device copy bandwidth (context, and the reference kernel for scaling
    # the HBM counters of a profile)
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(5):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * nbytes * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst

    # Settle: the GPU reaches its steady clocks only after tens of
    # milliseconds of this work (5 warm-up steps alone, about a millisecond,
    # left the timed steps 5-7% slower than 200 did), so the path runs
    # untimed for args.settle seconds before the warm-up steps.
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < args.settle:
        for _ in range(20):
            step()
        torch.cuda.synchronize()
    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        step(i)
    stop.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = start.elapsed_time(stop) / args.steps
    rel_ms = sum(ev.elapsed_ms(i * (n1 + n2) + 2, i * (n1 + n2) + 3) for i in range(args.steps)) / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_step:.4f} ms/step", file=sys.stderr, flush=True)
    # per-kernel breakdown from a separate, untimed pass with every event slot
    names = [f"prellm.{n}" for n in trevs.PRELLM_KERNELS] + [f"inllm.{n}" for n in trevs.INLLM_KERNELS]
    nb_steps = min(args.steps, 20)
    for i in range(nb_steps):
        step(i, all_events=True)
    torch.cuda.synchronize()
    kern_ms = {n: 0.0 for n in names}
    for i in range(nb_steps):
        base = i * (n1 + n2)
        for j, n in enumerate(names):
            kern_ms[n] += ev.elapsed_ms(base + 2 * j, base + 2 * j + 1) / nb_steps
    ev.close()

    # step and stage latency distribution (separate pass, events at the stage
    # boundaries)
    extras = {}
    if not args.no_extras:
        t1, t2 = stage_latency(pre, inl, stream, args.steps, trevs)
        tstep = t1 + t2
        extras["latency_ms"] = {
            "p50": float(np.percentile(tstep, 50)), "p90": float(np.percentile(tstep, 90)),
            "stage1_p50": float(np.percentile(t1, 50)), "stage1_p90": float(np.percentile(t1, 90)),
            "stage2_p50": float(np.percentile(t2, 50)), "stage2_p90": float(np.percentile(t2, 90)),
            "pass": f"{args.steps} steps, HIP events at the stage boundaries"}
        nb_ = algorithmic_bytes(w, s1["text_len"], args.softmax)
        t1s, t2s = np.percentile(t1, 50) * 1e-3, np.percentile(t2, 50) * 1e-3
        extras["stage_rates"] = {"stage1_tokens_per_s": w.B * w.N / t1s,
                                 "stage2_tokens_per_s": w.B * w.K1 / t2s,
                                 "stage1_hbm_frac": nb_["stage1"] / t1s / 1e9 / HBM_PEAK_GBPS,
                                 "stage2_hbm_frac": nb_["stage2"] / t2s / 1e9 / HBM_PEAK_GBPS}
        # the same step replayed from a captured HIP graph
        g_ms = graph_step_ms(pre, inl, args.steps, args.warmup)
        extras["graph_replay"] = {"ms_per_step": g_ms, "value": w.B * w.N / (g_ms * 1e-3),
                                  "path_hbm_frac": nb_["total"] / (g_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS}
        # the stage-2 softmax over each text row's whole causal row (Sec. 4.2's
        # text-to-vision attention within the layer's own attention)
        other = "causal" if args.softmax == "visual" else "visual"
        inl_other = trevs.Inllm(q, k, v, hid, pos, tl2, P=w.P, K_in=w.K1, n_keep_heads=w.n_keep,
                                k_keep=w.K2, softmax=other)
        other_ms = plain_step_ms(pre, inl_other, stream, args.steps, args.warmup)
        extras[f"softmax_{other}"] = {"ms_per_step": other_ms, "value": w.B * w.N / (other_ms * 1e-3)}
        del inl_other
        # stage 2 fed the per-row statistics of the layer's own (causal)
        # attention pass: no statistics pass in the library
        rs = layer_row_stats(q, k, w, causal=True)
        inl_rs = trevs.Inllm(q, k, v, hid, pos, tl2, P=w.P, K_in=w.K1, n_keep_heads=w.n_keep,
                             k_keep=w.K2, row_stats=rs)
        rs_ms = plain_step_ms(pre, inl_rs, stream, args.steps, args.warmup)
        extras["row_stats_from_layer"] = {"ms_per_step": rs_ms, "value": w.B * w.N / (rs_ms * 1e-3),
                                          "softmax": "causal"}
        del inl_rs, rs
        # stage 1 with a diversity set at the 3:1 pivot:diversity split of
        # Sec. 4.1 (K_d = K1 / 4 farthest-point tokens), then stage 2
        if args.k_div == 0 and w.N <= trevs.MAX_FPS_N:
            kd = w.K1 // 4
            pre_fps = trevs.Prellm(cls, Z, T, tl, k_keep=w.K1, n_seg=w.n_seg, textual_ratio=w.rho,
                                   ratio_mode=args.ratio_mode, k_div=kd)
            fps_ms = plain_step_ms(pre_fps, inl, stream, 10, 2)
            extras["diversity_set"] = {"k_div": kd, "ms_per_step": fps_ms, "value": w.B * w.N / (fps_ms * 1e-3)}
            del pre_fps

    nb = algorithmic_bytes(w, s1["text_len"], args.softmax)
    traffic = counter_traffic(w.name)
    rel_s = rel_ms * 1e-3
    achieved = nb["relevance"] / rel_s / 1e9
    t_step = ms_step * 1e-3
    tokens = w.B * w.N
    result = {
        "metric": METRIC,
        "value": tokens / t_step,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "ratio_mode": args.ratio_mode, "k_div": args.k_div,
                   "softmax": args.softmax, "B": w.B, "N": w.N, "d": w.d, "M_max": w.M_max,
                   "K1": w.K1, "K2": w.K2, "H_q": w.H_q, "H_kv": w.H_kv, "d_head": w.d_h,
                   "D": w.D, "n_keep_heads": w.n_keep, "P": w.P, "S": w.S},
        "roofline": {"bound": "hbm", "kernel": "prellm.relevance", "achieved": achieved,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": traffic, "bytes_per_launch": nb["relevance"]},
        "path_hbm_frac": nb["total"] / t_step / 1e9 / HBM_PEAK_GBPS,
        "path_hbm_target": 0.60,
        "path_bytes": nb,
        **extras,
        "relevance_us": rel_ms * 1e3,
        "kernels_us_separate_pass": {n: round(v * 1e3, 3) for n, v in kern_ms.items()},
        "copy_gbps": copy_gbps,
        "settle_s": args.settle,
        "wall_s": t_wall,
    }
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(w, s1, s2, args.cpu_seconds, args.ratio_mode, args.k_div,
                                              args.softmax)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
