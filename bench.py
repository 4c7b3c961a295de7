"""Benchmark: sender KV tokens scored + selected + compacted per second.

One step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM: cb_score (query-attention importance for every
layer and KV head), cb_select (top keep fraction per unit, source order) and
cb_compact (row gather of the kept K/V rows).  Default workload: the
Qwen3-8B attention shape, 36 layers, 32 query / 8 KV heads, head_dim 128,
T = 8192 sender positions, a 64-token receiver query, bf16, keep 0.25.

Prints one JSON line.  `value` is whole-job tokens/s (S*T positions per step
over all layers).  `roofline` reports the dominant stage (cb_score) against
MI355X's 8 TB/s HBM; per-stage times come from HIP events recorded on the
stream the kernels run on, around cb_score, cb_select_ws (the selection
kernel cb_pipeline runs, with its scratch clearing kernel) and cb_compact.  `cpu_baseline` times the CPU oracle (one thread)
on a bounded sample of units of the same workload and scales it to tokens/s.
Before the warmup steps an untimed settle phase (--settle-ms of whole steps)
lets the GPU clock reach its steady state; after the timed region, `cold`
times single steps each preceded by an untimed 512 MiB write that evicts the
inputs from the Infinity Cache.  `score_counters` carries the score kernel's
MFMA and wave counters recorded under profiles/ while its sources match.
`message` times the paper's own selector on the same inputs (position-level
score, span rule, continuous-row gather; --no-message skips it).

Single GPU only: the path shards by unit (layer, KV head, sender) with no
exchange, and no multi-GPU figure is produced here.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16
METRIC = "sender KV tokens scored+compacted/sec (all layers) and % of peak HBM GB/s"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(w, keep):
    """Bytes the method must move once: Q, K (one scan), importance written
    and read, indices written and read, kept K and V rows read, compact
    K and V written."""
    esz = w.esize
    U = w.units
    q = w.layers * w.q_heads * w.q_len * w.head_dim * esz
    k = U * w.seq_len * w.head_dim * esz
    imp = U * w.seq_len * 4
    idx = U * keep * 4
    rows = U * keep * w.head_dim * esz
    score = q + k + imp
    select = imp + idx
    compact = idx + 2 * rows + 2 * rows
    return dict(score=score, select=select, compact=compact, total=score + select + compact)


def score_kernel_sources():
    """The files cb_score's kernels are built from: the persistent kernel, its
    plan and launch, the importance instantiations and the internal header."""
    import glob

    csrc = os.path.join(ROOT, "paper_2609_32046_amd", "csrc")
    names = ["kernels.h", "score.hip", "score_impl.h"]
    names += [os.path.basename(f) for f in glob.glob(os.path.join(csrc, "score_bf16_d*.hip"))]
    names += [os.path.basename(f) for f in glob.glob(os.path.join(csrc, "score_f32_d*.hip"))]
    return [os.path.join(csrc, n) for n in sorted(names)]


def kernel_sources_sha256():
    """Hash of score_kernel_sources(): counters recorded under profiles/ for
    the score kernel are reported only while it matches."""
    import hashlib

    h = hashlib.sha256()
    for f in score_kernel_sources():
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(workload):
    """Counter-measured bytes per cb_score call (FETCH_SIZE + WRITE_SIZE,
    calibrated against a plain copy) from profiles/, or None when the kernel
    sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload.replace('-bf16', '')}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sources_sha256") != kernel_sources_sha256():
        return None
    return rec.get("score_stage_bytes_per_call")


def recorded_counters(workload):
    """MFMA and wave-cycle counters of the score kernel (rocprofv3 --pmc) from
    profiles/, or None when the kernel sources changed since they were taken."""
    path = os.path.join(ROOT, "profiles", f"counters_{workload.replace('-bf16', '')}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_sources_sha256") != kernel_sources_sha256():
        return None
    return rec.get("summary")


def message_path(cb, torch, w, lay, qd, kd, stream, dev, steps, warmup):
    """The paper's own selector on the same workload, timed like the graded
    path: cb_position_score (S_t = Q_t * C_t^2 with Pool_7, p = 2, alpha = 2),
    cb_select_spans at the 4x fan-out budget ceil(T/4) per sender with the
    first position and 40 latent positions forced and width-16 spans, and
    cb_gather_rows of the selected d_model-wide bf16 continuous rows."""
    S, T = w.senders, w.seq_len
    pbuf = cb.PositionBuffers(lay, device=dev)
    budget = cb.cb_budget_fanout(T, 4)
    idx = torch.empty((S, budget), dtype=torch.int32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(260932046)
    rows = torch.randn((S, T, w.d_model), generator=gen, device=dev).to(torch.bfloat16)
    out_rows = torch.empty((S * budget, w.d_model), dtype=torch.bfloat16, device=dev)
    row_bytes = w.d_model * 2

    def score():
        cb.cb_position_score(qd, kd, lay, pbuf.score, pbuf.ws, p=2.0, alpha=2.0, stream=stream)

    def spans():
        cb.cb_select_spans(pbuf.score, S, T, budget, idx, pbuf.span_ws, n_latent=40, stream=stream)

    def gather():
        cb.cb_gather_rows(rows, S, T, row_bytes, idx, budget, out_rows, stream=stream)

    for _ in range(warmup):
        score(), spans(), gather()
    torch.cuda.synchronize()
    region = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    region[0].record(stream)
    for _ in range(steps):
        score(), spans(), gather()
    region[1].record(stream)
    torch.cuda.synchronize()
    ms_per_step = region[0].elapsed_time(region[1]) / steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for e in ev:
        e[0].record(stream)
        score()
        e[1].record(stream)
        spans()
        e[2].record(stream)
        gather()
        e[3].record(stream)
    torch.cuda.synchronize()
    st = {k: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev]))
          for i, k in enumerate(("score", "spans", "gather"))}
    q_bytes = w.layers * w.q_heads * w.q_len * w.head_dim * w.esize
    k_bytes = w.units * w.seq_len * w.head_dim * w.esize
    ab = {"score": q_bytes + k_bytes + S * T * 4,                 # Q, K once; S_t written
          "spans": S * T * 4 + S * budget * 4,                    # S_t read; positions written
          "gather": S * budget * 4 + 2 * S * budget * row_bytes}  # positions; rows read + written
    ab["total"] = ab["score"] + ab["spans"] + ab["gather"]
    score_gbs = ab["score"] / (st["score"] * 1e-3) / 1e9
    del rows, out_rows, pbuf
    return {
        "what": "cb_position_score (p = 2, alpha = 2, Pool_7) + cb_select_spans (ceil(T/4) per "
                "sender, first position and 40 latents forced, width 16) + cb_gather_rows "
                f"({row_bytes}-byte bf16 rows)",
        "value": S * T / (ms_per_step * 1e-3), "unit": "tokens/s", "ms_per_step": ms_per_step,
        "steps": steps, "warmup": warmup, "budget_per_sender": budget,
        "stage_ms": st, "algorithmic_bytes": ab,
        "hbm_frac": ab["total"] / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "stage_gbs": {k: ab[k] / (st[k] * 1e-3) / 1e9 for k in st},
        "roofline": {"bound": "hbm",
                     "kernel": "cb_position_score (the persistent score kernel's position "
                               "variant and its layer/head reduction)",
                     "achieved": score_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": score_gbs / HBM_PEAK_GBS},
    }


def cpu_baseline(w, q, K, V, keep, budget_s=12.0):
    """The CPU oracle on a bounded sample of units, scaled to tokens/s."""
    import oracle
    import cb_workloads as W

    orc = oracle.Oracle()
    units = [(s, l, g) for s in range(w.senders) for l in range(w.layers)
             for g in range(w.kv_heads)]
    rng = np.random.default_rng(11)
    order = rng.permutation(len(units))
    done, t_total = 0, 0.0
    for i in order:
        s, l, g = units[i]
        qu = W.unit_q(w, q, l, g)
        ku = np.ascontiguousarray(K[s, l, g])[None, None, None]
        vu = np.ascontiguousarray(V[s, l, g])[None, None, None]
        t0 = time.perf_counter()
        imp = orc.score(qu, ku)
        idx = orc.select(imp, keep)
        orc.compact(ku, vu, idx)
        t_total += time.perf_counter() - t0
        done += 1
        if t_total >= budget_s:
            break
    per_unit = t_total / done
    tokens_per_s = w.senders * w.seq_len / (per_unit * w.units)
    cpu = platform.processor() or platform.machine()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": tokens_per_s, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of {w.units} units (score+select+compact), "
                      f"{t_total:.1f} s, scaled linearly to all units; 1 thread of "
                      f"{os.cpu_count()} on {cpu}"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="qwen3-8b-8k-bf16")
    ap.add_argument("--keep-ratio", type=float, default=None)
    # The GPU's clock ramps up over the first tens of milliseconds of
    # sustained work: an untimed, time-based settle phase before the warmup
    # steps reaches the steady state whatever --warmup is.
    ap.add_argument("--settle-ms", type=float, default=400.0)
    ap.add_argument("--cold-steps", type=int, default=20,
                    help="steps timed one by one after an untimed 512 MiB write")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-message", action="store_true",
                    help="skip the position-level message path (the `message` object)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); "
              "the path shards by (layer, KV head, sender) with no exchange between GPUs",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import cb_workloads as W
    import paper_2609_32046_amd as cb

    w = W.get(args.workload)
    ratio = args.keep_ratio if args.keep_ratio is not None else w.keep_ratios[0]
    log(f"bench: workload {w.name}, keep {ratio}; generating inputs")
    q = W.gen_q(w)
    K, V = W.gen_kv(w, progress=log)

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def up(a):
        t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
        t = t.to(dev)
        return t.view(torch.bfloat16) if a.dtype == np.uint16 else t

    qd, kd, vd = up(q), up(K), up(V)
    lay = cb.layout_of(w)
    buf = cb.Buffers(lay, ratio, device=dev)
    stream = torch.cuda.current_stream()
    log(f"bench: inputs resident ({(kd.numel() + vd.numel()) * kd.element_size() / 2**30:.2f} GiB K+V); "
        f"{args.warmup} warmup + {args.steps} timed steps")

    def step():
        """One pass of the whole hot path: the fused entry point."""
        cb.cb_pipeline(qd, kd, vd, lay, ratio, buf.importance, buf.idx, buf.k_out, buf.v_out,
                       buf.ws, stream=stream)

    def staged(ev):
        """The same work as three calls, with HIP events between them on the
        stream every kernel is ordered on (stage breakdown)."""
        ev[0].record(stream)
        cb.cb_score(qd, kd, lay, buf.importance, None, buf.ws, stream=stream)
        ev[1].record(stream)
        cb.cb_select_ws(buf.importance, buf.units, lay.seq_len, ratio, buf.idx, buf.sel_ws,
                        stream=stream)
        ev[2].record(stream)
        cb.cb_compact(kd, vd, buf.idx, lay, buf.keep, buf.k_out, buf.v_out, stream=stream)
        ev[3].record(stream)

    # Settle: whole steps, untimed, until settle_ms of wall time have passed.
    torch.cuda.synchronize()
    t_settle = time.perf_counter()
    settle_steps = 0
    while (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(20):
            step()
        settle_steps += 20
        torch.cuda.synchronize()
    settle_ms = (time.perf_counter() - t_settle) * 1e3

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Events only around the whole timed region: an event recorded between
    # steps leaves the GPU idle for a few microseconds.
    region_ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    region_ev[0].record(stream)
    for _ in range(args.steps):
        step()
    region_ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    log("bench: timed region done; stage breakdown")

    # Cold steps: before each, an untimed write of 512 MiB (twice the 256 MB
    # Infinity Cache) evicts the inputs; the step alone is timed with events.
    cold_ms = []
    if args.cold_steps > 0:
        flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        cold_ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        for i in range(args.cold_steps + 2):
            flush.fill_(i & 255)
            cold_ev[0].record(stream)
            step()
            cold_ev[1].record(stream)
            torch.cuda.synchronize()
            if i >= 2:
                cold_ms.append(cold_ev[0].elapsed_time(cold_ev[1]))
        del flush

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(min(3, args.steps)):
        staged(events[i])
    torch.cuda.synchronize()
    for i in range(args.steps):
        staged(events[i])
    torch.cuda.synchronize()

    st = {"score": [], "select": [], "compact": [], "staged": []}
    for ev in events:
        st["score"].append(ev[0].elapsed_time(ev[1]))
        st["select"].append(ev[1].elapsed_time(ev[2]))
        st["compact"].append(ev[2].elapsed_time(ev[3]))
        st["staged"].append(ev[0].elapsed_time(ev[3]))
    mean = {k: float(np.mean(v)) for k, v in st.items()}
    mean["step_events"] = region_ev[0].elapsed_time(region_ev[1]) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    tokens = w.senders * w.seq_len
    ab = algorithmic_bytes(w, buf.keep)
    # Reference: a plain device-to-device copy moving the compact stage's
    # bytes (read + write), the practical ceiling for a pure gather.
    half = ab["compact"] // 2
    csrc = torch.empty(half // 4, dtype=torch.int32, device=dev).fill_(1)
    cdst = torch.empty_like(csrc)
    copy_ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(3):
        cdst.copy_(csrc)
    copy_ev[0].record(stream)
    for _ in range(10):
        cdst.copy_(csrc)
    copy_ev[1].record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * csrc.numel() * 4 / (copy_ev[0].elapsed_time(copy_ev[1]) / 10 * 1e-3) / 1e9
    del csrc, cdst

    flops = 2.0 * w.units * w.rows * w.seq_len * w.head_dim   # one QK^T pass

    message = None
    if not args.no_message:
        log("bench: message path (position-level score, span rule, continuous rows)")
        message = message_path(cb, torch, w, lay, qd, kd, stream, dev, args.steps,
                               max(10, args.warmup // 5))

    score_gbs = ab["score"] / (mean["score"] * 1e-3) / 1e9
    k_bytes = w.units * w.seq_len * w.head_dim * w.esize
    counters = recorded_counters(w.name)
    # Issue floor of the score kernel on gfx950: per 64 logits and pass one
    # 16x16x32 MFMA interleaved with an fma, an exp2 and an add, measured at
    # 25.2 SIMD cycles by a microbenchmark at two waves per SIMD; 1024 SIMDs
    # at 2.4 GHz; both passes.
    floor_cycles_per_64 = 25.2
    logits_two_passes = 2.0 * w.units * w.rows * w.seq_len
    floor_ms = logits_two_passes / 64.0 * floor_cycles_per_64 / (1024 * 2.4e9) * 1e3
    out = {
        "metric": METRIC,
        "value": tokens / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded; shapes and value recipes of the workload, no dataset)",
        "config": {"workload": w.name, "layers": w.layers, "q_heads": w.q_heads,
                   "kv_heads": w.kv_heads, "head_dim": w.head_dim, "seq_len": w.seq_len,
                   "q_len": w.q_len, "senders": w.senders, "keep_ratio": ratio,
                   "keep": buf.keep, "units": w.units},
        "hbm_frac_pipeline": ab["total"] / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "algorithmic_bytes": ab,
        "step_ms_events": mean["step_events"],
        "stage_ms": {k: mean[k] for k in ("score", "select", "compact", "staged")},
        "stage_ms_median": {k: float(np.median(st[k])) for k in ("score", "select", "compact", "staged")},
        "stage_ms_min": {k: float(np.min(st[k])) for k in ("score", "select", "compact", "staged")},
        "stage_hbm_frac": {k: ab[k] / (mean[k] * 1e-3) / 1e9 / HBM_PEAK_GBS
                           for k in ("score", "select", "compact")},
        "stage_gbs": {k: ab[k] / (mean[k] * 1e-3) / 1e9 for k in ("score", "select", "compact")},
        # K as the score kernel streams it: both passes read every K row (the
        # second from the Infinity Cache or HBM)
        "score_k_stream_gbs": 2 * k_bytes / (mean["score"] * 1e-3) / 1e9,
        "settle": {"ms": settle_ms, "steps": settle_steps},
        "cold": ({"ms_per_step": float(np.mean(cold_ms)), "ms_median": float(np.median(cold_ms)),
                  "steps": len(cold_ms), "value": tokens / (float(np.mean(cold_ms)) * 1e-3),
                  "hbm_frac_pipeline": ab["total"] / (float(np.mean(cold_ms)) * 1e-3) / 1e9
                  / HBM_PEAK_GBS,
                  "flush": "untimed 512 MiB device write before each step"}
                 if cold_ms else None),
        "score_counters": counters,
        "score_mfma_tflops": flops / (mean["score"] * 1e-3) / 1e12,
        "score_issue_floor": {"cycles_per_64_logits_per_pass": floor_cycles_per_64,
                              "floor_ms": floor_ms, "frac": floor_ms / mean["score"]},
        "copy_reference": {"gbs": copy_gbs,
                           "compact_frac_of_copy": ab["compact"] / (mean["compact"] * 1e-3) / 1e9
                           / copy_gbs},
        "roofline": {"bound": "hbm",
                     "kernel": "cb_score (one persistent kernel: both score passes of every unit)",
                     "achieved": score_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": score_gbs / HBM_PEAK_GBS,
                     "traffic": recorded_traffic(w.name)},
        "message": message,
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a sample of units")
        out["cpu_baseline"] = cpu_baseline(w, q, K, V, buf.keep, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
