#!/usr/bin/env python3
"""Benchmark of the fused multi-sub-model LM head + CE + KL, forward + backward, on one MI355X.

One step = mls_distill_fwd + mls_distill_bwd over one batch of synthetic input that is
already resident in HBM: every sub-model's logits, online log-sum-exp, cross-entropy,
teacher-to-student KL, and the gradients grad_h_i and grad_W_i with the coefficients of
eq. (3). Prints one JSON line: throughput, per-kernel times, the roofline of the
dominant kernel and the CPU oracle's rate on a sample.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

With --diagnostics a step is instead the monitoring pass of paper section 3:
mls_diagnostics, one self-normalising pass over every sub-model's logits (pairwise
KL at temperature 1 and top-1 agreement of every pair of sub-models).

With --junction a step is the forward and backward of every inter-model junction
(eq. (1)) of a suite (mls_junction_fwd + mls_junction_bwd per junction).

With --decode a step is one speculative-decoding head step of a draft / verifier
pair (section 3, "Speculative Decoding Throughput"): gamma draft steps (head logits
+ nucleus sampling for the batch), the verifier's head logits over the batch's
gamma + 1 positions, and the verification (mls_head_logits, mls_sample,
mls_spec_verify).
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused LM-head+CE+KL fwd+bwd tokens/s (M=3, V=50304); % of bf16 MFMA peak"
METRIC_DIAG = "cross-model diagnostics (pairwise KL/top-1 agreement, one pass) tokens/s"
METRIC_JUNCTION = "inter-model junctions fwd+bwd tokens/s (every junction of the suite)"
METRIC_DECODE = ("speculative head step rows/s (gamma draft steps x batch + verifier "
                 "(gamma + 1) x batch rows)")
PEAK_FLOPS = {"bf16": 2.5e15, "f32": 157.3e12}  # MI355X dense MFMA peaks
HBM_PEAK = 8.0e12


def sources_sha256():
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2608_09703_amd", "csrc")
    for f in sorted(os.listdir(d)):
        h.update(f.encode())
        h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()


def profiled_traffic(workload, kernel, kind=False):
    """Per-launch bytes beyond L2 of `kernel` (reads + writes, from the TCC_EA0 request
    counters) in the committed rocprofv3 summary, or None when the summary is missing
    or the kernel sources changed since it was taken."""
    import re
    kind = {False: "kernels", True: "diagnostics"}.get(kind, kind)
    path = os.path.join(ROOT, "profiles", f"{workload}_{kind}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    info = json.loads(m.group(1))
    if info.get("sources_sha256") != sources_sha256():
        return None
    t = info.get("per_launch", {}).get(kernel)
    return None if t is None else t["fetch_bytes"] + t["write_bytes"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# The paper's own throughput figures, quoted as context only: it never times the
# loss block itself (it calls online distillation free, section 2 "Integrated
# Distillation").
PAPER_CONTEXT = {
    "training_compute": "-36% training compute for the 3B Matryoshka suite against token-matched "
                        "independent training (NVIDIA B200, bf16 mixed precision; GPU-hours x "
                        "nominal 4.5e15 FLOP/s; abstract, section 3 and appendix B)",
    "speculative_decoding": "+14% (nucleus p = 0.9, temperature 0.4) to +26% (greedy; 2,650 vs "
                            "2,100 tokens/s) decoding throughput with a 500M draft and 3B verifier "
                            "from one suite (NVIDIA A100 80GB; section 3, Speculative Decoding "
                            "Throughput)",
    "note": "context only, other hardware and other work: not a target for this measurement",
}


def host_info(threads):
    """Host facts recorded with every CPU baseline: the threads the oracle used,
    the host's CPU count and model, and the BLAS library numpy calls."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        libs = [f"{p.get('internal_api')} {p.get('version')} ({os.path.basename(p.get('filepath', ''))}, "
                f"{p.get('num_threads')} threads)"
                for p in threadpool_info() if p.get("user_api") == "blas"]
        if libs:
            blas = "; ".join(libs)
    except Exception:  # pragma: no cover
        pass
    return {"cores": int(threads), "host_cpus": os.cpu_count(), "cpu_model": model, "blas": blas}


def time_steps(torch, step, stream, n):
    """Per-step times (ms) of n calls of step, each bracketed by events on stream."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    for e0, e1 in evs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    return [e0.elapsed_time(e1) for e0, e1 in evs]


def step_stats(times):
    import statistics
    return {"median": statistics.median(times), "mean": statistics.fmean(times),
            "min": min(times), "max": max(times), "n": len(times)}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=0, help="oracle sample rows (0 = auto)")
    ap.add_argument("--vocab-chunk", type=int, default=0)
    ap.add_argument("--path", choices=("fwd_bwd", "recompute", "separate"), default="fwd_bwd",
                    help="fwd_bwd: mls_distill_fwd_bwd with its default plan (stored logits per "
                         "token chunk); recompute: the same call with MLS_FWD_BWD_RECOMPUTE; "
                         "separate: mls_distill_fwd then mls_distill_bwd")
    ap.add_argument("--diagnostics", action="store_true",
                    help="time the pairwise diagnostics pass instead of fwd+bwd")
    ap.add_argument("--junction", action="store_true",
                    help="time the inter-model junctions (forward + backward) instead")
    ap.add_argument("--decode", action="store_true",
                    help="time the speculative-decoding head step instead")
    ap.add_argument("--mfma-ceiling", action="store_true",
                    help="measure the device's bf16 MFMA ceiling (register operands, zero and random "
                         "data) instead")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (a known-size "
                         "kernel that checks the traffic counters of a profile run)")
    return ap.parse_args()


def cpu_baseline(wl, h, W, y, g_ce, g_kl, rows_req, diagnostics=False):
    """Times the float64 CPU oracle (forward + backward, or the diagnostics) on a
    sample of rows."""
    import numpy as np
    import oracle

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()
                       if p.get("user_api") == "blas"] or [os.cpu_count() or 1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    Wn = [x.float().cpu().numpy() for x in W]
    yn_all = y.cpu().numpy()

    def run(nrows):
        hn = [x[:nrows].float().cpu().numpy() for x in h]
        yn = yn_all[:nrows]
        t0 = time.perf_counter()
        if diagnostics:
            oracle.diagnostics(hn, Wn, yn)
        else:
            oracle.forward(hn, Wn, yn, tau=wl.tau)
            oracle.backward(hn, Wn, yn, g_ce, g_kl, tau=wl.tau)
        return time.perf_counter() - t0

    if rows_req > 0:
        rows = rows_req
        dt = run(rows)
    else:
        # grow the sample until one timed run costs 10-30 s of host time
        rows = 32
        while True:
            dt = run(rows)
            log(f"oracle sample {rows} rows: {dt:.1f} s")
            if dt >= 10.0 or rows >= wl.T:
                break
            rows = int(min(wl.T, max(2 * rows, rows * 14.0 / max(dt, 1e-3))))
            rows = max(16, rows // 16 * 16)
    out = {
        "value": rows / dt,
        "unit": "tokens/s",
        "kind": "oracle",
        "sample": f"float64 numpy oracle, {'diagnostics' if diagnostics else 'forward + backward'} "
                  f"on the first {rows} of {wl.T} tokens "
                  f"at full V={wl.V} and widths {list(wl.dims)}; {dt:.1f} s",
    }
    out.update(host_info(threads))
    return out


def junction_bytes(T, d_prev, d_fresh, act_bytes, grad_bytes):
    """Algorithmic HBM bytes of one junction forward and one backward launch: every
    operand read once and every result written once."""
    w = d_prev + d_fresh
    fwd = T * w * act_bytes + T * w * act_bytes                   # read o, e; write x
    bwd = T * w * grad_bytes + T * w * act_bytes + T * w * grad_bytes  # read g_x, o, e; write g_o, g_e
    return fwd, bwd


def cpu_junction(wl, inputs, rows_req):
    """Times the float64 oracle of every junction (forward + backward) on a sample of rows."""
    import numpy as np
    from oracle import junction as OJ
    npi = [[x.float().cpu().numpy() for x in trio] for trio in inputs]

    def run(nrows):
        t0 = time.perf_counter()
        for o, e, g in npi:
            OJ.forward(o[:nrows], e[:nrows])
            OJ.backward(o[:nrows], e[:nrows], g[:nrows])
        return time.perf_counter() - t0

    rows = rows_req if rows_req > 0 else 256
    while True:
        dt = run(rows)
        log(f"oracle sample {rows} rows: {dt:.2f} s")
        if rows_req > 0 or dt >= 10.0 or rows >= wl.T:
            break
        rows = int(min(wl.T, max(2 * rows, rows * 14.0 / max(dt, 1e-3))))
    # elementwise numpy: one thread
    out = {"value": rows / dt, "unit": "tokens/s",
           "kind": "oracle",
           "sample": f"float64 numpy oracle, forward + backward of every junction on the first "
                     f"{rows} of {wl.T} tokens; {dt:.1f} s"}
    out.update(host_info(1))
    return out


def main_junction(args):
    import torch
    from paper_2608_09703_amd import binding as B
    from paper_2608_09703_amd import workloads as WL

    name = args.workload or "c5_junctions"
    wl = WL.JUNCTIONS[name]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"junction workload {name}: T={wl.T} widths={wl.dims} {wl.act_dtype}/{wl.grad_dtype}")
    inputs = [WL.make_junction_inputs(wl, m, device=dev) for m in range(len(wl.junctions))]
    ea = 2 if wl.act_dtype == "bf16" else 4
    eg = 2 if wl.grad_dtype == "bf16" else 4
    act_code = B.MLS_BF16 if wl.act_dtype == "bf16" else B.MLS_F32
    grad_code = B.MLS_BF16 if wl.grad_dtype == "bf16" else B.MLS_F32
    calls = []
    fwd_bytes = bwd_bytes = 0
    for (dp, df), (o, e, gx) in zip(wl.junctions, inputs):
        j = B.make_junction(wl.T, dp, df, act_code, grad_code)
        x = torch.empty(wl.T, dp + df, dtype=o.dtype, device=dev)
        g_o = torch.empty(o.shape, dtype=gx.dtype, device=dev)
        g_e = torch.empty(e.shape, dtype=gx.dtype, device=dev)
        calls.append((j, o, e, gx, x, g_o, g_e))
        fb, bb = junction_bytes(wl.T, dp, df, ea, eg)
        fwd_bytes += fb
        bwd_bytes += bb
    sh = torch.cuda.current_stream(dev).cuda_stream

    def step():
        for j, o, e, gx, x, g_o, g_e in calls:
            B.junction_fwd(j, o.data_ptr(), e.data_ptr(), x.data_ptr(), sh)
        for j, o, e, gx, x, g_o, g_e in reversed(calls):
            B.junction_bwd(j, o.data_ptr(), e.data_ptr(), gx.data_ptr(), g_o.data_ptr(),
                           g_e.data_ptr(), sh)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    st = step_stats(time_steps(torch, step, stream, args.steps))
    ms_step = st["median"]
    B.profile_enable(True)  # per-kernel breakdown in a separate pass
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    B.profile_enable(False)
    prof = B.profile_report()
    kernels = {}
    for kname, (launches, tot) in prof.items():
        kernels[kname] = {"launches_per_step": launches / args.steps, "ms_per_step": tot / args.steps,
                          "avg_launch_ms": tot / launches}
        log(f"  {kname:14s} {launches / args.steps:5.1f} launches/step {tot / args.steps:8.4f} ms/step")
    per_step = {"junction_fwd": fwd_bytes, "junction_bwd": bwd_bytes}
    dom = max(per_step, key=lambda k: kernels[k]["ms_per_step"])
    achieved = per_step[dom] / (kernels[dom]["ms_per_step"] / 1e3)
    log(f"{ms_step:.4f} ms/step; {dom}: {achieved / 1e9:.0f} GB/s of algorithmic bytes")
    if args.copy_mib > 0:
        src = torch.ones(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_junction(wl, inputs, args.cpu_rows)
    out = {
        "metric": METRIC_JUNCTION,
        "value": wl.T / (ms_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_stats": st,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": f"{wl.act_dtype} activations, {wl.grad_dtype} gradients (fp32 reductions)",
        "data": "synthetic (seeded Gaussian sub-model outputs, fresh embeddings and gradients)",
        "config": {"workload": name, "T": wl.T, "widths": list(wl.dims), "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved / 1e9, "peak": HBM_PEAK / 1e9,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK,
                     "traffic": profiled_traffic(name, dom, "junction")},
        "kernels": kernels,
        "cpu_baseline": cpu,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(out), flush=True)


def cpu_decode(wl, x, rows_req):
    """Times the float64 oracle of the step (heads, draft draws, verification) on a
    sample of sequences."""
    import numpy as np
    from oracle import decode as OD
    B, G, V = wl.batch, wl.gamma, wl.V
    Wt = x["W_target"].float().cpu().numpy()
    Wd = x["W_draft"].float().cpu().numpy()
    ot = x["o_target"].float().cpu().numpy().reshape(B, G + 1, -1)
    od = x["o_draft"].float().cpu().numpy().reshape(G, B, -1)
    ud = x["u_draft"].cpu().numpy()
    ua = x["u_accept"].cpu().numpy()
    us = x["u_sample"].cpu().numpy()

    def run(n):
        t0 = time.perf_counter()
        dl = np.stack([OD.head_logits(od[k, :n], Wd) for k in range(G)], axis=1)  # [n, G, V]
        drafts = np.stack([OD.sample(dl[:, k], ud[k, :n], wl.temperature, wl.top_p)
                           for k in range(G)], axis=1)
        tl = OD.head_logits(ot[:n].reshape(n * (G + 1), -1), Wt).reshape(n, G + 1, V)
        OD.verify(dl, tl, drafts, ua[:n], us[:n], wl.temperature, wl.top_p)
        return time.perf_counter() - t0

    n = rows_req if rows_req > 0 else 2
    while True:
        dt = run(n)
        log(f"oracle sample {n} sequences: {dt:.1f} s")
        if rows_req > 0 or dt >= 10.0 or n >= B:
            break
        n = int(min(B, max(2 * n, n * 14.0 / max(dt, 1e-3))))
    rows = n * G + n * (G + 1)
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()
                       if p.get("user_api") == "blas"] or [os.cpu_count() or 1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count() or 1
    out = {"value": rows / dt, "unit": "rows/s", "kind": "oracle",
           "sample": f"float64 numpy oracle, the whole step for {n} of {B} sequences "
                     f"({rows} rows); {dt:.1f} s"}
    out.update(host_info(threads))
    return out


def device_peaks():
    """The device's CU count and clocks, with the peaks derived from them."""
    from paper_2608_09703_amd import binding as B
    cu, clk, mclk, bus = B.device_info()
    return {"compute_units": cu, "clock_mhz": clk / 1e3, "mem_clock_mhz": mclk / 1e3,
            "mem_bus_bits": bus,
            "bf16_peak_tflops_nominal": PEAK_FLOPS["bf16"] / 1e12,
            "bf16_peak_tflops_derived": cu * clk * 1e3 * 4096 / 1e12,
            "hbm_peak_gbs_nominal": HBM_PEAK / 1e9}


def main_decode(args):
    import torch
    from paper_2608_09703_amd import binding as B
    from paper_2608_09703_amd import workloads as WL

    name = args.workload or "spec_500m_3b"
    wl = WL.DECODE[name]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    Bt, G, V = wl.batch, wl.gamma, wl.V
    log(f"decode workload {name}: batch={Bt} gamma={G} V={V} draft d={wl.d_draft} "
        f"verifier d={wl.d_target} T={wl.temperature} top_p={wl.top_p}")
    x = WL.make_decode_inputs(wl, device=dev)
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    ldk = torch.empty(G, Bt, V, device=dev)         # draft logits, one slice per draft step
    lt = torch.empty(Bt * (G + 1), V, device=dev)
    tok = torch.empty(G, Bt, dtype=torch.int32, device=dev)
    u_acc = x["u_accept"].t().contiguous()          # [gamma, batch], drafting order
    n_acc = torch.empty(Bt, dtype=torch.int32, device=dev)
    nxt = torch.empty(Bt, dtype=torch.int32, device=dev)
    ws_b = B.spec_verify_workspace(Bt, G)
    ws = torch.empty(ws_b, dtype=torch.uint8, device=dev)
    samp = B.make_sampling(V, wl.temperature, wl.top_p)
    od = x["o_draft"].reshape(G, Bt, -1)
    # the draft rows' distribution records, kept by the sampler for the verification
    dpar = torch.empty(max(G, 1) * Bt * B.ROW_PARAMS_BYTES, dtype=torch.uint8, device=dev)
    dpar_k = [dpar.data_ptr() + k * Bt * B.ROW_PARAMS_BYTES for k in range(G)]
    cats = ["draft_head", "sample", "verify_head", "verify"]

    def run(cat, st):
        """The library calls of one kernel category of a step, on stream handle st."""
        if cat == "draft_head":
            for k in range(G):
                B.head_logits(Bt, V, wl.d_draft, B.MLS_BF16, od[k].data_ptr(),
                              x["W_draft"].data_ptr(), ldk[k].data_ptr(), st)
        elif cat == "sample":
            for k in range(G):
                B.sample(samp, Bt, ldk[k].data_ptr(), x["u_draft"][k].data_ptr(),
                         tok[k].data_ptr(), st, params=dpar_k[k])
        elif cat == "verify_head":
            B.head_logits(Bt * (G + 1), V, wl.d_target, B.MLS_BF16, x["o_target"].data_ptr(),
                          x["W_target"].data_ptr(), lt.data_ptr(), st)
        else:
            B.spec_verify(samp, Bt, G, ldk.data_ptr(), lt.data_ptr(), tok.data_ptr(),
                          u_acc.data_ptr(), x["u_sample"].data_ptr(), n_acc.data_ptr(),
                          nxt.data_ptr(), ws.data_ptr(), ws_b, st, draft_params=dpar.data_ptr())

    def step(st):
        for k in range(G):
            B.head_logits(Bt, V, wl.d_draft, B.MLS_BF16, od[k].data_ptr(),
                          x["W_draft"].data_ptr(), ldk[k].data_ptr(), st)
            B.sample(samp, Bt, ldk[k].data_ptr(), x["u_draft"][k].data_ptr(),
                     tok[k].data_ptr(), st, params=dpar_k[k])
        run("verify_head", st)
        run("verify", st)

    def capture(fn):
        """One call of fn captured as a HIP graph (after a run on the capture stream)."""
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            fn(side.cuda_stream)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(torch.cuda.current_stream(dev).cuda_stream)
        torch.cuda.synchronize()
        return g

    def timed(fn, n):
        """Median time of n calls, each bracketed by its own events."""
        return step_stats(time_steps(torch, fn, stream, n))["median"]

    for _ in range(args.warmup):
        step(sh)
    torch.cuda.synchronize()
    eager_out = [t.clone() for t in (tok, n_acc, nxt)]
    eager_ms = timed(lambda: step(sh), args.steps)
    # The step is launch-bound when each library call is issued from Python, so
    # the timed region replays a HIP graph of one step: the same kernels on the
    # same buffers, without host launch gaps.
    g_step = capture(step)
    g_cat = {c: capture(lambda st, c=c: run(c, st)) for c in cats}
    for t in (tok, n_acc, nxt):
        t.fill_(-7)
    g_step.replay()
    torch.cuda.synchronize()
    replay_ok = all(torch.equal(a, b) for a, b in zip(eager_out, (tok, n_acc, nxt)))
    for _ in range(args.warmup):
        g_step.replay()
    ms_step = timed(g_step.replay, args.steps)
    per = {c: timed(g_cat[c].replay, args.steps) for c in cats}
    replay_ok = replay_ok and all(torch.equal(a, b) for a, b in zip(eager_out, (tok, n_acc, nxt)))
    if not replay_ok:
        raise SystemExit("graph replay outputs differ from the eager step")
    rows = Bt * G + Bt * (G + 1)
    log(f"{ms_step:.3f} ms/step (graph replay; eager launches {eager_ms:.3f} ms/step), "
        f"mean accepted {n_acc.float().mean().item():.2f} of {G}")
    for c in cats:
        log(f"  {c:12s} {per[c]:8.4f} ms/step")
    # algorithmic work per step of each kernel category
    dd, dt_ = wl.d_draft, wl.d_target
    draft_bytes = G * (V * dd * 2 + Bt * dd * 2 + Bt * V * 4)
    verify_flops = 2.0 * Bt * (G + 1) * V * dt_
    verify_bytes = V * dt_ * 2 + Bt * (G + 1) * (dt_ * 2 + V * 4)
    sample_bytes = G * (Bt * V * 4 + Bt * 8)
    work = {
        "draft_head": ("hbm", draft_bytes, HBM_PEAK, "GB/s", 1e9),
        "verify_head": ("mfma", verify_flops, PEAK_FLOPS["bf16"], "TFLOP/s", 1e12)
        if verify_flops / verify_bytes > PEAK_FLOPS["bf16"] / HBM_PEAK
        else ("hbm", verify_bytes, HBM_PEAK, "GB/s", 1e9),
        "sample": ("hbm", sample_bytes, HBM_PEAK, "GB/s", 1e9),
    }
    dom = max(work, key=lambda c: per[c])
    bound, amount, peak, unit, scale = work[dom]
    achieved = amount / (per[dom] / 1e3)
    if args.copy_mib > 0:
        src = torch.ones(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_decode(wl, x, args.cpu_rows)
    out = {
        "metric": METRIC_DECODE,
        "value": rows / (ms_step / 1e3),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 heads and hidden states, fp32 logits and sampling",
        "data": "synthetic (seeded nested draft/verifier heads and hidden states, input uniforms)",
        "config": {"workload": name, "batch": Bt, "gamma": G, "V": V, "d_draft": dd,
                   "d_verifier": dt_, "temperature": wl.temperature, "top_p": wl.top_p,
                   "parallelism": "single GPU"},
        "mean_accepted": n_acc.float().mean().item(),
        "launch": "one step captured as a HIP graph and replayed (outputs checked against "
                  "the eager step)",
        "eager_ms_per_step": eager_ms,
        "roofline": {"bound": bound, "kernel": dom, "achieved": achieved / scale,
                     "peak": peak / scale, "unit": unit, "frac": achieved / peak,
                     "traffic": profiled_traffic(name, dom, "decode")},
        "ms_per_step_by_kernel": per,
        "cpu_baseline": cpu,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(out), flush=True)


def main_mfma_ceiling(args):
    """Rate of independent v_mfma_f32_32x32x16_bf16 on register operands (no memory,
    no LDS) with all-zero and with random bf16 operands: the ceiling any kernel built
    on this instruction can reach on this device, next to the nominal peak."""
    import torch
    from paper_2608_09703_amd import binding as B
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    sink = torch.empty(B.MFMA_PROBE_SINK_FLOATS, dtype=torch.float32, device=dev)
    iters = 20000
    res = {}
    for kind in ("zero", "random"):
        flops = B.mfma_probe(kind == "random", iters, None, 0, None)
        fn = lambda: B.mfma_probe(kind == "random", iters, sink.data_ptr(), sink.numel(),  # noqa: E731
                                  stream.cuda_stream)
        for _ in range(args.warmup):
            fn()
        st = step_stats(time_steps(torch, fn, stream, args.steps))
        res[kind] = {"ms_per_launch": st["median"], "tflops": flops / (st["median"] / 1e3) / 1e12,
                     "frac_of_nominal": flops / (st["median"] / 1e3) / PEAK_FLOPS["bf16"]}
        log(f"{kind:6s} operands: {res[kind]['tflops']:.0f} TFLOP/s "
            f"({100 * res[kind]['frac_of_nominal']:.1f}% of the nominal bf16 peak)")
    device = device_peaks()
    out = {
        "metric": "bf16 MFMA ceiling, v_mfma_f32_32x32x16_bf16 on register operands (TFLOP/s)",
        "value": res["random"]["tflops"], "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": res["random"]["ms_per_launch"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic register operands (zero, and random bf16 in +-[1, 2))",
        "config": {"workload": "mfma_ceiling", "blocks": 2048, "threads": 256,
                   "chains_per_wave": 8, "iters": iters, "parallelism": "single GPU"},
        "zero_operands": res["zero"], "random_operands": res["random"], "device": device,
        "roofline": {"bound": "mfma", "kernel": "mfma_probe", "achieved": res["random"]["tflops"],
                     "peak": PEAK_FLOPS["bf16"] / 1e12, "unit": "TFLOP/s",
                     "frac": res["random"]["frac_of_nominal"], "traffic": 0},
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the library runs on one GPU; a vocabulary-parallel split over "
                                   "several GPUs is designed but not implemented",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.junction:
        return main_junction(args)
    if args.decode:
        return main_decode(args)
    if args.mfma_ceiling:
        return main_mfma_ceiling(args)

    import torch
    from paper_2608_09703_amd import binding as B
    from paper_2608_09703_amd import api as D
    from paper_2608_09703_amd import workloads as WL

    name = args.workload or WL.HEADLINE
    wl = WL.WORKLOADS[name]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload {name}: M={wl.M} T={wl.T} dims={wl.dims} V={wl.V} {wl.dtype} "
        f"alpha={wl.alpha} tau={wl.tau}")
    h, W, y = WL.make_inputs(wl, device=dev)
    flags = B.MLS_FWD_BWD_RECOMPUTE if args.path == "recompute" else 0
    p = D.make_problem(h, W, y, tau=wl.tau, alpha=wl.alpha, vocab_chunk=args.vocab_chunk, flags=flags)
    buf = D.Buffers(p, dev)
    if args.path != "separate" and not args.diagnostics:
        fb_bytes = B.query_fwd_bwd_workspace(p)
        if fb_bytes > buf.workspace.numel():
            buf.workspace = torch.empty(fb_bytes, dtype=torch.uint8, device=dev)
    g_ce, g_kl = D.coefficients(wl.M, alpha=wl.alpha, tau=wl.tau)
    gce = torch.tensor(g_ce, dtype=torch.float32, device=dev)
    gkl = torch.tensor(g_kl, dtype=torch.float32, device=dev)
    gh = [torch.empty(x.shape, dtype=torch.float32, device=dev) for x in h]
    gW = [torch.empty(x.shape, dtype=torch.float32, device=dev) for x in W]
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    ws_ptr, ws_n = buf.workspace.data_ptr(), buf.workspace.numel()
    st_ptr = buf.stats.data_ptr()
    gh_p = [x.data_ptr() for x in gh]
    gW_p = [x.data_ptr() for x in gW]
    kl_pair = torch.empty(wl.M, wl.M, dtype=torch.float32, device=dev)
    agree = torch.empty(wl.M, wl.M, dtype=torch.float32, device=dev)

    def step():
        if args.diagnostics:
            B.diagnostics(p, kl_pair.data_ptr(), agree.data_ptr(), None, ws_ptr, ws_n, sh)
            return
        if args.path == "separate":
            B.distill_fwd(p, st_ptr, buf.ce.data_ptr(), buf.kl.data_ptr(), buf.entropy.data_ptr(),
                          ws_ptr, ws_n, sh)
            B.distill_bwd(p, st_ptr, gce.data_ptr(), gkl.data_ptr(), gh_p, gW_p, ws_ptr, ws_n, sh)
        else:
            B.distill_fwd_bwd(p, st_ptr, buf.ce.data_ptr(), buf.kl.data_ptr(),
                              buf.entropy.data_ptr(), gce.data_ptr(), gkl.data_ptr(), gh_p, gW_p,
                              ws_ptr, ws_n, sh)

    log(f"workspace {ws_n / 2**20:.0f} MiB, stats {buf.stats.numel() / 2**20:.1f} MiB")
    for k in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps done")

    # timed region: one event pair per step, no other work recorded; the median step
    times = time_steps(torch, step, stream, args.steps)
    st = step_stats(times)
    ms_step = st["median"]
    tokens_per_s = wl.T / (ms_step / 1e3)
    log(f"step times (ms): median {st['median']:.3f} mean {st['mean']:.3f} "
        f"min {st['min']:.3f} max {st['max']:.3f}")
    # per-kernel breakdown in a separate pass (the library's event timer brackets
    # every launch, which costs a little, so it stays out of the timed steps)
    B.profile_enable(True)
    torch.cuda.synchronize()
    for k in range(args.steps):
        step()
    torch.cuda.synchronize()
    B.profile_enable(False)
    prof = B.profile_report()
    # forward + backward: 6*T*V*sum(d); diagnostics: one 2*T*V*sum(d) pass
    flops_step = wl.algorithmic_flops() * (1.0 / 3.0 if args.diagnostics else 1.0)
    peak = PEAK_FLOPS[wl.dtype]
    pct = flops_step / (ms_step / 1e3) / peak * 100.0
    log(f"{args.steps} steps: {ms_step:.3f} ms/step, {tokens_per_s:,.0f} tokens/s, "
        f"{pct:.1f}% of {wl.dtype} MFMA peak (algorithmic)")
    device = device_peaks()
    log(f"peaks: nominal bf16 {PEAK_FLOPS['bf16'] / 1e12:.0f} TFLOP/s, from the device's "
        f"{device['compute_units']} CUs x {device['clock_mhz']:.0f} MHz x 4096 FLOP/clk: "
        f"{device['bf16_peak_tflops_derived']:.0f} TFLOP/s")

    # per-kernel times from the library's event timer (profiling pass)
    kernels = {}
    for kname, (launches, tot) in prof.items():
        kernels[kname] = {"launches_per_step": launches / args.steps,
                          "ms_per_step": tot / args.steps,
                          "avg_launch_ms": tot / launches}
        log(f"  {kname:14s} {launches / args.steps:5.1f} launches/step "
            f"{tot / args.steps:8.3f} ms/step  avg {tot / launches:8.4f} ms")
    # dense work per step of each MFMA kernel: the forward and the recompute each
    # contract 2*T*V*sum(d); the gradient GEMM launch holds both head products
    one = 2.0 * wl.T * wl.V * sum(wl.dims)
    dense = {"fused_fwd": one, "fused_bwd": one, "gemm_grads": 2.0 * one, "diag_tiles": one}
    dom = max((k for k in kernels if k in dense), key=lambda k: kernels[k]["ms_per_step"])
    per_launch = dense[dom] / kernels[dom]["launches_per_step"]
    achieved = per_launch / (kernels[dom]["avg_launch_ms"] / 1e3)
    roofline = {
        "bound": "mfma",
        "kernel": dom,
        "achieved": achieved / 1e12,
        "peak": peak / 1e12,
        "unit": "TFLOP/s",
        "frac": achieved / peak,
        # the recompute plan has a summary of its own (its launches differ from
        # the default plan's); --path separate runs the same launches
        "traffic": profiled_traffic(name, dom, args.diagnostics or
                                    ("recompute" if args.path != "fwd_bwd" else False)),
    }

    if args.copy_mib > 0:
        src = torch.ones(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.copy_mib} MiB done")
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample of rows")
        cpu = cpu_baseline(wl, h, W, y, g_ce, g_kl, args.cpu_rows, args.diagnostics)
        log(f"oracle: {cpu['value']:.2f} tokens/s on {cpu['cores']} threads")

    out = {
        "metric": METRIC_DIAG if args.diagnostics else
                  (METRIC if name == WL.HEADLINE else
                   f"fused LM-head+CE+KL fwd+bwd tokens/s (M={wl.M}, V={wl.V}); % of bf16 MFMA peak"),
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_stats": st,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded Gaussian hidden states and heads, uniform labels)",
        "config": {"workload": name, "M": wl.M, "T": wl.T, "batch": wl.batch, "seq": wl.seq,
                   "widths": list(wl.dims), "V": wl.V, "alpha": wl.alpha, "tau": wl.tau,
                   "ignore_frac": wl.ignore_frac, "parallelism": "single GPU",
                   "path": None if args.diagnostics else args.path},
        "pct_of_bf16_peak": pct if wl.dtype == "bf16" else None,
        "algorithmic_tflop_per_step": flops_step / 1e12,
        # a recomputing backward executes the logits product once more: 8 T V sum(d)
        "executed_tflop_per_step": flops_step * (4.0 / 3.0 if "fused_bwd" in kernels else 1.0) / 1e12,
        "device": device,
        "roofline": roofline,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
