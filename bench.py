#!/usr/bin/env python3
"""Benchmark of the GLIDE hybrid-attention hot path on one MI355X.

One step = one whole pass of the path over one synthetic batch:
  state init -> chunked prefill of the context over the whole layer stack ->
  every decode step of the workload (one call per step, all layers).
Inputs (q, k, v for prefill and for every decode step, Wf) are generated on
the GPU and resident in HBM before the timed region starts.

The default workload is the decode-heavy 32-layer Llama-3-8B-shaped stack:
batch 32, per-sequence context 16K-32K, windows geo(64 -> 4096), 128 decode
steps.  Its prefill reuses one layer's resident inputs for every layer (all
of a layer's inputs for 786K tokens take 9.7 GB; the whole stack's would not
fit).  Printed (one JSON line):
  value       decode tokens/s of the whole stack (batch / decode time per step)
  roofline    the decode step against HBM: algorithmic bytes (window K/V, new
              token in and into the ring, q in and O out, the fp32 state read
              every step and written once per fold period, Wf per layer) over
              the HIP-event time of the decode steps on the library's stream
  roofline_other  the prefill call against bf16 MFMA peak (algorithmic flops)
  decode_detail   per-step p10/p50/p90, and the stack called one layer at a
              time (eager and as one replayed HIP graph)
  b1_ctx8k    the batch-1, 8K-context stack: decode warm (its working set fits
              the 256 MB Infinity Cache) and cold (a 1 GiB copy sweeps the
              cache between steps; events around the decode call only),
              prefill, per-layer calls
  cpu_baseline  the CPU oracle on a bounded sample of the same decode step,
              with the threads it used and a one-thread figure; its prefill
              (the quadratic definition form) timed whole when that takes
              seconds, else sampled and extrapolated by its per-position cost
--workload selects another workload (c1 c2 c3 c3b c4u c4 c5 ...); the extra
batch-1 block is only added to the default one.
"""
import argparse
import json
import os
import sys
import time

HBM_PEAK = 8.0e12          # bytes/s, MI355X
MFMA_BF16_PEAK = 2.5e15    # dense bf16 flop/s
MFMA_FP32_PEAK = 157.3e12  # dense fp32 matrix flop/s
FOLD_PERIOD = 8            # decode writes a unit's state back once per this many steps
COLD_SWEEP_BYTES = 1 << 30  # > the 256 MB Infinity Cache


def _unit_decode_bytes(W, d, Df, G, e, state_write):
    """Bytes one (layer, sequence, KV head) unit moves in one decode step:
    window K/V (W tokens, the one leaving the window included), new k/v in,
    ring write, q in and O out, the fp32 state S, z read, plus `state_write`
    times their size written."""
    return (2 * W * d * e + 2 * d * e + 2 * d * e + 2 * G * d * e
            + (1 + state_write) * (Df * d * 4 + Df * 4))


def decode_bytes(wl, state_write=None):
    """Algorithmic bytes of one decode step over the stack.  By default the
    state write is charged once per fold period (what the deferred fold
    moves); state_write=1 charges it every step (the recurrence as written,
    one fold per token).  Every layer of the benchmark workloads has a
    non-empty linear part, so every unit reads its state."""
    e = 2 if wl.dtype.itemsize == 2 else 4
    d, Df, G = wl.head_dim, wl.feat_dim, wl.G
    tot = 0
    for W in wl.windows:
        sw = (1.0 / FOLD_PERIOD if W > 0 else 1.0) if state_write is None else state_write
        tot += _unit_decode_bytes(W, d, Df, G, e, sw) * wl.batch * wl.n_kv_heads + d * Df * e
    return int(round(tot))


def prefill_flops(wl, lens):
    """Algorithmic flops of a prefill of `lens[b]` tokens per sequence over the
    stack: phi of q and k, the banded QK^T and PV, the state update and the
    read-out (masked band work and intra-chunk overheads excluded)."""
    d, Df, G = wl.head_dim, wl.feat_dim, wl.G
    tot = 0
    for W in wl.windows:
        for n in lens:
            band = n * (n + 1) // 2 if W >= n else W * (W + 1) // 2 + (n - W) * W   # sum_t min(t+1, W)
            unit = 2 * ((G + 1) * n * d * Df + 2 * G * d * band + n * Df * d + G * n * Df * d)
            tot += unit * wl.n_kv_heads
    return tot


def _r(x, n=4):
    return {k: (round(v, n) if isinstance(v, float) else v) for k, v in x.items()}


class Run:
    """One workload resident on the GPU: library handle, state, workspace and
    every input of the prefill and of each decode step."""

    def __init__(self, wl, form=0, phi_kind=0, gated=False):
        import torch
        from paper_2607_24788_amd import glide, workload as W
        self.wl = wl
        self.form, self.phi_kind, self.gated = form, phi_kind, gated
        dev = torch.device("cuda:0")
        self.g = glide.Glide(wl.n_layers, wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.feat_dim,
                             wl.windows, dtype=wl.dtype, sm_scale=wl.tau, form=form, phi=phi_kind, gated=gated)
        self.lens = list(wl.context)
        self.cu = [0]
        for n in self.lens:
            self.cu.append(self.cu[-1] + n)
        T = self.T = self.cu[-1]
        L = wl.n_layers
        self.share_prefill = sum(wl.context) > 1_000_000 or wl.batch * max(wl.context) > 400_000
        n_pre = 1 if self.share_prefill else L
        self.phi = W.phi_weights(wl, device=dev)
        self.qp = torch.empty((n_pre, T, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
        self.kp = torch.empty((n_pre, T, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=dev)
        self.vp = torch.empty_like(self.kp)
        for l in range(n_pre):
            self.qp[l], self.kp[l], self.vp[l] = W.prefill_inputs(wl, l, self.lens, device=dev)
        S = wl.decode_steps
        self.dq = torch.empty((S, L, wl.batch, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
        self.dk = torch.empty((S, L, wl.batch, wl.n_kv_heads, wl.head_dim), dtype=wl.dtype, device=dev)
        self.dv = torch.empty_like(self.dk)
        for s in range(S):
            self.dq[s], self.dk[s], self.dv[s] = W.decode_inputs(wl, s, device=dev)
        self.pg = self.dg = None
        if gated:
            self.pg = torch.stack([W.prefill_log_gates(wl, l, self.lens, device=dev) for l in range(n_pre)])
            self.dg = torch.stack([W.decode_log_gates(wl, s, device=dev) for s in range(S)])
        self.pout = torch.empty((n_pre, T, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
        self.dout = torch.empty((L, wl.batch, wl.n_q_heads, wl.head_dim), dtype=wl.dtype, device=dev)
        self.state = self.g.new_state(dev)
        self.ws = self.g.new_workspace(T, dev)
        self.stream = torch.cuda.current_stream()

    def prefill(self):
        g, wl = self.g, self.wl
        if self.share_prefill:
            for l in range(wl.n_layers):
                g.prefill(self.state, self.phi[l:l + 1], self.qp, self.kp, self.vp, self.cu, self.pout, self.ws,
                          layer0=l, n_layers=1, chunk=wl.chunk, log_gates=self.pg)
        else:
            g.prefill(self.state, self.phi, self.qp, self.kp, self.vp, self.cu, self.pout, self.ws, chunk=wl.chunk,
                      log_gates=self.pg)

    def fresh(self):
        self.g.state_init(self.state)
        self.prefill()

    def decode(self, s):
        self.g.decode_step(self.state, self.phi, self.dq[s], self.dk[s], self.dv[s], self.dout, self.ws,
                           log_gates=None if self.dg is None else self.dg[s])

    def decode_layer(self, s, l):
        self.g.decode_step(self.state, self.phi[l:l + 1], self.dq[s, l:l + 1], self.dk[s, l:l + 1],
                           self.dv[s, l:l + 1], self.dout[l:l + 1], self.ws, layer0=l, n_layers=1,
                           log_gates=None if self.dg is None else self.dg[s, l:l + 1])

    def timed_steps(self, steps, warmup):
        """The timed region: `warmup` untimed, then `steps` whole passes (init,
        prefill, every decode step), HIP events on the library's stream."""
        import torch
        wl = self.wl
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps + warmup)]

        def one(e):
            self.g.state_init(self.state)
            e[0].record(self.stream)
            self.prefill()
            e[1].record(self.stream)
            for s in range(wl.decode_steps):
                self.decode(s)
            e[2].record(self.stream)

        for i in range(warmup):
            one(ev[i])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(warmup, warmup + steps):
            one(ev[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        pre_ms = sum(ev[i][0].elapsed_time(ev[i][1]) for i in range(warmup, warmup + steps)) / steps
        dec_ms = sum(ev[i][1].elapsed_time(ev[i][2]) for i in range(warmup, warmup + steps)) / steps
        return wall, pre_ms, dec_ms

    def figures(self, pre_ms, dec_ms):
        """Throughputs and roofline fractions of the timed region."""
        import torch
        wl = self.wl
        n = wl.decode_steps
        dec_step_s = dec_ms * 1e-3 / max(n, 1)
        dec_bytes = decode_bytes(wl)
        pre_flops = prefill_flops(wl, self.lens)
        mfma_peak = MFMA_BF16_PEAK if wl.dtype == torch.bfloat16 else MFMA_FP32_PEAK
        traffic = measured_traffic(wl.name) if self.form == 0 and self.phi_kind == 0 and not self.gated else None
        hbm = {"bound": "hbm", "kernel": "decode step (decode_kernel over the whole stack; split windows "
                                         "merged by their last piece)",
               "achieved": dec_bytes / dec_step_s / 1e9, "peak": HBM_PEAK / 1e9, "unit": "GB/s",
               "frac": dec_bytes / dec_step_s / HBM_PEAK,
               "traffic": traffic and traffic["decode_step_bytes"],
               "algorithmic_bytes_per_launch": dec_bytes,
               "bytes_if_state_written_every_step": decode_bytes(wl, state_write=1),
               "avg_launch_us": dec_step_s * 1e6}
        mfma = {"bound": "mfma", "kernel": "glide_prefill over the stack (prefill_main + segsum/scan/ringfill/"
                                          "advance/gather per layer batch)",
                "achieved": pre_flops / (pre_ms * 1e-3) / 1e12, "peak": mfma_peak / 1e12, "unit": "TFLOP/s",
                "frac": pre_flops / (pre_ms * 1e-3) / mfma_peak,
                "traffic": traffic and traffic["prefill_call_bytes"],
                "algorithmic_flops_per_launch": pre_flops, "avg_launch_us": pre_ms * 1e3}
        return {"decode_tokens_per_s": wl.batch * n / (dec_ms * 1e-3) if n else None,
                "decode_us_per_step": dec_step_s * 1e6 if n else None,
                "decode_hbm_frac": hbm["frac"] if n else None,
                "prefill_tokens_per_s": self.T / (pre_ms * 1e-3), "prefill_ms": pre_ms,
                "prefill_mfma_frac": mfma["frac"], "hbm": hbm, "mfma": mfma}

    def detail(self, reps=2):
        """Decode timings outside the timed region: every step of one pass on
        its own (median, p10, p90 of the whole-stack call), and the same steps
        as one library call per layer, the way a model that interleaves
        layers calls it: eagerly, and captured once in a HIP graph and
        replayed."""
        import torch
        wl = self.wl
        L, n = wl.n_layers, wl.decode_steps
        self.fresh()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        ev[0].record(self.stream)
        for s in range(n):
            self.decode(s)
            ev[s + 1].record(self.stream)
        torch.cuda.synchronize()
        us = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(n))
        pct = lambda f: us[min(n - 1, int(round(f * (n - 1))))]

        def per_layer():
            for s in range(n):
                for l in range(L):
                    self.decode_layer(s, l)

        def timed(run):
            best = None
            for _ in range(reps):
                self.fresh()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(self.stream)
                run()
                e1.record(self.stream)
                torch.cuda.synchronize()
                t = e0.elapsed_time(e1) * 1e3 / n
                best = t if best is None else min(best, t)
            return best

        eager_us = timed(per_layer)
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(self.stream)
        with torch.cuda.graph(graph, stream=side):
            per_layer()
        torch.cuda.synchronize()
        graph_us = timed(graph.replay)
        del graph
        db = decode_bytes(wl)
        return {"step_us_median": round(pct(0.5), 2), "step_us_p10": round(pct(0.1), 2),
                "step_us_p90": round(pct(0.9), 2),
                "tokens_per_s_at_median": round(wl.batch / (pct(0.5) * 1e-6), 2),
                "per_layer_calls_eager_us_per_step": round(eager_us, 2),
                "per_layer_calls_graph_us_per_step": round(graph_us, 2),
                "per_layer_calls_graph_us_per_layer": round(graph_us / L, 3),
                "per_layer_calls_graph_tokens_per_s": round(wl.batch / (graph_us * 1e-6), 2),
                "per_layer_calls_graph_hbm_frac": round(db / (graph_us * 1e-6) / HBM_PEAK, 4)}

    def cold_decode(self, steps=None):
        """Decode steps with the Infinity Cache swept between them (a 1 GiB
        device copy, untimed); events around each decode call only."""
        import torch
        wl = self.wl
        n = wl.decode_steps if steps is None else min(steps, wl.decode_steps)
        src = torch.empty(COLD_SWEEP_BYTES, dtype=torch.uint8, device="cuda")
        src.fill_(1)
        dst = torch.empty_like(src)
        self.fresh()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
        for s in range(n):
            dst.copy_(src)
            ev[s][0].record(self.stream)
            self.decode(s)
            ev[s][1].record(self.stream)
        torch.cuda.synchronize()
        us = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
        med = us[len(us) // 2]
        del src, dst
        return {"decode_us_median": round(med, 2), "decode_us_p10": round(us[int(0.1 * (n - 1))], 2),
                "decode_us_p90": round(us[int(round(0.9 * (n - 1)))], 2),
                "decode_tokens_per_s": round(wl.batch / (med * 1e-6), 2),
                "decode_hbm_frac": round(decode_bytes(wl) / (med * 1e-6) / HBM_PEAK, 4), "steps": n,
                "sweep": "1 GiB device-to-device copy before each step (untimed)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", default="c3")
    ap.add_argument("--form", type=int, default=0, choices=(0, 1, 2),
                    help="merge: 0 GLIDE's shared denominator (default); 1, 2 the Appendix's two hybrid "
                         "forms (separately normalised sum; state over the evicted tokens / every token)")
    ap.add_argument("--phi", type=int, default=0, choices=(0, 1, 2),
                    help="feature map: 0 ReLU (default), 1 ELU + 1, 2 softmax over the features")
    ap.add_argument("--gated", action="store_true",
                    help="the gated (GLA-style) linear state: log-gates uniform in [-0.4, 0] per token and KV head")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-detail", action="store_true",
                    help="skip the per-step decode distribution and the per-layer (eager and graph) decode runs")
    ap.add_argument("--no-extra", action="store_true", help="skip the batch-1 8K-context block")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run 5 device-to-device copies of MIB MiB (the known-size kernel that "
                         "calibrates the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested); the hybrid-attention "
              "step is implemented for one GPU (sharding across GPUs is a design note only)", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    import torch
    from paper_2607_24788_amd import workload as W

    torch.cuda.set_device(0)
    wl = W.workload(args.workload)
    big = sum(wl.context) > 1_000_000 or wl.batch * max(wl.context) > 400_000
    steps = args.steps if args.steps is not None else (3 if big else 10)
    warmup = args.warmup if args.warmup is not None else (1 if big else 2)
    if args.gated and args.form:
        print("the gated state combines with the shared denominator only (--form 0)", file=sys.stderr)
        sys.exit(2)
    run = Run(wl, args.form, args.phi, args.gated)
    wall, pre_ms, dec_ms = run.timed_steps(steps, warmup)
    f = run.figures(pre_ms, dec_ms)
    has_decode = wl.decode_steps > 0
    dominant, other = (f["hbm"], f["mfma"]) if has_decode else (f["mfma"], None)
    line = {
        "metric": "decode tokens/s per layer-stack + % HBM peak; prefill tokens/s + % MFMA",
        # prefill-only workloads report their prefill throughput instead
        "value": round(f["decode_tokens_per_s"] if has_decode else f["prefill_tokens_per_s"], 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(wall * 1e3 / steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {torch.bfloat16: "bf16", torch.float32: "fp32"}[wl.dtype],
        "data": "synthetic (seeded N(0,1)/sqrt(d) q,k,v; Wf ~ N(0,1/d))"
                + ("; prefill inputs of one layer reused by every layer" if run.share_prefill else ""),
        "config": dict(wl.describe(), chunk=wl.chunk, **({"form": args.form} if args.form else {}),
                       **({"phi": args.phi} if args.phi else {}), **({"gated": True} if args.gated else {})),
        "decode_tokens_per_s": f["decode_tokens_per_s"] and round(f["decode_tokens_per_s"], 2),
        "decode_us_per_step": f["decode_us_per_step"] and round(f["decode_us_per_step"], 2),
        "decode_hbm_frac": f["decode_hbm_frac"] and round(f["decode_hbm_frac"], 4),
        "prefill_tokens_per_s": round(f["prefill_tokens_per_s"], 1),
        "prefill_ms": round(pre_ms, 3),
        "prefill_mfma_frac": round(f["prefill_mfma_frac"], 4),
        "roofline": _r(dominant),
        "roofline_other": other and _r(other),
    }
    print(f"timed region done: {json.dumps({k: line[k] for k in ('value', 'ms_per_step')})}", file=sys.stderr,
          flush=True)
    if not args.no_detail and has_decode:
        line["decode_detail"] = run.detail()
        print("decode detail done", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline and has_decode and not args.gated:
        line["cpu_baseline"] = cpu_baseline(run, args.cpu_baseline_seconds)
        print("cpu baseline done", file=sys.stderr, flush=True)
    if args.workload == "c3" and not args.no_extra and args.form == 0 and args.phi == 0 and not args.gated:
        del run
        torch.cuda.empty_cache()
        line["b1_ctx8k"] = batch1_block(W.workload("c2"), args.no_detail)
        print("batch-1 block done", file=sys.stderr, flush=True)
    print(json.dumps(line), flush=True)


def batch1_block(wl, no_detail):
    """The batch-1, 8K-context stack: warm and cold-cache decode, prefill, and
    per-layer calls (not part of `value`)."""
    run = Run(wl)
    wall, pre_ms, dec_ms = run.timed_steps(10, 2)
    f = run.figures(pre_ms, dec_ms)
    out = {"workload": wl.name,
           "decode_tokens_per_s": round(f["decode_tokens_per_s"], 2),
           "decode_us_per_step": round(f["decode_us_per_step"], 2),
           "decode_hbm_frac_warm": round(f["decode_hbm_frac"], 4),
           "decode_algorithmic_bytes": f["hbm"]["algorithmic_bytes_per_launch"],
           "decode_traffic": f["hbm"]["traffic"],
           "prefill_tokens_per_s": round(f["prefill_tokens_per_s"], 1),
           "prefill_ms": round(pre_ms, 3),
           "prefill_mfma_frac": round(f["prefill_mfma_frac"], 4),
           "prefill_traffic": f["mfma"]["traffic"],
           "cold": run.cold_decode(64)}
    if not no_detail:
        out["decode_detail"] = run.detail()
    return out


def kernel_sources_hash():
    """sha256 prefix over the kernel sources (csrc/*.hip, csrc/*.h, include/glide.h)."""
    import glob
    import hashlib
    root = os.path.dirname(os.path.abspath(__file__))
    files = sorted(glob.glob(os.path.join(root, "paper_2607_24788_amd", "csrc", "*.hip")) +
                   glob.glob(os.path.join(root, "paper_2607_24788_amd", "csrc", "*.h")))
    files.append(os.path.join(root, "include", "glide.h"))
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_name):
    """HBM-side bytes per prefill call and per decode step from the rocprofv3
    FETCH_SIZE / WRITE_SIZE runs summarised in profiles/ (copy-calibrated);
    None when the kernels have changed since the counters were taken."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("sources_sha256_16") != kernel_sources_hash():
        return None
    w = t.get("workloads", {}).get(workload_name)
    if not w:
        return None
    return {"decode_step_bytes": round(w["decode_step_bytes"]), "prefill_call_bytes": round(w["prefill_call_bytes"])}


def copy_probe(mib):
    """Plain device-to-device copies of a known size: under rocprofv3 --pmc
    their FETCH_SIZE / WRITE_SIZE per dispatch give the factor that turns the
    counters into bytes."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "copies": 5}), flush=True)


def _omp():
    """libgomp, which the oracle's OpenMP regions run on (None if absent)."""
    import ctypes
    try:
        lib = ctypes.CDLL("libgomp.so.1")
    except OSError:
        return None
    lib.omp_get_max_threads.restype = ctypes.c_int
    lib.omp_set_num_threads.argtypes = [ctypes.c_int]
    return lib


def cpu_baseline(run, budget_s):
    """The CPU oracle (plain C, float64, OpenMP over (sequence, KV head)) on a
    bounded sample of the workload's decode step: the first and the last
    sequence through every layer, from the GPU's state after the benchmark
    (pending tokens folded), each step with its own inputs.  Sequences are
    independent, so the sample's tokens/s is the whole batch's.  Run with
    every thread OpenMP offers, then with one."""
    import numpy as np
    import torch

    import oracle
    from paper_2607_24788_amd import glide as gl

    wl, g = run.wl, run.g
    g.state_flush(run.state, run.phi)     # the oracle's state is the direct sum over the linear part
    torch.cuda.synchronize()
    seqs = sorted({0, wl.batch - 1})
    d = wl.head_dim

    def load_states():
        states = []
        for l in range(wl.n_layers):
            v = g.layer_views(run.state, l)
            W, R = v["window"], v["ring_slots"]
            pos = v["pos"][seqs, 0].cpu().numpy().astype(np.int64)
            st = {"S": v["S"][seqs].double().cpu().numpy(), "z": v["z"][seqs].double().cpu().numpy(),
                  "pos": pos.copy()}
            wk = np.zeros((len(seqs), wl.n_kv_heads, W, d))
            wv = np.zeros_like(wk)
            if R:
                kl = gl.kring_logical(v["kring_raw"][seqs].cpu(), R, d).double().numpy()
                vl = gl.vring_logical(v["vring_raw"][seqs].cpu(), R, d).double().numpy()
                for i in range(len(seqs)):
                    p = int(pos[i])
                    n = min(W, p)
                    idx = [(j % R) for j in range(p - n, p)]
                    wk[i, :, :n] = kl[i][:, idx]
                    wv[i, :, :n] = vl[i][:, idx]
            st["wk"], st["wv"] = wk, wv
            states.append(st)
        return states

    oras = [oracle.Oracle(wl.n_q_heads, wl.n_kv_heads, d, wl.feat_dim, W, tau=wl.tau, form=run.form,
                          phi=run.phi_kind) for W in wl.windows]
    wf = [run.phi[l].double().cpu().numpy() for l in range(wl.n_layers)]
    n_in = max(1, min(wl.decode_steps, 16))
    ins = [tuple(x[s][:, seqs].double().cpu().numpy() for x in (run.dq, run.dk, run.dv)) for s in range(n_in)]

    def timed(budget, max_steps):
        states = load_states()
        steps, el = 0, 0.0
        t0 = time.perf_counter()
        while True:
            q, k, v = ins[steps % n_in]
            for l in range(wl.n_layers):
                oras[l].decode(wf[l], states[l], q[l], k[l], v[l])
            steps += 1
            el = time.perf_counter() - t0
            if el >= budget or steps >= max_steps:
                return steps, el

    omp = _omp()
    threads = omp.omp_get_max_threads() if omp else int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    steps, el = timed(budget_s * 2 / 3, 1000)
    one = None
    if omp:
        omp.omp_set_num_threads(1)
        try:
            s1, e1 = timed(budget_s / 3, 1000)
        finally:
            omp.omp_set_num_threads(threads)
        one = {"value": round(len(seqs) * s1 / e1, 3), "unit": "tokens/s", "cores": 1,
               "sample": f"{s1} steps, {e1:.1f} s"}
    li = [0] * wl.n_layers if run.share_prefill else list(range(wl.n_layers))
    pre = prefill_sample(wl, run.lens, oras, wf,
                         lambda l, b=0: tuple(x[li[l], run.cu[b]:run.cu[b + 1]].double().cpu().numpy()
                                              for x in (run.qp, run.kp, run.vp)),
                         run.form)
    pre["cores"] = threads
    return {"value": round(len(seqs) * steps / el, 3), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{steps} full-stack decode steps ({wl.n_layers} layers) of sequences {seqs} of the batch "
                      f"of {wl.batch}, from the GPU state after the benchmark, {el:.1f} s; sequences are "
                      f"independent, so tokens/s = sequences x steps / time",
            "one_thread": one, "prefill": pre, "cpu_model": _cpu_model()}


def _sum_linear_and_band(n, W, form):
    """Over the positions t < n of one sequence: the summed size of the
    linear set (tokens before the window, every token up to t in form 2) and
    of the window."""
    band = n * (n + 1) // 2 if W >= n else W * (W + 1) // 2 + (n - W) * W
    lin = n * (n + 1) // 2 if form == 2 else ((n - W) * (n - W + 1) // 2 if n > W else 0)
    return lin, band


def prefill_sample(wl, lens, oras, wf, inputs, form, positions=24, full_s=10.0):
    """The oracle's prefill (its quadratic definition form, every output
    position evaluated from the whole history) on a bounded sample: sequence
    0 through the smallest-, middle- and largest-window layers at
    `positions` evenly spaced positions, then scaled to the whole prefill of
    the workload.  Per query head a position t costs the oracle
    (Df + d) x |linear set| + 3d x |window| multiply-adds, plus phi of every
    key row up to the last sampled position once per call; the phi time is
    measured on its own and the rest gives one rate per unit of that cost.
    The result is labelled extrapolated.  When the estimate of the whole
    prefill is under `full_s` seconds, the whole prefill (every layer,
    sequence and position) is timed instead.  inputs(l, b): q, k, v of
    sequence b of layer l."""
    import numpy as np
    d, Df, Hq, Hkv = wl.head_dim, wl.feat_dim, wl.n_q_heads, wl.n_kv_heads
    order = sorted(range(wl.n_layers), key=lambda l: wl.windows[l])
    layers = sorted({order[0], order[len(order) // 2], order[-1]})
    n0 = lens[0]
    pos = np.array(sorted({int((i + 0.5) * n0 / positions) for i in range(positions)}), dtype=np.int64)
    rows = (int(pos[-1]) + 1) * Hkv
    t_att = units = 0.0
    t_phi = None
    for l in layers:
        q, k, v = inputs(l)
        if t_phi is None:
            t0 = time.perf_counter()
            oras[l].phi(wf[l], k[:int(pos[-1]) + 1])
            t_phi = time.perf_counter() - t0
        t0 = time.perf_counter()
        oras[l].attend(wf[l], q, k, v, positions=pos)
        t_att += time.perf_counter() - t0 - t_phi
        W = wl.windows[l]
        for t in pos:
            beta = max(0, int(t) + 1 - W)
            lin = int(t) + 1 if form == 2 else beta
            units += Hq * ((Df + d) * lin + 3 * d * (int(t) + 1 - beta))
    rate = max(t_att, 1e-9) / units
    est = 0.0
    for W in wl.windows:
        for n in lens:
            lin, band = _sum_linear_and_band(n, W, form)
            est += t_phi / rows * n * Hkv + rate * Hq * ((Df + d) * lin + 3 * d * band)
    tokens = sum(lens)
    if est <= full_s:
        t0 = time.perf_counter()
        for l in range(wl.n_layers):
            for b in range(len(lens)):
                if lens[b]:
                    oras[l].attend(wf[l], *inputs(l, b))
        full = time.perf_counter() - t0
        return {"value": round(tokens / full, 4), "unit": "tokens/s", "kind": "oracle", "extrapolated": False,
                "sample": f"the whole prefill: {tokens} tokens x {wl.n_layers} layers, {full:.2f} s "
                          f"(the per-position estimate from a sample was {est:.2f} s)"}
    return {"value": round(tokens / est, 4), "unit": "tokens/s", "kind": "oracle", "extrapolated": True,
            "estimated_seconds": round(est, 1),
            "sample": f"sequence 0 ({n0} tokens) through layers {layers} (windows "
                      f"{[wl.windows[l] for l in layers]}) at {len(pos)} evenly spaced positions each: "
                      f"{t_att + len(layers) * t_phi:.1f} s, scaled to {tokens} tokens x {wl.n_layers} layers by "
                      f"the oracle's per-position cost ((Df + d) per linear-set token and 3d per window token, "
                      f"per query head) and its phi time per key row"}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
