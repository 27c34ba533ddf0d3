"""Throughput of the BGPO ELBO head on one MI355X.

One step = one bgpo_elbo_bwd_accumulate call over every Monte-Carlo sample of
the workload (mask draw, compaction, fused LM-head forward with online
log-sum-exp that also keeps the exponentials, l/g/loss, dZ = s (softmax -
onehot) from the kept exponentials, dX and dW accumulation), on
inputs already resident in device memory.  Default workload: the LLaDA-8B head
shape B=8 responses, L=512, d=4096, V=126464, n_t=64 samples.

Prints ONE JSON line: masked tokens/s (the sum over samples and responses of
masked positions, per second), the roofline of the dominant kernel measured
with HIP events inside the timed region, and the float64 CPU oracle timed on
a bounded sample of the same workload on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
WORKLOADS = {w.name: w for w in workloads.CONFIGS}
DEFAULT = workloads.LLADA_L512_NT64.name
GEMM_CLASSES = ("fwd", "recompute", "dx", "dw")
TRAFFIC_TABLE = os.path.join(ROOT, "profiles", "hbm_traffic_llada_head_B8_L512_nt64.json")


def kernel_source_hash() -> str:
    import glob
    import hashlib
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2510_11683_amd", "csrc", "*"))):
        h.update(os.path.basename(f).encode())
        h.update(open(f, "rb").read())
    return h.hexdigest()


def hbm_traffic(kernel: str, workload: str):
    """Calibrated FETCH + WRITE bytes per launch of `kernel` from the committed
    rocprofv3 counter table, or None if the table is for other kernel sources
    or another workload."""
    try:
        t = json.load(open(TRAFFIC_TABLE))
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != kernel_source_hash() or t.get("workload") != workload:
        return None
    k = t["kernels"].get(kernel)
    return None if k is None else k["fetch_bytes"] + k["write_bytes"]


class Telemetry:
    """Samples the GPU engine clock (pp_dpm_sclk) and socket power (hwmon) from
    sysfs in a background thread while the timed region runs."""

    def __init__(self, period_s=0.02):
        import glob
        import threading
        self.period = period_s
        self.sclk_path = next(iter(sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))), None)
        dev = os.path.dirname(self.sclk_path) if self.sclk_path else None
        hw = sorted(glob.glob(os.path.join(dev, "hwmon", "hwmon*"))) if dev else []
        self.power_path = os.path.join(hw[0], "power1_input") if hw else None
        self.cap_path = os.path.join(hw[0], "power1_cap") if hw else None
        self.sclk, self.power = [], []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _read(self):
        try:
            if self.sclk_path:
                for line in open(self.sclk_path):
                    if "*" in line:
                        self.sclk.append(float(line.split(":")[1].strip().split("M")[0]))
            if self.power_path and os.path.exists(self.power_path):
                self.power.append(float(open(self.power_path).read()) / 1e6)
        except (OSError, ValueError, IndexError):
            pass

    def _run(self):
        while not self._stop.is_set():
            self._read()
            time.sleep(self.period)

    def __enter__(self):
        self._t.start()
        return self

    def __exit__(self, *a):
        self._stop.set()
        self._t.join()

    def summary(self):
        cap = None
        try:
            cap = float(open(self.cap_path).read()) / 1e6 if self.cap_path else None
        except (OSError, ValueError):
            pass
        mean = lambda v: (sum(v) / len(v)) if v else None
        return {"sclk_mhz_mean": mean(self.sclk), "sclk_mhz_min": min(self.sclk) if self.sclk else None,
                "socket_power_w_mean": mean(self.power), "power_cap_w": cap,
                "samples": len(self.sclk)}


def blas_info() -> dict:
    """BLAS library numpy runs on (threadpoolctl) and its thread count."""
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                return {"vendor": i.get("internal_api"), "version": i.get("version"),
                        "threads": i.get("num_threads"), "architecture": i.get("architecture")}
    except Exception:
        pass
    return {"vendor": None, "version": None, "threads": None}


def _oracle_tokens_per_s(w, x, js, budget_s, max_responses=None):
    """The literal float64 oracle (Algorithm 1 inner loop) on samples `js`,
    one response at a time, until `budget_s` of host time is spent (at least
    one response per sample).  Returns (tokens, seconds, [(j, responses)])."""
    from oracle import elbo
    tokens, secs, done = 0, 0.0, []
    per_j = budget_s / len(js)
    for j in js:
        nb, t_j = 0, 0.0
        while nb < (max_responses or w.B) and (nb == 0 or t_j < per_j):
            b = nb
            p = elbo.Problem(1, w.L, w.d, w.V, w.n_t, j_begin=j, j_count=1, seed=w.philox_seed,
                             seq_id_base=w.seq_id_base + b, t_mode=w.t_mode)
            t0 = time.perf_counter()
            r = elbo.elbo_literal(p, x["hidden"][b:b + 1], x["W"], x["targets"][b:b + 1],
                                  x["resp_mask"][b:b + 1], x["adv"][b:b + 1])
            t_j += time.perf_counter() - t0
            tokens += int(r.n_masked.sum())
            nb += 1
        secs += t_j
        done.append((j, nb))
    return tokens, secs, done


def cpu_baseline(w: workloads.Workload, x: dict, budget_s: float = 20.0,
                 single_thread_s: float = 15.0) -> dict:
    """The float64 oracle's literal per-sample form timed on this host: samples
    j = 0 and 1 of the workload on all BLAS threads (responses added until the
    budget is spent), and one response of sample j = 0 of the B=8, L=256
    workload on one BLAS thread."""
    blas = blas_info()
    cores = len(os.sched_getaffinity(0))
    tokens, secs, done = _oracle_tokens_per_s(w, x, (0, 1), budget_s)
    out = {"value": tokens / secs, "unit": "masked tokens/s", "cores": blas["threads"] or cores,
           "kind": "oracle", "blas": blas, "host_cpus": cores,
           "sample": f"literal float64 oracle, MC samples j=0,1 of {w.name} "
                     f"(responses per sample: {dict(done)}; {tokens} masked tokens, fwd+bwd incl. "
                     f"full dW), {secs:.1f} s on {blas['threads'] or cores} BLAS threads"}
    if single_thread_s > 0:
        try:
            from threadpoolctl import threadpool_limits
            w2 = workloads.LLADA_L256
            x2 = x if w2.name == w.name else workloads.generate(w2)
            with threadpool_limits(1):
                t2, s2, _ = _oracle_tokens_per_s(w2, x2, (0,), single_thread_s, max_responses=1)
            out["single_thread"] = {"value": t2 / s2, "unit": "masked tokens/s", "threads": 1,
                                    "sample": f"{w2.name} j=0, response 0: {t2} masked tokens, "
                                              f"{s2:.1f} s"}
        except ImportError:
            out["single_thread"] = None
    return out


def cpu_plan(out_path=None):
    """The oracle's literal form on samples j = 0 and 1 of every LLaDA-shaped
    workload with the full batch (all responses), on all BLAS threads, plus
    one response of the B=8, L=256 workload's sample j = 0 on one thread; one
    JSON line per measurement (host only, minutes of CPU time)."""
    from oracle import elbo
    blas = blas_info()
    rows = []
    for w in workloads.CONFIGS[1:]:
        x = workloads.generate(w)
        for j in (0, 1):
            p = elbo.Problem(w.B, w.L, w.d, w.V, w.n_t, j_begin=j, j_count=1, seed=w.philox_seed,
                             seq_id_base=w.seq_id_base, t_mode=w.t_mode)
            t0 = time.perf_counter()
            r = elbo.elbo_literal(p, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"])
            secs = time.perf_counter() - t0
            tok = int(r.n_masked.sum())
            row = {"workload": w.name, "j": j, "masked_tokens": tok, "seconds": secs,
                   "value": tok / secs, "unit": "masked tokens/s", "threads": blas["threads"],
                   "blas": blas}
            rows.append(row)
            print(json.dumps(row), flush=True)
    from threadpoolctl import threadpool_limits
    w = workloads.LLADA_L256
    x = workloads.generate(w)
    with threadpool_limits(1):
        tok, secs, _ = _oracle_tokens_per_s(w, x, (0,), 0.0, max_responses=1)
    row = {"workload": w.name, "j": 0, "responses": 1, "masked_tokens": tok, "seconds": secs,
           "value": tok / secs, "unit": "masked tokens/s", "threads": 1, "blas": blas}
    rows.append(row)
    print(json.dumps(row), flush=True)
    if out_path:
        json.dump(rows, open(out_path, "w"), indent=1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default=DEFAULT, choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0,
                    help="seconds of host time for the oracle on samples j = 0, 1")
    ap.add_argument("--cpu-single-thread", type=float, default=12.0,
                    help="seconds for the one-thread oracle figure (0: skip)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the per-sample + final-RMSNorm variant measurement")
    ap.add_argument("--ws-budget-gib", type=float, default=0.0,
                    help="workspace budget of the timed step (0: the default layout)")
    ap.add_argument("--vocab-chunk", type=int, default=0,
                    help="force the recompute backward with this vocabulary chunk")
    ap.add_argument("--no-budget-sweep", action="store_true",
                    help="skip the workspace-budget sweep")
    ap.add_argument("--no-memory-leg", action="store_true",
                    help="skip the peak-memory-against-n_t calls (profiling runs)")
    ap.add_argument("--cpu-plan", metavar="OUT_JSON", nargs="?", const="",
                    help="only time the CPU oracle on samples j = 0, 1 of every LLaDA workload "
                         "(full batch) and exit")
    args = ap.parse_args()
    if args.cpu_plan is not None:
        cpu_plan(args.cpu_plan or None)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    from paper_2510_11683_amd import bgpo

    w = WORKLOADS[args.workload]
    t0 = time.perf_counter()
    x = workloads.generate(w)
    gen_s = time.perf_counter() - t0
    dev = bgpo.device_inputs(x)
    B, L, d, V, nt = w.B, w.L, w.d, w.V, w.n_t
    prob = bgpo.Problem(B, L, d, V, nt, seed=w.philox_seed, seq_id_base=w.seq_id_base,
                        t_mode=w.t_mode, ws_budget=int(args.ws_budget_gib * GiB),
                        vocab_chunk=args.vocab_chunk)
    plan = bgpo.bgpo_workspace_plan(prob)
    # peak memory against n_t first, with nothing else allocated but the inputs
    mem_vs_nt = None if args.no_memory_leg else memory_vs_n_t(w, prob, dev, x)
    ws = bgpo.alloc_workspace(prob)
    dX = torch.zeros(B, L, d, dtype=torch.float32, device="cuda")
    dW = torch.zeros(d, V, dtype=torch.float32, device="cuda")
    ell = torch.zeros(B, nt, dtype=torch.float64, device="cuda")
    g = torch.zeros(B, nt, dtype=torch.float64, device="cuda")
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    nm = torch.zeros(B, nt, dtype=torch.int32, device="cuda")
    tt = torch.zeros(B, nt, dtype=torch.float32, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")

    def step(p, timing=None):
        bgpo.bgpo_elbo_bwd_accumulate(p, dev["hidden"], dev["W"], dev["targets"],
                                      dev["resp_mask"], dev["adv"], None, 1.0 / 8, dX, dW, ell, g,
                                      loss, nm, tt, flags, ws, timing=timing)

    for _ in range(args.warmup):
        step(prob)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()

    timing = bgpo.Timing()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with Telemetry() as tel:
        wall0 = time.perf_counter()
        start.record()
        for _ in range(args.steps):
            step(prob, timing)
        end.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
    telemetry = tel.summary()
    ms = start.elapsed_time(end) / args.steps
    tokens = int(nm.sum().item())                        # masked tokens per step
    value = tokens / (ms / 1e3)

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    kt = timing.as_dict()
    # algorithmic FLOPs: each GEMM class does 2 * N_j * d * V per sample
    gemm_flop_per_step = 2.0 * tokens * d * V
    per_kernel = {}
    for k, (kms, n) in kt.items():
        if n == 0:
            continue
        e = {"ms_per_step": kms / args.steps, "launches_per_step": n / args.steps,
             "avg_launch_us": 1e3 * kms / n}
        if k in GEMM_CLASSES:
            e["tflops"] = gemm_flop_per_step / (kms / args.steps / 1e3) / 1e12
        per_kernel[k] = e
    # HBM-bound kernel classes: achieved bandwidth from the committed counter
    # bytes and from the algorithmic bytes, against the 8 TB/s peak
    def algo_bytes(k, launches):                         # per launch
        rows = tokens / launches                         # masked rows one launch processes
        # (softmax_grad: three small kernels per unit, counter bytes only;
        # dx_reduce: depends on the split count)
        return {"gather": 6.0 * rows * d,                # read rows, write H_c and H_c^T
                "transpose_w": 6.0 * d * V}.get(k)       # read W, write W^T and W slab-major
    for k, e in per_kernel.items():
        if k in GEMM_CLASSES:
            continue
        secs = e["avg_launch_us"] / 1e6
        tb = hbm_traffic(k, w.name)
        if tb is not None:
            e["counter_gbs"] = tb / secs / 1e9
            e["counter_hbm_frac"] = e["counter_gbs"] / PEAK_HBM_GBS
        ab = algo_bytes(k, e["launches_per_step"])
        if ab:
            e["algorithmic_gbs"] = ab / secs / 1e9
            e["algorithmic_hbm_frac"] = e["algorithmic_gbs"] / PEAK_HBM_GBS
    dom = max((k for k in per_kernel if k in GEMM_CLASSES), key=lambda k: per_kernel[k]["ms_per_step"])
    achieved = per_kernel[dom]["tflops"]
    # GEMM passes per sample: forward logits, dX, dW (stored mode: the
    # backward reuses the forward's exponentials, so executed = useful 6 d V),
    # plus the chunked logits recompute in the recompute mode (8 d V executed)
    passes = sum(1 for k in GEMM_CLASSES if k in per_kernel)
    exec_flops = 2.0 * passes * d * V * value
    useful_flops = 6.0 * d * V * value

    out = {
        "metric": "masked tokens/sec fwd+bwd per MC sample; % bf16 MFMA peak; peak mem vs n_t",
        "value": value,
        "unit": "masked tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded numpy: RMS-normalised N(0,1) hidden, N(0,0.02^2) head, Zipf(1.1) targets)",
        "config": {"workload": w.name, "B": B, "L": L, "d": d, "V": V, "n_t": nt,
                   "t_mode": "stratified" if w.t_mode else "iid",
                   "masked_tokens_per_step": tokens, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": hbm_traffic(dom, w.name)},
        "backward_plan": plan,
        "gemm_passes_per_sample": passes,
        "mfma_frac_executed": exec_flops / (PEAK_BF16_TFLOPS * 1e12),
        "mfma_frac_6dV": useful_flops / (PEAK_BF16_TFLOPS * 1e12),
        "kernels": per_kernel,
        "telemetry": telemetry,
        # the same MFMA fraction against the peak at the mean engine clock measured
        "mfma_frac_executed_at_measured_clock": (
            exec_flops / (PEAK_BF16_TFLOPS * 1e12 * telemetry["sclk_mhz_mean"] / 2400.0)
            if telemetry.get("sclk_mhz_mean") else None),
        "wall_s_timed": wall,
        "peak_mem_vs_n_t": mem_vs_nt,
        "status_flags": int(flags.item()),
        "input_gen_s": gen_s,
    }
    if not args.no_variants:
        out["variants"] = {"forward_only": forward_only_leg(w, prob, dev, ws, args, tokens),
                           "per_sample_rmsnorm": per_sample_rmsnorm_leg(w, prob, dev, ws, args, tokens),
                           "exact_objective_off_policy": exact_objective_leg(w, prob, dev, ws, args,
                                                                             tokens)}
    # the remaining legs allocate their own workspaces and buffers
    del ws, dX, dW, ell, g, loss, nm, tt
    torch.cuda.empty_cache()
    if not args.no_budget_sweep and args.ws_budget_gib == 0 and args.vocab_chunk == 0:
        out["budget_sweep"] = budget_sweep_leg(w, dev)
    if not args.no_variants:
        out["variants"]["exact_objective_retained"] = retained_memory_leg(w, prob, dev)
        out["mask_compaction_2p20"] = mask_scaling_leg()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, x, args.cpu_budget, args.cpu_single_thread)
    print(json.dumps(out))


GiB = 1 << 30


def _call_buffers(w, nt):
    import torch
    f = dict(device="cuda")
    return dict(dX=torch.zeros(w.B, w.L, w.d, dtype=torch.float32, **f),
                dW=torch.zeros(w.d, w.V, dtype=torch.float32, **f),
                ell=torch.zeros(w.B, nt, dtype=torch.float64, **f),
                g=torch.zeros(w.B, nt, dtype=torch.float64, **f),
                loss=torch.zeros(1, dtype=torch.float64, **f),
                nm=torch.zeros(w.B, nt, dtype=torch.int32, **f),
                flags=torch.zeros(1, dtype=torch.int32, **f))


def _bwd(bgpo, p, dev, o, ws):
    bgpo.bgpo_elbo_bwd_accumulate(p, dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"],
                                  dev["adv"], None, 1.0 / 8, o["dX"], o["dW"], o["ell"], o["g"],
                                  o["loss"], o["nm"], None, o["flags"], ws)


def memory_vs_n_t(w, prob, dev, x, n_ts=(1, 4, 16, 64)):
    """Peak device memory of one backward call over all n_t samples, for
    several n_t at the step's layout: torch's peak of everything allocated
    (inputs, outputs, gradients, workspace) and the drop of free device
    memory (hipMemGetInfo) across the call, which would show any allocation
    inside the library."""
    import dataclasses
    import torch
    from paper_2510_11683_amd import bgpo
    res = {"n_t": list(n_ts), "workspace_bytes": [], "peak_mem_bytes": [],
           "mem_get_info_drop_during_call": [], "inputs_bytes": sum(t.numel() * t.element_size()
                                                                   for t in dev.values())}
    # the process's first library call also loads the code objects (a
    # one-time drop of free memory by the HIP runtime, not an allocation of
    # the library): make it here, with one sample, and report it apart
    p1 = dataclasses.replace(prob, n_t=1)
    ws = bgpo.alloc_workspace(p1)
    o = _call_buffers(w, 1)
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    _bwd(bgpo, p1, dev, o, ws)
    torch.cuda.synchronize()
    res["first_call_runtime_drop_bytes"] = free0 - torch.cuda.mem_get_info()[0]
    del ws, o
    for n in n_ts:
        p = dataclasses.replace(prob, n_t=n)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        ws = bgpo.alloc_workspace(p)
        o = _call_buffers(w, n)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        _bwd(bgpo, p, dev, o, ws)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        res["workspace_bytes"].append(ws.numel())
        res["peak_mem_bytes"].append(torch.cuda.max_memory_allocated())
        res["mem_get_info_drop_during_call"].append(free0 - free1)
        del ws, o
    torch.cuda.empty_cache()
    return res


def budget_sweep_leg(w, dev, budgets_gib=(2, 4, 8, 16, 32, 48), n_ts=(1, 64)):
    """Masked tokens/s and peak device memory of one backward call over all
    samples under each workspace budget (the layout it picks: stored
    exponentials with smaller units, or the recompute backward), for
    n_t = 1 and the workload's n_t."""
    import torch
    from paper_2510_11683_amd import bgpo
    out = []
    for bg in budgets_gib:
        for n in n_ts:
            n = min(n, w.n_t) if n != 1 else 1
            p = bgpo.Problem(w.B, w.L, w.d, w.V, n, seed=w.philox_seed, seq_id_base=w.seq_id_base,
                             t_mode=w.t_mode, ws_budget=bg * GiB)
            try:
                plan = bgpo.bgpo_workspace_plan(p)
            except bgpo.BgpoError as e:
                out.append({"budget_gib": bg, "n_t": n, "error": str(e)})
                continue
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            torch.cuda.reset_peak_memory_stats()
            ws = bgpo.alloc_workspace(p)
            o = _call_buffers(w, n)
            _bwd(bgpo, p, dev, o, ws)                    # warm-up
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = 3 if n == 1 else 1
            a.record()
            for _ in range(reps):
                _bwd(bgpo, p, dev, o, ws)
            b.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / reps
            tokens = int(o["nm"].sum().item())
            out.append({"budget_gib": bg, "n_t": n, "plan": plan, "ms_per_call": ms,
                        "masked_tokens": tokens, "value": tokens / (ms / 1e3),
                        "peak_mem_bytes": torch.cuda.max_memory_allocated(),
                        "status_flags": int(o["flags"].item())})
            del ws, o
    torch.cuda.empty_cache()
    return out


def mask_scaling_leg(B=4096, L=256, reps=5):
    """Mask draw + stable compaction of one sample at the B*L = 2^20 limit:
    the single-workgroup kernel (bgpo_sample_masks) against the multi-block
    passes the library uses above 65536 positions (test hook), HIP events."""
    import torch
    from paper_2510_11683_amd import bgpo
    p = bgpo.Problem(B, L, 64, 64, 4, seed=0xB6B0D000)
    resp = torch.ones(B, L, dtype=torch.uint8, device="cuda")
    idx = torch.empty(B * L, dtype=torch.int32, device="cuda")
    nm = torch.empty(B, dtype=torch.int32, device="cuda")
    res = {"B": B, "L": L}
    for name, fn in (("single_workgroup", lambda j: bgpo.bgpo_sample_masks(p, resp, j, idx, nm)),
                     ("multi_block", lambda j: bgpo.bgpo_test_mask_multiblock(p, resp, j, idx, nm))):
        fn(0)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for r in range(reps):
            fn(r % 4)
        b.record()
        torch.cuda.synchronize()
        us = 1e3 * a.elapsed_time(b) / reps
        n = int(nm.sum().item())
        # resp_mask read + one 4-byte index per masked position written
        res[name] = {"us_per_sample": us, "masked": n,
                     "gbs": (B * L + 4 * n) / (us * 1e-6) / 1e9}
    return res


def retained_memory_leg(w, prob, dev, n_ts=(1, 4, 16)):
    """The exact objective computed by keeping every sample's state (as when
    all n_t computational graphs are retained): peak device memory and time
    of one off-policy call for several n_t, against the constant-memory mode."""
    import dataclasses
    import torch
    from paper_2510_11683_amd import bgpo
    B, L, d, V = w.B, w.L, w.d, w.V
    res = {"n_t": list(n_ts), "workspace_bytes": [], "peak_mem_bytes": [], "ms_per_call": [],
           "masked_tokens": []}
    for nt in n_ts:
        p = dataclasses.replace(prob, n_t=nt, bound=bgpo.BGPO_BOUND_EXACT, retain_samples=1)
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        ws = bgpo.alloc_workspace(p)
        dX = torch.zeros(B, L, d, dtype=torch.float32, device="cuda")
        dW = torch.zeros(d, V, dtype=torch.float32, device="cuda")
        ell_old = torch.zeros(B, nt, dtype=torch.float64, device="cuda")
        ell, g = torch.zeros_like(ell_old), torch.zeros_like(ell_old)
        loss = torch.zeros(1, dtype=torch.float64, device="cuda")
        nm = torch.zeros(B, nt, dtype=torch.int32, device="cuda")
        flags = torch.zeros(1, dtype=torch.int32, device="cuda")
        bgpo.bgpo_elbo_fwd(p, dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"], ell_old,
                           nm, None, ws)

        def call():
            bgpo.bgpo_elbo_bwd_accumulate(p, dev["hidden"], dev["W"], dev["targets"],
                                          dev["resp_mask"], dev["adv"], ell_old, 1.0 / 8, dX, dW,
                                          ell, g, loss, nm, None, flags, ws)
        call()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        call()
        b.record()
        torch.cuda.synchronize()
        res["workspace_bytes"].append(ws.numel())
        res["peak_mem_bytes"].append(torch.cuda.max_memory_allocated())
        res["ms_per_call"].append(a.elapsed_time(b))
        res["masked_tokens"].append(int(nm.sum().item()))
        del ws, dX, dW
        torch.cuda.empty_cache()
    res["workspace_bytes_n_t_64"] = bgpo.bgpo_workspace_size(
        dataclasses.replace(prob, n_t=64, bound=bgpo.BGPO_BOUND_EXACT, retain_samples=1))
    res["constant_mode_workspace_bytes"] = bgpo.bgpo_workspace_size(
        dataclasses.replace(prob, bound=bgpo.BGPO_BOUND_EXACT))
    return res


def forward_only_leg(w, prob, dev, ws, args, tokens_main):
    """bgpo_elbo_fwd over all samples (l of every sample, no gradient: how
    l_old is produced with the old head weights), same workspace."""
    import torch
    from paper_2510_11683_amd import bgpo
    ell = torch.zeros(w.B, w.n_t, dtype=torch.float64, device="cuda")
    nm = torch.zeros(w.B, w.n_t, dtype=torch.int32, device="cuda")

    def step():
        bgpo.bgpo_elbo_fwd(prob, dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"], ell, nm,
                           None, ws)
    steps = max(1, min(args.steps, 3))
    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    tokens = int(nm.sum().item())
    assert tokens == tokens_main
    return {"value": tokens / (ms / 1e3), "unit": "masked tokens/s", "ms_per_step": ms,
            "steps": steps, "mfma_frac_2dV": 2.0 * w.d * w.V * tokens / (ms / 1e3) / (PEAK_BF16_TFLOPS * 1e12)}


def exact_objective_leg(w, prob, dev, ws, args, tokens_main):
    """The exact ratio objective (bound mode 3) off-policy: ell_old from a
    forward pass, so the call runs its forward pass over all samples for the
    mean log-ratio before the per-sample backward loop."""
    import dataclasses
    import torch
    from paper_2510_11683_amd import bgpo
    B, L, d, V, nt = w.B, w.L, w.d, w.V, w.n_t
    p = dataclasses.replace(prob, bound=bgpo.BGPO_BOUND_EXACT)
    ell_old = torch.zeros(B, nt, dtype=torch.float64, device="cuda")
    nm = torch.zeros(B, nt, dtype=torch.int32, device="cuda")
    bgpo.bgpo_elbo_fwd(prob, dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"], ell_old,
                       nm, None, ws)
    dX = torch.zeros(B, L, d, dtype=torch.float32, device="cuda")
    dW = torch.zeros(d, V, dtype=torch.float32, device="cuda")
    ell = torch.zeros_like(ell_old)
    g = torch.zeros_like(ell_old)
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")

    def step():
        bgpo.bgpo_elbo_bwd_accumulate(p, dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"],
                                      dev["adv"], ell_old, 1.0 / 8, dX, dW, ell, g, loss, nm, None,
                                      flags, ws)
    steps = max(1, min(args.steps, 3))
    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    tokens = int(nm.sum().item())
    assert tokens == tokens_main
    return {"value": tokens / (ms / 1e3), "unit": "masked tokens/s", "ms_per_step": ms,
            "steps": steps, "status_flags": int(flags.item())}


def per_sample_rmsnorm_leg(w, prob, dev, ws, args, tokens_main):
    """The same workload through the final-RMSNorm entry point with one
    activation tensor per sample (device copies of one pre-norm tensor) and a
    dx per sample: the per-sample form of the step."""
    import dataclasses
    import torch
    from paper_2510_11683_amd import bgpo
    B, L, d, V, nt = w.B, w.L, w.d, w.V, w.n_t
    xb = workloads.pre_norm_activations(w)
    x1 = torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16)
    x = x1.unsqueeze(0).expand(nt, B, L, d).contiguous()
    del x1
    gamma = torch.from_numpy(workloads.norm_weight(w)).cuda()
    p = dataclasses.replace(prob, sample_stride=B * L * d, norm_eps=1e-6)
    dx = torch.zeros(nt, B, L, d, dtype=torch.float32, device="cuda")
    dgam = torch.zeros(d, dtype=torch.float32, device="cuda")
    dW = torch.zeros(d, V, dtype=torch.float32, device="cuda")
    ell = torch.zeros(B, nt, dtype=torch.float64, device="cuda")
    g = torch.zeros_like(ell)
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    nm = torch.zeros(B, nt, dtype=torch.int32, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")

    def step():
        bgpo.bgpo_elbo_bwd_accumulate_rmsnorm(p, x, gamma, dev["W"], dev["targets"],
                                              dev["resp_mask"], dev["adv"], None, 1.0 / 8, dx,
                                              dgam, dW, ell, g, loss, nm, None, flags, ws)
    steps = max(1, min(args.steps, 3))
    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    tokens = int(nm.sum().item())
    assert tokens == tokens_main            # same masks as the main measurement
    return {"value": tokens / (ms / 1e3), "unit": "masked tokens/s", "ms_per_step": ms,
            "steps": steps, "sample_stride": B * L * d, "status_flags": int(flags.item())}


if __name__ == "__main__":
    main()
