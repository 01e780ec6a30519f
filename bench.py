#!/usr/bin/env python3
"""Benchmark: memory-efficient attention forward + backward on one MI355X.

Headline workload: self-attention, batch 1, 16 heads, n_q = n_k = 16384, d = 64,
bf16 inputs with float32 accumulation, Q/K/V/dO i.i.d. N(0, 1) from fixed seeds
(synthetic; the paper also measures on standard-normal inputs, Section 5.1).

One step = the whole hot path over that batch, as a training step issues it:
the forward call (lazy-softmax tile kernel, writing o, lse and o's rounding
residual) and one backward call (D preprocess, dK/dV kernel, dQ kernel).
Per-kernel figures come from a second timed loop that issues the backward as
two calls -- dK/dV, then dQ -- so that HIP events on the launch stream time
each kernel (the small D preprocess runs in each of the two calls there).

Credited work (algorithmic, unmasked (query, key) pairs P = B*H*n_q*n_k, or
B*H*n(n+1)/2 causal): forward 4*d*P flop (Q K^T and P V), backward 10*d*P flop
(the recomputed Q K^T, dO V^T, P^T dO, dS K, dS^T Q).  value = 14*d*P / mean
step time over the K timed steps (enqueued back to back, no host gaps);
per-kernel figures are medians over the same steps.

Also measured (objects on the same JSON line): the causal 4x32x8192 d = 128
workload (forward + backward), the long-key forward (n_q = 16384, n_k = 2^20),
decode-shaped attention (HBM-bound), key padding, the shader clock and board
power sampled with amd-smi while steps run, and the float64 oracle on the
host's cores (all threads and one thread).

Prints ONE JSON line on stdout.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import subprocess
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 flop/clk (dense, no sparsity)
PEAK_HBM_GBS = 8000.0
METRIC = "attention fwd+bwd TFLOP/s and % bf16 MFMA peak at n=16384,d=64; peak workspace"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
HEADLINE = "selfattn_bf16_b1h16_n16384_d64"
CAUSAL_D128 = "causal_bf16_b4h32_n8192_d128"
LONGKV = "longkv_bf16_b1h1_nq16384_nk1048576_d64"
DECODE_WORKLOAD = "decode_bf16_b8h16_nq1_nk65536_d64"


def csrc_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2112_05682_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str = HEADLINE):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("csrc_digest") != csrc_digest():
        return None
    ent = data.get("workloads", {}).get(workload, {}).get(kernel)
    if not ent:
        return None
    return ent.get("hbm_bytes_per_launch")


def pairs_of(w) -> int:
    per = w.n_q * w.n_k if not w.causal else w.n_q * (w.n_q + 1) // 2
    return w.batch * w.heads * per


def med(xs):
    return statistics.median(xs) if xs else None


class ClockSampler:
    """Samples the shader clock of every XCD and the socket power with
    `amd-smi metric -c -p` in a background thread while work runs."""

    def __init__(self):
        self.samples = []
        self._stop = threading.Event()
        self._t = None
        self.error = None

    def _one(self):
        r = subprocess.run(["amd-smi", "metric", "-g", "0", "-c", "-p", "--json"],
                           capture_output=True, text=True, timeout=20)
        data = json.loads(r.stdout)
        g = data["gpu_data"][0] if isinstance(data, dict) else data[0]
        clocks = [v["clk"]["value"] for k, v in g["clock"].items()
                  if k.startswith("gfx_") and isinstance(v, dict) and isinstance(v.get("clk"), dict)
                  and isinstance(v["clk"].get("value"), (int, float))]
        power = g.get("power", {}).get("socket_power", {}).get("value")
        return clocks, power

    def _run(self):
        while not self._stop.is_set():
            try:
                self.samples.append(self._one())
            except Exception as e:  # tool missing or output changed: report, do not fail the bench
                self.error = repr(e)[:200]
                return

    def __enter__(self):
        self._t = threading.Thread(target=self._run, daemon=True)
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join(timeout=30)

    def summary(self):
        cl = [statistics.mean(c) for c, _ in self.samples if c]
        pw = [p for _, p in self.samples if isinstance(p, (int, float))]
        if not cl:
            return {"tool": "amd-smi metric -c -p", "samples": 0, "error": self.error}
        return {"tool": "amd-smi metric -c -p", "samples": len(cl),
                "gfx_mhz_median": round(med(cl), 1), "gfx_mhz_min": round(min(cl), 1),
                "gfx_mhz_max": round(max(cl), 1),
                "socket_power_w_median": round(med(pw), 1) if pw else None,
                "note": "mean over the 8 XCDs per sample; peak figures assume 2400 MHz"}


def time_steps(step, n_events: int, steps: int):
    """Runs `steps` steps enqueued back to back, each recording n_events events
    on the current stream; returns (total ms, [[segment ms] per step])."""
    import torch

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_events)] for _ in range(steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s_ in range(steps):
        step(evs[s_])
    stop.record()
    torch.cuda.synchronize()
    total = start.elapsed_time(stop)
    segs = [[e[i].elapsed_time(e[i + 1]) for i in range(n_events - 1)] for e in evs]
    return total, segs


def fwd_bwd_step(w, x):
    """The step of a workload: forward (with residual), then one backward call
    (preprocess, dK/dV, dQ), with three events around them."""
    from paper_2112_05682_amd import attention_bwd, attention_fwd

    q, k, v, do = x["q"], x["k"], x["v"], x["do"]

    def step(ev):
        ev[0].record()
        o, lse, o_lo = attention_fwd(q, k, v, causal=w.causal, residual=True)
        ev[1].record()
        attention_bwd(q, k, v, o, lse, do, causal=w.causal, o_lo=o_lo)
        ev[2].record()

    return step


def split_step(w, x):
    """The same work with the backward split into a dK/dV call and a dQ call,
    four events: the per-kernel times."""
    from paper_2112_05682_amd import attention_bwd, attention_fwd

    q, k, v, do = x["q"], x["k"], x["v"], x["do"]

    def step(ev):
        ev[0].record()
        o, lse, o_lo = attention_fwd(q, k, v, causal=w.causal, residual=True)
        ev[1].record()
        attention_bwd(q, k, v, o, lse, do, causal=w.causal, need_dq=False, o_lo=o_lo)
        ev[2].record()
        attention_bwd(q, k, v, o, lse, do, causal=w.causal, need_dkdv=False, o_lo=o_lo)
        ev[3].record()

    return step


def timed_workload(w, x, steps: int, warmup: int):
    """Warm-up, then `steps` whole steps (value) and `steps` split steps
    (per-kernel medians); returns (total ms of the whole steps, their segment
    times [fwd, bwd], the split steps' segment times [fwd, dK/dV, dQ])."""
    import torch

    step, split = fwd_bwd_step(w, x), split_step(w, x)
    for _ in range(warmup):
        step([torch.cuda.Event(enable_timing=True) for _ in range(3)])
        split([torch.cuda.Event(enable_timing=True) for _ in range(4)])
    total, segs = time_steps(step, 3, steps)
    _, ksegs = time_steps(split, 4, steps)
    return total, segs, ksegs


def kernel_table(w, segs, whole):
    """Per-kernel medians (over steps) of the three timed segments of the
    split steps, with credited flop and the fraction of the bf16 peak; the
    forward, backward and step summaries from the whole steps' [fwd, bwd]
    segments."""
    P = pairs_of(w)
    f = {"fwd": 4.0 * w.d * P, "bwd_dkdv": 8.0 * w.d * P, "bwd_dq": 2.0 * w.d * P}
    names = ("fwd", "bwd_dkdv", "bwd_dq")
    out = {}
    for i, n_ in enumerate(names):
        xs = [s[i] for s in segs]
        m = med(xs)
        out[n_] = {"median_ms": round(m, 4), "mean_ms": round(statistics.mean(xs), 4),
                   "algorithmic_flop": f[n_], "tflops": round(f[n_] / m / 1e9, 2),
                   "frac_of_peak": round(f[n_] / m / 1e9 / PEAK_BF16_TFLOPS, 4)}
    out["bwd_dkdv"]["includes"] = "D preprocess"
    out["bwd_dq"]["includes"] = "D preprocess; executes 6*d*P, credited 2*d*P"
    fwd_ms = med([s[0] for s in whole])
    bwd_ms = med([s[1] for s in whole])
    summary = {"fwd_median_ms": round(fwd_ms, 4), "bwd_median_ms": round(bwd_ms, 4),
               "fwd_tflops": round(4.0 * w.d * P / fwd_ms / 1e9, 2),
               "bwd_tflops": round(10.0 * w.d * P / bwd_ms / 1e9, 2),
               "step_tflops_median": round(14.0 * w.d * P / med([sum(s) for s in whole]) / 1e9, 2)}
    summary["fwd_frac_of_peak"] = round(summary["fwd_tflops"] / PEAK_BF16_TFLOPS, 4)
    summary["bwd_frac_of_peak"] = round(summary["bwd_tflops"] / PEAK_BF16_TFLOPS, 4)
    summary["step_frac_of_peak_median"] = round(summary["step_tflops_median"] / PEAK_BF16_TFLOPS, 4)
    return out, summary


def kernel_names(w):
    two_group = w.d == 64
    return {"fwd": "attn_fwd_pp_kernel" if two_group else "attn_fwd_kernel",
            "bwd_dkdv": "attn_bwd_dkdv_pp_kernel" if two_group else "attn_bwd_dkdv_kernel",
            "bwd_dq": "attn_bwd_dq_pp_kernel" if two_group else "attn_bwd_dq_kernel"}


def roofline_of(w, kernels):
    dom = max(("fwd", "bwd_dkdv"), key=lambda n_: kernels[n_]["median_ms"])
    name = kernel_names(w)[dom]
    a = kernels[dom]["tflops"]
    return {"kernel": name, "bound": "mfma", "achieved": a, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(a / PEAK_BF16_TFLOPS, 4), "traffic": load_traffic(name, w.name),
            "time": "median per launch over the timed steps (HIP events on the launch stream"
                    + ("; includes the D preprocess)" if dom == "bwd_dkdv" else ")")}


def bench_fwd_bwd_workload(name, dev, steps: int, warmup: int):
    """Forward + backward of another workload (the causal d = 128 one)."""
    import torch

    from paper_2112_05682_amd.inputs import WORKLOADS, workload_inputs

    w = WORKLOADS[name]
    x = {k_: t.to(dev) for k_, t in workload_inputs(w, with_grad=True).items()}
    total, segs, ksegs = timed_workload(w, x, steps, warmup)
    kernels, summary = kernel_table(w, ksegs, segs)
    P = pairs_of(w)
    del x
    return {"workload": w.name, "steps": steps, "pairs": P,
            "ms_per_step": round(total / steps, 4),
            "value": round(14.0 * w.d * P / (total / steps) / 1e9, 2), "unit": "TFLOP/s",
            "frac_of_bf16_peak": round(14.0 * w.d * P / (total / steps) / 1e9 / PEAK_BF16_TFLOPS, 4),
            **summary, "kernels": kernels, "roofline": roofline_of(w, kernels),
            "inputs": "N(0,%g^2) %s, causal=%s" % (w.std, w.dtype, w.causal)}


def bench_longkv(dev, calls: int, warmup: int):
    """Forward only, 1 head, 16384 queries against 2^20 keys, d = 64: the keys
    are split over workgroups and the per-split summaries combined (Section 4);
    the time includes the combine."""
    import torch

    from paper_2112_05682_amd import attention_fwd
    from paper_2112_05682_amd.inputs import WORKLOADS, workload_inputs

    w = WORKLOADS[LONGKV]
    x = {k_: t.to(dev) for k_, t in workload_inputs(w, with_grad=False).items()}

    def step(ev):
        ev[0].record()
        attention_fwd(x["q"], x["k"], x["v"], causal=w.causal)
        ev[1].record()

    for _ in range(warmup):
        step([torch.cuda.Event(enable_timing=True) for _ in range(2)])
    _, segs = time_steps(step, 2, calls)
    m = med([s[0] for s in segs])
    f = 4.0 * w.d * pairs_of(w)
    del x
    return {"workload": w.name, "calls": calls, "median_ms": round(m, 4),
            "algorithmic_flop": f, "tflops": round(f / m / 1e9, 2),
            "frac_of_bf16_peak": round(f / m / 1e9 / PEAK_BF16_TFLOPS, 4),
            "kernel": "attn_fwd_pp_kernel (key splits) + attn_combine_kernel",
            "includes": "combine of the key splits"}


def bench_decode(dev, calls: int = 100, warmup: int = 5):
    """Decode-shaped forward (one query per batch and head against n_k keys):
    HBM-bound, so its roofline is the 8 TB/s HBM peak.  Algorithmic bytes per
    call: K and V once (4 n_k d per (batch, head) for 16-bit inputs), Q and O
    (4 n_q d) and the lse (4 n_q); the time includes the combine of the key
    ranges.  HIP events on torch's current stream, the stream the kernels run on."""
    import torch

    from paper_2112_05682_amd import attention_fwd
    from paper_2112_05682_amd.inputs import WORKLOADS, workload_inputs

    w = WORKLOADS[DECODE_WORKLOAD]
    x = {k_: t.to(dev) for k_, t in workload_inputs(w, with_grad=False).items()}

    def step(ev):
        ev[0].record()
        attention_fwd(x["q"], x["k"], x["v"], causal=w.causal)
        ev[1].record()

    for _ in range(warmup):
        step([torch.cuda.Event(enable_timing=True) for _ in range(2)])
    _, segs = time_steps(step, 2, calls)
    ms = med([s[0] for s in segs])
    bh = w.batch * w.heads
    nbytes = bh * (4 * w.n_k * w.d + 4 * w.n_q * w.d + 4 * w.n_q)
    gbs = nbytes / (ms * 1e-3) / 1e9
    del x
    out = {"workload": w.name, "kernel": "attn_decode_kernel", "bound": "hbm", "calls": calls,
           "median_ms": round(ms, 4), "algorithmic_bytes": nbytes, "achieved": round(gbs, 1),
           "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
           "traffic": load_traffic("attn_decode_kernel", w.name), "includes": "combine of the key ranges"}
    ceiling = read_ceiling()
    if ceiling:
        out["read_ceiling"] = ceiling
        out["frac_of_read_ceiling"] = round(gbs / ceiling["GBps"], 4)
    return out


def read_ceiling():
    """Best streaming-read rate of a plain read kernel (tests/native/hbm_read:
    2 GiB read once with 16-byte loads, several launch shapes) in a child
    process: the practical HBM ceiling for a kernel that reads K and V once."""
    exe = os.path.join(ROOT, "tests", "native", "hbm_read")
    if not os.path.exists(exe):
        return None
    try:
        r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    except subprocess.TimeoutExpired:
        return None
    lines = [json.loads(l) for l in r.stdout.splitlines() if l.startswith("{")]
    if r.returncode != 0 or not lines or "best_shape" not in lines[-1]:
        return None
    best = lines[-1]
    return {"tool": "tests/native/hbm_read", "shape": best["best_shape"], "GBps": best["GBps"],
            "frac_of_8TBps": best["frac_of_8TBps"]}


def bench_key_padding(dev, calls: int = 10, warmup: int = 2):
    """Forward + backward on a key-padded batch: 4 sequences of 8192 keys of
    which 8192, 6144, 4096 and 2048 are valid (kv_len), 16 heads, d = 64,
    bf16, against the same call without padding.  Credited work counts the
    unmasked pairs only (14 d per pair), so equal TFLOP/s means the padded
    keys cost nothing."""
    import torch

    from paper_2112_05682_amd import attention_bwd, attention_fwd
    from paper_2112_05682_amd.inputs import attention_inputs

    B, H, n, d = 4, 16, 8192, 64
    lens = [8192, 6144, 4096, 2048]
    x = {k_: t.to(dev) for k_, t in attention_inputs(B, H, n, n, d, "bf16").items()}
    kl = torch.tensor(lens, dtype=torch.int32, device=dev)
    out = {}
    for name, kv_len, keys in (("padded", kl, sum(lens)), ("full", None, B * n)):
        def step(ev, kv_len=kv_len):
            ev[0].record()
            o, lse, o_lo = attention_fwd(x["q"], x["k"], x["v"], kv_len=kv_len, residual=True)
            attention_bwd(x["q"], x["k"], x["v"], o, lse, x["do"], kv_len=kv_len, o_lo=o_lo)
            ev[1].record()

        for _ in range(warmup):
            step([torch.cuda.Event(enable_timing=True) for _ in range(2)])
        _, segs = time_steps(step, 2, calls)
        ms = med([s[0] for s in segs])
        out[name] = {"median_ms": round(ms, 4), "tflops": round(14.0 * d * H * n * keys / (ms * 1e-3) / 1e12, 1)}
    del x
    return {"workload": "selfattn_bf16_b4h16_n8192_d64_kvlen", "kv_len": lens, "calls": calls,
            "includes": "forward + backward (dK/dV and dQ in one call)",
            "valid_key_fraction": sum(lens) / (B * n), **out,
            "time_ratio": round(out["padded"]["median_ms"] / out["full"]["median_ms"], 4)}


# ----------------------------------------------------------- CPU baseline
# The float64 oracle as it stands, timed on the host's cores: with all its
# OpenMP threads, and with one (oracle.set_num_threads).

ORACLE_SAMPLES = {
    # name: (batch, heads, n_q, n_k, d, dtype, causal, with backward, description)
    "headline_2heads": (1, 2, 16384, 16384, 64, "bf16", False, True,
                        "2 of the 16 heads of the benchmark workload (n_q = n_k = 16384, d = 64), "
                        "float64 forward + backward"),
    "headline_1head_n4096": (1, 1, 4096, 4096, 64, "bf16", False, True,
                             "1 head at n_q = n_k = 4096, d = 64 (the benchmark's per-pair work at a "
                             "quarter of its length), float64 forward + backward"),
    "fp32_n256_full": (1, 1, 256, 256, 64, "fp32", False, True,
                       "the fp32 1x1x256x256 d = 64 workload in full, forward + backward"),
    "bf16_h8_n4096_fwd_full": (1, 8, 4096, 4096, 64, "bf16", False, False,
                               "the bf16 1x8x4096x4096 d = 64 workload in full, forward"),
    "causal_d128_1slice": (1, 1, 8192, 8192, 128, "bf16", True, True,
                           "1 of the 128 (batch, head) slices of the causal 4x32x8192 d = 128 workload, "
                           "float64 forward + backward"),
}


def oracle_sample(name: str) -> dict:
    import oracle
    from paper_2112_05682_amd.inputs import attention_inputs

    B, H, nq, nk, d, dtype, causal, bwd, desc = ORACLE_SAMPLES[name]
    x = attention_inputs(B, H, nq, nk, d, dtype, std=0.5 if causal and d == 128 else 1.0, with_grad=bwd)
    arrs = {k_: t.double().numpy() for k_, t in x.items()}
    t0 = time.perf_counter()
    oracle.fwd(arrs["q"], arrs["k"], arrs["v"], scale=d ** -0.5, causal=causal)
    if bwd:
        oracle.bwd(arrs["q"], arrs["k"], arrs["v"], arrs["do"], scale=d ** -0.5, causal=causal)
    dt = time.perf_counter() - t0
    pairs = B * H * (nq * nk if not causal else nq * (nq + 1) // 2)
    flops = (14.0 if bwd else 4.0) * d * pairs
    return {"sample": desc, "seconds": round(dt, 3), "threads": oracle.num_threads(),
            "gflops": round(flops / dt / 1e9, 3), "credited_flop": flops}


def oracle_longkv_rows(n_rows: int = 512) -> dict:
    """The long-key workload's forward (1 head, n_q = 16384, n_k = 2^20,
    d = 64) on n_rows query rows spread evenly over all query positions
    (rows are independent in the forward)."""
    import numpy as np

    import oracle
    from paper_2112_05682_amd.inputs import WORKLOADS, workload_inputs

    w = WORKLOADS[LONGKV]
    x = workload_inputs(w, with_grad=False)
    q, k, v = (x[n][0, 0].double().numpy() for n in ("q", "k", "v"))
    rows = np.linspace(0, w.n_q - 1, n_rows).astype(np.int64)
    t0 = time.perf_counter()
    oracle.fwd_rows(q, k, v, rows, scale=w.d ** -0.5, causal=w.causal)
    dt = time.perf_counter() - t0
    flops = 4.0 * w.d * n_rows * w.n_k
    return {"sample": "%d of the %d query rows of the long-key workload (n_k = 2^20, d = 64), spread over all "
                      "positions, float64 forward" % (n_rows, w.n_q),
            "seconds": round(dt, 3), "threads": oracle.num_threads(), "gflops": round(flops / dt / 1e9, 3),
            "credited_flop": flops}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def cpu_baseline() -> dict:
    all_core = oracle_sample("headline_2heads")
    extra = {"fp32_n256_full": oracle_sample("fp32_n256_full"),
             "bf16_h8_n4096_fwd_full": oracle_sample("bf16_h8_n4096_fwd_full"),
             "causal_d128_1slice": oracle_sample("causal_d128_1slice"),
             "longkv_512rows": oracle_longkv_rows()}
    import oracle

    n_all = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        one = oracle_sample("headline_1head_n4096")
    finally:
        oracle.set_num_threads(n_all)
    return {
        "value": round(all_core["gflops"] / 1e3, 6),
        "unit": "TFLOP/s",
        "cores": all_core["threads"],
        "kind": "oracle",
        "sample": all_core["sample"] + " (%.1f s); credited 14*d*pairs flop / time" % all_core["seconds"],
        "seconds": all_core["seconds"],
        "host_cpu": cpu_model(),
        "host_threads": os.cpu_count(),
        "omp_num_threads_env": os.environ.get("OMP_NUM_THREADS"),
        "one_thread": one,
        "other_workloads": extra,
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="headline workload only (no causal d = 128, long-key, decode, key-padding lines)")
    ap.add_argument("--clock-seconds", type=float, default=4.0,
                    help="sustained steps while amd-smi samples the clock (0: skip)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device copy (HBM counter calibration)")
    ap.add_argument("--only", default=None,
                    choices=["causal_d128", "longkv", "decode", "key_padding"],
                    help="run just this one measurement and print its object (for profiler runs)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d, WORLD_SIZE %d requested)" % (args.gpus, world), file=sys.stderr)
        return 2

    import torch

    from paper_2112_05682_amd import _lib, attention_bwd, attention_fwd
    from paper_2112_05682_amd.inputs import WORKLOADS, workload_inputs

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    if args.only:
        dev = torch.device("cuda", 0)
        run = {"causal_d128": lambda: bench_fwd_bwd_workload(CAUSAL_D128, dev, args.steps, args.warmup),
               "longkv": lambda: bench_longkv(dev, args.steps, args.warmup),
               "decode": lambda: bench_decode(dev, args.steps, args.warmup),
               "key_padding": lambda: bench_key_padding(dev, args.steps, args.warmup)}[args.only]
        print(json.dumps({args.only: run()}), flush=True)
        return 0
    w = WORKLOADS[args.workload]
    dev = torch.device("cuda", 0)
    x = {k_: t.to(dev) for k_, t in workload_inputs(w, with_grad=True).items()}
    q, k, v, do = x["q"], x["k"], x["v"], x["do"]
    torch.cuda.synchronize()
    P = pairs_of(w)
    f_step = 14.0 * w.d * P
    step = fwd_bwd_step(w, x)

    # Peak memory in excess of inputs and outputs (the paper's "memory
    # overhead", Section 5.1) during one forward + backward with every output
    # kept alive, from torch's allocator.
    torch.cuda.reset_peak_memory_stats(dev)
    base_alloc = torch.cuda.memory_allocated(dev)
    o_, lse_, olo_ = attention_fwd(q, k, v, causal=w.causal, residual=True)
    grads_ = attention_bwd(q, k, v, o_, lse_, do, causal=w.causal, o_lo=olo_)
    torch.cuda.synchronize()
    peak_extra = torch.cuda.max_memory_allocated(dev) - base_alloc
    out_bytes = sum(t.numel() * t.element_size() for t in (o_, *grads_))  # o, dq, dk, dv
    del o_, lse_, olo_, grads_

    # The timed steps: enqueued back to back, events read after the final
    # synchronisation.
    total_ms, segs, ksegs = timed_workload(w, x, args.steps, args.warmup)
    ms_step = total_ms / args.steps
    kernels, summary = kernel_table(w, ksegs, segs)

    # Clock and power while the same steps run for a few seconds (not timed).
    clock = None
    if args.clock_seconds > 0:
        n_clk = max(1, int(args.clock_seconds * 1e3 / ms_step))
        with ClockSampler() as cs:
            time.sleep(0.3)
            for _ in range(n_clk):
                step([torch.cuda.Event(enable_timing=True) for _ in range(3)])
            torch.cuda.synchronize()
        clock = cs.summary()
        clock["during"] = "%d back-to-back steps of the headline workload (%.1f s)" % (
            n_clk, n_clk * ms_step / 1e3)
        # The same for each kernel alone (half the time each): the clock and
        # power the chip settles at under that kernel's instruction mix.
        o1, l1, lo1 = attention_fwd(q, k, v, causal=w.causal, residual=True)
        alone = {"fwd": lambda: attention_fwd(q, k, v, causal=w.causal),
                 "bwd_dkdv": lambda: attention_bwd(q, k, v, o1, l1, do, causal=w.causal, need_dq=False, o_lo=lo1),
                 "bwd_dq": lambda: attention_bwd(q, k, v, o1, l1, do, causal=w.causal, need_dkdv=False, o_lo=lo1)}
        clock["per_kernel"] = {}
        for name_, fn in alone.items():
            n_k_ = max(1, int(args.clock_seconds * 0.5e3 / kernels[name_]["median_ms"]))
            with ClockSampler() as cs:
                time.sleep(0.3)
                for _ in range(n_k_):
                    fn()
                torch.cuda.synchronize()
            ks_ = cs.summary()
            ks_["during"] = "%d back-to-back calls (%.1f s)" % (n_k_, n_k_ * kernels[name_]["median_ms"] / 1e3)
            clock["per_kernel"][name_] = ks_
        del o1, l1, lo1

    p = _lib.problem(w.batch, w.heads, w.n_q, w.n_k, w.d, _lib.MEA_BF16, w.causal, w.d ** -0.5)
    lib_ws = max(_lib.fwd_workspace_size(p), _lib.bwd_workspace_size(p))
    lse_bytes = w.batch * w.heads * w.n_q * 4
    res_bytes = w.batch * w.heads * w.n_q * w.d * 2
    n2_bytes = w.batch * w.heads * w.n_q * w.n_k * 4
    del x, q, k, v, do, step
    torch.cuda.empty_cache()

    extras = {}
    if not args.no_extras:
        extras["causal_d128"] = bench_fwd_bwd_workload(CAUSAL_D128, dev, steps=30, warmup=3)
        torch.cuda.empty_cache()
        extras["longkv"] = bench_longkv(dev, calls=30, warmup=3)
        torch.cuda.empty_cache()
        extras["decode"] = bench_decode(dev)
        torch.cuda.empty_cache()
        extras["key_padding"] = bench_key_padding(dev)
        torch.cuda.empty_cache()

    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    value = f_step / (ms_step * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "heads": w.heads, "n_q": w.n_q,
                   "n_k": w.n_k, "d": w.d, "causal": w.causal,
                   "inputs": "N(0,%g^2) %s%s" % (w.std, w.dtype,
                                                 ", q and k x%g" % w.qk_mult if w.qk_mult != 1.0 else ""),
                   "accumulation": "fp32"},
        "frac_of_bf16_peak": round(value / PEAK_BF16_TFLOPS, 4),
        **summary,
        "kernels": kernels,
        "workspace": {"library_bytes": lib_ws, "lse_bytes": lse_bytes, "o_residual_bytes": res_bytes,
                      "peak_bytes": lib_ws + lse_bytes + res_bytes,
                      "measured_peak_above_inputs_outputs": max(0, peak_extra - out_bytes),
                      "n2_fp32_matrix_bytes": n2_bytes,
                      "reduction_vs_n2": round(n2_bytes / (lib_ws + lse_bytes + res_bytes), 1)},
        "roofline": roofline_of(w, kernels),
        "clock": clock,
        **extras,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
