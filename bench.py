#!/usr/bin/env python3
"""Benchmark: memory-efficient attention forward + backward on one MI355X.

Workload: self-attention, batch 1, 16 heads, n_q = n_k = 16384, d = 64, bf16
inputs with float32 accumulation, Q/K/V/dO i.i.d. N(0, 1) from fixed seeds
(synthetic; the paper also measures on standard-normal inputs).

One step = the whole hot path over that batch: the forward call (lazy-softmax
tile kernel) and the backward (D preprocess, dK/dV kernel, dQ kernel).  The
backward is issued as two library calls -- one computing dK and dV, one
computing dQ -- so that HIP events on the launch stream time each kernel; the
small D preprocess therefore runs twice per step (counted inside the timed
region, which only makes the step slower).

Credited work (algorithmic, unmasked (query, key) pairs P = B*H*n_q*n_k):
forward 4*d*P flop (Q K^T and P V), backward 10*d*P flop (the recomputed
Q K^T, dO V^T, P^T dO, dS K, dS^T Q).  value = 14*d*P / step time.

Prints ONE JSON line on stdout.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 flop/clk (dense, no sparsity)
PEAK_HBM_GBS = 8000.0
METRIC = "attention fwd+bwd TFLOP/s and % bf16 MFMA peak at n=16384,d=64; peak workspace"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def csrc_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2112_05682_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("csrc_digest") != csrc_digest():
        return None
    ent = data.get("kernels", {}).get(kernel)
    if not ent:
        return None
    return ent.get("hbm_bytes_per_launch")


DECODE_WORKLOAD = "decode_bf16_b8h16_nq1_nk65536_d64"


def bench_decode(w, dev, calls: int = 50, warmup: int = 5):
    """Decode-shaped forward (one query per batch and head against n_k keys):
    HBM-bound, so its roofline is the 8 TB/s HBM peak.  Algorithmic bytes per
    call: K and V once (4 n_k d per (batch, head) for 16-bit inputs), Q and O
    (4 n_q d) and the lse (4 n_q); the time includes the combine of the key
    ranges.  HIP events on torch's current stream, the stream the kernels run on."""
    import torch

    from paper_2112_05682_amd import attention_fwd
    from paper_2112_05682_amd.inputs import workload_inputs

    x = {k_: t.to(dev) for k_, t in workload_inputs(w, with_grad=False).items()}
    for _ in range(warmup):
        attention_fwd(x["q"], x["k"], x["v"], causal=w.causal)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(calls):
        attention_fwd(x["q"], x["k"], x["v"], causal=w.causal)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / calls
    bh = w.batch * w.heads
    nbytes = bh * (4 * w.n_k * w.d + 4 * w.n_q * w.d + 4 * w.n_q)
    gbs = nbytes / (ms * 1e-3) / 1e9
    del x
    return {"workload": w.name, "kernel": "attn_decode_kernel", "bound": "hbm", "calls": calls,
            "ms": round(ms, 4), "algorithmic_bytes": nbytes, "achieved": round(gbs, 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
            "traffic": load_traffic("attn_decode_kernel"), "includes": "combine of the key ranges"}


def bench_key_padding(dev, calls: int = 5, warmup: int = 2):
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

    def run(kv_len):
        o, lse, o_lo = attention_fwd(x["q"], x["k"], x["v"], kv_len=kv_len, residual=True)
        attention_bwd(x["q"], x["k"], x["v"], o, lse, x["do"], kv_len=kv_len, o_lo=o_lo)

    out = {}
    for name, kv_len, keys in (("padded", kl, sum(lens)), ("full", None, B * n)):
        for _ in range(warmup):
            run(kv_len)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(calls):
            run(kv_len)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / calls
        out[name] = {"ms": round(ms, 4), "tflops": round(14.0 * d * H * n * keys / (ms * 1e-3) / 1e12, 1)}
    del x
    return {"workload": "selfattn_bf16_b4h16_n8192_d64_kvlen", "kv_len": lens, "calls": calls,
            "includes": "forward + backward (dK/dV and dQ in one call)",
            "valid_key_fraction": sum(lens) / (B * n), **out,
            "time_ratio": round(out["padded"]["ms"] / out["full"]["ms"], 4)}


def cpu_baseline(w):
    """Time the float64 oracle (forward + backward) on whole (batch, head)
    slices of the workload (heads are independent, so a slice is exact)."""
    import oracle
    from paper_2112_05682_amd.inputs import attention_inputs

    # Two full heads of the workload: about 10 s on 16 host threads.
    heads = int(os.environ.get("MEA_CPU_SAMPLE_HEADS", "2"))
    x = attention_inputs(1, heads, w.n_q, w.n_k, w.d, w.dtype, w.std, w.qk_mult)
    q, k, v, do = (x[n].double().numpy() for n in ("q", "k", "v", "do"))
    t0 = time.perf_counter()
    oracle.fwd(q, k, v, scale=w.d ** -0.5, causal=w.causal)
    oracle.bwd(q, k, v, do, scale=w.d ** -0.5, causal=w.causal)
    dt = time.perf_counter() - t0
    pairs = heads * (w.n_q * w.n_k if not w.causal else w.n_q * (w.n_q + 1) // 2)
    flops = 14.0 * w.d * pairs
    return {
        "value": flops / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": "%d of %d heads (n_q = %d, n_k = %d, d = %d), float64 forward + backward "
                  "(%.1f s); credited 14*d*pairs flop / time" % (heads, w.heads, w.n_q, w.n_k,
                                                                 w.d, dt),
        "seconds": dt,
        "host_cpu": platform.processor() or platform.machine(),
    }


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="selfattn_bf16_b1h16_n16384_d64")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 256 MiB device copy (HBM counter calibration)")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the decode-shaped forward measurement")
    ap.add_argument("--no-key-padding", action="store_true",
                    help="skip the key-padding measurement")
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
    w = WORKLOADS[args.workload]
    dev = torch.device("cuda", 0)
    x = {k_: t.to(dev) for k_, t in workload_inputs(w, with_grad=True).items()}
    q, k, v, do = x["q"], x["k"], x["v"], x["do"]
    torch.cuda.synchronize()

    pairs = w.batch * w.heads * (w.n_q * w.n_k if not w.causal else w.n_q * (w.n_q + 1) // 2)
    f_fwd, f_dkdv, f_dq_credit = 4.0 * w.d * pairs, 8.0 * w.d * pairs, 2.0 * w.d * pairs
    f_step = 14.0 * w.d * pairs

    def step(ev):
        # ev: four events recorded before the forward, after it, after the
        # dK/dV call and after the dQ call.
        ev[0].record()
        o, lse, o_lo = attention_fwd(q, k, v, causal=w.causal, residual=True)
        ev[1].record()
        attention_bwd(q, k, v, o, lse, do, causal=w.causal, need_dq=False, o_lo=o_lo)
        ev[2].record()
        attention_bwd(q, k, v, o, lse, do, causal=w.causal, need_dkdv=False, o_lo=o_lo)
        ev[3].record()

    def events():
        return [torch.cuda.Event(enable_timing=True) for _ in range(4)]

    for _ in range(args.warmup):
        step(events())
    torch.cuda.synchronize()

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

    # The timed steps are enqueued back to back (no synchronisation inside the
    # timed region, so the GPU never waits for the host between kernels); the
    # per-kernel event pairs of every step are read after the final
    # synchronisation.
    step_ev = [events() for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for s_ in range(args.steps):
        step(step_ev[s_])
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    t_fwd = sum(e[0].elapsed_time(e[1]) for e in step_ev)
    t_dkdv = sum(e[1].elapsed_time(e[2]) for e in step_ev)
    t_dq = sum(e[2].elapsed_time(e[3]) for e in step_ev)
    ms_step = total_ms / args.steps
    t_fwd, t_dkdv, t_dq = (t / args.steps for t in (t_fwd, t_dkdv, t_dq))

    kernels = {
        "fwd": {"ms": t_fwd, "algorithmic_flop": f_fwd, "tflops": f_fwd / t_fwd / 1e9},
        "bwd_dkdv": {"ms": t_dkdv, "algorithmic_flop": f_dkdv,
                     "tflops": f_dkdv / t_dkdv / 1e9, "includes": "D preprocess"},
        "bwd_dq": {"ms": t_dq, "algorithmic_flop": f_dq_credit,
                   "tflops": f_dq_credit / t_dq / 1e9,
                   "includes": "D preprocess; executes 6*d*P, credited 2*d*P"},
    }
    dom = max(("fwd", "bwd_dkdv"), key=lambda n_: kernels[n_]["ms"])
    # 16-bit d = 64 runs the two-group forward and dK/dV kernels; other shapes
    # the 4-wave ones.
    two_group = w.d == 64
    dom_kernel_name = {"fwd": "attn_fwd_pp_kernel" if two_group else "attn_fwd_kernel",
                       "bwd_dkdv": "attn_bwd_dkdv_pp_kernel" if two_group else "attn_bwd_dkdv_kernel"}[dom]
    achieved = kernels[dom]["tflops"]
    traffic = load_traffic(dom_kernel_name)

    p = _lib.problem(w.batch, w.heads, w.n_q, w.n_k, w.d, _lib.MEA_BF16, w.causal, w.d ** -0.5)
    lib_ws = max(_lib.fwd_workspace_size(p), _lib.bwd_workspace_size(p))
    lse_bytes = w.batch * w.heads * w.n_q * 4
    n2_bytes = w.batch * w.heads * w.n_q * w.n_k * 4

    decode = None if args.no_decode else bench_decode(WORKLOADS[DECODE_WORKLOAD], dev)
    key_padding = None if args.no_key_padding else bench_key_padding(dev)

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
        "fwd_tflops": round(kernels["fwd"]["tflops"], 2),
        "bwd_tflops": round(10.0 * w.d * pairs / ((t_dkdv + t_dq) * 1e-3) / 1e12, 2),
        "fwd_frac_of_peak": round(kernels["fwd"]["tflops"] / PEAK_BF16_TFLOPS, 4),
        "bwd_frac_of_peak": round(10.0 * w.d * pairs / ((t_dkdv + t_dq) * 1e-3) / 1e12
                                  / PEAK_BF16_TFLOPS, 4),
        "kernels_ms": {n_: round(kv["ms"], 4) for n_, kv in kernels.items()},
        "workspace": {"library_bytes": lib_ws, "lse_bytes": lse_bytes,
                      "peak_bytes": lib_ws + lse_bytes,
                      "measured_peak_above_inputs_outputs": max(0, peak_extra - out_bytes),
                      "n2_fp32_matrix_bytes": n2_bytes,
                      "reduction_vs_n2": round(n2_bytes / (lib_ws + lse_bytes), 1)},
        "roofline": {"kernel": dom_kernel_name, "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic},
    }
    if decode is not None:
        out["decode"] = decode
    if key_padding is not None:
        out["key_padding"] = key_padding
    if not args.no_cpu_baseline:
        cb = cpu_baseline(w)
        out["cpu_baseline"] = {kk: (round(vv, 6) if isinstance(vv, float) else vv)
                               for kk, vv in cb.items() if kk not in ("host_cpu",)}
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
