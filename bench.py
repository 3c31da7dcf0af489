#!/usr/bin/env python3
"""Benchmark of the HSTU jagged-attention hot path on one MI355X.

One step = one pass of the whole path over the batch (inputs resident in
HBM): hstu_attn_fwd (work-list scheduling, fused attention forward with
the in-register bias and time bucketisation) then hstu_attn_bwd
(recomputing backward with dQ/dK/dV and the bias-table gradients); for
the training workload the whole layer, hstu_layer_fwd (attention +
LayerNorm(A V) (.) U) then hstu_layer_bwd.  Default workload: the
8192-long shape (B=8 sequences of length U[4096, 8192], h=4,
d_qk=d_v=128, N=8192, bf16).

Prints one JSON line: tokens/s (whole job), the per-kernel breakdown,
the roofline position of the dominant kernel measured live with HIP
events on its own stream, and the CPU oracle timed on a bounded sample
of the same workload.
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
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
METRIC = "HSTU jagged attn fwd+bwd tokens/s & TFLOP/s at N=8192; % bf16 MFMA peak"


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="long", help="tiny|medium|training|long|target")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the oracle timing (profiling runs)")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--no-aux", action="store_true",
                    help="skip the MFMA probe, bucketize and clock measurements")
    ap.add_argument("--bucketize", action="store_true",
                    help="only the standalone bucketize kernel on the workload's timestamps")
    ap.add_argument("--mfalcon", action="store_true",
                    help="only the M-FALCON cached passes on the target workload")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only copy 256 MiB device-to-device 3 times (the reference that "
                         "scales rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes), then exit")
    return ap.parse_args()


def percentile(xs, q):
    xs = sorted(xs)
    k = (len(xs) - 1) * q
    lo, hi = int(k), min(int(k) + 1, len(xs) - 1)
    return xs[lo] + (xs[hi] - xs[lo]) * (k - lo)


def gpu_clock():
    """The clock lines rocm-smi prints for the device (best effort)."""
    import subprocess
    try:
        r = subprocess.run(["rocm-smi", "--showclocks"], capture_output=True, text=True, timeout=20)
    except (OSError, subprocess.SubprocessError):
        return None
    lines = [ln.strip() for ln in r.stdout.splitlines() if "clock level" in ln]
    return lines or None


def bucketize_measurement(hstu, torch, d, batch, stream):
    """The standalone bucketize kernel's write rate on the workload's
    timestamps: warm (ten launches back to back between two events, per
    launch) and cold (one launch after flushing the 256 MB last-level cache
    by writing 512 MB), with the runtime's plain fill of the same buffer
    (timed like warm) as a reachable write rate."""
    out = {}
    po = hstu.hstu_pair_offsets(d["seq_offsets"], stream=stream)
    total_pairs = int(po[-1].item())
    buckets = torch.empty(total_pairs, dtype=torch.uint8, device="cuda")
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    nbytes = total_pairs + 8 * batch.total_tokens

    def bucketize():
        hstu.hstu_time_bucketize(d["seq_offsets"], d["timestamps"], d["rab_time"].numel(),
                                 pair_offsets=po, total_pairs=total_pairs, out=buckets,
                                 stream=stream)

    def timed(fn, reps, before=None):
        ts = []
        for _ in range(6):
            if before is not None:
                before()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / reps)
        return percentile(ts[1:], 0.5)

    for mode, ms in (("warm", timed(bucketize, 10)), ("cold", timed(bucketize, 1, flush.zero_))):
        out[f"bucketize_{mode}"] = {"ms": ms, "gbs": nbytes / (ms * 1e-3) / 1e9,
                                    "frac_hbm": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                                    "bytes": nbytes}
    ms = timed(buckets.zero_, 10)
    out["plain_fill_reference"] = {"ms": ms, "gbs": total_pairs / (ms * 1e-3) / 1e9,
                                   "bytes": total_pairs}
    del flush
    return out


def aux_measurements(hstu, torch, d, batch, stream):
    """Outside the timed region: the matrix-core rate of a kernel that only
    issues bf16 MFMAs (the measured ceiling the attention kernels are also
    compared against), and the standalone bucketize kernel's write rate
    with the 256 MB last-level cache warm and flushed."""
    out = {}
    sink = torch.empty(256, dtype=torch.float32, device="cuda")
    rates = []
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        flop = hstu.hstu_probe_mfma_bf16(20000, 2, sink, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        rates.append(flop / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    out["mfma_probe"] = {"tflops": max(rates[1:]), "frac_of_spec": max(rates[1:]) / PEAK_BF16_TFLOPS,
                         "kernel": "bf16 v_mfma_f32_32x32x16, 8 independent chains per wave, "
                                   "2 waves per SIMD, every CU"}
    out.update(bucketize_measurement(hstu, torch, d, batch, stream))
    out["mfalcon"] = mfalcon_measurement(hstu, torch, stream)
    out["projections"] = projection_measurement(hstu, torch, stream)
    out["stochastic_length"] = sl_measurement(hstu, torch, stream)
    out["gpu_clock"] = gpu_clock()
    return out


def _time_ms(torch, stream, fn, reps=6):
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return percentile(ts[1:], 0.5)


def projection_measurement(hstu, torch, stream):
    """The layer's linear maps at the training shape (T = 60383 tokens of the
    training workload, d_model = 512, h = 8, d = 64, so F = 2048): f_1 with
    SiLU (Eq. 1), f_2 with bias and residual (Eq. 3), and their backward
    calls (input and weight gradients, bias sums); rate = matrix FLOPs of
    each call / its time."""
    from paper_2402_17152_amd import inputs
    T = int(inputs.make_batch("training").seq_offsets[-1])
    D, h, dqk, dv = 512, 8, 64, 64
    hv, F = h * dv, 2 * h * (dqk + dv)
    P = inputs.make_proj(T, D, h, dqk, dv, dtype="bf16", seed=7)
    d = {k: inputs.array_to_device(v) for k, v in P.items()}
    z, z_pre = hstu.hstu_proj_in_fwd(d["x"], d["w1"], d["b1"], h, dqk, dv, stream=stream)
    y = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
    dz = [d["dz"][:, a:b].contiguous().view(T, h, -1)
          for a, b in ((0, hv), (hv, 2 * hv), (2 * hv, 2 * hv + h * dqk), (2 * hv + h * dqk, F))]
    p = hstu.proj_problem(d["x"], h, dqk, dv)
    ws = hstu.proj_workspace(p, D)
    outs_in = (torch.empty_like(d["x"]), torch.empty((F, D), dtype=torch.float32, device="cuda"),
               torch.empty(F, dtype=torch.float32, device="cuda"))
    outs_out = (torch.empty_like(d["g"]), torch.empty((D, hv), dtype=torch.float32, device="cuda"),
                torch.empty(D, dtype=torch.float32, device="cuda"))
    calls = {
        "proj_in_fwd": (2 * T * D * F, lambda: hstu.hstu_proj_in_fwd(
            d["x"], d["w1"], d["b1"], h, dqk, dv, z=z, z_pre=z_pre, stream=stream)),
        "proj_out_fwd": (2 * T * hv * D, lambda: hstu.hstu_proj_out_fwd(
            d["g"], d["w2"], d["b2"], d["x"], h, dqk, dv, y=y, stream=stream)),
        "proj_out_bwd": (4 * T * hv * D, lambda: hstu.hstu_proj_out_bwd(
            d["g"], d["w2"], d["dy"], h, dqk, dv, out=outs_out, ws=ws, stream=stream)),
        "proj_in_bwd": (4 * T * D * F, lambda: hstu.hstu_proj_in_bwd(
            d["x"], d["w1"], z_pre, *dz, h, dqk, dv, dx_add=d["dy"], out=outs_in, ws=ws,
            stream=stream)),
    }
    res = {"shape": f"T={T}, d_model={D}, h={h}, d_qk=d_v=64, F={F}, bf16"}
    tot_ms, tot_flop = 0.0, 0
    for name, (flop, fn) in calls.items():
        ms = _time_ms(torch, stream, fn, reps=8)
        res[name] = {"ms": ms, "tflops": flop / (ms * 1e-3) / 1e12, "flop": flop}
        tot_ms += ms
        tot_flop += flop
    res["all_four"] = {"ms": tot_ms, "tflops": tot_flop / (tot_ms * 1e-3) / 1e12}
    return res


def sl_measurement(hstu, torch, stream):
    """Stochastic Length (Eq. 4) on the training workload (B = 64, power-law
    lengths up to N = 4096, h = 8, d = 64) at alpha = 1.6 (L = 776), random
    selection: the sampler plus the gather of q, k, v, u and timestamps, the
    sparsity before and after, and the attention forward + backward on the
    shrunk batch against the full one."""
    import numpy as np
    from paper_2402_17152_amd import inputs
    batch = inputs.make_batch("training")
    d = inputs.to_device(batch)
    N = batch.spec.max_seq_len
    L = hstu.hstu_sl_subseq_len(N, 1.6)
    kn = hstu.hstu_sl_keep_numerator(N, 1.6)
    u, e = inputs.make_sl_draws(len(batch.lengths), batch.seq_offsets[-1], seed=5)
    ud, ed = torch.from_numpy(u).cuda(), torch.from_numpy(e).cuda()
    T = batch.total_tokens
    new_offs = torch.empty(len(batch.lengths) + 1, dtype=torch.int64, device="cuda")
    gather = torch.empty(T, dtype=torch.int64, device="cuda")
    ws = torch.empty(hstu.hstu_sl_workspace_bytes(len(batch.lengths)), dtype=torch.uint8,
                     device="cuda")
    bufs = {k: torch.empty_like(d[k]) for k in ("q", "k", "v", "u", "timestamps")}

    def sample():
        hstu.hstu_stochastic_length(d["seq_offsets"], d["timestamps"], L, kn, hstu.HSTU_SL_RANDOM,
                                    ud, ed, out=(new_offs, gather), ws=ws, stream=stream)
        for k, dst in bufs.items():
            hstu.hstu_gather_rows(d[k], gather, new_offs[-1:], max_rows=T, dst=dst, stream=stream)
    ms_sample = _time_ms(torch, stream, sample)
    offs_new = new_offs.cpu().numpy()
    T2 = int(offs_new[-1])
    sp0, s20 = hstu.hstu_sl_sparsity(batch.seq_offsets, N)
    sp1, s21 = hstu.hstu_sl_sparsity(offs_new, N)

    def attn(dd, offs, ntok):
        q, k, v = dd["q"][:ntok], dd["k"][:ntok], dd["v"][:ntok]
        do = d["do"][:ntok]
        def run():
            hstu.hstu_attn_fwd(q, k, v, offs, dd["timestamps"][:ntok], d["rab_pos"], d["rab_time"],
                               N, stream=stream)
            hstu.hstu_attn_bwd(q, k, v, do, offs, dd["timestamps"][:ntok], d["rab_pos"],
                               d["rab_time"], N, stream=stream)
        return _time_ms(torch, stream, run)
    ms_full = attn(d, d["seq_offsets"], T)
    ms_sl = attn(bufs, new_offs, T2)
    return {"workload": f"training: B={len(batch.lengths)}, T={T}, N={N}, alpha=1.6, L={L}, "
                        "random selection",
            "sampler_and_gather_ms": ms_sample, "tokens_before": T, "tokens_after": T2,
            "sparsity_before": sp0, "sparsity_after": sp1, "s2_before": s20, "s2_after": s21,
            "attn_fwd_bwd_ms_full": ms_full, "attn_fwd_bwd_ms_sl": ms_sl,
            "attention_speedup": ms_full / ms_sl}


def mfalcon_measurement(hstu, torch, stream):
    """M-FALCON on the target workload (16 users, 2048 prefix tokens, 1024
    candidates, h=4, d=128, N=3072): the uncached target-aware forward over
    prefix ++ all candidates against cached passes that compute only the
    candidate rows from the prefix's cached K and V, as one microbatch of
    1024, four of 256 and sixteen of 64 (inputs of each microbatch gathered
    beforehand), called one by one and replayed from a captured graph."""
    import numpy as np
    from paper_2402_17152_amd import inputs
    batch = inputs.make_batch("target")
    s = batch.spec
    d = inputs.to_device(batch)
    N = s.max_seq_len
    offs, nt = batch.seq_offsets, batch.num_targets
    B = len(nt)
    nh = np.diff(offs) - nt

    def idx(parts):
        return torch.from_numpy(np.concatenate(parts).astype(np.int64)).cuda()

    pre = idx([np.arange(offs[b], offs[b] + nh[b]) for b in range(B)])
    kc, vc = d["k"].index_select(0, pre), d["v"].index_select(0, pre)
    cts = d["timestamps"].index_select(0, pre)
    coffs = torch.from_numpy(np.concatenate([[0], np.cumsum(nh)]).astype(np.int64)).cuda()

    def microbatches(b_m):
        mbs = []
        for i in range((int(nt.max()) + b_m - 1) // b_m):
            c0, c1 = np.minimum(i * b_m, nt), np.minimum((i + 1) * b_m, nt)
            r = idx([np.arange(offs[b] + nh[b] + c0[b], offs[b] + nh[b] + c1[b])
                     for b in range(B)])
            co = torch.from_numpy(np.concatenate([[0], np.cumsum(c1 - c0)]).astype(np.int64))
            q, k, v = (d[x].index_select(0, r) for x in ("q", "k", "v"))
            ts = d["timestamps"].index_select(0, r)
            p = hstu.problem_for(q, v, co, N, d["rab_time"])
            mbs.append((q, k, v, co.cuda(), ts, torch.empty_like(v), hstu.cached_workspace(p)))
        return mbs

    full_out = torch.empty_like(d["v"])
    ws_full = hstu.workspace(hstu.problem_for(d["q"], d["v"], d["seq_offsets"], N, d["rab_time"]))
    ms_uncached = _time_ms(torch, stream, lambda: hstu.hstu_attn_fwd(
        d["q"], d["k"], d["v"], d["seq_offsets"], d["timestamps"], d["rab_pos"], d["rab_time"],
        N, num_targets=d["num_targets"], out=full_out, ws=ws_full, stream=stream))
    cand = int(nt.sum())
    flop_cached = 2 * (s.d_qk + s.d_v) * s.num_heads * int((nt * (nh + 1)).sum())
    res = {"workload": "target: 16 users x (2048 prefix + 1024 candidates), h=4, d=128, N=3072",
           "uncached_ms": ms_uncached,
           "cached_flop": flop_cached}
    for b_m in (1024, 256, 64):
        mbs = microbatches(b_m)

        def run(st=stream):
            for (q, k, v, co, ts, o, ws) in mbs:
                hstu.hstu_attn_fwd_cached(q, k, v, co, ts, kc, vc, coffs, cts, d["rab_pos"],
                                          d["rab_time"], N, out=o, ws=ws, stream=st)
        ms = _time_ms(torch, stream, run)
        # The same passes replayed from a HIP graph (captured once; each
        # replay launches every pass's kernels without host calls in between).
        run()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run(st=torch.cuda.current_stream())
        ms_graph = _time_ms(torch, stream, g.replay)
        res[f"cached_b{b_m}"] = {"ms": ms, "passes": len(mbs),
                                 "tflops": flop_cached / (ms * 1e-3) / 1e12,
                                 "candidates_per_s": cand / (ms * 1e-3),
                                 "speedup_vs_uncached": ms_uncached / ms,
                                 "graph_ms": ms_graph,
                                 "graph_speedup_vs_uncached": ms_uncached / ms_graph}
        del g
    return res


def source_hash(*names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2402_17152_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counters_traffic(kernel: str, workload: str, src: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if
    it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != src:
        return None
    return rec.get("hbm_bytes_per_launch")


def dq_partial_bytes(batch, block_rows=32, block_keys=128):
    """Bytes of f16 partial dQ blocks the two-role backward stores (and
    its reduce pass reads back): one 32-row x d_qk block per 32-row step of
    every 128-key block and head."""
    s = batch.spec
    slots = 0
    for L in np.diff(batch.seq_offsets):
        S = (int(L) + block_rows - 1) // block_rows
        K = (int(L) + block_keys - 1) // block_keys
        slots += K * S - 2 * K * (K - 1)
    return slots * s.num_heads * s.d_qk * block_rows * 2


def dq_atomic_bytes(batch, block_keys=128):
    """Bytes the bf16 backward adds to its fp32 dQ accumulator with
    atomics: every (sequence, 128-key block, head) work item adds a
    d_qk-wide fp32 row for each row it visits (from its first key to the
    sequence end; candidate key blocks visit their own rows only)."""
    s = batch.spec
    offs = batch.seq_offsets
    nt = batch.num_targets
    rows = 0
    for b in range(len(offs) - 1):
        L = int(offs[b + 1] - offs[b])
        n_h = L - (int(nt[b]) if nt is not None else 0)
        for j0 in range(0, L, block_keys):
            i_end = min(j0 + block_keys, L) if j0 >= n_h else L
            rows += i_end - j0
    return rows * s.num_heads * s.d_qk * 4


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(batch, flops_full):
    """The oracle, untuned, over the whole workload: one forward (and, for
    the fwd+bwd workloads, one backward with the seeded dO) on the host
    cores, OpenMP over (sequence, head) tasks; tokens/s = T / wall time."""
    import oracle

    threads = oracle.num_threads()
    N = batch.spec.max_seq_len
    args = (batch.seq_offsets, N, batch.timestamps, batch.rab_pos, batch.rab_time,
            batch.f64("q"), batch.f64("k"), batch.f64("v"))
    t0 = time.perf_counter()
    oracle.attn_fwd(*args, num_targets=batch.num_targets)
    if batch.spec.backward:
        oracle.attn_bwd(*args, batch.f64("do"), num_targets=batch.num_targets)
    dt = time.perf_counter() - t0
    tasks = len(batch.lengths) * batch.spec.num_heads
    return {
        "value": batch.total_tokens / dt,
        "unit": "tokens/s",
        "cores": min(threads, tasks),
        "kind": "oracle",
        "sample": (f"the whole workload (T={batch.total_tokens}, {len(batch.lengths)} sequences x "
                   f"{batch.spec.num_heads} heads): fp64 oracle fwd"
                   f"{'+bwd' if batch.spec.backward else ''}, {flops_full:.3e} FLOP in {dt:.1f} s "
                   f"= {flops_full / dt / 1e9:.2f} GFLOP/s on {threads} OpenMP threads "
                   f"({_cpu_model()})"),
        "gflops": flops_full / dt / 1e9,
        "seconds": dt,
        "cpu_model": _cpu_model(),
    }


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the library runs on exactly one GPU (the path shards by sequence and "
              "needs no collective until the bias-gradient all-reduce, which is not built); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.calibrate_copy:
        n = 256 << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": n, "copies": 3}), flush=True)
        return

    from paper_2402_17152_amd import hstu, inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.mfalcon:
        print(json.dumps(mfalcon_measurement(hstu, torch, torch.cuda.current_stream())), flush=True)
        return
    batch = inputs.make_batch(args.workload)
    spec = batch.spec
    d = inputs.to_device(batch)
    if args.bucketize:
        res = bucketize_measurement(hstu, torch, d, batch, torch.cuda.current_stream())
        print(json.dumps({"workload": args.workload, "total_tokens": batch.total_tokens, **res}),
              flush=True)
        return
    T = batch.total_tokens
    N = spec.max_seq_len
    f_fwd, f_bwd = inputs.flops(batch)
    flops_step = f_fwd + (f_bwd if spec.backward else 0)
    p = hstu.problem_for(d["q"], d["v"], d["seq_offsets"], N, d["rab_time"])
    ws = hstu.workspace(p)
    D = spec.num_heads * spec.d_v
    dt = d["q"].dtype
    attn_out = torch.empty((T, D), dtype=torch.float32, device="cuda")
    y = torch.empty((T, D), dtype=dt, device="cuda")
    mean = torch.empty(T, dtype=torch.float32, device="cuda")
    rstd = torch.empty(T, dtype=torch.float32, device="cuda")
    grads = (torch.empty_like(d["q"]), torch.empty_like(d["k"]), torch.empty_like(d["v"]),
             torch.empty_like(d["rab_pos"]), torch.empty_like(d["rab_time"]))
    stream = torch.cuda.current_stream()

    # The training workload times the whole layer (attention, LayerNorm
    # gate, and their backward); the others the attention alone.
    layer = spec.name == "training"
    out_bf = torch.empty((T, spec.num_heads, spec.d_v), dtype=dt, device="cuda")
    lgrads = None
    if layer:
        lgrads = (grads[0], grads[1], grads[2], torch.empty((T, D), dtype=dt, device="cuda"), None,
                  None, grads[3], grads[4])
    dy = d["do"].reshape(T, D)

    def step():
        if layer:
            hstu.hstu_layer_fwd(d["q"], d["k"], d["v"], d["u"], d["seq_offsets"], d["timestamps"],
                                d["rab_pos"], d["rab_time"], N, num_targets=d["num_targets"],
                                attn_out=attn_out, y=y, ln_mean=mean, ln_rstd=rstd, ws=ws,
                                stream=stream)
            if spec.backward:
                hstu.hstu_layer_bwd(d["q"], d["k"], d["v"], d["u"], attn_out, mean, rstd, dy,
                                    d["seq_offsets"], d["timestamps"], d["rab_pos"],
                                    d["rab_time"], N, num_targets=d["num_targets"],
                                    grads=lgrads, ws=ws, stream=stream)
            return
        hstu.hstu_attn_fwd(d["q"], d["k"], d["v"], d["seq_offsets"], d["timestamps"],
                           d["rab_pos"], d["rab_time"], N, num_targets=d["num_targets"],
                           out=out_bf, ws=ws, stream=stream)
        if spec.backward:
            hstu.hstu_attn_bwd(d["q"], d["k"], d["v"], d["do"], d["seq_offsets"],
                               d["timestamps"], d["rab_pos"], d["rab_time"], N,
                               num_targets=d["num_targets"], grads=grads, ws=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    hstu.hstu_timing_reset()
    if not args.no_kernel_timing:
        hstu.hstu_timing_enable(True)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    evs[0].record(stream)
    for k in range(args.steps):
        step()
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    hstu.hstu_timing_enable(False)
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = [evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps)]

    kernels = {}
    for name in ("attn_fwd", "ln_gate", "ln_gate_bwd", "attn_bwd", "dq_reduce"):
        tot, n = hstu.hstu_timing_read(name)
        if n:
            kernels[name] = {"avg_ms": tot / n, "launches": n}
    # Algorithmic work per launch: FLOPs of the contractions for attention,
    # bytes read + written for the epilogue.
    # fp32 attention output read, u read and y written in the problem's dtype
    ln_bytes = T * D * (4 + 2 * (2 if spec.dtype == "bf16" else 4)) + 8 * T
    if "attn_fwd" in kernels:
        kernels["attn_fwd"]["tflops"] = f_fwd / (kernels["attn_fwd"]["avg_ms"] * 1e-3) / 1e12
    if "attn_bwd" in kernels:
        kernels["attn_bwd"]["tflops"] = f_bwd / (kernels["attn_bwd"]["avg_ms"] * 1e-3) / 1e12
    if "dq_reduce" in kernels:
        # f16 partial blocks read, bf16 dQ written
        rb = dq_partial_bytes(batch) + T * spec.num_heads * spec.d_qk * 2
        kernels["dq_reduce"]["gbs"] = rb / (kernels["dq_reduce"]["avg_ms"] * 1e-3) / 1e9
    if "ln_gate" in kernels:
        kernels["ln_gate"]["gbs"] = ln_bytes / (kernels["ln_gate"]["avg_ms"] * 1e-3) / 1e9
    if "ln_gate_bwd" in kernels:
        e = 2 if spec.dtype == "bf16" else 4
        lnb_bytes = T * D * (4 + 4 * e) + 8 * T
        kernels["ln_gate_bwd"]["gbs"] = lnb_bytes / (kernels["ln_gate_bwd"]["avg_ms"] * 1e-3) / 1e9

    peak = PEAK_BF16_TFLOPS if spec.dtype == "bf16" else PEAK_FP32_TFLOPS
    dom = "attn_bwd" if spec.backward else "attn_fwd"
    roofline = None
    if dom in kernels:
        src = source_hash("attn_bwd.hip" if dom == "attn_bwd" else "attn_fwd.hip", "common.h")
        ach = kernels[dom]["tflops"]
        roofline = {"bound": "mfma", "kernel": dom, "achieved": ach, "peak": peak,
                    "unit": "TFLOP/s", "frac": ach / peak,
                    "traffic": counters_traffic(dom, args.workload, src),
                    "flop_per_launch": f_bwd if dom == "attn_bwd" else f_fwd,
                    "source_hash": src}
        if dom == "attn_bwd" and spec.dtype == "bf16":
            if layer:
                # Two-term dO: the single-role kernel adds the dQ partial sums
                # of its 128-key work items to memory as fp32 atomics.
                qb = dq_atomic_bytes(batch)
                roofline["dq_atomic_bytes"] = qb
                roofline["dq_atomic_tbs"] = qb / (kernels[dom]["avg_ms"] * 1e-3) / 1e12
            else:
                # The two-role kernel stores them as f16 blocks (each with
                # a power-of-two scale); a reduce pass (kernels.dq_reduce)
                # reads them back.
                roofline["dq_partial_bytes"] = dq_partial_bytes(batch)

    aux = None if args.no_aux else aux_measurements(hstu, torch, d, batch, stream)
    if roofline is not None and aux is not None:
        roofline["peak_measured"] = aux["mfma_probe"]["tflops"]
        roofline["frac_measured"] = roofline["achieved"] / aux["mfma_probe"]["tflops"]

    tflops = flops_step / (ms * 1e-3) / 1e12
    rec = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_p10_p50_p90": [percentile(per_step, 0.1), percentile(per_step, 0.5),
                                    percentile(per_step, 0.9)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic (seeded generator; no dataset)",
        "config": {
            "workload": f"{spec.name}: B={len(batch.lengths)} jagged sequences, T={T}, "
                        f"h={spec.num_heads}, d_qk={spec.d_qk}, d_v={spec.d_v}, N={N}, "
                        f"{'target-aware' if spec.target_aware else 'causal'}; step = "
                        + ("layer fwd (attention + LayerNorm gate)" + (" + layer bwd (LayerNorm-gate "
                           "backward, attention backward with bias gradients)" if spec.backward else "")
                           if layer else "attention fwd" + (" + attention bwd with bias gradients"
                                                            if spec.backward else "")),
            "num_seqs": len(batch.lengths),
            "total_tokens": T,
            "max_seq_len": N,
            "parallelism": "single GPU",
        },
        "tflops": tflops,
        "pct_bf16_peak": 100.0 * tflops / PEAK_BF16_TFLOPS,
        "flop_per_step": flops_step,
        "wall_s_timed": t_wall,
        "kernels": kernels,
        "roofline": roofline,
        "aux": aux,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(batch, flops_step)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
