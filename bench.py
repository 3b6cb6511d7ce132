#!/usr/bin/env python3
"""Throughput benchmark of the global CG convolution on one MI355X.

Workload (the configuration the headline metric is quoted on): point-cloud
token sets, B=8, N=16384 tokens, L_max=6 (49 components), C=32 channels,
fp32 -- synthetic inputs shaped like the paper's point-cloud experiments
(features = real spherical harmonics of ellipsoid surface normals times
per-channel weights; see workloads/).  One step = one cgconv_forward of the
whole batch (forward DFTs, sparse CG product, inverse DFTs), inputs already
resident in HBM.

Prints ONE JSON line.  Besides the contract fields it carries
  roofline      the dominant kernel (the CG stage, VALU-bound) against the
                fp32 vector peak (157.3 TFLOP/s), timed live with HIP
                events on the stream the kernels run on; traffic from the
                committed rocprofv3 counter summary if it was taken on the
                current kernel source
  stages        per-stage average time and achieved bandwidth of each kernel
  cpu_baseline  the CPU oracle (direct O(N^2) definition) on sampled output
                rows of the same inputs; those rows also check the GPU output
Flags: --gpus N (only 1 is supported), --steps K, --warmup W,
--no-cpu-baseline, --cpu-seconds S, --workload NAME (other synthetic
workloads, for exploration), --bf16, --copy-calibration (a plain device copy
of known size, the reference for rocprofv3 byte counters), --mixed (the
convolution with per-path channel mixing, cgconv_forward_mixed, with seeded
random weights: its own JSON line, the mixing stage against the bf16 matrix
core peak), --backward (cgconv_backward, both gradients, for a seeded
output gradient: its own JSON line), --gate (cgconv_gate_value with the
workload's q and k as u and v: its own JSON line, gate_value against the
fp32 vector peak), --gate-backward (cgconv_gate_value_backward, both
gradients, for a seeded upstream gradient: its own JSON line), --graph (cgconv_forward_graph on the graph workload,
B=4, N=4096, L=6, C=32, with Laplacian eigenbases: its own JSON line, the
forward transform against the bf16 matrix core peak), --boundary linear (any mode on a plan with the
zero-padded token boundary: DFTs of length 2N).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
# fp32 vector peak: 256 CUs x 4 SIMDs x 32 lanes per cycle x 2 flop x 2.4 GHz.
# A SIMD completes one wave64 fp32 FMA (v_fmac_f32, not packed) every 2
# cycles when two or more waves are ready; one wave alone issues at most one
# every 4 cycles, i.e. half this rate.
VALU_PEAK_TFLOPS = 256 * 4 * 32 * 2 * 2.4e9 / 1e12
METRIC = "CG-conv tokens/sec at N=16384, L_max=6, C=32; achieved HBM GB/s vs peak"
METRIC_MIXED = "CG-conv with per-path channel mixing, tokens/sec at N=16384, L_max=6, C=32"
METRIC_INTER = ("inter-channel CG-conv (4 heads x 8 channels, all channel pairs, per-degree reduction to 8), "
                "tokens/sec at N=16384, L_max=6")
METRIC_GRAPH = "CG-conv in a graph Fourier basis, tokens/sec at N=4096, L_max=6, C=32"
METRIC_LINEAR = "CG-conv with the zero-padded (linear) boundary, tokens/sec at N=16384, L_max=6, C=32"
METRIC_BACKWARD = "CG-conv backward (grad_q and grad_k), tokens/sec at N=16384, L_max=6, C=32"
METRIC_GATE = "invariant softmax gating + value tensor product, tokens/sec at N=16384, L_max=6, C=32"
METRIC_GATE_BACKWARD = ("gating + value tensor product backward (grad_u and grad_v), tokens/sec at N=16384, "
                        "L_max=6, C=32")
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak, published
# sources of every kernel of the fused forward (the step's counter bytes
# cover all three stages) and of the plan that launches them
CG_SOURCES = ["paper_2509_24093_amd/csrc/cg_gen.hip", "paper_2509_24093_amd/csrc/cg_fused.hip",
              "paper_2509_24093_amd/csrc/fft.hip", "paper_2509_24093_amd/csrc/cgconv.cpp",
              "paper_2509_24093_amd/csrc/cg_common.h", "paper_2509_24093_amd/csrc/fft_reg.h",
              "paper_2509_24093_amd/csrc/codegen/gen_cg.cpp", "paper_2509_24093_amd/csrc/cg_table.cpp",
              "paper_2509_24093_amd/csrc/kernels.h"]
PMC_SUMMARY = os.path.join(ROOT, "profiles", "cg_kernel_pointcloud_pmc.md")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cg_source_hash() -> str:
    h = hashlib.sha256()
    for rel in CG_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def committed_counters(workload):
    """The committed rocprofv3 counter summary (calibrated HBM bytes per CG
    launch and per whole step) if it was taken on the current CG kernel
    source and this workload, else (None, reason)."""
    if not os.path.exists(PMC_SUMMARY):
        return None, "no counter summary committed"
    text = open(PMC_SUMMARY).read()
    start = text.find("```json")
    if start < 0:
        return None, "counter summary has no json block"
    end = text.find("```", start + 7)
    d = json.loads(text[start + 7:end])
    if d.get("cg_source_hash") != cg_source_hash():
        return None, "CG kernel changed since the counters were taken"
    if d.get("workload") != workload:
        return None, "counters were taken on another workload"
    return d, "rocprofv3 FETCH_SIZE+WRITE_SIZE, copy-calibrated"


def copy_calibration():
    import torch
    n = 1 << 28  # 1 GiB of fp32
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}), flush=True)


def copy_peak_gbs(nbytes=1 << 30, reps=10):
    """Measured HBM ceiling: bytes read plus written per second by a plain
    device-to-device copy of nbytes on the current stream (HIP events on that
    stream, after warm-up copies)."""
    import torch
    src = torch.ones(nbytes // 4, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2 * nbytes / (ms * 1e-3) / 1e9


def hbm_ceiling(nbytes=1 << 30, reps=10):
    """Measured HBM ceiling: the hand-written streaming kernels of
    libhbmprobe.so (16-byte accesses: copy, copy with nontemporal loads and
    stores, read only, write only), each at a few grid sizes, timed with HIP
    events on the current stream after warm-up launches, next to torch's
    device copy.  Returns {name: GB/s (bytes read + written per second)} with
    the grid size of each best result."""
    import ctypes

    import torch
    from paper_2509_24093_amd.build import PROBE_LIB
    lib = ctypes.CDLL(PROBE_LIB)
    lib.hbm_probe.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                              ctypes.c_void_p]
    lib.hbm_probe.restype = ctypes.c_int
    src = torch.ones(nbytes // 4, device="cuda")
    dst = torch.empty_like(src)
    stream = torch.cuda.current_stream().cuda_stream
    out = {}
    for mode, name, moved in ((0, "copy", 2), (1, "copy_nontemporal", 2), (2, "read", 1), (3, "write", 1)):
        best = (0.0, 0)
        for blocks in (1024, 2048, 4096, 8192):
            def launch():
                if lib.hbm_probe(src.data_ptr(), dst.data_ptr(), nbytes, mode, blocks, stream) != 0:
                    raise RuntimeError("hbm_probe launch failed")
            for _ in range(2):
                launch()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                launch()
            e1.record()
            torch.cuda.synchronize()
            gbs = moved * nbytes / (e0.elapsed_time(e1) / reps * 1e-3) / 1e9
            best = max(best, (gbs, blocks))
        out[name + "_gbs"] = round(best[0], 1)
        out[name + "_blocks"] = best[1]
    del src, dst
    out["torch_copy_gbs"] = round(copy_peak_gbs(nbytes, reps), 1)
    return out


def cpu_baseline(q, k, L, budget_s, got, linear=False):
    """Oracle direct mode on sampled output rows; returns the bench object and
    the parity of the GPU output on those rows."""
    import numpy as np
    from oracle.conv import cgconv_direct_linear_rows, cgconv_direct_rows
    rows_fn = cgconv_direct_linear_rows if linear else cgconv_direct_rows
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max((d.get("num_threads", 1) for d in threadpool_info()), default=1)
    except Exception:
        blas_threads = None
    B, N = q.shape[0], q.shape[1]
    rng = np.random.default_rng(2024)
    # rows in chunks of 8 per batch element, cycling over b, until the budget
    # is spent; (0, 0) and (B-1, N-1) are always included
    rows, ref, chunk_s = [], [], []
    t0 = time.perf_counter()
    chunk = 0
    while True:
        tc = time.perf_counter()
        b = chunk % B
        picks = [int(x) for x in rng.integers(0, N, size=8)]
        if chunk == 0:
            picks[0] = 0
        if chunk == B - 1:
            picks[0] = N - 1
        part = [(b, i) for i in picks]
        ref.extend(rows_fn(q, k, L, part))
        rows.extend(part)
        chunk_s.append(time.perf_counter() - tc)
        chunk += 1
        if time.perf_counter() - t0 >= budget_s and chunk >= B:
            break
    dt = time.perf_counter() - t0
    R = len(rows)
    # three consecutive thirds of the chunks timed as separate runs; the
    # reported rate is their median
    thirds = [chunk_s[i * len(chunk_s) // 3:(i + 1) * len(chunk_s) // 3] for i in range(3)]
    rates = sorted(8 * len(t) / sum(t) for t in thirds if t)
    num = den = 0.0
    for n, (b, i) in enumerate(rows):
        d = got[b, i].astype(np.float64) - ref[n]
        num += float((d * d).sum())
        den += float((ref[n] * ref[n]).sum())
    cores = len(os.sched_getaffinity(0))
    value = rates[len(rates) // 2] if rates else R / dt
    obj = {"value": value, "unit": "tokens/s", "cores": blas_threads or cores, "kind": "oracle",
           "sample": f"direct O(N^2) definition on {R} sampled output rows (b, i) of the same workload "
                     f"(all K components and C channels per row), fp64 numpy, {dt:.1f} s; median of "
                     f"three runs of {len(chunk_s) // 3}+ chunks of 8 rows "
                     f"({', '.join(f'{r:.2f}' for r in rates)} rows/s); host exposes {cores} cores"}
    return obj, (num / den) ** 0.5 if den > 0 else 0.0, R


def cpu_fft_baseline(q, k, L, budget_s, got):
    """The oracle's FFT mode (the convolution theorem in fp64 numpy, dense
    R_full) over whole channels, batch element by batch element and channel
    by channel until the budget is spent or the whole tensor is done;
    returns the bench object (token-equivalents per second: tokens times the
    fraction of the channels done) and the parity of the GPU output on
    what was computed."""
    import numpy as np
    from oracle.conv import cgconv_fft
    B, N, K, C = q.shape
    n_done, dt, num, den = 0, 0.0, 0.0, 0.0
    for b in range(B):
        for c in range(C):
            t0 = time.perf_counter()
            ref = cgconv_fft(q[b:b + 1], k[b:b + 1], L, channels=[c])
            dt += time.perf_counter() - t0
            d = got[b:b + 1, ..., c:c + 1].astype(np.float64) - ref
            num += float((d * d).sum())
            den += float((ref * ref).sum())
            n_done += 1
            if dt >= budget_s:
                break
        if dt >= budget_s:
            break
    cores = len(os.sched_getaffinity(0))
    what = "the whole tensor" if n_done == B * C else f"{n_done} of {B * C} (batch element, channel) signals"
    obj = {"value": N * n_done / C / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle (FFT mode)",
           "sample": f"{what}, all {N} tokens each ({N * n_done / C:.0f} token-equivalents), fp64 numpy FFT mode "
                     f"with the dense R_full contraction, {dt:.1f} s"}
    return obj, (num / den) ** 0.5 if den > 0 else 0.0, n_done == B * C


def dft_length(N, boundary):
    """Length of the token DFTs: N (cyclic) or the smallest power of two
    >= 2N - 1 (zero-padded boundary)."""
    if boundary == "cyclic":
        return N
    n = 2
    while n < 2 * N - 1:
        n *= 2
    return n


KERNEL_OF_STAGE = {"cg_fused": "cg_fused_kernel", "cg_small": "cg_small_kernel"}


def cg_roofline(stage_avg, B, N, L, C, n_products, nnz, traffic, traffic_src):
    """Roofline object of the CG stage (fused or unfused) from its average
    launch time: algorithmic flops per launch against the fp32 vector peak."""
    K = (L + 1) ** 2
    Cp = (C + 1) // 2
    F = N // 2 + 1
    points = B * F * C
    cg_flops_per_point = 6 * n_products + 4 * nnz
    dom = "cg_fused" if "cg_fused" in stage_avg else ("cg_small" if "cg_small" in stage_avg else "cg")
    cg_ms = stage_avg[dom]
    flops = points * cg_flops_per_point
    flop_model = (f"(6*{n_products} distinct complex products + 4*{nnz} non-zeros) per "
                  f"(b, frequency 0..N/2, channel) point, {points} points")
    if dom == "cg_fused":
        # the fused kernel also runs the length-64 DFTs over n2: 5 n log2 n
        # flops per complex transform, K*C forward and K*ceil(C/2) inverse
        # columns per class
        n1 = N // 64
        dft = 5 * 64 * 6
        flops += dft * B * n1 * K * (C + Cp)
        flop_model += f" + {dft}-flop length-64 DFTs on {B * n1 * K * (C + Cp)} columns"
    elif dom == "cg_small":
        # the one-block kernel runs both whole DFTs: 5 N log2 N flops per
        # complex transform, K*C forward and K*ceil(C/2) inverse columns
        dft = 5 * N * (N.bit_length() - 1)
        flops += dft * B * K * (C + Cp)
        flop_model += f" + {dft}-flop length-{N} DFTs on {B * K * (C + Cp)} columns"
    achieved_tflops = flops / (cg_ms * 1e-3) / 1e12
    return {
        "kernel": f"{KERNEL_OF_STAGE.get(dom) or ('cg_split_kernel' if L >= 7 else 'cg_gen_kernel')}<{L}>",
        "bound": "alu",
        "achieved": round(achieved_tflops, 2),
        "peak": round(VALU_PEAK_TFLOPS, 1),
        "unit": "TFLOP/s",
        "frac": round(achieved_tflops / VALU_PEAK_TFLOPS, 4),
        "traffic": traffic,
        "traffic_source": traffic_src,
        "flops_per_launch": flops,
        "flop_model": flop_model,
        "launch_ms": round(cg_ms, 4),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="pointcloud")
    ap.add_argument("--bf16", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--mixed", action="store_true")
    ap.add_argument("--interchannel", action="store_true")
    ap.add_argument("--heads", type=int, default=4)
    ap.add_argument("--backward", action="store_true")
    ap.add_argument("--gate", action="store_true")
    ap.add_argument("--gate-backward", action="store_true")
    ap.add_argument("--boundary", choices=["cyclic", "linear"], default="cyclic")
    ap.add_argument("--graph", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the benchmark runs on one GPU "
              "(the path shards over batch and channels with no exchange between GPUs)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2509_24093_amd as P
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration()
        return

    if args.graph:
        bench_graph(args)
        return
    w = W.WORKLOADS[args.workload]
    B, N, L, C = w["B"], w["N"], w["L"], w["C"]
    K = (L + 1) ** 2
    log(f"[bench] generating {args.workload} inputs B={B} N={N} L={L} C={C}")
    q, k = W.make(args.workload)
    if args.bf16:
        qd = torch.from_numpy(W.to_bf16_bits(q).view(np.int16)).cuda().view(torch.bfloat16)
        kd = torch.from_numpy(W.to_bf16_bits(k).view(np.int16)).cuda().view(torch.bfloat16)
        esize = 2
    else:
        qd = torch.from_numpy(q).cuda()
        kd = torch.from_numpy(k).cuda()
        esize = 4
    out = torch.empty_like(qd)
    plan = P.Plan(B, N, L, C, boundary=args.boundary)
    if args.mixed:
        bench_mixed(args, plan, q, k, qd, kd, out, B, N, L, C)
        return
    if args.interchannel:
        bench_interchannel(args, plan, q, k, qd, kd, B, N, L, C)
        return
    if args.backward:
        bench_backward(args, plan, q, k, qd, kd, B, N, L, C)
        return
    if args.gate:
        bench_gate(args, plan, q, k, qd, kd, out, B, N, L, C)
        return
    if args.gate_backward:
        bench_gate_backward(args, plan, q, k, qd, kd, B, N, L, C)
        return
    n_paths, nnz_real, ws_bytes = plan.info()
    nnz, n_products = plan.contraction_info()
    log(f"[bench] plan: paths={n_paths} nnz={nnz_real} real / {nnz} complex-basis, products={n_products} "
        f"workspace={ws_bytes / 2**30:.2f} GiB")

    log(f"[bench] timing {args.steps} steps")
    ms, stage_avg, timing = _timed(args, lambda: plan(qd, kd, out), plan)
    tokens = B * N
    S = B * N * K * C * esize                     # one feature tensor in bytes
    # bytes each kernel must move (inputs read + outputs written), fp32
    # spectra of the DFT length Nf (N, or 2N with the zero-padded boundary)
    Nf = dft_length(N, args.boundary)
    Sc = B * Nf * K * C * 4
    Cp = (C + 1) // 2
    Sp = B * Nf * K * Cp * 8
    if "cg_fused" in stage_avg:
        io = {"fft_fwd_1": 2 * S + 2 * Sc, "cg_fused": 2 * Sc + Sp, "fft_inv_2": Sp + S}
    elif "cg_small" in stage_avg:
        io = {"cg_small": 3 * S}
    elif Nf > 256:
        io = {"fft_fwd_1": 2 * S + 2 * Sc, "fft_fwd_2": 4 * Sc, "cg": 2 * Sc + Sp, "fft_inv_1": 2 * Sp,
              "fft_inv_2": Sp + S}
    else:
        io = {"fft_fwd": 2 * S + 2 * Sc, "cg": 2 * Sc + Sp, "fft_inv": Sp + S}
    stages = {s: {"ms": round(t, 4), "bytes": io.get(s), "gbs": round(io.get(s, 0) / (t * 1e-3) / 1e9, 1)}
              for s, t in stage_avg.items()}
    counters, traffic_src = committed_counters(args.workload) if not args.bf16 else (None, "bf16 run")
    if args.boundary != "cyclic":
        counters, traffic_src = None, "counters were taken with the cyclic boundary"
    roofline = cg_roofline(stage_avg, B, Nf, L, C, n_products, nnz,
                           counters["cg_hbm_bytes_per_launch"] if counters else None, traffic_src)
    hbm_alg_gbs = 3 * S / (ms * 1e-3) / 1e9
    ceiling = hbm_ceiling()
    copy_gbs = max(ceiling["copy_gbs"], ceiling["copy_nontemporal_gbs"], ceiling["torch_copy_gbs"])
    log(f"[bench] HBM ceiling (1 GiB): copy {ceiling['copy_gbs']:.0f}, nontemporal copy "
        f"{ceiling['copy_nontemporal_gbs']:.0f}, read {ceiling['read_gbs']:.0f}, write {ceiling['write_gbs']:.0f}, "
        f"torch copy {ceiling['torch_copy_gbs']:.0f} GB/s")
    for st in stages.values():
        st["frac_of_copy"] = round(st["gbs"] / copy_gbs, 4) if st.get("bytes") else None
    result = {
        "metric": METRIC if args.boundary == "cyclic" else METRIC_LINEAR,
        "value": tokens / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16-storage/f32" if args.bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": B, "N": N, "L_max": L, "C": C, "boundary": args.boundary,
                   "parallelism": "single GPU"},
        "hbm": {"algorithmic_bytes_per_step": 3 * S, "achieved_gbs": round(hbm_alg_gbs, 1),
                "peak_gbs": HBM_PEAK_GBS, "frac": round(hbm_alg_gbs / HBM_PEAK_GBS, 4),
                "counter_bytes_per_step": counters["step_hbm_bytes"] if counters else None,
                "counter_gbs": round(counters["step_hbm_bytes"] / (ms * 1e-3) / 1e9, 1) if counters else None,
                "counter_frac": round(counters["step_hbm_bytes"] / (ms * 1e-3) / (HBM_PEAK_GBS * 1e9), 4)
                if counters else None,
                "copy_measured_gbs": round(copy_gbs, 1), "ceiling": ceiling,
                "frac_of_copy": round(hbm_alg_gbs / copy_gbs, 4),
                "counter_frac_of_copy": round(counters["step_hbm_bytes"] / (ms * 1e-3) / 1e9 / copy_gbs, 4)
                if counters else None},
        "roofline": roofline,
        "stages": stages,
        "timing": timing,
    }
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle baseline (~{args.cpu_seconds:.0f} s)")
        got = out.float().cpu().numpy() if args.bf16 else out.cpu().numpy()
        if args.bf16:
            q = W.bf16_bits_to_f32(W.to_bf16_bits(q))
            k = W.bf16_bits_to_f32(W.to_bf16_bits(k))
        obj, parity, R = cpu_baseline(q, k, L, args.cpu_seconds, got, linear=args.boundary == "linear")
        result["cpu_baseline"] = obj
        result["parity_rel_l2_sampled_rows"] = parity
        log(f"[bench] parity on {R} rows: rel_l2 = {parity:.3e}")
        if args.boundary == "cyclic":
            log(f"[bench] CPU oracle FFT mode (at most ~{args.cpu_seconds:.0f} s)")
            fobj, fpar, whole = cpu_fft_baseline(q, k, L, args.cpu_seconds, got)
            result["cpu_fft_baseline"] = fobj
            result["parity_rel_l2_whole_tensor" if whole else "parity_rel_l2_fft_channels"] = fpar
            log(f"[bench] parity on {'the whole tensor' if whole else 'whole channels'}: rel_l2 = {fpar:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


def bench_mixed(args, plan, q, k, qd, kd, out, B, N, L, C):
    """cgconv_forward_mixed on the same inputs with weights W_p ~ N(0, 1/C)."""
    import numpy as np
    import torch

    import paper_2509_24093_amd as P
    paths = [tuple(int(x) for x in row) for row in P.cgconv_paths(L)]
    n_paths = len(paths)
    wts = (np.random.default_rng(2025).normal(size=(n_paths, C, C)) / np.sqrt(C)).astype(np.float32)
    wd = torch.from_numpy(wts).cuda()
    log(f"[bench] timing {args.steps} mixed steps")
    ms, stage_avg, timing = _timed(args, lambda: plan.forward_mixed(qd, kd, wd, out), plan)
    mix_ms = stage_avg["cg_mix"]
    F = N // 2 + 1
    pts = B * F
    outs = int(sum(2 * J + 1 for _, _, J in paths))          # per-path outputs (J, M) per channel
    mix_flops = 4 * outs * C * C * pts                        # real W x complex T, multiply-add
    pair_tiles = sum(J + 1 for _, _, J in paths)               # tile passes per 8 points
    mfma_flops = 6 * 32 * 32 * 16 * 2 * pair_tiles * ((pts + 7) // 8)  # bf16 MFMAs executed
    achieved = mfma_flops / (mix_ms * 1e-3) / 1e12
    result = {
        "timing": timing,
        "metric": METRIC_MIXED,
        "value": B * N / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (mixing: bf16 hi/lo split on MFMA, fp32 accumulate)",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": B, "N": N, "L_max": L, "C": C, "boundary": args.boundary, "paths": n_paths,
                   "weights": "N(0, 1/C), seed 2025", "parallelism": "single GPU"},
        "roofline": {
            "kernel": f"cg_mix_kernel<{L}>",
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": None,
            "flops_per_launch": mfma_flops,
            "flop_model": (f"bf16 MFMA flops executed: 6 v_mfma_f32_32x32x16_bf16 (3 per 16 input channels, "
                           f"hi/lo split) per 32x32 tile pass, {pair_tiles} tile passes per 8 points, "
                           f"{(pts + 7) // 8} blocks of 8 points; the fp32-equivalent mixing work is "
                           f"4*{outs}*C^2 per point = {mix_flops} flops"),
            "mixing_tflops_fp32_equivalent": round(mix_flops / (mix_ms * 1e-3) / 1e12, 2),
            "launch_ms": round(mix_ms, 4),
        },
        "stages": {s: {"ms": round(t, 4)} for s, t in stage_avg.items()},
    }
    if not args.no_cpu_baseline and args.boundary != "cyclic":
        log("[bench] no CPU baseline for the mixed convolution with the zero-padded boundary")
    if not args.no_cpu_baseline and args.boundary == "cyclic":
        from oracle.mix import cgconv_mixed_direct_rows
        log(f"[bench] CPU oracle baseline, mixed (~{args.cpu_seconds:.0f} s)")
        got = out.cpu().numpy()
        rng = np.random.default_rng(2026)
        rows, ref = [], []
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_seconds or len(rows) < 2:
            part = [(int(rng.integers(0, B)), int(rng.integers(0, N)))]
            if not rows:
                part = [(0, 0)]
            ref.extend(cgconv_mixed_direct_rows(q, k, L, wts, part))
            rows.extend(part)
        dt = time.perf_counter() - t0
        num = sum(float(((got[b, i].astype(np.float64) - ref[n]) ** 2).sum()) for n, (b, i) in enumerate(rows))
        den = sum(float((r * r).sum()) for r in ref)
        cores = len(os.sched_getaffinity(0))
        result["cpu_baseline"] = {"value": len(rows) / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
                                  "sample": f"direct definition with per-path mixing on {len(rows)} sampled output "
                                            f"rows (b, i), fp64 numpy, {dt:.1f} s"}
        result["parity_rel_l2_sampled_rows"] = (num / den) ** 0.5
        log(f"[bench] mixed parity on {len(rows)} rows: rel_l2 = {result['parity_rel_l2_sampled_rows']:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


def bench_interchannel(args, plan, q, k, qd, kd, B, N, L, C):
    """cgconv_forward_interchannel with H heads of m = C/H channels, every
    channel pair of a head, reduced per degree to m_out = m channels by
    seeded weights ~ N(0, 1/m^2)."""
    import numpy as np
    import torch

    H = args.heads
    m = C // H
    mo = m
    wts = (np.random.default_rng(2031).normal(size=(H, L + 1, mo, m * m)) / m).astype(np.float32)
    wd = torch.from_numpy(wts).cuda()
    out = torch.empty((B, N, (L + 1) ** 2, H * mo), dtype=torch.float32, device="cuda")
    log(f"[bench] timing {args.steps} inter-channel steps (heads {H}, m {m}, m_out {mo})")
    ms, stage_avg, timing = _timed(args, lambda: plan.forward_interchannel(qd, kd, wd, heads=H, out=out), plan)
    nnz, n_products = plan.contraction_info()
    F = N // 2 + 1
    pts = B * F * H * 64                       # lanes: (point, pair slot); m*m of 64 slots carry pairs
    pair_pts = B * F * H * m * m
    cg_flops = pair_pts * (6 * n_products + 4 * nnz)
    mfma_flops = B * H * ((F + 3) // 4) * sum(2 * 16 * 16 * 64 * (1 if mu == 0 else 1) * (L + 1 - mu)
                                              for mu in range(L + 1))
    ims = stage_avg["cg_inter"]
    achieved = cg_flops / (ims * 1e-3) / 1e12
    result = _common(args, METRIC_INTER, ms, B, N, L, C, "f32 (reduction: fp32 MFMA)", timing)
    result["config"].update({"heads": H, "channels_per_head": m, "m_out": mo, "weights": "N(0, 1/m^2), seed 2031"})
    result["roofline"] = {
        "kernel": f"cg_inter_kernel<{L}>",
        "bound": "alu",
        "achieved": round(achieved, 2),
        "peak": round(VALU_PEAK_TFLOPS, 1),
        "unit": "TFLOP/s",
        "frac": round(achieved / VALU_PEAK_TFLOPS, 4),
        "traffic": None,
        "flops_per_launch": cg_flops,
        "flop_model": (f"(6*{n_products} distinct complex products + 4*{nnz} non-zeros) per (b, frequency 0..N/2, "
                       f"head, channel pair) point, {pair_pts} points; the per-degree reduction runs on the matrix "
                       f"cores: {mfma_flops} fp32 MFMA flops per launch (16x16x4, rows padded to 16)"),
        "reduction_mfma_tflops": round(mfma_flops / (ims * 1e-3) / 1e12, 2),
        "launch_ms": round(ims, 4),
    }
    result["stages"] = {s: {"ms": round(t, 4)} for s, t in stage_avg.items()}
    if not args.no_cpu_baseline and args.boundary == "cyclic":
        from oracle.conv import cgconv_direct_rows
        from oracle.inter import pair_channels, reduce_degrees
        log(f"[bench] CPU oracle baseline, inter-channel (~{args.cpu_seconds:.0f} s)")
        got = out.cpu().numpy()
        rng = np.random.default_rng(2032)
        rows, num, den = 0, 0.0, 0.0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_seconds or rows < 2:
            b, i = (0, 0) if rows == 0 else (int(rng.integers(0, B)), int(rng.integers(0, N)))
            qe, ke = pair_channels(q[b:b + 1], k[b:b + 1], H)
            u = cgconv_direct_rows(qe, ke, L, [(0, i)])          # (1, K, H m^2)
            ref = reduce_degrees(u[None], L, H, wts)[0, 0]      # (K, H m_out)
            d = got[b, i].astype(np.float64) - ref
            num += float((d * d).sum())
            den += float((ref * ref).sum())
            rows += 1
        dt = time.perf_counter() - t0
        cores = len(os.sched_getaffinity(0))
        result["cpu_baseline"] = {"value": rows / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
                                  "sample": f"direct definition over every channel pair with the per-degree "
                                            f"reduction, {rows} sampled output rows (b, i), fp64 numpy, {dt:.1f} s"}
        result["parity_rel_l2_sampled_rows"] = (num / den) ** 0.5
        log(f"[bench] inter-channel parity on {rows} rows: rel_l2 = {result['parity_rel_l2_sampled_rows']:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


def _common(args, metric, ms, B, N, L, C, dtype, timing=None):
    r = {"metric": metric, "value": B * N / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": dtype, "data": "synthetic",
            "config": {"workload": args.workload, "batch": B, "N": N, "L_max": L, "C": C, "boundary": args.boundary,
                       "parallelism": "single GPU"}}
    if timing is not None:
        r["timing"] = timing
    return r


def _timed(args, step, plan, calls_per_step=1):
    """Warm up, then time args.steps calls of step(), each between two HIP
    events on the current stream (the one the library enqueues on), with the
    plan's stage timing off; the host synchronises before and after the
    timed steps.  Then a separate pass of up to 20 steps with the stage
    timing on gives the per-kernel averages.  Returns (median ms per step,
    {stage: average ms per timed call}, timing record)."""
    import torch
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record()
        step()
        b.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    per_step = sorted(a.elapsed_time(b) for a, b in ev)
    ms = per_step[len(per_step) // 2] if len(per_step) % 2 else 0.5 * (per_step[len(per_step) // 2 - 1] +
                                                                          per_step[len(per_step) // 2])
    n_stage = min(args.steps, 20)
    plan.enable_timing(n_stage * calls_per_step)
    for _ in range(n_stage):
        step()
    stage_ms, ncalls = plan.stage_times()
    plan.enable_timing(0)
    rec = {"method": f"HIP events around each of the {args.steps} timed steps on the stream the kernels run on; "
                     f"median; stage times from a separate pass of {n_stage} steps",
           "median_ms": round(ms, 4), "min_ms": round(per_step[0], 4), "max_ms": round(per_step[-1], 4),
           "wall_ms_per_step": round(wall_ms, 4)}
    return ms, {s: v / max(ncalls, 1) for s, v in stage_ms.items()}, rec


def bench_backward(args, plan, q, k, qd, kd, B, N, L, C):
    """cgconv_backward (both gradients) for a seeded output gradient ~ N(0, 1).
    Each gradient is one forward-shaped pipeline on the same kernels, so the
    stage times are averages over the 2 * steps pipelines."""
    import numpy as np
    import torch

    import paper_2509_24093_amd as P
    g = np.random.default_rng(2027).normal(size=q.shape).astype(np.float32)
    gd = torch.from_numpy(g).cuda()
    gq, gk = torch.empty_like(qd), torch.empty_like(qd)
    stream = torch.cuda.current_stream().cuda_stream

    def step():
        P.cgconv_backward(plan._h, qd.data_ptr(), kd.data_ptr(), gd.data_ptr(), gq.data_ptr(), gk.data_ptr(),
                          stream)
    log(f"[bench] timing {args.steps} backward steps")
    ms, stage_avg, timing = _timed(args, step, plan, calls_per_step=2)
    nnz, n_products = plan.contraction_info()
    counters, src = committed_counters(args.workload)
    if args.boundary != "cyclic":
        counters, src = None, "counters were taken with the cyclic boundary"
    roofline = cg_roofline(stage_avg, B, dft_length(N, args.boundary), L, C, n_products, nnz,
                           counters["cg_hbm_bytes_per_launch"] if counters else None,
                           (src + "; taken on the forward, same kernel and launch shape") if counters else src)
    result = _common(args, METRIC_BACKWARD, ms, B, N, L, C, "f32", timing)
    result["roofline"] = roofline
    result["stages_per_gradient"] = {s: {"ms": round(t, 4)} for s, t in stage_avg.items()}
    if not args.no_cpu_baseline:
        from oracle.backward import backward_direct_rows
        log(f"[bench] CPU oracle baseline, backward (~{args.cpu_seconds:.0f} s)")
        got = {"q": gq.cpu().numpy(), "k": gk.cpu().numpy()}
        rng = np.random.default_rng(2028)
        rows, num, den = [], 0.0, 0.0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_seconds or len(rows) < 2:
            b = len(rows) % B
            part = [(b, 0 if not rows else int(rng.integers(0, N)))]
            for wrt in ("q", "k"):
                ref = backward_direct_rows(q, k, g, L, part, wrt, boundary=args.boundary)[0]
                d = got[wrt][part[0]].astype(np.float64) - ref
                num += float((d * d).sum())
                den += float((ref * ref).sum())
            rows.extend(part)
        dt = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": len(rows) / dt, "unit": "tokens/s", "cores": len(os.sched_getaffinity(0)),
                                  "kind": "oracle",
                                  "sample": f"direct sums of both gradients on {len(rows)} sampled rows (b, j), "
                                            f"all components and channels, fp64 numpy, {dt:.1f} s"}
        result["parity_rel_l2_sampled_rows"] = (num / den) ** 0.5
        log(f"[bench] backward parity on {len(rows)} rows: rel_l2 = {result['parity_rel_l2_sampled_rows']:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


def bench_gate(args, plan, q, k, qd, kd, out, B, N, L, C):
    """cgconv_gate_value with u = q and v = k of the workload."""
    import numpy as np

    import paper_2509_24093_amd as P
    log(f"[bench] timing {args.steps} gating steps")
    ms, stage_avg, timing = _timed(args, lambda: plan.gate_value(qd, kd, out), plan)
    K = (L + 1) ** 2
    _, coef = P.cgconv_cg_table(L)
    nnz_real = len(coef)
    lanes = B * N * C
    per_lane = K * K + 2 * nnz_real + 3 * K
    flops = per_lane * lanes
    gv_ms = stage_avg["gate_value"]
    achieved = flops / (gv_ms * 1e-3) / 1e12
    result = _common(args, METRIC_GATE, ms, B, N, L, C, "f32", timing)
    result["roofline"] = {
        "kernel": f"gate_value_kernel<{L}>",
        "bound": "alu",
        "achieved": round(achieved, 2),
        "peak": round(VALU_PEAK_TFLOPS, 1),
        "unit": "TFLOP/s",
        "frac": round(achieved / VALU_PEAK_TFLOPS, 4),
        "traffic": None,
        "flops_per_launch": flops,
        "flop_model": (f"per (b, i, c) lane: {K}^2 products u_x v_y + 2 flops (multiply-add by the "
                       f"coefficient) per real-basis non-zero ({nnz_real}) + 3K for the norms and the gate; "
                       f"{lanes} lanes"),
        "algorithmic_bytes_per_launch": 3 * K * 4 * lanes,
        "achieved_gbs": round(3 * K * 4 * lanes / (gv_ms * 1e-3) / 1e9, 1),
        "launch_ms": round(gv_ms, 4),
    }
    result["stages"] = {s: {"ms": round(t, 4)} for s, t in stage_avg.items()}
    if not args.no_cpu_baseline:
        from oracle.gate import gate_value
        log(f"[bench] CPU oracle baseline, gating (~{args.cpu_seconds:.0f} s)")
        got = out.cpu().numpy()
        num = den = 0.0
        chans = []
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_seconds and len(chans) < C:
            c = len(chans)
            ref = gate_value(q[0:1, :, :, c:c + 1], k[0:1, :, :, c:c + 1], L)
            d = got[0:1, :, :, c:c + 1].astype(np.float64) - ref
            num += float((d * d).sum())
            den += float((ref * ref).sum())
            chans.append(c)
        dt = time.perf_counter() - t0
        tokens = N * len(chans) / C
        result["cpu_baseline"] = {"value": tokens / dt, "unit": "tokens/s", "cores": len(os.sched_getaffinity(0)),
                                  "kind": "oracle",
                                  "sample": f"batch element 0, all {N} tokens, channels 0..{len(chans) - 1} of {C} "
                                            f"({tokens:.0f} token-equivalents), fp64 numpy, {dt:.1f} s"}
        result["parity_rel_l2_sampled_channels"] = (num / den) ** 0.5
        log(f"[bench] gating parity on {len(chans)} channels: rel_l2 = {result['parity_rel_l2_sampled_channels']:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


def bench_gate_backward(args, plan, q, k, qd, kd, B, N, L, C):
    """cgconv_gate_value_backward (grad_u and grad_v) with u = q, v = k of
    the workload and a seeded upstream gradient ~ N(0, 1)."""
    import numpy as np
    import torch

    import paper_2509_24093_amd as P
    g = np.random.default_rng(2029).normal(size=q.shape).astype(np.float32)
    gd = torch.from_numpy(g).cuda()
    gu, gv = torch.empty_like(qd), torch.empty_like(qd)
    stream = torch.cuda.current_stream().cuda_stream

    def step():
        P.cgconv_gate_value_backward(plan._h, qd.data_ptr(), kd.data_ptr(), gd.data_ptr(), gu.data_ptr(),
                                     gv.data_ptr(), stream)
    log(f"[bench] timing {args.steps} gating backward steps")
    ms, stage_avg, timing = _timed(args, step, plan)
    K = (L + 1) ** 2
    _, coef = P.cgconv_cg_table(L)
    nnz_real = len(coef)
    lanes = B * N * C
    per_lane = 2 * (K * K + 2 * nnz_real) + 8 * K
    flops = per_lane * lanes
    bw_ms = stage_avg["gate_bwd"]
    achieved = flops / (bw_ms * 1e-3) / 1e12
    result = _common(args, METRIC_GATE_BACKWARD, ms, B, N, L, C, "f32", timing)
    result["roofline"] = {
        "kernel": f"gate_bwd_kernel<{L}, false> + gate_bwd_kernel<{L}, true> (one launch per gradient)",
        "bound": "alu",
        "achieved": round(achieved, 2),
        "peak": round(VALU_PEAK_TFLOPS, 1),
        "unit": "TFLOP/s",
        "frac": round(achieved / VALU_PEAK_TFLOPS, 4),
        "traffic": None,
        "flops_per_launch": flops,
        "flop_model": (f"per (b, i, c) lane: two real-basis tensor products (one per gradient), each {K}^2 "
                       f"products + 2 flops per non-zero ({nnz_real}), + 8K for the scales, the gate and "
                       f"its sums; {lanes} lanes"),
        "algorithmic_bytes_per_launch": 5 * K * 4 * lanes,
        "achieved_gbs": round(5 * K * 4 * lanes / (bw_ms * 1e-3) / 1e9, 1),
        "launch_ms": round(bw_ms, 4),
    }
    result["stages"] = {s: {"ms": round(t, 4)} for s, t in stage_avg.items()}
    if not args.no_cpu_baseline:
        from oracle.gate import gate_value_backward
        log(f"[bench] CPU oracle baseline, gating backward (~{args.cpu_seconds:.0f} s)")
        got = {"u": gu.cpu().numpy(), "v": gv.cpu().numpy()}
        num = den = 0.0
        chans = []
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_seconds and len(chans) < C:
            c = len(chans)
            sl = (slice(0, 1), slice(None), slice(None), slice(c, c + 1))
            ru, rv = gate_value_backward(q[sl], k[sl], g[sl], L)
            for name, ref in (("u", ru), ("v", rv)):
                d = got[name][sl].astype(np.float64) - ref
                num += float((d * d).sum())
                den += float((ref * ref).sum())
            chans.append(c)
        dt = time.perf_counter() - t0
        tokens = N * len(chans) / C
        result["cpu_baseline"] = {"value": tokens / dt, "unit": "tokens/s", "cores": len(os.sched_getaffinity(0)),
                                  "kind": "oracle",
                                  "sample": f"both gradients, batch element 0, all {N} tokens, channels "
                                            f"0..{len(chans) - 1} of {C} ({tokens:.0f} token-equivalents), "
                                            f"fp64 numpy, {dt:.1f} s"}
        result["parity_rel_l2_sampled_channels"] = (num / den) ** 0.5
        log(f"[bench] gating backward parity on {len(chans)} channels: "
            f"rel_l2 = {result['parity_rel_l2_sampled_channels']:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


def bench_graph(args):
    """cgconv_forward_graph on the graph workload: per sample the normalised
    Laplacian eigenbasis of the 16-nearest-neighbour graph of its points."""
    import numpy as np
    import torch

    import paper_2509_24093_amd as P
    import workloads as W
    w = W.WORKLOADS["graph"]
    B, N, L, C = w["B"], w["N"], w["L"], w["C"]
    log(f"[bench] generating the graph workload B={B} N={N} L={L} C={C} (Laplacian eigenbases on the host)")
    q, k, U = W.graph_pointcloud(B, N, L, C, w["seed"])
    qd, kd, Ud = (torch.from_numpy(a).cuda() for a in (q, k, U))
    plan = P.GraphPlan(B, N, L, C)
    out = torch.empty_like(qd)
    log(f"[bench] timing {args.steps} graph steps")
    ms, stage_avg, timing = _timed(args, lambda: plan(Ud, qd, kd, out), plan)
    K = (L + 1) ** 2
    Kp = -(-N // 32) * 32
    Mp = -(-N // 128) * 128
    KCp = -(-(K * C) // 128) * 128
    mfma_flops = 3 * 2 * Mp * (2 * KCp) * Kp * B       # executed bf16 MFMA work of the forward transform
    fp32_equiv = 2 * N * N * (2 * K * C) * B             # the transform itself
    gm = stage_avg["gft_gemm_fwd"]
    achieved = mfma_flops / (gm * 1e-3) / 1e12
    result = _common(args, METRIC_GRAPH, ms, B, N, L, C, "f32 (transforms: bf16 hi/lo split on MFMA, fp32 accumulate)", timing)
    result["config"] = {"workload": "graph", "batch": B, "N": N, "L_max": L, "C": C,
                        "basis": "normalised Laplacian eigenvectors of the 16-NN graph", "parallelism": "single GPU"}
    result["roofline"] = {
        "kernel": "gft_gemm_kernel (forward transform)",
        "bound": "mfma",
        "achieved": round(achieved, 2),
        "peak": MFMA_BF16_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
        "traffic": None,
        "flops_per_launch": mfma_flops,
        "flop_model": (f"bf16 MFMA flops executed: 3 products (hi*hi, hi*lo, lo*hi) x 2 x Mp={Mp} x Np={2 * KCp} "
                       f"x Kp={Kp} per batch element, {B} elements; the transform itself is "
                       f"2*N^2*2KC*B = {fp32_equiv} fp32 flops"),
        "transform_tflops_fp32_equivalent": round(fp32_equiv / (gm * 1e-3) / 1e12, 2),
        "launch_ms": round(gm, 4),
    }
    result["stages"] = {s: {"ms": round(t, 4)} for s, t in stage_avg.items()}
    if not args.no_cpu_baseline:
        from oracle.gft import gft_cgconv
        log(f"[bench] CPU oracle baseline, graph (~{args.cpu_seconds:.0f} s)")
        got = out.cpu().numpy()
        num = den = 0.0
        chans = []
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_seconds and len(chans) < C:
            c = len(chans)
            ref = gft_cgconv(U[0:1], q[0:1, :, :, c:c + 1], k[0:1, :, :, c:c + 1], L)
            d = got[0:1, :, :, c:c + 1].astype(np.float64) - ref
            num += float((d * d).sum())
            den += float((ref * ref).sum())
            chans.append(c)
        dt = time.perf_counter() - t0
        tokens = N * len(chans) / C
        result["cpu_baseline"] = {"value": tokens / dt, "unit": "tokens/s", "cores": len(os.sched_getaffinity(0)),
                                  "kind": "oracle",
                                  "sample": f"batch element 0, all {N} nodes, channels 0..{len(chans) - 1} of {C} "
                                            f"({tokens:.0f} token-equivalents), fp64 numpy, {dt:.1f} s"}
        result["parity_rel_l2_sampled_channels"] = (num / den) ** 0.5
        log(f"[bench] graph parity on {len(chans)} channels: rel_l2 = {result['parity_rel_l2_sampled_channels']:.3e}")
    else:
        result["cpu_baseline"] = None
    plan.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
