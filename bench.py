"""Benchmark: MXNorm + MXFP8 cast throughput on one MI355X.

A step is one forward pass of the fused MXNorm kernel (block absmax, row RMS
estimate, E8M0 scales, E4M3 codes -- Algorithm 2) over the Llama-3-8B-shaped
activation tensor x bf16 [32768, 4096] (seeded N(0,1) with 1% outlier
channels).  The value is algorithmic HBM bytes per step (2 B read + 1 B code
+ 1/32 B scale per element, + 4 B of rho per row) divided by the measured
step time.  Alongside, on the same inputs: the hand-written RMSNorm + MXFP8
cast baseline (gain-free, as in the paper's kernel benchmark, and with gain),
the NVFP4 variants, a device-to-device copy for reference, and the CPU oracle
on a bounded sample.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
Prints one JSON line.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
WORKLOAD = "llama3-8b-d4096"
NV_WORKLOAD = "llama3-8b-d4096-nvfp4"
ROTATE_MIN_BYTES = 768 << 20       # > 3x the 256 MiB Infinity Cache
# the norm/cast kernel body and its launch configuration
KERNEL_SRC = [os.path.join(ROOT, "paper_2603_13180_amd", "csrc", f)
              for f in ("norm_cast.h", "mxnorm.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_mxnorm_mxfp8_llama3-8b-d4096.txt")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=300,
                    help="untimed launches first: the device takes about 200 back-to-back "
                         "launches (~13 ms) to settle to its sustained rate")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--sweep", metavar="OUT_JSON",
                    help="instead of the headline line, run the paper's kernel sweep "
                         "(17 hidden sizes x 5 token counts) and write per-shape results")
    ap.add_argument("--layer", metavar="OUT_JSON",
                    help="instead of the headline line, run the MXNormLinear layer benchmark "
                         "(norm + MX matmul at Llama-3-8B projection shapes) and write results")
    ap.add_argument("--backward", metavar="OUT_JSON",
                    help="instead of the headline line, time the MXNormLinear backward "
                         "(casts, STE, both matmuls) at Llama-3-8B projection shapes")
    ap.add_argument("--sweep-formats",
                    default="e4m3-b32,nvfp4,e4m3-b16,e4m3-b64,e2m1-b16,e2m1-b32,e2m1-b64",
                    help="comma list of e4m3-b{16,32,64}, e2m1-b{16,32,64}, nvfp4")
    return ap.parse_args()


# the paper's kernel-benchmark grid (appendix "Performance Benchmark Details"):
# hidden sizes k * 2^r, k in {1, 3, 5, 7}, within [2^10, 2^14]; tokens 2^12 .. 2^16
SWEEP_D = sorted({k * 2 ** r for k in (1, 3, 5, 7) for r in range(15)
                  if 1024 <= k * 2 ** r <= 16384})
SWEEP_T = [4096, 8192, 16384, 32768, 65536]


def graph_time(launch, n_sets, reps, rounds, stream):
    """ms per launch of `launch(i)` for i in 0..n_sets-1, captured once as a
    HIP graph and replayed `reps` times per round; median over rounds."""
    import numpy as np
    import torch
    for i in range(n_sets):
        launch(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for i in range(n_sets):
            launch(i)
    out = []
    with torch.cuda.stream(stream):   # replays and events on one stream
        g.replay()
        torch.cuda.synchronize()
        for _ in range(rounds):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(reps):
                g.replay()
            b.record(stream)
            torch.cuda.synchronize()
            out.append(a.elapsed_time(b) / (reps * n_sets))
    del g
    return float(np.median(out))


def run_sweep(path, formats):
    """Per-shape MXNorm and RMSNorm+cast (both gain-free, as in the paper's
    kernel benchmark) times and the geometric-mean speedup per format."""
    import math
    import numpy as np
    import torch
    from paper_2603_13180_amd import mxnorm

    dev = torch.device("cuda:0")
    mxnorm.load()
    stream = torch.cuda.Stream(dev)
    gen = torch.Generator(device=dev)
    results = []
    summary = {}
    for fmt in formats:
        speedups = []
        for d in SWEEP_D:
            for T in SWEEP_T:
                gen.manual_seed(d * 100003 + T)
                xbytes = T * d * 2
                n_sets = max(2, -(-ROTATE_MIN_BYTES // xbytes))
                x = torch.randn(n_sets, T, d, generator=gen, device=dev).to(torch.bfloat16)
                if fmt == "nvfp4":
                    codes = torch.empty(n_sets, T, d // 2, dtype=torch.uint8, device=dev)
                    scales = torch.empty(n_sets, T, d // 16, dtype=torch.uint8, device=dev)
                    nbytes = nvfp4_bytes(T, d) - 4 * T
                    sg = mxnorm.mxnorm_default_global_scale(d, 16, 2)
                    sr = mxnorm.rmsnorm_default_global_scale(d, 1.0)
                    mx = lambda i: mxnorm.mxnorm_nvfp4_fwd(x[i], sg, codes=codes[i], scales=scales[i],
                                                          want_rho=False)
                    rm = lambda i: mxnorm.rmsnorm_nvfp4_fwd(x[i], None, sr, codes=codes[i],
                                                           scales=scales[i], want_rho=False)
                else:
                    # "<elem>-b<block>": E8M0 scales per block, E4M3 or E2M1 codes
                    elem, blk = fmt.split("-b")
                    blk = int(blk)
                    cw = d if elem == "e4m3" else d // 2
                    codes = torch.empty(n_sets, T, cw, dtype=torch.uint8, device=dev)
                    scales = torch.empty(n_sets, T, d // blk, dtype=torch.uint8, device=dev)
                    nbytes = T * d * 2 + T * cw + T * (d // blk)
                    mx = lambda i: mxnorm.mxnorm_mx_fwd(x[i], blk, elem, codes=codes[i],
                                                       scales=scales[i], want_rho=False)
                    rm = lambda i: mxnorm.rmsnorm_mx_fwd(x[i], None, blk, elem, codes=codes[i],
                                                        scales=scales[i], want_rho=False)
                # about 20 ms of device time per round
                est_ms = nbytes / 5.0e12 * 1e3
                reps = max(2, int(20.0 / max(est_ms * n_sets, 1e-3)))
                t_mx, t_rm = [], []
                for _ in range(3):    # interleave the two kernels
                    t_mx.append(graph_time(mx, n_sets, reps, 1, stream))
                    t_rm.append(graph_time(rm, n_sets, reps, 1, stream))
                m, r = float(np.median(t_mx)), float(np.median(t_rm))
                speedups.append(r / m)
                results.append({"format": fmt, "d": d, "tokens": T, "mxnorm_us": round(m * 1e3, 3),
                                "rmsnorm_us": round(r * 1e3, 3), "speedup": round(r / m, 4),
                                "mxnorm_GBps": round(nbytes / (m * 1e-3) / 1e9, 1),
                                "rmsnorm_GBps": round(nbytes / (r * 1e-3) / 1e9, 1)})
                print(json.dumps(results[-1]), file=sys.stderr, flush=True)
                del x, codes, scales
                torch.cuda.empty_cache()
        summary[fmt] = {
            "geomean_speedup": round(math.exp(sum(math.log(v) for v in speedups) / len(speedups)), 4),
            "min_speedup": round(min(speedups), 4), "max_speedup": round(max(speedups), 4),
            "shapes": len(speedups)}
    doc = {"method": "HIP-graph replays of one launch per rotating buffer set (>= 768 MiB of "
                     "input in rotation), median of 3 interleaved rounds; gain-free kernels, "
                     "N(0,1) bf16 inputs drawn on the GPU (seeded); bytes = algorithmic bytes",
           "hidden": SWEEP_D, "tokens": SWEEP_T, "summary": summary, "results": results}
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
    print(json.dumps({"sweep": path, "summary": summary}))


# MI355X dense matrix-core peaks (TFLOP/s) for the MX matmul's element types
PEAK_MFMA_TFLOPS = {"e4m3": 5000.0, "e2m1": 10100.0}
LAYER_D = 4096                       # Llama-3-8B hidden size
LAYER_N = {"qkv": 6144, "gate_up": 28672}   # projections that follow a norm
LAYER_T = [4096, 8192, 16384, 32768, 65536]


def layer_case(fmt, T, N, stream, gen, rounds=3, budget_ms=40.0):
    """One MXNormLinear shape: MXNorm -> MX matmul against RMSNorm (gain) +
    MX cast -> the same matmul, each pair captured as one graph and timed in
    interleaved rounds.  Returns a result dict."""
    import numpy as np
    import torch
    from paper_2603_13180_amd import mxnorm

    dev = torch.device("cuda:0")
    d = LAYER_D
    x = torch.randn(T, d, generator=gen, device=dev).to(torch.bfloat16)
    w = (0.02 * torch.randn(N, d, generator=gen, device=dev)).to(torch.bfloat16)
    gam = (1.0 + 0.1 * torch.randn(d, generator=gen, device=dev)).to(torch.bfloat16)
    wc_g, ws_g = mxnorm.mx_cast_fwd(w, gam, block=32, elem=fmt)   # MXCast(W gamma)
    wc, ws = mxnorm.mx_cast_fwd(w, None, block=32, elem=fmt)      # MXCast(W)
    cw = d if fmt == "e4m3" else d // 2
    codes = torch.empty(T, cw, dtype=torch.uint8, device=dev)
    scales = torch.empty(T, d // 32, dtype=torch.uint8, device=dev)
    out = torch.empty(T, N, dtype=torch.bfloat16, device=dev)

    def mx_layer(_):
        mxnorm.mxnorm_mx_fwd(x, 32, fmt, codes=codes, scales=scales, want_rho=False)
        mxnorm.mx_matmul_fwd(codes, scales, wc_g, ws_g, d, elem=fmt, out_dtype=torch.bfloat16,
                             out=out)

    def rms_layer(_):
        mxnorm.rmsnorm_mx_fwd(x, gam, 32, fmt, codes=codes, scales=scales, want_rho=False)
        mxnorm.mx_matmul_fwd(codes, scales, wc, ws, d, elem=fmt, out_dtype=torch.bfloat16,
                             out=out)

    def gemm(_):
        mxnorm.mx_matmul_fwd(codes, scales, wc, ws, d, elem=fmt, out_dtype=torch.bfloat16,
                             out=out)

    def mx_norm(_):
        mxnorm.mxnorm_mx_fwd(x, 32, fmt, codes=codes, scales=scales, want_rho=False)

    def rms_norm(_):
        mxnorm.rmsnorm_mx_fwd(x, gam, 32, fmt, codes=codes, scales=scales, want_rho=False)

    flops = 2.0 * T * N * d
    est_ms = flops / 1.5e15 * 1e3
    reps = max(2, int(budget_ms / est_ms))
    t = {k: [] for k in ("mx", "rms", "gemm", "mx_norm", "rms_norm")}
    for _ in range(rounds):
        t["mx"].append(graph_time(mx_layer, 1, reps, 1, stream))
        t["rms"].append(graph_time(rms_layer, 1, reps, 1, stream))
        t["gemm"].append(graph_time(gemm, 1, reps, 1, stream))
        t["mx_norm"].append(graph_time(mx_norm, 1, 4 * reps, 1, stream))
        t["rms_norm"].append(graph_time(rms_norm, 1, 4 * reps, 1, stream))
    m = {k: float(np.median(v)) for k, v in t.items()}
    tf = flops / (m["gemm"] * 1e-3) / 1e12
    del x, w, codes, scales, out, wc, ws, wc_g, ws_g
    torch.cuda.empty_cache()
    return {"format": fmt, "tokens": T, "N": N, "d": d,
            "mxnorm_linear_us": round(m["mx"] * 1e3, 2),
            "rmsnorm_cast_linear_us": round(m["rms"] * 1e3, 2),
            "layer_speedup": round(m["rms"] / m["mx"], 4),
            # the matmul is common to both layers: the same ratio from the
            # separately timed parts, free of the matmul's run-to-run noise
            "layer_speedup_from_parts":
                round((m["rms_norm"] + m["gemm"]) / (m["mx_norm"] + m["gemm"]), 4),
            "matmul_us": round(m["gemm"] * 1e3, 2),
            "matmul_TFLOPs": round(tf, 1),
            "matmul_frac_of_peak": round(tf / PEAK_MFMA_TFLOPS[fmt], 4),
            "mxnorm_us": round(m["mx_norm"] * 1e3, 2),
            "rmsnorm_gamma_cast_us": round(m["rms_norm"] * 1e3, 2)}


def run_layer(path):
    """The MXNormLinear forward at the Llama-3-8B projections that consume a
    norm (QKV and gate+up, d = 4096) over the paper's token counts, MXFP8 and
    MXFP4 (E8M0 scales, 32-element blocks)."""
    import math
    import torch
    from paper_2603_13180_amd import mxnorm

    mxnorm.load()
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(dev)
    gen = torch.Generator(device=dev)
    results, summary = [], {}
    for fmt in ("e4m3", "e2m1"):
        sp, spp = [], []
        for name, N in LAYER_N.items():
            for T in LAYER_T:
                gen.manual_seed(T * 31 + N)
                r = layer_case(fmt, T, N, stream, gen)
                r["projection"] = name
                results.append(r)
                sp.append(r["layer_speedup"])
                spp.append(r["layer_speedup_from_parts"])
                print(json.dumps(r), file=sys.stderr, flush=True)
        gm = lambda v: round(math.exp(sum(math.log(u) for u in v) / len(v)), 4)
        summary[fmt] = {"geomean_layer_speedup": gm(sp), "min": min(sp), "max": max(sp),
                        "geomean_layer_speedup_from_parts": gm(spp), "shapes": len(sp)}
    doc = {"method": "each layer variant (norm kernel + MX matmul, bf16 output) captured as a "
                     "HIP graph, replayed ~40 ms per round, median of 3 interleaved rounds; "
                     "RMSNorm path applies the gain and multiplies MXCast(W), the MXNorm path "
                     "multiplies MXCast(W gamma); N(0,1) activations, 0.02 N(0,1) weights",
           "summary": summary, "results": results}
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
    print(json.dumps({"layer": path, "summary": summary}))


def ste_bytes(T, d):
    """Algorithmic bytes of one STE launch: x, grad_Z read and grad_x (bf16)
    written per element, rho per row, gamma read and grad_gamma written once."""
    return T * d * 6 + 4 * T + 2 * d + 4 * d


def cast_t_bytes(T, d):
    """Algorithmic bytes of the column cast of rho~ X to MXFP8."""
    return T * d * 2 + T * d + T * d // 32 + 4 * T


def backward_case(fmt, T, N, stream, gen, rounds=3, budget_ms=40.0):
    """The MXNormLinear backward at one shape: every stage captured alone and
    the whole chain captured as one graph, medians of interleaved rounds."""
    import numpy as np
    import torch
    from paper_2603_13180_amd import mxnorm

    dev = torch.device("cuda:0")
    d = LAYER_D
    x = torch.randn(T, d, generator=gen, device=dev).to(torch.bfloat16)
    w = (0.02 * torch.randn(N, d, generator=gen, device=dev)).to(torch.bfloat16)
    gam = (1.0 + 0.1 * torch.randn(d, generator=gen, device=dev)).to(torch.bfloat16)
    gh = (0.01 * torch.randn(T, N, generator=gen, device=dev)).to(torch.bfloat16)
    _, _, rho = mxnorm.mxnorm_mx_fwd(x, 32, fmt)
    cw = lambda n: n if fmt == "e4m3" else n // 2
    u8 = lambda *shape: torch.empty(*shape, dtype=torch.uint8, device=dev)
    gh_c, gh_s = u8(T, cw(N)), u8(T, N // 32)
    wt_c, wt_s = u8(d, cw(N)), u8(d, N // 32)
    ght_c, ght_s = u8(N, cw(T)), u8(N, T // 32)
    xt_c, xt_s = u8(d, cw(T)), u8(d, T // 32)
    gz = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    gx = torch.empty(T, d, dtype=torch.bfloat16, device=dev)
    gg = torch.empty(d, dtype=torch.float32, device=dev)
    gw = torch.empty(N, d, dtype=torch.float32, device=dev)
    ws = u8(max(16, mxnorm.load().mxnorm_ste_bwd_workspace_bytes(T, d)))

    stages = {
        "cast_grad_h": lambda _: mxnorm.mx_cast_fwd(gh, None, 32, fmt, codes=gh_c, scales=gh_s),
        "cast_t_w": lambda _: mxnorm.mx_cast_t_fwd(w, None, 32, fmt, codes=wt_c, scales=wt_s),
        "matmul_grad_z": lambda _: mxnorm.mx_matmul_fwd(gh_c, gh_s, wt_c, wt_s, N, elem=fmt,
                                                        out_dtype=torch.bfloat16, out=gz),
        "ste": lambda _: mxnorm.mxnorm_ste_bwd(x, gz, gam, rho, grad_x=gx, grad_gamma=gg,
                                               workspace=ws),
        "cast_t_grad_h": lambda _: mxnorm.mx_cast_t_fwd(gh, None, 32, fmt, codes=ght_c,
                                                        scales=ght_s),
        "cast_t_rho_x": lambda _: mxnorm.mx_cast_t_fwd(x, rho, 32, fmt, codes=xt_c,
                                                       scales=xt_s),
        "matmul_grad_w": lambda _: mxnorm.mx_matmul_fwd(ght_c, ght_s, xt_c, xt_s, T, elem=fmt,
                                                        out_dtype=torch.float32, out=gw,
                                                        b_gain=gam),
    }

    def whole(i):
        for f in stages.values():
            f(i)

    flops = 2.0 * 2 * T * N * d
    reps = max(2, int(budget_ms / (flops / 1.5e15 * 1e3)))
    t = {k: [] for k in list(stages) + ["backward"]}
    for _ in range(rounds):
        t["backward"].append(graph_time(whole, 1, reps, 1, stream))
        for k, f in stages.items():
            t[k].append(graph_time(f, 1, reps, 1, stream))
    m = {k: float(np.median(v)) for k, v in t.items()}
    out = {"format": fmt, "tokens": T, "N": N, "d": d,
           "backward_us": round(m["backward"] * 1e3, 2),
           "stages_us": {k: round(m[k] * 1e3, 2) for k in stages},
           "matmul_TFLOPs": {k: round(2.0 * T * N * d / (m[k] * 1e-3) / 1e12, 1)
                             for k in ("matmul_grad_z", "matmul_grad_w")},
           "ste_GBps": round(ste_bytes(T, d) / (m["ste"] * 1e-3) / 1e9, 1),
           "cast_t_rho_x_GBps": round((T * d * 2 + T * cw(d) + T * d // 32 + 4 * T)
                                      / (m["cast_t_rho_x"] * 1e-3) / 1e9, 1)}
    del x, w, gh, gz, gx, gw, ws
    torch.cuda.empty_cache()
    return out


def run_backward(path):
    import torch
    from paper_2603_13180_amd import mxnorm
    mxnorm.load()
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(dev)
    gen = torch.Generator(device=dev)
    results = []
    for fmt in ("e4m3", "e2m1"):
        for name, N in LAYER_N.items():
            for T in (4096, 16384, 32768):
                gen.manual_seed(T + N)
                r = backward_case(fmt, T, N, stream, gen)
                r["projection"] = name
                results.append(r)
                print(json.dumps(r), file=sys.stderr, flush=True)
    doc = {"method": "each stage and the whole chain captured as HIP graphs, replayed ~40 ms "
                     "per round, median of 3 interleaved rounds; N(0,1) activations, "
                     "0.02 N(0,1) weights, 0.01 N(0,1) output gradients",
           "results": results}
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)
    print(json.dumps({"backward": path, "shapes": len(results)}))


def mxfp8_bytes(T, d):
    return T * d * 2 + T * d + T * (d // 32) + 4 * T


def nvfp4_bytes(T, d):
    return T * d * 2 + T * d // 2 + T * (d // 16) + 4 * T


def source_hash():
    h = hashlib.sha256()
    for f in KERNEL_SRC:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source; else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def time_launches(fn, n_sets, steps, warmup, stream):
    import torch
    for i in range(warmup):
        fn(i % n_sets)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(steps):
        fn(i % n_sets)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps  # ms per launch


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# every workload preset, with the oracle entry point that computes it
CPU_CONFIGS = (("llama3-125m-d768", "mxfp8"), ("llama3-1b-d2048", "mxfp8"),
               ("llama3-8b-d4096", "mxfp8"), ("llama3-8b-d4096-nvfp4", "nvfp4"),
               ("llama3-8b-longctx-stress", "mxfp8"))


def _oracle_fn(fmt, d):
    import numpy as np
    import oracle
    if fmt == "mxfp8":
        return oracle.mxnorm_mxfp8, mxfp8_bytes
    s_g = float(np.float32(oracle.mxnorm_default_global_scale(d, 16, 2)))
    return (lambda x: oracle.mxnorm_nvfp4(x, s_g)), nvfp4_bytes


def _time_rows(fn, x, budget_s, step=512):
    """Single-threaded: chunks of `step` rows from the start of x until
    budget_s has passed or x is used up.  Returns (rows, seconds)."""
    fn(x[:4])   # builds/loads the library outside the timing
    done = 0
    t0 = time.perf_counter()
    while done < x.shape[0] and time.perf_counter() - t0 < budget_s:
        fn(x[done:done + step])
        done += step
    return min(done, x.shape[0]), time.perf_counter() - t0


def cpu_baseline(x_rows, d, budget_s=10.0, per_config_s=2.0, parallel_rows=32768):
    """The oracle as it stands on the host cores.  Primary: single-threaded,
    on the first rows of the headline workload until about budget_s has been
    spent.  Also: a bounded single-threaded sample of each workload preset,
    and the same oracle run row-parallel on threads over the cores this
    process may use (its C calls release the GIL), as a secondary number."""
    from concurrent.futures import ThreadPoolExecutor
    import numpy as np
    from paper_2603_13180_amd import synth

    fn, nbytes = _oracle_fn("mxfp8", d)
    done, el = _time_rows(fn, x_rows, budget_s)
    per = {}
    for name, fmt in CPU_CONFIGS:
        P = synth.PRESETS[name]
        rows = min(P.T, 8192)
        xs = x_rows if name == WORKLOAD else synth.generate(name, rows=np.arange(rows)).x
        f, nb = _oracle_fn(fmt, P.d)
        n, t = _time_rows(f, xs[:rows], per_config_s, step=256)
        per[name] = {"format": fmt, "rows": n, "s": round(t, 2),
                     "GB/s": round(nb(n, P.d) / t / 1e9, 4), "rows_per_s": round(n / t, 1),
                     "full_tensor_s_est": round(P.T * t / n, 1)}
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    threads = max(1, min(avail, 64))
    xp = x_rows[:parallel_rows]
    chunks = [c for c in np.array_split(np.arange(xp.shape[0]), 8 * threads) if len(c)]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(lambda ix: fn(xp[ix[0]:ix[-1] + 1]), chunks))
    tp = time.perf_counter() - t0
    return {
        "value": round(nbytes(done, d) / el / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": "first %d rows of %s (%d elements), single-threaded C oracle, %.1f s"
                  % (done, WORKLOAD, done * d, el),
        "rows_per_s": round(done / el, 1),
        "nproc": os.cpu_count(),
        "cores_available": avail,
        "cpu_model": cpu_model(),
        "per_config": per,
        "row_parallel": {"threads": threads, "rows": int(xp.shape[0]), "s": round(tp, 2),
                         "GB/s": round(nbytes(xp.shape[0], d) / tp / 1e9, 4),
                         "rows_per_s": round(xp.shape[0] / tp, 1),
                         "sample": "first %d rows of %s, row chunks on %d threads"
                                   % (xp.shape[0], WORKLOAD, threads)},
    }


def main():
    args = parse()
    if args.sweep:
        run_sweep(args.sweep, args.sweep_formats.split(","))
        return
    if args.layer:
        run_layer(args.layer)
        return
    if args.backward:
        run_backward(args.backward)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(rows are independent; see the sharding notes).  Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2603_13180_amd import mxnorm, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    mxnorm.load()

    w = synth.generate(WORKLOAD)
    T, d = w.preset.T, w.preset.d
    x0 = torch.from_numpy(w.x.view(np.int16)).view(torch.bfloat16).to(dev)
    g = torch.from_numpy(w.gamma.view(np.int16)).view(torch.bfloat16).to(dev)
    n_sets = max(2, -(-ROTATE_MIN_BYTES // x0.numel() // 2))
    xs = [x0] + [x0.clone() for _ in range(n_sets - 1)]
    codes = [torch.empty(T, d, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    scales = [torch.empty(T, d // 32, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    rho = [torch.empty(T, dtype=torch.float32, device=dev) for _ in range(n_sets)]
    ncodes = [torch.empty(T, d // 2, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    nscales = [torch.empty(T, d // 16, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    stream = torch.cuda.current_stream(dev)

    def mxn(i):
        mxnorm.mxnorm_mxfp8_fwd(xs[i], codes=codes[i], scales=scales[i], rho=rho[i])

    def rms(i):
        mxnorm.rmsnorm_mxfp8_fwd(xs[i], None, codes=codes[i], scales=scales[i], rho=rho[i])

    def post(i):
        mxnorm.mxnorm_postround_mx_fwd(xs[i], 32, "e4m3", codes=codes[i], scales=scales[i],
                                       rho=rho[i])

    def rms_g(i):
        mxnorm.rmsnorm_mxfp8_fwd(xs[i], g, codes=codes[i], scales=scales[i], rho=rho[i])

    s_g = mxnorm.mxnorm_default_global_scale(d, 16, 2)
    gmax = float(np.abs(synth.bf16_bits_to_f32(w.gamma)).max())
    s_r = mxnorm.rmsnorm_default_global_scale(d, gmax)

    def nv_mxn(i):
        mxnorm.mxnorm_nvfp4_fwd(xs[i], s_g, codes=ncodes[i], scales=nscales[i], rho=rho[i])

    def nv_rms(i):
        mxnorm.rmsnorm_nvfp4_fwd(xs[i], None, mxnorm.rmsnorm_default_global_scale(d, 1.0),
                                 codes=ncodes[i], scales=nscales[i], rho=rho[i])

    def nv_rms_g(i):
        mxnorm.rmsnorm_nvfp4_fwd(xs[i], g, s_r, codes=ncodes[i], scales=nscales[i], rho=rho[i])

    # the headline: exactly `steps` timed MXNorm MXFP8 steps
    ms = time_launches(mxn, n_sets, args.steps, args.warmup, stream)
    b8 = mxfp8_bytes(T, d)
    gbps = b8 / (ms * 1e-3) / 1e9

    # every kernel, in interleaved rounds so that clock and thermal drift hit
    # all of them alike; the speedups use the per-kernel medians
    kernels = (("mxnorm_mxfp8", mxn, b8), ("rmsnorm_mxfp8", rms, b8),
               ("mxnorm_postround_mxfp8", post, b8),
               ("rmsnorm_mxfp8_gamma", rms_g, b8 + 2 * d),
               ("mxnorm_nvfp4", nv_mxn, nvfp4_bytes(T, d)),
               ("rmsnorm_nvfp4", nv_rms, nvfp4_bytes(T, d)),
               ("rmsnorm_nvfp4_gamma", nv_rms_g, nvfp4_bytes(T, d) + 2 * d))
    rounds, per_round = 7, max(20, args.steps // 5)
    times = {name: [] for name, _, _ in kernels}
    for _ in range(rounds):
        for name, fn, _ in kernels:
            times[name].append(time_launches(fn, n_sets, per_round, 3, stream))
    side = {}
    for name, _, nbytes in kernels:
        m = float(np.median(times[name]))
        side[name] = {"ms": round(m, 5), "GB/s": round(nbytes / (m * 1e-3) / 1e9, 1),
                      "pct_of_peak": round(100 * nbytes / (m * 1e-3) / 1e9 / PEAK_HBM_GBPS, 2)}

    # practical ceilings on this device: the same traffic and access pattern
    # with no arithmetic (mixed, read-only, write-only), and a D2D copy
    from paper_2603_13180_amd import streamref
    small = [torch.empty(T, d // 32, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    ref = {}
    for mode, nbytes in (("mixed", b8 - 4 * T), ("read", T * d * 2 + 16 * T),
                         ("write", T * d + T * (d // 32)),
                         ("nvfp4", nvfp4_bytes(T, d) - 4 * T)):
        def run_ref(i, mode=mode):
            if mode == "nvfp4":
                streamref.stream_reference(xs[i], ncodes[i], nscales[i], mode)
            else:
                streamref.stream_reference(
                    xs[i], codes[i], small[i] if mode != "read" else small[i][:, :16], mode)
        m = time_launches(run_ref, n_sets, 50, 5, stream)
        ref[mode] = round(nbytes / (m * 1e-3) / 1e9, 1)
    dst = torch.empty_like(x0)
    m = time_launches(lambda i: dst.copy_(xs[i]), n_sets, 50, 5, stream)
    copy_gbps = 2 * x0.numel() * 2 / (m * 1e-3) / 1e9

    # the backward's streaming kernels at the same shape: the STE (x and a
    # synthetic grad_Z) and the column cast of rho~ X, inputs and outputs in
    # rotation like the forward's
    gzs = [torch.randn(T, d, device=dev).to(torch.bfloat16) for _ in range(n_sets)]
    gxo = [torch.empty(T, d, dtype=torch.bfloat16, device=dev) for _ in range(n_sets)]
    ggo = torch.empty(d, dtype=torch.float32, device=dev)
    wsp = torch.empty(mxnorm.load().mxnorm_ste_bwd_workspace_bytes(T, d), dtype=torch.uint8,
                      device=dev)
    tc = [torch.empty(d, T, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    ts = [torch.empty(d, T // 32, dtype=torch.uint8, device=dev) for _ in range(n_sets)]
    # each kernel beside the stream with its traffic and no arithmetic (the
    # STE's: x and grad_Z read, grad_X written; the column cast's: its
    # tiling, transposed bytes), in interleaved rounds after a common warm-up
    # so that clock and power transients hit a kernel and its stream alike;
    # per-kernel medians
    bkern = (("ste", lambda i: mxnorm.mxnorm_ste_bwd(
                 xs[i], gzs[i], g, rho[i], grad_x=gxo[i], grad_gamma=ggo, workspace=wsp)),
             ("ste_ref", lambda i: streamref.stream_reference_ste(xs[i], gzs[i], gxo[i])),
             ("ct", lambda i: mxnorm.mx_cast_t_fwd(xs[i], rho[i], codes=tc[i], scales=ts[i])),
             ("ct_ref", lambda i: streamref.stream_reference_transpose(xs[i], rho[i], tc[i],
                                                                       ts[i])))
    for _, fn in bkern:
        time_launches(fn, n_sets, 30, 0, stream)
    btimes = {name: [] for name, _ in bkern}
    for _ in range(7):
        for name, fn in bkern:
            btimes[name].append(time_launches(fn, n_sets, 20, 3, stream))
    ms_ste, ms_ste_ref, ms_ct, ms_ct_ref = (float(np.median(btimes[k]))
                                            for k in ("ste", "ste_ref", "ct", "ct_ref"))
    ste_ref_gbps = 3 * T * d * 2 / (ms_ste_ref * 1e-3) / 1e9
    ct_ref_gbps = cast_t_bytes(T, d) / (ms_ct_ref * 1e-3) / 1e9
    bwd = {"ste_bwd": {"us": round(ms_ste * 1e3, 2),
                       "GB/s": round(ste_bytes(T, d) / (ms_ste * 1e-3) / 1e9, 1)},
           "cast_t_rho_x_mxfp8": {"us": round(ms_ct * 1e3, 2),
                                  "GB/s": round(cast_t_bytes(T, d) / (ms_ct * 1e-3) / 1e9, 1)}}
    for v in bwd.values():
        v["pct_of_peak"] = round(100 * v["GB/s"] / PEAK_HBM_GBPS, 2)
    bwd["ste_bwd"]["stream_reference_GBps"] = round(ste_ref_gbps, 1)
    bwd["ste_bwd"]["frac_of_stream_reference"] = round(bwd["ste_bwd"]["GB/s"] / ste_ref_gbps, 4)
    ct = bwd["cast_t_rho_x_mxfp8"]
    ct["stream_reference_GBps"] = round(ct_ref_gbps, 1)
    ct["frac_of_stream_reference"] = round(ct["GB/s"] / ct_ref_gbps, 4)
    bwd["method"] = ("median of 7 interleaved rounds of 20 launches per kernel, each kernel "
                     "beside its stream")
    del gzs, gxo, wsp, tc, ts

    # the MX matmul the MXNorm output feeds (Llama-3-8B QKV projection)
    del ncodes, nscales, small
    torch.cuda.empty_cache()
    lgen = torch.Generator(device=dev)
    lgen.manual_seed(7)
    lay = layer_case("e4m3", T, LAYER_N["qkv"], torch.cuda.Stream(dev), lgen)

    traffic = measured_traffic()
    line = {
        "metric": "MXNorm+MXFP8 cast HBM GB/s (% of peak); speedup vs RMSNorm+cast",
        "value": round(gbps, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: MXNorm (p=2, B=32, RCEIL) fwd, x bf16 [%d, %d] N(0,1) with 1%% "
                        "outlier channels x20 -> E4M3 codes + E8M0 scales + rho" % (WORKLOAD, T, d),
            "tokens": T, "d": d, "block": 32, "p": 2, "scale_mode": "rceil",
            "rotating_buffer_sets": n_sets,
        },
        "pct_of_peak": round(100 * gbps / PEAK_HBM_GBPS, 2),
        "rows_per_s": round(T / (ms * 1e-3), 1),
        "speedup_vs_rmsnorm_cast":
            round(side["rmsnorm_mxfp8"]["ms"] / side["mxnorm_mxfp8"]["ms"], 4),
        "speedup_vs_rmsnorm_gamma_cast":
            round(side["rmsnorm_mxfp8_gamma"]["ms"] / side["mxnorm_mxfp8"]["ms"], 4),
        "speedup_method": "median of %d interleaved rounds of %d launches per kernel"
                          % (rounds, per_round),
        "nvfp4": {
            "workload": NV_WORKLOAD,
            "GB/s": side["mxnorm_nvfp4"]["GB/s"],
            "pct_of_peak": side["mxnorm_nvfp4"]["pct_of_peak"],
            "speedup_vs_rmsnorm_cast": round(side["rmsnorm_nvfp4"]["ms"] / side["mxnorm_nvfp4"]["ms"], 4),
            "speedup_vs_rmsnorm_gamma_cast":
                round(side["rmsnorm_nvfp4_gamma"]["ms"] / side["mxnorm_nvfp4"]["ms"], 4),
            "stream_reference_GBps": ref["nvfp4"],
            "frac_of_stream_reference": round(side["mxnorm_nvfp4"]["GB/s"] / ref["nvfp4"], 4),
        },
        "kernels": side,
        "mx_matmul": {
            "shape": "MXNormLinear QKV: [%d, %d] x [%d, %d]^T MXFP8 -> bf16" % (T, d, lay["N"], d),
            "TFLOP/s": lay["matmul_TFLOPs"], "frac_of_fp8_peak": lay["matmul_frac_of_peak"],
            "layer_speedup_vs_rmsnorm_gamma_cast": lay["layer_speedup"],
            "layer_speedup_from_parts": lay["layer_speedup_from_parts"]},
        "backward_kernels": bwd,
        "copy_d2d_GBps": round(copy_gbps, 1),
        "stream_reference_GBps": ref,
        "frac_of_stream_reference": round(gbps / ref["mixed"], 4),
        "roofline": {
            "bound": "hbm",
            "achieved": round(gbps, 1),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(gbps / PEAK_HBM_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": b8,
        },
        "cpu_baseline": None,
    }
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(w.x, d)
    print(json.dumps(line))


if __name__ == "__main__":
    main()
