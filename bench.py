"""Benchmark: ConvCRF mean-field inference on one MI355X.

One step = one full call of the library (softmax init + T mean-field rounds)
on one synthetic batch already resident in HBM.  Prints one JSON line with
the throughput in megapixel-iterations per second, the roofline of the
dominant kernel (the kernel with the largest share of the time, by HIP events
recorded by the library around every launch on the launch stream; its
duration is that share of the timed region) and the double-precision CPU
oracle timed on this host as a baseline.

    python bench.py [--steps K] [--warmup W] [--workload pascal]
                    [--variant fused|materialised|resident] [--no-cpu-baseline]
                    [--backward]

--backward times the reverse mode instead: one step = one call of
convcrf_meanfield_backward (the forward rounds recomputed and kept, then every
round undone, with the compatibility and kernel-parameter derivatives).
--features runs the learnable-smoothness-feature variant (Sec. 4.2, "+T"):
two feature planes, the pixel positions plus seeded N(0, 0.5) noise (with
--backward, dL/dF is returned as well).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "megapixel·iterations/sec and ms per 5-iter inference (C=21, 512², k=7)"
METRIC_BWD = ("megapixel·iterations/sec and ms per 5-iter derivative (forward recomputed, "
              "then reversed; C=21, 512², k=7)")
UNIT = "MP·iter/s"

# MI355X: FP32 vector peak 157.3 TFLOP/s (256 CUs at 2.4 GHz, 128 FP32 FMA
# lanes per CU per clock).  The library is built without packed FP32; gfx950
# reaches that lane rate only by issuing VALU instructions of two waves of a
# SIMD in the same cycle, which needs all-VGPR operands (measured with an FMA
# loop: 118-123 lanes per clock per CU at two or more waves per SIMD, 59 at
# one, about 62 with an SGPR or DPP operand).  HBM3E: 8 TB/s.
PEAK_VALU_FP32 = 157.3e12
PEAK_VALU_LANE_OPS = 256 * 128 * 2.4e9     # VALU lane-instructions per second at that peak
PEAK_HBM = 8.0e12

ITER_SRC = os.path.join(ROOT, "paper_1805_04777_amd", "csrc", "iter.hip")
COUNTERS = os.path.join(ROOT, "profiles", "counters.json")


def flops_per_pixel_iter(C: int, k: int) -> int:
    """Algorithmic flops of one pixel-iteration: message 2C(k^2-1), Gaussian
    weights 12 per tap (3 differences, squared norm, exponent, exp, add),
    compatibility 2C^2 (the C x C matrix-vector product; the library folds
    Potts into Z = U + M, which needs fewer), unary add and softmax 5C + 1."""
    taps = k * k - 1
    return 2 * C * taps + 12 * taps + 2 * C * C + 5 * C + 1


def bytes_per_pixel(C: int, first: bool) -> int:
    """Algorithmic HBM bytes of one fused launch per pixel: read Q_t (not on
    the first launch, which reads U instead), U and the RGB image, write
    Q_{t+1}; fp32."""
    return 4 * C * (2 if first else 3) + 12


def algorithmic_per_launch(kname: str, wl, D: int = 0):
    """(flops, HBM bytes) one launch of `kname` must spend on workload `wl`
    (averaged over its launches in one call); fp32; D learnable smoothness
    feature planes (0 without).  fused_iter is one later iteration (reads
    Q_t, U and the image, writes Q_t+1), fused_first the first one (reads U
    and the image, writes Q_1; its softmax of U is counted with the update's)."""
    C, k, T, px = wl.C, wl.filter_size, wl.iters, wl.pixels
    if kname == "fused_iter":
        return flops_per_pixel_iter(C, k) * px, bytes_per_pixel(C, False) * px
    if kname == "fused_first":
        return (flops_per_pixel_iter(C, k) + 5 * C + 1) * px, bytes_per_pixel(C, True) * px
    if kname == "materialised_iter":
        taps = k * k - 1
        return ((flops_per_pixel_iter(C, k) - 12 * taps) * px,
                ((bytes_per_pixel(C, True) + (T - 1) * bytes_per_pixel(C, False)) / T + 4 * taps) * px)
    if kname == "build_kernel":
        taps = k * k - 1
        return 12 * taps * px, (12 + 4 * taps) * px
    if kname == "fused_resident":
        # one launch = T iterations; bytes: U and the image read, Q written
        # (the tiles' border rings are the only other traffic)
        return T * flops_per_pixel_iter(C, k) * px, (8 * C + 12) * px
    s2 = wl.blur * wl.blur
    npx = px // s2
    if kname == "blur_message":
        # pooled grid: read pooled Q and colours (and D pooled feature planes,
        # whose Gaussian costs 3D + 2 per tap), write pooled message
        fg = 3 * D + 2 if D else 0
        return (2 * C + 12 + fg) * (k * k - 1) * npx, (8 * C + 12 + 4 * D) * npx
    if kname == "blur_update":
        # per pixel: bilinear sample of C pooled messages (3 FMA each), unary
        # add, softmax, s*s average; reads U, writes the pooled Q (T - 1
        # launches) or the full Q (the last one)
        return ((6 + 1 + 5 + 1) * C * px,
                4 * C * px + 4 * C * npx + ((T - 1) * 4 * C * npx + 4 * C * px) / T)
    if kname == "blur_iteration":
        # one fused iteration (4 x 4 pooling): the pooled message of every
        # cell (weights 12, with D pooled feature planes their Gaussian 3D + 2,
        # and message 2C per tap) and per pixel the bilinear sample (3C FMA),
        # unary add and softmax (5C + 1) and the cell average (C); reads U,
        # the pooled Q_t, colours and features, writes the pooled Q_t+1
        # (T - 1 launches) or the full Q (the last)
        taps = k * k - 1
        fg = 3 * D + 2 if D else 0
        return ((2 * C + 12 + fg) * taps * npx + (6 * C + 5 * C + 1 + C) * px,
                4 * C * px + (4 * C + 12 + 4 * D) * npx + ((T - 1) * 4 * C * npx + 4 * C * px) / T)
    if kname == "blur_pool":
        if wl.blur == 4:
            # one launch per call: softmax(U), the image and the D feature
            # planes, averaged over the cells; reads them, writes the pooled
            # planes
            return (5 * C + 1 + C + 3 + D) * px, 4 * (C + 3 + D) * (px + npx)
        # one launch per pooled tensor (the image, the features, softmax(U)),
        # averaged over them
        n = 3 if D else 2
        return ((5 * C + 1 + C + 3 + D) * px / n, 4 * (C + 3 + D) * (px + npx) / n)
    if kname == "softmax":
        return (5 * C + 1) * px, 8 * C * px
    if kname == "sync_reset":
        return 0, 0
    # reverse mode (compatibility and kernel-parameter derivatives requested)
    taps = k * k - 1
    if kname == "bwd_message" and wl.blur > 1:
        # on the pooled grid (the derivative of the blur variant): as below
        # per pooled cell
        npx = px // (wl.blur * wl.blur)
        if D:
            return ((8 * C + 22 + 5 * D + 6) * taps + 2 * C * C) * npx, (16 * C + 12 + 12 * D) * npx
        return (6 * C + 22) * taps * npx + 2 * C * C * npx, (16 * C + 12) * npx
    if kname == "feature_iter":
        # per tap: the appearance weight (12), the feature distance and its
        # Gaussian (3D + 2), the message (2C); per pixel unary add and softmax
        # (5C + 1); reads Q_t, U, the image and the features, writes Q_t+1
        return ((12 + 3 * D + 2 + 2 * C) * taps + 5 * C + 1) * px, (12 * C + 12 + 4 * D) * px
    if kname == "bwd_message":
        # per tap: the weight (12), dk = <dM_p, Q_q> (2C), dQ += w dM (2C),
        # M += w Q (2C), the five parameter sums (10); per pixel the outer
        # product dP M^T (2C^2); reads Q^t, dM, dP and the image, writes dQ^t.
        # With features: the feature Gaussian (3D + 2), dk(x+d, x) (2C) and
        # dL/dF (2D + 4) per tap; the features read, dL/dF read and written
        if D:
            return ((8 * C + 22 + 5 * D + 6) * taps + 2 * C * C) * px, (16 * C + 12 + 12 * D) * px
        return (6 * C + 22) * taps * px + 2 * C * C * px, (16 * C + 12) * px
    if kname == "bwd_point":
        # T + 1 launches per call.  T undo a round: dot, dZ, dU and the Potts
        # dM (7C flops); read Q, dQ and, except on the first, dU; write dU
        # and dM (with Potts no -dZ plane is written).  The last one takes
        # only the initial softmax's adjoint (5C; read Q, dQ, dU, write dU).
        # dQ is grad_q on the first; with blur the later ones read it on the
        # pooled grid (the pooling's transpose applied in place).
        dq_later = 4 * C / (wl.blur * wl.blur)
        rounds = 7 * C * T + 5 * C
        rbytes = (12 * C * T + 4 * C + dq_later * (T - 1) + 4 * C * (T - 1)
                  + 12 * C + dq_later)
        return rounds * px / (T + 1), rbytes * px / (T + 1)
    if kname == "bwd_reduce":
        return 0, 0
    if kname == "bwd_blur_transpose":
        # one launch per round (with Potts -dL/dZ follows from dL/dM): the
        # bilinear upsampling transposed for dL/dM, each full-resolution
        # value reaching four cells (8 flop per pixel and class; the
        # full-resolution planes read, the pooled ones written); with
        # features one more at the end, the pooling's transpose of dL/dF
        # (pooled read, full resolution written).  Averaged over the launches.
        s2 = wl.blur * wl.blur
        n = T + (1 if D else 0)
        fl = 8 * C * px * T + D * px
        by = 4 * (C * T + D) * (px + px / s2)
        return fl / n, by / n
    raise KeyError(kname)


def source_hash(path: str = ITER_SRC) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def counters_key(workload: str, kernel: str, D: int = 0) -> str:
    """Key of a kernel's record in profiles/counters.json; runs with learnable
    features have their own records."""
    return f"{workload}{'+features' if D else ''}/{kernel}"


def load_counters(workload: str, kernel: str, D: int = 0):
    """Counter figures per launch of `kernel` on `workload` from the committed
    rocprofv3 passes (profiles/counters.json): HBM bytes (FETCH_SIZE and
    WRITE_SIZE, scaled by what they read for a plain copy) and VALU
    instructions (SQ_INSTS_VALU); None unless they were taken on the current
    source of the kernel (the file a record names, csrc/iter.hip if none)."""
    try:
        with open(COUNTERS) as f:
            rec = json.load(f)[counters_key(workload, kernel, D)]
    except (OSError, KeyError, ValueError):
        return None
    src = os.path.join(os.path.dirname(ITER_SRC), rec.get("source", "iter.hip"))
    try:
        if rec.get("source_sha256_16") != source_hash(src):
            return None
    except OSError:
        return None
    return rec


def cpu_baseline(wl, U, I, budget_s: float = 10.0, backward: bool = False, features=None):
    """The oracle as it stands, on this host: the full workload, repeated
    until `budget_s` seconds have passed (median per call); with `backward`,
    its derivative (forward recomputed, then reversed) on the same inputs."""
    import numpy as np
    import oracle
    oracle.build()
    p = oracle.OracleParams(filter_size=wl.filter_size, blur=wl.blur, w_app=wl.w_app,
                            theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta,
                            w_smooth=wl.w_smooth, theta_gamma=wl.theta_gamma)
    times = []
    t_all = time.perf_counter()
    G = np.random.default_rng(77).normal(0.0, 1.0, U.shape) if backward else None
    while True:
        t0 = time.perf_counter()
        if backward:
            oracle.meanfield_backward(U, I, p, wl.iters, G, features=features)
        else:
            oracle.meanfield(U, I, p, wl.iters, features=features)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_all >= budget_s or len(times) >= 50:
            break
    t = float(np.median(times))
    mpi = wl.pixels * wl.iters / 1e6
    single = None if backward or features is not None else cpu_single_thread(wl)
    return {"value": round(mpi / t, 3), "unit": UNIT, "cores": oracle.num_threads(),
            "kind": "oracle", "single_thread": single,
            "sample": f"the full {wl.name} workload ({wl.B}x{wl.C}x{wl.H}x{wl.W}, k={wl.filter_size}, "
                      f"blur={wl.blur}, T={wl.iters}){', derivative' if backward else ''}"
                      f"{', learnable features D=2' if features is not None else ''}, "
                      f"{len(times)} calls, median {t * 1e3:.1f} ms/call, double precision"}


def cpu_single_thread(wl):
    """The oracle on one host thread (OMP_NUM_THREADS=1, in a child process,
    since OpenMP reads it at start-up), on the top quarter of the first
    image of the workload (the same per-pixel work; a few seconds)."""
    import subprocess
    rows = max(1, wl.H // 4)
    code = (
        "import sys, time, json\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "import oracle\n"
        "from paper_1805_04777_amd import synth\n"
        f"wl = synth.WORKLOADS[{wl.name!r}]\n"
        "U, I, _ = synth.make_inputs(wl.with_(B=1))\n"
        f"U = U[:, :, :{rows}].copy(); I = I[:, :, :{rows}].copy()\n"
        "p = oracle.OracleParams(filter_size=wl.filter_size, blur=wl.blur, w_app=wl.w_app,"
        " theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta, w_smooth=wl.w_smooth,"
        " theta_gamma=wl.theta_gamma)\n"
        "t0 = time.perf_counter(); oracle.meanfield(U, I, p, wl.iters); t = time.perf_counter() - t0\n"
        "print(json.dumps({'s': t, 'threads': oracle.num_threads()}))\n")
    env = dict(os.environ, OMP_NUM_THREADS="1")
    try:
        r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                           timeout=120, check=True)
        rec = json.loads(r.stdout.strip().splitlines()[-1])
    except Exception as e:  # noqa: BLE001 - reported, not fatal
        return {"error": str(e)[:200]}
    mpi = rows * wl.W * wl.iters / 1e6
    return {"value": round(mpi / rec["s"], 4), "unit": UNIT, "cores": rec["threads"],
            "sample": f"rows 0..{rows - 1} of image 0 ({rows}x{wl.W}), one call, "
                      f"{rec['s'] * 1e3:.0f} ms"}


def copy_reference(torch, mib: int, steps: int) -> int:
    """Plain copy of `mib` MiB, `steps` times: each dispatch reads and writes
    exactly mib MiB, which calibrates the rocprofv3 byte counters."""
    n = mib * (1 << 20) // 4
    x = torch.rand(n, device="cuda:0")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(json.dumps({"copy_mib": mib, "ms_per_copy": round(ms, 5),
                      "GB_per_s": round(2 * mib * (1 << 20) / (ms / 1e3) / 1e9, 1)}), flush=True)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="pascal")
    ap.add_argument("--variant", choices=["fused", "materialised", "resident"], default="fused")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--backward", action="store_true",
                    help="time convcrf_meanfield_backward instead of the inference")
    ap.add_argument("--features", action="store_true",
                    help="learnable smoothness features (two planes)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="instead: time a plain device-to-device copy of this many MiB "
                         "(reference dispatch for the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: this library runs on one GPU; --gpus {args.gpus} is not supported "
              "(batch items or row bands would shard across GPUs, which is not built)",
              file=sys.stderr)
        return 2

    import torch

    if args.copy_mib:
        return copy_reference(torch, args.copy_mib, args.steps)

    from paper_1805_04777_amd import convcrf as cc
    from paper_1805_04777_amd import synth

    wl = synth.WORKLOADS[args.workload]
    U, I, _ = synth.make_inputs(wl)
    dev = torch.device("cuda:0")
    Ut = torch.from_numpy(U).to(dev)
    It = torch.from_numpy(I).to(dev)
    out = torch.empty_like(Ut)
    variant = {"fused": cc.VARIANT_FUSED, "materialised": cc.VARIANT_MATERIALISED,
               "resident": cc.VARIANT_RESIDENT}[args.variant]
    D = 2 if args.features else 0
    Fn = None
    if args.features:
        import numpy as np
        yy, xx = np.meshgrid(np.arange(wl.H, dtype=np.float32), np.arange(wl.W, dtype=np.float32),
                             indexing="ij")
        Fn = (np.stack([yy, xx])[None].repeat(wl.B, axis=0) + np.random.default_rng(78).normal(
            0.0, 0.5, (wl.B, 2, wl.H, wl.W))).astype(np.float32)
    p = cc.Params(filter_size=wl.filter_size, blur=wl.blur, variant=variant, w_app=wl.w_app,
                  theta_alpha=wl.theta_alpha, theta_beta=wl.theta_beta, w_smooth=wl.w_smooth,
                  theta_gamma=wl.theta_gamma,
                  features=None if Fn is None else torch.from_numpy(Fn).to(dev))
    crf = cc.ConvCRF(0)
    stream = torch.cuda.current_stream(dev)
    if args.backward:
        import numpy as np
        Gt = torch.from_numpy(np.random.default_rng(77).normal(
            0.0, 1.0, U.shape).astype(np.float32)).to(dev)

        def step():
            crf.meanfield_backward(Ut, It, p, wl.iters, Gt, grad_compat=True, grad_kernel=True,
                                   out=out, stream=stream)
    else:
        def step():
            crf.meanfield(Ut, It, p, wl.iters, out=out, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # timed pass: K steps, nothing recorded between the library's launches
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    ms = total_ms / args.steps
    value = wl.pixels * wl.iters / 1e6 / (ms / 1e3)
    # distribution pass: each call between its own pair of events
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(args.steps)]
    for e_start, e_stop in pairs:
        e_start.record(stream)
        step()
        e_stop.record(stream)
    torch.cuda.synchronize()
    import numpy as np
    per_call = np.array([a.elapsed_time(b) for a, b in pairs])
    dist = {"p10": round(float(np.percentile(per_call, 10)), 5),
            "p50": round(float(np.median(per_call)), 5),
            "p90": round(float(np.percentile(per_call, 90)), 5)}
    # kernel pass: the same K steps with HIP events recorded by the library
    # around every launch, on the launch stream
    crf.profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()

    # per-kernel time of the K calls; the dominant kernel is the one with the
    # largest total, priced by its own algorithmic flops and bytes
    per = {n: crf.profile_read(n) for n in cc.KERNEL_NAMES}
    crf.profile_enable(False)
    launched = {n: v for n, v in per.items() if v[1] > 0}
    kname = max(launched, key=lambda n: launched[n][0])
    k_ms, k_n = launched[kname]
    # Events around every launch add about a microsecond each, so the
    # kernel's duration is taken from the timed region instead: its share of
    # the evented time, applied to the time per call, over its launches per
    # call.
    share = k_ms / sum(v[0] for v in launched.values())
    avg_s = ms / 1e3 * share / (k_n / args.steps)
    avg_s_events = k_ms / 1e3 / k_n
    F, Bytes = algorithmic_per_launch(kname, wl, D)
    alu_frac = F / avg_s / PEAK_VALU_FP32
    hbm_frac = Bytes / avg_s / PEAK_HBM
    # Which ceiling binds is decided by the counters, when they were taken on
    # the current source: the kernel's measured HBM traffic per second
    # against 8 TB/s, and its measured VALU lane-instructions per second
    # against the 157.3 TFLOP/s lane rate; the higher utilisation is the
    # binding one.  Without current counters the algorithmic fractions decide.
    ctr = load_counters(args.workload, kname, D)
    if ctr:
        hbm_util = ctr["bytes_per_launch"] / avg_s / PEAK_HBM
        valu_util = ctr["valu_insts_per_launch"] * 64 / avg_s / PEAK_VALU_LANE_OPS
        bound = "alu" if valu_util > hbm_util else "hbm"
        rule = "counters: measured HBM bytes/s vs 8 TB/s against measured VALU lane-ops/s vs peak"
    else:
        hbm_util = valu_util = None
        bound = "alu" if alu_frac >= hbm_frac else "hbm"
        rule = "no counters on the current source: the larger algorithmic fraction"
    if bound == "alu":
        roof = {"bound": "alu", "achieved": round(F / avg_s / 1e12, 3), "peak": round(PEAK_VALU_FP32 / 1e12, 1),
                "unit": "TFLOP/s", "frac": round(alu_frac, 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(Bytes / avg_s / 1e9, 1), "peak": PEAK_HBM / 1e9,
                "unit": "GB/s", "frac": round(hbm_frac, 4)}
    roof["traffic"] = ctr["bytes_per_launch"] if ctr else None
    roof.update({
        "kernel": kname, "launches": k_n, "avg_launch_us": round(avg_s * 1e6, 3),
        "avg_launch_us_per_launch_events": round(avg_s_events * 1e6, 3),
        "algorithmic_flop_per_launch": int(F), "algorithmic_bytes_per_launch": int(Bytes),
        "alu_frac": round(alu_frac, 4), "hbm_frac": round(hbm_frac, 4),
        "bound_rule": rule,
        "hbm_util_counters": None if hbm_util is None else round(hbm_util, 4),
        "valu_util_counters": None if valu_util is None else round(valu_util, 4),
        "evented_ms_per_step_by_kernel": {n: round(v[0] / args.steps, 5) for n, v in launched.items()},
    })

    rec = {
        "metric": METRIC_BWD if args.backward else METRIC, "value": round(value, 2),
        "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "ms_per_call_distribution": dist,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded Voronoi images and noisy unaries)",
        "config": {"workload": f"{wl.name}: B={wl.B} C={wl.C} {wl.H}x{wl.W} k={wl.filter_size} "
                               f"blur={wl.blur} T={wl.iters} Potts, "
                               + ("derivative (dU, dmu, d kernel parameters)" if args.backward
                                  else args.variant)
                               + (", learnable smoothness features D=2" if args.features else ""),
                   "global_batch": wl.B, "variant": args.variant,
                   "direction": "backward" if args.backward else "forward"},
        "roofline": roof,
    }
    crf.close()
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl, U, I, backward=args.backward, features=Fn)
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
