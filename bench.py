"""Benchmark of the MEC hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--layer NAME] [--algo lowered|fused]

One step is one MEC convolution of the layer: the compact lowering of I into
L followed by the o_h slab products (mec_lower + mec_gemm, exactly the two
kernels mec_conv2d(MEC_ALGO_LOWERED) enqueues), on inputs already resident in
device memory. Buffers rotate over several sets so that the 256 MB
memory-attached last-level cache cannot serve a step from the previous one.
Timing, with HIP events on the stream the kernels run on: the K timed steps
run between two events with nothing else on the stream (ms_per_step, value);
then the same K steps run again with an event around every kernel launch
(the per-kernel durations of the rooflines). The events are created without
the system-scope fence, so recording one between two launches adds no cache
maintenance to the interval it measures.

Prints ONE JSON line: effective TFLOP/s (2*MAC/time) of the whole step, the
workspace bytes against im2col's, the roofline of the dominant kernel (the slab
products) and of the lowering, the fused variant's rate, and the CPU oracle's
rate on the host cores (a baseline, not the target).
"""
import argparse
import json
import os
import sys
import time

REPO = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, REPO)

METRIC = "effective conv TFLOP/s (2·MAC/time) + workspace bytes vs im2col, 1×MI355X"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}   # dense MFMA peaks of the MI355X
PEAK_HBM_GBS = 8000.0
DEFAULT_LAYER = "resnet_mid"


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--layer", default=DEFAULT_LAYER)
    ap.add_argument("--algo", default="lowered", choices=["lowered", "fused", "im2col"],
                    help="MEC from L (default), MEC fused, or the im2col + product baseline")
    ap.add_argument("--sets", type=int, default=4, help="rotating buffer sets")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the layer's batch size i_n (0 keeps the layer's own)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time for the oracle baseline (0 skips it)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one plain device-to-device copy of this many MiB "
                         "(a known-size reference for rocprofv3 byte counters)")
    ap.add_argument("--traffic", default=None,
                    help="profile summary holding the slab-product kernel's per-launch HBM "
                         "bytes from rocprofv3 counters (default: profiles/slab_gemm_<dtype>_<layer>_"
                         "<algo>_traffic.md when present)")
    return ap.parse_args()


def _code_only(text):
    """C/C++/HIP source with comments and whitespace removed (string literals
    kept): edits to comments do not change the kernels."""
    import re
    pattern = re.compile(r'//[^\n]*|/\*.*?\*/|"(?:\\.|[^"\\])*"', re.S)
    text = pattern.sub(lambda m: m.group(0) if m.group(0).startswith('"') else " ", text)
    return "".join(text.split())


def csrc_digest():
    """sha256 over the native sources without their comments; a traffic figure
    taken from another version of the kernels is not reported."""
    import hashlib
    d = os.path.join(REPO, "paper_1706_06873_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".h", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(d, name), encoding="utf-8") as f:
                h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def load_traffic(path, kdt, layer_name, algo):
    """Per-launch HBM bytes of the slab-product kernel from a profile summary:
    the line starting with 'traffic-json:' holds FETCH_SIZE and WRITE_SIZE (KiB
    per dispatch), the factors that make each counter read a plain copy of known
    size correctly, and the digest of the sources the counters were taken on."""
    if path is None:
        path = os.path.join(REPO, "profiles", "slab_gemm_%s_%s_%s_traffic.md" % (kdt, layer_name, algo))
    if not os.path.exists(path):
        return None
    with open(path) as f:
        for line in f:
            if line.startswith("traffic-json:"):
                t = json.loads(line[len("traffic-json:"):])
                break
        else:
            return None
    if t.get("workload") != "%s %s" % (layer_name, algo) or t.get("csrc_sha256") != csrc_digest():
        return None
    return int(round((t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs as a single process on one GPU", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1706_06873_amd as mec
    from paper_1706_06873_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    layer = wl.LAYERS[args.layer]
    if args.batch > 0:
        import dataclasses
        layer = dataclasses.replace(layer, i_n=args.batch)
    dims = layer.dims
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    dt_code = mec.BF16 if layer.dtype == "bf16" else mec.F32
    es = 2 if layer.dtype == "bf16" else 4
    macs = i_n * o_h * o_w * k_c * k_h * k_w * i_c
    flops = 2.0 * macs
    ws_bytes = mec.workspace_bytes(*dims, dtype=dt_code, algo=mec.LOWERED)
    im2col_bytes = mec.im2col_bytes(*dims, dtype=dt_code)
    size_I = i_n * i_h * i_w * i_c
    size_K = k_h * k_w * i_c * k_c
    size_O = i_n * o_h * o_w * k_c
    size_L = ws_bytes // es
    size_M = im2col_bytes // es
    P = k_h * k_w * i_c  # im2col row length

    dev = torch.device("cuda:0")
    I0, K0 = wl.make_inputs(layer)
    sets = []
    for j in range(args.sets):
        I = I0.to(dev)
        if j:
            I = I.clone()
        lshape = (i_n, o_w, o_h, k_h, k_w, i_c) if args.algo == "im2col" else (i_n, o_w, i_h, k_w, i_c)
        sets.append(dict(I=I, K=K0.to(dev),
                         L=torch.empty(lshape, dtype=I0.dtype, device=dev),
                         O=torch.empty((i_n, o_h, o_w, k_c), dtype=torch.float32, device=dev)))
    stream = torch.cuda.Stream(device=dev)  # default priority
    torch.cuda.synchronize()

    def step(bufs, ev=None):
        if args.algo == "fused":
            if ev:
                ev[0].record(stream)
            mec.conv2d(bufs["I"], bufs["K"], s_h, s_w, algo="fused", O=bufs["O"], stream=stream)
            if ev:
                ev[1].record(stream)
            return
        if ev:
            ev[0].record(stream)
        if args.algo == "im2col":
            mec.im2col(bufs["I"], k_h, k_w, k_c, s_h, s_w, M=bufs["L"], stream=stream)
        else:
            mec.lower(bufs["I"], k_h, k_w, k_c, s_h, s_w, L=bufs["L"], stream=stream)
        if ev:
            ev[1].record(stream)
        if args.algo == "im2col":
            # the product of M and K: MEC's product phase of the 1x1 convolution
            # whose pixels (n, y, x) carry the patches as channels
            mec.gemm(bufs["L"].view(i_n, o_w, o_h, 1, P), bufs["K"].view(1, 1, P, k_c),
                     o_h, o_w, 1, 1, O=bufs["O"], stream=stream)
        else:
            mec.gemm(bufs["L"], bufs["K"], i_h, i_w, s_h, s_w, O=bufs["O"], stream=stream)
        if ev:
            ev[2].record(stream)

    from paper_1706_06873_amd.timing import HipEvent
    with torch.cuda.stream(stream):
        for w in range(args.warmup):
            step(sets[w % len(sets)])
        torch.cuda.synchronize()
        # the timed steps: nothing on the stream but the steps themselves
        start, end = HipEvent(), HipEvent()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        start.record(stream)
        for k in range(args.steps):
            step(sets[k % len(sets)])
        end.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        # the same steps again, an event around every launch: per-kernel durations
        n_ev = 2 if args.algo == "fused" else 3
        evs = [[HipEvent() for _ in range(n_ev)] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for k in range(args.steps):
            step(sets[k % len(sets)], evs[k])
        torch.cuda.synchronize()

    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    if args.algo == "fused":
        kern_ms = [e[0].elapsed_time(e[1]) for e in evs]
        lower_ms = None
    else:
        lower_ms = sorted(e[0].elapsed_time(e[1]) for e in evs)
        kern_ms = [e[1].elapsed_time(e[2]) for e in evs]
    kern_ms = sorted(kern_ms)
    kern_avg = sum(kern_ms) / len(kern_ms)
    value = flops / (ms_per_step * 1e-3) / 1e12

    # roofline of the dominant kernel: algorithmic flops per launch / its average duration
    peak = PEAK_TFLOPS[layer.dtype]
    achieved = flops / (kern_avg * 1e-3) / 1e12
    kname = "slab_gemm_%s_kernel" % ("bf16" if layer.dtype == "bf16" else "f32")
    if args.algo == "fused":
        alg_bytes = es * (size_I + size_K) + 4 * size_O
        kname += " (from I)"
    elif args.algo == "im2col":
        alg_bytes = es * (size_M + size_K) + 4 * size_O
        kname += " (im2col product, k_h = 1)"
    else:
        alg_bytes = es * (size_L + size_K) + 4 * size_O
    # a kernel whose arithmetic intensity is below the ridge point is HBM-bound
    ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)
    bound = "mfma" if flops / alg_bytes >= ridge else "hbm"
    traffic = load_traffic(args.traffic, "bf16" if layer.dtype == "bf16" else "f32", layer.name, args.algo) if args.batch <= 0 else None
    if bound == "mfma":
        roof = {"bound": "mfma", "kernel": kname, "achieved": round(achieved, 2),
                "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": traffic, "alg_flops": flops, "alg_bytes": alg_bytes,
                "avg_ms": round(kern_avg, 5)}
    else:
        gbs = alg_bytes / (kern_avg * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": kname, "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic,
                "alg_flops": flops, "alg_bytes": alg_bytes, "avg_ms": round(kern_avg, 5)}

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": layer.dtype,
        "data": "synthetic (seeded, %s)" % layer.note,
        "config": {"workload": "%s: i_n=%d, I %dx%dx%d (%s), K %dx%dx%dx%d, s=%d/%d, o=%dx%d"
                               % (layer.name, i_n, i_h, i_w, i_c, layer.dtype, k_h, k_w, i_c, k_c,
                                  s_h, s_w, o_h, o_w),
                   "algo": args.algo, "buffer_sets": args.sets},
        "workspace_bytes": {"lowered": ws_bytes, "fused": 0, "im2col": im2col_bytes}[args.algo],
        "im2col_bytes": im2col_bytes,
        "workspace_vs_im2col": round(im2col_bytes / ws_bytes, 4),
        "wall_s": round(wall, 4),
        "gemm_ms": {"avg": round(kern_avg, 5), "median": round(kern_ms[len(kern_ms) // 2], 5),
                    "min": round(kern_ms[0], 5)},
        "roofline": roof,
    }
    if lower_ms is not None:
        lavg = sum(lower_ms) / len(lower_ms)
        lbytes = es * (size_I + (size_M if args.algo == "im2col" else size_L))
        out["lower_ms"] = {"avg": round(lavg, 5), "median": round(lower_ms[len(lower_ms) // 2], 5),
                           "min": round(lower_ms[0], 5)}
        out["roofline_lower"] = {"bound": "hbm",
                                 "kernel": "im2col_*_kernel" if args.algo == "im2col" else "lower_*_kernel",
                                 "achieved": round(lbytes / (lavg * 1e-3) / 1e9, 1),
                                 "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                 "frac": round(lbytes / (lavg * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                                 "alg_bytes": lbytes}
    if args.copy_mib > 0:
        # A plain copy of known size through the library's own row-copy
        # kernel: with i_w = k_w = 1 the lowering is L = I element for element.
        rows = args.copy_mib * (1 << 20) // 4096
        src = torch.ones((1, rows, 1, 1024), dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        mec.lower(src, 1, 1, 1, 1, 1, L=dst, stream=stream)
        torch.cuda.synchronize()
        if not torch.equal(src, dst):
            raise RuntimeError("reference copy mismatch")
        out["copy_reference_bytes"] = {"read": src.numel() * 4, "write": dst.numel() * 4}
        del src, dst
    out["cpu_baseline"] = cpu_baseline(layer, I0, K0, macs, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def cpu_baseline(layer, I, K, macs, seconds):
    """The oracle's direct convolution, as it stands, on the host cores: the
    full layer, repeated until about `seconds` of CPU work."""
    if seconds <= 0:
        return None
    import oracle
    from paper_1706_06873_amd import workloads as wl

    Ia, Ka = wl.to_oracle_array(I), wl.to_oracle_array(K)
    reps, t_total = 0, 0.0
    while t_total < seconds or reps == 0:
        t0 = time.perf_counter()
        oracle.conv2d_direct(Ia, Ka, layer.s_h, layer.s_w)
        t_total += time.perf_counter() - t0
        reps += 1
        if reps >= 1000:
            break
    out = {"value": round(2.0 * macs * reps / t_total / 1e12, 6), "unit": "TFLOP/s",
           "cores": oracle.num_threads(), "kind": "oracle",
           "sample": "full %s layer (all %d images), direct fp64-accumulated convolution, "
                     "%d repetition(s) in %.1f s" % (layer.name, layer.i_n, reps, t_total),
           "cpu_model": cpu_model()}
    # the oracle's lowering (a plain copy loop): bytes of I read + L written per second, on
    # all the cores above and on one
    nbytes = Ia.nbytes * (1 + oracle.lowered_elems(*layer.dims) / Ia.size)
    for key, threads in (("lowering_gbps_all_cores", out["cores"]), ("lowering_gbps_1_core", 1)):
        oracle.set_num_threads(threads)
        reps, t = 0, 0.0
        while t < 0.5 or reps < 2:
            t0 = time.perf_counter()
            oracle.mec_lower(Ia, layer.k_h, layer.k_w, layer.k_c, layer.s_h, layer.s_w)
            t += time.perf_counter() - t0
            reps += 1
        out[key] = round(nbytes * reps / t / 1e9, 2)
    oracle.set_num_threads(out["cores"])
    return out


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
