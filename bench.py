"""Benchmark of the MEC hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--layer NAME] [--algo lowered|fused|im2col]
                    [--sweep all|none]

One step is one MEC convolution of the layer on inputs already resident in
device memory: the compact lowering of I into L followed by the o_h slab
products (mec_lower + mec_gemm, exactly the two kernels
mec_conv2d(MEC_ALGO_LOWERED) enqueues), or the fused kernel
(mec_conv2d(MEC_ALGO_FUSED)). The default layer is the largest fp32 one,
AlexNet conv1 (i_n=128, 227x227x3, 11x11x96 kernel, stride 4), from L.
Every operand a kernel reads rotates over at least 512 MB of buffer sets
(twice the 256 MB memory-attached last-level cache), so that no launch finds
it in that cache from an earlier one.

Timing, with HIP events on the stream the kernels run on (created without the
system-scope fence, so recording one adds no cache maintenance to what it
measures):
  * untimed steps for --settle seconds (the GPU's clocks leave their idle
    state), then the W warm-up steps;
  * the K timed steps run between two events with nothing else on the stream
    (ms_per_step, value);
  * each kernel's duration is then timed on its own: K launches of that one
    kernel back to back between two events (the per-kernel averages of the
    rooflines), the lowering first so that the products read a lowered L.

Prints ONE JSON line: effective TFLOP/s (2*MAC/time) of the whole step, the
workspace bytes against im2col's, the roofline of the dominant kernel (the slab
products) and of the lowering, the CPU oracle's rate on the host cores (a
baseline, not the target) and, under "configs", the same step and per-kernel
figures for every synthetic layer (tiny, resnet_mid, vgg_first, alexnet_conv1,
deep_bf16), each from L and fused.
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
DEFAULT_LAYER = "alexnet_conv1"
MIN_ROTATION_BYTES = 1 << 30   # bytes each kernel's rotating buffers span, at least
READ_ROTATION_BYTES = 1 << 29  # bytes each operand a kernel reads rotates over, at least
SWEEP_ALGOS = ("lowered", "fused")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--settle", type=float, default=0.3,
                    help="seconds of untimed steps before the warm-up steps (clocks leave idle)")
    ap.add_argument("--layer", default=DEFAULT_LAYER)
    ap.add_argument("--algo", default="lowered", choices=["lowered", "fused", "im2col"],
                    help="MEC from L (default), MEC fused, or the im2col + product baseline")
    ap.add_argument("--sweep", default="all", choices=["all", "none"],
                    help="also time every synthetic layer from L and fused (default), or not")
    ap.add_argument("--sets", type=int, default=4,
                    help="rotating buffer sets, at least (more where a kernel's buffers are small)")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the layer's batch size i_n (0 keeps the layer's own)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time for the oracle baseline (0 skips it)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one plain device-to-device copy of this many MiB "
                         "(a known-size reference for rocprofv3 byte counters)")
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


def profile_path(dtype, layer_name, algo):
    return os.path.join(REPO, "profiles", "slab_gemm_%s_%s_%s.md" % (dtype, layer_name, algo))


def load_traffic(dtype, layer_name, algo, digest):
    """Per-launch HBM bytes of the slab products and of the lowering from the
    layer's profile summary: its lines 'traffic-json:' (products) and
    'traffic-lower-json:' (lowering) hold FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch), the factors that make each counter read a plain copy of known
    size correctly, and the digest of the sources the counters were taken on.
    A figure taken on other sources is not reported (None)."""
    path = profile_path(dtype, layer_name, algo)
    out = {"products": None, "lower": None, "products_kernel": None, "lower_kernel": None}
    if not os.path.exists(path):
        return out
    with open(path) as f:
        for line in f:
            for key, tag in (("products", "traffic-json:"), ("lower", "traffic-lower-json:")):
                if line.startswith(tag):
                    t = json.loads(line[len(tag):])
                    if t.get("workload") == "%s %s" % (layer_name, algo) and t.get("csrc_sha256") == digest:
                        out[key] = int(round((t["fetch_kib"] * t["fetch_scale"] +
                                              t["write_kib"] * t["write_scale"]) * 1024))
                        out[key + "_kernel"] = t.get("kernel")
    return out


def rotation_sets(nbytes, nsets):
    """Buffer sets for an operand of `nbytes` that a kernel reads: enough that
    one rotation through them spans READ_ROTATION_BYTES, at least `nsets`, at
    most 256."""
    return min(max(nsets, -(-READ_ROTATION_BYTES // max(nbytes, 1))), 256)


class Config:
    """One layer and algorithm: sizes, algorithmic work, buffers and launches."""

    def __init__(self, mec, wl, torch, layer, algo, nsets, dev, stream):
        self.mec, self.torch, self.layer, self.algo, self.stream = mec, torch, layer, algo, stream
        self.dims = dims = layer.dims
        i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
        self.o_h, self.o_w = o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
        self.dt_code = mec.BF16 if layer.dtype == "bf16" else mec.F32
        self.es = es = 2 if layer.dtype == "bf16" else 4
        self.macs = i_n * o_h * o_w * k_c * k_h * k_w * i_c
        self.flops = 2.0 * self.macs
        self.ws_lowered = mec.workspace_bytes(*dims, dtype=self.dt_code, algo=mec.LOWERED)
        self.ws_im2col = mec.im2col_bytes(*dims, dtype=self.dt_code)
        self.ws = {"lowered": self.ws_lowered, "fused": 0, "im2col": self.ws_im2col}[algo]
        self.size_I = i_n * i_h * i_w * i_c
        self.size_K = k_h * k_w * i_c * k_c
        self.size_O = i_n * o_h * o_w * k_c
        self.size_W = self.ws // es   # |L| or |M| elements (0 fused)
        self.P = k_h * k_w * i_c      # im2col row length
        self.I0, self.K0 = wl.make_inputs(layer)
        # Buffer sets. Every operand a kernel reads (I and K; the workspace,
        # which the products read) rotates over at least READ_ROTATION_BYTES
        # on its own, twice the 256 MB memory-attached last-level cache, so no
        # launch finds it there from an earlier one; O, only written, over the
        # sets that make the products' operands span MIN_ROTATION_BYTES
        # together. Launch k takes entry k of each list modulo its length.
        # (Over 5 sets, vgg_first's 9.8 MB I stayed in that cache while 1 GiB
        # of O went through it: its fused products took 44 us there against
        # 62 us with I read from HBM.)
        read_sets = lambda nbytes: rotation_sets(nbytes, nsets)
        src = self.size_I if algo == "fused" else self.size_W
        prod_foot = es * (src + self.size_K) + 4 * self.size_O
        n_o = min(max(nsets, -(-MIN_ROTATION_BYTES // prod_foot)), 256)
        self.Is = [self.I0.to(dev) if j == 0 else self.I0.to(dev).clone()
                   for j in range(read_sets(es * self.size_I))]
        self.Ks = [self.K0.to(dev) for _ in range(read_sets(es * self.size_K))]
        self.Os = [torch.empty((i_n, o_h, o_w, k_c), dtype=torch.float32, device=dev) for _ in range(n_o)]
        # the workspace the library asks for, in bytes
        self.Ws = [] if algo == "fused" else [torch.empty(self.ws, dtype=torch.uint8, device=dev)
                                               for _ in range(read_sets(self.ws))]
        self.nsets = {"I": len(self.Is), "K": len(self.Ks), "W": len(self.Ws), "O": n_o}
        self.k = 0

    def next(self):
        """The buffers of the next launch."""
        k = self.k
        self.k += 1
        b = dict(I=self.Is[k % len(self.Is)], K=self.Ks[k % len(self.Ks)], O=self.Os[k % len(self.Os)])
        if self.Ws:
            b["W"] = self.Ws[k % len(self.Ws)]
        return b

    def lower(self, b):
        m, (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w) = self.mec, self.dims
        if self.algo == "im2col":
            M = b["W"].view(self.I0.dtype).view(i_n, self.o_w, self.o_h, k_h, k_w, i_c)
            m.im2col(b["I"], k_h, k_w, k_c, s_h, s_w, M=M, stream=self.stream)
        else:
            L = b["W"].view(self.I0.dtype).view(i_n, self.o_w, i_h, k_w, i_c)
            m.lower(b["I"], k_h, k_w, k_c, s_h, s_w, L=L, stream=self.stream)

    def products(self, b):
        m, (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w) = self.mec, self.dims
        if self.algo == "fused":
            m.conv2d(b["I"], b["K"], s_h, s_w, algo="fused", O=b["O"], stream=self.stream)
        elif self.algo == "im2col":
            # the product of M and K: MEC's product phase of the 1x1 convolution
            # whose pixels (n, y, x) carry the patches as channels
            M = b["W"].view(self.I0.dtype).view(i_n, self.o_w, self.o_h, 1, self.P)
            m.gemm(M, b["K"].view(1, 1, self.P, k_c), self.o_h, self.o_w, 1, 1, O=b["O"],
                   stream=self.stream)
        else:
            L = b["W"].view(self.I0.dtype).view(i_n, self.o_w, i_h, k_w, i_c)
            m.gemm(L, b["K"], i_h, i_w, s_h, s_w, O=b["O"], stream=self.stream)

    def step(self, b):
        if self.algo != "fused":
            self.lower(b)
        self.products(b)

    def alg_bytes(self):
        """Algorithmic HBM bytes of the products kernel per launch: each
        element of L (or I when fused, or M) and K read once, O written once."""
        src = self.size_I if self.algo == "fused" else self.size_W
        return self.es * (src + self.size_K) + 4 * self.size_O

    def lower_bytes(self):
        return self.es * (self.size_I + self.size_W)


def timed(HipEvent, stream, fn, cfg, n):
    """Average ms of n calls of fn over the rotating buffers, between two events."""
    import torch
    bufs = [cfg.next() for _ in range(n)]
    start, end = HipEvent(), HipEvent()
    torch.cuda.synchronize()
    start.record(stream)
    for b in bufs:
        fn(b)
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / n


def settle(cfg, seconds):
    """Untimed steps for about `seconds` of wall time, so that the GPU's clocks
    have left their idle state before the warm-up steps; returns the count."""
    import torch
    n, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            cfg.step(cfg.next())
            n += 1
        torch.cuda.synchronize()
    return n


def measure(cfg, HipEvent, steps, warmup, digest, settle_s):
    """Step time and per-kernel durations of one configuration, with rooflines."""
    import torch
    with torch.cuda.stream(cfg.stream):
        settled = settle(cfg, settle_s)
        for w in range(warmup):
            cfg.step(cfg.next())
        t0 = time.perf_counter()
        ms_step = timed(HipEvent, cfg.stream, cfg.step, cfg, steps)
        wall = time.perf_counter() - t0
        lower_ms = None
        if cfg.algo != "fused":
            lower_ms = timed(HipEvent, cfg.stream, cfg.lower, cfg, steps)
        prod_ms = timed(HipEvent, cfg.stream, cfg.products, cfg, steps)

    layer = cfg.layer
    peak = PEAK_TFLOPS[layer.dtype]
    traffic = load_traffic(layer.dtype, layer.name, cfg.algo, digest)
    # the kernel's own name where the layer's profile (taken on these sources)
    # recorded it, else its family
    kname = traffic["products_kernel"] or "slab_gemm_%s_*kernel" % layer.dtype
    kname += {"fused": " (from I)", "im2col": " (im2col product, k_h = 1)", "lowered": ""}[cfg.algo]
    ab = cfg.alg_bytes()
    ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)
    if layer.name == "tiny":
        bound = "launch"   # 450 flops: the launch, not a roofline, is what it costs
    else:
        bound = "mfma" if cfg.flops / ab >= ridge else "hbm"
    if bound == "hbm":
        ach = ab / (prod_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": kname, "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4)}
    else:
        ach = cfg.flops / (prod_ms * 1e-3) / 1e12
        roof = {"bound": bound, "kernel": kname, "achieved": round(ach, 3), "peak": peak,
                "unit": "TFLOP/s", "frac": round(ach / peak, 4) if bound == "mfma" else None}
    roof.update({"traffic": traffic["products"], "alg_flops": cfg.flops, "alg_bytes": ab,
                 "avg_ms": round(prod_ms, 5)})
    out = {"ms_per_step": round(ms_step, 5),
           "tflops": round(cfg.flops / (ms_step * 1e-3) / 1e12, 3),
           "settle_steps": settled,
           "wall_s": round(wall, 4),
           "gemm_ms": round(prod_ms, 5),
           "roofline": roof}
    if lower_ms is not None:
        lb = cfg.lower_bytes()
        gbs = lb / (lower_ms * 1e-3) / 1e9
        out["lower_ms"] = round(lower_ms, 5)
        out["roofline_lower"] = {
            "bound": "hbm" if layer.name != "tiny" else "launch",
            "kernel": "im2col_*_kernel" if cfg.algo == "im2col" else (traffic["lower_kernel"] or "lower_*_kernel"),
            "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 4) if layer.name != "tiny" else None,
            "traffic": traffic["lower"], "alg_bytes": lb}
    out["buffer_sets"] = cfg.nsets
    out["workspace_bytes"] = cfg.ws
    out["im2col_bytes"] = cfg.ws_im2col
    out["workspace_vs_mec_closed_form"] = round(cfg.ws / cfg.ws_lowered, 4) if cfg.algo == "lowered" else None
    return out


def workload_name(layer, o_h, o_w):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = layer.dims
    return ("%s: i_n=%d, I %dx%dx%d (%s), K %dx%dx%dx%d, s=%d/%d, o=%dx%d"
            % (layer.name, i_n, i_h, i_w, i_c, layer.dtype, k_h, k_w, i_c, k_c, s_h, s_w, o_h, o_w))


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
    from paper_1706_06873_amd.timing import HipEvent

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    layer = wl.LAYERS[args.layer]
    if args.batch > 0:
        import dataclasses
        layer = dataclasses.replace(layer, i_n=args.batch)
    dev = torch.device("cuda:0")
    stream = torch.cuda.Stream(device=dev)  # default priority
    digest = csrc_digest()

    cfg = Config(mec, wl, torch, layer, args.algo, args.sets, dev, stream)
    torch.cuda.synchronize()
    head = measure(cfg, HipEvent, args.steps, args.warmup, digest, args.settle)
    if args.batch > 0:   # counters were taken at the layer's own batch
        head["roofline"]["traffic"] = None
        if "roofline_lower" in head:
            head["roofline_lower"]["traffic"] = None
    I0, K0, macs = cfg.I0, cfg.K0, cfg.macs
    value = cfg.flops / (head["ms_per_step"] * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": layer.dtype,
        "data": "synthetic (seeded, %s)" % layer.note,
        "config": {"workload": workload_name(layer, cfg.o_h, cfg.o_w),
                   "algo": args.algo, "buffer_sets": cfg.nsets},
        "workspace_bytes": cfg.ws,
        "im2col_bytes": cfg.ws_im2col,
        "workspace_vs_im2col": round(cfg.ws_im2col / cfg.ws_lowered, 4),
        "wall_s": head["wall_s"],
        "gemm_ms": head["gemm_ms"],
        "roofline": head["roofline"],
    }
    if "lower_ms" in head:
        out["lower_ms"] = head["lower_ms"]
        out["roofline_lower"] = head["roofline_lower"]
    del cfg
    torch.cuda.empty_cache()

    if args.sweep == "all":
        sweep = {}
        for name in wl.LAYER_ORDER:
            for algo in SWEEP_ALGOS:
                key = "%s/%s" % (name, algo)
                if name == layer.name and algo == args.algo and args.batch <= 0:
                    sweep[key] = dict(head, workload=out["config"]["workload"])
                    continue
                c = Config(mec, wl, torch, wl.LAYERS[name], algo, args.sets, dev, stream)
                r = measure(c, HipEvent, args.steps, args.warmup, digest, args.settle)
                r["workload"] = workload_name(c.layer, c.o_h, c.o_w)
                sweep[key] = r
                del c
                torch.cuda.empty_cache()
        out["configs"] = sweep

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
