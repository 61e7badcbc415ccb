"""Timing suite over the paper's benchmark layers on one MI355X.

    python -m paper_1706_06873_amd.suite table2 [--batch 32] [--dtype f32|bf16|both] [--yardstick]
    python -m paper_1706_06873_amd.suite stride [--batch 32] [--dtype f32]
    python -m paper_1706_06873_amd.suite resnet101 [--batch 1] [--dtype f32]
    python -m paper_1706_06873_amd.suite train [--layers resnet_mid,cv9,...] [--yardstick]

``table2`` runs the twelve layers of Table 2 (cv1-cv12), ``stride`` runs cv1
(227x227x3 input, 11x11x96 kernel) with s_h = s_w = 1..10 as in Fig. 4(a),
``resnet101`` runs the five layers of Table 3 (cv4, cv9-cv12) and ends with a
summary line weighing each layer by its count in ResNet-101, as Table 3 does:
weighted workspace (MiB) and weighted time of MEC against im2col. ``train``
times the training passes (fp32) per layer, each call between HIP events:
``conv2d_dgrad`` and ``conv2d_wgrad`` whole, and their parts -- the dL
products against K and the fold (the input gradient's general path; layers
taking the sub-pixel phases of the padded gradient run those instead), the
lowering and the partial A_h^T G_h sums with their reduction; with
``--yardstick`` it also times torch's own convolution gradients (the vendor
library) on the same shapes in NCHW, for context. ``table2 --yardstick`` (and
the other forward modes) also times the vendor GEMM (hipBLASLt through torch)
on the same im2col matrix, for context: im2col + vendor GEMM.
For every layer it times MEC from L (compact lowering + slab products), MEC
fused, and the im2col baseline (im2col lowering + one product through the
same kernels), each kernel between HIP events on its stream, on seeded
synthetic inputs already in device memory (every operand a kernel reads
rotating over at least 512 MB of buffer sets, twice the last-level cache, and
O over sets that make the fused form's operands span 1 GiB, after untimed
launches that let the clocks settle, as the benchmark does), and prints one
JSON line with the times, the effective TFLOP/s (2 x MAC / time) and the
workspace of MEC against im2col. Parity of every one of these shapes with the CPU oracle is
checked by the GPU tests, not here.
"""
import argparse
import dataclasses
import json
import sys
import time

import torch

import paper_1706_06873_amd as mec
from paper_1706_06873_amd import workloads as wl
from paper_1706_06873_amd.timing import HipEvent


MIN_ROTATION_BYTES = 1 << 30   # I, K and O of the fused form, together
READ_ROTATION_BYTES = 1 << 29  # each operand a kernel reads, on its own
MAX_SETS = 256


def _auto_sets(I0, K0, o_elems):
    """Sets of O: one rotation through I, K and O of the fused form spans at
    least 1 GiB (between 2 and MAX_SETS)."""
    foot = I0.numel() * I0.element_size() + K0.numel() * K0.element_size() + 4 * o_elems
    return max(2, min(MAX_SETS, -(-MIN_ROTATION_BYTES // foot)))


def _read_sets(nbytes):
    """Sets of an operand that a kernel reads (I, K, L or M): one rotation
    through them spans at least 512 MB, twice the 256 MB last-level cache, so
    no launch finds it there from an earlier one (between 2 and MAX_SETS)."""
    return max(2, min(MAX_SETS, -(-READ_ROTATION_BYTES // max(1, nbytes))))


def _time_layer(layer, reps, warmup, sets, yardstick=False, settle=0.2):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = layer.dims
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    dt = mec.BF16 if layer.dtype == "bf16" else mec.F32
    macs = i_n * o_h * o_w * k_c * k_h * k_w * i_c
    P = k_h * k_w * i_c
    dev = torch.device("cuda:0")
    I0, K0 = wl.make_inputs(layer)
    es = I0.element_size()
    if sets > 0:  # one count for every operand
        n_I = n_K = n_O = n_L = n_M = sets
    else:
        n_I, n_K = _read_sets(I0.numel() * es), _read_sets(K0.numel() * es)
        n_O = _auto_sets(I0, K0, i_n * o_h * o_w * k_c)
        n_L, n_M = _read_sets(i_n * o_w * i_h * k_w * i_c * es), _read_sets(i_n * o_w * o_h * P * es)
    Is = [I0.to(dev) if j == 0 else I0.to(dev).clone() for j in range(n_I)]
    Ks = [K0.to(dev) for _ in range(n_K)]
    Os = [torch.empty((i_n, o_h, o_w, k_c), dtype=torch.float32, device=dev) for _ in range(n_O)]
    nsets = {"I": n_I, "K": n_K, "O": n_O}
    launch = [0]  # launch k takes entry k of each list modulo its length

    def next_bufs(Ws):
        k = launch[0]
        launch[0] += 1
        b = dict(I=Is[k % n_I], K=Ks[k % n_K], O=Os[k % n_O])
        if Ws:
            b["W"] = Ws[k % len(Ws)]
        return b

    stream = torch.cuda.Stream(device=dev)
    res = {}
    for algo in ("lowered", "fused", "im2col"):
        Ws = None
        if algo == "lowered":
            Ws = [torch.empty((i_n, o_w, i_h, k_w, i_c), dtype=I0.dtype, device=dev) for _ in range(n_L)]
            nsets["L"] = n_L
        elif algo == "im2col":
            Ws = [torch.empty((i_n, o_w, o_h, k_h, k_w, i_c), dtype=I0.dtype, device=dev) for _ in range(n_M)]
            nsets["M"] = n_M

        def run(b, ev=None):
            rec = (lambda i: ev[i].record(stream)) if ev else (lambda i: None)
            rec(0)
            if algo == "fused":
                mec.conv2d(b["I"], b["K"], s_h, s_w, algo="fused", O=b["O"], stream=stream)
                rec(1)
                rec(2)
                return
            if algo == "lowered":
                mec.lower(b["I"], k_h, k_w, k_c, s_h, s_w, L=b["W"], stream=stream)
            else:
                mec.im2col(b["I"], k_h, k_w, k_c, s_h, s_w, M=b["W"], stream=stream)
            rec(1)
            if algo == "lowered":
                mec.gemm(b["W"], b["K"], i_h, i_w, s_h, s_w, O=b["O"], stream=stream)
            else:
                mec.gemm(b["W"].view(i_n, o_w, o_h, 1, P), b["K"].view(1, 1, P, k_c), o_h, o_w,
                         1, 1, O=b["O"], stream=stream)
            rec(2)

        with torch.cuda.stream(stream):
            # untimed launches until the clocks have settled, then the warm-up
            t0 = time.time()
            k = 0
            while time.time() - t0 < settle:
                run(next_bufs(Ws))
                k += 1
                if k % 16 == 0:
                    torch.cuda.synchronize()
            for w in range(warmup):
                run(next_bufs(Ws))
            torch.cuda.synchronize()
            evs = [[HipEvent() for _ in range(3)] for _ in range(reps)]
            bufs = [next_bufs(Ws) for _ in range(reps)]
            for r in range(reps):
                run(bufs[r], evs[r])
            torch.cuda.synchronize()
        tot = sorted(e[0].elapsed_time(e[2]) * 1e3 for e in evs)
        low = sorted(e[0].elapsed_time(e[1]) * 1e3 for e in evs)
        prod = sorted(e[1].elapsed_time(e[2]) * 1e3 for e in evs)
        med = lambda v: v[len(v) // 2]
        res[algo] = {"us": round(med(tot), 2), "tflops": round(2.0 * macs / (med(tot) * 1e-6) / 1e12, 2)}
        if algo != "fused":
            res[algo]["lower_us"] = round(med(low), 2)
            res[algo]["product_us"] = round(med(prod), 2)
        if algo == "im2col" and yardstick:
            # context only: the vendor GEMM (hipBLASLt through torch) on the same
            # im2col matrix, rows (n, x, y); its result is not in O's layout
            Mv, Kv = bufs[0]["W"].view(-1, P), bufs[0]["K"].view(P, k_c)
            with torch.cuda.stream(stream):
                for _ in range(warmup):
                    torch.matmul(Mv, Kv)
                torch.cuda.synchronize()
                gev = [[HipEvent() for _ in range(2)] for _ in range(reps)]
                for r in range(reps):
                    gev[r][0].record(stream)
                    torch.matmul(Mv, Kv)
                    gev[r][1].record(stream)
                torch.cuda.synchronize()
            g = med(sorted(e[0].elapsed_time(e[1]) * 1e3 for e in gev))
            res["im2col"]["vendor_gemm_us"] = round(g, 2)
            res["im2col"]["im2col_plus_vendor_gemm_us"] = round(med(low) + g, 2)
        del Ws, bufs
        torch.cuda.empty_cache()
    ws_mec = mec.workspace_bytes(*layer.dims, dtype=dt, algo=mec.LOWERED)
    ws_im2col = mec.im2col_bytes(*layer.dims, dtype=dt)
    return {"layer": layer.name, "dims": list(layer.dims), "o": [o_h, o_w], "dtype": layer.dtype,
            "gflop": round(2.0 * macs / 1e9, 3), "sets": nsets, "workspace_mec": ws_mec,
            "workspace_im2col": ws_im2col, "im2col_over_mec": round(ws_im2col / ws_mec, 3),
            "timings": res,
            "mec_speedup_vs_im2col": round(res["im2col"]["us"] / min(res["lowered"]["us"],
                                                                       res["fused"]["us"]), 3)}


def _time_train(layer, reps, warmup, yardstick):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = layer.dims
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    macs = i_n * o_h * o_w * k_c * k_h * k_w * i_c
    dev = torch.device("cuda:0")
    I0, K0 = wl.make_inputs(layer)
    G0 = torch.rand((i_n, o_h, o_w, k_c), generator=torch.Generator().manual_seed(layer.seed + 7))
    I, K, G = I0.to(dev), K0.to(dev), (G0 * 2 - 1).to(dev)
    dI = torch.empty_like(I)
    dK = torch.empty_like(K)
    dL = torch.empty((i_n, o_w, i_h, k_w, i_c), dtype=torch.float32, device=dev)
    L = torch.empty_like(dL)
    part = torch.empty(mec.grad_workspace_bytes(*layer.dims, grad_pass=mec.GRAD_KERNEL_FROM_L),
                       dtype=torch.uint8, device=dev)
    ws_i = torch.empty(mec.grad_workspace_bytes(*layer.dims, grad_pass=mec.GRAD_INPUT),
                       dtype=torch.uint8, device=dev)
    ws_k = torch.empty(mec.grad_workspace_bytes(*layer.dims, grad_pass=mec.GRAD_KERNEL),
                       dtype=torch.uint8, device=dev)
    stream = torch.cuda.Stream(device=dev)
    steps = {
        "conv2d_dgrad": lambda: mec.conv2d_dgrad(G, K, i_h, i_w, s_h, s_w, dI=dI, workspace=ws_i,
                                                 stream=stream),
        "conv2d_wgrad": lambda: mec.conv2d_wgrad(I, G, k_h, k_w, s_h, s_w, dK=dK, workspace=ws_k,
                                                 stream=stream),
        "dgrad_products": lambda: mec.dgrad_gemm(G, K, i_h, i_w, s_h, s_w, dL=dL, stream=stream),
        "fold": lambda: mec.fold(dL, i_w, s_w, dI=dI, stream=stream),
        "lower": lambda: mec.lower(I, k_h, k_w, k_c, s_h, s_w, L=L, stream=stream),
        "wgrad_products": lambda: mec.wgrad_gemm(L, G, k_h, i_w, s_h, s_w, dK=dK, workspace=part,
                                                 stream=stream),
    }
    if yardstick:
        In = I.permute(0, 3, 1, 2).contiguous()
        Kn = K.permute(3, 2, 0, 1).contiguous()
        Gn = G.permute(0, 3, 1, 2).contiguous()
        steps["vendor_dgrad"] = lambda: torch.nn.grad.conv2d_input(In.shape, Kn, Gn, stride=(s_h, s_w))
        steps["vendor_wgrad"] = lambda: torch.nn.grad.conv2d_weight(In, Kn.shape, Gn, stride=(s_h, s_w))
    times = {}
    with torch.cuda.stream(stream):
        for name, fn in steps.items():
            for _ in range(warmup):
                fn()
            torch.cuda.synchronize()
            ev = [(HipEvent(), HipEvent())
                  for _ in range(reps)]
            for a, b in ev:
                a.record(stream)
                fn()
                b.record(stream)
            torch.cuda.synchronize()
            t = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
            times[name] = round(t[len(t) // 2], 2)
    tf = lambda us: round(2.0 * macs / (us * 1e-6) / 1e12, 2)
    out = {"layer": layer.name, "dims": list(layer.dims), "gflop": round(2.0 * macs / 1e9, 3),
           "us": times,
           "dgrad_us": times["conv2d_dgrad"], "wgrad_us": times["conv2d_wgrad"],
           "dgrad_tflops": tf(times["conv2d_dgrad"]), "wgrad_tflops": tf(times["conv2d_wgrad"]),
           "dgrad_workspace": ws_i.numel(), "wgrad_workspace": ws_k.numel()}
    out["dgrad_products_tflops"] = tf(times["dgrad_products"])
    out["wgrad_products_tflops"] = tf(times["wgrad_products"])
    out["dgrad_products_frac_fp32_mfma"] = round(out["dgrad_products_tflops"] / 157.3, 3)
    out["wgrad_products_frac_fp32_mfma"] = round(out["wgrad_products_tflops"] / 157.3, 3)
    fold_bytes = 4 * (dL.numel() + dI.numel())
    out["fold_tbps"] = round(fold_bytes / (times["fold"] * 1e-6) / 1e12, 3)
    if yardstick:
        out["vendor_dgrad_tflops"] = tf(times["vendor_dgrad"])
        out["vendor_wgrad_tflops"] = tf(times["vendor_wgrad"])
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("which", choices=["table2", "stride", "resnet101", "train"])
    ap.add_argument("--yardstick", action="store_true",
                    help="train: also time torch's convolution gradients; forward modes: "
                         "the vendor GEMM on the im2col matrix")
    ap.add_argument("--batch", type=int, default=None,
                    help="images per layer (default 32; 1 for resnet101, as in Table 3)")
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16", "both"])
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--sets", type=int, default=0,
                    help="rotating buffer sets of every operand (0: enough that each operand read spans 512 MB and O with I and K 1 GiB, at most %d)"
                         % MAX_SETS)
    ap.add_argument("--settle", type=float, default=0.2,
                    help="seconds of untimed launches per layer and algorithm before the warm-up")
    ap.add_argument("--layers", default="", help="comma-separated subset")
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        print("the suite needs a GPU", file=sys.stderr)
        return 1
    dtypes = ["f32", "bf16"] if args.dtype == "both" else [args.dtype]
    batch = args.batch or (1 if args.which == "resnet101" else 32)
    if args.which == "train":
        names = args.layers.split(",") if args.layers else ["resnet_mid", "alexnet_conv1",
                                                            "vgg_first"] + list(wl.TABLE2)
        for name in names:
            layer = wl.LAYERS[name] if name in wl.LAYERS else wl.table2_layer(name, batch)
            if args.batch and name in wl.LAYERS:
                layer = dataclasses.replace(layer, i_n=args.batch)
            print(json.dumps(_time_train(layer, args.reps, args.warmup, args.yardstick)),
                  flush=True)
        return 0
    if args.which == "table2":
        names = args.layers.split(",") if args.layers else list(wl.TABLE2)
        layers = [wl.table2_layer(n, batch, d) for d in dtypes for n in names]
    elif args.which == "resnet101":
        names = args.layers.split(",") if args.layers else list(wl.TABLE3_WEIGHTS)
        layers = [wl.table2_layer(n, batch, d) for d in dtypes for n in names]
    else:
        strides = [int(x) for x in args.layers.split(",")] if args.layers else list(range(1, 11))
        layers = [wl.table2_layer("cv1", batch, d, stride=s) for d in dtypes for s in strides]
    rows = []
    for layer in layers:
        rows.append(_time_layer(layer, args.reps, args.warmup, args.sets, args.yardstick, args.settle))
        print(json.dumps(rows[-1]), flush=True)
    if args.which == "resnet101":
        for d in dtypes:
            print(json.dumps(weighted_summary([r for r in rows if r["dtype"] == d], batch)),
                  flush=True)
    return 0


def weighted_summary(rows, batch):
    """Table 3's weighted totals: each layer's workspace and time times its
    count in ResNet-101, summed, for MEC (from L and fused) and im2col."""
    mib = 2.0 ** 20
    tot = {"workspace_im2col_mib": 0.0, "workspace_mec_mib": 0.0, "im2col_us": 0.0,
           "mec_lowered_us": 0.0, "mec_fused_us": 0.0}
    for r in rows:
        wgt = wl.TABLE3_WEIGHTS[r["layer"]]
        tot["workspace_im2col_mib"] += wgt * r["workspace_im2col"] / mib
        tot["workspace_mec_mib"] += wgt * r["workspace_mec"] / mib
        tot["im2col_us"] += wgt * r["timings"]["im2col"]["us"]
        tot["mec_lowered_us"] += wgt * r["timings"]["lowered"]["us"]
        tot["mec_fused_us"] += wgt * r["timings"]["fused"]["us"]
    out = {"summary": "ResNet-101 weighted (Table 3 layers and weights)", "batch": batch,
           "dtype": rows[0]["dtype"] if rows else None,
           "layers": {r["layer"]: wl.TABLE3_WEIGHTS[r["layer"]] for r in rows}}
    out.update({k: round(v, 3) for k, v in tot.items()})
    if tot["workspace_mec_mib"] > 0:
        out["workspace_ratio"] = round(tot["workspace_im2col_mib"] / tot["workspace_mec_mib"], 3)
    if tot["mec_lowered_us"] > 0:
        out["time_ratio_lowered"] = round(tot["im2col_us"] / tot["mec_lowered_us"], 3)
        out["time_ratio_fused"] = round(tot["im2col_us"] / tot["mec_fused_us"], 3)
    return out


if __name__ == "__main__":
    sys.exit(main())
