"""Timing suite over the paper's benchmark layers on one MI355X.

    python -m paper_1706_06873_amd.suite table2 [--batch 32] [--dtype f32|bf16|both]
    python -m paper_1706_06873_amd.suite stride [--batch 32] [--dtype f32]
    python -m paper_1706_06873_amd.suite resnet101 [--batch 1] [--dtype f32]

``table2`` runs the twelve layers of Table 2 (cv1-cv12), ``stride`` runs cv1
(227x227x3 input, 11x11x96 kernel) with s_h = s_w = 1..10 as in Fig. 4(a),
``resnet101`` runs the five layers of Table 3 (cv4, cv9-cv12) and ends with a
summary line weighing each layer by its count in ResNet-101, as Table 3 does:
weighted workspace (MiB) and weighted time of MEC against im2col.
For every layer it times MEC from L (compact lowering + slab products), MEC
fused, and the im2col baseline (im2col lowering + one product through the
same kernels), each kernel between HIP events on its stream, on seeded
synthetic inputs already in device memory, and prints one JSON line with the
times, the effective TFLOP/s (2 x MAC / time) and the workspace of MEC
against im2col. Parity of every one of these shapes with the CPU oracle is
checked by the GPU tests, not here.
"""
import argparse
import json
import sys

import torch

import paper_1706_06873_amd as mec
from paper_1706_06873_amd import workloads as wl


def _time_layer(layer, reps, warmup, sets):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = layer.dims
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    dt = mec.BF16 if layer.dtype == "bf16" else mec.F32
    macs = i_n * o_h * o_w * k_c * k_h * k_w * i_c
    P = k_h * k_w * i_c
    dev = torch.device("cuda:0")
    I0, K0 = wl.make_inputs(layer)
    bufs = [dict(I=I0.to(dev) if j == 0 else I0.to(dev).clone(), K=K0.to(dev),
                 O=torch.empty((i_n, o_h, o_w, k_c), dtype=torch.float32, device=dev))
            for j in range(sets)]
    stream = torch.cuda.Stream(device=dev)
    res = {}
    for algo in ("lowered", "fused", "im2col"):
        if algo == "lowered":
            for b in bufs:
                b["W"] = torch.empty((i_n, o_w, i_h, k_w, i_c), dtype=I0.dtype, device=dev)
        elif algo == "im2col":
            for b in bufs:
                b["W"] = torch.empty((i_n, o_w, o_h, k_h, k_w, i_c), dtype=I0.dtype, device=dev)

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
            for w in range(warmup):
                run(bufs[w % sets])
            torch.cuda.synchronize()
            evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
            for r in range(reps):
                run(bufs[r % sets], evs[r])
            torch.cuda.synchronize()
        tot = sorted(e[0].elapsed_time(e[2]) * 1e3 for e in evs)
        low = sorted(e[0].elapsed_time(e[1]) * 1e3 for e in evs)
        prod = sorted(e[1].elapsed_time(e[2]) * 1e3 for e in evs)
        med = lambda v: v[len(v) // 2]
        res[algo] = {"us": round(med(tot), 2), "tflops": round(2.0 * macs / (med(tot) * 1e-6) / 1e12, 2)}
        if algo != "fused":
            res[algo]["lower_us"] = round(med(low), 2)
            res[algo]["product_us"] = round(med(prod), 2)
        for b in bufs:
            b.pop("W", None)
        torch.cuda.empty_cache()
    ws_mec = mec.workspace_bytes(*layer.dims, dtype=dt, algo=mec.LOWERED)
    ws_im2col = mec.im2col_bytes(*layer.dims, dtype=dt)
    return {"layer": layer.name, "dims": list(layer.dims), "o": [o_h, o_w], "dtype": layer.dtype,
            "gflop": round(2.0 * macs / 1e9, 3), "workspace_mec": ws_mec,
            "workspace_im2col": ws_im2col, "im2col_over_mec": round(ws_im2col / ws_mec, 3),
            "timings": res,
            "mec_speedup_vs_im2col": round(res["im2col"]["us"] / min(res["lowered"]["us"],
                                                                       res["fused"]["us"]), 3)}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("which", choices=["table2", "stride", "resnet101"])
    ap.add_argument("--batch", type=int, default=None,
                    help="images per layer (default 32; 1 for resnet101, as in Table 3)")
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16", "both"])
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--sets", type=int, default=2, help="rotating buffer sets")
    ap.add_argument("--layers", default="", help="comma-separated subset")
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        print("the suite needs a GPU", file=sys.stderr)
        return 1
    dtypes = ["f32", "bf16"] if args.dtype == "both" else [args.dtype]
    batch = args.batch or (1 if args.which == "resnet101" else 32)
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
        rows.append(_time_layer(layer, args.reps, args.warmup, args.sets))
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
