"""Benchmark: effective TFLOP/s (nonzero blocks) of factorized sparse attention,
forward + backward with recomputation, on one MI355X.

One step = forward and backward over each of the two measured workloads:
  strided, n = 12,288, l = 128, B = 64, batch 2, 8 merged heads of 64
  fixed,   n = 65,536, l = 256, c = 32, B = 64, batch 1, 8 merged heads of 64
Inputs are seeded N(0, 1) bf16 tensors already resident in device memory; the
block layouts are built once before timing.  Every present B x B block is
credited 14 B^2 d FLOPs per (batch, head): 4 B^2 d forward (QK^T, PV) and
10 B^2 d backward (QK^T recomputed, dO V^T, P^T dO, dS^T Q, dS K).

Prints one JSON line.  The fp64 oracle is timed on the host cores on one
(batch, head) slice of each workload and scaled to the whole step.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective TFLOP/s (nonzero blocks) fwd+bwd and % bf16 MFMA peak at n=12288/65536"
PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
HBM_PEAK_GBS = 8000.0
BENCH_WORKLOADS = ("strided_n12288_l128_merged", "fixed_n65536_l256_c32_merged")


def heads_per_layout(w, n_layouts):
    """Heads reading each layout: alternating heads split A1 (layout 0) and A2;
    with a summary subblock per head, head h reads the layout of subblock
    h mod (l / c) (layout 1 + that subblock for the odd heads when they
    alternate)."""
    from paper_1904_10509_amd.inputs import FIXED_PER_HEAD, MODE_A1, MODE_INTERLEAVED
    sub = w.stride // w.summary if w.pattern == FIXED_PER_HEAD else 0
    counts = [0] * n_layouts
    for h in range(w.heads):
        if w.mode == MODE_INTERLEAVED:
            g = (1 + (h % sub if sub else 0)) if h % 2 else 0
        else:
            g = 0 if (w.mode == MODE_A1 or sub == 0) else h % sub
        counts[g] += 1
    return counts


def credited_flops(w, nnz):
    """14 B^2 d per present block per (batch, head), over the layout each head reads."""
    blocks = sum(z * w.batch * hpl for z, hpl in zip(nnz, heads_per_layout(w, len(nnz))))
    return 14.0 * w.block * w.block * w.d_head * blocks, 4.0 * w.block * w.block * w.d_head * blocks


def mfma_flops_upper_bound(w, nnz):
    """MFMA work the kernels issue per present block and (batch, head) when no
    part of a block is skipped: forward 2 products (QK^T, PV), dQ kernel 3
    (QK^T, dO V^T, dS K), dK/dV kernel 4 (QK^T, dO V^T, P^T dO, dS^T Q).  The
    kernels skip the products of 32-wide chunks in which no pair of a wave's
    rows and columns is attended, so the work issued is at most this."""
    blocks = sum(z * w.batch * hpl for z, hpl in zip(nnz, heads_per_layout(w, len(nnz))))
    return 18.0 * w.block * w.block * w.d_head * blocks


def attended_pairs(w):
    """sum_i |S_i| per (batch, head) for the merged sets of Sec. 4.3 (closed forms;
    with a summary subblock per head every head has the same count)."""
    import numpy as np
    from paper_1904_10509_amd.inputs import MODE_MERGED, STRIDED
    if w.mode != MODE_MERGED:
        return None
    i = np.arange(w.n, dtype=np.int64)
    if w.pattern == STRIDED:
        cnt = np.minimum(i, w.stride) + 1 + np.maximum(0, i // w.stride - 1)
    else:
        cnt = i % w.stride + 1 + (i // w.stride) * w.summary
    return int(cnt.sum())


def algorithmic_bwd_bytes(w):
    """Backward call: read Q, K, V, O, dO, LSE; write dQ, dK, dV; D written and read."""
    e = w.batch * w.heads * w.n
    return 8 * e * w.d_head * 2 + 3 * e * 4


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "traffic_sparse_attn_bwd_fixed_n65536.json")


def kernel_sources_sha256():
    """Digest of the HIP sources, to tell whether stored counter data is current."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_1904_10509_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(f.encode())
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload_name):
    """HBM bytes per backward call from the stored rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes (copy-calibrated), or None when absent or taken on other kernel sources."""
    try:
        with open(TRAFFIC_RECORD) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload_name or rec.get("source_sha256") != kernel_sources_sha256():
        return None
    return rec.get("bytes_per_launch")


def copy_calibration(torch, dev):
    """A copy-like elementwise kernel of known size (torch.neg: 256 MiB read,
    256 MiB written), run when counters are collected so FETCH_SIZE /
    WRITE_SIZE can be scaled to bytes."""
    src = torch.empty(128 << 20, dtype=torch.bfloat16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


def cpu_baseline(workloads, inputs, budget_s=10.0):
    """Time the fp64 oracle on whole (batch, head) slices of each workload, full
    sequence, slice after slice until about budget_s seconds of CPU work are
    spent (at least one slice per workload), and scale the mean time per slice
    by batch * heads to the whole step."""
    from oracle import oracle
    from paper_1904_10509_amd.inputs import as_oracle_array

    est_s, credited, parts, spent = 0.0, 0.0, [], 0.0
    for w, nnz, x in workloads:
        times = []
        for sidx in range(w.batch * w.heads):
            b, h = divmod(sidx, w.heads)
            sl = [as_oracle_array(x[name][b:b + 1, h:h + 1]) for name in ("q", "k", "v", "dout")]
            t0 = time.perf_counter()
            oracle.backward(*sl, pattern=w.pattern, mode=w.mode, l=w.stride, c=w.summary, scale=w.scale)
            times.append(time.perf_counter() - t0)
            spent += times[-1]
            if spent >= budget_s:
                break
        est_s += sum(times) / len(times) * w.batch * w.heads
        credited += credited_flops(w, nnz)[0]
        parts.append(f"{w.name}: {len(times)} of {w.batch * w.heads} (batch, head) slices in {sum(times):.2f} s")
    return {
        "value": credited / est_s / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": "; ".join(parts) + "; full fwd+bwd (the oracle's backward recomputes its forward),"
                  " mean time per slice scaled by batch*heads",
        "est_step_s": est_s,
    }


# The paper's Table 2: time per training iteration of whole models (dense
# attention against the two sparse patterns), on its own hardware.  Quoted only
# as the ratios next to which the attention-only ratios here are set.
TABLE2 = {
    "text, n=12,288": {"dense": "dense_n12288_merged", "fixed": "fixed_n12288_l128_c32_merged",
                       "strided": "strided_n12288_l128_merged",
                       "paper_time_per_iter": {"dense": 1.31, "fixed": 0.55, "strided": 0.35}},
    "image, n=3,072": {"dense": "dense_n3072_merged", "fixed": "fixed_n3072_l128_c32_merged",
                       "strided": "strided_n3072_l128_merged",
                       "paper_time_per_iter": {"dense": 0.54, "fixed": 0.47, "strided": 0.38}},
}


def table2(args):
    """Attention forward + backward time, dense causal against fixed and strided,
    at the two contexts of Table 2 (same kernels; dense is the stride-n limit)."""
    import torch

    from paper_1904_10509_amd import sparse_attn as sa
    from paper_1904_10509_amd.inputs import WORKLOADS, workload_inputs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    out = {"metric": "attention fwd+bwd time, dense causal vs sparse (kernel analogue of Table 2)",
           "unit": "ms", "higher_is_better": False, "steps": args.steps, "warmup": args.warmup,
           "dtype": "bf16", "data": "synthetic", "contexts": {}}
    for ctx, spec in TABLE2.items():
        res = {}
        for kind in ("dense", "fixed", "strided"):
            w = WORKLOADS[spec[kind]]
            x = workload_inputs(w)
            lay = sa.build_layout(w.n, w.block, w.stride, w.summary, w.pattern, w.mode, device=dev)
            q, k, v, dout = (x[n_].to(dev) for n_ in ("q", "k", "v", "dout"))
            o = torch.empty_like(q)
            lse = torch.empty(q.shape[:3], dtype=torch.float32, device=dev)
            grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
            need = sa.sparse_attn_bwd_workspace_size(*lay.pattern_args, w.batch, w.heads, w.d_head, sa.SA_BF16)
            ws = torch.empty(need, dtype=torch.uint8, device=dev)

            def step():
                sa.forward(q, k, v, lay, w.scale, out=o, lse=lse)
                sa.backward(q, k, v, o, dout, lse, lay, w.scale, grads=grads, workspace=ws)

            for _ in range(args.warmup):
                step()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(args.steps):
                step()
            e1.record()
            torch.cuda.synchronize()
            cred, _ = credited_flops(w, lay.nnz)
            ms = e0.elapsed_time(e1) / args.steps
            res[kind] = {"workload": w.name, "ms": ms, "nnz_blocks": lay.nnz,
                         "credited_tflops": cred / (ms * 1e-3) / 1e12}
        paper = spec["paper_time_per_iter"]
        for kind in ("fixed", "strided"):
            res[kind]["speedup_vs_dense"] = res["dense"]["ms"] / res[kind]["ms"]
            res[kind]["paper_speedup_vs_dense"] = paper["dense"] / paper[kind]
        out["contexts"][ctx] = res
    print(json.dumps(out), flush=True)


# Decoding steps at the two long-sequence shapes: one new position per
# sequence, a batch of sequences, the K / V cache resident in HBM.
DECODE = {
    "fixed n=65,536 (l 256, c 32, 8 heads of 64)":
        dict(n=65536, l=256, c=32, pattern=1, heads=8, d=64, batch=32, seed=21),
    "fixed, a summary subblock per head, n=65,536 (l 256, c 32, 8 heads of 64)":
        dict(n=65536, l=256, c=32, pattern=2, heads=8, d=64, batch=32, seed=23),
    "strided n=1,048,576 (l 1,024, 4 heads of 64)":
        dict(n=1048576, l=1024, c=0, pattern=0, heads=4, d=64, batch=16, seed=22),
}


def decode_bench(args):
    """Time per decoding step (sparse_attn_decode at positions n - steps .. n - 1,
    one per step, as in generation) and the bandwidth of the K / V rows it
    reads (|S_pos| rows of K and of V per (sequence, head)) against HBM."""
    import torch

    from paper_1904_10509_amd import sparse_attn as sa

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    out = {"metric": "decoding step time and K/V bandwidth (sparse_attn_decode)", "unit": "us", "dtype": "bf16",
           "data": "synthetic", "steps": args.steps, "warmup": args.warmup, "shapes": {}}
    for name, c in DECODE.items():
        g = torch.Generator(device=dev).manual_seed(c["seed"])
        shape = (c["batch"], c["heads"], c["n"], c["d"])
        kc = torch.randn(shape, generator=g, device=dev, dtype=torch.bfloat16)
        vc = torch.randn(shape, generator=g, device=dev, dtype=torch.bfloat16)
        qs = torch.randn((args.steps + args.warmup, c["batch"], c["heads"], c["d"]), generator=g, device=dev,
                         dtype=torch.bfloat16)
        o = torch.empty_like(qs[0])
        lse = torch.empty((c["batch"], c["heads"]), dtype=torch.float32, device=dev)
        ws_bytes = sa.sparse_attn_decode_workspace_size(c["n"] - 1, c["l"], c["c"], c["pattern"], sa.SA_MODE_MERGED,
                                                        c["batch"], c["heads"], c["d"], sa.SA_BF16)
        ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device=dev)
        total = args.steps + args.warmup
        positions = [c["n"] - total + s for s in range(total)]

        def step(s):
            sa.decode(qs[s], kc, vc, positions[s], c["l"], c["c"], c["pattern"], sa.SA_MODE_MERGED,
                      out=o, lse=lse, workspace=ws)

        for s in range(args.warmup):
            step(s)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for s in range(args.warmup, total):
            step(s)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        # |S_pos| of the merged sets (closed forms of Sec. 4.3, the same for every
        # summary subblock), averaged over the timed positions
        rows = 0
        for pos in positions[args.warmup:]:
            if c["pattern"] == 0:
                rows += min(pos, c["l"]) + 1 + max(0, pos // c["l"] - 1)
            else:
                rows += pos % c["l"] + 1 + (pos // c["l"]) * c["c"]
        rows /= args.steps
        kv_bytes = 2.0 * rows * c["d"] * 2 * c["batch"] * c["heads"]
        gbs = kv_bytes / (us * 1e-6) / 1e9
        out["shapes"][name] = {"batch": c["batch"], "heads": c["heads"], "d": c["d"], "cache_len": c["n"],
                               "keys_per_step": rows, "us_per_step": us, "kv_bytes_per_step": kv_bytes,
                               "tokens_per_s": c["batch"] / (us * 1e-6),
                               "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                            "frac": gbs / HBM_PEAK_GBS}}
        del kc, vc
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


# Strided A2 heads two ways: the block-sparse kernels over the A2 layout, and
# the transposed form (dense causal attention per residue class, Sec. 5.5).
TRANSPOSED = {
    "text, n=12,288 (l 128, 2 x 8 heads of 64)": dict(n=12288, l=128, batch=2, heads=8, d=64, block=64,
                                                        class_block=32, seed=31),
    "audio, n=1,048,576 (l 1,024, 4 heads of 64)": dict(n=1048576, l=1024, batch=1, heads=4, d=64, block=64,
                                                          class_block=64, seed=32),
}


def transposed_bench(args):
    """Forward + backward time of strided A2 attention and of strided merged
    attention (A1 u A2), block-sparse against transposed, with FLOPs counted
    per attended pair (14 d per pair and head: 4 d forward, 10 d backward),
    the honest count for both."""
    import torch

    import numpy as np

    from paper_1904_10509_amd import sparse_attn as sa

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    out = {"metric": "strided A2 and merged fwd+bwd: block-sparse vs transposed (Sec. 5.5)", "unit": "ms",
           "dtype": "bf16",
           "data": "synthetic", "steps": args.steps, "warmup": args.warmup, "shapes": {}}
    for name, c in TRANSPOSED.items():
        g = torch.Generator(device=dev).manual_seed(c["seed"])
        shape = (c["batch"], c["heads"], c["n"], c["d"])
        q, k, v, dout = (torch.randn(shape, generator=g, device=dev, dtype=torch.bfloat16) for _ in range(4))
        m = c["n"] // c["l"]
        pairs = c["l"] * m * (m + 1) // 2 * c["batch"] * c["heads"]
        flop = 14.0 * c["d"] * pairs
        res = {}
        lay_b = sa.build_layout(c["n"], c["block"], c["l"], 0, sa.SA_STRIDED, sa.SA_MODE_A2, device=dev)
        lay_t = sa.transposed_a2_layout(c["n"], c["l"], c["class_block"], device=dev)
        o = torch.empty_like(q)
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
        lse_b = torch.empty(shape[:3], dtype=torch.float32, device=dev)
        lse_t = torch.empty((c["batch"] * c["heads"], c["l"], m), dtype=torch.float32, device=dev)
        ws_b = torch.empty(max(16, sa.sparse_attn_bwd_workspace_size(*lay_b.pattern_args, c["batch"], c["heads"],
                                                                     c["d"], sa.SA_BF16)), dtype=torch.uint8,
                           device=dev)
        ws_t = torch.empty(max(16, sa.sparse_attn_bwd_workspace_size(*lay_t.pattern_args,
                                                                     c["batch"] * c["heads"], c["l"], c["d"],
                                                                     sa.SA_BF16)), dtype=torch.uint8, device=dev)

        def block_step():
            sa.forward(q, k, v, lay_b, out=o, lse=lse_b)
            sa.backward(q, k, v, o, dout, lse_b, lay_b, grads=grads, workspace=ws_b)

        def transposed_step():
            sa.forward_a2_transposed(q, k, v, c["l"], lay_t, out=o, lse=lse_t)
            sa.backward_a2_transposed(q, k, v, o, dout, lse_t, c["l"], lay_t, grads=grads, workspace=ws_t)

        for kind, fn in (("block", block_step), ("transposed", transposed_step)):
            for _ in range(args.warmup):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(args.steps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            res[kind] = {"ms": ms, "pair_tflops": flop / (ms * 1e-3) / 1e12}
        res["block"]["layout_blocks"] = lay_b.nnz
        res["transposed"]["class_layout_blocks"] = lay_t.nnz
        res["speedup"] = res["block"]["ms"] / res["transposed"]["ms"]
        res["attended_pairs"] = pairs
        del lay_b, lay_t, ws_b, ws_t, lse_t

        # merged heads: the merged layout against the band + transposed rest
        i = np.arange(c["n"], dtype=np.int64)
        m_pairs = int((np.minimum(i, c["l"]) + 1 + np.maximum(0, i // c["l"] - 1)).sum()) * c["batch"] * c["heads"]
        m_flop = 14.0 * c["d"] * m_pairs
        lay_m = sa.build_layout(c["n"], c["block"], c["l"], 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, device=dev)
        band = sa.band_layout(c["n"], c["block"], c["l"], device=dev)
        ws_m = torch.empty(max(16, sa.sparse_attn_bwd_workspace_size(*lay_m.pattern_args, c["batch"], c["heads"],
                                                                     c["d"], sa.SA_BF16)), dtype=torch.uint8,
                           device=dev)
        ws_mt = torch.empty(sa.sparse_attn_transposed_workspace_size(c["n"], c["block"], c["l"], c["class_block"],
                                                                     c["batch"], c["heads"], c["d"], sa.SA_BF16),
                            dtype=torch.uint8, device=dev)

        def merged_block_step():
            sa.forward(q, k, v, lay_m, out=o, lse=lse_b)
            sa.backward(q, k, v, o, dout, lse_b, lay_m, grads=grads, workspace=ws_m)

        def merged_transposed_step():
            sa.forward_merged_transposed(q, k, v, band, c["class_block"], out=o, lse=lse_b, workspace=ws_mt)
            sa.backward_merged_transposed(q, k, v, o, dout, lse_b, band, c["class_block"], grads=grads,
                                          workspace=ws_mt)

        merged = {}
        for kind, fn in (("block", merged_block_step), ("transposed", merged_transposed_step)):
            for _ in range(args.warmup):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(args.steps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / args.steps
            merged[kind] = {"ms": ms, "pair_tflops": m_flop / (ms * 1e-3) / 1e12}
        merged["block"]["layout_blocks"] = lay_m.nnz
        merged["transposed"]["band_layout_blocks"] = band.nnz
        merged["speedup"] = merged["block"]["ms"] / merged["transposed"]["ms"]
        merged["attended_pairs"] = m_pairs
        res["merged"] = merged
        out["shapes"][name] = res
        del lay_m, band, ws_m, ws_mt
        del q, k, v, dout, o, grads
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 256 MiB device copy (reference for HBM byte counters)")
    ap.add_argument("--workloads", default=",".join(BENCH_WORKLOADS),
                    help="comma-separated workload names (default: the two measured workloads of the metric); "
                         "other workloads give side measurements, not the metric's line")
    ap.add_argument("--table2", action="store_true",
                    help="instead of the metric's line, time dense causal against fixed and strided attention at "
                         "the two contexts of the paper's Table 2")
    ap.add_argument("--decode", action="store_true",
                    help="instead of the metric's line, time decoding steps (sparse_attn_decode) at the two "
                         "long-sequence shapes")
    ap.add_argument("--transposed", action="store_true",
                    help="instead of the metric's line, time strided A2 attention block-sparse against the "
                         "transposed form (dense causal per residue class)")
    args = ap.parse_args()
    if args.transposed:
        transposed_bench(args)
        return
    if args.decode:
        decode_bench(args)
        return
    if args.table2:
        table2(args)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(see the sharding design note); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_1904_10509_amd import sparse_attn as sa
    from paper_1904_10509_amd.inputs import WORKLOADS, workload_inputs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    if args.copy_calibration:
        copy_calibration(torch, dev)

    runs = []
    names = [x for x in args.workloads.split(",") if x]
    for name in names:
        w = WORKLOADS[name]
        x = workload_inputs(w)
        lay = sa.build_layout(w.n, w.block, w.stride, w.summary, w.pattern, w.mode, device=dev)
        q, k, v, dout = (x[n_].to(dev) for n_ in ("q", "k", "v", "dout"))
        o = torch.empty_like(q)
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device=dev)
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
        need = sa.sparse_attn_bwd_workspace_size(*lay.pattern_args, w.batch, w.heads, w.d_head, sa.SA_BF16)
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
        runs.append(dict(w=w, x=x, lay=lay, q=q, k=k, v=v, dout=dout, o=o, lse=lse, grads=grads, ws=ws))
    torch.cuda.synchronize()

    def step(events=None):
        for idx, r in enumerate(runs):
            if events is not None:
                events[idx][0].record(stream)
            sa.forward(r["q"], r["k"], r["v"], r["lay"], r["w"].scale, out=r["o"], lse=r["lse"])
            if events is not None:
                events[idx][1].record(stream)
            sa.backward(r["q"], r["k"], r["v"], r["o"], r["dout"], r["lse"], r["lay"], r["w"].scale,
                        grads=r["grads"], workspace=r["ws"])
            if events is not None:
                events[idx][2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in runs] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(ev[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    per = {}
    total_credited = 0.0
    fwd_ms_all, bwd_ms_all = [], []
    for idx, r in enumerate(runs):
        w = r["w"]
        fwd_ms = sum(ev[s][idx][0].elapsed_time(ev[s][idx][1]) for s in range(args.steps)) / args.steps
        bwd_ms = sum(ev[s][idx][1].elapsed_time(ev[s][idx][2]) for s in range(args.steps)) / args.steps
        cred, cred_fwd = credited_flops(w, r["lay"].nnz)
        total_credited += cred
        fwd_ms_all.append(fwd_ms)
        bwd_ms_all.append(bwd_ms)
        pairs = attended_pairs(w)
        per[w.name] = {
            "n": w.n, "nnz_blocks": r["lay"].nnz, "credited_flop": cred,
            "element_level_flop": None if pairs is None else 14.0 * w.d_head * pairs * w.batch * w.heads,
            "mfma_flop_upper_bound": mfma_flops_upper_bound(w, r["lay"].nnz),
            "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
            "fwd_tflops": cred_fwd / (fwd_ms * 1e-3) / 1e12,
            "bwd_tflops": (cred - cred_fwd) / (bwd_ms * 1e-3) / 1e12,
            "fwd_bwd_tflops": cred / ((fwd_ms + bwd_ms) * 1e-3) / 1e12,
            "pct_bf16_peak": 100 * cred / ((fwd_ms + bwd_ms) * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        }
    ms_per_step = wall * 1e3 / args.steps
    value = total_credited / (ms_per_step * 1e-3) / 1e12

    # roofline of the dominant call: the backward of the largest workload
    dom = max(range(len(runs)), key=lambda i: bwd_ms_all[i])
    dw = runs[dom]["w"]
    cred, cred_fwd = credited_flops(dw, runs[dom]["lay"].nnz)
    achieved = (cred - cred_fwd) / (bwd_ms_all[dom] * 1e-3) / 1e12
    roofline = {
        "kernel": f"sparse_attn_bwd on {dw.name} (bwd_pre + bwd_dq_bf16 + bwd_dkdv_bf16 launches)",
        "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
        "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(dw.name),
        "avg_ms": bwd_ms_all[dom], "algorithmic_bytes": algorithmic_bwd_bytes(dw),
    }

    out = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": " + ".join(names),
                   "workloads": {r["w"].name: r["w"].describe() for r in runs}},
        "pct_bf16_peak": 100 * value / PEAK_BF16_TFLOPS,
        "per_workload": per,
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline([(r["w"], r["lay"].nnz, r["x"]) for r in runs], None)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
