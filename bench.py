"""Benchmark: effective TFLOP/s (nonzero blocks) of factorized sparse attention,
forward + backward with recomputation, on one MI355X.

One step = forward and backward over each of the two measured workloads:
  strided, n = 12,288, l = 128, B = 64, batch 2, 8 merged heads of 64
  fixed,   n = 65,536, l = 256, c = 32, B = 64, batch 1, 8 merged heads of 64
Inputs are seeded N(0, 1) bf16 tensors already resident in device memory; the
block layouts are built once before timing.  The fixed workload (the one with
the most attended pairs) runs its backward in two calls of
sparse_attn_bwd_stage, the row statistics with dQ (one launch in the library)
and then dK / dV, and the timed steps record HIP events on the library's
stream only around that dK / dV call (an event costs the stream a few
microseconds); the strided workload's backward is one call.  After the timed
steps, two untimed passes time each workload alone and split it into its
forward and backward calls.

The metric credits every present B x B block 14 B^2 d FLOPs per (batch,
head): 4 B^2 d forward (QK^T, PV) and 10 B^2 d backward (QK^T recomputed,
dO V^T, P^T dO, dS^T Q, dS K).  The kernels skip the parts of blocks that no
pair attends, and the strided pattern computes its A2 part by residue
classes, so the credited rate is not matrix-core utilisation: the line also
gives the element-level rate (14 d FLOPs per attended pair), and its roofline
object is the dominant kernel, the dK / dV stage at n = 65,536, priced at its
element-level work (8 d FLOPs per attended pair: S, dP, dV, dK) over its own
event-timed duration.

Prints one JSON line.  The fp64 oracle is timed on the host cores on whole
(batch, head) slices of each workload and scaled to the whole step.
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


def algorithmic_dkdv_bytes(w):
    """dK / dV stage: read Q, K, V, dO and the two row statistics; write dK, dV."""
    e = w.batch * w.heads * w.n
    return 6 * e * w.d_head * 2 + 2 * e * 4


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "traffic_bwd_dkdv_fixed_n65536.json")


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
    """HBM bytes per dK / dV launch from the stored rocprofv3 FETCH_SIZE / WRITE_SIZE
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
    256 MiB written), and a 256 MiB read through direct-to-LDS loads
    (dma_read_kernel), run when counters are collected so FETCH_SIZE /
    WRITE_SIZE can be scaled to bytes for either kind of load."""
    src = torch.empty(128 << 20, dtype=torch.bfloat16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    # the same 256 MiB read once more through direct-to-LDS loads (the kernels'
    # tile staging): 1,024 workgroups x 4 waves x 64 KiB
    L = probe_lib()
    sink = torch.empty(1024 * 256, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    for _ in range(3):
        if L.sa_probe_dma_read_launch(1024, 64, src.data_ptr(), sink.data_ptr(), stream.cuda_stream) != 0:
            raise RuntimeError("probe launch failed")
    torch.cuda.synchronize()
    del src, dst, sink


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


def probe_lib():
    """The measurement probe library (libsa_probe.so: the matrix-core peak and clock, the LDS read rate, the
    workgroup-to-XCD placement)."""
    import ctypes
    path = os.path.join(ROOT, "paper_1904_10509_amd", "libsa_probe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(path)
    L.sa_probe_mfma_flop.restype = ctypes.c_double
    L.sa_probe_mfma_flop.argtypes = [ctypes.c_int, ctypes.c_int]
    L.sa_probe_mfma_launch.restype = ctypes.c_int
    L.sa_probe_mfma_launch.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    L.sa_probe_lds_bytes.restype = ctypes.c_double
    L.sa_probe_lds_bytes.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    L.sa_probe_lds_launch.restype = ctypes.c_int
    L.sa_probe_lds_launch.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p]
    L.sa_probe_dma_read_launch.restype = ctypes.c_int
    L.sa_probe_dma_read_launch.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_void_p]
    L.sa_probe_xcd_map_launch.restype = ctypes.c_int
    L.sa_probe_xcd_map_launch.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    return L


def xcd_map(torch, dev, grids=(768, 2048, 65536)):
    """For grids of several sizes, how many workgroups L ran on XCD L mod 8
    (the placement the kernels' work orders assume)."""
    L = probe_lib()
    stream = torch.cuda.current_stream(dev)
    out = {}
    for g in grids:
        xcd = torch.zeros(g, dtype=torch.int32, device=dev)
        sink = torch.empty(g * 256, dtype=torch.float32, device=dev)
        if L.sa_probe_xcd_map_launch(g, xcd.data_ptr(), sink.data_ptr(), stream.cuda_stream) != 0:
            raise RuntimeError("probe launch failed")
        torch.cuda.synchronize()
        ids = xcd.cpu()
        want = torch.arange(g, dtype=torch.int32) % 8
        out[str(g)] = {"on_xcd_index_mod_8": int((ids == want).sum()), "workgroups": g}
    return out


def lds_read_rate(torch, dev, iters=4000, reps=5):
    """LDS read rate per compute unit for ds_read_b128 and ds_read_b64_tr_b16
    (8 resident workgroups of 4 waves per CU, 16 KiB of LDS each, 8 independent
    reads per lane and iteration), with the shader clock during each."""
    L = probe_lib()
    props = torch.cuda.get_device_properties(dev)
    cus = props.multi_processor_count
    groups = cus * 8
    sink = torch.empty(groups * 256, dtype=torch.int32, device=dev)
    clocks = torch.zeros(2, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream(dev)
    out = {}
    for kind, label in ((0, "ds_read_b128"), (1, "ds_read_b64_tr_b16")):
        nbytes = L.sa_probe_lds_bytes(kind, groups, iters)
        best_ms = None
        for r in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if L.sa_probe_lds_launch(kind, groups, iters, sink.data_ptr(), clocks.data_ptr(), stream.cuda_stream) != 0:
                raise RuntimeError("probe launch failed")
            e1.record(stream)
            torch.cuda.synchronize()
            if r > 0:
                ms = e0.elapsed_time(e1)
                best_ms = ms if best_ms is None else min(best_ms, ms)
        cyc, ticks = (int(x) for x in clocks.cpu())
        ghz = cyc / (ticks / 100e6) / 1e9 if ticks > 0 else None
        rate = nbytes / (best_ms * 1e-3)
        out[label] = {"tb_per_s": rate / 1e12, "clock_ghz": ghz,
                      "bytes_per_clk_per_cu": rate / cus / (ghz * 1e9) if ghz else None}
    out["method"] = ("8 workgroups of 256 threads per CU, all resident (16 KiB of LDS each); every lane "
                     "issues 8 independent reads per iteration at consecutive 16-byte slots; best of 5 launches by "
                     "HIP events; clock from s_memtime over s_memrealtime across one wave's loop")
    return out


def mfma_peak(torch, dev, iters=4096, reps=5):
    """Achievable bf16 matrix-core rate (every wave issuing independent
    16 x 16 x 32 products, 8 waves per SIMD) and the shader clock during it."""
    L = probe_lib()
    props = torch.cuda.get_device_properties(dev)
    groups = props.multi_processor_count * 8
    sink = torch.empty(groups * 256, dtype=torch.float32, device=dev)
    clocks = torch.zeros(2, dtype=torch.int64, device=dev)
    stream = torch.cuda.current_stream(dev)
    flop = L.sa_probe_mfma_flop(groups, iters)
    best = 0.0
    for r in range(reps + 1):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        if L.sa_probe_mfma_launch(groups, iters, sink.data_ptr(), clocks.data_ptr(), stream.cuda_stream) != 0:
            raise RuntimeError("probe launch failed")
        e1.record(stream)
        torch.cuda.synchronize()
        if r > 0:  # the first launch warms up
            best = max(best, flop / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    cyc, ticks = (int(x) for x in clocks.cpu())
    return {"tflops": best, "frac_of_peak": best / PEAK_BF16_TFLOPS,
            "clock_ghz": cyc / (ticks / 100e6) / 1e9 if ticks > 0 else None,
            "workgroups": groups, "compute_units": props.multi_processor_count,
            "method": "8 waves per SIMD, each issuing v_mfma_f32_16x16x32_bf16 on 8 independent accumulators; "
                      "best of 5 launches by HIP events; clock = shader cycles (s_memtime) over 100 MHz "
                      "real-time ticks (s_memrealtime) across one wave's loop"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=30)
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
    ap.add_argument("--mfma-peak", action="store_true",
                    help="instead of the metric's line, measure the achievable bf16 matrix-core rate and clock, "
                         "the LDS read rate per compute unit and the workgroup-to-XCD placement")
    args = ap.parse_args()
    if args.mfma_peak:
        import torch
        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        print(json.dumps({"metric": "achievable bf16 MFMA rate (v_mfma_f32_16x16x32_bf16)",
                          "peak_datasheet_tflops": PEAK_BF16_TFLOPS, **mfma_peak(torch, dev),
                          "lds_read": lds_read_rate(torch, dev), "xcd_map": xcd_map(torch, dev)}), flush=True)
        return
    if args.decode:
        decode_bench(args)
        return
    if args.table2:
        table2(args)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path; run with --gpus 1",
              file=sys.stderr)
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

    # The roofline's kernel is the dK / dV stage of the workload with the most
    # attended pairs; that workload's backward runs as two calls, the row
    # statistics with dQ (one launch in the library) and then dK / dV, with
    # events around the second.  Every other workload's backward is one call
    # (the strided one then runs its short residue classes' dQ and dK / dV as
    # one launch).
    dom = max(range(len(runs)), key=lambda i: (attended_pairs(runs[i]["w"]) or 0) * runs[i]["w"].batch
              * runs[i]["w"].heads)
    split_calls = (("row_stats_and_dq", sa.SA_BWD_ROW_STATS | sa.SA_BWD_DQ), ("dkdv", sa.SA_BWD_DKDV))
    whole_call = (("backward", sa.SA_BWD_ALL_STAGES),)
    calls = [split_calls if i == dom else whole_call for i in range(len(runs))]
    LAST = 1 + len(split_calls)  # events per workload: before the forward, after it, after each call

    def step(events=None, marks="dkdv"):
        """One step.  events[idx] holds the events of workload idx: before the
        forward, after it, and after each backward call.  marks = "dkdv"
        records only the two around the dominant workload's dK / dV call (the
        timed steps: each event costs the stream a few microseconds), "total"
        only the first and the last, "all" every one."""
        for idx, r in enumerate(runs):
            ev = events[idx] if events is not None else None
            if ev is not None and marks != "dkdv":
                ev[0].record(stream)
            sa.forward(r["q"], r["k"], r["v"], r["lay"], r["w"].scale, out=r["o"], lse=r["lse"])
            if ev is not None and marks == "all":
                ev[1].record(stream)
            n_calls = len(calls[idx])
            for si, (name, st) in enumerate(calls[idx]):
                if ev is not None and marks == "dkdv" and name == "dkdv":
                    ev[1 + si].record(stream)
                sa.backward(r["q"], r["k"], r["v"], r["o"], r["dout"], r["lse"], r["lay"], r["w"].scale,
                            grads=r["grads"], workspace=r["ws"], stages=st)
                if ev is not None and (marks == "all" or (marks == "dkdv" and name == "dkdv")):
                    ev[2 + si].record(stream)
                if ev is not None and marks == "total" and si == n_calls - 1:
                    ev[LAST].record(stream)

    def new_events():
        return [[[torch.cuda.Event(enable_timing=True) for _ in range(LAST + 1)] for _ in runs]
                for _ in range(args.steps)]

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # the timed steps: events only around each dK / dV stage (the roofline's kernel)
    ev = new_events()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(ev[s], "dkdv")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    def avg_ms(evs, idx, a, b):
        return sum(evs[s_][idx][a].elapsed_time(evs[s_][idx][b]) for s_ in range(args.steps)) / args.steps

    dkdv_ms = avg_ms(ev, dom, len(split_calls), 1 + len(split_calls))
    # after the timed steps, untimed: each workload's own time (events at its
    # ends only), then its split into forward and backward stages (every event)
    ev_total, ev_all = new_events(), new_events()
    for s in range(args.steps):
        step(ev_total[s], "total")
    for s in range(args.steps):
        step(ev_all[s], "all")
    torch.cuda.synchronize()

    per = {}
    total_credited = total_element = 0.0
    for idx, r in enumerate(runs):
        w = r["w"]
        total_ms = avg_ms(ev_total, idx, 0, LAST)
        n_calls = len(calls[idx])
        fwd_ms, bwd_ms = avg_ms(ev_all, idx, 0, 1), avg_ms(ev_all, idx, 1, 1 + n_calls)
        stage_ms = {name: avg_ms(ev_all, idx, 1 + si, 2 + si) for si, (name, _) in enumerate(calls[idx])}
        cred, cred_fwd = credited_flops(w, r["lay"].nnz)
        total_credited += cred
        pairs = attended_pairs(w)
        elem = None if pairs is None else 14.0 * w.d_head * pairs * w.batch * w.heads
        total_element += elem or 0.0
        per[w.name] = {
            "n": w.n, "nnz_blocks": r["lay"].nnz, "credited_flop": cred, "element_level_flop": elem,
            "attended_pairs_per_head": pairs,
            "ms": total_ms, "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
            "bwd_stage_ms": stage_ms,
            "dkdv_ms_timed_steps": dkdv_ms if idx == dom else None,
            "timing_note": ("ms: forward + backward from events at the workload's ends; fwd_ms, bwd_ms and "
                            "bwd_stage_ms from a pass with an event after every stage (a few us each); both "
                            "passes run after the timed steps"),
            "credited_tflops": cred / (total_ms * 1e-3) / 1e12,
            "credited_pct_bf16_peak": 100 * cred / (total_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "element_level_tflops": None if elem is None else elem / (total_ms * 1e-3) / 1e12,
            "element_level_pct_bf16_peak": None if elem is None else
            100 * elem / (total_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        }
        if w.pattern == 0:
            per[w.name]["note"] = ("strided: A2 runs by residue classes (dense causal attention per class), so the "
                                   "credited rate counts blocks the kernels never form; it is the metric's "
                                   "artefact, not matrix-core utilisation (see element_level_tflops)")
    ms_per_step = wall * 1e3 / args.steps
    value = total_credited / (ms_per_step * 1e-3) / 1e12

    # roofline of the dominant kernel: the dK / dV stage (one bwd_dkdv_bf16_kernel
    # launch) of the workload with the most attended pairs, priced at its
    # element-level work, 8 d FLOPs per attended pair (S, dP, dV, dK), over its
    # event-timed duration in the timed steps
    dw = runs[dom]["w"]
    dkdv_flop = 8.0 * dw.d_head * attended_pairs(dw) * dw.batch * dw.heads
    achieved = dkdv_flop / (dkdv_ms * 1e-3) / 1e12
    roofline = {
        "kernel": f"bwd_dkdv_bf16_kernel (dK/dV stage of sparse_attn_bwd) on {dw.name}",
        "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
        "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(dw.name),
        "avg_ms": dkdv_ms, "flop_per_launch": dkdv_flop,
        "flop_basis": "8 d per attended pair (S, dP, dV, dK) x pairs per head x batch x heads",
        "algorithmic_bytes": algorithmic_dkdv_bytes(dw),
    }

    out = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": " + ".join(names),
                   "workloads": {r["w"].name: r["w"].describe() for r in runs}},
        "credited_frac": value / PEAK_BF16_TFLOPS,
        "element_level_tflops": total_element / (ms_per_step * 1e-3) / 1e12,
        "element_level_frac": total_element / (ms_per_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
        "per_workload": per,
        "roofline": roofline,
        "mfma_probe": mfma_peak(torch, dev),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline([(r["w"], r["lay"].nnz, r["x"]) for r in runs], None)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
