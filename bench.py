"""Decode-throughput benchmark of the fused EntroPack decode on one MI355X.

Default workload (the 27B-class LLM MLP set): gate and up 17408 x 5120 and
down 5120 x 17408 BF16 weights (seeded synthetic, Gaussian rows with
lognormal std and 0.05 % x8 outliers), each converted to the row-scaled FP8
e4m3 container and EntroPack-coded at 4.0 bits/weight with 4096-weight tiles
by the library's CPU encoder.  One step decodes all three tensors to FP8 e4m3
plus per-row dequant scales in a single launch of a prepared stack (ep_stack_decode), with the
blobs already resident in HBM.

Reported: decoded weights/s (value), achieved GB/s of the decode kernel
against the 8 TB/s HBM3E peak (algorithmic bytes = every compressed byte read
+ every weight and dequant byte written), and the CPU oracle decoder's
throughput on the same blobs on this host's cores.

Other workloads (--workload): attn_fp16 (3072 x 3072 at 3.0 bpp to FP16),
dit_stack (30 diffusion-transformer blocks, 180 layers at 2.5 bpp to BF16 in one
launch), mlp_down_int8 (the MLP down projection in the INT8 container at
6.0 bpp to INT8, followed by the INT8 MFMA product with 8192 x 17408
activations, timed separately: decode time over product time is reported),
encode_mlp (the GPU encoder on the MLP set's three BF16 tensors, FP8 container
at 4.0 bpp; a step encodes all three; the CPU baseline is the oracle encoder
on the down projection), fused_mfma_m<m> (the fused decode and MFMA product
ep_decode_gemm_i8 of the INT8-container down projection with the first m rows of the
activations, timed beside decode-then-GEMM and the product alone on resident weights),
fused_bf16_m<m> (the fused decode and BF16 MFMA product ep_decode_gemm_bf16 of the
diffusion-transformer MLP input projection 10240 x 3840 at 2.5 bpp with m rows of bf16
activations, timed beside a BF16 decode followed by the library BF16 GEMM),
fused_down_m1 / _m2 / _m4 / _m8 (the fused decode and
small-batch product ep_decode_matmul_i8: the INT8-container down projection
times the first 1, 2, 4 or 8 rows of the activations, one launch per step;
algorithmic bytes = compressed blob + X read, Y and dequant written),
tile_sweep (the paper's reference-layer shape 10240 x 3840 at 4.0 bpp to BF16,
encoded and decoded at tile sizes of 128 to 3640 vectors: stored rate, tile
count and decode time per size; value is the 512-vector point).

The roofline's `traffic` field is the decode kernel's measured HBM bytes per
launch, read from the committed rocprofv3 counter summary of this workload
(FETCH_SIZE and WRITE_SIZE, each scaled by the factor the same counter shows
for a plain device copy of known size); `counters` carries the kernel's VALU,
SALU and LDS utilisation from the committed SQ counter summary.  Both are null
when their summary is absent or was taken from a different decode kernel
source than the one built.

Parity gate: before anything is timed, the CPU-baseline leg decodes the same blobs with the
oracle, and one GPU step's output (every weight, and the dequant scales) must equal it bit for
bit, or the run stops (config.parity_gate records the check; --no-cpu-baseline skips both).

Timing: the W warm-up steps are followed, untimed, by further steps until
SETTLE_S seconds have passed since the warm-up began (config.settle_steps
says how many), because a GPU fresh from idle runs its first milliseconds at
lower clocks; then exactly K steps are timed with HIP events on the launch
stream.

--copy-calibration runs only a plain 1 GiB device-to-device copy (five times),
the reference kernel for those counter factors.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decoded weights/s and achieved HBM GB/s (% roofline), 1 MI355X"
HBM_PEAK_GBPS = 8000.0
SETTLE_S = 0.3
INT8_PEAK_TOPS = 5000.0   # dense MFMA int8, MI355X
BF16_PEAK_TFLOPS = 2500.0   # dense MFMA bf16, MI355X
# the decode kernels' sources: their device code, then the file that instantiates
# the kernels bench.py times
DECODE_SRCS = [os.path.join(ROOT, "paper_2609_34185_amd", "csrc", n)
               for n in ("decode_kernels.h", "decode.hip")]
COPY_BYTES = 1 << 30


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload(name, E, W, threads):
    """Returns (description dict, [(label, blob, out_dtype)])."""
    if name == "mlp_fp8":
        d = W.llm_mlp()
        items = []
        for n in ("gate", "up", "down"):
            b, st = E.encode(d[n], 4.0, container=E.CONT_FP8_ROW, nthreads=threads)
            log(f"encoded {n}: {b.size} B, {st['rate_stored']:.4f} bpp")
            items.append((n, b, E.FP8_E4M3))
        desc = {"workload": "27B-class LLM MLP set: gate+up 17408x5120, down 5120x17408; FP8-e4m3 "
                            "row container coded at 4.0 bpp, 4096-weight tiles; decoded to FP8 e4m3 "
                            "+ per-row dequant in one launch",
                "tensors": 3, "target_bpp": 4.0, "tile_weights": 4096, "out": "fp8_e4m3+dequant"}
    elif name == "attn_fp16":
        b, st = E.encode(W.attention_projection(), 3.0, nthreads=threads)
        items = [("attn", b, E.FP16)]
        desc = {"workload": "attention projection 3072x3072 at 3.0 bpp, decoded to FP16",
                "tensors": 1, "target_bpp": 3.0, "tile_weights": 4096, "out": "fp16"}
    elif name == "mlp_down_int8":
        d = W.llm_mlp()
        b, st = E.encode(d["down"], 6.0, container=E.CONT_INT8_ROW, nthreads=threads)
        items = [("down", b, E.INT8)]
        desc = {"workload": "MLP down 5120x17408, INT8 row container at 6.0 bpp, decoded to INT8 "
                            "+ per-row dequant", "tensors": 1, "target_bpp": 6.0,
                "tile_weights": 4096, "out": "int8+dequant"}
    elif name == "dit_stack":
        items = []
        for blk in range(30):
            for lname, w in W.dit_block(blk):
                b, st = E.encode(w, 2.5, nthreads=threads)
                items.append((lname, b, E.BF16))
            log(f"encoded block {blk}")
        desc = {"workload": "diffusion-transformer stack: 30 blocks x (4 x 3840x3840, 10240x3840, "
                            "3840x10240) at 2.5 bpp, 180 layers decoded to BF16 in one launch",
                "tensors": 180, "target_bpp": 2.5, "tile_weights": 4096, "out": "bf16"}
    else:
        raise SystemExit(f"unknown workload {name}")
    return desc, items


def encode_bench(args, E, W, threads):
    """--workload encode_mlp: the GPU encoder on the 27B-class MLP set (gate, up, down BF16,
    FP8 row container at 4.0 bpp, as the decode workload is prepared), inputs resident in
    HBM.  A step encodes all three tensors (each call returns a finished host blob)."""
    import numpy as np
    import torch
    d = W.llm_mlp()
    names = ("gate", "up", "down")
    dev = {n: torch.from_numpy(d[n].view(np.int16)).cuda() for n in names}
    weights = sum(d[n].size for n in names)
    s = torch.cuda.current_stream().cuda_stream

    def step():
        return [E.encode_gpu(dev[n].data_ptr(), d[n].shape[0], d[n].shape[1], 4.0,
                             container=E.CONT_FP8_ROW, stream=s) for n in names]

    first = step()
    ref = [E.encode(d[n], 4.0, container=E.CONT_FP8_ROW, nthreads=threads)[0] for n in names]
    assert all(np.array_equal(a[0], b) for a, b in zip(first, ref)), "GPU and CPU encoder blobs differ"
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.steps
    line = {
        "metric": "encoded weights/s (GPU encoder; blobs byte-identical to the CPU encoder)",
        "value": weights / sec, "unit": "weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": sec * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": "GPU encode of the 27B-class LLM MLP set: gate+up 17408x5120, "
                               "down 5120x17408 BF16 in HBM, FP8 row container at 4.0 bpp, "
                               "host blobs out", "tensors": 3, "weights": weights,
                   "stored_bytes": int(sum(b.size for b in ref))},
    }
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        log("timing the CPU oracle encoder on the down projection")
        t0 = time.perf_counter()
        O.encode(d["down"], 4.0, container=1)
        osec = time.perf_counter() - t0
        line["cpu_baseline"] = {"value": d["down"].size / osec, "unit": "weights/s", "cores": 1,
                                "kind": "oracle", "sample": "the down projection (89,128,960 "
                                "weights) encoded once by the plain C oracle encoder",
                                "seconds": round(osec, 3)}
    print(json.dumps(line), flush=True)


def fused_bench(args, E, W, threads, m):
    """--workload fused_down_m<m>: Y = X W'^T for the INT8-container MLP down projection
    (5120 x 17408 at 6.0 bpp) and the first m rows of the 8192 x 17408 activations, W' never
    written.  The first result is checked against the product of the GPU-decoded W'."""
    import numpy as np
    import torch
    w = W.llm_mlp(["down"])["down"]
    blob, _ = E.encode(w, 6.0, container=E.CONT_INT8_ROW, nthreads=threads)
    info = E.blob_info(blob)
    x_host = np.ascontiguousarray(W.llm_activations()[:m])
    d_blob = E.to_device(blob, torch.device("cuda", 0))
    x = torch.from_numpy(x_host).cuda()
    y = torch.empty((m, info.rows), dtype=torch.int32, device="cuda")
    dq = torch.empty(info.rows, dtype=torch.float32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        E.decode_matmul_i8(info, d_blob.data_ptr(), x.data_ptr(), m, y.data_ptr(), dq.data_ptr(),
                           status.data_ptr(), stream.cuda_stream)

    step()
    wd, _, _ = E.decode(blob, E.INT8, d_blob=d_blob, info=info)
    ref = x_host.astype(np.int64) @ wd.cpu().numpy().astype(np.int64).T
    torch.cuda.synchronize()
    assert np.array_equal(y.cpu().numpy(), ref), "fused product differs from decode-then-multiply"
    t0 = time.perf_counter()
    for _ in range(args.warmup):
        step()
    settle = 0
    while time.perf_counter() - t0 < SETTLE_S:
        for _ in range(10):
            step()
        settle += 10
        torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(args.steps):
        step()
    b.record(stream)
    torch.cuda.synchronize()
    assert int(status.item()) == 0, "decode reported a corrupt stream"
    ms = a.elapsed_time(b) / args.steps
    weights = info.rows * info.cols
    algo = blob.size + m * info.cols + 4 * m * info.rows + 4 * info.rows
    gbps = algo / (ms * 1e-3) / 1e9
    line = {
        "metric": "fused decode + product: decoded weights/s and achieved HBM GB/s (% roofline)",
        "value": weights / (ms * 1e-3), "unit": "weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "i32", "data": "synthetic",
        "config": {"workload": f"fused decode and product: MLP down 5120x17408 in the INT8 row "
                               f"container at 6.0 bpp times X = {m} x 17408 int8 rows, Y int32 "
                               f"exact, decoded weights never written", "rows_x": m,
                   "weights": weights, "bytes_per_step": algo, "settle_steps": settle},
        "roofline": {"bound": "hbm", "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": gbps / HBM_PEAK_GBPS, "traffic": None},
    }
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        log("timing the CPU oracle: decode, then the product")
        t = time.perf_counter()
        wo, _ = O.decode(blob, O.INT8)
        O.gemm_i8_nt(x_host, wo)
        osec = time.perf_counter() - t
        line["cpu_baseline"] = {"value": weights / osec, "unit": "weights/s", "cores": 1,
                                "kind": "oracle", "sample": f"the whole down projection decoded by "
                                f"the plain C oracle, then its exact product with the {m} rows",
                                "seconds": round(osec, 3), "cpu": cpu_model()}
    print(json.dumps(line), flush=True)


def time_steps(args, step, stream):
    """Warm-up, settle, then the mean over args.steps launches (HIP events on `stream`)."""
    import torch
    t0 = time.perf_counter()
    for _ in range(args.warmup):
        step()
    while time.perf_counter() - t0 < SETTLE_S:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(args.steps):
        step()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / args.steps


def fused_mfma_bench(args, E, W, threads, m):
    """--workload fused_mfma_m<m>: Y = X W'^T for the INT8-container MLP down projection
    (5120 x 17408 at 6.0 bpp) and the first m rows of the 8192 x 17408 activations by the fused
    decode and MFMA product (ep_decode_gemm_i8_prepared on a workspace whose tables
    ep_decode_gemm_i8_prepare built once; W' never written as a whole), timed beside
    decode-then-GEMM (a prepared one-layer stack decoded to INT8 by ep_stack_decode, then
    ep_gemm_i8_nt) and beside the product alone on resident decoded weights: the analog of the
    paper's decode-cost curve over tokens per call (App. A.5, Fig. cost).  The variants that
    build their tables at every call (ep_decode_gemm_i8, ep_decode_tiles) are timed too.  The
    fused Y must equal decode-then-GEMM's Y."""
    import numpy as np
    import torch
    w = W.llm_mlp(["down"])["down"]
    blob, _ = E.encode(w, 6.0, container=E.CONT_INT8_ROW, nthreads=threads)
    info = E.blob_info(blob)
    x = torch.from_numpy(np.ascontiguousarray(W.llm_activations()[:m])).cuda()
    d_blob = E.to_device(blob, torch.device("cuda", 0))
    y = torch.empty((m, info.rows), dtype=torch.int32, device="cuda")
    y2 = torch.empty((m, info.rows), dtype=torch.int32, device="cuda")
    wd = torch.empty((info.rows, info.cols), dtype=torch.int8, device="cuda")
    dq = torch.empty(info.rows, dtype=torch.float32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = E.decode_gemm_i8_workspace(info)
    d_ws = torch.empty(ws, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    s = stream.cuda_stream
    E.decode_gemm_i8_prepare(info, d_blob.data_ptr(), d_ws.data_ptr(), ws, s)
    sws = E.stack_workspace(1)
    d_sws = torch.empty(sws, dtype=torch.uint8, device="cuda")
    stack = E.stack_prepare([(info, d_blob.data_ptr(), wd.data_ptr(), dq.data_ptr(), E.INT8)],
                            d_sws.data_ptr(), sws, s)

    def fused_step():
        E.decode_gemm_i8_prepared(info, d_blob.data_ptr(), x.data_ptr(), m, y.data_ptr(),
                                  d_ws.data_ptr(), ws, dq.data_ptr(), status.data_ptr(), s)

    def fused_built_step():
        E.decode_gemm_i8(info, d_blob.data_ptr(), x.data_ptr(), m, y.data_ptr(), d_ws.data_ptr(), ws,
                         dq.data_ptr(), status.data_ptr(), s)

    def decode_step():
        E.stack_decode(stack, status.data_ptr(), s)

    def decode_tiles_step():
        E.decode_tiles(info, d_blob.data_ptr(), E.INT8, wd.data_ptr(), dq.data_ptr(), 0, info.n_tiles,
                       status.data_ptr(), s)

    def gemm_step():
        E.gemm_i8_nt(x.data_ptr(), wd.data_ptr(), y2.data_ptr(), m, info.rows, info.cols, s)

    for f in (fused_step, decode_step, gemm_step):
        f()
    torch.cuda.synchronize()
    assert int(status.item()) == 0, "decode reported a corrupt stream"
    assert torch.equal(y, y2), "fused product differs from decode-then-GEMM"
    fused_built_step()
    torch.cuda.synchronize()
    assert torch.equal(y, y2), "fused product (tables built) differs from decode-then-GEMM"
    ms = time_steps(args, fused_step, stream)
    ms_built = time_steps(args, fused_built_step, stream)
    ms_dec = time_steps(args, decode_step, stream)
    ms_tiles = time_steps(args, decode_tiles_step, stream)
    ms_gemm = time_steps(args, gemm_step, stream)
    assert int(status.item()) == 0, "decode reported a corrupt stream"
    weights = info.rows * info.cols
    ops = 2.0 * m * info.rows * info.cols
    line = {
        "metric": "fused decode + MFMA product: decoded weights/s and int8 TOP/s (% of MFMA peak)",
        "value": weights / (ms * 1e-3), "unit": "weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "i32", "data": "synthetic",
        "config": {"workload": f"fused decode and MFMA product: MLP down 5120x17408 in the INT8 row "
                               f"container at 6.0 bpp times X = {m} x 17408 int8 rows, Y int32 exact",
                   "rows_x": m, "weights": weights,
                   "decode_then_gemm_ms": {"decode": ms_dec, "gemm": ms_gemm, "total": ms_dec + ms_gemm},
                   "tables_built_every_call_ms": {"fused": ms_built, "decode": ms_tiles,
                                                  "decode_then_gemm": ms_tiles + ms_gemm},
                   "resident_gemm_ms": ms_gemm,
                   "fused_over_decode_then_gemm": ms / (ms_dec + ms_gemm),
                   "overhead_vs_resident_pct": 100.0 * (ms / ms_gemm - 1.0),
                   "decode_then_gemm_overhead_vs_resident_pct": 100.0 * (ms_dec / ms_gemm)},
        "roofline": {"bound": "mfma", "achieved": ops / (ms * 1e-3) / 1e12, "peak": INT8_PEAK_TOPS,
                     "unit": "TFLOP/s", "frac": ops / (ms * 1e-3) / 1e12 / INT8_PEAK_TOPS,
                     "traffic": None},
    }
    print(json.dumps(line), flush=True)


def fused_bf16_bench(args, E, W, threads, m):
    """--workload fused_bf16_m<m>: Y = X W'^T (fp32) for the diffusion-transformer MLP input
    projection (10240 x 3840 Student-t rows at 2.5 bpp, the paper's reference-layer shape) and
    m rows of bf16 activations by the fused decode and BF16 MFMA product
    (ep_decode_gemm_bf16_prepared, tables prepared once; W' never written as a whole), timed
    beside decode-then-GEMM (a prepared one-layer stack decoded to BF16 by ep_stack_decode,
    then torch's BF16 GEMM, used only as the comparison) and beside that GEMM alone on the
    resident decoded weights.  The fused Y is checked against the fp32 product of the decoded
    weights before anything is timed."""
    import numpy as np
    import torch
    w = dict(W.dit_block(0))["blocks.0.mlp_in"]
    blob, _ = E.encode(w, 2.5, nthreads=threads)
    info = E.blob_info(blob)
    rng = np.random.default_rng(7)
    x = torch.from_numpy(rng.standard_normal((m, info.cols)).astype(np.float32)).cuda().to(torch.bfloat16)
    d_blob = E.to_device(blob, torch.device("cuda", 0))
    y = torch.empty((m, info.rows), dtype=torch.float32, device="cuda")
    wd = torch.empty((info.rows, info.cols), dtype=torch.bfloat16, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = E.decode_gemm_bf16_workspace(info)
    d_ws = torch.empty(ws, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    s = stream.cuda_stream
    E.decode_gemm_bf16_prepare(info, d_blob.data_ptr(), d_ws.data_ptr(), ws, s)
    sws = E.stack_workspace(1)
    d_sws = torch.empty(sws, dtype=torch.uint8, device="cuda")
    stack = E.stack_prepare([(info, d_blob.data_ptr(), wd.data_ptr(), 0, E.BF16)], d_sws.data_ptr(), sws, s)

    def fused_step():
        E.decode_gemm_bf16_prepared(info, d_blob.data_ptr(), x.data_ptr(), m, y.data_ptr(),
                                    d_ws.data_ptr(), ws, 0, status.data_ptr(), s)

    def decode_step():
        E.stack_decode(stack, status.data_ptr(), s)

    def gemm_step():
        torch.nn.functional.linear(x, wd)   # a 2-D product (no batched GEMM)

    fused_step()
    decode_step()
    torch.cuda.synchronize()
    assert int(status.item()) == 0, "decode reported a corrupt stream"
    ref = x.float() @ wd.float().t().contiguous()
    torch.cuda.synchronize()
    assert torch.allclose(y, ref, rtol=1e-3, atol=1e-3 * float(ref.abs().max())), \
        "fused BF16 product differs from the product of the decoded weights"
    ms = time_steps(args, fused_step, stream)
    ms_dec = time_steps(args, decode_step, stream)
    ms_gemm = time_steps(args, gemm_step, stream)
    assert int(status.item()) == 0, "decode reported a corrupt stream"
    weights = info.rows * info.cols
    flops = 2.0 * m * info.rows * info.cols
    line = {
        "metric": "fused decode + BF16 MFMA product: decoded weights/s and TFLOP/s (% of MFMA peak)",
        "value": weights / (ms * 1e-3), "unit": "weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"fused decode and BF16 MFMA product: DiT MLP input projection 10240x3840 "
                               f"at 2.5 bpp times X = {m} x 3840 bf16 rows, Y fp32",
                   "rows_x": m, "weights": weights,
                   "decode_then_gemm_ms": {"decode": ms_dec, "gemm": ms_gemm, "total": ms_dec + ms_gemm},
                   "fused_over_decode_then_gemm": ms / (ms_dec + ms_gemm)},
        "roofline": {"bound": "mfma", "achieved": flops / (ms * 1e-3) / 1e12, "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": flops / (ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
                     "traffic": None},
    }
    print(json.dumps(line), flush=True)


SWEEP_V = (128, 256, 512, 1024, 1820, 2048, 3640)


def tile_sweep(args, E, W, threads):
    """--workload tile_sweep: one layer of the reference shape (10240 x 3840, the DiT stack's
    first MLP input projection) at 4.0 bpp, decoded to BF16, for several tile sizes V (the
    paper's 4096, 8192, 16384 and 32768 symbols per tile are V = 455, 910, 1820, 3640)."""
    import torch
    w = dict(W.dit_block(0))["blocks.0.mlp_in"]
    weights = w.size
    rows = []
    for V in SWEEP_V:
        blob, st = E.encode(w, 4.0, tile_vectors=V, nthreads=threads)
        info = E.blob_info(blob)
        d_blob = E.to_device(blob)
        out = torch.empty((info.rows, info.cols), dtype=torch.bfloat16, device="cuda")
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        s = torch.cuda.current_stream()

        def step():
            E.decode_tiles(info, d_blob.data_ptr(), E.BF16, out.data_ptr(), 0, 0, info.n_tiles,
                           status.data_ptr(), s.cuda_stream)

        t0 = time.perf_counter()
        while time.perf_counter() - t0 < SETTLE_S:
            for _ in range(10):
                step()
            torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        for _ in range(args.steps):
            step()
        b.record(s)
        torch.cuda.synchronize()
        assert int(status.item()) == 0, "decode reported a corrupt stream"
        ms = a.elapsed_time(b) / args.steps
        steady = info.prob_bits == 11 and info.path in (1, 3) and V >= 32   # slot-table steady state (any V >= 32)
        rows.append({"V": V, "symbols_per_tile": 9 * V, "tiles": info.n_tiles,
                     "stored_bpp": round(8.0 * blob.size / weights, 4),
                     "erel_pct": round(100.0 * st["erel_coded"], 3), "ms": ms,
                     "weights_per_s": weights / (ms * 1e-3),
                     "gbps": (blob.size + 2 * weights) / (ms * 1e-3) / 1e9,
                     "steady_state": steady})
        log(f"V={V}: {rows[-1]['stored_bpp']} bpp, E_rel {rows[-1]['erel_pct']} %, {ms * 1e3:.1f} us")
    ref = [r for r in rows if r["V"] == 512][0]
    line = {
        "metric": "decoded weights/s per tile size (reference layer)", "value": ref["weights_per_s"],
        "unit": "weights/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ref["ms"], "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u32", "data": "synthetic",
        "config": {"workload": "tile-size sweep: 10240x3840 BF16 (Student-t rows) at 4.0 bpp, "
                               "decoded to BF16, one tensor per launch", "weights": weights,
                   "sweep": rows},
        "roofline": {"bound": "hbm", "achieved": ref["gbps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": ref["gbps"] / HBM_PEAK_GBPS, "traffic": None},
    }
    print(json.dumps(line), flush=True)


def source_digest() -> str:
    """sha256 of the decode kernels' sources, in DECODE_SRCS order."""
    h = hashlib.sha256()
    for path in DECODE_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def profile_summary(name: str):
    """The `key: value` lines of profiles/<name>, or None when the file is
    absent or was taken from a decode kernel source other than the one built."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith(("#", " ", "\t")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    return kv if kv.get("decode_source_sha256") == source_digest() else None


def measured_counters(workload_name: str):
    """Unit utilisation of the decode kernel from its committed SQ counter summary, or None."""
    kv = profile_summary(f"decode_{workload_name}_sq_counters.txt")
    if kv is None:
        return None
    try:
        return {"valu_busy": float(kv["valu_busy_pct"]) / 100,
                "salu_busy": float(kv["salu_busy_pct"]) / 100,
                "lds_busy": float(kv["lds_busy_pct"]) / 100,
                "lds_bank_conflict_stall": float(kv["lds_bank_conflict_pct"]) / 100,
                "valu_lane_ops_per_weight": float(kv["valu_lane_ops_per_weight"]),
                "source": f"profiles/decode_{workload_name}_sq_counters.txt"}
    except (KeyError, ValueError):
        return None


def measured_traffic(workload_name: str):
    """HBM bytes per decode launch from profiles/decode_<workload>_traffic.txt, or None."""
    kv = profile_summary(f"decode_{workload_name}_traffic.txt")
    if kv is None:
        return None
    try:
        fetch = float(kv["fetch_kib_per_launch"]) * float(kv["copy_fetch_factor"])
        write = float(kv["write_kib_per_launch"]) * float(kv["copy_write_factor"])
        return 1024.0 * (fetch + write)
    except (KeyError, ValueError):
        return None


def copy_calibration():
    """A plain device copy of COPY_BYTES, five times: the counters' reference kernel."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 5}), flush=True)


def gemm_leg(E, W, out, info, reps=20, warm=30):
    """Time the INT8 MFMA product of the decoded weights with the 8192 x 17408 activations."""
    import torch
    act = torch.from_numpy(W.llm_activations()).cuda()
    m, n, k = act.shape[0], info.rows, info.cols
    y = torch.empty((m, n), dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream()

    def run():
        E.gemm_i8_nt(act.data_ptr(), out.data_ptr(), y.data_ptr(), m, n, k, s.cuda_stream)

    for _ in range(warm):   # about 20 ms: lets the clocks settle under MFMA load
        run()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(reps):
        run()
    b.record(s)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    tops = 2.0 * m * n * k / (ms * 1e-3) / 1e12
    return {"shape": [m, n, k], "ms": ms, "tops": tops,
            "roofline": {"bound": "mfma", "achieved": tops, "peak": INT8_PEAK_TOPS,
                         "unit": "TOP/s", "frac": tops / INT8_PEAK_TOPS}}


def cold_cache_ms(step, reps=15):
    """Per-launch times with the 256 MB last-level cache flushed before each launch."""
    import torch
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    times = []
    for _ in range(reps):
        flush.zero_()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        step()
        b.record(s)
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    times.sort()
    return {"min": times[0], "median": times[len(times) // 2], "reps": reps}


def copy_bandwidth(reps=10):
    """Achieved bandwidth of a plain 1 GiB device-to-device copy (bytes read plus bytes
    written per second, HIP events): the practical ceiling a streaming kernel is held against
    beside the 8 TB/s nominal figure."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    s = torch.cuda.current_stream()
    for _ in range(3):
        dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(s)
    for _ in range(reps):
        dst.copy_(src)
    b.record(s)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    return 2 * COPY_BYTES / (ms * 1e-3) / 1e9


def cpu_baseline(items, threads):
    """The oracle decoder on the same blobs, tiles split over `threads` host threads.  Returns
    (the timing record, the oracle's outputs [(weights, dequant or None)] for the parity gate)."""
    import numpy as np
    from oracle import oracle as O
    ocode = {1: O.BF16, 2: O.FP16, 3: O.FP32, 4: O.FP8, 5: O.INT8}
    jobs = []
    outs = []
    weights = 0
    for label, blob, dt in items:
        h = O.header(blob)
        out = np.zeros((h["rows"], h["cols"]), dtype=O.OUT_NPTYPE[ocode[dt]])
        dq = np.zeros(h["rows"], dtype=np.float32)
        outs.append((out, dq))
        weights += h["rows"] * h["cols"]
        n = h["n_tiles"]
        parts = max(1, min(threads, n))
        for p in range(parts):
            jobs.append((blob, ocode[dt], out, dq, n * p // parts, n * (p + 1) // parts))

    def run(j):
        blob, code, out, dq, t0, t1 = j
        O.decode(blob, code, t0, t1, out=out, dequant=dq)

    # three passes (about 20 s of CPU work on the MLP set); the median is reported
    secs = []
    with ThreadPoolExecutor(threads) as ex:
        for _ in range(3):
            t = time.perf_counter()
            list(ex.map(run, jobs))
            secs.append(time.perf_counter() - t)
    sec = sorted(secs)[1]
    # one thread on a bounded sample: the first tensor's first 4096 tiles
    label, blob, dt = items[0]
    h = O.header(blob)
    t1 = min(4096, h["n_tiles"])
    out, dq = outs[0]
    t = time.perf_counter()
    O.decode(blob, ocode[dt], 0, t1, out=out, dequant=dq)
    sec1 = time.perf_counter() - t
    w1 = min(t1 * h["V"] * 8, h["rows"] * h["cols"])
    # the single-thread run rewrote the first tiles of the first tensor with the same values
    rec = {"value": weights / sec, "unit": "weights/s", "cores": threads, "kind": "oracle",
           "host_cores": len(os.sched_getaffinity(0)),
           "sample": f"all {len(items)} tensors ({weights} weights) decoded by the plain C "
                     f"oracle, tiles split over {threads} threads ({len(os.sched_getaffinity(0))} "
                     f"cores visible); median of 3 passes",
           "seconds": round(sec, 3),
           "cpu": cpu_model(),
           "single_thread": {"value": w1 / sec1, "unit": "weights/s", "cores": 1,
                             "sample": f"{label}: tiles [0, {t1}) ({w1} weights)",
                             "seconds": round(sec1, 3)}}
    return rec, [(out, dq if O.header(blob)["container"] else None)
                 for (out, dq), (_, blob, _) in zip(outs, items)]


def parity_gate(keep, refs, torch):
    """Bit-exact comparison of every decoded weight (and dequant scale) of one GPU step with the
    oracle's decode of the same blobs, before anything is timed."""
    import numpy as np
    n = 0
    for k, (ref, ref_dq) in enumerate(refs):
        out, dq = keep[3 * k + 1], keep[3 * k + 2]
        got = out.view(torch.uint8 if out.element_size() == 1 else
                       torch.int16 if out.element_size() == 2 else torch.int32).cpu().numpy()
        if not np.array_equal(got.reshape(ref.shape), ref.view(got.dtype)):   # bit patterns
            raise SystemExit(f"parity gate: tensor {k} differs from the oracle's decode")
        if ref_dq is not None and not np.array_equal(dq.cpu().numpy(), ref_dq):
            raise SystemExit(f"parity gate: dequant scales of tensor {k} differ from the oracle's")
        n += ref.size
    return {"tensors": len(refs), "weights": n, "bit_exact": True}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mlp_fp8")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the decode shards by tile range with no exchange; see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_34185_amd import entropack as E
    from paper_2609_34185_amd import workloads as W

    E.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.workload == "encode_mlp":
        encode_bench(args, E, W, min(16, len(os.sched_getaffinity(0))))
        return
    if args.workload == "tile_sweep":
        tile_sweep(args, E, W, min(16, len(os.sched_getaffinity(0))))
        return
    if args.workload.startswith("fused_bf16_m"):
        fused_bf16_bench(args, E, W, min(16, len(os.sched_getaffinity(0))),
                         int(args.workload[len("fused_bf16_m"):]))
        return
    if args.workload.startswith("fused_mfma_m"):
        fused_mfma_bench(args, E, W, min(16, len(os.sched_getaffinity(0))),
                         int(args.workload[len("fused_mfma_m"):]))
        return
    if args.workload.startswith("fused_down_m"):
        m = int(args.workload[len("fused_down_m"):])
        fused_bench(args, E, W, min(16, len(os.sched_getaffinity(0))), m)
        return
    threads = min(16, len(os.sched_getaffinity(0)))

    t = time.perf_counter()
    desc, items = workload(args.workload, E, W, threads)
    log(f"workload ready in {time.perf_counter() - t:.1f} s")

    layers, keep = [], []
    weights, algo_bytes = 0, 0
    for label, blob, dt in items:
        info = E.blob_info(blob)
        d_blob = E.to_device(blob, dev)
        out = torch.empty((info.rows, info.cols), dtype=E.torch_dtype(dt), device=dev)
        dq = torch.empty(info.rows, dtype=torch.float32, device=dev) if info.container else None
        keep += [d_blob, out, dq]
        layers.append((info, d_blob.data_ptr(), out.data_ptr(), dq.data_ptr() if dq is not None else 0, dt))
        weights += info.rows * info.cols
        algo_bytes += blob.size + info.rows * info.cols * E.ITEMSIZE[dt] + (4 * info.rows if info.container else 0)
    stored_bpp = 8.0 * sum(b.size for _, b, _ in items) / weights
    ws = max(1, E.stack_workspace(len(layers)))
    d_ws = torch.empty(ws, dtype=torch.uint8, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    # descriptors written once, outside the timed region; a step is one launch
    stack = E.stack_prepare(layers, d_ws.data_ptr(), ws, stream.cuda_stream)

    def step():
        E.stack_decode(stack, status.data_ptr(), stream.cuda_stream)

    # the CPU-baseline leg runs first: the oracle's outputs are the parity gate's reference
    cpu = refs = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle decoder")
        cpu, refs = cpu_baseline(items, threads)
    step()
    torch.cuda.synchronize()
    assert int(status.item()) == 0, "decode reported a corrupt stream"
    gate = None
    if refs is not None:
        log("parity gate: every decoded weight against the oracle")
        gate = parity_gate(keep, refs, torch)
        del refs

    t0 = time.perf_counter()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    settle = 0
    while time.perf_counter() - t0 < SETTLE_S:
        for _ in range(10):
            step()
        settle += 10
        torch.cuda.synchronize()
    assert int(status.item()) == 0, "decode reported a corrupt stream"

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = start.elapsed_time(end) / args.steps
    assert int(status.item()) == 0, "decode reported a corrupt stream"

    cold = cold_cache_ms(step)
    copy_gbps = copy_bandwidth()
    gemm = None
    if args.workload == "mlp_down_int8":
        log("timing the INT8 product of the decoded weights")
        gemm = gemm_leg(E, W, keep[1], layers[0][0])
        gemm["decode_over_gemm"] = ms / gemm["ms"]

    sec = ms / 1e3
    gbps = algo_bytes / sec / 1e9
    traffic = measured_traffic(args.workload)
    line = {
        "metric": METRIC,
        "value": weights / sec,
        "unit": "weights/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": dict(desc, weights=weights, stored_bpp=round(stored_bpp, 4),
                       bytes_per_step=algo_bytes, wall_s=round(wall, 4), settle_steps=settle,
                       cold_cache_ms=cold, measured_copy_gbps=round(copy_gbps, 1),
                       frac_of_measured_copy=round(gbps / copy_gbps, 4)),
        "roofline": {"bound": "hbm", "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": gbps / HBM_PEAK_GBPS, "traffic": traffic},
    }
    line["counters"] = measured_counters(args.workload)
    if gemm is not None:
        line["config"]["gemm"] = gemm
    line["config"]["parity_gate"] = gate
    if cpu is not None:
        line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
