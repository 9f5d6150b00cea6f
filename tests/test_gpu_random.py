"""GPU parity on seeded random configurations.

Each case draws a shape (rows of 1 to 300, row lengths of 8 to 1600), a tile size, a
target rate, a container, the probability precision b (or the encoder's own rule), a body
distribution with outliers and two output types, encodes with the oracle encoder, and
decodes on the GPU through the decode path ep_blob_info chose and, in one case out of four,
through the global-table path; every output element (bits) and every dequant scale must
equal the oracle's decode.  The fixed seed makes the set reproducible; it reaches
combinations the hand-written cases do not (short and long rows against small and large
tiles, every container with every output type, b from 9 to 12).
"""
import sys

import numpy as np
import pytest

from paper_2609_34185_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

N_CASES = 40
OUT = ["COORD2", "BF16", "FP16", "FP32", "FP8", "INT8", "E5M2", "UINT8"]


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def E():
    from paper_2609_34185_amd import entropack
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    entropack.lib()
    return entropack


def codes(E, oracle, name):
    return {"COORD2": (E.COORD2_I32, oracle.COORD2), "BF16": (E.BF16, oracle.BF16),
            "FP16": (E.FP16, oracle.FP16), "FP32": (E.FP32, oracle.FP32),
            "FP8": (E.FP8_E4M3, oracle.FP8), "INT8": (E.INT8, oracle.INT8),
            "E5M2": (E.FP8_E5M2, oracle.FP8E5), "UINT8": (E.UINT8, oracle.UINT8)}[name]


def gpu_bits(t):
    t = t.cpu()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float8_e4m3fn, torch.float8_e5m2):
        return t.view(torch.uint8).numpy()
    return t.numpy()


def draw_case(i: int):
    rng = np.random.default_rng([7, i])
    rows = int(rng.integers(1, 301))
    cols = 8 * int(rng.integers(1, 201))
    body = str(rng.choice(["gauss", "t5"]))
    w = W.draw_tensor(rng, rows, cols, body=body, log_mu=float(rng.uniform(-6, 0)),
                      log_sigma=float(rng.uniform(0, 0.8)), outlier_rate=float(rng.choice([0, 0.002])),
                      outlier_factor=float(rng.uniform(2, 12)))
    kw = dict(tile_vectors=int(rng.choice([1, 7, 32, 45, 100, 512, 700])),
              container=int(rng.integers(0, 5)))
    pb = int(rng.choice([0, 0, 9, 10, 11, 12]))
    if pb:
        kw["prob_bits"] = pb
    target = float(rng.uniform(1.5, 8.0))
    outs = ["COORD2"] + [str(x) for x in rng.choice(OUT[1:], 2, replace=False)]
    force_global = bool(rng.integers(0, 4) == 0)
    return w, target, kw, outs, force_global


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_configuration(E, oracle, i):
    w, target, kw, outs, force_global = draw_case(i)
    say(f"  case {i}: {w.shape} at {target:.2f} bpp {kw} -> {outs}"
        f"{' (global-table path)' if force_global else ''}")
    blob, _ = oracle.encode(w, target, **kw)
    info = E.blob_info(blob)
    if force_global:
        info.path = 4
    d_blob = E.to_device(blob)
    for name in outs:
        ecode, ocode = codes(E, oracle, name)
        out, dq, st = E.decode(blob, ecode, d_blob=d_blob, info=info)
        torch.cuda.synchronize()
        ref, ref_dq = oracle.decode(blob, ocode)
        assert int(st.item()) == 0, name
        got = gpu_bits(out)
        if not np.array_equal(got, ref):
            bad = np.argwhere(got != ref)
            r, c = bad[0]
            raise AssertionError(f"{name}: {len(bad)} mismatches, first at {r},{c}: "
                                 f"gpu {got[r, c]} oracle {ref[r, c]}")
        if info.container:
            assert np.array_equal(dq.cpu().numpy(), ref_dq), name


N_LISTS = 10


def draw_layer(rng):
    rows = int(rng.integers(1, 161))
    cols = 8 * int(rng.integers(1, 121))
    w = W.draw_tensor(rng, rows, cols, body=str(rng.choice(["gauss", "t5"])),
                      log_mu=float(rng.uniform(-5, -1)), log_sigma=float(rng.uniform(0, 0.6)))
    kw = dict(tile_vectors=int(rng.choice([7, 32, 100, 512])), container=int(rng.integers(0, 5)))
    pb = int(rng.choice([0, 0, 9, 12]))
    if pb:
        kw["prob_bits"] = pb
    return w, float(rng.uniform(1.5, 7.5)), kw, str(rng.choice(OUT))


@pytest.mark.parametrize("i", range(N_LISTS))
def test_random_layer_list(E, oracle, i):
    """A list of 1 to 12 random layers (paths, containers and output types mixed) decoded in
    one launch: by ep_decode_layers (descriptors by value up to 8 layers, in the workspace
    above) and by a prepared stack; every layer against the oracle."""
    rng = np.random.default_rng([8, i])
    n = int(rng.integers(1, 13))
    drawn = [draw_layer(rng) for _ in range(n)]
    blobs = [oracle.encode(w, t, **kw)[0] for w, t, kw, _ in drawn]
    infos = [E.blob_info(b) for b in blobs]
    say(f"  list {i}: {n} layers, paths {[x.path for x in infos]}, "
        f"outputs {[d[3] for d in drawn]}")
    dev = [E.to_device(b) for b in blobs]
    for how in ("layers", "stack"):
        outs, dqs, layers = [], [], []
        for (w, _, _, name), info, d in zip(drawn, infos, dev):
            code = codes(E, oracle, name)[0]
            o = torch.empty((info.rows, info.cols), dtype=E.torch_dtype(code), device="cuda")
            q = torch.zeros(info.rows, dtype=torch.float32, device="cuda") if info.container else None
            outs.append(o)
            dqs.append(q)
            layers.append((info, d.data_ptr(), o.data_ptr(), q.data_ptr() if q is not None else 0, code))
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        if how == "layers":
            ws = E.decode_layers_workspace(n)
            d_ws = torch.empty(max(1, ws), dtype=torch.uint8, device="cuda")
            E.decode_layers(layers, d_ws.data_ptr(), ws, status.data_ptr(), s)
        else:
            ws = E.stack_workspace(n)
            d_ws = torch.empty(max(1, ws), dtype=torch.uint8, device="cuda")
            st = E.stack_prepare(layers, d_ws.data_ptr(), ws, s)
            E.stack_decode(st, status.data_ptr(), s)
        torch.cuda.synchronize()
        assert int(status.item()) == 0, how
        for k, ((_, _, _, name), blob, info, o, q) in enumerate(zip(drawn, blobs, infos, outs, dqs)):
            ref, ref_dq = oracle.decode(blob, codes(E, oracle, name)[1])
            assert np.array_equal(gpu_bits(o), ref), (how, k, name)
            if info.container:
                assert np.array_equal(q.cpu().numpy(), ref_dq), (how, k)


N_FUSED = 10


@pytest.mark.parametrize("i", range(N_FUSED))
def test_random_fused_products(E, oracle, i):
    """The fused decode and MFMA products on random tensors and rows of X: the INT8 product
    (INT8 row container) exact against the oracle's decode and exact product; the BF16
    product (any blob) within its fp32 summation bound against the oracle's bf16 decode
    multiplied in fp64."""
    rng = np.random.default_rng([9, i])
    rows = int(rng.integers(1, 201))
    cols = 8 * int(rng.integers(1, 151))
    m = int(rng.choice([1, 3, 16, 17, 33, 64, 100, 257]))
    w = W.draw_tensor(rng, rows, cols, body="gauss", log_mu=float(rng.uniform(-5, -1)),
                      log_sigma=0.4)
    V = int(rng.choice([7, 45, 512]))
    s = torch.cuda.current_stream().cuda_stream
    say(f"  fused {i}: {w.shape}, V = {V}, m = {m}")
    # INT8 product on the INT8 row container
    blob, _ = oracle.encode(w, float(rng.uniform(3, 7)), container=oracle.CONT_INT8, tile_vectors=V)
    info = E.blob_info(blob)
    d_blob = E.to_device(blob)
    x = rng.integers(-127, 128, (m, cols), dtype=np.int8)
    d_x = torch.from_numpy(x).cuda()
    y = torch.empty((m, rows), dtype=torch.int32, device="cuda")
    dq = torch.empty(rows, dtype=torch.float32, device="cuda")
    ws = E.decode_gemm_i8_workspace(info)
    d_ws = torch.empty(ws, dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    E.decode_gemm_i8(info, d_blob.data_ptr(), d_x.data_ptr(), m, y.data_ptr(), d_ws.data_ptr(), ws,
                     dq.data_ptr(), status.data_ptr(), s)
    torch.cuda.synchronize()
    wd, ref_dq = oracle.decode(blob, oracle.INT8)
    assert int(status.item()) == 0
    assert np.array_equal(y.cpu().numpy(), oracle.gemm_i8_nt(x, wd))
    assert np.array_equal(dq.cpu().numpy(), ref_dq)
    # BF16 product on a direct blob
    blob, _ = oracle.encode(w, float(rng.uniform(2, 6)), tile_vectors=V)
    info = E.blob_info(blob)
    d_blob = E.to_device(blob)
    xb = torch.from_numpy(rng.standard_normal((m, cols)).astype(np.float32)).to(torch.bfloat16).cuda()
    yb = torch.empty((m, rows), dtype=torch.float32, device="cuda")
    ws = E.decode_gemm_bf16_workspace(info)
    d_ws = torch.empty(ws, dtype=torch.uint8, device="cuda")
    E.decode_gemm_bf16(info, d_blob.data_ptr(), xb.data_ptr(), m, yb.data_ptr(), d_ws.data_ptr(), ws,
                       0, status.data_ptr(), s)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    wbits, _ = oracle.decode(blob, oracle.BF16)
    wf = (wbits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    xf = xb.float().cpu().numpy().astype(np.float64)
    exact = xf @ wf.T
    bound = (cols + 18) * 2.0 ** -24 * (np.abs(xf) @ np.abs(wf).T)
    assert (np.abs(yb.cpu().numpy().astype(np.float64) - exact) <= bound).all()


N_ENCODE = 15


@pytest.mark.parametrize("i", range(N_ENCODE))
def test_random_gpu_encoder(E, oracle, i):
    """The GPU encoder on random tensors (BF16 or FP32 input, every container, tile sizes,
    rates and precisions as above): the blob equals the oracle encoder's byte for byte."""
    w, target, kw, _, _ = draw_case(100 + i)
    rng = np.random.default_rng([10, i])
    if rng.integers(0, 2):
        w = (w.astype(np.uint32) << 16).view(np.float32)   # the same values as FP32 input
    say(f"  GPU encode {i}: {w.shape} {w.dtype} at {target:.2f} bpp {kw}")
    ref, _ = oracle.encode(w, target, **kw)
    src = torch.from_numpy(w.view(np.int16) if w.dtype == np.uint16 else w).cuda()
    dt = E.FP32 if w.dtype == np.float32 else E.BF16
    blob, _ = E.encode_gpu(src.data_ptr(), w.shape[0], w.shape[1], target, dtype=dt,
                           stream=torch.cuda.current_stream().cuda_stream, **kw)
    assert np.array_equal(blob, ref)
