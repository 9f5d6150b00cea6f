"""GPU parity of the fused decode and small-batch product (ep_decode_matmul_i8).

Y = X W'^T, with W' the INT8 container matrix of a blob and X a few int8 rows,
must equal the oracle's product of the oracle-decoded W' exactly, on every
element: the steady state with per-lane sums for 1, 2, 4 and 8 rows of X (rows
at least a tile long, tiles crossing rows), rows shorter than a tile (every
vector added on its own), ragged tiles (the generic loop), b = 12 (the search
path), the full-size 27B-class MLP down projection at 6.0 bpp, and the delta
output.  The call overwrites Y, so a second call into the same buffer must
give the same result.
"""
import sys

import numpy as np
import pytest

from paper_2609_34185_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def E():
    from paper_2609_34185_amd import entropack
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    entropack.lib()
    return entropack


def activations(seed: int, m: int, cols: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(-127, 128, (m, cols), dtype=np.int8)


def fused(E, blob: np.ndarray, x: np.ndarray, twice: bool = False):
    """(Y, delta, status) of the fused product on the GPU."""
    info = E.blob_info(blob)
    d_blob = torch.from_numpy(blob).cuda()
    d_x = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    m = x.shape[0]
    y = torch.full((m, info.rows), 7, dtype=torch.int32, device="cuda")
    dq = torch.zeros(info.rows, dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    for _ in range(2 if twice else 1):
        E.decode_matmul_i8(info, d_blob.data_ptr(), d_x.data_ptr(), m, y.data_ptr(), dq.data_ptr(),
                           st.data_ptr(), s)
    torch.cuda.synchronize()
    return y.cpu().numpy(), dq.cpu().numpy(), int(st.item())


def reference(oracle, blob: np.ndarray, x: np.ndarray):
    w, dq = oracle.decode(blob, oracle.INT8)
    return oracle.gemm_i8_nt(x, w), dq


CASES = [
    # name, generator, target, encode kwargs, rows of X
    ("long_rows_m1", lambda: W.ragged_tensor(11, 96, 8 * 1000, scale=0.05), 6.0, {}, 1),
    ("long_rows_m2", lambda: W.ragged_tensor(12, 80, 8 * 1100, scale=0.05), 6.0, {}, 2),
    ("long_rows_m3", lambda: W.ragged_tensor(13, 64, 8 * 640, scale=0.05), 4.0, {}, 3),
    ("long_rows_m4", lambda: W.ragged_tensor(14, 72, 8 * 777, scale=0.05), 6.0, {}, 4),
    ("long_rows_m8", lambda: W.ragged_tensor(15, 70, 8 * 1024, scale=0.05), 6.0, {}, 8),
    ("row_just_short_of_a_tile_m5", lambda: W.ragged_tensor(16, 64, 8 * 500, scale=0.05), 6.0, {}, 5),
    ("short_rows_m4", lambda: W.ragged_tensor(17, 300, 512, scale=0.05), 6.0, {}, 4),
    ("ragged_tiles_m2", lambda: W.ragged_tensor(18, 37, 136, scale=0.05), 6.0, dict(tile_vectors=45), 2),
    ("ragged_tiles_m7", lambda: W.ragged_tensor(19, 41, 8 * 333, scale=0.05), 5.0, dict(tile_vectors=96), 7),
    ("b12_search_m3", lambda: W.ragged_tensor(20, 64, 8 * 600, scale=0.05), 6.0, dict(prob_bits=12), 3),
    ("one_vector_m1", lambda: W.ragged_tensor(21, 1, 8, scale=0.05), 6.0, {}, 1),
]


@pytest.mark.parametrize("name,gen,target,kw,m", CASES, ids=[c[0] for c in CASES])
def test_fused_product_matches_oracle(E, oracle, name, gen, target, kw, m):
    w = gen()
    say(f"  fused {name}: {w.shape} at {target}, m = {m}")
    blob, _ = oracle.encode(w, target, container=oracle.CONT_INT8, **kw)
    x = activations(len(name), m, w.shape[1])
    y_ref, dq_ref = reference(oracle, blob, x)
    y, dq, st = fused(E, blob, x, twice=True)
    assert st == 0
    assert np.array_equal(y, y_ref)
    assert np.array_equal(dq, dq_ref)


def test_fused_product_config5_down(E, oracle):
    """The INT8-container MLP down projection (5120 x 17408, 6.0 bpp) times the first
    rows of the 8192 x 17408 activations, every element of Y."""
    say("  fused cfg5: encoding the down projection (INT8 container, 6.0 bpp)")
    w = W.llm_mlp(["down"])["down"]
    blob, _ = E.encode(w, 6.0, container=E.CONT_INT8_ROW)
    act = W.llm_activations()
    w_ref, dq_ref = oracle.decode(blob, oracle.INT8)
    for m in (1, 4, 8):
        x = act[:m]
        say(f"  fused cfg5: m = {m}")
        y, dq, st = fused(E, blob, x)
        assert st == 0
        assert np.array_equal(y, oracle.gemm_i8_nt(x, w_ref))
        assert np.array_equal(dq, dq_ref)


def test_fused_product_rejects_bad_arguments(E, oracle):
    w = W.ragged_tensor(22, 32, 256, scale=0.05)
    blob_int8, _ = oracle.encode(w, 6.0, container=oracle.CONT_INT8)
    blob_fp8, _ = oracle.encode(w, 6.0, container=oracle.CONT_FP8)
    x = activations(1, 9, 256)
    d_x = torch.from_numpy(x).cuda()
    y = torch.zeros((9, 32), dtype=torch.int32, device="cuda")
    lib = E.lib()
    for blob, m, code in ((blob_fp8, 1, E.ERR_UNSUPPORTED), (blob_int8, 0, E.ERR_ARG),
                          (blob_int8, 9, E.ERR_ARG)):
        info = E.blob_info(blob)
        d_blob = torch.from_numpy(blob).cuda()
        rc = lib.ep_decode_matmul_i8(E.C.byref(info), d_blob.data_ptr(), d_x.data_ptr(), m,
                                     y.data_ptr(), None, None, None)
        assert rc == code
    info = E.blob_info(blob_int8)
    d_blob = torch.from_numpy(blob_int8).cuda()
    assert lib.ep_decode_matmul_i8(E.C.byref(info), d_blob.data_ptr(), None, 1, y.data_ptr(),
                                   None, None, None) == E.ERR_ARG


# ---- the fused decode and MFMA product (any number of rows of X) ---------------------

def fused_mfma(E, blob: np.ndarray, x: np.ndarray, twice: bool = False, prepared: bool = False,
               path: int = 0):
    """(Y, delta, status) of ep_decode_gemm_i8 on the GPU; Y starts as garbage.  With
    `prepared`, ep_decode_gemm_i8_prepare first builds the tables into the workspace and
    ep_decode_gemm_i8_prepared runs on it."""
    info = E.blob_info(blob)
    if path:
        info.path = path
    d_blob = torch.from_numpy(blob).cuda()
    d_x = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    m = x.shape[0]
    y = torch.full((m, info.rows), 7, dtype=torch.int32, device="cuda")
    dq = torch.zeros(info.rows, dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = E.decode_gemm_i8_workspace(info)
    d_ws = torch.full((max(1, ws),), 0xA5, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    run = E.decode_gemm_i8
    if prepared:
        E.decode_gemm_i8_prepare(info, d_blob.data_ptr(), d_ws.data_ptr(), ws, s)
        run = E.decode_gemm_i8_prepared
    for _ in range(2 if twice else 1):
        run(info, d_blob.data_ptr(), d_x.data_ptr(), m, y.data_ptr(), d_ws.data_ptr(), ws,
            dq.data_ptr(), st.data_ptr(), s)
    torch.cuda.synchronize()
    return y.cpu().numpy(), dq.cpu().numpy(), int(st.item())


MFMA_CASES = [
    # name, generator, target, encode kwargs, rows of X
    ("long_rows_m16", lambda: W.ragged_tensor(31, 96, 8 * 1000, scale=0.05), 6.0, {}, 16),
    ("long_rows_m1", lambda: W.ragged_tensor(32, 40, 8 * 700, scale=0.05), 6.0, {}, 1),
    ("long_rows_m17", lambda: W.ragged_tensor(33, 50, 8 * 640, scale=0.05), 4.0, {}, 17),
    ("long_rows_m64", lambda: W.ragged_tensor(34, 72, 8 * 777, scale=0.05), 6.0, {}, 64),
    ("long_rows_m100", lambda: W.ragged_tensor(35, 33, 8 * 1024, scale=0.05), 6.0, {}, 100),
    ("long_rows_m256", lambda: W.ragged_tensor(36, 48, 8 * 520, scale=0.05), 6.0, {}, 256),
    ("long_rows_m300", lambda: W.ragged_tensor(37, 20, 8 * 300, scale=0.05), 6.0, {}, 300),
    ("short_rows_m40", lambda: W.ragged_tensor(38, 300, 512, scale=0.05), 6.0, {}, 40),
    ("tiny_rows_m33", lambda: W.ragged_tensor(39, 200, 24, scale=0.05), 6.0, dict(tile_vectors=45), 33),
    ("ragged_tiles_m20", lambda: W.ragged_tensor(40, 41, 8 * 333, scale=0.05), 5.0, dict(tile_vectors=96), 20),
    ("b12_search_m48", lambda: W.ragged_tensor(41, 64, 8 * 600, scale=0.05), 6.0, dict(prob_bits=12), 48),
    ("one_vector_m5", lambda: W.ragged_tensor(42, 1, 8, scale=0.05), 6.0, {}, 5),
    # 40-row blocks (three slab tiles); 64-row blocks (four) in two rounds of workgroups
    ("blocks_of_40_rows_m40", lambda: W.ragged_tensor(45, 10240, 64, scale=0.05), 6.0, {}, 40),
    ("two_rounds_m7", lambda: W.ragged_tensor(46, 16640, 64, scale=0.05), 6.0, {}, 7),
    ("two_rounds_m72", lambda: W.ragged_tensor(47, 16640, 64, scale=0.05), 6.0, {}, 72),
]


@pytest.mark.parametrize("prepared", [False, True], ids=["tables_built", "tables_prepared"])
@pytest.mark.parametrize("name,gen,target,kw,m", MFMA_CASES, ids=[c[0] for c in MFMA_CASES])
def test_fused_mfma_product_matches_oracle(E, oracle, name, gen, target, kw, m, prepared):
    """Every element of Y against the oracle's decode followed by its exact product: token
    counts from 1 to 300 (K split over waves below 256 rows of X, whole token tiles above),
    rows longer and shorter than a tile, blocks of 16 rows cut by tiles, blocks of 40 and 64
    rows (three and four slab tiles against one, two or more X tiles per work item), the
    64-row blocks in two rounds of workgroups, ragged tiles (the generic loop), b = 12 (the
    search path), and two calls into the same Y; with the tables built in every workgroup and
    copied from a prepared workspace."""
    w = gen()
    say(f"  fused MFMA {name}: {w.shape} at {target}, m = {m}, prepared = {prepared}")
    blob, _ = oracle.encode(w, target, container=oracle.CONT_INT8, **kw)
    x = activations(100 + len(name), m, w.shape[1])
    y_ref, dq_ref = reference(oracle, blob, x)
    y, dq, st = fused_mfma(E, blob, x, twice=True, prepared=prepared)
    assert st == 0
    assert np.array_equal(y, y_ref)
    assert np.array_equal(dq, dq_ref)


@pytest.mark.parametrize("prepared", [False, True], ids=["tables_built", "tables_prepared"])
def test_fused_mfma_product_global_table_path(E, oracle, prepared):
    """The same product when the tables are read through the global-table path."""
    w = W.ragged_tensor(43, 64, 8 * 512, scale=0.05)
    blob, _ = oracle.encode(w, 6.0, container=oracle.CONT_INT8)
    x = activations(7, 24, w.shape[1])
    y_ref, dq_ref = reference(oracle, blob, x)
    y, dq, st = fused_mfma(E, blob, x, prepared=prepared, path=4)
    assert st == 0
    assert np.array_equal(y, y_ref)
    assert np.array_equal(dq, dq_ref)


def test_fused_mfma_product_config5_down(E, oracle):
    """The INT8-container MLP down projection (5120 x 17408, 6.0 bpp) times the first 1, 16, 64
    and 256 rows of the 8192 x 17408 activations: every element of Y."""
    w = W.llm_mlp(["down"])["down"]
    blob, _ = E.encode(w, 6.0, container=E.CONT_INT8_ROW)
    act = W.llm_activations()
    w_ref, dq_ref = oracle.decode(blob, oracle.INT8)
    for m, prepared in ((1, True), (16, False), (16, True), (64, True), (256, False)):
        x = act[:m]
        say(f"  fused MFMA cfg5: m = {m}, prepared = {prepared}")
        y, dq, st = fused_mfma(E, blob, x, prepared=prepared)
        assert st == 0
        assert np.array_equal(y, oracle.gemm_i8_nt(x, w_ref))
        assert np.array_equal(dq, dq_ref)


def test_fused_mfma_product_rejects_bad_arguments(E, oracle):
    w = W.ragged_tensor(44, 32, 256, scale=0.05)
    blob_int8, _ = oracle.encode(w, 6.0, container=oracle.CONT_INT8)
    blob_fp8, _ = oracle.encode(w, 6.0, container=oracle.CONT_FP8)
    x = activations(1, 20, 256)
    d_x = torch.from_numpy(x).cuda()
    y = torch.zeros((20, 32), dtype=torch.int32, device="cuda")
    lib = E.lib()
    info8 = E.blob_info(blob_int8)
    ws = E.decode_gemm_i8_workspace(info8)
    d_ws = torch.empty(ws, dtype=torch.uint8, device="cuda")
    for blob, m, wsb, code in ((blob_fp8, 1, ws, E.ERR_UNSUPPORTED), (blob_int8, 0, ws, E.ERR_ARG),
                               (blob_int8, 20, ws - 1, E.ERR_ARG)):
        info = E.blob_info(blob)
        d_blob = torch.from_numpy(blob).cuda()
        rc = lib.ep_decode_gemm_i8(E.C.byref(info), d_blob.data_ptr(), d_x.data_ptr(), m,
                                   y.data_ptr(), None, d_ws.data_ptr(), wsb, None, None)
        assert rc == code
        rc = lib.ep_decode_gemm_i8_prepared(E.C.byref(info), d_blob.data_ptr(), d_x.data_ptr(), m,
                                            y.data_ptr(), None, d_ws.data_ptr(), wsb, None, None)
        assert rc == code
        if m:
            rc = lib.ep_decode_gemm_i8_prepare(E.C.byref(info), d_blob.data_ptr(), d_ws.data_ptr(),
                                               wsb, None)
            assert rc == code


# ---- the fused decode and BF16 MFMA product --------------------------------------
def bf16_bits(f: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest even) and return the bits."""
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def bf16_values(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def bf16_activations(seed: int, m: int, cols: int) -> np.ndarray:
    return bf16_bits(np.random.default_rng(seed).standard_normal((m, cols)).astype(np.float32))


def fused_bf16(E, blob: np.ndarray, xbits: np.ndarray, prepared: bool = False, twice: bool = False):
    """(Y fp32, delta, status) of ep_decode_gemm_bf16 on the GPU; Y starts as garbage."""
    info = E.blob_info(blob)
    d_blob = torch.from_numpy(blob).cuda()
    d_x = torch.from_numpy(np.ascontiguousarray(xbits).view(np.int16)).cuda()
    m = xbits.shape[0]
    y = torch.full((m, info.rows), 7.0, dtype=torch.float32, device="cuda")
    dq = torch.zeros(info.rows, dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = E.decode_gemm_bf16_workspace(info)
    d_ws = torch.full((max(1, ws),), 0xA5, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream().cuda_stream
    run = E.decode_gemm_bf16
    if prepared:
        E.decode_gemm_bf16_prepare(info, d_blob.data_ptr(), d_ws.data_ptr(), ws, s)
        run = E.decode_gemm_bf16_prepared
    for _ in range(2 if twice else 1):
        run(info, d_blob.data_ptr(), d_x.data_ptr(), m, y.data_ptr(), d_ws.data_ptr(), ws,
            dq.data_ptr(), st.data_ptr(), s)
    torch.cuda.synchronize()
    return y.cpu().numpy(), dq.cpu().numpy(), int(st.item())


def check_bf16_product(oracle, blob: np.ndarray, xbits: np.ndarray, y: np.ndarray):
    """Y against the exact product of the oracle's bf16 decode, within the fp32 summation
    bound: every product of two bf16 values is exact in fp32, and at most C + 16 + 2
    roundings of 2^-24 relative size fall on any partial sum, so
    |Y - X W'^T| <= (C + 18) 2^-24 sum_j |X[t][j] W'[r][j]|."""
    wbits, _ = oracle.decode(blob, oracle.BF16)
    w = bf16_values(wbits)
    x = bf16_values(xbits)
    exact = x @ w.T
    bound = (x.shape[1] + 18) * 2.0 ** -24 * (np.abs(x) @ np.abs(w).T)
    err = np.abs(y.astype(np.float64) - exact)
    worst = np.argmax(err - bound)
    assert (err <= bound).all(), (f"{int((err > bound).sum())} elements beyond the bound; worst "
                                  f"{np.unravel_index(worst, err.shape)}: err {err.flat[worst]:.3e} "
                                  f"bound {bound.flat[worst]:.3e}")
    # the bound is a small fraction of Y's typical size, so a wrong row, column or scale
    # (errors of that size) cannot hide within it
    assert np.median(bound) < 0.05 * np.sqrt(np.mean(exact ** 2))


BF16_CASES = [
    # name, generator, target, encode kwargs, rows of X
    ("direct_long_rows_m16", lambda: W.ragged_tensor(61, 96, 8 * 1000), 4.0, {}, 16),
    ("direct_m1", lambda: W.ragged_tensor(62, 40, 8 * 700), 3.0, {}, 1),
    ("direct_m17_short_rows", lambda: W.ragged_tensor(63, 300, 512), 4.0, {}, 17),
    ("direct_m64_ragged_tiles", lambda: W.ragged_tensor(64, 41, 8 * 333), 5.0, dict(tile_vectors=96), 64),
    ("direct_m300", lambda: W.ragged_tensor(65, 20, 8 * 300), 4.0, {}, 300),
    ("direct_b12_search_m20", lambda: W.ragged_tensor(66, 64, 8 * 600), 4.0, dict(prob_bits=12), 20),
    ("int8_container_m16", lambda: W.ragged_tensor(67, 64, 8 * 777, scale=0.05), 6.0,
     dict(container="INT8"), 16),
    ("fp8_container_m33", lambda: W.ragged_tensor(68, 50, 8 * 640, scale=0.05), 4.0,
     dict(container="FP8"), 33),
    ("direct_two_rounds_m40", lambda: W.ragged_tensor(69, 16640, 64), 4.0, {}, 40),
]


@pytest.mark.parametrize("prepared", [False, True], ids=["tables_built", "tables_prepared"])
@pytest.mark.parametrize("name,gen,target,kw,m", BF16_CASES, ids=[c[0] for c in BF16_CASES])
def test_fused_bf16_product_matches_oracle(E, oracle, name, gen, target, kw, m, prepared):
    """Every element of Y within the fp32 summation bound of the exact product of the oracle's
    bf16 decode: direct blobs and both containers, rows longer and shorter than a tile,
    ragged tiles, the search path, 1 to 300 rows of X (K split over waves below 256 rows), two
    calls into the same Y, and the tables built in every workgroup or prepared."""
    w = gen()
    kw = dict(kw)
    if kw.get("container") == "INT8":
        kw["container"] = oracle.CONT_INT8
    elif kw.get("container") == "FP8":
        kw["container"] = oracle.CONT_FP8
    say(f"  fused BF16 {name}: {w.shape} at {target}, m = {m}, prepared = {prepared}")
    blob, _ = oracle.encode(w, target, **kw)
    xbits = bf16_activations(200 + len(name), m, w.shape[1])
    y, dq, st = fused_bf16(E, blob, xbits, prepared=prepared, twice=True)
    assert st == 0
    check_bf16_product(oracle, blob, xbits, y)
    if E.blob_info(blob).container:
        assert np.array_equal(dq, oracle.decode(blob, oracle.BF16)[1])


def test_fused_bf16_product_dit_layer(E, oracle):
    """The diffusion-transformer MLP input projection (10240 x 3840 at 2.5 bpp, the paper's
    reference-layer shape) times 16 and 64 rows of bf16 activations: every element within
    the bound."""
    w = dict(W.dit_block(0))["blocks.0.mlp_in"]
    blob, _ = E.encode(w, 2.5)
    for m, prepared in ((16, False), (64, True)):
        say(f"  fused BF16 DiT mlp_in: m = {m}, prepared = {prepared}")
        xbits = bf16_activations(300 + m, m, w.shape[1])
        y, _, st = fused_bf16(E, blob, xbits, prepared=prepared)
        assert st == 0
        check_bf16_product(oracle, blob, xbits, y)


def test_fused_bf16_product_rejects_bad_arguments(E, oracle):
    w = W.ragged_tensor(69, 32, 256)
    blob, _ = oracle.encode(w, 4.0)
    info = E.blob_info(blob)
    d_blob = torch.from_numpy(blob).cuda()
    x = torch.zeros((20, 256), dtype=torch.int16, device="cuda")
    y = torch.zeros((20, 32), dtype=torch.float32, device="cuda")
    ws = E.decode_gemm_bf16_workspace(info)
    assert ws > E.decode_gemm_i8_workspace(info)   # bf16 slabs are twice the size
    d_ws = torch.empty(ws, dtype=torch.uint8, device="cuda")
    lib = E.lib()
    for m, wsb in ((0, ws), (70000, ws), (20, ws - 1)):
        for fn in (lib.ep_decode_gemm_bf16, lib.ep_decode_gemm_bf16_prepared):
            rc = fn(E.C.byref(info), d_blob.data_ptr(), x.data_ptr(), m, y.data_ptr(), None,
                    d_ws.data_ptr(), wsb, None, None)
            assert rc == E.ERR_ARG
    assert lib.ep_decode_gemm_bf16_prepare(E.C.byref(info), d_blob.data_ptr(), d_ws.data_ptr(), ws - 1,
                                           None) == E.ERR_ARG
    # the INT8 product refuses a tensor outside the INT8 container; the BF16 one takes it
    assert lib.ep_decode_gemm_i8(E.C.byref(info), d_blob.data_ptr(), x.data_ptr(), 20, y.data_ptr(),
                                 None, d_ws.data_ptr(), ws, None, None) == E.ERR_UNSUPPORTED
