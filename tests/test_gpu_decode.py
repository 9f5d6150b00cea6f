"""GPU parity: the HIP decode (through the C ABI) against the oracle decoder.

Every blob here comes from the oracle encoder; the GPU output must equal the
oracle's bit for bit (doubled coordinates, weights in every output dtype, and
the container dequant scales), with a clean status word.
"""
import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from paper_2609_34185_amd import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

DTYPES = ["COORD2", "BF16", "FP16", "FP32", "FP8", "INT8", "E5M2", "UINT8"]


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def E():
    from paper_2609_34185_amd import entropack
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    entropack.lib()
    return entropack


# Launches of few four-tile tasks run two-tile tasks (one chain per wave) unless
# EP_SMALL_TASK_LIMIT says otherwise; the small-size tests below run both ways.
TASKS = ["one_chain", "two_chain"]


class task_mode:
    """Context: "two_chain" sets EP_SMALL_TASK_LIMIT=0 (always four-tile tasks)."""

    def __init__(self, mode):
        self.mode = mode

    def __enter__(self):
        self.old = os.environ.get("EP_SMALL_TASK_LIMIT")
        if self.mode == "two_chain":
            os.environ["EP_SMALL_TASK_LIMIT"] = "0"
        else:
            os.environ.pop("EP_SMALL_TASK_LIMIT", None)

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("EP_SMALL_TASK_LIMIT", None)
        else:
            os.environ["EP_SMALL_TASK_LIMIT"] = self.old


def codes(E, oracle, name):
    return {"COORD2": (E.COORD2_I32, oracle.COORD2), "BF16": (E.BF16, oracle.BF16),
            "FP16": (E.FP16, oracle.FP16), "FP32": (E.FP32, oracle.FP32),
            "FP8": (E.FP8_E4M3, oracle.FP8), "INT8": (E.INT8, oracle.INT8),
            "E5M2": (E.FP8_E5M2, oracle.FP8E5), "UINT8": (E.UINT8, oracle.UINT8)}[name]


def gpu_bits(t):
    """Host numpy view of a device tensor's bits, matching the oracle's arrays."""
    t = t.cpu()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float8_e4m3fn, torch.float8_e5m2):
        return t.view(torch.uint8).numpy()
    return t.numpy()


def check_blob(E, oracle, blob, dtypes=DTYPES, tag="", path=None):
    """Decode `blob` on the GPU to every type in `dtypes` and compare with the oracle bit for
    bit.  `path` forces a decode path other than the one ep_blob_info chose (any path that can
    hold the tables must give the same result)."""
    info = E.blob_info(blob)
    if path is not None:
        info.path = path
    d_blob = E.to_device(blob)
    for name in dtypes:
        ecode, ocode = codes(E, oracle, name)
        say(f"  decode {tag} {info.rows}x{info.cols} b={info.prob_bits} path={info.path} -> {name}")
        out, dq, st = E.decode(blob, ecode, d_blob=d_blob, info=info)
        torch.cuda.synchronize()
        ref, ref_dq = oracle.decode(blob, ocode)
        assert int(st.item()) == 0
        got = gpu_bits(out)
        if not np.array_equal(got, ref):
            bad = np.argwhere(got != ref)
            r, c = bad[0]
            raise AssertionError(f"{name}: {len(bad)} mismatches, first at {r},{c}: "
                                 f"gpu {got[r, c]} oracle {ref[r, c]}")
        if info.container:
            assert np.array_equal(dq.cpu().numpy(), ref_dq)
    return info


def test_config1_all_dtypes_search_path(E, oracle):
    blob, st = oracle.encode(W.single_linear(), 4.0, prob_bits=12)
    info = check_blob(E, oracle, blob, tag="cfg1")
    assert info.path == 2


@pytest.mark.parametrize("tasks", TASKS)
def test_config1_all_dtypes_lut_path(E, oracle, tasks):
    blob, st = oracle.encode(W.single_linear(), 4.0, prob_bits=11)
    with task_mode(tasks):
        info = check_blob(E, oracle, blob, tag=f"cfg1-b11 {tasks}")
    assert info.path == 1


@pytest.mark.parametrize("tasks", TASKS)
def test_config2_fp16_bf16(E, oracle, tasks):
    blob, st = oracle.encode(W.attention_projection(), 3.0)
    with task_mode(tasks):
        check_blob(E, oracle, blob, dtypes=["COORD2", "FP16", "BF16", "FP8", "INT8"],
                   tag=f"cfg2 {tasks}")


@pytest.mark.parametrize("b", [9, 10, 11, 12, 13, 14, 15])
def test_every_probability_precision(E, oracle, b):
    w = W.ragged_tensor(20 + b, 96, 704)
    blob, st = oracle.encode(w, 4.5, prob_bits=b)
    check_blob(E, oracle, blob, dtypes=["COORD2", "BF16"], tag=f"b{b}")


def search_fits(b, sum_A):
    """Whether the bucketed-search tables (u16 cumulative values, 2^k + 1 bucket bounds per
    table for some k in min(b, 11) .. 8, metadata) fit the 128 KiB the payload rings leave."""
    cum = (2 * (sum_A + 16) + 3) & ~3
    for k in range(min(b, 11), 7, -1):
        meta = (cum + 2 * 16 * ((1 << k) + 1) + 3) & ~3
        if ((meta + 128 + 511) & ~511) <= 128 * 1024:
            return sum_A <= 0xFFFF0
    return False


def expected_path(info):
    """The decode path rule: narrow slot entries while every doubled coordinate lies in
    [-256, 255], wide ones up to [-1024, 1023] (both for b <= 11), else bucketed search when
    its tables fit the LDS, else the global-table path."""
    if info.prob_bits <= 11 and -256 <= info.coord2_min and info.coord2_max <= 255:
        return 1
    if info.prob_bits <= 11 and -1024 <= info.coord2_min and info.coord2_max <= 1023:
        return 3
    return 2 if search_fits(info.prob_bits, info.sum_alphabet) else 4


@pytest.mark.parametrize("target", [6.0, 8.0, 10.0])
def test_high_rates_large_alphabets(E, oracle, target):
    """High targets give wide coordinate ranges and large tables (b = 12 at 8 bpp): wide
    slot entries or the bucketed-search path decode them; both build their tables in LDS
    from the blob."""
    w = W.attention_projection()[:512, :2048]
    blob, st = oracle.encode(w, target)
    info = check_blob(E, oracle, blob, dtypes=["COORD2", "BF16", "FP16"], tag=f"rate{target}")
    assert info.path == expected_path(info) and info.path in (2, 3)
    say(f"    b={info.prob_bits} sum_A={info.sum_alphabet} coord2 [{info.coord2_min}, {info.coord2_max}]")


@pytest.mark.parametrize("b", [9, 10, 11])
def test_wide_slot_entries(E, oracle, b):
    """Coordinates beyond a signed byte at b <= 11 take the wide slot entries (f - 1, u - F
    and a 10-bit coordinate field): every output type, full and ragged tiles, both row
    modes of the steady state (C/8 below and above V - 32)."""
    for rows, cols in ((96, 2048), (131, 3000), (64, 4096)):
        w = (W.ragged_tensor(40 + b, rows, cols).astype(np.uint32) << 16).view(np.float32).copy()
        w[:, :8] *= 8.0   # a few large columns widen the coordinate range
        blob, st = oracle.encode(w, 6.0, prob_bits=b)
        info = E.blob_info(blob)
        say(f"    {rows}x{cols} b={info.prob_bits} coord2 [{info.coord2_min}, {info.coord2_max}]")
        assert info.path == 3, (info.prob_bits, info.coord2_min, info.coord2_max)
        for tasks in TASKS if b == 11 else TASKS[:1]:
            with task_mode(tasks):
                check_blob(E, oracle, blob, tag=f"wide{b} {tasks}")


def escalated_blobs(oracle):
    """Two blobs of App. C.1's precision escalation, from a tensor whose sampled rows miss
    large values in the other rows: at 10 bpp the alphabet escalates b to 13 (bucketed search
    in LDS); at 14 bpp it exceeds 2^15 and the scale is coarsened at b = 15 (sum of the table
    ranges 77,519, largest 31,209: beyond any LDS table, the global-table path)."""
    R, Cc = 40, 65536
    rng = np.random.default_rng(12)
    w = (rng.standard_normal((R, Cc)) * 1e-3).astype(np.float32)
    outside = [r for r in range(R) if r not in set(oracle.sample_rows(R, Cc).tolist())]
    out = []
    for val, target in ((0.02, 10.0), (0.5, 14.0)):
        w[outside, 5] = val
        blob, st = oracle.encode(w, target, prob_bits=11)
        out.append((blob, st))
    return out


def test_escalated_precision_blobs(E, oracle):
    """Every valid blob decodes on the GPU, bit-exact: the escalated one (b = 13) from LDS
    search tables, the coarsened one (b = 15, tables too large for LDS) through the
    global-table path, whose frequencies stay in the blob in global memory."""
    (b13, s13), (b15, s15) = escalated_blobs(oracle)
    assert s13["b"] == 13 and s13["coarsenings"] == 0
    assert s15["b"] == 15 and s15["coarsenings"] >= 1
    i13, i15 = E.blob_info(b13), E.blob_info(b15)
    say(f"    b=13 sum_A={i13.sum_alphabet} path={i13.path}; b=15 sum_A={i15.sum_alphabet} path={i15.path}")
    assert i13.path == expected_path(i13) == 2
    assert i15.path == expected_path(i15) == 4 and i15.sum_alphabet == 77519
    check_blob(E, oracle, b13, dtypes=["COORD2", "BF16"], tag="esc b13")
    check_blob(E, oracle, b15, dtypes=["COORD2", "BF16", "FP32", "FP16"], tag="coarsened b15")


@pytest.mark.parametrize("case", ["cfg1", "ragged45", "c8", "fp8c", "int8c", "b9", "b15", "wide", "V1"])
def test_global_table_path_on_any_blob(E, oracle, case):
    """The global-table path holds any valid table, so forcing it on blobs that would take
    another path must give the same bits: every output type, ragged tiles, containers with
    their scales, b from 9 to 15 and wide coordinates."""
    gen = {
        "cfg1": lambda: oracle.encode(W.single_linear(), 4.0, prob_bits=12),
        "ragged45": lambda: oracle.encode(W.ragged_tensor(1, 37, 136), 3.3, tile_vectors=45),
        "c8": lambda: oracle.encode(W.ragged_tensor(2, 300, 8), 4.0, tile_vectors=33),
        "fp8c": lambda: oracle.encode(W.ragged_tensor(3, 128, 512, scale=0.05), 4.0, container=1),
        "int8c": lambda: oracle.encode(W.ragged_tensor(4, 128, 512, scale=0.05), 6.0, container=2),
        "b9": lambda: oracle.encode(W.ragged_tensor(6, 64, 256), 2.0, prob_bits=9),
        "b15": lambda: oracle.encode(W.ragged_tensor(7, 64, 1024), 9.0, prob_bits=15),
        "wide": lambda: oracle.encode(W.attention_projection()[:256, :2048], 8.0),
        "V1": lambda: oracle.encode(W.ragged_tensor(8, 1, 4096), 3.0, tile_vectors=1),
    }[case]
    blob, _ = gen()
    check_blob(E, oracle, blob, tag=f"global {case}", path=4)


def test_decode_refuses_a_path_that_cannot_hold_the_tables(E, oracle):
    """A caller-edited info naming a slot-table path for tables it cannot hold is refused on
    the host with EP_ERR_ARG, before any launch."""
    (b13, _), _ = escalated_blobs(oracle)
    info = E.blob_info(b13)
    info.path = 1
    with pytest.raises(E.EntroPackError) as ei:
        E.decode(b13, E.COORD2_I32, info=info)
    assert ei.value.code == E.ERR_ARG


@pytest.mark.parametrize("tasks", TASKS)
@pytest.mark.parametrize("shape,V", [((1, 8), 512), ((3, 24), 32), ((7, 400), 45),
                                     ((33, 264), 512), ((130, 72), 100), ((300, 8), 33),
                                     ((65, 1000), 77), ((1, 4096), 1), ((5, 1024), 64)])
def test_ragged_shapes_and_tiles(E, oracle, shape, V, tasks):
    """Tensors of one tile to a few hundred, ragged last tiles and odd tile counts (a two-tile
    task with one tile, a four-tile task with one to three)."""
    w = W.ragged_tensor(8, *shape)
    blob, st = oracle.encode(w, 3.0, tile_vectors=V)
    with task_mode(tasks):
        check_blob(E, oracle, blob, dtypes=["COORD2", "BF16", "FP8"], tag=f"V{V} {tasks}")


@pytest.mark.parametrize("tasks", TASKS)
@pytest.mark.parametrize("shape,V", [((400, 136), 45), ((200, 520), 77), ((120, 1024), 100),
                                     ((64, 2048), 33)])
def test_partial_last_round_in_the_steady_state(E, oracle, shape, V, tasks):
    """Tiles whose length is not a multiple of 32 vectors run the slot-table steady state with
    a partial last round; a lane's vectors then lie 32 (ceil(V / 32) - 1) vectors apart, so
    with rows of 17, 65, 128 and 256 vectors they span up to three rows, and the row scale
    of each vector must still be its own (every output type)."""
    w = W.ragged_tensor(50 + V, *shape)
    blob, st = oracle.encode(w, 4.0, tile_vectors=V)
    info = E.blob_info(blob)
    assert info.prob_bits == 11 and info.path in (1, 3)
    with task_mode(tasks):
        check_blob(E, oracle, blob, tag=f"partial V{V} {tasks}")


@pytest.mark.parametrize("tasks", TASKS)
@pytest.mark.parametrize("V", [455, 1820])
def test_paper_tile_sizes_at_full_size(E, oracle, V, tasks):
    """The paper's default tile sizes of 4096 and 16384 symbols (Table tileoverhead: 455 and
    1820 vectors, not multiples of 32) on the reference-layer shape 10240 x 3840 at 4.0 bpp,
    decoded at full size to BF16 and to doubled coordinates: every element equals the oracle.
    The slot-table steady state runs these tiles with a partial last round.  Blobs come from
    the library encoder, byte-identical to the oracle's (checked on the first tiles' bytes of
    the same layer in the CPU encoder tests; here the two decoders are compared)."""
    w = dict(W.dit_block(0))["blocks.0.mlp_in"]
    blob, st = E.encode(w, 4.0, tile_vectors=V)
    info = E.blob_info(blob)
    assert info.tile_vectors == V and info.path in (1, 3) and info.prob_bits == 11
    say(f"    V={V}: {info.n_tiles} tiles, {st['rate_stored']:.4f} bpp, path {info.path}")
    with task_mode(tasks):
        check_blob(E, oracle, blob, dtypes=["COORD2", "BF16"], tag=f"V{V} {tasks}")


def test_tile_ranges_write_only_their_tiles(E, oracle):
    blob, st = oracle.encode(W.ragged_tensor(3, 200, 520), 3.5, tile_vectors=64)
    info = E.blob_info(blob)
    d_blob = E.to_device(blob)
    full, _ = oracle.decode(blob, oracle.BF16)
    out = torch.full((info.rows, info.cols), 7, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    st_t = torch.zeros(1, dtype=torch.int32, device="cuda")
    for t0, t1 in [(0, 3), (3, 4), (4, 4), (5, info.n_tiles)]:
        E.decode(blob, E.BF16, d_blob=d_blob, info=info, tile_begin=t0, tile_end=t1, out=out,
                 status=st_t)
    torch.cuda.synchronize()
    got = gpu_bits(out).reshape(-1)
    ref = full.reshape(-1)
    V8 = 64 * 8
    assert np.array_equal(got[:4 * V8], ref[:4 * V8])
    assert np.all(got[4 * V8:5 * V8] == 7)                 # tile 4 was never decoded
    assert np.array_equal(got[5 * V8:], ref[5 * V8:])
    assert int(st_t.item()) == 0


def test_degenerate_tensors(E, oracle):
    # all zeros: one coset, zero scales-by-fallback, every output zero
    z = np.zeros((64, 128), dtype=np.float32)
    blob, st = oracle.encode(z, 4.0)
    info = check_blob(E, oracle, blob, dtypes=["COORD2", "BF16", "INT8"], tag="zeros")
    assert info.coset_f1 == 0
    # constant rows
    c = np.full((16, 64), 0.25, dtype=np.float32)
    blob, st = oracle.encode(c, 2.0)
    check_blob(E, oracle, blob, dtypes=["COORD2", "FP16"], tag="const")


@pytest.mark.parametrize("tasks", TASKS)
def test_saturation(E, oracle, tasks):
    rng = np.random.default_rng(4)
    w = (rng.standard_normal((32, 256)) * 3e4).astype(np.float32)
    w[0, :8] = 1e5
    blob, st = oracle.encode(w, 5.0)
    with task_mode(tasks):
        check_blob(E, oracle, blob, dtypes=["FP16", "FP8", "INT8", "BF16", "E5M2"], tag=f"sat {tasks}")
    w[1, :8] = 9e4   # beyond e5m2's 57344
    blob, st = oracle.encode(w, 5.0)
    with task_mode(tasks):
        check_blob(E, oracle, blob, dtypes=["E5M2"], tag=f"sat e5m2 {tasks}")


@pytest.mark.parametrize("shape,target,kw", [
    ((96, 8 * 1000), 4.0, {}),                        # full tasks, slot-table steady state
    ((64, 8 * 640), 7.0, {}),                         # larger coordinates
    ((37, 136), 4.0, dict(tile_vectors=45)),          # ragged tiles: the generic loop
    ((64, 8 * 600), 6.0, dict(prob_bits=12)),         # the bucketed-search path
])
def test_fp8_e5m2_and_uint8_containers(E, oracle, shape, target, kw):
    """The FP8 e5m2 row container and the UINT8 tensor container (the paper's dtype table),
    decoded to their types with their scales."""
    w = W.ragged_tensor(31, *shape, scale=0.05)
    blob, _ = oracle.encode(w, target, container=oracle.CONT_FP8E5, **kw)
    check_blob(E, oracle, blob, dtypes=["E5M2", "COORD2", "FP32"], tag="e5m2 container")
    blob, _ = oracle.encode(w, target, container=oracle.CONT_UINT8, **kw)
    check_blob(E, oracle, blob, dtypes=["UINT8", "COORD2"], tag="uint8 container")


def test_corrupt_payload_sets_status_without_fault(E, oracle):
    blob, st = oracle.encode(W.ragged_tensor(6, 128, 512), 4.0)
    info = E.blob_info(blob)
    bad = blob.copy()
    bad[info.off_payload + 200: info.off_payload + 260] ^= 0x5A
    assert oracle.decode_status(bad) == oracle.ERR_CORRUPT
    out, dq, stt = E.decode(bad, E.COORD2_I32)
    torch.cuda.synchronize()
    assert int(stt.item()) != 0


# ---- the paper-shaped workloads at full size ------------------------------------

@pytest.fixture(scope="module")
def mlp():
    say("  generating the 27B-class MLP set (seed 2)")
    return W.llm_mlp()


@pytest.fixture(scope="module")
def mlp_fp8_blobs(oracle, mlp):
    names = ["gate", "up", "down"]
    with ThreadPoolExecutor(3) as ex:
        res = list(ex.map(lambda n: oracle.encode(mlp[n], 4.0, container=oracle.CONT_FP8), names))
    return {n: r[0] for n, r in zip(names, res)}


def test_config3_full_size_fp8_in_one_launch(E, oracle, mlp_fp8_blobs):
    """The benchmark's configuration: gate, up and down decoded by one ep_decode_layers call."""
    names = ["gate", "up", "down"]
    infos = {n: E.blob_info(mlp_fp8_blobs[n]) for n in names}
    dev = {n: E.to_device(mlp_fp8_blobs[n]) for n in names}
    outs = {n: torch.zeros((infos[n].rows, infos[n].cols), dtype=torch.float8_e4m3fn, device="cuda")
            for n in names}
    dqs = {n: torch.zeros(infos[n].rows, dtype=torch.float32, device="cuda") for n in names}
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    layers = [(infos[n], dev[n].data_ptr(), outs[n].data_ptr(), dqs[n].data_ptr(), E.FP8_E4M3)
              for n in names]
    ws = max(1, E.decode_layers_workspace(len(layers)))
    d_ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
    say("  ep_decode_layers over gate/up/down")
    E.decode_layers(layers, d_ws.data_ptr(), ws, st.data_ptr(),
                    torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    with ThreadPoolExecutor(3) as ex:
        refs = dict(zip(names, ex.map(lambda n: oracle.decode(mlp_fp8_blobs[n], oracle.FP8), names)))
    for n in names:
        assert infos[n].path == 1
        assert np.array_equal(gpu_bits(outs[n]), refs[n][0]), n
        assert np.array_equal(dqs[n].cpu().numpy(), refs[n][1]), n


def test_prepared_stack_decodes_like_the_oracle(E, oracle, mlp_fp8_blobs):
    """ep_stack_prepare once, then ep_stack_decode twice into cleared outputs: both decodes
    equal the oracle (the descriptors stay valid across launches)."""
    names = ["gate", "up", "down"]
    infos = {n: E.blob_info(mlp_fp8_blobs[n]) for n in names}
    dev = {n: E.to_device(mlp_fp8_blobs[n]) for n in names}
    outs = {n: torch.zeros((infos[n].rows, infos[n].cols), dtype=torch.float8_e4m3fn, device="cuda")
            for n in names}
    dqs = {n: torch.zeros(infos[n].rows, dtype=torch.float32, device="cuda") for n in names}
    layers = [(infos[n], dev[n].data_ptr(), outs[n].data_ptr(), dqs[n].data_ptr(), E.FP8_E4M3)
              for n in names]
    ws = E.stack_workspace(len(layers))
    d_ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    st = E.stack_prepare(layers, d_ws.data_ptr(), ws, stream)
    assert st.n_layers == 3 and st.path == 1 and st.total_tasks == 65280 // 4
    refs = {n: oracle.decode(mlp_fp8_blobs[n], oracle.FP8) for n in names}
    for rep in range(2):
        for n in names:
            outs[n].view(torch.uint8).fill_(0x55)
            dqs[n].fill_(-1.0)
        status = torch.zeros(1, dtype=torch.int32, device="cuda")
        say(f"  ep_stack_decode, launch {rep}")
        E.stack_decode(st, status.data_ptr(), stream)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        for n in names:
            assert np.array_equal(gpu_bits(outs[n]), refs[n][0]), (rep, n)
            assert np.array_equal(dqs[n].cpu().numpy(), refs[n][1]), (rep, n)


def test_stack_rejects_bad_arguments(E):
    st = E.Stack()
    assert E.lib().ep_stack_decode(None, None, None) == E.ERR_ARG
    st.n_layers = 2   # never prepared: no workspace
    assert E.lib().ep_stack_decode(E.C.byref(st), None, None) == E.ERR_ARG
    assert E.lib().ep_stack_prepare(None, 1, None, 0, E.C.byref(st), None) == E.ERR_ARG


def test_config3_product_encoder_reproduces_oracle_blobs(E, mlp, mlp_fp8_blobs):
    """The benchmark encodes with the library's encoder; at full size it emits the same bytes."""
    for n in ["gate", "down"]:
        b, _ = E.encode(mlp[n], 4.0, container=E.CONT_FP8_ROW)
        assert np.array_equal(b, mlp_fp8_blobs[n]), n


def test_config5_down_int8_container(E, oracle, mlp):
    blob, st = oracle.encode(mlp["down"], 6.0, container=oracle.CONT_INT8)
    info = check_blob(E, oracle, blob, dtypes=["INT8", "COORD2"], tag="cfg5")
    assert info.path == 3   # coordinates beyond a signed byte: wide slot entries


def test_mixed_path_stack_in_one_launch(E, oracle, mlp, mlp_fp8_blobs):
    """Layers whose tables take different decode paths decode in one launch: the config-3
    FP8 set (narrow slot tables), the config-5 INT8-container down projection (wide slot
    tables), the two escalated blobs (LDS search tables; the global-table path) and three
    ragged layers (the generic loop), through ep_decode_layers (nine layers: descriptors in the
    workspace) and through a prepared stack decoded twice."""
    b5, _ = oracle.encode(mlp["down"], 6.0, container=oracle.CONT_INT8)
    (b13, _), (b15, _) = escalated_blobs(oracle)
    items = [(mlp_fp8_blobs[n], "FP8") for n in ("gate", "up", "down")]
    items += [(b5, "INT8"), (b13, "BF16"), (b15, "BF16")]
    for seed, shape, V in ((1, (37, 136), 45), (2, (300, 8), 33), (5, (65, 1000), 77)):
        items.append((oracle.encode(W.ragged_tensor(seed, *shape), 3.0, tile_vectors=V)[0], "FP16"))
    infos = [E.blob_info(b) for b, _ in items]
    assert [i.path for i in infos[:6]] == [1, 1, 1, 3, 2, 4]
    dev = [E.to_device(b) for b, _ in items]
    outs = [torch.empty((i.rows, i.cols), dtype=E.torch_dtype(codes(E, oracle, dt)[0]), device="cuda")
            for i, (_, dt) in zip(infos, items)]
    dqs = [torch.zeros(i.rows, dtype=torch.float32, device="cuda") if i.container else None for i in infos]
    layers = [(i, d.data_ptr(), o.data_ptr(), q.data_ptr() if q is not None else 0, codes(E, oracle, dt)[0])
              for i, d, o, q, (_, dt) in zip(infos, dev, outs, dqs, items)]
    with ThreadPoolExecutor(8) as ex:
        refs = list(ex.map(lambda it: oracle.decode(it[0], codes(E, oracle, it[1])[1]), items))
    stream = torch.cuda.current_stream().cuda_stream

    def check(tag):
        for k, (o, q, (ref, ref_dq)) in enumerate(zip(outs, dqs, refs)):
            assert np.array_equal(gpu_bits(o), ref), (tag, k, infos[k].path)
            if q is not None:
                assert np.array_equal(q.cpu().numpy(), ref_dq), (tag, k)

    def clear():
        for o in outs:
            o.view(torch.uint8).fill_(0x55)

    clear()
    ws = E.decode_layers_workspace(len(layers))
    d_ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    say("  ep_decode_layers over 9 layers on 5 decode paths")
    E.decode_layers(layers, d_ws.data_ptr(), ws, st.data_ptr(), stream)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    check("decode_layers")
    sws = E.stack_workspace(len(layers))
    d_sws = torch.zeros(sws, dtype=torch.uint8, device="cuda")
    stk = E.stack_prepare(layers, d_sws.data_ptr(), sws, stream)
    for rep in range(2):
        clear()
        st.zero_()
        say(f"  mixed prepared stack, launch {rep}")
        E.stack_decode(stk, st.data_ptr(), stream)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        check(f"stack {rep}")


def test_config4_stack_two_blocks_one_launch(E, oracle):
    """Two diffusion-transformer blocks (12 layers at full layer shapes) in one
    ep_decode_layers launch; more than 8 layers use the workspace descriptor list."""
    say("  generating 2 DiT blocks")
    layers_np = W.dit_stack(2, workers=2)
    with ThreadPoolExecutor(8) as ex:
        blobs = list(ex.map(lambda lw: oracle.encode(lw[1], 2.5)[0], layers_np))
    infos = [E.blob_info(b) for b in blobs]
    dev = [E.to_device(b) for b in blobs]
    outs = [torch.zeros((i.rows, i.cols), dtype=torch.bfloat16, device="cuda") for i in infos]
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    layers = [(i, d.data_ptr(), o.data_ptr(), 0, E.BF16) for i, d, o in zip(infos, dev, outs)]
    ws = E.decode_layers_workspace(len(layers))
    assert ws > 0
    d_ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
    say("  ep_decode_layers over 12 layers")
    E.decode_layers(layers, d_ws.data_ptr(), ws, st.data_ptr(),
                    torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    with ThreadPoolExecutor(8) as ex:
        refs = list(ex.map(lambda b: oracle.decode(b, oracle.BF16)[0], blobs))
    for (name, _), o, r in zip(layers_np, outs, refs):
        assert np.array_equal(gpu_bits(o), r), name


def test_config4_full_stack_sampled_tiles(E, oracle):
    """The full diffusion-transformer configuration as the benchmark runs it: 30 blocks (180
    layers, 4.13e9 weights) at 2.5 bpp, one prepared-stack launch to BF16.  The oracle decodes
    sampled tiles of every layer (first, last and three drawn at random) one by one; each
    must equal the GPU's output over that tile's weights.  Blobs come from the library's CPU
    encoder, whose bytes equal the oracle encoder's (checked here on one layer, and on the
    encoder parity set in the CPU tests)."""
    blobs, names = [], []
    with ThreadPoolExecutor(8) as ex:   # blocks drawn ahead while earlier ones encode
        drawn = list(ex.map(W.dit_block, range(30)))
    for blk, block in enumerate(drawn):
        for name, w in block:
            b, _ = E.encode(w, 2.5)
            if blk == 0 and name.endswith(".q"):
                assert np.array_equal(b, oracle.encode(w, 2.5)[0])
            blobs.append(b)
            names.append(name)
        drawn[blk] = None
        if blk % 5 == 4:
            say(f"  encoded {blk + 1} blocks")
    infos = [E.blob_info(b) for b in blobs]
    dev = [E.to_device(b) for b in blobs]
    outs = [torch.empty((i.rows, i.cols), dtype=torch.bfloat16, device="cuda") for i in infos]
    for o in outs:
        o.view(torch.int16).fill_(0x7FC1)   # NaN pattern, which a decode never writes
    layers = [(i, d.data_ptr(), o.data_ptr(), 0, E.BF16) for i, d, o in zip(infos, dev, outs)]
    ws = E.stack_workspace(len(layers))
    d_ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    st = E.stack_prepare(layers, d_ws.data_ptr(), ws, stream)
    assert st.n_layers == 180 and st.total_tasks == 1008000 // 4
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    say("  ep_stack_decode over 180 layers")
    E.stack_decode(st, status.data_ptr(), stream)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    # every weight of every layer was written: no sentinel left anywhere
    for name, o in zip(names, outs):
        assert not bool((o.view(torch.int16) == 0x7FC1).any()), name
    rng = np.random.default_rng(44)
    for name, blob, info, o in zip(names, blobs, infos, outs):
        picks = sorted({0, info.n_tiles - 1, *rng.choice(info.n_tiles, 3, replace=False).tolist()})
        flat = o.view(torch.int16).view(-1)
        for t in picks:
            ref, _ = oracle.decode(blob, oracle.BF16, t, t + 1)
            a, b = t * 4096, min((t + 1) * 4096, info.rows * info.cols)
            got = flat[a:b].cpu().numpy().view(np.uint16)
            assert np.array_equal(got, ref.reshape(-1)[a:b]), (name, t)
    say("  sampled tiles of all 180 layers equal the oracle")
