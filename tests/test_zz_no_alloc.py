"""GPU test of ep_decode_layers_noalloc, the decode entry point that allocates nothing (its
descriptor list lives in a static device array of the library): on two calls in a row, the
second with fewer and smaller layers, its output equals ep_decode_layers' output bit for bit
(and both equal the oracle's), and a list longer than the array is refused."""
import sys
from concurrent.futures import ThreadPoolExecutor

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


def bits(t):
    t = t.cpu()
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float8_e4m3fn, torch.float8_e5m2):
        return t.view(torch.uint8).numpy()
    return t.numpy()


def layer_list(E, oracle, specs):
    """Encode (oracle) and upload; returns (infos, device blobs, layers for the C ABI of both
    entry points, their outputs, oracle references).  specs: (seed, rows, cols, target, kw, E dtype, oracle dtype)."""
    with ThreadPoolExecutor(8) as ex:
        blobs = list(ex.map(lambda sp: oracle.encode(W.ragged_tensor(sp[0], sp[1], sp[2], scale=0.05),
                                                       sp[3], **sp[4])[0], specs))
    infos = [E.blob_info(b) for b in blobs]
    dev = [E.to_device(b) for b in blobs]

    def outputs():
        return [(torch.full((i.rows, i.cols), 0x55, dtype=torch.uint8, device="cuda")
                 .view(E.torch_dtype(sp[5])) if E.ITEMSIZE[sp[5]] == 1 else
                 torch.zeros((i.rows, i.cols), dtype=E.torch_dtype(sp[5]), device="cuda"),
                 torch.zeros(i.rows, dtype=torch.float32, device="cuda") if i.container else None)
                for i, sp in zip(infos, specs)]

    outs_ws, outs_na = outputs(), outputs()

    def layers(outs):
        return [(i, d.data_ptr(), o.data_ptr(), q.data_ptr() if q is not None else 0, sp[5])
                for i, d, (o, q), sp in zip(infos, dev, outs, specs)]

    refs = [oracle.decode(b, sp[6]) for b, sp in zip(blobs, specs)]
    # the device blobs go back with the lists: the launches read them through raw pointers
    return infos, dev, layers(outs_ws), layers(outs_na), outs_ws, outs_na, refs


def run_both(E, oracle, specs, tag):
    infos, dev, lw, ln, ow, on, refs = layer_list(E, oracle, specs)
    stream = torch.cuda.current_stream().cuda_stream
    ws = max(1, E.decode_layers_workspace(len(lw)))
    d_ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
    st_w = torch.zeros(1, dtype=torch.int32, device="cuda")
    st_n = torch.zeros(1, dtype=torch.int32, device="cuda")
    say(f"  {tag}: ep_decode_layers over {len(lw)} layers, paths {[i.path for i in infos]}")
    E.decode_layers(lw, d_ws.data_ptr(), ws, st_w.data_ptr(), stream)
    say(f"  {tag}: ep_decode_layers_noalloc over {len(ln)} layers")
    E.decode_layers_noalloc(ln, st_n.data_ptr(), stream)
    torch.cuda.synchronize()
    sw, sn = int(st_w.item()), int(st_n.item())
    assert sw == 0, f"workspace status {sw}"
    assert sn == 0, f"no-alloc status {sn}"
    for k, ((a, qa), (b, qb), (ref, ref_dq)) in enumerate(zip(ow, on, refs)):
        assert np.array_equal(bits(b), bits(a)), (tag, k)
        assert np.array_equal(bits(b), ref), (tag, k)
        if qa is not None:
            assert np.array_equal(qb.cpu().numpy(), qa.cpu().numpy()), (tag, k)
            assert np.array_equal(qb.cpu().numpy(), ref_dq), (tag, k)


def test_noalloc_decode_equals_workspace_decode(E, oracle):
    O = oracle
    big = [  # 12 layers: slot tables (narrow and wide), search tables, containers, ragged tiles
        (1, 256, 2048, 4.0, {}, E.BF16, O.BF16),
        (2, 300, 1024, 3.0, {}, E.FP16, O.FP16),
        (3, 128, 4096, 4.0, dict(container=1), E.FP8_E4M3, O.FP8),
        (4, 128, 4096, 6.0, dict(container=2), E.INT8, O.INT8),
        (5, 77, 136, 3.3, dict(tile_vectors=45), E.BF16, O.BF16),
        (6, 96, 2048, 8.0, {}, E.FP32, O.FP32),
        (7, 64, 1024, 4.5, dict(prob_bits=13), E.COORD2_I32, O.COORD2),
        (8, 300, 8, 4.0, dict(tile_vectors=33), E.BF16, O.BF16),
        (9, 512, 512, 2.5, {}, E.BF16, O.BF16),
        (10, 200, 520, 3.5, dict(tile_vectors=64), E.FP16, O.FP16),
        (11, 64, 3000, 6.0, {}, E.BF16, O.BF16),
        (12, 40, 4096, 4.0, dict(container=3), E.FP8_E5M2, O.FP8E5),
    ]
    small = [  # then 3 smaller layers: the array keeps the first call's longer list behind
        (21, 33, 264, 3.0, {}, E.BF16, O.BF16),
        (22, 16, 512, 4.0, dict(container=1), E.FP8_E4M3, O.FP8),
        (23, 7, 400, 3.0, dict(tile_vectors=45), E.FP16, O.FP16),
    ]
    run_both(E, oracle, big, "call 1")
    run_both(E, oracle, small, "call 2")


def test_noalloc_refuses_more_layers_than_its_array(E):
    arr = (E.Layer * 513)()
    assert E.lib().ep_decode_layers_noalloc(arr, 513, None, None) == E.ERR_ARG
    assert b"512" in E.lib().ep_last_error()
