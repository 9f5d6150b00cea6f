"""GPU parity of the INT8 MFMA product (ep_gemm_i8_nt) and of decode-then-GEMM.

The oracle computes Y = A B^T exactly in int64 (returned as int32); the GPU
result must be equal element for element: on every element for the small and
ragged shapes, on sampled rows for the full-size decode-then-GEMM case (the
INT8-container MLP down projection, 5120 x 17408 at 6.0 bpp, against 8192 x
17408 activations).
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


def gemm_gpu(E, a: np.ndarray, b: np.ndarray) -> np.ndarray:
    da = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    db = torch.from_numpy(np.ascontiguousarray(b)).cuda()
    y = torch.full((a.shape[0], b.shape[0]), -1, dtype=torch.int32, device="cuda")
    E.gemm_i8_nt(da.data_ptr(), db.data_ptr(), y.data_ptr(), a.shape[0], b.shape[0], a.shape[1],
                 torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("m,n,k", [(128, 128, 64), (200, 130, 208), (1, 1, 16), (257, 129, 1024),
                                   (512, 384, 4096), (4300, 4000, 80), (4096, 2560, 48),
                                   (300, 520, 1168), (2304, 2560, 1168), (2048, 1280, 1936),
                                   (16, 5120, 17408)])
def test_gemm_matches_oracle_everywhere(E, oracle, m, n, k):
    """Every element, with Y filled with -1 beforehand.  On a 256-CU device the launch
    takes 4300 x 4000 as 256 whole tiles plus 16 tiles split in halves (ragged in m, n and
    k), 4096 x 2560 as whole tiles only, and 2304 x 2560 as whole tiles plus halves.  K
    walks in 128-byte steps through a ring of five operand slots; k = 1168 (10 steps, the
    last partial) wraps it twice.  Launches of at most 128 units (whole or half tiles)
    split K over several workgroups per unit, whose partial sums meet in Y by atomics after
    a clear: 257 x 129 (2 parts), 512 x 384 (8), 300 x 520 (2), 2048 x 1280 (3 parts of 6,
    6 and 4 steps) and the MLP down projection's shape against 16 rows of activations
    (6 parts of 23 and 21 steps)."""
    rng = np.random.default_rng([11, m, n, k])
    a = rng.integers(-128, 128, (m, k), dtype=np.int8)
    b = rng.integers(-128, 128, (n, k), dtype=np.int8)
    say(f"  gemm {m}x{n}x{k}")
    assert np.array_equal(gemm_gpu(E, a, b), oracle.gemm_i8_nt(a, b))


def test_gemm_extreme_operands(E, oracle):
    """All -128 operands: every sum is 16384 k, the largest magnitude the int8 ranges allow."""
    a = np.full((96, 2048), -128, dtype=np.int8)
    b = np.full((160, 2048), -128, dtype=np.int8)
    y = gemm_gpu(E, a, b)
    assert (y == 16384 * 2048).all()
    assert np.array_equal(y, oracle.gemm_i8_nt(a, b))


def test_gemm_rejects_bad_arguments(E):
    a = torch.zeros((4, 32), dtype=torch.int8, device="cuda")
    y = torch.zeros((4, 4), dtype=torch.int32, device="cuda")
    lib = E.lib()
    assert lib.ep_gemm_i8_nt(a.data_ptr(), a.data_ptr(), y.data_ptr(), 4, 4, 24, None) == E.ERR_ARG
    assert lib.ep_gemm_i8_nt(a.data_ptr(), a.data_ptr(), y.data_ptr(), 0, 4, 32, None) == E.ERR_ARG
    assert lib.ep_gemm_i8_nt(None, a.data_ptr(), y.data_ptr(), 4, 4, 32, None) == E.ERR_ARG


def test_config5_decode_then_gemm(E, oracle):
    """Decode the INT8-container down projection on the GPU, multiply by the activations on
    MFMA, and compare sampled rows with the oracle's product of the oracle-decoded weights,
    then every element with an independent library GEMM."""
    say("  cfg5: generating and encoding the down projection (INT8 container, 6.0 bpp)")
    w = W.llm_mlp(["down"])["down"]
    blob, _ = E.encode(w, 6.0, container=E.CONT_INT8_ROW)
    ref_w, ref_dq = oracle.decode(blob, oracle.INT8)
    info = E.blob_info(blob)
    out, dq, st = E.decode(blob, E.INT8, info=info)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert np.array_equal(out.cpu().numpy(), ref_w)
    assert np.array_equal(dq.cpu().numpy(), ref_dq)
    say("  cfg5: activations 8192 x 17408 and the MFMA product")
    act = W.llm_activations()
    d_act = torch.from_numpy(act).cuda()
    y = torch.empty((act.shape[0], info.rows), dtype=torch.int32, device="cuda")
    E.gemm_i8_nt(d_act.data_ptr(), out.data_ptr(), y.data_ptr(), act.shape[0], info.rows,
                 info.cols, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, act.shape[0] - 1],
                                     np.random.default_rng(5).choice(act.shape[0], 14, replace=False)]))
    say(f"  cfg5: oracle product on {rows.size} sampled rows")
    ref = oracle.gemm_i8_nt(act, ref_w, rows=rows)
    got = y[torch.from_numpy(rows).cuda()].cpu().numpy()
    assert np.array_equal(got, ref)
    # every element against an independent GEMM (the vendor library behind torch._int_mm,
    # used only as a checker here): int32 sums of int8 products are exact in both
    if hasattr(torch, "_int_mm"):
        say("  cfg5: all of Y against torch._int_mm")
        ind = torch._int_mm(d_act, out.view(torch.int8).t())
        torch.cuda.synchronize()
        assert torch.equal(ind, y)
