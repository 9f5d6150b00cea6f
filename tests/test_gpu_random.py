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
