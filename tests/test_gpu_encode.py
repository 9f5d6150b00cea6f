"""GPU parity of the GPU encoder (ep_encode_gpu).

The GPU encoder must produce the oracle encoder's blob byte for byte (same
scale, tables, row scales, states, offsets and payload) on the same seeded
inputs, and the same statistics: the small and ragged cases of the CPU
encoder's parity set (tile sizes that leave partial tiles and odd tile
counts, both containers, b = 9, high rate, the literal state credit, FP16 and
FP32 input), the escalation path, degenerate inputs, and two full-size
tensors (the 3072 x 3072 attention projection, and the 27B-class MLP down
projection in the FP8 row container, also encoded by two host threads at once).
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


def to_device(w: np.ndarray, E, dtype=None):
    """(device tensor, dtype code) of a host matrix: float32, or uint16 bits."""
    w = np.ascontiguousarray(w)
    if dtype is None:
        dtype = E.FP32 if w.dtype == np.float32 else E.BF16
    src = torch.from_numpy(w.view(np.int16) if w.dtype == np.uint16 else w)
    return src.cuda(), dtype


def gpu_encode(E, w, target, dtype=None, **kw):
    d, dt = to_device(w, E, dtype)
    blob, st = E.encode_gpu(d.data_ptr(), w.shape[0], w.shape[1], target, dtype=dt,
                            stream=torch.cuda.current_stream().cuda_stream, **kw)
    return blob, st


def same_stats(g, o):
    assert g["scale"] == o["scale"]
    assert g["prob_bits"] == o["b"]
    assert g["bytes"] == o["bytes"]
    assert g["escalations"] == o["escalations"] and g["coarsenings"] == o["coarsenings"]


CASES = [
    ("cfg1", lambda: W.single_linear(), 4.0, dict(prob_bits=12)),
    ("cfg2_rows", lambda: W.attention_projection()[:700], 3.0, {}),
    ("ragged", lambda: W.ragged_tensor(1, 37, 136), 3.3, dict(tile_vectors=45)),
    ("c8", lambda: W.ragged_tensor(2, 300, 8), 4.0, dict(tile_vectors=33)),
    ("fp8_container", lambda: W.ragged_tensor(3, 128, 512, scale=0.05), 4.0, dict(container=1)),
    ("int8_container", lambda: W.ragged_tensor(4, 128, 512, scale=0.05), 6.0, dict(container=2)),
    ("fp8e5m2_container", lambda: W.ragged_tensor(23, 96, 512, scale=0.05), 4.0, dict(container=3)),
    ("uint8_container", lambda: W.ragged_tensor(24, 80, 520, scale=0.05), 4.0, dict(container=4)),
    ("high_rate", lambda: W.ragged_tensor(5, 64, 1024), 9.0, {}),
    ("b9", lambda: W.ragged_tensor(6, 64, 256), 2.0, dict(prob_bits=9)),
    ("literal_credit", lambda: W.ragged_tensor(7, 96, 512), 3.0, dict(state_credit_bits=16.0)),
    ("one_vector", lambda: W.ragged_tensor(8, 1, 8), 4.0, {}),
    ("v1_tiles", lambda: W.ragged_tensor(9, 5, 64), 4.0, dict(tile_vectors=1)),
]


@pytest.mark.parametrize("name,gen,target,kw", CASES, ids=[c[0] for c in CASES])
def test_gpu_encoder_matches_oracle_bytes(E, oracle, name, gen, target, kw):
    w = gen()
    say(f"  encode {name} {w.shape} at {target}")
    b_or, s_or = oracle.encode(w, target, **kw)
    b_gpu, s_gpu = gpu_encode(E, w, target, **kw)
    assert np.array_equal(b_gpu, b_or)
    same_stats(s_gpu, s_or)


@pytest.mark.parametrize("container", [0, 1, 2])
def test_gpu_encoder_stats_equal_cpu_encoder(E, container):
    """Every statistic equals the CPU encoder's (same definitions); the two relative errors,
    whose row sums the GPU takes as a tree instead of in element order, to 1e-12."""
    w = W.ragged_tensor(3, 128, 1000, scale=0.05)
    _, s_cpu = E.encode(w, 4.0, container=container)
    _, s_gpu = gpu_encode(E, w, 4.0, container=container)
    for k in s_cpu:
        if k.startswith("erel"):
            assert s_gpu[k] == pytest.approx(s_cpu[k], rel=1e-12), k
        else:
            assert s_gpu[k] == s_cpu[k], k


def test_gpu_encoder_escalation_matches_oracle(E, oracle):
    R, Cc = 40, 65536
    rng = np.random.default_rng(12)
    w = (rng.standard_normal((R, Cc)) * 1e-3).astype(np.float32)
    outside = [r for r in range(R) if r not in set(oracle.sample_rows(R, Cc).tolist())]
    w[outside, 5] = 0.02
    b_or, s_or = oracle.encode(w, 10.0, prob_bits=11)
    b_gpu, s_gpu = gpu_encode(E, w, 10.0, prob_bits=11)
    assert s_gpu["escalations"] == s_or["escalations"] > 0
    assert np.array_equal(b_gpu, b_or)


def test_gpu_encoder_fp16_input_matches_oracle(E, oracle):
    rng = np.random.default_rng(8)
    h = (rng.standard_normal((64, 256)) * 0.03).astype(np.float16).view(np.uint16)
    b_or, _ = oracle.encode(h, 4.0, dtype=oracle.FP16)
    b_gpu, _ = gpu_encode(E, h, 4.0, dtype=E.FP16)
    assert np.array_equal(b_gpu, b_or)


def test_gpu_encoder_degenerate_rows_match_oracle(E, oracle):
    """All-zero rows (mu = eta, refit falls back to s mu) and constant rows."""
    w = W.ragged_tensor(10, 48, 256)
    w[3] = 0
    w[7] = 0.25
    w[20:24] = 0
    b_or, _ = oracle.encode(w, 3.0)
    b_gpu, _ = gpu_encode(E, w, 3.0)
    assert np.array_equal(b_gpu, b_or)


def test_gpu_encoder_rejects_bad_input(E):
    bad = np.zeros((4, 16), dtype=np.float32)
    bad[1, 3] = np.inf
    with pytest.raises(E.EntroPackError) as e:
        gpu_encode(E, bad, 4.0)
    assert e.value.code == E.ERR_ARG
    with pytest.raises(E.EntroPackError) as e:
        gpu_encode(E, np.zeros((4, 12), dtype=np.float32), 4.0)
    assert e.value.code == E.ERR_ARG


RDO_CASES = [
    ("rdo_k5", lambda: W.ragged_tensor(3, 96, 512), 3.0, dict(rdo_candidates=5, rdo_sweeps=1)),
    ("rdo_k9_t2", lambda: W.attention_projection()[:300], 3.0, dict(rdo_candidates=9, rdo_sweeps=2)),
    ("rdo_fp8", lambda: W.ragged_tensor(4, 128, 512, scale=0.05), 4.0,
     dict(container=1, rdo_candidates=5, rdo_sweeps=1)),
    ("rdo_int8_ragged", lambda: W.ragged_tensor(5, 77, 136), 6.0,
     dict(container=2, tile_vectors=45, rdo_candidates=4, rdo_sweeps=3)),
]


@pytest.mark.parametrize("name,gen,target,kw", RDO_CASES, ids=[c[0] for c in RDO_CASES])
def test_gpu_encoder_row_refinement_matches_oracle_bytes(E, oracle, name, gen, target, kw):
    """The per-row refinement (Section 3.5, App. C.2) with its candidate passes on the GPU."""
    w = gen()
    b_or, s_or = oracle.encode(w, target, **kw)
    b_gpu, s_gpu = gpu_encode(E, w, target, **kw)
    assert np.array_equal(b_gpu, b_or)
    assert s_gpu["rdo_rows_moved"] == s_or["rdo_rows_moved"]


def test_gpu_encoder_full_size_attention(E, oracle):
    w = W.attention_projection()
    say("  encode 3072 x 3072 at 3.0 (oracle, then GPU)")
    b_or, s_or = oracle.encode(w, 3.0)
    b_gpu, s_gpu = gpu_encode(E, w, 3.0)
    assert np.array_equal(b_gpu, b_or)
    same_stats(s_gpu, s_or)


@pytest.fixture(scope="module")
def mlp_down_fp8(oracle):
    w = W.llm_mlp(["down"])["down"]
    say(f"  oracle encode of MLP down {w.shape} in the FP8 row container at 4.0")
    b_or, s_or = oracle.encode(w, 4.0, container=1)
    return w, b_or, s_or


def test_gpu_encoder_full_size_mlp_down_fp8(E, mlp_down_fp8):
    w, b_or, s_or = mlp_down_fp8
    b_gpu, s_gpu = gpu_encode(E, w, 4.0, container=1)
    assert np.array_equal(b_gpu, b_or)
    same_stats(s_gpu, s_or)


def test_gpu_encoder_concurrent_calls(E, mlp_down_fp8):
    """Two host threads encode the same tensor at once, each on its own stream; their
    payload copies (45 MB, several staging chunks) take the library's pinned staging buffers
    in turn.  Both blobs equal the oracle's."""
    import threading
    w, b_or, _ = mlp_down_fp8
    d, dt = to_device(w, E)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    out, errs = [None, None], []

    def run(i):
        try:
            out[i] = E.encode_gpu(d.data_ptr(), w.shape[0], w.shape[1], 4.0, dtype=dt,
                                  stream=streams[i].cuda_stream, container=1)[0]
        except Exception as e:   # re-raised below, in the test's thread
            errs.append(e)

    threads = [threading.Thread(target=run, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errs, errs
    for b in out:
        assert np.array_equal(b, b_or)
