"""Pins of the coset-conditioned model, the code length and the stored-size
estimate (Sections 3.3, 3.4; Appendix C.3, Table tileoverhead)."""
import numpy as np
import pytest

from paper_2609_34185_amd import workloads as W


@pytest.mark.parametrize("b", [9, 11, 12, 15])
def test_normalisation_sums_and_support(oracle, b):
    rng = np.random.default_rng(b)
    for trial in range(40):
        A = int(rng.integers(1, min(600, 1 << b) + 1))
        n = rng.geometric(rng.uniform(0.01, 0.9), size=A).astype(np.uint64) - 1
        n[rng.random(A) < 0.3] = 0
        if n.sum() == 0:
            n[rng.integers(A)] = 1
        f = oracle.normalize(n, b)
        assert int(f.sum()) == 1 << b
        assert np.array_equal(f > 0, n > 0)


def test_normalisation_special_cases(oracle):
    # one observed symbol takes the whole range and costs zero bits
    f = oracle.normalize([0, 0, 7, 0], 11)
    assert f.tolist() == [0, 0, 2048, 0]
    assert oracle.code_length([0, 0, 7, 0], f, 11) == 0.0
    # exactly M observed symbols each get frequency 1
    f = oracle.normalize(np.arange(1, 513), 9)
    assert np.all(f == 1)
    # proportional counts are reproduced exactly
    f = oracle.normalize([1, 2, 1, 4], 11)
    assert f.tolist() == [256, 512, 256, 1024]
    # more observed symbols than slots is refused
    from oracle.oracle import OracleError
    with pytest.raises(OracleError):
        oracle.normalize(np.ones(513), 9)


def test_code_length_gibbs_bound(oracle):
    """C_CE is at least the empirical entropy cost and approaches it as b grows."""
    rng = np.random.default_rng(3)
    n = np.round(5e5 * np.exp(-0.5 * (np.arange(-40, 41) / 6.0) ** 2)).astype(np.uint64)
    N = float(n.sum())
    p = n[n > 0] / N
    h = -(n[n > 0] * np.log2(p)).sum()
    prev = None
    for b in range(9, 16):
        c = oracle.code_length(n, oracle.normalize(n, b), b)
        assert c >= h - 1e-6
        if prev is not None:
            assert c <= prev + 1e-6
        prev = c
    assert prev / h - 1 < 2e-4


def test_conditioning_gain_identity(oracle):
    """Pooled minus coset-conditioned cost equals sum_i I(a_i; c) [eq. conditioning_gain],
    measured on the oracle's own field map and model, with near-exact probabilities (b=15)."""
    rng = np.random.default_rng(9)
    y = rng.standard_normal((60000, 8)) * 1.7
    tp, c = oracle.nearest_e8(y)
    f9 = oracle.fields(tp)
    b = 15

    def cost(vals):
        lo = vals.min()
        n = np.bincount(vals - lo).astype(np.uint64)
        return oracle.code_length(n, oracle.normalize(n, b), b)

    pooled = cost(f9[:, 0]) + sum(cost(f9[:, i]) for i in range(1, 9))
    cond = cost(f9[:, 0]) + sum(cost(f9[f9[:, 0] == cc, i]) for i in range(1, 9) for cc in (0, 1))

    def H(vals):
        _, n = np.unique(vals, return_counts=True)
        p = n / n.sum()
        return -(p * np.log2(p)).sum()

    mi = 0.0
    for i in range(1, 9):
        joint = f9[:, i].astype(np.int64) * 2 + f9[:, 0]
        mi += H(f9[:, i]) + H(f9[:, 0]) - H(joint)
    gain_bits_per_vec = (pooled - cond) / f9.shape[0]
    assert mi > 0.05
    assert abs(gain_bits_per_vec - mi) < 2e-3 * 9


def _golden_tile_table():
    import os
    rows = []
    path = os.path.join(os.path.dirname(__file__), "golden", "tile_overhead.txt")
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            t, S, V, tiles, b, meta, pct = line.split()
            rows.append((int(S), int(V), int(tiles), int(meta)))
    return rows


TILE_TABLE = _golden_tile_table()


@pytest.mark.parametrize("S,V_paper,tiles,meta_bytes", TILE_TABLE)
def test_tile_metadata_matches_paper_table(oracle, S, V_paper, tiles, meta_bytes):
    """Encode a 10240 x 3840 tensor (constant tiny values: cheap to quantise) and read the
    tile-metadata bytes off the blob layout."""
    R, Cc = 10240, 3840
    V = max(32, S // 9)
    assert V == V_paper
    w = np.full((R, Cc), 0.01, dtype=np.float32)
    w[:, ::2] = -0.01
    blob, st = oracle.encode(w, 4.0, tile_vectors=V, search_steps=1)
    h = oracle.header(blob)
    assert h["n_tiles"] == tiles
    payload = (2 * h["payload_words"] + 3) // 4 * 4
    scales = 4 * R
    meta = h["total_bytes"] - 48 - h["table_bytes"] - scales - payload
    assert meta == meta_bytes


def test_estimate_payload_window(oracle):
    """Actual payload bits lie in (C_CE - 16 J n_tile, C_CE]: a tile's states absorb at most
    16 bits each, and rANS with exact frequencies costs at most the model length plus rounding."""
    w = W.single_linear()
    blob, st = oracle.encode(w, 4.0, prob_bits=12)
    J, nt = 32, st["n_tiles"]
    assert st["cce_full"] - 16 * J * nt < st["payload_bits"] <= st["cce_full"] * 1.002
    # information retained per state is log2(x/2^15), 8 bits on average
    assert 7.0 < st["mean_state_bits"] < 9.0


def test_estimate_matches_encoded_size(oracle):
    """With the default credit of 8 bits per state the estimate of the full tensor's fields
    predicts the encoded size within a fraction of a percent."""
    w = W.attention_projection()[:1024]
    blob, st = oracle.encode(w, 3.0)
    tp, _, _ = oracle.quantize(w, st["scale"])
    f9 = oracle.fields(tp.reshape(-1, 8))
    cce, est_bits, tb = oracle.estimate(f9, 1024, int(st["b"]), 512, 8.0, 0)
    assert abs(cce - st["cce_full"]) < 1e-6 * cce
    assert abs(est_bits / (8 * st["bytes"]) - 1) < 5e-3
    assert tb == st["table_bytes"]
