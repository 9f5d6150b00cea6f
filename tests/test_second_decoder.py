"""A second, independent decoder of the stored representation, in plain Python.

It re-reads the byte layout and re-implements the rANS decode (Section 3.7,
eq. rans_decode; Appendix C.3) and the field inverse (eq. point_inverse) with
pure-Python loops and a linear symbol search, to guard the C oracle's decoder
against a one-author mistake.  Small inputs only.
"""
import struct

import numpy as np

from paper_2609_34185_amd import workloads as W


def decode_py(blob: bytes):
    (magic, ver, R, C, b, V, n_tiles, cont, tb, n_words) = struct.unpack_from("<10I", blob, 0)
    assert magic == 0x314B5045 and ver == 1
    pos = 48
    f0, f1 = struct.unpack_from("<2H", blob, pos)
    tabs = {0: (0, [f0, f1])}
    pos += 4
    for c in (0, 1):
        for i in range(1, 9):
            mn, A = struct.unpack_from("<iI", blob, pos)
            f = list(struct.unpack_from(f"<{A}H", blob, pos + 8))
            tabs[(i, c)] = (mn, f)
            pos += 8 + (2 * A + 3) // 4 * 4
    assert pos == 48 + tb
    sigma = np.frombuffer(blob, np.float32, R, pos)
    pos += 4 * R + (4 * R if cont else 0)
    states = np.frombuffer(blob, np.uint32, 32 * n_tiles, pos).reshape(n_tiles, 32)
    pos += 128 * n_tiles
    offs = np.frombuffer(blob, np.uint32, n_tiles + 1, pos)
    pos += 4 * (n_tiles + 1)
    words = np.frombuffer(blob, np.uint16, n_words, pos)
    M = 1 << b
    nvec = R * C // 8
    two_p = np.zeros(R * C, dtype=np.int64)
    for t in range(n_tiles):
        v0 = t * V
        nv = min(V, nvec - v0)
        x = [int(s) for s in states[t]]
        ptr = int(offs[t])
        fields = [[0] * 9 for _ in range(32)]
        for step in range(9 * ((nv + 31) // 32)):
            k, i = divmod(step, 9)
            for lane in range(32):
                if lane + 32 * k >= nv:
                    continue
                mn, f = tabs[0] if i == 0 else tabs[(i, fields[lane][0])]
                u = x[lane] % M
                cum = 0
                for sym, fs in enumerate(f):          # linear search of the interval
                    if cum <= u < cum + fs:
                        break
                    cum += fs
                x[lane] = fs * (x[lane] // M) + u - cum
                if x[lane] < 1 << 15:
                    x[lane] = (x[lane] << 16) + int(words[ptr])
                    ptr += 1
                fields[lane][i] = sym + mn
                if i == 8:
                    c = fields[lane][0]
                    z = fields[lane][1:8]
                    pi = sum(z) % 2
                    p2 = [2 * zz + c for zz in z] + [2 * (2 * fields[lane][8] + pi) + c]
                    v = v0 + lane + 32 * k
                    two_p[8 * v: 8 * v + 8] = p2
        assert all(s == 1 << 15 for s in x), "terminal states"
        assert ptr == offs[t + 1], "tile payload boundary"
    return two_p.reshape(R, C), sigma


def test_second_decoder_agrees_with_oracle(oracle):
    w = W.single_linear()[:96]
    blob, st = oracle.encode(w, 4.0, prob_bits=12)
    tp_py, sigma = decode_py(blob.tobytes())
    tp_or, _ = oracle.decode(blob, oracle.COORD2)
    assert np.array_equal(tp_py, tp_or)
    ref, _, _ = oracle.quantize(w, st["scale"])
    assert np.array_equal(tp_py, ref)


def test_second_decoder_ragged_tiles(oracle):
    w = W.ragged_tensor(3, 13, 200)
    blob, st = oracle.encode(w, 5.0, tile_vectors=45)
    tp_py, _ = decode_py(blob.tobytes())
    tp_or, _ = oracle.decode(blob, oracle.COORD2)
    assert np.array_equal(tp_py, tp_or)
