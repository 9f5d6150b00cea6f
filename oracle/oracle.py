"""ctypes binding of the EntroPack CPU oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg load this
module.  ``build()`` compiles ``oracle.c`` with gcc into ``liboracle.so`` next
to it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
# ORACLE_LIB names another build of the same source (the sanitizer run of the CPU pins)
LIB = os.environ.get("ORACLE_LIB") or os.path.join(HERE, "liboracle.so")

BF16, FP16, FP32, FP8, INT8, FP8E5, UINT8, COORD2 = 1, 2, 3, 4, 5, 6, 7, 100
CONT_DIRECT, CONT_FP8, CONT_INT8, CONT_FP8E5, CONT_UINT8 = 0, 1, 2, 3, 4
OK, ERR_ARG, ERR_FORMAT, ERR_UNSUPPORTED, ERR_NOMEM, ERR_CORRUPT = 0, -1, -2, -3, -4, -6

STATS = ["scale", "b", "rhat_sub", "r_stored", "bytes", "payload_bits", "cce_full", "n_tiles",
         "max_A", "erel_coded", "erel_orig", "mean_state_bits", "table_bytes", "sample_rows",
         "escalations", "coarsenings", "rdo_rows_moved", "rdo_budget_bytes", "rdo_lambda"]

OUT_ITEMSIZE = {BF16: 2, FP16: 2, FP32: 4, FP8: 1, INT8: 1, FP8E5: 1, UINT8: 1, COORD2: 4}
OUT_NPTYPE = {BF16: np.uint16, FP16: np.uint16, FP32: np.float32, FP8: np.uint8, INT8: np.int8, FP8E5: np.uint8, UINT8: np.uint8,
              COORD2: np.int32}


class Params(C.Structure):
    _fields_ = [("target_bpp", C.c_double), ("tile_vectors", C.c_int32),
                ("prob_bits", C.c_int32), ("search_steps", C.c_int32),
                ("container", C.c_int32), ("scale_lo", C.c_double), ("scale_hi", C.c_double),
                ("sample_vectors", C.c_int64), ("state_credit_bits", C.c_double),
                ("rdo_candidates", C.c_int32), ("rdo_sweeps", C.c_int32)]


def params(target_bpp, tile_vectors=512, prob_bits=0, search_steps=12, container=0,
           scale_lo=1e-3, scale_hi=8.0, sample_vectors=1 << 18, state_credit_bits=8.0,
           rdo_candidates=0, rdo_sweeps=0):
    return Params(float(target_bpp), int(tile_vectors), int(prob_bits), int(search_steps),
                  int(container), float(scale_lo), float(scale_hi), int(sample_vectors),
                  float(state_credit_bits), int(rdo_candidates), int(rdo_sweeps))


def build(force: bool = True) -> str:
    if os.environ.get("ORACLE_LIB"):
        return LIB
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-shared", "-fPIC", SRC,
                               "-lm", "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = C.CDLL(LIB)
        p, i64, i32, dbl = C.c_void_p, C.c_int64, C.c_int32, C.c_double
        L.ora_encode.argtypes = [p, C.c_int, i64, i64, C.POINTER(Params),
                                 C.POINTER(C.POINTER(C.c_uint8)), C.POINTER(C.c_uint64), p]
        L.ora_decode.argtypes = [p, C.c_uint64, C.c_int, p, p, C.c_uint32, C.c_uint32]
        L.ora_blob_free.argtypes = [p]
        L.ora_blob_header.argtypes = [p, C.c_uint64, p]
        L.ora_nearest_d8.argtypes = [p, i64, p]
        L.ora_nearest_e8.argtypes = [p, i64, p, p]
        L.ora_fields.argtypes = [p, i64, p]
        L.ora_points.argtypes = [p, i64, p]
        L.ora_normalize.argtypes = [p, i32, i32, p]
        L.ora_code_length.argtypes = [p, p, i32, i32]
        L.ora_code_length.restype = dbl
        L.ora_rans_words.argtypes = [p, i64, i32, i32, p, p, p, p, p]
        L.ora_snap.argtypes = [p, i64, C.c_int, p]
        L.ora_values.argtypes = [p, i64, C.c_int, p]
        L.ora_quantize.argtypes = [p, C.c_int, i64, i64, C.c_int, dbl, p, p, p]
        L.ora_sample_rows.argtypes = [i64, i64, i64, p]
        L.ora_rdo_ratios.argtypes = [C.c_int, p]
        L.ora_sample_rows.restype = i64
        L.ora_estimate.argtypes = [p, i64, i64, i32, i32, dbl, i32, p]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, code, what):
        super().__init__(f"{what} failed with status {code}")
        self.code = code


def _chk(rc, what):
    if rc != OK:
        raise OracleError(rc, what)


def _ptr(a):
    return a.ctypes.data_as(C.c_void_p)


def _dtype_code(w: np.ndarray, dtype):
    if dtype is not None:
        return dtype
    if w.dtype == np.float32:
        return FP32
    if w.dtype == np.uint16:
        return BF16
    raise ValueError("pass dtype for uint16 FP16 bits")


def encode(w: np.ndarray, target_bpp: float, dtype=None, **kw):
    """Encode an R x C weight matrix (uint16 BF16/FP16 bits or float32).
    Returns (blob bytes as np.uint8 array, stats dict)."""
    w = np.ascontiguousarray(w)
    R, Cc = w.shape
    prm = params(target_bpp, **kw)
    out = C.POINTER(C.c_uint8)()
    n = C.c_uint64(0)
    st = np.zeros(32, dtype=np.float64)
    rc = lib().ora_encode(_ptr(w), _dtype_code(w, dtype), R, Cc, C.byref(prm), C.byref(out),
                          C.byref(n), _ptr(st))
    _chk(rc, "ora_encode")
    blob = np.ctypeslib.as_array(out, shape=(n.value,)).copy()
    lib().ora_blob_free(C.cast(out, C.c_void_p))
    return blob, {k: float(st[i]) for i, k in enumerate(STATS)}


def header(blob: np.ndarray) -> dict:
    h = np.zeros(9, dtype=np.uint64)
    _chk(lib().ora_blob_header(_ptr(blob), blob.size, _ptr(h)), "ora_blob_header")
    keys = ["rows", "cols", "b", "V", "n_tiles", "container", "table_bytes", "payload_words",
            "total_bytes"]
    return {k: int(v) for k, v in zip(keys, h)}


def decode(blob: np.ndarray, out_dtype: int, t0: int = 0, t1=None, out=None, dequant=None):
    """Decode tiles [t0, t1) into a full R x C output; returns (out, dequant)."""
    h = header(blob)
    if t1 is None:
        t1 = h["n_tiles"]
    if out is None:
        out = np.zeros((h["rows"], h["cols"]), dtype=OUT_NPTYPE[out_dtype])
    if dequant is None and h["container"]:
        dequant = np.zeros(h["rows"], dtype=np.float32)
    rc = lib().ora_decode(_ptr(blob), blob.size, out_dtype, _ptr(out),
                          _ptr(dequant) if dequant is not None else None, t0, t1)
    _chk(rc, "ora_decode")
    return out, dequant


def decode_status(blob: np.ndarray, out_dtype: int = COORD2) -> int:
    """Status code of a full decode (for corruption tests)."""
    try:
        h = header(blob)
    except OracleError as e:
        return e.code
    out = np.zeros((h["rows"], h["cols"]), dtype=OUT_NPTYPE[out_dtype])
    dq = np.zeros(h["rows"], dtype=np.float32)
    return lib().ora_decode(_ptr(blob), blob.size, out_dtype, _ptr(out), _ptr(dq), 0,
                            h["n_tiles"])


def nearest_d8(y: np.ndarray) -> np.ndarray:
    y = np.ascontiguousarray(y, dtype=np.float64).reshape(-1, 8)
    z = np.zeros(y.shape, dtype=np.int32)
    _chk(lib().ora_nearest_d8(_ptr(y), y.shape[0], _ptr(z)), "ora_nearest_d8")
    return z


def nearest_e8(y: np.ndarray):
    """Returns (2p as int32 [n, 8], coset int32 [n])."""
    y = np.ascontiguousarray(y, dtype=np.float64).reshape(-1, 8)
    tp = np.zeros(y.shape, dtype=np.int32)
    c = np.zeros(y.shape[0], dtype=np.int32)
    _chk(lib().ora_nearest_e8(_ptr(y), y.shape[0], _ptr(tp), _ptr(c)), "ora_nearest_e8")
    return tp, c


def fields(two_p: np.ndarray) -> np.ndarray:
    tp = np.ascontiguousarray(two_p, dtype=np.int32).reshape(-1, 8)
    f = np.zeros((tp.shape[0], 9), dtype=np.int32)
    _chk(lib().ora_fields(_ptr(tp), tp.shape[0], _ptr(f)), "ora_fields")
    return f


def points(f9: np.ndarray) -> np.ndarray:
    f = np.ascontiguousarray(f9, dtype=np.int32).reshape(-1, 9)
    tp = np.zeros((f.shape[0], 8), dtype=np.int32)
    _chk(lib().ora_points(_ptr(f), f.shape[0], _ptr(tp)), "ora_points")
    return tp


def normalize(counts, b: int) -> np.ndarray:
    n = np.ascontiguousarray(counts, dtype=np.uint64)
    f = np.zeros(n.size, dtype=np.uint32)
    _chk(lib().ora_normalize(_ptr(n), n.size, b, _ptr(f)), "ora_normalize")
    return f


def code_length(counts, freqs, b: int) -> float:
    n = np.ascontiguousarray(counts, dtype=np.uint64)
    f = np.ascontiguousarray(freqs, dtype=np.uint32)
    return float(lib().ora_code_length(_ptr(n), _ptr(f), n.size, b))


def snap(y, dtype: int) -> np.ndarray:
    y = np.ascontiguousarray(y, dtype=np.float64)
    out = np.zeros(y.shape, dtype=OUT_NPTYPE[dtype])
    _chk(lib().ora_snap(_ptr(y), y.size, dtype, _ptr(out)), "ora_snap")
    return out


def values(bits: np.ndarray, dtype: int) -> np.ndarray:
    b = np.ascontiguousarray(bits)
    out = np.zeros(b.shape, dtype=np.float64)
    _chk(lib().ora_values(_ptr(b), b.size, dtype, _ptr(out)), "ora_values")
    return out


def quantize(w: np.ndarray, s: float, container: int = 0, dtype=None):
    """Returns (2p int32 R x C, coded values float32 R x C, mu float64 R)."""
    w = np.ascontiguousarray(w)
    R, Cc = w.shape
    tp = np.zeros((R, Cc), dtype=np.int32)
    xv = np.zeros((R, Cc), dtype=np.float32)
    mu = np.zeros(R, dtype=np.float64)
    _chk(lib().ora_quantize(_ptr(w), _dtype_code(w, dtype), R, Cc, container, float(s), _ptr(tp),
                            _ptr(xv), _ptr(mu)), "ora_quantize")
    return tp, xv, mu


def rdo_ratios(K: int) -> np.ndarray:
    """Candidate scale ratios of the per-row refinement (Section 3.5), in candidate order."""
    out = np.zeros(K, dtype=np.float64)
    _chk(lib().ora_rdo_ratios(K, _ptr(out)), "ora_rdo_ratios")
    return out


def sample_rows(R: int, Cc: int, sample_vectors: int = 1 << 18) -> np.ndarray:
    rows = np.zeros(R, dtype=np.int64)
    k = lib().ora_sample_rows(R, Cc, sample_vectors, _ptr(rows))
    if k < 0:
        raise OracleError(k, "ora_sample_rows")
    return rows[:k].copy()


def estimate(f9: np.ndarray, rows: int, b: int, V: int = 512, kappa: float = 16.0,
             container: int = 0):
    """(C_CE bits, estimated stored bits, table bytes) of a field set."""
    f = np.ascontiguousarray(f9, dtype=np.int32).reshape(-1, 9)
    out = np.zeros(3, dtype=np.float64)
    _chk(lib().ora_estimate(_ptr(f), f.shape[0], rows, b, V, kappa, container, _ptr(out)),
         "ora_estimate")
    return float(out[0]), float(out[1]), float(out[2])


def gemm_i8_nt(a: np.ndarray, b: np.ndarray, rows=None) -> np.ndarray:
    """Exact int32 Y = A B^T (int8 A[m,k], B[n,k]); only `rows` of Y if given."""
    a = np.ascontiguousarray(a, dtype=np.int8)
    b = np.ascontiguousarray(b, dtype=np.int8)
    m, k = a.shape
    n = b.shape[0]
    assert b.shape[1] == k
    L = lib()
    L.ora_gemm_i8_nt.restype = C.c_int
    L.ora_gemm_i8_nt.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_int64,
                                 C.c_int64, C.c_void_p, C.c_int64]
    if rows is None:
        y = np.zeros((m, n), dtype=np.int32)
        rc = L.ora_gemm_i8_nt(_ptr(a), _ptr(b), _ptr(y), m, n, k, None, 0)
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        y = np.zeros((r.size, n), dtype=np.int32)
        rc = L.ora_gemm_i8_nt(_ptr(a), _ptr(b), _ptr(y), m, n, k, _ptr(r), r.size)
    _chk(rc, "gemm_i8_nt")
    return y


def _table(values: np.ndarray, b: int):
    """One table built from `values` (Section 3.3): (min, A, counts over [min, max],
    frequencies normalised to 2^b, or None when the range exceeds 2^b)."""
    if values.size == 0:
        return 0, 0, np.zeros(0, np.uint64), np.zeros(0, np.uint32)
    lo, hi = int(values.min()), int(values.max())
    counts = np.bincount(values - lo, minlength=hi - lo + 1).astype(np.uint64)
    if counts.size > (1 << b):
        return lo, counts.size, counts, None
    return lo, counts.size, counts, normalize(counts, b)


def rans_words(f9: np.ndarray, V: int, b: int, tmin, tA, freqs) -> int:
    """Payload words of the tiled interleaved rANS coding of the fields f9 (nvec x 9) with
    17 tables (Section 3.6): table 0 for the coset, 1 + 8 c + (i - 1) for field i under
    coset c, covering tA[t] values from tmin[t] with normalised frequencies freqs[t]."""
    f = np.ascontiguousarray(f9, dtype=np.int32)
    lo = np.ascontiguousarray(tmin, dtype=np.int32)
    A = np.ascontiguousarray(tA, dtype=np.int32)
    fr = np.concatenate([np.asarray(x, dtype=np.uint32) for x in freqs] + [np.zeros(1, np.uint32)])
    words = np.zeros(1, dtype=np.uint64)
    _chk(lib().ora_rans_words(_ptr(f), f.shape[0], V, b, _ptr(lo), _ptr(A), _ptr(fr),
                              _ptr(words), None), "ora_rans_words")
    return int(words[0])


def coding_ablation(blob: np.ndarray) -> dict:
    """Stored size of a blob's own lattice points re-encoded under the three coding models of
    the entropy-model ablation (App. A.3, Table coding; eqs. cond, parity, conditioning_gain):
      'entropack': coset table + one table per (field, coset), fields (c, z1..z7, m);
      'pooled':    coset table + one table per field for both cosets (no conditioning);
      'direct_z8': as 'entropack' with z8 = 2m + pi coded in place of m (no parity reduction).
    Every variant keeps the points, row scales, tiles and precision b, builds its tables from
    its own fields (counts normalised to 2^b), and re-runs the tiled rANS encoder on its
    symbols.  Its stored size is the blob layout's (header, serialized tables, scales, states,
    offsets, payload) with its own tables and payload; the pooled model stores 9 tables, the
    others 17.  code_bits is each model's ideal code length C_CE under its tables (eq. length)."""
    h = header(blob)
    b, V, R = h["b"], h["V"], h["rows"]
    two_p, _ = decode(blob, COORD2)
    f9 = fields(two_p)
    c = f9[:, 0]
    z8 = (two_p.reshape(-1, 8)[:, 7] - c) // 2
    n = h["rows"] * h["cols"]
    fixed = (48 + 4 * R + (4 * R if h["container"] else 0) + 128 * h["n_tiles"]
             + 4 * (h["n_tiles"] + 1))
    cn = np.array([(c == 0).sum(), (c == 1).sum()], dtype=np.uint64)
    cf = normalize(cn, b)
    res = {"b": b, "weights": n, "stored_bits": {}, "code_bits": {}, "payload_words": {}}
    for name in ("entropack", "pooled", "direct_z8"):
        g = f9.copy()
        if name == "direct_z8":
            g[:, 8] = z8
        tmin, tA = [0] * 17, [0] * 17
        freqs = [np.zeros(0, np.uint32)] * 17
        tA[0], freqs[0] = 2, cf
        bits = code_length(cn, cf, b)
        tbytes = 4                                  # the coset pair f0, f1
        for i in range(1, 9):
            parts = [(None, g[:, i])] if name == "pooled" else [(k, g[c == k, i]) for k in (0, 1)]
            for k, vals in parts:
                lo, A, cnt, fr = _table(vals, b)
                if fr is None:
                    raise ValueError(f"{name}: field {i} spans {A} values, more than 2^{b}")
                if cnt.size:
                    bits += code_length(cnt, fr, b)
                tbytes += 8 + (2 * A + 3) // 4 * 4
                for kk in ((0, 1) if k is None else (k,)):
                    t = 1 + 8 * kk + (i - 1)
                    tmin[t], tA[t], freqs[t] = lo, A, fr
        words = rans_words(g, V, b, tmin, tA, freqs)
        stored = 8.0 * (fixed + tbytes + (2 * words + 3) // 4 * 4)
        res["stored_bits"][name] = stored
        res["code_bits"][name] = bits
        res["payload_words"][name] = words
        res[name + "_bpp"] = stored / n
    return res
