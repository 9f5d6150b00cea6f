"""Python binding of libentropack.so (argument marshalling only).

Every step of encoding runs in the library's C++ encoder and every step of
decoding runs in its HIP kernels; this module converts numpy arrays and torch
device tensors to pointers and back.  PyTorch is used only for device memory
and streams.  The library must be built first (``__graft_entry__.build()``);
if it is missing, loading raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os
import weakref

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libentropack.so")

# ---- constants (mirror include/entropack.h) -------------------------------------
OK, ERR_ARG, ERR_FORMAT, ERR_UNSUPPORTED, ERR_NOMEM, ERR_HIP, ERR_CORRUPT = 0, -1, -2, -3, -4, -5, -6
BF16, FP16, FP32, FP8_E4M3, INT8, FP8_E5M2, UINT8, COORD2_I32 = 1, 2, 3, 4, 5, 6, 7, 100
CONT_DIRECT, CONT_FP8_ROW, CONT_INT8_ROW, CONT_FP8E5M2_ROW, CONT_UINT8_TENSOR = 0, 1, 2, 3, 4
STATUS_PAYLOAD_OVERRUN, STATUS_BAD_FINAL_STATE, STATUS_BAD_END_OFFSET = 1, 2, 4

ITEMSIZE = {BF16: 2, FP16: 2, FP32: 4, FP8_E4M3: 1, INT8: 1, FP8_E5M2: 1, UINT8: 1, COORD2_I32: 4}


class EncodeParams(C.Structure):
    _fields_ = [("target_bpp", C.c_double), ("tile_vectors", C.c_int32),
                ("prob_bits", C.c_int32), ("search_steps", C.c_int32),
                ("container", C.c_int32), ("scale_lo", C.c_double), ("scale_hi", C.c_double),
                ("sample_vectors", C.c_int64), ("state_credit_bits", C.c_double),
                ("nthreads", C.c_int32), ("rdo_candidates", C.c_int32),
                ("rdo_sweeps", C.c_int32), ("reserved", C.c_int32)]


class EncodeStats(C.Structure):
    _fields_ = [("scale", C.c_double), ("rate_estimate_sample", C.c_double),
                ("rate_stored", C.c_double), ("code_length_bits", C.c_double),
                ("erel_coded", C.c_double), ("erel_original", C.c_double),
                ("mean_state_bits", C.c_double), ("bytes", C.c_uint64),
                ("payload_bits", C.c_uint64), ("prob_bits", C.c_uint32),
                ("n_tiles", C.c_uint32), ("max_alphabet", C.c_uint32),
                ("sample_rows", C.c_uint32), ("escalations", C.c_uint32),
                ("coarsenings", C.c_uint32), ("rdo_rows_moved", C.c_uint32),
                ("reserved", C.c_uint32)]


class Blob(C.Structure):
    _fields_ = [("data", C.POINTER(C.c_uint8)), ("size", C.c_uint64)]


class TensorInfo(C.Structure):
    _fields_ = [("rows", C.c_uint32), ("cols", C.c_uint32), ("prob_bits", C.c_uint32),
                ("tile_vectors", C.c_uint32), ("n_tiles", C.c_uint32),
                ("container", C.c_uint32), ("table_bytes", C.c_uint32),
                ("payload_words", C.c_uint32), ("total_bytes", C.c_uint64),
                ("off_tables", C.c_uint64), ("off_sigma", C.c_uint64),
                ("off_delta", C.c_uint64), ("off_states", C.c_uint64),
                ("off_offsets", C.c_uint64), ("off_payload", C.c_uint64),
                ("max_alphabet", C.c_uint32), ("coord2_min", C.c_int32),
                ("coord2_max", C.c_int32), ("max_abs_weight", C.c_float),
                ("path", C.c_uint32), ("sum_alphabet", C.c_uint32),
                ("table_off", C.c_uint32 * 16), ("table_min", C.c_int32 * 16),
                ("table_A", C.c_uint32 * 16), ("coset_f0", C.c_uint32),
                ("coset_f1", C.c_uint32)]


class Layer(C.Structure):
    _fields_ = [("info", TensorInfo), ("d_blob", C.c_void_p), ("d_out", C.c_void_p),
                ("d_dequant", C.c_void_p), ("out_dtype", C.c_int32), ("reserved", C.c_int32)]


class Stack(C.Structure):
    _fields_ = [("d_workspace", C.c_void_p), ("n_layers", C.c_int32), ("path", C.c_uint32),
                ("total_tasks", C.c_uint32), ("lds_bytes", C.c_uint32),
                ("reserved", C.c_uint32 * 4)]


class EntroPackError(RuntimeError):
    def __init__(self, code: int, what: str, msg: str):
        super().__init__(f"{what}: status {code}: {msg}")
        self.code = code


_lib = None


def lib():
    """The loaded native library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        vp, u32, i32, i64, u64 = C.c_void_p, C.c_uint32, C.c_int32, C.c_int64, C.c_uint64
        L.ep_encode_params_default.argtypes = [C.POINTER(EncodeParams)]
        L.ep_encode_params_default.restype = None
        L.ep_encode_cpu.argtypes = [vp, C.c_int, i64, i64, C.POINTER(EncodeParams),
                                    C.POINTER(Blob), C.POINTER(EncodeStats)]
        L.ep_encode_gpu.argtypes = [vp, C.c_int, i64, i64, C.POINTER(EncodeParams),
                                    C.POINTER(Blob), C.POINTER(EncodeStats), vp]
        L.ep_blob_free.argtypes = [C.POINTER(Blob)]
        L.ep_blob_free.restype = None
        L.ep_blob_info.argtypes = [vp, u64, C.POINTER(TensorInfo)]
        L.ep_decode_tiles.argtypes = [C.POINTER(TensorInfo), vp, C.c_int, vp, vp, u32, u32, vp, vp]
        L.ep_decode_layers_workspace.argtypes = [C.c_int]
        L.ep_decode_layers_workspace.restype = u64
        L.ep_decode_layers.argtypes = [C.POINTER(Layer), C.c_int, vp, u64, vp, vp]
        L.ep_decode_layers_noalloc.argtypes = [C.POINTER(Layer), C.c_int, vp, vp]
        L.ep_stack_workspace.argtypes = [C.c_int]
        L.ep_stack_workspace.restype = u64
        L.ep_stack_prepare.argtypes = [C.POINTER(Layer), C.c_int, vp, u64, C.POINTER(Stack), vp]
        L.ep_stack_decode.argtypes = [C.POINTER(Stack), vp, vp]
        L.ep_gemm_i8_nt.argtypes = [vp, vp, vp, i64, i64, i64, vp]
        L.ep_decode_matmul_i8.argtypes = [C.POINTER(TensorInfo), vp, vp, C.c_int, vp, vp, vp, vp]
        L.ep_decode_gemm_i8.argtypes = [C.POINTER(TensorInfo), vp, vp, i64, vp, vp, vp, u64, vp, vp]
        L.ep_decode_gemm_i8_prepared.argtypes = [C.POINTER(TensorInfo), vp, vp, i64, vp, vp, vp, u64,
                                                 vp, vp]
        L.ep_decode_gemm_i8_prepare.argtypes = [C.POINTER(TensorInfo), vp, vp, u64, vp]
        L.ep_decode_gemm_bf16.argtypes = [C.POINTER(TensorInfo), vp, vp, i64, vp, vp, vp, u64, vp, vp]
        L.ep_decode_gemm_bf16_prepared.argtypes = [C.POINTER(TensorInfo), vp, vp, i64, vp, vp, vp, u64,
                                                   vp, vp]
        L.ep_decode_gemm_bf16_prepare.argtypes = [C.POINTER(TensorInfo), vp, vp, u64, vp]
        L.ep_decode_gemm_bf16_workspace.argtypes = [C.POINTER(TensorInfo)]
        L.ep_decode_gemm_bf16_workspace.restype = u64
        L.ep_decode_gemm_i8_workspace.argtypes = [C.POINTER(TensorInfo)]
        L.ep_decode_gemm_i8_workspace.restype = u64
        L.ep_last_error.restype = C.c_char_p
        _lib = L
    return _lib


EXPORTS = ["ep_encode_params_default", "ep_encode_cpu", "ep_encode_gpu", "ep_blob_free", "ep_blob_info",
           "ep_decode_tiles", "ep_decode_layers_workspace", "ep_decode_layers",
           "ep_decode_layers_noalloc",
           "ep_stack_workspace", "ep_stack_prepare", "ep_stack_decode", "ep_gemm_i8_nt",
           "ep_decode_matmul_i8", "ep_decode_gemm_i8", "ep_decode_gemm_i8_workspace",
           "ep_decode_gemm_i8_prepare", "ep_decode_gemm_i8_prepared",
           "ep_decode_gemm_bf16", "ep_decode_gemm_bf16_workspace", "ep_decode_gemm_bf16_prepare",
           "ep_decode_gemm_bf16_prepared",
           "ep_last_error"]


def _check(rc: int, what: str):
    if rc != OK:
        raise EntroPackError(rc, what, lib().ep_last_error().decode())


def default_params(target_bpp: float, **kw) -> EncodeParams:
    p = EncodeParams()
    lib().ep_encode_params_default(C.byref(p))
    p.target_bpp = float(target_bpp)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _blob_array(out: Blob) -> np.ndarray:
    """The blob the library allocated, as a uint8 numpy array over the same memory (no
    copy); ep_blob_free releases it once no array refers to that memory any more."""
    addr = C.cast(out.data, C.c_void_p).value
    buf = (C.c_uint8 * out.size).from_address(addr)
    weakref.finalize(buf, _free_blob, addr, out.size)
    return np.frombuffer(buf, dtype=np.uint8)


def _free_blob(addr: int, size: int) -> None:
    b = Blob(C.cast(addr, C.POINTER(C.c_uint8)), size)
    lib().ep_blob_free(C.byref(b))


def encode(w: np.ndarray, target_bpp: float, dtype: int | None = None, **kw):
    """Encode an R x C matrix (uint16 BF16 bits, or float32; FP16 bits with dtype=FP16).
    Returns (blob as a uint8 numpy array over the library's memory, no copy; stats dict)."""
    w = np.ascontiguousarray(w)
    if dtype is None:
        dtype = FP32 if w.dtype == np.float32 else BF16
    p = default_params(target_bpp, **kw)
    out = Blob()
    st = EncodeStats()
    _check(lib().ep_encode_cpu(w.ctypes.data_as(C.c_void_p), dtype, w.shape[0], w.shape[1],
                               C.byref(p), C.byref(out), C.byref(st)), "ep_encode_cpu")
    return _blob_array(out), {k: getattr(st, k) for k, _ in EncodeStats._fields_}


def encode_gpu(d_w: int, rows: int, cols: int, target_bpp: float, dtype: int = BF16,
               stream: int = 0, **kw):
    """Encode an R x C device matrix (pointer d_w: BF16/FP16 bits or FP32) with the GPU
    encoder.  Returns (blob as a uint8 numpy array, stats dict), as encode()."""
    p = default_params(target_bpp, **kw)
    out = Blob()
    st = EncodeStats()
    _check(lib().ep_encode_gpu(d_w, dtype, rows, cols, C.byref(p), C.byref(out), C.byref(st),
                               stream or None), "ep_encode_gpu")
    return _blob_array(out), {k: getattr(st, k) for k, _ in EncodeStats._fields_}


def blob_info(blob: np.ndarray) -> TensorInfo:
    info = TensorInfo()
    b = np.ascontiguousarray(blob, dtype=np.uint8)
    _check(lib().ep_blob_info(b.ctypes.data_as(C.c_void_p), b.size, C.byref(info)), "ep_blob_info")
    return info


def decode_tiles(info: TensorInfo, d_blob: int, out_dtype: int, d_out: int, d_dequant: int = 0,
                 tile_begin: int = 0, tile_end: int | None = None, d_status: int = 0,
                 stream: int = 0):
    """Raw entry point: all buffers are device addresses (ints)."""
    if tile_end is None:
        tile_end = info.n_tiles
    _check(lib().ep_decode_tiles(C.byref(info), d_blob, out_dtype, d_out, d_dequant or None,
                                 tile_begin, tile_end, d_status or None, stream or None),
           "ep_decode_tiles")


def decode_layers_workspace(n: int) -> int:
    return int(lib().ep_decode_layers_workspace(n))


def _layer_array(layers):
    arr = (Layer * len(layers))()
    for i, (info, blob, out, dq, dt) in enumerate(layers):
        arr[i].info = info
        arr[i].d_blob = blob
        arr[i].d_out = out
        arr[i].d_dequant = dq or None
        arr[i].out_dtype = dt
    return arr


def decode_layers(layers, d_ws: int, ws_bytes: int, d_status: int = 0, stream: int = 0):
    """layers: sequence of (TensorInfo, d_blob, d_out, d_dequant, out_dtype)."""
    arr = _layer_array(layers)
    _check(lib().ep_decode_layers(arr, len(layers), d_ws, ws_bytes, d_status or None,
                                  stream or None), "ep_decode_layers")


def decode_layers_noalloc(layers, d_status: int = 0, stream: int = 0):
    """As decode_layers, with the descriptors in the library's static device array (no
    workspace, no allocation; at most 512 layers)."""
    arr = _layer_array(layers)
    _check(lib().ep_decode_layers_noalloc(arr, len(layers), d_status or None, stream or None),
           "ep_decode_layers_noalloc")


def stack_workspace(n: int) -> int:
    return int(lib().ep_stack_workspace(n))


def stack_prepare(layers, d_ws: int, ws_bytes: int, stream: int = 0) -> Stack:
    """Write the device descriptors of `layers` once; returns the prepared stack."""
    st = Stack()
    arr = _layer_array(layers)
    _check(lib().ep_stack_prepare(arr, len(layers), d_ws, ws_bytes, C.byref(st), stream or None),
           "ep_stack_prepare")
    return st


def stack_decode(st: Stack, d_status: int = 0, stream: int = 0):
    _check(lib().ep_stack_decode(C.byref(st), d_status or None, stream or None), "ep_stack_decode")


def gemm_i8_nt(d_a: int, d_b: int, d_y: int, m: int, n: int, k: int, stream: int = 0):
    _check(lib().ep_gemm_i8_nt(d_a, d_b, d_y, m, n, k, stream or None), "ep_gemm_i8_nt")


def decode_matmul_i8(info: TensorInfo, d_blob: int, d_x: int, m: int, d_y: int, d_dequant: int = 0,
                     d_status: int = 0, stream: int = 0):
    """Y (m x R int32) = X (m x C int8) times the decoded INT8 container matrix, transposed."""
    _check(lib().ep_decode_matmul_i8(C.byref(info), d_blob, d_x, m, d_y, d_dequant or None,
                                     d_status or None, stream or None), "ep_decode_matmul_i8")


def decode_gemm_i8_workspace(info: TensorInfo) -> int:
    return int(lib().ep_decode_gemm_i8_workspace(C.byref(info)))


def decode_gemm_i8(info: TensorInfo, d_blob: int, d_x: int, m: int, d_y: int, d_ws: int,
                   ws_bytes: int, d_dequant: int = 0, d_status: int = 0, stream: int = 0):
    """Y (m x R int32) = X (m x C int8) times the decoded INT8 container matrix, transposed,
    on the matrix cores, for any m (the fused decode and MFMA product)."""
    _check(lib().ep_decode_gemm_i8(C.byref(info), d_blob, d_x, m, d_y, d_dequant or None, d_ws,
                                   ws_bytes, d_status or None, stream or None), "ep_decode_gemm_i8")


def decode_gemm_i8_prepare(info: TensorInfo, d_blob: int, d_ws: int, ws_bytes: int, stream: int = 0):
    """Build the tensor's decode tables once into the workspace (synchronous)."""
    _check(lib().ep_decode_gemm_i8_prepare(C.byref(info), d_blob, d_ws, ws_bytes, stream or None),
           "ep_decode_gemm_i8_prepare")


def decode_gemm_i8_prepared(info: TensorInfo, d_blob: int, d_x: int, m: int, d_y: int, d_ws: int,
                            ws_bytes: int, d_dequant: int = 0, d_status: int = 0, stream: int = 0):
    """decode_gemm_i8 on a workspace that decode_gemm_i8_prepare filled for this blob."""
    _check(lib().ep_decode_gemm_i8_prepared(C.byref(info), d_blob, d_x, m, d_y, d_dequant or None,
                                            d_ws, ws_bytes, d_status or None, stream or None),
           "ep_decode_gemm_i8_prepared")


def decode_gemm_bf16_workspace(info: TensorInfo) -> int:
    return int(lib().ep_decode_gemm_bf16_workspace(C.byref(info)))


def decode_gemm_bf16(info: TensorInfo, d_blob: int, d_x: int, m: int, d_y: int, d_ws: int,
                     ws_bytes: int, d_dequant: int = 0, d_status: int = 0, stream: int = 0):
    """Y (m x R fp32) = X (m x C bf16) times the tensor's bf16 decode, transposed, on the
    matrix cores, for any m (the fused decode and BF16 MFMA product)."""
    _check(lib().ep_decode_gemm_bf16(C.byref(info), d_blob, d_x, m, d_y, d_dequant or None, d_ws,
                                     ws_bytes, d_status or None, stream or None), "ep_decode_gemm_bf16")


def decode_gemm_bf16_prepare(info: TensorInfo, d_blob: int, d_ws: int, ws_bytes: int, stream: int = 0):
    """Build the tensor's decode tables once into the workspace (synchronous)."""
    _check(lib().ep_decode_gemm_bf16_prepare(C.byref(info), d_blob, d_ws, ws_bytes, stream or None),
           "ep_decode_gemm_bf16_prepare")


def decode_gemm_bf16_prepared(info: TensorInfo, d_blob: int, d_x: int, m: int, d_y: int, d_ws: int,
                              ws_bytes: int, d_dequant: int = 0, d_status: int = 0, stream: int = 0):
    """decode_gemm_bf16 on a workspace that decode_gemm_bf16_prepare filled for this blob."""
    _check(lib().ep_decode_gemm_bf16_prepared(C.byref(info), d_blob, d_x, m, d_y, d_dequant or None,
                                              d_ws, ws_bytes, d_status or None, stream or None),
           "ep_decode_gemm_bf16_prepared")


# ---- torch conveniences (device memory and streams only) ------------------------
def _torch():
    import torch
    return torch


TORCH_DTYPE = {}


def torch_dtype(code: int):
    t = _torch()
    return {BF16: t.bfloat16, FP16: t.float16, FP32: t.float32, FP8_E4M3: t.float8_e4m3fn,
            INT8: t.int8, FP8_E5M2: t.float8_e5m2, UINT8: t.uint8, COORD2_I32: t.int32}[code]


def to_device(blob: np.ndarray, device="cuda"):
    t = _torch()
    return t.from_numpy(np.ascontiguousarray(blob, dtype=np.uint8)).to(device)


def decode(blob: np.ndarray, out_dtype: int, d_blob=None, tile_begin=0, tile_end=None,
           out=None, dequant=None, status=None, info=None):
    """Decode a blob on the current CUDA/HIP device into a new (or given) torch tensor.
    Returns (out, dequant or None, status tensor)."""
    t = _torch()
    info = info or blob_info(blob)
    if d_blob is None:
        d_blob = to_device(blob)
    if out is None:
        out = t.zeros((info.rows, info.cols), dtype=torch_dtype(out_dtype), device=d_blob.device)
    if dequant is None and info.container:
        dequant = t.zeros(info.rows, dtype=t.float32, device=d_blob.device)
    if status is None:
        status = t.zeros(1, dtype=t.int32, device=d_blob.device)
    stream = t.cuda.current_stream(d_blob.device).cuda_stream
    decode_tiles(info, d_blob.data_ptr(), out_dtype, out.data_ptr(),
                 dequant.data_ptr() if dequant is not None else 0, tile_begin, tile_end,
                 status.data_ptr(), stream)
    return out, dequant, status
