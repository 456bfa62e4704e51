"""Python binding of libq4nx.so (ctypes): argument marshalling only.

Every function has the name of the C entry point it calls (include/q4nx.h).
Host functions take and return NumPy arrays; device functions take torch
tensors that live on the GPU (torch provides device memory and streams) and
enqueue the library's HIP kernels on the current torch stream, or on the
stream passed explicitly.  Nothing here computes any part of the projection.

If the shared library is missing this module raises at import: there is no
fallback path.  Q4NX_LIBRARY, if set, names another build of the same library
to load instead (the host-sanitized build of build.py --sanitize).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("Q4NX_LIBRARY") or os.path.join(_HERE, "libq4nx.so")

Q4NX_OK = 0
Q4NX_ERR_INVALID_ARG = 1
Q4NX_ERR_SHAPE = 2
Q4NX_ERR_ALIGNMENT = 3
Q4NX_ERR_BUFFER_TOO_SMALL = 4
Q4NX_ERR_HIP = 5
Q4NX_F32 = 0
Q4NX_BF16 = 1
Q4NX_MAX_BATCH = 8
Q4NX_WEIGHTS_Q4NX = 0
Q4NX_WEIGHTS_MXFP4 = 1
Q4NX_WEIGHTS_BF16 = 2

EXPORTED = ["q4nx_packed_size", "q4nx_pack", "q4nx_unpack", "q4nx_quantize", "q4nx_dequant", "q4nx_gemv",
            "q4nx_gemv_batched", "q4nx_gemm", "q4nx_gemm_bf16", "q4nx_flowkv_workspace_size",
            "q4nx_flowkv_decode", "q4nx_flowkv_decode_static", "q4nx_mx_packed_size", "q4nx_mx_pack", "q4nx_mx_unpack", "q4nx_mx_quantize", "q4nx_mx_dequant",
            "q4nx_mx_gemv", "q4nx_mx_gemv_batched", "q4nx_mx_gemm", "q4nx_gemm_workspace_size", "q4nx_gemm_ex", "q4nx_stream_read",
            "q4nx_status_str", "q4nx_last_error"]

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2602_06063_amd/build.py`")

# torch ships its own HIP runtime under the same soname (libamdhip64.so.7).
# Loading torch first makes the dynamic loader satisfy libq4nx's dependency
# with that copy, so the process holds one HIP runtime and device pointers and
# streams from torch are valid inside the library.
try:
    import torch as _torch  # noqa: F401
except ImportError:  # host-only use (pack / unpack) without torch
    _torch = None

lib = ctypes.CDLL(LIB_PATH)

_vp, _i64, _i32, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t


class q4nx_gemv_desc(ctypes.Structure):
    _fields_ = [("blob", _vp), ("x", _vp), ("y", _vp), ("N", _i64), ("K", _i64)]


lib.q4nx_packed_size.argtypes = [_i64, _i64]
lib.q4nx_packed_size.restype = _sz
lib.q4nx_pack.argtypes = [_vp, _vp, _vp, _i64, _i64, _vp, _sz]
lib.q4nx_pack.restype = ctypes.c_int
lib.q4nx_unpack.argtypes = [_vp, _sz, _i64, _i64, _vp, _vp, _vp]
lib.q4nx_unpack.restype = ctypes.c_int
lib.q4nx_quantize.argtypes = [_vp, _i64, _i64, _vp, _vp]
lib.q4nx_quantize.restype = ctypes.c_int
lib.q4nx_dequant.argtypes = [_vp, _i64, _i64, _vp, ctypes.c_int, _vp]
lib.q4nx_dequant.restype = ctypes.c_int
lib.q4nx_gemv.argtypes = [_vp, _vp, _vp, ctypes.c_int, _i64, _i64, _vp]
lib.q4nx_gemv.restype = ctypes.c_int
lib.q4nx_gemv_batched.argtypes = [ctypes.POINTER(q4nx_gemv_desc), _i32, ctypes.c_int, _vp]
lib.q4nx_gemv_batched.restype = ctypes.c_int
lib.q4nx_gemm.argtypes = [_i64, _i64, _i64, _vp, _vp, _vp, ctypes.c_int, _vp]
lib.q4nx_gemm.restype = ctypes.c_int
lib.q4nx_gemm_bf16.argtypes = [_i64, _i64, _i64, _vp, _vp, _vp, ctypes.c_int, _vp]
lib.q4nx_gemm_bf16.restype = ctypes.c_int
lib.q4nx_flowkv_workspace_size.argtypes = [_i64, _i64, _i64]
lib.q4nx_flowkv_workspace_size.restype = _sz
lib.q4nx_flowkv_decode.argtypes = [_vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, ctypes.c_float, _vp,
                                   ctypes.c_int, _vp, _sz, _vp]
lib.q4nx_flowkv_decode.restype = ctypes.c_int
lib.q4nx_flowkv_decode_static.argtypes = [_vp, _vp, _vp, _i64, _i64, _i64, _i64, _i64, _i64, ctypes.c_float, _vp,
                                          ctypes.c_int, _vp]
lib.q4nx_flowkv_decode_static.restype = ctypes.c_int
lib.q4nx_mx_packed_size.argtypes = [_i64, _i64]
lib.q4nx_mx_packed_size.restype = _sz
lib.q4nx_mx_pack.argtypes = [_vp, _vp, _i64, _i64, _vp, _sz]
lib.q4nx_mx_pack.restype = ctypes.c_int
lib.q4nx_mx_unpack.argtypes = [_vp, _sz, _i64, _i64, _vp, _vp]
lib.q4nx_mx_unpack.restype = ctypes.c_int
lib.q4nx_mx_quantize.argtypes = [_vp, _i64, _i64, _vp, _vp]
lib.q4nx_mx_quantize.restype = ctypes.c_int
lib.q4nx_mx_dequant.argtypes = [_vp, _i64, _i64, _vp, ctypes.c_int, _vp]
lib.q4nx_mx_dequant.restype = ctypes.c_int
lib.q4nx_mx_gemv.argtypes = [_vp, _vp, _vp, ctypes.c_int, _i64, _i64, _vp]
lib.q4nx_mx_gemv.restype = ctypes.c_int
lib.q4nx_mx_gemv_batched.argtypes = [ctypes.POINTER(q4nx_gemv_desc), _i32, ctypes.c_int, _vp]
lib.q4nx_mx_gemv_batched.restype = ctypes.c_int
lib.q4nx_mx_gemm.argtypes = [_i64, _i64, _i64, _vp, _vp, _vp, ctypes.c_int, _vp]
lib.q4nx_mx_gemm.restype = ctypes.c_int
lib.q4nx_gemm_workspace_size.argtypes = [ctypes.c_int, _i64, _i64, _i64]
lib.q4nx_gemm_workspace_size.restype = _sz
lib.q4nx_gemm_ex.argtypes = [ctypes.c_int, _i64, _i64, _i64, _vp, _vp, _vp, ctypes.c_int, _vp, _sz, _vp]
lib.q4nx_gemm_ex.restype = ctypes.c_int
lib.q4nx_stream_read.argtypes = [_vp, _sz, _vp, _vp]
lib.q4nx_stream_read.restype = ctypes.c_int
lib.q4nx_status_str.argtypes = [ctypes.c_int]
lib.q4nx_status_str.restype = ctypes.c_char_p
lib.q4nx_last_error.argtypes = []
lib.q4nx_last_error.restype = ctypes.c_char_p


class Q4NXError(RuntimeError):
    def __init__(self, status: int, fn: str):
        self.status = status
        msg = lib.q4nx_status_str(status).decode()
        detail = lib.q4nx_last_error().decode()
        super().__init__(f"{fn}: {msg} ({detail})" if detail else f"{fn}: {msg}")


def _check(status: int, fn: str):
    if status != Q4NX_OK:
        raise Q4NXError(status, fn)


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ------------------------------------------------------------------ host
def q4nx_packed_size(N: int, K: int) -> int:
    return int(lib.q4nx_packed_size(N, K))


def q4nx_pack(codes: np.ndarray, scales: np.ndarray, offsets: np.ndarray) -> np.ndarray:
    """codes u8[N][K], scales/offsets bf16 bits u16[N][K/32] -> blob u8."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    N, K = codes.shape
    scales = np.ascontiguousarray(scales, dtype=np.uint16)
    offsets = np.ascontiguousarray(offsets, dtype=np.uint16)
    if scales.size != N * (K // 32) or offsets.size != N * (K // 32):
        raise ValueError("scales and offsets need N * K/32 entries")
    size = q4nx_packed_size(N, K)
    blob = np.empty(max(size, 1), dtype=np.uint8)
    _check(lib.q4nx_pack(_np_ptr(codes), _np_ptr(scales), _np_ptr(offsets), N, K, _np_ptr(blob), size),
           "q4nx_pack")
    return blob[:size]


def q4nx_mx_packed_size(N: int, K: int) -> int:
    return int(lib.q4nx_mx_packed_size(N, K))


def q4nx_mx_pack(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """codes u8[N][K] (FP4 E2M1), scales u8[N][K/32] (E8M0) -> MXFP4-variant blob u8."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    N, K = codes.shape
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    if scales.size != N * (K // 32):
        raise ValueError("scales need N * K/32 entries")
    size = q4nx_mx_packed_size(N, K)
    blob = np.empty(max(size, 1), dtype=np.uint8)
    _check(lib.q4nx_mx_pack(_np_ptr(codes), _np_ptr(scales), N, K, _np_ptr(blob), size), "q4nx_mx_pack")
    return blob[:size]


def q4nx_mx_unpack(blob: np.ndarray, N: int, K: int):
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    codes = np.empty((N, K), np.uint8)
    scales = np.empty((N, max(K // 32, 1)), np.uint8)
    _check(lib.q4nx_mx_unpack(_np_ptr(blob), blob.size, N, K, _np_ptr(codes), _np_ptr(scales)), "q4nx_mx_unpack")
    return codes, scales


def q4nx_unpack(blob: np.ndarray, N: int, K: int):
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    codes = np.empty((N, K), np.uint8)
    scales = np.empty((N, max(K // 32, 1)), np.uint16)
    offsets = np.empty((N, max(K // 32, 1)), np.uint16)
    _check(lib.q4nx_unpack(_np_ptr(blob), blob.size, N, K, _np_ptr(codes), _np_ptr(scales), _np_ptr(offsets)),
           "q4nx_unpack")
    return codes, scales, offsets


# ------------------------------------------------------------------ device
def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if hasattr(stream, "cuda_stream"):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _dptr(t) -> int:
    if not t.is_cuda:
        raise ValueError("expected a GPU tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _need(t, nbytes: int, what: str):
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what}: {have} bytes, need {nbytes}")


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return Q4NX_F32
    if t.dtype == torch.bfloat16:
        return Q4NX_BF16
    raise ValueError("outputs must be float32 or bfloat16")


def q4nx_quantize(W, N: int, K: int, blob, stream=None):
    """blob <- Q4NX quantization of the float32 weights W[N][K] (device)."""
    _need(W, 4 * N * K, "W")
    _need(blob, q4nx_packed_size(N, K), "blob")
    _check(lib.q4nx_quantize(_dptr(W), N, K, _dptr(blob), _stream(stream)), "q4nx_quantize")


def q4nx_dequant(blob, N: int, K: int, W, stream=None):
    """W[N][K] (float32 or bfloat16 tensor) <- Eq. 3 of every packed weight."""
    _need(blob, q4nx_packed_size(N, K), "blob")
    _need(W, N * K * W.element_size(), "W")
    _check(lib.q4nx_dequant(_dptr(blob), N, K, _dptr(W), _dtype_code(W), _stream(stream)), "q4nx_dequant")


def q4nx_gemv(blob, x, y, N: int, K: int, stream=None):
    """y[N] <- W x; x is a bf16 (or 16-bit bit-pattern) tensor of K values."""
    _need(blob, q4nx_packed_size(N, K), "blob")
    _need(x, 2 * K, "x")
    _need(y, N * y.element_size(), "y")
    _check(lib.q4nx_gemv(_dptr(blob), _dptr(x), _dptr(y), _dtype_code(y), N, K, _stream(stream)), "q4nx_gemv")


def q4nx_gemv_batched(items, stream=None):
    """items: sequence of (blob, x, y, N, K); all y share one dtype."""
    items = list(items)
    arr = (q4nx_gemv_desc * max(len(items), 1))()
    for i, (blob, x, y, N, K) in enumerate(items):
        _need(blob, q4nx_packed_size(N, K), "blob")
        _need(x, 2 * K, "x")
        _need(y, N * y.element_size(), "y")
        arr[i] = q4nx_gemv_desc(_dptr(blob), _dptr(x), _dptr(y), N, K)
    ydt = _dtype_code(items[0][2]) if items else Q4NX_F32
    if any(_dtype_code(it[2]) != ydt for it in items):
        raise ValueError("all outputs of a batch must share one dtype")
    _check(lib.q4nx_gemv_batched(arr, len(items), ydt, _stream(stream)), "q4nx_gemv_batched")


def q4nx_gemm(M: int, N: int, K: int, X, blob, Y, stream=None):
    """Y[M][N] <- X[M][K] W^T with W dequantized to bf16."""
    _need(blob, q4nx_packed_size(N, K), "blob")
    _need(X, 2 * M * K, "X")
    _need(Y, M * N * Y.element_size(), "Y")
    _check(lib.q4nx_gemm(M, N, K, _dptr(X), _dptr(blob), _dptr(Y), _dtype_code(Y), _stream(stream)),
           "q4nx_gemm")


def q4nx_gemm_bf16(M: int, N: int, K: int, X, W, Y, stream=None):
    """Y[M][N] <- X[M][K] W^T with W already bf16 [N][K] (the second phase of
    the two-phase prefill: W from q4nx_dequant with a bf16 output)."""
    _need(W, 2 * N * K, "W")
    _need(X, 2 * M * K, "X")
    _need(Y, M * N * Y.element_size(), "Y")
    _check(lib.q4nx_gemm_bf16(M, N, K, _dptr(X), _dptr(W), _dptr(Y), _dtype_code(Y), _stream(stream)),
           "q4nx_gemm_bf16")


def q4nx_mx_quantize(W, N: int, K: int, blob, stream=None):
    """blob <- MXFP4-variant quantization of the float32 weights W[N][K] (device)."""
    _need(W, 4 * N * K, "W")
    _need(blob, q4nx_mx_packed_size(N, K), "blob")
    _check(lib.q4nx_mx_quantize(_dptr(W), N, K, _dptr(blob), _stream(stream)), "q4nx_mx_quantize")


def q4nx_mx_dequant(blob, N: int, K: int, W, stream=None):
    """W[N][K] (float32 or bfloat16 tensor) <- X * fp4(q) of every weight of an MXFP4-variant blob."""
    _need(blob, q4nx_mx_packed_size(N, K), "blob")
    _need(W, N * K * W.element_size(), "W")
    _check(lib.q4nx_mx_dequant(_dptr(blob), N, K, _dptr(W), _dtype_code(W), _stream(stream)), "q4nx_mx_dequant")


def q4nx_mx_gemv(blob, x, y, N: int, K: int, stream=None):
    """y[N] <- W x for an MXFP4-variant blob."""
    _need(blob, q4nx_mx_packed_size(N, K), "blob")
    _need(x, 2 * K, "x")
    _need(y, N * y.element_size(), "y")
    _check(lib.q4nx_mx_gemv(_dptr(blob), _dptr(x), _dptr(y), _dtype_code(y), N, K, _stream(stream)),
           "q4nx_mx_gemv")


def q4nx_mx_gemv_batched(items, stream=None):
    """items: sequence of (blob, x, y, N, K) over MXFP4-variant blobs; all y share one dtype."""
    items = list(items)
    arr = (q4nx_gemv_desc * max(len(items), 1))()
    for i, (blob, x, y, N, K) in enumerate(items):
        _need(blob, q4nx_mx_packed_size(N, K), "blob")
        _need(x, 2 * K, "x")
        _need(y, N * y.element_size(), "y")
        arr[i] = q4nx_gemv_desc(_dptr(blob), _dptr(x), _dptr(y), N, K)
    ydt = _dtype_code(items[0][2]) if items else Q4NX_F32
    if any(_dtype_code(it[2]) != ydt for it in items):
        raise ValueError("all outputs of a batch must share one dtype")
    _check(lib.q4nx_mx_gemv_batched(arr, len(items), ydt, _stream(stream)), "q4nx_mx_gemv_batched")


def q4nx_mx_gemm(M: int, N: int, K: int, X, blob, Y, stream=None):
    """Y[M][N] <- X[M][K] W^T for an MXFP4-variant blob (W exact in bf16)."""
    _need(blob, q4nx_mx_packed_size(N, K), "blob")
    _need(X, 2 * M * K, "X")
    _need(Y, M * N * Y.element_size(), "Y")
    _check(lib.q4nx_mx_gemm(M, N, K, _dptr(X), _dptr(blob), _dptr(Y), _dtype_code(Y), _stream(stream)),
           "q4nx_mx_gemm")


def q4nx_gemm_workspace_size(w_format: int, M: int, N: int, K: int) -> int:
    return int(lib.q4nx_gemm_workspace_size(w_format, M, N, K))


def q4nx_gemm_ex(w_format: int, M: int, N: int, K: int, X, W, Y, work=None, stream=None):
    """Y[M][N] <- X[M][K] W^T for W in the given format (Q4NX_WEIGHTS_*); with a
    workspace of q4nx_gemm_workspace_size(w_format, M, N, K) bytes the plan may
    split K and, for Q4NX weights and a large M, dequantize W to bf16 first."""
    wbytes = {Q4NX_WEIGHTS_Q4NX: q4nx_packed_size(N, K), Q4NX_WEIGHTS_MXFP4: q4nx_mx_packed_size(N, K),
              Q4NX_WEIGHTS_BF16: 2 * N * K}.get(w_format, 0)
    _need(W, wbytes, "W")
    _need(X, 2 * M * K, "X")
    _need(Y, M * N * Y.element_size(), "Y")
    wp, wn = (None, 0) if work is None else (_dptr(work), work.numel() * work.element_size())
    _check(lib.q4nx_gemm_ex(w_format, M, N, K, _dptr(X), _dptr(W), _dptr(Y), _dtype_code(Y), wp, wn, _stream(stream)),
           "q4nx_gemm_ex")


def q4nx_stream_read(src, sink, stream=None):
    """Measurement aid: read all of `src` once (sink: 8192 float32, one fold per wave)."""
    _need(sink, 4 * 8192, "sink")
    _check(lib.q4nx_stream_read(_dptr(src), src.numel() * src.element_size(), _dptr(sink), _stream(stream)),
           "q4nx_stream_read")


def q4nx_flowkv_workspace_size(H: int, d: int, n_keys: int) -> int:
    return lib.q4nx_flowkv_workspace_size(H, d, n_keys)


def q4nx_flowkv_decode(q, K, V, H: int, G: int, d: int, L: int, t: int, window: int, scale: float, o, work,
                       stream=None):
    """o[H][d] <- FlowKV decode attention of the query q[H][d] over the cache
    K, V [G][L][d] at position t (window 0 = full attention)."""
    _need(q, 2 * H * d, "q")
    _need(K, 2 * G * L * d, "K")
    _need(V, 2 * G * L * d, "V")
    _need(o, H * d * o.element_size(), "o")
    _check(lib.q4nx_flowkv_decode(_dptr(q), _dptr(K), _dptr(V), H, G, d, L, t, window, scale, _dptr(o),
                                  _dtype_code(o), _dptr(work), work.numel() * work.element_size(), _stream(stream)),
           "q4nx_flowkv_decode")


def q4nx_flowkv_decode_static(q, K, V, H: int, G: int, d: int, L: int, t: int, window: int, scale: float, o,
                              stream=None):
    """q4nx_flowkv_decode with the chunk partials in the library's static
    device scratch (no workspace argument, nothing allocated)."""
    _need(q, 2 * H * d, "q")
    _need(K, 2 * G * L * d, "K")
    _need(V, 2 * G * L * d, "V")
    _need(o, H * d * o.element_size(), "o")
    _check(lib.q4nx_flowkv_decode_static(_dptr(q), _dptr(K), _dptr(V), H, G, d, L, t, window, scale, _dptr(o),
                                         _dtype_code(o), _stream(stream)),
           "q4nx_flowkv_decode_static")
