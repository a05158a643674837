"""Python binding of libsoniq (gfx950): SONIQ's per-channel mixed-precision
quantized matrix multiply (arXiv 2311.14114, Sec. 3 codec and Alg. 1 Phase II
integer MAC).

The functions carry the C-ABI names of ``include/soniq.h`` and only marshal
arguments: torch tensors provide device pointers and the current HIP stream;
every step runs in the library's HIP kernels.  There is no CPU fallback: if
``libsoniq.so`` is missing, importing the binding's entry points raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsoniq.so")

SONIQ_OK = 0
SONIQ_ERR_INVALID_ARGUMENT = 1
SONIQ_ERR_UNSUPPORTED = 2
SONIQ_ERR_OUT_OF_MEMORY = 3
SONIQ_ERR_HIP = 4
SONIQ_WQ_SYMMETRIC = 0
SONIQ_WQ_TWOS_FRACTION = 1
SONIQ_WPACK_SIGN_NIBBLES = 0x100
SONIQ_WPACK_F8F6F4 = 0x200
SONIQ_WPACK_DENSE = 0x400
SONIQ_MAX_K = 65536

# Every symbol include/soniq.h declares.
EXPORTED = [
    "soniq_pack_weights", "soniq_pack_weights_ex", "soniq_pack_weights_grouped",
    "soniq_pack_weights_conv3x3", "soniq_act_create", "soniq_act_create_conv3x3",
    "soniq_quantize_act", "soniq_quantize_act_conv3x3", "soniq_mp_gemm", "soniq_quantize_mp_gemm",
    "soniq_quantize_mp_gemm_scratch",
    "soniq_mp_gemm_quantize_next", "soniq_mp_gemm_quantize_next_max",
    "soniq_weights_info",
    "soniq_plan_input_channels", "soniq_weights_unpack_debug",
    "soniq_act_unpack_debug", "soniq_act_wait_timeouts", "soniq_debug_stream_read",
    "soniq_weights_destroy",
    "soniq_act_destroy",
    "soniq_last_error",
]


class SoniqError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"soniq status {status}: {msg}")
        self.status = status


class WeightsInfo(ctypes.Structure):
    _fields_ = [
        ("N", ctypes.c_int64), ("K", ctypes.c_int64), ("S", ctypes.c_int32),
        ("a_signed", ctypes.c_int32), ("wq_mode", ctypes.c_int32),
        ("a_bits", ctypes.c_uint8 * 2), ("w_bits", ctypes.c_uint8 * 2),
        ("a_count", ctypes.c_int64 * 2), ("a_count_padded", ctypes.c_int64 * 2),
        ("w_count", ctypes.c_int64 * 2), ("packed_w_bytes", ctypes.c_int64),
        ("packed_w_bytes_algorithmic", ctypes.c_int64),
        ("act_group_bits", ctypes.c_int32), ("act_scales", ctypes.c_int32),
        ("f8f6f4", ctypes.c_int32), ("dense_w_bytes", ctypes.c_int64),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsoniq.so (fails loudly when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "or python -m paper_2311_14114_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32, st = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int
        L.soniq_pack_weights.restype = st
        L.soniq_pack_weights.argtypes = [vp, i64, i64, i64, vp, vp, i32, vp, ctypes.POINTER(vp)]
        L.soniq_pack_weights_ex.restype = st
        L.soniq_pack_weights_ex.argtypes = [vp, i64, i64, i64, vp, vp, i32, i32, vp, ctypes.POINTER(vp)]
        L.soniq_pack_weights_grouped.restype = st
        L.soniq_pack_weights_grouped.argtypes = [vp, i64, i64, i64, vp, vp, i32, i32, i32, vp,
                                                 ctypes.POINTER(vp)]
        L.soniq_pack_weights_conv3x3.restype = st
        L.soniq_pack_weights_conv3x3.argtypes = [vp, i64, i64, vp, vp, i32, i32, vp,
                                                 ctypes.POINTER(vp)]
        L.soniq_act_create_conv3x3.restype = st
        L.soniq_act_create_conv3x3.argtypes = [vp, i64, i64, i64, ctypes.POINTER(vp)]
        L.soniq_act_create.restype = st
        L.soniq_act_create.argtypes = [vp, i64, ctypes.POINTER(vp)]
        L.soniq_quantize_act.restype = st
        L.soniq_quantize_act.argtypes = [vp, vp, i64, i64, vp]
        L.soniq_quantize_act_conv3x3.restype = st
        L.soniq_quantize_act_conv3x3.argtypes = [vp, vp, i64, i64, i64, i64, vp]
        L.soniq_mp_gemm.restype = st
        L.soniq_mp_gemm.argtypes = [vp, vp, vp, i64, vp, vp]
        L.soniq_mp_gemm_quantize_next.restype = st
        L.soniq_mp_gemm_quantize_next.argtypes = [vp, vp, vp, vp, vp, i64, vp, vp]
        L.soniq_mp_gemm_quantize_next_max.restype = st
        L.soniq_mp_gemm_quantize_next_max.argtypes = [vp, vp, vp, vp, i64, vp, vp]
        L.soniq_quantize_mp_gemm.restype = st
        L.soniq_quantize_mp_gemm.argtypes = [vp, vp, vp, i64, i64, vp, i64, vp, vp]
        L.soniq_quantize_mp_gemm_scratch.restype = st
        L.soniq_quantize_mp_gemm_scratch.argtypes = [vp, vp, i64, i64, vp, i64, vp, vp]
        L.soniq_weights_info.restype = st
        L.soniq_weights_info.argtypes = [vp, ctypes.POINTER(WeightsInfo)]
        L.soniq_plan_input_channels.restype = st
        L.soniq_plan_input_channels.argtypes = [vp, i64, vp, vp, vp, vp]
        L.soniq_weights_unpack_debug.restype = st
        L.soniq_weights_unpack_debug.argtypes = [vp, vp, vp]
        L.soniq_act_unpack_debug.restype = st
        L.soniq_act_unpack_debug.argtypes = [vp, vp, vp]
        L.soniq_act_wait_timeouts.restype = st
        L.soniq_act_wait_timeouts.argtypes = [vp, ctypes.POINTER(ctypes.c_uint64)]
        L.soniq_debug_stream_read.restype = st
        L.soniq_debug_stream_read.argtypes = [vp, i64, vp, vp]
        L.soniq_weights_destroy.restype = None
        L.soniq_weights_destroy.argtypes = [vp]
        L.soniq_act_destroy.restype = None
        L.soniq_act_destroy.argtypes = [vp]
        L.soniq_last_error.restype = ctypes.c_char_p
        L.soniq_last_error.argtypes = []
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != SONIQ_OK:
        raise SoniqError(status, lib().soniq_last_error().decode())


def _u8(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.uint8)


def _stream(stream):
    if stream is not None:
        return ctypes.c_void_p(int(stream))
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype_name: str):
    import torch
    if not (isinstance(t, torch.Tensor) and t.is_cuda):
        raise TypeError(f"expected a device tensor ({dtype_name})")
    return ctypes.c_void_p(t.data_ptr())


class Weights:
    """Owner of a packed weights handle (soniq_weights)."""

    def __init__(self, handle: ctypes.c_void_p, N: int, K: int):
        self.handle = handle
        self.N, self.K = N, K
        self.info = soniq_weights_info(self)
        # accumulators per output: precision groups, or sub-group blocks
        self.S = self.info.act_scales

    def close(self):
        if self.handle:
            lib().soniq_weights_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Activations:
    """Owner of a packed activation handle (soniq_act)."""

    def __init__(self, handle: ctypes.c_void_p, weights: Weights, max_M: int):
        self.handle = handle
        self.weights = weights      # keeps the weights alive
        self.max_M = max_M
        self.M = 0

    def close(self):
        if self.handle:
            lib().soniq_act_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def soniq_pack_weights(W, w_bits, a_bits, a_signed: bool, wq_mode: int = SONIQ_WQ_SYMMETRIC,
                       stream=None, act_group_bits: int = 0, sign_nibbles: bool = False,
                       f8f6f4: bool = False, dense: bool = False) -> Weights:
    """Quantize, re-order and bit-pack W (device float32 [N, K], row-major).
    act_group_bits > 0 gives the activations sub-group scales (blocks of
    that many bits of storage inside each precision group); sign_nibbles
    stores 1-bit channels in 4-bit containers (SONIQ_WPACK_SIGN_NIBBLES);
    f8f6f4 also keeps the narrow operands in fp4/fp6 MFMA operand formats
    (SONIQ_WPACK_F8F6F4); dense also keeps every code in exactly its width
    for the GEMV forms (SONIQ_WPACK_DENSE)."""
    import torch
    if W.dtype != torch.float32 or W.dim() != 2 or W.stride(1) != 1:
        raise TypeError("W must be a 2-D float32 device tensor with unit column stride")
    N, K = W.shape
    wb, ab = _u8(w_bits), _u8(a_bits)
    if wb.shape != (N,) or ab.shape != (K,):
        raise ValueError("w_bits must have N entries and a_bits K entries")
    h = ctypes.c_void_p()
    _check(lib().soniq_pack_weights_grouped(_dev(W, "float32"), N, K, W.stride(0),
                                            wb.ctypes.data_as(ctypes.c_void_p),
                                            ab.ctypes.data_as(ctypes.c_void_p),
                                            1 if a_signed else 0,
                                            int(wq_mode) | (SONIQ_WPACK_SIGN_NIBBLES if sign_nibbles else 0)
                                            | (SONIQ_WPACK_F8F6F4 if f8f6f4 else 0)
                                            | (SONIQ_WPACK_DENSE if dense else 0),
                                            int(act_group_bits), _stream(stream),
                                            ctypes.byref(h)))
    return Weights(h, N, K)


def soniq_pack_weights_conv3x3(Wf, w_bits, c_bits, a_signed: bool,
                               wq_mode: int = SONIQ_WQ_SYMMETRIC, stream=None,
                               sign_nibbles: bool = False) -> Weights:
    """Pack a 3x3 filter (device float32 [N, C, 3, 3], contiguous) for the
    implicit-GEMM convolution; c_bits holds one width per input channel.
    The handle behaves as weights of K = 9*C columns (k = c*9 + kh*3 + kw)."""
    import torch
    if Wf.dtype != torch.float32 or Wf.dim() != 4 or tuple(Wf.shape[2:]) != (3, 3) \
            or not Wf.is_contiguous():
        raise TypeError("the filter must be a contiguous float32 [N, C, 3, 3] device tensor")
    N, C = Wf.shape[0], Wf.shape[1]
    wb, cb = _u8(w_bits), _u8(c_bits)
    if wb.shape != (N,) or cb.shape != (C,):
        raise ValueError("w_bits must have N entries and c_bits C entries")
    h = ctypes.c_void_p()
    _check(lib().soniq_pack_weights_conv3x3(_dev(Wf, "float32"), N, C,
                                            wb.ctypes.data_as(ctypes.c_void_p),
                                            cb.ctypes.data_as(ctypes.c_void_p),
                                            1 if a_signed else 0,
                                            int(wq_mode) | (SONIQ_WPACK_SIGN_NIBBLES if sign_nibbles else 0),
                                            _stream(stream), ctypes.byref(h)))
    return Weights(h, N, 9 * C)


def soniq_act_create_conv3x3(weights: Weights, B: int, H: int, W: int) -> Activations:
    h = ctypes.c_void_p()
    _check(lib().soniq_act_create_conv3x3(weights.handle, int(B), int(H), int(W), ctypes.byref(h)))
    return Activations(h, weights, int(B) * int(H) * int(W))


def soniq_act_create(weights: Weights, max_M: int) -> Activations:
    h = ctypes.c_void_p()
    _check(lib().soniq_act_create(weights.handle, int(max_M), ctypes.byref(h)))
    return Activations(h, weights, int(max_M))


def soniq_quantize_act(act: Activations, A, stream=None) -> None:
    """Quantize and pack A (device float32 [M, K], row-major) into `act`."""
    import torch
    if A.dtype != torch.float32 or A.dim() != 2 or A.stride(1) != 1:
        raise TypeError("A must be a 2-D float32 device tensor with unit column stride")
    if A.shape[1] != act.weights.K:
        raise ValueError("A has the wrong number of input channels")
    _check(lib().soniq_quantize_act(act.handle, _dev(A, "float32"), A.shape[0], A.stride(0),
                                    _stream(stream)))
    act.M = A.shape[0]


def soniq_quantize_act_conv3x3(act: Activations, X, stream=None) -> None:
    """Quantize and pack the activations of a stride-1, pad-1 3x3 convolution
    straight from its input X (device float32 [B, C, H, W], contiguous); the
    handle's weights are the [N, C, 3, 3] filter viewed as [N, 9C]."""
    import torch
    if X.dtype != torch.float32 or X.dim() != 4 or not X.is_contiguous():
        raise TypeError("X must be a contiguous 4-D float32 device tensor")
    B, C, H, W = X.shape
    _check(lib().soniq_quantize_act_conv3x3(act.handle, _dev(X, "float32"), B, C, H, W,
                                            _stream(stream)))
    act.M = B * H * W


def soniq_mp_gemm(act: Activations, weights: Weights, out=None, acc=None, stream=None):
    """Y[M, N] (bf16) from the last quantized activations; optional int32
    accumulator dump acc[S, M, N].  Returns Y."""
    import torch
    M, N = act.M, weights.N
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1 or out.shape[0] < M:
        raise TypeError("out must be a bf16 [M, >=N] device tensor with unit column stride")
    accp = None
    if acc is not None:
        if acc.dtype != torch.int32 or not acc.is_contiguous() or tuple(acc.shape) != (weights.S, M, N):
            raise TypeError("acc must be a contiguous int32 [S, M, N] device tensor")
        accp = _dev(acc, "int32")
    _check(lib().soniq_mp_gemm(act.handle, weights.handle, _dev(out, "bf16"), out.stride(0),
                               accp, _stream(stream)))
    return out



def soniq_quantize_mp_gemm(act: Activations, weights: Weights, A, out=None, acc=None, stream=None):
    """soniq_quantize_act(act, A) then soniq_mp_gemm(act, weights) in one call
    (a single launch for a batch of one row).  Returns Y."""
    import torch
    if A.dtype != torch.float32 or A.dim() != 2 or A.stride(1) != 1:
        raise TypeError("A must be a 2-D float32 device tensor with unit column stride")
    if A.shape[1] != act.weights.K:
        raise ValueError("A has the wrong number of input channels")
    M, N = A.shape[0], weights.N
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1 or out.shape[0] < M:
        raise TypeError("out must be a bf16 [M, >=N] device tensor with unit column stride")
    accp = None
    if acc is not None:
        if acc.dtype != torch.int32 or not acc.is_contiguous() or tuple(acc.shape) != (weights.S, M, N):
            raise TypeError("acc must be a contiguous int32 [S, M, N] device tensor")
        accp = _dev(acc, "int32")
    _check(lib().soniq_quantize_mp_gemm(act.handle, weights.handle, _dev(A, "float32"), M, A.stride(0),
                                        _dev(out, "bf16"), out.stride(0), accp, _stream(stream)))
    act.M = M
    return out


def soniq_quantize_mp_gemm_scratch(weights: Weights, A, out=None, acc=None, stream=None):
    """soniq_quantize_mp_gemm without an activation handle: the library's
    per-device scratch holds the packed activations, and the call allocates
    nothing (pass `out` to keep the binding from allocating Y).  Returns Y."""
    import torch
    if A.dtype != torch.float32 or A.dim() != 2 or A.stride(1) != 1:
        raise TypeError("A must be a 2-D float32 device tensor with unit column stride")
    if A.shape[1] != weights.K:
        raise ValueError("A has the wrong number of input channels")
    M, N = A.shape[0], weights.N
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1 or out.shape[0] < M:
        raise TypeError("out must be a bf16 [M, >=N] device tensor with unit column stride")
    accp = None
    if acc is not None:
        if acc.dtype != torch.int32 or not acc.is_contiguous() or tuple(acc.shape) != (weights.S, M, N):
            raise TypeError("acc must be a contiguous int32 [S, M, N] device tensor")
        accp = _dev(acc, "int32")
    _check(lib().soniq_quantize_mp_gemm_scratch(weights.handle, _dev(A, "float32"), M, A.stride(0),
                                                _dev(out, "bf16"), out.stride(0), accp,
                                                _stream(stream)))
    return out


def soniq_mp_gemm_quantize_next(act: Activations, weights: Weights, next_act: Activations,
                                s_next, out=None, acc=None, stream=None):
    """soniq_mp_gemm(act, weights) whose epilogue also quantizes the outputs
    into next_act with the static scales s_next (one per next-layer
    activation group, or per block for sub-group weights).  out=None skips
    Y; returns out."""
    import torch
    M, N = act.M, weights.N
    sn = np.ascontiguousarray(np.asarray(s_next, np.float32).ravel())
    if sn.shape[0] < next_act.weights.S:
        raise ValueError("one static scale per next-layer activation group (or block)")
    outp, ldy = None, N
    if out is not None:
        if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1 or out.shape[0] < M:
            raise TypeError("out must be a bf16 [M, >=N] device tensor with unit column stride")
        outp, ldy = _dev(out, "bf16"), out.stride(0)
    accp = None
    if acc is not None:
        if acc.dtype != torch.int32 or not acc.is_contiguous() or tuple(acc.shape) != (weights.S, M, N):
            raise TypeError("acc must be a contiguous int32 [S, M, N] device tensor")
        accp = _dev(acc, "int32")
    _check(lib().soniq_mp_gemm_quantize_next(act.handle, weights.handle, next_act.handle,
                                             sn.ctypes.data_as(ctypes.c_void_p), outp, ldy, accp,
                                             _stream(stream)))
    next_act.M = M
    return out


def soniq_mp_gemm_quantize_next_max(act: Activations, weights: Weights, next_act: Activations,
                                    out=None, acc=None, stream=None):
    """soniq_mp_gemm(act, weights) storing Y (out, allocated when None) whose
    epilogue also folds each next-layer group's largest |Y|; next_act then
    holds soniq_quantize_act of float(Y) with that batch maximum.  Returns
    out."""
    import torch
    M, N = act.M, weights.N
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.stride(1) != 1 or out.shape[0] < M:
        raise TypeError("out must be a bf16 [M, >=N] device tensor with unit column stride")
    accp = None
    if acc is not None:
        if acc.dtype != torch.int32 or not acc.is_contiguous() or tuple(acc.shape) != (weights.S, M, N):
            raise TypeError("acc must be a contiguous int32 [S, M, N] device tensor")
        accp = _dev(acc, "int32")
    _check(lib().soniq_mp_gemm_quantize_next_max(act.handle, weights.handle, next_act.handle,
                                                 _dev(out, "bf16"), out.stride(0), accp,
                                                 _stream(stream)))
    next_act.M = M
    return out


def soniq_weights_info(weights: Weights) -> WeightsInfo:
    info = WeightsInfo()
    _check(lib().soniq_weights_info(weights.handle, ctypes.byref(info)))
    return info


def soniq_plan_input_channels(a_bits):
    """Host-only input-channel plan: (pos[K], seg_len[2], seg_pad[2], S)."""
    ab = _u8(a_bits)
    K = ab.shape[0]
    pos = np.empty(K, np.int64)
    seg_len = np.zeros(2, np.int64)
    seg_pad = np.zeros(2, np.int64)
    S = ctypes.c_int32()
    _check(lib().soniq_plan_input_channels(ab.ctypes.data_as(ctypes.c_void_p), K,
                                           pos.ctypes.data_as(ctypes.c_void_p),
                                           seg_len.ctypes.data_as(ctypes.c_void_p),
                                           seg_pad.ctypes.data_as(ctypes.c_void_p),
                                           ctypes.byref(S)))
    return pos, seg_len, seg_pad, S.value


def soniq_weights_unpack_debug(weights: Weights):
    """Codes int32 [N, K] (original order) and scales float32 [N]."""
    codes = np.empty((weights.N, weights.K), np.int32)
    s_w = np.empty(weights.N, np.float32)
    _check(lib().soniq_weights_unpack_debug(weights.handle, codes.ctypes.data_as(ctypes.c_void_p),
                                            s_w.ctypes.data_as(ctypes.c_void_p)))
    return codes, s_w


def soniq_act_unpack_debug(act: Activations):
    """Codes int32 [M, K] (original order) and scales float32 [S] (one per
    precision group, or per sub-group block)."""
    codes = np.empty((act.M, act.weights.K), np.int32)
    s_a = np.zeros(max(2, act.weights.S), np.float32)
    _check(lib().soniq_act_unpack_debug(act.handle, codes.ctypes.data_as(ctypes.c_void_p),
                                        s_a.ctypes.data_as(ctypes.c_void_p)))
    return codes, s_a[: act.weights.S].copy()


def soniq_debug_stream_read(src, nbytes: int, sink, offset: int = 0, stream=None) -> None:
    """One plain read of nbytes of the device tensor src from byte offset
    `offset` (a measurement aid: the ceiling a bandwidth-bound kernel is
    held against); sink, an int32 device tensor of at least
    ceil(nbytes / 8192) elements, receives one XOR per workgroup."""
    import torch
    if not (isinstance(src, torch.Tensor) and src.is_cuda and src.is_contiguous()):
        raise TypeError("src must be a contiguous device tensor")
    if offset < 0 or offset + nbytes > src.numel() * src.element_size():
        raise ValueError("the read lies outside src")
    if sink.dtype != torch.int32 or not sink.is_cuda or sink.numel() < (nbytes + 8191) // 8192:
        raise TypeError("sink must be an int32 device tensor of ceil(nbytes / 8192) elements")
    _check(lib().soniq_debug_stream_read(ctypes.c_void_p(src.data_ptr() + offset), nbytes,
                                         _dev(sink, "int32"), _stream(stream)))


def soniq_act_wait_timeouts(act: Activations) -> int:
    """Workgroups of the single-pass quantizer whose grid wait timed out
    since the handle was made (results unchanged; the call was slow)."""
    n = ctypes.c_uint64(0)
    _check(lib().soniq_act_wait_timeouts(act.handle, ctypes.byref(n)))
    return int(n.value)
