"""CPU oracle for SONIQ's inference hot path (arXiv 2311.14114).

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this package.  The
product library never loads it, and it shares no code with the HIP path.

The arithmetic lives in ``soniq_oracle.c`` (plain C loops, OpenMP over rows);
this module only marshals numpy arrays.  Each function names the passage of
the paper it follows:

* ``quantize_weights`` -- group max-abs scale (Sec. 3, codec item 1), signed
  codes on the symmetric grid, or on the two's-complement fraction grid of
  Eq. (1) (codec item 3).
* ``quantize_act`` -- one scale per activation precision group (Sec. 2.4 C2,
  Alg. 1 channel permutation); unsigned codec of codec item 2, or the signed
  symmetric grid.
* ``quantize_act_grouped`` -- sub-group scales: blocks of GroupSize_act
  bits inside each precision group (Sec. 3 design-space parameters; the
  group-wise activation normalization of the transformer setup, Sec. 5).
* ``mac`` -- integer multiply-accumulate, one int32 sum per activation group
  or sub-group (Alg. 1, Phase II integer forward).
* ``quantize_act_static`` -- the same codes with caller-given (calibrated)
  group scales: what a producing kernel can quantize its own outputs with
  (Sec. 4 fuses quantization into the preceding operation).
* ``epilogue_ref`` -- y = bf16(s_w * sum_g s_a[g] * ACC[g]) in fp64;
  ``epilogue_replay_f32`` the fixed-order fp32 value before rounding.
* ``run`` -- the whole path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "soniq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

SIGNED, UNSIGNED, TWOS_FRACTION = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (IEEE fp32, no contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-std=c11", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        i64, i32, f32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_void_p
        L.orc_threads.restype = i32
        L.orc_threads.argtypes = []
        L.orc_qmax.restype = i64
        L.orc_qmax.argtypes = [i32, i32]
        L.orc_scale.restype = f32
        L.orc_scale.argtypes = [f32, i32, i32]
        L.orc_code.restype = ctypes.c_int32
        L.orc_code.argtypes = [f32, f32, i32, i32]
        L.orc_quantize_weights.restype = None
        L.orc_quantize_weights.argtypes = [vp, i64, i64, i64, vp, i32, vp, vp]
        L.orc_segments.restype = i32
        L.orc_segments.argtypes = [vp, i64, vp, vp]
        L.orc_quantize_act.restype = i32
        L.orc_quantize_act.argtypes = [vp, i64, i64, i64, vp, i32, vp, vp, vp, vp]
        L.orc_quantize_act_grouped.restype = i32
        L.orc_quantize_act_grouped.argtypes = [vp, i64, i64, i64, vp, i32, i32, i32, vp, vp, vp, vp]
        L.orc_mac.restype = i32
        L.orc_mac.argtypes = [vp, vp, vp, i64, i64, i64, i32, vp]
        L.orc_mac_at.restype = None
        L.orc_mac_at.argtypes = [vp, vp, vp, i64, i32, i64, vp, vp, vp]
        L.orc_bf16_from_f64.restype = ctypes.c_uint16
        L.orc_bf16_from_f64.argtypes = [ctypes.c_double]
        L.orc_bf16_from_f32.restype = ctypes.c_uint16
        L.orc_bf16_from_f32.argtypes = [f32]
        L.orc_epilogue_ref.restype = None
        L.orc_epilogue_ref.argtypes = [vp, vp, vp, i64, i64, i32, vp]
        L.orc_epilogue_replay.restype = None
        L.orc_epilogue_replay.argtypes = [vp, vp, vp, i64, i64, i32, vp]
        L.orc_epilogue_replay_f32.restype = None
        L.orc_epilogue_replay_f32.argtypes = [vp, vp, vp, i64, i64, i32, vp]
        L.orc_quantize_act_static.restype = i32
        L.orc_quantize_act_static.argtypes = [vp, i64, i64, i64, vp, i32, vp, vp]
        L.orc_quantize_act_static_grouped.restype = i32
        L.orc_quantize_act_static_grouped.argtypes = [vp, i64, i64, i64, vp, i32, i32, i32, vp, vp, vp]
        L.orc_container.restype = i32
        L.orc_container.argtypes = [i32]
        L.orc_pack.restype = i64
        L.orc_pack.argtypes = [vp, i64, i32, i32, vp]
        L.orc_unpack.restype = None
        L.orc_unpack.argtypes = [vp, i64, i32, i32, vp]
        _lib = L
    return _lib


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(lib().orc_threads())


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def qmax(bits: int, mode: int) -> int:
    """Largest code magnitude (grid denominator for Eq. (1) mode)."""
    return int(lib().orc_qmax(bits, mode))


def scale(maxabs: float, bits: int, mode: int) -> np.float32:
    return np.float32(lib().orc_scale(np.float32(maxabs), bits, mode))


def code(x: float, s: float, bits: int, mode: int) -> int:
    return int(lib().orc_code(np.float32(x), np.float32(s), bits, mode))


def quantize_weights(W, w_bits, mode: int = SIGNED):
    """Per-output-channel max-abs scales and signed codes of W[N,K]."""
    W = _c(W, np.float32)
    N, K = W.shape
    wb = _c(w_bits, np.uint8)
    assert wb.shape == (N,)
    q = np.empty((N, K), np.int32)
    s = np.empty((N,), np.float32)
    lib().orc_quantize_weights(_p(W), N, K, K, _p(wb), mode, _p(q), _p(s))
    return q, s


def segments(a_bits):
    ab = _c(a_bits, np.uint8)
    sb = np.zeros(2, np.uint8)
    so = np.empty(ab.shape[0], np.uint8)
    S = lib().orc_segments(_p(ab), ab.shape[0], _p(sb), _p(so))
    if S < 0:
        raise ValueError("activation widths must be 1..8 with at most two distinct values")
    return S, sb[:S].copy(), so


def quantize_act(A, a_bits, a_signed: bool):
    """Per-precision-group scales and codes of A[M,K]."""
    A = _c(A, np.float32)
    M, K = A.shape
    ab = _c(a_bits, np.uint8)
    assert ab.shape == (K,)
    q = np.empty((M, K), np.int32)
    s = np.zeros(2, np.float32)
    sb = np.zeros(2, np.uint8)
    so = np.empty(K, np.uint8)
    S = lib().orc_quantize_act(_p(A), M, K, K, _p(ab), 1 if a_signed else 0,
                               _p(q), _p(s), _p(sb), _p(so))
    if S < 0:
        raise ValueError("activation widths must be 1..8 with at most two distinct values")
    return q, s[:S].copy(), sb[:S].copy(), so


def quantize_act_grouped(A, a_bits, a_signed: bool, group_bits: int):
    """Sub-group scales: each precision group cut into blocks of
    group_bits / container channels in the Alg. 1 order, one scale per
    block.  Returns codes, scales[S], block widths[S], block of each
    channel[K] (group_bits = 0: one block per precision group)."""
    A = _c(A, np.float32)
    M, K = A.shape
    ab = _c(a_bits, np.uint8)
    assert ab.shape == (K,)
    cap = K + 2
    q = np.empty((M, K), np.int32)
    s = np.zeros(cap, np.float32)
    sb = np.zeros(cap, np.uint8)
    so = np.empty(K, np.int32)
    S = lib().orc_quantize_act_grouped(_p(A), M, K, K, _p(ab), 1 if a_signed else 0,
                                       int(group_bits), cap, _p(q), _p(s), _p(sb), _p(so))
    if S < 0:
        raise ValueError("bad widths or group size")
    return q, s[:S].copy(), sb[:S].copy(), so


def mac(q_a, q_w, seg_of, S: int):
    """ACC[g][m][n] as int32 (g = the scale group of each channel, seg_of);
    raises if a sum leaves int32."""
    q_a = _c(q_a, np.int32)
    q_w = _c(q_w, np.int32)
    so = _c(seg_of, np.int32)
    M, K = q_a.shape
    N = q_w.shape[0]
    acc = np.empty((S, M, N), np.int32)
    rc = lib().orc_mac(_p(q_a), _p(q_w), _p(so), M, N, K, S, _p(acc))
    if rc != 0:
        raise OverflowError("accumulator leaves int32")
    return acc


def mac_at(q_a, q_w, seg_of, S: int, ms, ns):
    """ACC[g] at sampled (m, n) pairs -> int64 [count, S]."""
    q_a = _c(q_a, np.int32)
    q_w = _c(q_w, np.int32)
    so = _c(seg_of, np.int32)
    ms = _c(ms, np.int64)
    ns = _c(ns, np.int64)
    out = np.empty((ms.shape[0], S), np.int64)
    lib().orc_mac_at(_p(q_a), _p(q_w), _p(so), q_a.shape[1], S, ms.shape[0],
                     _p(ms), _p(ns), _p(out))
    return out


def bf16_from_f64(v: float) -> int:
    return int(lib().orc_bf16_from_f64(float(v)))


def bf16_from_f32(v: float) -> int:
    return int(lib().orc_bf16_from_f32(np.float32(v)))


def epilogue_ref(acc, s_a, s_w):
    """bf16 bits (uint16) of s_w[n] * sum_g s_a[g] * ACC[g][m][n], fp64 math."""
    acc = _c(acc, np.int32)
    S, M, N = acc.shape
    sa = _c(s_a, np.float32)
    sw = _c(s_w, np.float32)
    y = np.empty((M, N), np.uint16)
    lib().orc_epilogue_ref(_p(acc), _p(sa), _p(sw), M, N, S, _p(y))
    return y


def epilogue_replay(acc, s_a, s_w):
    """bf16 bits of the same value evaluated in the fixed fp32 order."""
    acc = _c(acc, np.int32)
    S, M, N = acc.shape
    sa = _c(s_a, np.float32)
    sw = _c(s_w, np.float32)
    y = np.empty((M, N), np.uint16)
    lib().orc_epilogue_replay(_p(acc), _p(sa), _p(sw), M, N, S, _p(y))
    return y


def epilogue_replay_f32(acc, s_a, s_w):
    """The fixed-order fp32 epilogue value before its bf16 rounding."""
    acc = _c(acc, np.int32)
    S, M, N = acc.shape
    sa = _c(s_a, np.float32)
    sw = _c(s_w, np.float32)
    y = np.empty((M, N), np.float32)
    lib().orc_epilogue_replay_f32(_p(acc), _p(sa), _p(sw), M, N, S, _p(y))
    return y


def quantize_act_static(A, a_bits, a_signed: bool, s_a):
    """Codes of A[M,K] with the caller's group scales (one per precision
    group, narrow width first) instead of the batch maximum."""
    A = _c(A, np.float32)
    M, K = A.shape
    ab = _c(a_bits, np.uint8)
    sa = _c(s_a, np.float32)
    q = np.empty((M, K), np.int32)
    S = lib().orc_quantize_act_static(_p(A), M, K, K, _p(ab), 1 if a_signed else 0, _p(sa), _p(q))
    if S < 0 or sa.shape[0] < S:
        raise ValueError("bad widths or too few scales")
    return q


def quantize_act_static_grouped(A, a_bits, a_signed: bool, group_bits: int, s_blocks):
    """Codes of A[M,K] with the caller's scale per sub-group block (the
    blocks of quantize_act_grouped).  Returns codes and the block of each
    channel."""
    A = _c(A, np.float32)
    M, K = A.shape
    ab = _c(a_bits, np.uint8)
    sb = _c(s_blocks, np.float32)
    q = np.empty((M, K), np.int32)
    so = np.empty(K, np.int32)
    S = lib().orc_quantize_act_static_grouped(_p(A), M, K, K, _p(ab), 1 if a_signed else 0,
                                              int(group_bits), K + 2, _p(sb), _p(q), _p(so))
    if S < 0 or sb.shape[0] < S:
        raise ValueError("bad widths or group size, or too few scales")
    return q, so


def container(bits: int) -> int:
    return int(lib().orc_container(bits))


def pack(codes, bits: int, mode: int):
    c = _c(codes, np.int32).ravel()
    per = 32 // container(bits)
    words = np.empty(((c.shape[0] + per - 1) // per,), np.uint32)
    lib().orc_pack(_p(c), c.shape[0], bits, mode, _p(words))
    return words


def unpack(words, n: int, bits: int, mode: int):
    w = _c(words, np.uint32)
    out = np.empty((n,), np.int32)
    lib().orc_unpack(_p(w), n, bits, mode, _p(out))
    return out


def bf16_to_f32(y_bits):
    """Widen bf16 bit patterns (uint16) to float32 values."""
    return (np.asarray(y_bits, np.uint16).astype(np.uint32) << 16).view(np.float32)


def run(A, W, a_bits, w_bits, a_signed: bool, wmode: int = SIGNED):
    """The whole path on the CPU: codes, scales, ACC and both epilogues."""
    q_w, s_w = quantize_weights(W, w_bits, wmode)
    q_a, s_a, seg_bits, seg_of = quantize_act(A, a_bits, a_signed)
    S = len(seg_bits)
    acc = mac(q_a, q_w, seg_of, S)
    return dict(q_w=q_w, s_w=s_w, q_a=q_a, s_a=s_a, seg_bits=seg_bits,
                seg_of=seg_of, S=S, acc=acc,
                y_ref=epilogue_ref(acc, s_a, s_w),
                y_replay=epilogue_replay(acc, s_a, s_w))
