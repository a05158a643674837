"""Seeded synthetic inputs shaped like SONIQ's CNN and Transformer workloads.

This module only draws random numbers and lays them out (including the
im2col lowering of a 3x3 convolution).  It holds none of the method's
arithmetic: no scales, codes, packing or products.  Both the oracle side
(tests, CPU baseline) and the GPU side (tests, benchmark) take their inputs
from here, so both see identical bytes.

Every case is a dict with
  A        float32 [M, K]   activations (row-major)
  W        float32 [N, K]   weights, output channel n is row n
  a_bits   uint8   [K]      per-input-channel width (two levels)
  w_bits   uint8   [N]      per-output-channel width (two levels)
  a_signed bool             False = unsigned activation codec
  name, seed and shape metadata.

Draw order inside one case: activations, weights, activation-precision
split, weight-precision split.  A split picks the low-width channel set as
``rng.permutation(C)[:round(frac * C)]``; channels are never pre-sorted, so
every case exercises the precision-group permutation.
"""
from __future__ import annotations

import numpy as np

BASE_SEED = 231114114

# name -> (seed id, description)
CONFIGS = {
    "tiny_linear": 1,
    "conv3x3_im2col": 2,
    "xfmr_qkv": 31,
    "xfmr_ffn_up": 32,
    "xfmr_ffn_down": 33,
    "decode_11008_m1": 41,
    "decode_4096_m1": 42,
    "decode_11008_m8": 43,
    "decode_4096_m8": 44,
    "decode_11008_m1_w36": 45,
    "decode_11008_m8_w36": 46,
    "decode_11008_m1_sign": 47,
    "square_8192": 5,
}


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _split(rng: np.random.Generator, C: int, frac_lo: float, lo: int, hi: int) -> np.ndarray:
    """Per-channel widths: round(frac_lo*C) seeded channels at lo, the rest at hi."""
    bits = np.full(C, hi, np.uint8)
    n_lo = int(round(frac_lo * C))
    bits[rng.permutation(C)[:n_lo]] = lo
    return bits


def generic(M: int, N: int, K: int, *, a_lo: int, a_hi: int, a_frac_lo: float,
            w_lo: int, w_hi: int, w_frac_lo: float, a_signed: bool = True,
            a_std: float = 1.0, w_std: float = 0.02, seed: int = 0,
            a_abs: bool = False, name: str = "generic") -> dict:
    """A ~ N(0, a_std) (|.| if a_abs), W ~ N(0, w_std), seeded two-level splits."""
    rng = _rng(seed)
    A = rng.standard_normal((M, K), dtype=np.float32) * np.float32(a_std)
    if a_abs:
        A = np.abs(A)
    W = rng.standard_normal((N, K), dtype=np.float32) * np.float32(w_std)
    a_bits = _split(rng, K, a_frac_lo, a_lo, a_hi)
    w_bits = _split(rng, N, w_frac_lo, w_lo, w_hi)
    return dict(name=name, seed=seed, M=M, N=N, K=K, A=A, W=W, a_bits=a_bits,
                w_bits=w_bits, a_signed=a_signed)


def im2col_3x3(X: np.ndarray) -> np.ndarray:
    """Stride-1, pad-1 3x3 lowering of X[B,C,H,W] to [B*H*W, C*9].

    Row index b*H*W + oh*W + ow; column index c*9 + kh*3 + kw (the order of
    torch.nn.functional.unfold).  Border taps read the zero padding.
    """
    B, C, H, Wd = X.shape
    Xp = np.pad(X, ((0, 0), (0, 0), (1, 1), (1, 1)))
    win = np.lib.stride_tricks.sliding_window_view(Xp, (3, 3), axis=(2, 3))
    # win: [B, C, H, W, 3, 3] -> [B, H, W, C, 3, 3]
    return np.ascontiguousarray(win.transpose(0, 2, 3, 1, 4, 5)).reshape(B * H * Wd, C * 9)


def tiny_linear() -> dict:
    """Single linear layer: A[64,256] ~N(0,1), 50% of K at 4b signed, rest 8b;
    W[256,256] ~N(0,0.02), 75% of N at 2b, rest 4b."""
    return generic(64, 256, 256, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=4,
                   w_frac_lo=0.75, seed=BASE_SEED + 1, name="tiny_linear")


def conv3x3_im2col(batch: int = 32, channels: int = 256, hw: int = 14) -> dict:
    """ResNet-18-like 3x3 conv 256->256 at 14x14, batch 32, as an im2col GEMM
    (M = 6272, K = 2304, N = 256).  Post-ReLU activations |N(0,1)|, unsigned,
    60% of input channels at 4b and 40% at 8b (all 9 taps of a channel share
    its width); weights ~N(0,0.05), 80% of output channels 1-bit, 20% 4-bit."""
    rng = _rng(BASE_SEED + 2)
    X = np.abs(rng.standard_normal((batch, channels, hw, hw), dtype=np.float32))
    Wt = rng.standard_normal((channels, channels, 3, 3), dtype=np.float32) * np.float32(0.05)
    ch_bits = _split(rng, channels, 0.6, 4, 8)
    w_bits = _split(rng, channels, 0.8, 1, 4)
    A = im2col_3x3(X)
    W = np.ascontiguousarray(Wt.reshape(channels, channels * 9))
    a_bits = np.repeat(ch_bits, 9)
    return dict(name="conv3x3_im2col", seed=BASE_SEED + 2, M=A.shape[0], N=channels,
                K=A.shape[1], A=A, W=W, a_bits=a_bits, w_bits=w_bits, a_signed=False, X=X)


def conv3x3(batch: int, channels: int, h: int, w: int, n_out: int, *, a_lo: int = 4,
            a_hi: int = 8, a_frac_lo: float = 0.6, w_lo: int = 1, w_hi: int = 4,
            w_frac_lo: float = 0.8, a_signed: bool = False, seed: int = 0,
            name: str = "conv3x3") -> dict:
    """A 3x3 stride-1 pad-1 convolution X[batch, channels, h, w] -> n_out
    channels, in the draw order of conv3x3_im2col: X (|N(0,1)| when unsigned,
    else N(0,1)), filters ~N(0,0.05), per-input-channel widths (shared by the
    channel's 9 taps), per-output-channel widths.  Carries X and its lowering
    A = im2col_3x3(X)."""
    rng = _rng(seed)
    X = rng.standard_normal((batch, channels, h, w), dtype=np.float32)
    if not a_signed:
        X = np.abs(X)
    Wt = rng.standard_normal((n_out, channels, 3, 3), dtype=np.float32) * np.float32(0.05)
    ch_bits = _split(rng, channels, a_frac_lo, a_lo, a_hi)
    w_bits = _split(rng, n_out, w_frac_lo, w_lo, w_hi)
    A = im2col_3x3(X)
    return dict(name=name, seed=seed, M=A.shape[0], N=n_out, K=A.shape[1], A=A,
                W=np.ascontiguousarray(Wt.reshape(n_out, channels * 9)),
                a_bits=np.repeat(ch_bits, 9), w_bits=w_bits, a_signed=a_signed, X=X)


def _xfmr(K: int, N: int, seed_id: int, name: str, M: int = 4096) -> dict:
    """Transformer encoder linear (hidden 768, FFN 3072, seq 128 x batch 32):
    A ~N(0,1) with round(1% of K) outlier channels scaled x20 held at 8b, the
    rest at 4b (signed); W ~N(0,0.02), 70% of N at 2b, 30% at 8b."""
    rng = _rng(BASE_SEED + seed_id)
    A = rng.standard_normal((M, K), dtype=np.float32)
    W = rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)
    n_out = int(round(0.01 * K))
    a_bits = np.full(K, 4, np.uint8)
    out = rng.permutation(K)[:n_out]
    a_bits[out] = 8
    A[:, out] *= np.float32(20.0)
    w_bits = _split(rng, N, 0.7, 2, 8)
    return dict(name=name, seed=BASE_SEED + seed_id, M=M, N=N, K=K, A=A, W=W,
                a_bits=a_bits, w_bits=w_bits, a_signed=True)


def xfmr_qkv() -> dict:
    return _xfmr(768, 2304, 31, "xfmr_qkv")


def xfmr_ffn_up() -> dict:
    return _xfmr(768, 3072, 32, "xfmr_ffn_up")


def xfmr_ffn_down() -> dict:
    return _xfmr(3072, 768, 33, "xfmr_ffn_down")


def _decode(N: int, M: int, seed_id: int, name: str) -> dict:
    """Decode GEMV: x[M,4096] ~N(0,1), 80% 4b / 20% 8b signed; W[N,4096]
    ~N(0,0.02), 75% 2b / 25% 4b."""
    return generic(M, N, 4096, a_lo=4, a_hi=8, a_frac_lo=0.8, w_lo=2, w_hi=4,
                   w_frac_lo=0.75, seed=BASE_SEED + seed_id, name=name)


def decode_11008_m1() -> dict:
    return _decode(11008, 1, 41, "decode_11008_m1")


def decode_4096_m1() -> dict:
    return _decode(4096, 1, 42, "decode_4096_m1")


def decode_11008_m8() -> dict:
    return _decode(11008, 8, 43, "decode_11008_m8")


def decode_4096_m8() -> dict:
    return _decode(4096, 8, 44, "decode_4096_m8")


def _decode_w36(M: int, seed_id: int, name: str) -> dict:
    """Decode GEMV with weight widths off the container sizes: x[M,4096]
    ~N(0,1), 80% 4b / 20% 8b signed; W[11008,4096] ~N(0,0.02), 75% 3b /
    25% 6b (any width from 1 to 8 bits is a valid SONIQ precision)."""
    return generic(M, 11008, 4096, a_lo=4, a_hi=8, a_frac_lo=0.8, w_lo=3, w_hi=6,
                   w_frac_lo=0.75, seed=BASE_SEED + seed_id, name=name)


def decode_11008_m1_w36() -> dict:
    return _decode_w36(1, 45, "decode_11008_m1_w36")


def decode_11008_m8_w36() -> dict:
    return _decode_w36(8, 46, "decode_11008_m8_w36")


def decode_11008_m1_sign() -> dict:
    """Decode GEMV with sign (1-bit) channels on both sides: x[1,4096]
    ~N(0,1), 75% 1b / 25% 4b signed; W[11008,4096] ~N(0,0.02), 75% 1b /
    25% 4b (the sign x sign runs are XNOR-popcount products)."""
    return generic(1, 11008, 4096, a_lo=1, a_hi=4, a_frac_lo=0.75, w_lo=1, w_hi=4,
                   w_frac_lo=0.75, seed=BASE_SEED + 47, name="decode_11008_m1_sign")


def square_8192(size: int = 8192) -> dict:
    """M = N = K = 8192, A ~N(0,1), W ~N(0,0.02), 50% 4b / 50% 8b on both
    operands with seeded interleaving."""
    return generic(size, size, size, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=4, w_hi=8,
                   w_frac_lo=0.5, seed=BASE_SEED + 5, name="square_8192")


def _grouped(base: dict, group_bits: int = 512) -> dict:
    """The same inputs with sub-group activation scales: each precision
    group cut into blocks of group_bits of storage (Sec. 5 normalizes
    transformer activations in 512-bit groups)."""
    case = dict(base)
    case["name"] = f"{base['name']}_g{group_bits}"
    case["act_group_bits"] = group_bits
    return case


def xfmr_qkv_g512() -> dict:
    return _grouped(xfmr_qkv())


def xfmr_ffn_down_g512() -> dict:
    return _grouped(xfmr_ffn_down())


def decode_11008_m1_g512() -> dict:
    return _grouped(decode_11008_m1())


def decode_11008_m8_g512() -> dict:
    return _grouped(decode_11008_m8())


BUILDERS = {
    "tiny_linear": tiny_linear,
    "conv3x3_im2col": conv3x3_im2col,
    "xfmr_qkv": xfmr_qkv,
    "xfmr_ffn_up": xfmr_ffn_up,
    "xfmr_ffn_down": xfmr_ffn_down,
    "decode_11008_m1": decode_11008_m1,
    "decode_4096_m1": decode_4096_m1,
    "decode_11008_m8": decode_11008_m8,
    "decode_4096_m8": decode_4096_m8,
    "decode_11008_m1_w36": decode_11008_m1_w36,
    "decode_11008_m8_w36": decode_11008_m8_w36,
    "decode_11008_m1_sign": decode_11008_m1_sign,
    "square_8192": square_8192,
    "xfmr_qkv_g512": xfmr_qkv_g512,
    "xfmr_ffn_down_g512": xfmr_ffn_down_g512,
    "decode_11008_m1_g512": decode_11008_m1_g512,
    "decode_11008_m8_g512": decode_11008_m8_g512,
}


def make(name: str) -> dict:
    return BUILDERS[name]()
