"""GPU parity of the MFMA-native fp4/fp6 copies (SONIQ_WPACK_F8F6F4): tiles
of narrow weights (1/2/4-bit containers) against narrow activation groups
(2/4-bit containers) run on v_mfma_scale_f32_16x16x128_f8f6f4 with the
codes in e2m1 / e3m2, where every stored code is exact; the int32
accumulators and the outputs must still equal the oracle's integer MAC
(Alg. 1 Phase II) and fixed-order epilogue bit for bit, and equal the
integer path of the same weights."""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def run(case, f8f6f4, wq_mode=0, sign_nibbles=False):
    M, N, K = case["M"], case["N"], case["K"]
    w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                              case["a_signed"], wq_mode, sign_nibbles=sign_nibbles, f8f6f4=f8f6f4)
    assert w.info.f8f6f4 == int(f8f6f4)
    act = sq.soniq_act_create(w, M)
    sq.soniq_quantize_act(act, torch.from_numpy(case["A"]).cuda())
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
    Y = sq.soniq_mp_gemm(act, w, acc=acc)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), _bits(Y)


def check(case, wq_mode=0, sign_nibbles=False):
    print(f"[gpu] f8f6f4 {case['name']} M={case['M']} N={case['N']} K={case['K']}", flush=True)
    acc, y = run(case, True, wq_mode, sign_nibbles)
    mode = oracle.TWOS_FRACTION if wq_mode == 1 else oracle.SIGNED
    r = oracle.run(case["A"], case["W"], case["a_bits"], case["w_bits"], case["a_signed"], mode)
    np.testing.assert_array_equal(acc, r["acc"])
    np.testing.assert_array_equal(y, r["y_replay"])
    acc_i, y_i = run(case, False, wq_mode, sign_nibbles)
    np.testing.assert_array_equal(acc, acc_i)
    np.testing.assert_array_equal(y, y_i)


@pytest.mark.parametrize("name", ["tiny_linear", "xfmr_qkv", "xfmr_ffn_up", "xfmr_ffn_down",
                                  "conv3x3_im2col"])
def test_workloads(name):
    case = workloads.make(name)
    check(case, sign_nibbles=name == "conv3x3_im2col")


def test_conv_sign_bits():
    """1-bit weights kept as sign bits (not nibbles) also map to fp4 +-1."""
    check(workloads.make("conv3x3_im2col"))


def test_decode_weights_at_a_prefill_batch():
    """The decode layer's weights (W[11008, 4096], 2/4-bit) at a batch of 128
    rows, which runs the MFMA tiles (batches of 8 or fewer run the GEMV)."""
    case = workloads.generic(128, 11008, 4096, a_lo=4, a_hi=8, a_frac_lo=0.8, w_lo=2, w_hi=4,
                             w_frac_lo=0.75, a_signed=True, seed=4141, name="decode_weights_m128")
    check(case)


def test_square_8192():
    """The 8192^3 case (4/8-bit both sides: its 4-bit x 4-bit tiles run in
    fp6 x fp6), every accumulator and output."""
    check(workloads.square_8192())


EDGE = [  # (M, N, K, a_lo, a_hi, w_lo, w_hi, a_signed, wq_mode)
    (64, 256, 192, 4, 8, 2, 8, True, 0),      # 3 granules: a half fgranule at the end
    (130, 300, 65, 4, 8, 2, 4, True, 0),      # one granule per group, ragged rows
    (200, 128, 1000, 2, 8, 2, 8, False, 0),   # unsigned 2-bit activations (fp4)
    (100, 200, 500, 4, 8, 2, 4, True, 1),     # two's-fraction grid: codes -8 and -2
    (96, 250, 700, 4, 4, 4, 4, True, 0),      # one width each side (tiles past the class)
    (257, 129, 300, 3, 6, 1, 3, False, 0),    # 3-bit in 4-bit containers, sign weights
]


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s[:3])) + f"_a{s[3]}{s[4]}w{s[5]}{s[6]}m{s[8]}")
def test_edges(shape):
    M, N, K, alo, ahi, wlo, whi, sgn, mode = shape
    case = workloads.generic(M, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.6, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.6, a_signed=sgn, a_abs=not sgn, seed=M + N + K,
                             name="f8f6f4_edge")
    check(case, wq_mode=mode)


def test_scratch_entry_with_copies():
    """The allocation-free entry point on weights with the copies."""
    case = workloads.make("xfmr_qkv")
    w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                              True, f8f6f4=True)
    A = torch.from_numpy(case["A"]).cuda()
    Ys = sq.soniq_quantize_mp_gemm_scratch(w, A)
    r = oracle.run(case["A"], case["W"], case["a_bits"], case["w_bits"], True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bits(Ys), r["y_replay"])
