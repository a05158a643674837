"""GPU parity of the 3x3 convolution entry point (soniq_quantize_act_conv3x3):
activations quantized straight from the input tensor X, then the usual
integer GEMM, against the oracle run on the lowered matrix im2col_3x3(X).

Same bar as the other parity tests: codes, scales and int32 accumulators
bit-exact, bf16 outputs equal to the fixed-order fp32 replay.
"""
import numpy as np
import pytest
import torch

import paper_2311_14114_amd as sq
import workloads
from test_gpu_parity import _bf16_bits, compare_full, oracle_run

pytestmark = pytest.mark.gpu


def gpu_run_conv(case, act=None, w=None):
    X = torch.from_numpy(case["X"]).cuda()
    B, C, H, W = case["X"].shape
    M, N = case["M"], case["N"]
    print(f"[gpu] {case['name']} X={tuple(X.shape)} N={N} signed={case['a_signed']}", flush=True)
    if w is None:
        w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                                  case["a_signed"])
    if act is None:
        act = sq.soniq_act_create(w, M)
    sq.soniq_quantize_act_conv3x3(act, X)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
    sq.soniq_mp_gemm(act, w, out=Y, acc=acc)
    torch.cuda.synchronize()
    out = dict(S=w.S, y=_bf16_bits(Y), acc=acc.cpu().numpy(), w=w, act=act)
    out["q_w"], out["s_w"] = sq.soniq_weights_unpack_debug(w)
    out["q_a"], out["s_a"] = sq.soniq_act_unpack_debug(act)
    return out


SMALL = [
    # (B, C, H, W, N, a_lo, a_hi, a_frac_lo, w_lo, w_hi, a_signed)
    (1, 1, 1, 1, 16, 4, 8, 1.0, 2, 4, False),     # one pixel, one channel, one group
    (2, 16, 5, 7, 32, 4, 8, 0.6, 1, 4, False),    # ragged 16-row blocks (M = 70)
    (2, 16, 5, 7, 32, 4, 8, 0.6, 2, 8, True),     # signed codes
    (3, 40, 9, 6, 48, 2, 8, 0.5, 4, 8, False),    # 2-bit group (zero point 2)
    (1, 7, 3, 20, 20, 3, 6, 0.4, 1, 4, False),    # widths in wider containers, no zero point
    (2, 12, 4, 4, 24, 1, 8, 0.5, 2, 4, True),     # 1-bit sign group: generic quantizer
    (4, 64, 8, 8, 128, 4, 8, 0.6, 1, 4, False),   # several blocks per image
    (2, 3, 1, 70, 8, 4, 8, 0.5, 2, 4, False),     # one image row wider than a wave
]


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: "x".join(map(str, s[:5])) + ("s" if s[-1] else "u"))
def test_conv_parity_small(spec):
    B, C, H, W, N, alo, ahi, af, wlo, whi, sgn = spec
    case = workloads.conv3x3(B, C, H, W, N, a_lo=alo, a_hi=ahi, a_frac_lo=af, w_lo=wlo, w_hi=whi,
                             a_signed=sgn, seed=B * 1000 + C)
    compare_full(gpu_run_conv(case), oracle_run(case))


def test_conv_parity_full_resnet_layer():
    """The 256 -> 256 3x3 layer at 14x14, batch 32 (M = 6272, K = 2304)."""
    case = workloads.make("conv3x3_im2col")
    compare_full(gpu_run_conv(case), oracle_run(case))


def test_conv_matches_the_lowered_path_and_repeats():
    """Two calls in a row on one handle (the second with new values and a
    smaller batch) each give the codes the lowered-matrix entry point gives."""
    big = workloads.conv3x3(3, 24, 6, 6, 32, seed=7)
    small = workloads.conv3x3(1, 24, 6, 6, 32, seed=8)
    small["W"], small["w_bits"], small["a_bits"] = big["W"], big["w_bits"], big["a_bits"]
    w = sq.soniq_pack_weights(torch.from_numpy(big["W"]).cuda(), big["w_bits"], big["a_bits"], False)
    act = sq.soniq_act_create(w, big["M"])
    ref = sq.soniq_act_create(w, big["M"])
    for case in (big, small):
        g = gpu_run_conv(case, act=act, w=w)
        sq.soniq_quantize_act(ref, torch.from_numpy(case["A"]).cuda())
        torch.cuda.synchronize()
        q_ref, s_ref = sq.soniq_act_unpack_debug(ref)
        np.testing.assert_array_equal(g["q_a"], q_ref)
        np.testing.assert_array_equal(g["s_a"], s_ref)
        compare_full(g, oracle_run(case))


def test_conv_rejects_bad_shapes():
    case = workloads.conv3x3(1, 8, 4, 4, 16, seed=2)
    w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"], False)
    act = sq.soniq_act_create(w, case["M"])
    X = torch.from_numpy(case["X"]).cuda()
    with pytest.raises(sq.SoniqError) as e:
        sq.soniq_quantize_act_conv3x3(act, X[:, :7].contiguous())   # 9*C != K
    assert e.value.status == sq.SONIQ_ERR_INVALID_ARGUMENT
    with pytest.raises(sq.SoniqError) as e:
        sq.soniq_quantize_act_conv3x3(act, torch.cat([X, X]))        # B*H*W > max_M
    assert e.value.status == sq.SONIQ_ERR_INVALID_ARGUMENT
    # the taps of one channel at different widths
    ab = case["a_bits"].copy()
    ab[1] = 8 if ab[0] == 4 else 4
    w2 = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], ab, False)
    act2 = sq.soniq_act_create(w2, case["M"])
    with pytest.raises(sq.SoniqError) as e:
        sq.soniq_quantize_act_conv3x3(act2, X)
    assert e.value.status == sq.SONIQ_ERR_UNSUPPORTED
