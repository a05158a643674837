"""GPU parity of the implicit-GEMM 3x3 convolution (soniq_pack_weights_conv3x3,
soniq_act_create_conv3x3): the input is quantized once into a haloed code
image and the GEMM gathers each tap's units from it, with no lowered matrix
anywhere.  Against the oracle on the lowered matrix im2col_3x3(X): codes
(read back as the lowered matrix's), scales and every int32 accumulator
bit-exact, bf16 outputs equal to the fixed-order replay, and the same bits
as the lowered path of the same layer."""
import numpy as np
import pytest
import torch

import paper_2311_14114_amd as sq
import workloads
from test_gpu_parity import _bf16_bits, compare_full, oracle_run

pytestmark = pytest.mark.gpu


def gpu_run_implicit(case, sign_nibbles=False):
    X = torch.from_numpy(case["X"]).cuda()
    B, C, H, W = case["X"].shape
    M, N = case["M"], case["N"]
    print(f"[gpu] implicit {case['name']} X={tuple(X.shape)} N={N} signed={case['a_signed']}",
          flush=True)
    Wf = torch.from_numpy(np.ascontiguousarray(case["W"].reshape(N, C, 3, 3))).cuda()
    ch_bits = case["a_bits"][::9]
    w = sq.soniq_pack_weights_conv3x3(Wf, case["w_bits"], ch_bits, case["a_signed"],
                                      sign_nibbles=sign_nibbles)
    act = sq.soniq_act_create_conv3x3(w, B, H, W)
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
    # (B, C, H, W, N, a_lo, a_hi, a_frac_lo, w_lo, w_hi, a_signed, sign_nibbles)
    (1, 2, 1, 1, 16, 4, 8, 0.5, 2, 4, False, False),   # one pixel: every tap but the centre is halo
    (2, 16, 5, 7, 32, 4, 8, 0.6, 1, 4, False, False),  # ragged 16-row blocks (M = 70), sign bits
    (2, 16, 5, 7, 32, 4, 8, 0.6, 1, 4, False, True),   # sign weights in nibbles
    (2, 20, 5, 7, 40, 4, 8, 0.6, 2, 8, True, False),   # signed codes
    (1, 7, 3, 20, 20, 3, 6, 0.4, 2, 4, False, False),  # 3/6-bit in 4/8-bit containers, no zero point
    (4, 64, 8, 8, 128, 4, 8, 0.6, 4, 8, False, False), # several blocks per image
    (2, 33, 6, 9, 130, 4, 8, 0.5, 4, 4, True, False),  # odd channel counts, N past a tile
    (2, 3, 1, 70, 8, 4, 8, 0.5, 2, 4, False, False),   # one image row wider than a wave
    # the other weight container pairs
    (2, 16, 5, 7, 48, 4, 8, 0.6, 5, 8, False, False),  # 8/8: two widths in one container
    (2, 16, 5, 7, 40, 4, 8, 0.6, 1, 7, True, False),   # 1/8
    (1, 24, 6, 6, 33, 3, 6, 0.5, 2, 2, False, False),  # 2/2: one width
    (2, 16, 4, 5, 40, 4, 8, 0.6, 1, 2, True, False),   # 1/2
    (1, 16, 5, 5, 20, 4, 8, 0.6, 1, 1, False, False),  # 1/1: sign weights only
    # one activation width (S = 1)
    (2, 16, 5, 7, 32, 8, 8, 0.6, 1, 4, False, False),  # 8-bit activations only
    (2, 12, 4, 6, 40, 3, 3, 0.6, 2, 8, True, False),   # 3-bit signed activations only
]


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: "x".join(map(str, s[:5])) + ("s" if s[10] else "u") + ("n" if s[11] else ""))
def test_implicit_conv_small(spec):
    B, C, H, W, N, alo, ahi, af, wlo, whi, sgn, nib = spec
    case = workloads.conv3x3(B, C, H, W, N, a_lo=alo, a_hi=ahi, a_frac_lo=af, w_lo=wlo, w_hi=whi,
                             a_signed=sgn, seed=B * 1000 + C + 7)
    compare_full(gpu_run_implicit(case, sign_nibbles=nib), oracle_run(case))


@pytest.mark.parametrize("nibbles", [False, True])
def test_implicit_conv_workload(nibbles):
    """The CNN workload (32 x 256 x 14 x 14 -> 256, unsigned 4/8-bit, 1/4-bit
    weights) in full: codes, scales, accumulators and outputs."""
    case = workloads.make("conv3x3_im2col")
    g = gpu_run_implicit(case, sign_nibbles=nibbles)
    compare_full(g, oracle_run(case))


def test_implicit_conv_smaller_batch_and_errors():
    """A second call with fewer images into the same handle; entry points
    that need a lowered matrix refuse the handle."""
    case = workloads.conv3x3(3, 24, 6, 6, 48, seed=99)
    B, C, H, W = case["X"].shape
    Wf = torch.from_numpy(np.ascontiguousarray(case["W"].reshape(48, C, 3, 3))).cuda()
    w = sq.soniq_pack_weights_conv3x3(Wf, case["w_bits"], case["a_bits"][::9], False)
    act = sq.soniq_act_create_conv3x3(w, B, H, W)
    small = workloads.conv3x3(1, 24, 6, 6, 48, seed=99)
    small["W"], small["w_bits"], small["a_bits"] = case["W"], case["w_bits"], case["a_bits"]
    X1 = torch.from_numpy(small["X"]).cuda()
    sq.soniq_quantize_act_conv3x3(act, torch.from_numpy(case["X"]).cuda())
    sq.soniq_quantize_act_conv3x3(act, X1)
    acc = torch.empty((w.S, small["M"], 48), dtype=torch.int32, device="cuda")
    Y = sq.soniq_mp_gemm(act, w, acc=acc)
    torch.cuda.synchronize()
    r = oracle_run(small)
    np.testing.assert_array_equal(acc.cpu().numpy(), r["acc"])
    np.testing.assert_array_equal(_bf16_bits(Y), r["y_replay"])
    with pytest.raises(sq.SoniqError):
        sq.soniq_quantize_act(act, torch.zeros((36, 9 * C), dtype=torch.float32, device="cuda"))
    with pytest.raises(sq.SoniqError):
        sq.soniq_act_create(w, 10)
    with pytest.raises(sq.SoniqError):   # other image size
        sq.soniq_quantize_act_conv3x3(act, torch.zeros((1, C, 7, 6), dtype=torch.float32, device="cuda"))
