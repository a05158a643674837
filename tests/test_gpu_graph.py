"""HIP graph replay of the hot path (quantize_act + mp_gemm, as bench.py
times it): every replay, with eager work and synchronizations between the
replays, equals an eager run on the same data bit for bit."""
import numpy as np
import pytest
import torch

import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy()


@pytest.mark.parametrize("name", ["conv3x3_im2col", "xfmr_qkv", "tiny_linear", "decode_4096_m1",
                                  "decode_11008_m8"])
def test_graph_replay_matches_eager(name):
    case = workloads.make(name)
    M, N = case["M"], case["N"]
    print(f"[gpu] graph replay {name} M={M} N={N} K={case['K']}", flush=True)
    W = torch.from_numpy(case["W"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], case["a_signed"])
    act_g = sq.soniq_act_create(w, M)
    act_e = sq.soniq_act_create(w, M)
    A0 = torch.from_numpy(case["A"]).cuda()
    # inputs of the replays: the workload's activations at several scales
    # (signs kept, so unsigned groups stay non-negative)
    inputs = [A0 * s for s in (1.0, 0.37, 2.5, 1.0)]
    A_buf = inputs[0].clone()
    Yg = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")

    # one eager call on the capture stream, then the capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        sq.soniq_quantize_act(act_g, A_buf)
        sq.soniq_mp_gemm(act_g, w, out=Yg)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        sq.soniq_quantize_act(act_g, A_buf)
        sq.soniq_mp_gemm(act_g, w, out=Yg)
    torch.cuda.synchronize()

    for r, A in enumerate(inputs):
        A_buf.copy_(A)           # eager work between replays
        Yg.zero_()
        g.replay()
        torch.cuda.synchronize()
        sq.soniq_quantize_act(act_e, A)
        Ye = sq.soniq_mp_gemm(act_e, w)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bits(Yg), _bits(Ye), err_msg=f"replay {r}")
        _, s_g = sq.soniq_act_unpack_debug(act_g)
        _, s_e = sq.soniq_act_unpack_debug(act_e)
        np.testing.assert_array_equal(s_g, s_e, err_msg=f"replay {r} scales")
