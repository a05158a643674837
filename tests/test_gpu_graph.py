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


def _capture(side, fn):
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        fn()
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("name", ["xfmr_qkv_g512", "grouped_small"])
def test_graph_replay_grouped(name):
    """Sub-group scales (the single pass, and the three-launch form for a
    small batch) replayed from a graph, checked against eager calls."""
    if name == "grouped_small":
        case = workloads.generic(300, 200, 1000, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                                 w_frac_lo=0.6, a_signed=True, seed=8, name=name)
        case["act_group_bits"] = 512
    else:
        case = workloads.make(name)
    M, N = case["M"], case["N"]
    print(f"[gpu] graph replay {name} M={M} N={N} K={case['K']}", flush=True)
    W = torch.from_numpy(case["W"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], case["a_signed"],
                              act_group_bits=case["act_group_bits"])
    act_g, act_e = sq.soniq_act_create(w, M), sq.soniq_act_create(w, M)
    A0 = torch.from_numpy(case["A"]).cuda()
    A_buf = A0.clone()
    Yg = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    step = lambda: sq.soniq_quantize_mp_gemm(act_g, w, A_buf, out=Yg)
    with torch.cuda.stream(side):
        step()
    torch.cuda.synchronize()
    g = _capture(side, step)
    for r, s in enumerate((1.0, 0.37, 2.5, 1.0)):
        A = A0 * s
        A_buf.copy_(A)
        Yg.zero_()
        g.replay()
        torch.cuda.synchronize()
        Ye = sq.soniq_quantize_mp_gemm(act_e, w, A)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bits(Yg), _bits(Ye), err_msg=f"replay {r}")


@pytest.mark.parametrize("gbits", [0, 512])
def test_graph_replay_quantize_next(gbits):
    """Two layers with the second's activations quantized in the first
    GEMM's epilogue, replayed from a graph, checked against eager calls
    (gbits > 0: both layers with sub-group activation scales)."""
    l1 = workloads.generic(256, 384, 256, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.6, a_signed=True, seed=3, name="l1")
    l2 = workloads.generic(256, 128, 384, a_lo=4, a_hi=8, a_frac_lo=0.7, w_lo=2, w_hi=4,
                           w_frac_lo=0.5, a_signed=True, seed=4, name="l2")
    print(f"[gpu] graph replay quantize_next gbits={gbits}", flush=True)
    w1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True,
                               act_group_bits=gbits)
    w2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], True,
                               act_group_bits=gbits)
    s2 = np.linspace(0.05, 0.2, w2.S).astype(np.float32)
    A0 = torch.from_numpy(l1["A"]).cuda()
    A_buf = A0.clone()
    a1g, a2g = sq.soniq_act_create(w1, 256), sq.soniq_act_create(w2, 256)
    a1e, a2e = sq.soniq_act_create(w1, 256), sq.soniq_act_create(w2, 256)
    Yg = torch.empty((256, 128), dtype=torch.bfloat16, device="cuda")

    def chain(a1, a2, A, Y):
        sq.soniq_quantize_act(a1, A)
        sq.soniq_mp_gemm_quantize_next(a1, w1, a2, s2)
        return sq.soniq_mp_gemm(a2, w2, out=Y)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        chain(a1g, a2g, A_buf, Yg)  # the first call prepares a2g outside the graph
    torch.cuda.synchronize()
    g = _capture(side, lambda: chain(a1g, a2g, A_buf, Yg))
    for r, s in enumerate((1.0, 0.5, 3.0, 1.0)):
        A = A0 * s
        A_buf.copy_(A)
        Yg.zero_()
        g.replay()
        torch.cuda.synchronize()
        Ye = chain(a1e, a2e, A, torch.empty_like(Yg))
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bits(Yg), _bits(Ye), err_msg=f"replay {r}")
