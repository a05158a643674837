"""GPU parity of soniq_quantize_mp_gemm (quantize + GEMM in one call; a batch
of one row is quantized inside the GEMV launch): against the oracle, and bit
for bit against the two calls it stands for, including the packed row and
scales it leaves in the handle."""
import numpy as np
import pytest
import torch

import paper_2311_14114_amd as sq
import workloads
from test_gpu_parity import _bf16_bits, compare_full, oracle_run

pytestmark = pytest.mark.gpu


def run_fused(case, act=None, w=None):
    M, N = case["M"], case["N"]
    print(f"[gpu] fused {case['name']} M={M} N={N} K={case['K']}", flush=True)
    if w is None:
        w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                                  case["a_signed"])
    if act is None:
        act = sq.soniq_act_create(w, M)
    A = torch.from_numpy(case["A"]).cuda()
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
    Y = sq.soniq_quantize_mp_gemm(act, w, A, acc=acc)
    torch.cuda.synchronize()
    out = dict(S=w.S, y=_bf16_bits(Y), acc=acc.cpu().numpy(), w=w, act=act)
    out["q_w"], out["s_w"] = sq.soniq_weights_unpack_debug(w)
    out["q_a"], out["s_a"] = sq.soniq_act_unpack_debug(act)
    return out


def two_calls(case, w):
    act = sq.soniq_act_create(w, case["M"])
    sq.soniq_quantize_act(act, torch.from_numpy(case["A"]).cuda())
    acc = torch.empty((w.S, case["M"], case["N"]), dtype=torch.int32, device="cuda")
    Y = sq.soniq_mp_gemm(act, w, acc=acc)
    torch.cuda.synchronize()
    q_a, s_a = sq.soniq_act_unpack_debug(act)
    return _bf16_bits(Y), acc.cpu().numpy(), q_a, s_a


def G(M, N, K, alo, ahi, af, wlo, whi, wf, signed, seed, name):
    return workloads.generic(M, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=af, w_lo=wlo, w_hi=whi,
                             w_frac_lo=wf, a_signed=signed, a_abs=not signed, seed=seed, name=name)


CASES = [
    ("decode_11008_m1", lambda: workloads.make("decode_11008_m1")),
    ("decode_4096_m1", lambda: workloads.make("decode_4096_m1")),
    ("signed_2_4", lambda: G(1, 256, 256, 4, 8, 0.5, 2, 4, 0.75, True, 1, "signed_2_4")),
    ("unsigned_1bit_w", lambda: G(1, 200, 1000, 4, 8, 0.6, 1, 4, 0.8, False, 2, "unsigned_1bit_w")),
    ("byte_blocks", lambda: G(1, 64, 2048, 4, 8, 0.7, 4, 8, 0.5, True, 3, "byte_blocks")),
    ("one_group", lambda: G(1, 48, 4096, 4, 8, 1.0, 2, 4, 0.5, False, 4, "one_group")),
    # fall back to the two calls
    ("two_bit_acts", lambda: G(1, 64, 320, 2, 8, 0.5, 2, 4, 0.5, False, 5, "two_bit_acts")),
    ("k_not_mult4", lambda: G(1, 40, 258, 4, 8, 0.5, 2, 4, 0.5, True, 6, "k_not_mult4")),
    ("k_over_4096", lambda: G(1, 32, 4608, 4, 8, 0.5, 2, 4, 0.5, True, 7, "k_over_4096")),
    ("batch_of_3", lambda: G(3, 96, 512, 4, 8, 0.5, 2, 4, 0.5, True, 8, "batch_of_3")),
]


@pytest.mark.parametrize("name,make", CASES, ids=[c[0] for c in CASES])
def test_fused_parity(name, make):
    case = make()
    g = run_fused(case)
    compare_full(g, oracle_run(case))
    y2, acc2, q2, s2 = two_calls(case, g["w"])
    np.testing.assert_array_equal(g["y"], y2)
    np.testing.assert_array_equal(g["acc"], acc2)
    np.testing.assert_array_equal(g["q_a"], q2)
    np.testing.assert_array_equal(g["s_a"], s2)


def test_fused_repeat_calls():
    """Two rows through one handle in a row, each matching the oracle."""
    a = workloads.make("decode_4096_m1")
    b = dict(a)
    b["A"] = np.ascontiguousarray(a["A"] * np.float32(-0.5) + np.float32(0.25))
    w = sq.soniq_pack_weights(torch.from_numpy(a["W"]).cuda(), a["w_bits"], a["a_bits"], a["a_signed"])
    act = sq.soniq_act_create(w, 1)
    for case in (a, b, a):
        compare_full(run_fused(case, act=act, w=w), oracle_run(case))


def test_fused_many_calls_one_handle():
    """Successive one-row calls through one handle, each on new data, equal
    the two calls they stand for (packed row, image and scales included)."""
    case = G(1, 512, 2048, 4, 8, 0.7, 2, 4, 0.6, True, 9, "fused_seq")
    w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                              True)
    act = sq.soniq_act_create(w, 1)
    rng = np.random.default_rng(9)
    for i in range(24):
        c = dict(case)
        c["A"] = np.ascontiguousarray(case["A"] * np.float32(rng.uniform(-3, 3)) +
                                      rng.standard_normal(case["A"].shape).astype(np.float32))
        c["name"] = f"fused_seq_{i}"
        g = run_fused(c, act=act, w=w)
        y2, acc2, q2, s2 = two_calls(c, w)
        np.testing.assert_array_equal(g["acc"], acc2, err_msg=f"call {i}")
        np.testing.assert_array_equal(g["y"], y2, err_msg=f"call {i}")
        np.testing.assert_array_equal(g["q_a"], q2, err_msg=f"call {i}")
        np.testing.assert_array_equal(g["s_a"], s2, err_msg=f"call {i}")


def test_fused_graph_replay():
    """The one-launch call captured in a HIP graph and replayed on new rows,
    with eager work between the replays, equals eager calls bit for bit."""
    case = workloads.make("decode_11008_m1")
    N = case["N"]
    w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                              case["a_signed"])
    act_g = sq.soniq_act_create(w, 1)
    act_e = sq.soniq_act_create(w, 1)
    A0 = torch.from_numpy(case["A"]).cuda()
    inputs = [A0 * s for s in (1.0, -0.5, 3.0, 1.0, 0.01)]
    A_buf = inputs[0].clone()
    Yg = torch.empty((1, N), dtype=torch.bfloat16, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        sq.soniq_quantize_mp_gemm(act_g, w, A_buf, out=Yg)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        sq.soniq_quantize_mp_gemm(act_g, w, A_buf, out=Yg)
    torch.cuda.synchronize()
    for r, A in enumerate(inputs):
        A_buf.copy_(A)
        Yg.zero_()
        g.replay()
        torch.cuda.synchronize()
        Ye = sq.soniq_quantize_mp_gemm(act_e, w, A)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bf16_bits(Yg), _bf16_bits(Ye), err_msg=f"replay {r}")
        # the handle keeps the row the replay quantized
        q_g, s_g = sq.soniq_act_unpack_debug(act_g)
        q_e, s_e = sq.soniq_act_unpack_debug(act_e)
        np.testing.assert_array_equal(q_g, q_e, err_msg=f"replay {r} codes")
        np.testing.assert_array_equal(s_g, s_e, err_msg=f"replay {r} scales")
