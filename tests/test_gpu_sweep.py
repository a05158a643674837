"""Seeded sweep of random shapes and widths through the newer paths, each
case against the oracle to the parity bar: sub-group activation scales,
1-bit weights in 4-bit containers, and the next layer quantized in the
producing GEMM's epilogue.  Sizes stay small (the oracle runs each case in
well under a second)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu

WIDTHS_SIGNED = [(2, 8), (3, 5), (4, 8), (4, 4), (8, 8), (5, 7)]
WIDTHS_W = [(1, 4), (2, 8), (1, 2), (4, 8), (2, 4), (8, 8), (1, 1), (3, 6)]


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _case(rng, seed, grouped):
    M = int(rng.choice([1, 3, 9, 17, 64, 130, 300, 700]))
    K = int(rng.integers(16, 1500))
    N = int(rng.integers(8, 400))
    a = WIDTHS_SIGNED[int(rng.integers(len(WIDTHS_SIGNED)))]
    w = WIDTHS_W[int(rng.integers(len(WIDTHS_W)))]
    signed = bool(rng.integers(2)) or not grouped
    if grouped and not signed:
        a = (3, 6)   # unsigned widths below their containers: no zero point
    case = workloads.generic(M, N, K, a_lo=a[0], a_hi=a[1], a_frac_lo=float(rng.uniform(0.2, 0.9)),
                             w_lo=w[0], w_hi=w[1], w_frac_lo=float(rng.uniform(0.2, 0.9)),
                             a_signed=signed, seed=seed, a_abs=not signed, name="sweep")
    case["A"] = (case["A"] * rng.uniform(0.1, 10.0, K).astype(np.float32)).astype(np.float32)
    return case


def _check(y, acc, q_a, s_a, r_q, r_s, r_acc, r_sw):
    np.testing.assert_array_equal(s_a, r_s)
    np.testing.assert_array_equal(q_a, r_q)
    np.testing.assert_array_equal(acc, r_acc)
    np.testing.assert_array_equal(y, oracle.epilogue_replay(r_acc, r_s, r_sw))


@pytest.mark.parametrize("seed", range(12))
def test_sweep_grouped_and_nibbles(seed):
    rng = np.random.default_rng(1000 + seed)
    grouped = seed % 2 == 0
    case = _case(rng, 2000 + seed, grouped)
    gbits = int(rng.choice([512, 1024, 2048])) if grouped else 0
    nib = not grouped
    M, N, K = case["M"], case["N"], case["K"]
    print(f"[gpu] sweep {seed} M={M} N={N} K={K} a={sorted(set(case['a_bits']))} "
          f"w={sorted(set(case['w_bits']))} signed={case['a_signed']} g={gbits} nib={nib}", flush=True)
    w = sq.soniq_pack_weights(torch.from_numpy(case["W"]).cuda(), case["w_bits"], case["a_bits"],
                              case["a_signed"], act_group_bits=gbits, sign_nibbles=nib)
    act = sq.soniq_act_create(w, M)
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
    Y = sq.soniq_quantize_mp_gemm(act, w, torch.from_numpy(case["A"]).cuda(), acc=acc)
    torch.cuda.synchronize()
    q_a, s_a = sq.soniq_act_unpack_debug(act)
    q_w, s_w = oracle.quantize_weights(case["W"], case["w_bits"])
    if grouped:
        r_q, r_s, _, r_of = oracle.quantize_act_grouped(case["A"], case["a_bits"], case["a_signed"], gbits)
    else:
        r_q, r_s, _, r_of = oracle.quantize_act(case["A"], case["a_bits"], case["a_signed"])
    r_acc = oracle.mac(r_q, q_w, r_of, len(r_s))
    _check(_bits(Y), acc.cpu().numpy(), q_a, s_a, r_q, r_s, r_acc, s_w)


@pytest.mark.parametrize("seed", range(6))
def test_sweep_quantize_next(seed):
    rng = np.random.default_rng(3000 + seed)
    M = int(rng.choice([1, 5, 40, 200]))
    K1, N1, N2 = int(rng.integers(16, 600)), int(rng.integers(16, 700)), int(rng.integers(8, 200))
    l1 = workloads.generic(M, N1, K1, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.5, a_signed=True, seed=4000 + seed, name="s1")
    a2 = WIDTHS_SIGNED[int(rng.integers(len(WIDTHS_SIGNED)))]
    signed2 = bool(rng.integers(2))
    l2 = workloads.generic(M, N2, N1, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.6, w_lo=1, w_hi=4,
                           w_frac_lo=0.5, a_signed=signed2, seed=5000 + seed, name="s2")
    print(f"[gpu] sweep next {seed} M={M} K1={K1} N1={N1} N2={N2} a2={a2} signed={signed2}", flush=True)
    r1 = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], True)
    y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])
    _, s_cal, _, _ = oracle.quantize_act(y1, l2["a_bits"], signed2)
    s2 = (s_cal * np.float32(rng.uniform(0.5, 1.5))).astype(np.float32)
    r_q = oracle.quantize_act_static(y1, l2["a_bits"], signed2, s2)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, _, seg_of2 = oracle.segments(l2["a_bits"])
    r_acc = oracle.mac(r_q, q_w2, seg_of2, S2)
    w1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True)
    w2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], signed2,
                               sign_nibbles=bool(seed % 2))
    a1, a2h = sq.soniq_act_create(w1, M), sq.soniq_act_create(w2, M)
    sq.soniq_quantize_act(a1, torch.from_numpy(l1["A"]).cuda())
    sq.soniq_mp_gemm_quantize_next(a1, w1, a2h, s2)
    acc = torch.empty((S2, M, N2), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(a2h, w2, acc=acc)
    torch.cuda.synchronize()
    q_a, s_a = sq.soniq_act_unpack_debug(a2h)
    _check(_bits(Y2), acc.cpu().numpy(), q_a, s_a, r_q, s2[:S2], r_acc, s_w2)
