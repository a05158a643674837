"""The allocation-free entry point (soniq_quantize_mp_gemm_scratch), for
callers that cannot allocate device memory: called through the C-ABI, its
outputs and int32 accumulators equal those of soniq_quantize_mp_gemm on an
activation handle, bit for bit, on two calls in a row whose second batch is
smaller (the scratch keeps the first call's contents), for the single-pass,
two-pass, sub-group-scale and one-row quantizers; a batch too large for the
scratch is rejected before anything runs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy()


CASES = [  # (name, M first, M second, K, N, a_lo, a_hi, w_lo, w_hi, signed, group_bits)
    ("single_pass", 1400, 300, 768, 256, 4, 8, 2, 8, True, 0),
    ("unsigned_conv_like", 2048, 96, 2304, 256, 4, 8, 1, 4, False, 0),
    ("sub_group_scales", 1536, 200, 1024, 192, 4, 8, 2, 8, True, 512),
    ("decode", 8, 1, 4096, 1100, 4, 8, 2, 4, True, 0),
]


@pytest.mark.parametrize("c", CASES, ids=lambda c: c[0])
def test_scratch_entry_matches_handle_entry(c):
    name, M1, M2, K, N, alo, ahi, wlo, whi, sgn, gbits = c
    case = workloads.generic(M1, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.6, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.7, a_signed=sgn, a_abs=not sgn, seed=M1 + K + N,
                             name=name)
    print(f"[gpu] scratch entry {name} M={M1},{M2} K={K} N={N} g={gbits}", flush=True)
    W = torch.from_numpy(case["W"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], sgn, act_group_bits=gbits)
    act = sq.soniq_act_create(w, M1)
    A_full = torch.from_numpy(case["A"]).cuda()
    for M in (M1, M2):
        A = A_full[:M] * (1.0 if M == M1 else 0.5)     # other data in the second call
        Yh = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        acc_h = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
        sq.soniq_quantize_mp_gemm(act, w, A, out=Yh, acc=acc_h)
        Ys = torch.full((M, N), 7.0, dtype=torch.bfloat16, device="cuda")
        acc_s = torch.full((w.S, M, N), -5, dtype=torch.int32, device="cuda")
        sq.soniq_quantize_mp_gemm_scratch(w, A, out=Ys, acc=acc_s)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(acc_s.cpu().numpy(), acc_h.cpu().numpy(), err_msg=f"M={M}")
        np.testing.assert_array_equal(_bits(Ys), _bits(Yh), err_msg=f"M={M}")
        if M == M2 and not gbits:
            # and the oracle, on the smaller call
            r = oracle.run(A.cpu().numpy(), case["W"], case["a_bits"], case["w_bits"], sgn)
            np.testing.assert_array_equal(acc_s.cpu().numpy(), r["acc"])
            np.testing.assert_array_equal(_bits(Ys).view(np.uint16), r["y_replay"])


def test_scratch_entry_rejects_oversized_batches():
    """A batch whose packed rows exceed the scratch: UNSUPPORTED, Y untouched."""
    K, N, M = 8192, 64, 16384
    rng = np.random.default_rng(5)
    W = torch.from_numpy((rng.standard_normal((N, K)) * 0.02).astype(np.float32)).cuda()
    w = sq.soniq_pack_weights(W, np.full(N, 4, np.uint8), np.full(K, 8, np.uint8), True)
    A = torch.zeros((M, K), dtype=torch.float32, device="cuda")
    Y = torch.full((M, N), 3.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(sq.SoniqError) as e:
        sq.soniq_quantize_mp_gemm_scratch(w, A, out=Y)
    assert e.value.status == sq.SONIQ_ERR_UNSUPPORTED
    assert b"scratch" in sq.lib().soniq_last_error()
    torch.cuda.synchronize()
    assert bool((Y == 3.0).all())
    # the largest configuration of the benchmark fits: M = K = 8192 at 4/8 bits
    A2 = torch.from_numpy(rng.standard_normal((8192, K)).astype(np.float32)).cuda()
    ab = np.where(np.arange(K) % 2 == 0, 4, 8).astype(np.uint8)
    w2 = sq.soniq_pack_weights(W, np.full(N, 4, np.uint8), ab, True)
    act = sq.soniq_act_create(w2, 8192)
    Yh = sq.soniq_quantize_mp_gemm(act, w2, A2)
    Ys = sq.soniq_quantize_mp_gemm_scratch(w2, A2)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bits(Ys), _bits(Yh))
