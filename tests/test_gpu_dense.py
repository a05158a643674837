"""GPU parity of the dense weight copy (SONIQ_WPACK_DENSE): the GEMV forms
(batches of at most 8 rows) read every code in exactly its channel's width,
so 3-, 5-, 6- and 7-bit channels no longer take the next power-of-two
container (the f4 row's dense packing; Sec. 7 finds CNN palettes of 1 and
5-8 bits).  Same bar as the other parity tests: codes, scales and every
int32 accumulator bit-exact, bf16 outputs equal to the fixed-order replay;
and the same bits as the same layer packed without the dense copy."""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads
from test_gpu_parity import _bf16_bits, compare_full, oracle_run

pytestmark = pytest.mark.gpu


def run(case, dense):
    M, N, K = case["M"], case["N"], case["K"]
    W = torch.from_numpy(case["W"]).cuda()
    A = torch.from_numpy(case["A"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], case["a_signed"], dense=dense)
    act = sq.soniq_act_create(w, M)
    sq.soniq_quantize_act(act, A)
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
    Y = sq.soniq_mp_gemm(act, w, acc=acc)
    torch.cuda.synchronize()
    out = dict(S=w.S, y=_bf16_bits(Y), acc=acc.cpu().numpy(), w=w, act=act)
    out["q_w"], out["s_w"] = sq.soniq_weights_unpack_debug(w)
    out["q_a"], out["s_a"] = sq.soniq_act_unpack_debug(act)
    return out


CASES = [  # (M, N, K, a_lo, a_hi, w_lo, w_hi, a_signed)
    (1, 300, 512, 4, 8, 3, 6, True),     # 3/6-bit weights, one row
    (3, 200, 700, 4, 8, 5, 7, False),    # 5/7-bit, unsigned activations, ragged K
    (8, 256, 1024, 4, 8, 1, 3, True),    # sign bits and 3 bits, 8 rows
    (2, 130, 300, 1, 8, 1, 5, True),     # 1-bit activations against 1-bit weights
    (5, 96, 4096, 3, 6, 2, 7, True),     # long K (several batches of runs per thread)
    (1, 64, 256, 4, 8, 6, 6, True),      # one width
    (4, 100, 640, 4, 8, 4, 8, True),     # power-of-two widths through the dense path
    (1, 1000, 4096, 4, 8, 3, 6, True),   # a decode-like row
    # sign weights against a sign activation group: XNOR-popcount runs
    (1, 200, 1000, 1, 8, 1, 4, True),    # one row, beside an 8-bit group
    (8, 160, 2048, 1, 4, 1, 2, True),    # eight rows
    (3, 64, 700, 1, 1, 1, 1, True),      # sign x sign only, ragged K
    (2, 48, 4160, 1, 8, 1, 6, True),     # K / 64 odd: half of the last quad-run past K
]


@pytest.mark.parametrize("c", CASES, ids=lambda c: f"M{c[0]}_N{c[1]}_K{c[2]}_w{c[5]}{c[6]}_a{c[3]}{c[4]}")
def test_dense_gemv(c):
    M, N, K, alo, ahi, wlo, whi, sgn = c
    case = workloads.generic(M, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.7, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.6, a_signed=sgn, seed=M * 7 + N + K, name="dense")
    print(f"[gpu] dense M={M} N={N} K={K} w={wlo}/{whi} a={alo}/{ahi}", flush=True)
    g = run(case, True)
    compare_full(g, oracle_run(case))
    plain = run(case, False)
    np.testing.assert_array_equal(g["acc"], plain["acc"])
    np.testing.assert_array_equal(g["y"], plain["y"])


def test_dense_bytes_and_batches_above_8():
    """The dense copy holds 256*b bytes per 128-channel quad-run of each
    16-row block (b its width, Kp rounded up to 128 channels);
    batches above 8 rows run the GEMM tiles on the units, bit-exact."""
    case = workloads.generic(40, 200, 500, a_lo=4, a_hi=8, a_frac_lo=0.7, w_lo=3, w_hi=6,
                             w_frac_lo=0.6, a_signed=True, seed=3, name="dense40")
    g = run(case, True)
    compare_full(g, oracle_run(case))
    info = sq.soniq_weights_info(g["w"])
    n_lo = int((case["w_bits"] == 3).sum())
    n_hi = 200 - n_lo
    Kp = int(info.a_count_padded[0] + info.a_count_padded[1])
    blocks = lambda n: (n + 15) // 16
    # blocks in plan order: the narrow class padded to whole 128-column tiles
    nb_lo = -(-blocks(n_lo) // 8) * 8
    nb_all = -(-(nb_lo + blocks(n_hi)) // 8) * 8
    nquad = -(-Kp // 128)
    expect = 256 * nquad * (3 * nb_lo + 6 * (nb_all - nb_lo))
    assert info.dense_w_bytes == expect
    assert info.dense_w_bytes < info.packed_w_bytes


def test_dense_rejects_other_copies():
    case = workloads.generic(4, 64, 256, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=3, w_hi=6,
                             w_frac_lo=0.5, a_signed=True, seed=5, name="dense_bad")
    W = torch.from_numpy(case["W"]).cuda()
    for kw in (dict(f8f6f4=True), dict(act_group_bits=512)):
        with pytest.raises(sq.SoniqError) as e:
            sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], True, dense=True, **kw)
        assert e.value.status == sq.SONIQ_ERR_UNSUPPORTED


@pytest.mark.parametrize("name", ["decode_11008_m1_w36", "decode_11008_m8_w36", "decode_11008_m1_sign"])
def test_dense_workload_full(name):
    """The dense decode workloads at full size, as bench.py --dense runs
    them (the same handles and entry points), compared in full."""
    case = workloads.make(name)
    print(f"[gpu] dense workload {name}", flush=True)
    compare_full(run(case, True), oracle_run(case))


@pytest.mark.parametrize("M", [1, 5])
def test_dense_one_call_and_scratch(M):
    """soniq_quantize_mp_gemm and the allocation-free entry point on a
    dense handle (quantize, then the dense GEMV) give the two-call result."""
    case = workloads.generic(M, 300, 1500, a_lo=4, a_hi=8, a_frac_lo=0.8, w_lo=3, w_hi=6,
                             w_frac_lo=0.7, a_signed=True, seed=77 + M, name="dense_call")
    print(f"[gpu] dense one-call M={M}", flush=True)
    ref = run(case, True)
    w = ref["w"]
    A = torch.from_numpy(case["A"]).cuda()
    act = sq.soniq_act_create(w, M)
    for _ in range(2):
        acc = torch.empty((w.S, M, case["N"]), dtype=torch.int32, device="cuda")
        Y = sq.soniq_quantize_mp_gemm(act, w, A, acc=acc)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(acc.cpu().numpy(), ref["acc"])
        np.testing.assert_array_equal(_bf16_bits(Y), ref["y"])
        acc2 = torch.empty_like(acc)
        Y2 = sq.soniq_quantize_mp_gemm_scratch(w, A, acc=acc2)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(acc2.cpu().numpy(), ref["acc"])
        np.testing.assert_array_equal(_bf16_bits(Y2), ref["y"])
