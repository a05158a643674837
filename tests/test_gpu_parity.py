"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle.

Bar: weight and activation codes, scales and every int32 accumulator are
bit-exact; bf16 outputs equal the oracle's fixed-order fp32 replay bit for
bit and lie within the tolerance of the fp64 reference (relative 1e-2, or
2^-15 of the magnitude sum where cancellation makes the output tiny).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu


def _bf16_bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def gpu_run(case, wq_mode=0, ldw_pad=0, lda_pad=0, ldy_pad=0, with_acc=True, debug=True,
            sign_nibbles=False):
    M, N, K = case["M"], case["N"], case["K"]
    print(f"[gpu] {case['name']} M={M} N={N} K={K} wq_mode={wq_mode}", flush=True)
    Wb = torch.zeros((N, K + ldw_pad), dtype=torch.float32, device="cuda")
    Wb[:, :K] = torch.from_numpy(case["W"]).cuda()
    Ab = torch.zeros((M, K + lda_pad), dtype=torch.float32, device="cuda")
    Ab[:, :K] = torch.from_numpy(case["A"]).cuda()
    W, A = Wb[:, :K], Ab[:, :K]
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], case["a_signed"], wq_mode,
                              sign_nibbles=sign_nibbles)
    act = sq.soniq_act_create(w, M)
    sq.soniq_quantize_act(act, A)
    Yb = torch.empty((M, N + ldy_pad), dtype=torch.bfloat16, device="cuda")
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda") if with_acc else None
    sq.soniq_mp_gemm(act, w, out=Yb[:, :N], acc=acc)
    torch.cuda.synchronize()
    out = dict(S=w.S, y=_bf16_bits(Yb[:, :N]), w=w, act=act)
    if with_acc:
        out["acc"] = acc.cpu().numpy()
    if debug:
        out["q_w"], out["s_w"] = sq.soniq_weights_unpack_debug(w)
        out["q_a"], out["s_a"] = sq.soniq_act_unpack_debug(act)
    return out


def oracle_run(case, wq_mode=0):
    mode = oracle.TWOS_FRACTION if wq_mode == 1 else oracle.SIGNED
    return oracle.run(case["A"], case["W"], case["a_bits"], case["w_bits"], case["a_signed"], mode)


def check_y(y, y_ref, acc, s_a, s_w):
    yg = oracle.bf16_to_f32(y).astype(np.float64)
    yr = oracle.bf16_to_f32(y_ref).astype(np.float64)
    T = np.abs(s_w.astype(np.float64))[None, :] * sum(
        np.abs(float(s_a[g]) * acc[g].astype(np.float64)) for g in range(acc.shape[0]))
    tol = np.maximum(1e-2 * np.abs(yr), 2.0 ** -15 * T)
    bad = np.abs(yg - yr) > tol
    assert not bad.any(), f"{bad.sum()} outputs outside tolerance"


def compare_full(g, r):
    assert g["S"] == r["S"]
    np.testing.assert_array_equal(g["s_w"], r["s_w"])
    np.testing.assert_array_equal(g["q_w"], r["q_w"])
    np.testing.assert_array_equal(g["s_a"], r["s_a"])
    np.testing.assert_array_equal(g["q_a"], r["q_a"])
    np.testing.assert_array_equal(g["acc"], r["acc"])
    np.testing.assert_array_equal(g["y"], r["y_replay"])
    check_y(g["y"], r["y_ref"], r["acc"], r["s_a"], r["s_w"])


FULL = ["tiny_linear", "conv3x3_im2col", "xfmr_qkv", "xfmr_ffn_up", "xfmr_ffn_down",
        "decode_11008_m1", "decode_4096_m1", "decode_11008_m8", "decode_4096_m8"]


@pytest.mark.parametrize("name", FULL)
def test_workload_parity_full(name):
    case = workloads.make(name)
    compare_full(gpu_run(case), oracle_run(case))


NIBBLE_SIGN = [  # (M, N, K, a_lo, a_hi, w_lo, w_hi, a_signed): 1-bit weights in 4-bit containers
    (200, 256, 2304, 4, 8, 1, 4, False),
    (70, 130, 300, 4, 8, 1, 8, True),
    (3, 64, 200, 4, 8, 1, 2, True),        # batch of 3 on the GEMV
    (1, 100, 64, 4, 8, 1, 1, True),        # every output 1-bit, one row
    (150, 100, 129, 1, 8, 1, 2, True),     # 1-bit activations too
]


@pytest.mark.parametrize("shape", NIBBLE_SIGN, ids=lambda s: "x".join(map(str, s[:3])) + f"_w{s[5]}{s[6]}")
def test_sign_weights_in_nibbles(shape):
    """SONIQ_WPACK_SIGN_NIBBLES changes only the storage of 1-bit channels:
    the same codes, accumulators and outputs as the oracle."""
    M, N, K, alo, ahi, wlo, whi, sgn = shape
    case = workloads.generic(M, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.6, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.8, a_signed=sgn, seed=M + 3 * N + K, a_abs=not sgn,
                             name="sign_nibbles")
    compare_full(gpu_run(case, sign_nibbles=True), oracle_run(case))


def test_conv_workload_sign_nibbles():
    case = workloads.make("conv3x3_im2col")
    compare_full(gpu_run(case, sign_nibbles=True), oracle_run(case))


def test_square_8192_full():
    """Full-size 8192^3 at the benchmark's launch configuration, compared
    element by element: every code and scale, all 2 x 8192 x 8192 int32
    accumulators against the oracle's MAC, and every bf16 output against the
    oracle's fixed-order replay and within tolerance of its fp64 reference."""
    case = workloads.square_8192()
    g = gpu_run(case, with_acc=False, debug=True)
    q_w, s_w = oracle.quantize_weights(case["W"], case["w_bits"])
    q_a, s_a, seg_bits, seg_of = oracle.quantize_act(case["A"], case["a_bits"], case["a_signed"])
    np.testing.assert_array_equal(g["s_w"], s_w)
    np.testing.assert_array_equal(g["s_a"], s_a)
    np.testing.assert_array_equal(g["q_w"], q_w)
    np.testing.assert_array_equal(g["q_a"], q_a)
    del g["q_w"], g["q_a"]
    # the accumulators through a second call with the dump; its outputs must
    # be the same bits as the call without it
    w, act = g["w"], g["act"]
    acc = torch.empty((w.S, case["M"], case["N"]), dtype=torch.int32, device="cuda")
    Y = sq.soniq_mp_gemm(act, w, acc=acc)
    torch.cuda.synchronize()
    y = _bf16_bits(Y)
    np.testing.assert_array_equal(g["y"], y)
    acc_g = acc.cpu().numpy()
    del acc, Y
    print("[gpu] square_8192: oracle MAC over all outputs", flush=True)
    ref = oracle.mac(q_a, q_w, seg_of, len(seg_bits))
    np.testing.assert_array_equal(acc_g, ref)
    del acc_g
    np.testing.assert_array_equal(y, oracle.epilogue_replay(ref, s_a, s_w))
    y_ref = oracle.epilogue_ref(ref, s_a, s_w)
    for r0 in range(0, case["M"], 1024):  # bounded temporaries
        sl = slice(r0, r0 + 1024)
        check_y(y[sl], y_ref[sl], ref[:, sl], s_a, s_w)


EDGE = [  # (M, N, K, a_lo, a_hi, w_lo, w_hi, a_signed)
    (1, 1, 1, 4, 8, 2, 4, True),
    (1, 65, 63, 4, 8, 2, 4, True),
    (2, 130, 65, 2, 8, 1, 4, False),
    (7, 63, 200, 4, 4, 4, 8, True),
    (8, 300, 129, 1, 8, 1, 2, True),
    (9, 63, 200, 4, 8, 2, 8, True),
    (129, 257, 130, 4, 8, 2, 4, False),
    (200, 1, 64, 8, 8, 8, 8, True),
    (131, 129, 1000, 3, 6, 5, 7, True),
    (257, 200, 333, 1, 2, 1, 3, False),
    (3, 64, 4095, 4, 8, 2, 4, True),
    (150, 100, 129, 1, 8, 1, 2, True),     # sign-bit x sign-bit padding, GEMM path
    (20, 70, 65, 1, 1, 1, 1, True),        # all channels 1-bit
    (1030, 100, 300, 4, 8, 2, 4, True),    # 16-row block quantizer, ragged last block
    (1041, 70, 260, 4, 8, 1, 4, False),    # unsigned, ragged
    (1024, 64, 1028, 4, 8, 4, 8, True),    # two position slots per thread
]


@pytest.mark.parametrize("shape", EDGE, ids=lambda s: "x".join(map(str, s[:3])) + f"_a{s[3]}{s[4]}w{s[5]}{s[6]}{'s' if s[7] else 'u'}")
def test_edge_shapes(shape):
    M, N, K, alo, ahi, wlo, whi, sgn = shape
    case = workloads.generic(M, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.6, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.7, a_signed=sgn, seed=M * 1000 + N + K,
                             a_abs=not sgn, name="edge")
    compare_full(gpu_run(case), oracle_run(case))


@pytest.mark.parametrize("alo,ahi", [(1, 8), (2, 4), (3, 5), (6, 7), (1, 2)])
@pytest.mark.parametrize("sgn", [True, False])
@pytest.mark.parametrize("M", [3, 150])
def test_activation_widths(alo, ahi, sgn, M):
    case = workloads.generic(M, 96, 250, a_lo=alo, a_hi=ahi, a_frac_lo=0.5, w_lo=2, w_hi=8,
                             w_frac_lo=0.5, a_signed=sgn, seed=alo * 10 + ahi + M, name="awidth")
    compare_full(gpu_run(case), oracle_run(case))


@pytest.mark.parametrize("wlo,whi", [(1, 8), (2, 3), (4, 5), (6, 7), (1, 1), (8, 8)])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("M", [5, 140])
def test_weight_widths_and_grids(wlo, whi, mode, M):
    case = workloads.generic(M, 150, 190, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.5, seed=wlo * 10 + whi + M + 100 * mode, name="wwidth")
    compare_full(gpu_run(case, wq_mode=mode), oracle_run(case, wq_mode=mode))


GEMV_W = [(2, 4), (2, 8), (4, 8), (1, 4), (1, 2), (8, 8), (3, 4)]
GEMV_A = [(4, 8, True), (4, 8, False), (4, 4, True), (3, 8, True), (2, 8, True), (8, 8, True)]


@pytest.mark.parametrize("wlo,whi", GEMV_W)
@pytest.mark.parametrize("alo,ahi,sgn", GEMV_A)
@pytest.mark.parametrize("M", [1, 2, 5, 8])
def test_small_batch_paths(wlo, whi, alo, ahi, sgn, M):
    """Batch <= 8: nibble dot products (4-bit activation groups against 2- and
    4-bit weight blocks), byte dot products otherwise, ragged N and K."""
    case = workloads.generic(M, 333, 1000, a_lo=alo, a_hi=ahi, a_frac_lo=0.7, w_lo=wlo,
                             w_hi=whi, w_frac_lo=0.6, a_signed=sgn, a_abs=not sgn,
                             seed=wlo * 1000 + whi * 100 + alo * 10 + ahi + M * 7 + sgn,
                             name="gemv")
    compare_full(gpu_run(case), oracle_run(case))


@pytest.mark.parametrize("M,K", [(1, 9000), (2, 9000), (8, 3000)])
def test_small_batch_long_rows(M, K):
    """Several load batches per workgroup and several activation staging rounds."""
    case = workloads.generic(M, 100, K, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=4, w_hi=8,
                             w_frac_lo=0.5, seed=K + M, name="gemv_long")
    compare_full(gpu_run(case), oracle_run(case))


@pytest.mark.parametrize("K,lda_pad,wlo,whi", [
    (1000, 0, 2, 4),    # per-row quantizer; nibble-path blocks
    (1000, 0, 4, 8),    # byte-path blocks widen the image's 4-bit units
    (1000, 0, 1, 4),    # sign-bit blocks
    (20000, 0, 2, 8),   # small-batch quantizer; several staging rounds
    (1001, 3, 2, 4),    # unaligned row: two-pass quantizer
])
def test_single_row_image(K, lda_pad, wlo, whi):
    """A GEMV of one row stages the contiguous row image its quantizer left
    beside the units; every quantizer of one row writes it."""
    case = workloads.generic(1, 200, K, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.5, seed=K + wlo + lda_pad, name="row_image")
    compare_full(gpu_run(case, lda_pad=lda_pad), oracle_run(case))


def test_single_row_image_after_other_writers():
    """The image follows whatever last quantized the handle: larger batches
    (which leave no image), the fused one-call form, and one row again."""
    big = workloads.generic(24, 300, 2000, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=4,
                            w_frac_lo=0.5, seed=77, name="row_image_seq")
    W = torch.from_numpy(big["W"]).cuda()
    w = sq.soniq_pack_weights(W, big["w_bits"], big["a_bits"], True)
    act = sq.soniq_act_create(w, 24)
    for step, (M, lo, fused) in enumerate([(1, 0, False), (24, 0, False), (1, 5, False),
                                           (3, 2, False), (1, 9, True), (1, 9, False),
                                           (1, 11, True)]):
        print(f"[gpu] row image step {step}: M={M} row {lo} fused={fused}", flush=True)
        A_np = big["A"][lo:lo + M].copy()
        A = torch.from_numpy(A_np).cuda()
        acc = torch.empty((w.S, M, 300), dtype=torch.int32, device="cuda")
        if fused:
            Y = sq.soniq_quantize_mp_gemm(act, w, A, acc=acc)
        else:
            sq.soniq_quantize_act(act, A)
            Y = sq.soniq_mp_gemm(act, w, acc=acc)
        torch.cuda.synchronize()
        r = oracle.run(A_np, big["W"], big["a_bits"], big["w_bits"], True)
        np.testing.assert_array_equal(acc.cpu().numpy(), r["acc"])
        np.testing.assert_array_equal(_bf16_bits(Y), r["y_replay"])
    # a GEMV after the fused call reads the image the fused call left
    Y2 = sq.soniq_mp_gemm(act, w)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bf16_bits(Y2), r["y_replay"])


def test_stream_read_probe():
    """The plain-read probe bench.py holds the GEMV against reads every byte:
    its per-workgroup XORs equal the host's, ragged last workgroup included."""
    n = 8192 * 37 + 48
    src = torch.randint(0, 256, (n + 64,), dtype=torch.uint8, device="cuda")
    sink = torch.zeros(38, dtype=torch.int32, device="cuda")
    sq.soniq_debug_stream_read(src, n, sink, offset=16)
    torch.cuda.synchronize()
    words = np.zeros((38 * 8192) // 4, np.uint32)
    words.view(np.uint8)[:n] = src.cpu().numpy()[16:16 + n]
    ref = np.bitwise_xor.reduce(words.reshape(38, 2048), axis=1)
    np.testing.assert_array_equal(sink.cpu().numpy().view(np.uint32), ref)


def test_strides_and_unaligned_rows():
    case = workloads.generic(70, 100, 131, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=4,
                             w_frac_lo=0.5, seed=5, name="strides")
    compare_full(gpu_run(case, ldw_pad=3, lda_pad=5, ldy_pad=7), oracle_run(case))
    case = workloads.generic(5, 100, 132, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=4,
                             w_frac_lo=0.5, seed=6, name="strides2")
    compare_full(gpu_run(case, ldw_pad=1, lda_pad=1, ldy_pad=1), oracle_run(case))


@pytest.mark.parametrize("extreme", [False, True], ids=["random", "all_max"])
def test_largest_padded_k(extreme):
    """K at the accumulator limit (65472 8-bit channels, padded K 65472 <=
    SONIQ_MAX_K): every code at its maximum gives ACC = 127*127*K, just
    under 2^31 / 2; the quantizer and GEMM take their wide-row forms."""
    M, N, K = 20, 130, 65472
    case = workloads.generic(M, N, K, a_lo=8, a_hi=8, a_frac_lo=1.0, w_lo=8, w_hi=8,
                             w_frac_lo=1.0, a_signed=True, seed=77, name="kmax")
    if extreme:
        case["A"][:] = 1.0
        case["W"][:] = 0.5
    g, r = gpu_run(case), oracle_run(case)
    if extreme:
        assert r["acc"].max() == 127 * 127 * K
    compare_full(g, r)


def test_zero_inputs():
    case = workloads.generic(40, 70, 100, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=1, w_hi=4,
                             w_frac_lo=0.5, seed=9, name="zeros")
    case["A"][:] = 0.0
    case["W"][::3] = 0.0
    compare_full(gpu_run(case), oracle_run(case))
    case = workloads.generic(4, 70, 100, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=1, w_hi=4,
                             w_frac_lo=0.5, seed=10, name="zeros-group")
    case["A"][:, case["a_bits"] == 8] = 0.0       # one activation group all zero
    compare_full(gpu_run(case), oracle_run(case))


def test_tiny_and_huge_magnitudes():
    case = workloads.generic(33, 40, 77, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=8,
                             w_frac_lo=0.5, seed=11, a_std=1e-30, w_std=1e30, name="scale")
    compare_full(gpu_run(case), oracle_run(case))


def test_repeat_calls_and_smaller_batch():
    """Results do not depend on an earlier, larger call through the same
    handles, and repeated calls are bit-identical (no races)."""
    big = workloads.generic(300, 130, 260, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=4,
                            w_frac_lo=0.5, seed=12, name="big")
    W = torch.from_numpy(big["W"]).cuda()
    w = sq.soniq_pack_weights(W, big["w_bits"], big["a_bits"], True)
    act = sq.soniq_act_create(w, 300)
    ys = []
    for M in (300, 300, 7, 131, 7):
        A = torch.from_numpy(big["A"][:M].copy()).cuda()
        sq.soniq_quantize_act(act, A)
        acc = torch.empty((w.S, M, 130), dtype=torch.int32, device="cuda")
        Y = sq.soniq_mp_gemm(act, w, acc=acc)
        torch.cuda.synchronize()
        r = oracle.run(big["A"][:M], big["W"], big["a_bits"], big["w_bits"], True)
        np.testing.assert_array_equal(acc.cpu().numpy(), r["acc"])
        np.testing.assert_array_equal(_bf16_bits(Y), r["y_replay"])
        ys.append(_bf16_bits(Y))
    np.testing.assert_array_equal(ys[0], ys[1])
    np.testing.assert_array_equal(ys[2], ys[4])


def test_api_errors_on_device():
    case = workloads.tiny_linear()
    W = torch.from_numpy(case["W"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], True)
    w2 = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], True)
    act = sq.soniq_act_create(w, 16)
    with pytest.raises(sq.SoniqError):
        sq.soniq_mp_gemm(act, w)                 # nothing quantized yet
    A = torch.from_numpy(case["A"]).cuda()
    with pytest.raises(sq.SoniqError):
        sq.soniq_quantize_act(act, A)            # M = 64 > max_M = 16
    sq.soniq_quantize_act(act, A[:16])
    with pytest.raises(sq.SoniqError):
        sq.soniq_mp_gemm(act, w2)                # activations of other weights
    info = sq.soniq_weights_info(w)
    assert info.N == 256 and info.K == 256 and info.S == 2
    assert list(info.a_bits) == [4, 8] and list(info.w_bits) == [2, 4]
    assert info.packed_w_bytes_algorithmic == (192 * 2 + 64 * 4) * 256 // 8


# Batches of at least 2^20 elements that fit the registers of one resident
# grid are quantized in one pass (rows per workgroup RB and float4 per
# thread T chosen from K); each case below lands on a different (RB, T),
# with a ragged last workgroup.  Both the single pass and the two-pass
# path (SONIQ_ACT_COOP=0) must match the oracle.
COOP = [  # (M, K, a_lo, a_hi, a_signed)      RB, T
    (8200, 128, 4, 8, True),                # 16, 6 (K4 = 32: 8 rows per 256-step)
    (1400, 768, 4, 8, False),               # 16, 12
    (343, 3072, 2, 4, True),                # 4, 12 (2-bit pieces of 4 rows)
    (460, 2304, 4, 8, False),               # 8, 18 (the conv row length)
    (1100, 1000, 4, 8, True),               # 4, 6 (K4 = 250 < 256)
    (4100, 260, 2, 8, False),               # 16, 6 (K4 = 65: three rows per step)
]


@pytest.mark.parametrize("coop", [True, False], ids=["single_pass", "two_pass"])
@pytest.mark.parametrize("shape", COOP, ids=lambda s: f"{s[0]}x{s[1]}_a{s[2]}{s[3]}{'s' if s[4] else 'u'}")
def test_single_pass_quantize(shape, coop, monkeypatch):
    M, K, alo, ahi, sgn = shape
    if not coop:
        monkeypatch.setenv("SONIQ_ACT_COOP", "0")
    case = workloads.generic(M, 64, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.6, w_lo=2, w_hi=4,
                             w_frac_lo=0.5, a_signed=sgn, a_abs=not sgn, seed=M + K,
                             name="coop")
    compare_full(gpu_run(case), oracle_run(case))


def test_single_pass_repeat_calls():
    """The grid barrier's counters reset themselves: repeated calls, a
    smaller grid after a larger one and new data all stay bit-exact."""
    big = workloads.generic(1400, 64, 768, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=4,
                            w_frac_lo=0.5, seed=21, name="coop-repeat")
    W = torch.from_numpy(big["W"]).cuda()
    w = sq.soniq_pack_weights(W, big["w_bits"], big["a_bits"], True)
    act = sq.soniq_act_create(w, 1400)
    for M, scale in ((1400, 1.0), (1400, 3.0), (1366, 0.5), (1400, 1.0)):
        A_np = (big["A"][:M] * np.float32(scale)).copy()
        sq.soniq_quantize_act(act, torch.from_numpy(A_np).cuda())
        acc = torch.empty((w.S, M, 64), dtype=torch.int32, device="cuda")
        Y = sq.soniq_mp_gemm(act, w, acc=acc)
        torch.cuda.synchronize()
        r = oracle.run(A_np, big["W"], big["a_bits"], big["w_bits"], True)
        _, s_a = sq.soniq_act_unpack_debug(act)
        np.testing.assert_array_equal(s_a, r["s_a"])
        np.testing.assert_array_equal(acc.cpu().numpy(), r["acc"])
        np.testing.assert_array_equal(_bf16_bits(Y), r["y_replay"])
    assert sq.soniq_act_wait_timeouts(act) == 0  # the grid was resident every time


@pytest.mark.parametrize("M,K", [(1400, 768), (460, 2304)])
def test_single_pass_wait_timeout(M, K, monkeypatch):
    """With a spin limit of zero every workgroup but the grid's last arrival
    gives up waiting and takes the maxima from the whole batch itself; the
    codes, scales and outputs are the same, and the next call (normal
    limit) finds the grid state clean."""
    case = workloads.generic(M, 64, K, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=4,
                             w_frac_lo=0.5, a_signed=False, a_abs=True, seed=M * 3 + K,
                             name="coop-timeout")
    ref = oracle_run(case)
    monkeypatch.setenv("SONIQ_COOP_SPINS", "0")
    g = gpu_run(case)
    compare_full(g, ref)
    # the workgroup that arrived first polled before the last arrival
    assert sq.soniq_act_wait_timeouts(g["act"]) >= 1
    monkeypatch.delenv("SONIQ_COOP_SPINS")
    g = gpu_run(case)
    compare_full(g, ref)
    assert sq.soniq_act_wait_timeouts(g["act"]) == 0
