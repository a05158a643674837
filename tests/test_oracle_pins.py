"""Pins of the CPU oracle against what the paper and mathematics fix.

Every check here is independent of the oracle's own formulas: brute-force
searches, hand-worked fixtures (tests/golden/), enumeration of Eq. (1),
library routines for special cases (numpy integer matmul, fp64 BLAS, torch's
bf16 cast), invariants (error bound of Sec. 2.3, permutation and padding
invariance of Sec. 3 / Fig. "normalization"), and a noise-model sanity check.
"""
import itertools
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- helpers
def brute_code(r: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """argmin over the integer grid [lo, hi] of |r - q|, ties to the even q.

    r is the fp32 quotient; differences are formed in fp64 (exact)."""
    grid = np.arange(lo, hi + 1, dtype=np.float64)
    d = np.abs(r.astype(np.float64)[:, None] - grid[None, :])
    best = d.min(axis=1, keepdims=True)
    cand = d == best
    # among tied candidates prefer the even one
    even = (np.arange(lo, hi + 1) % 2 == 0)[None, :]
    pick_even = cand & even
    has_even = pick_even.any(axis=1)
    idx = np.where(has_even, pick_even.argmax(axis=1), cand.argmax(axis=1))
    return (lo + idx).astype(np.int64)


def read_sections(path):
    sec, cur = {}, None
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        if line.startswith("["):
            cur = line.strip("[]")
            sec[cur] = []
        else:
            sec[cur].append(line.split())
    return sec


# ------------------------------------------------------------- O1: grids
def test_qmax_closed_forms():
    for b in range(1, 9):
        assert oracle.qmax(b, oracle.UNSIGNED) == 2 ** b - 1      # codec item 2
        assert oracle.qmax(b, oracle.TWOS_FRACTION) == 2 ** (b - 1)  # Eq. (1) denominator
        assert oracle.qmax(b, oracle.SIGNED) == (1 if b == 1 else 2 ** (b - 1) - 1)
    assert oracle.qmax(0, oracle.SIGNED) == -1
    assert oracle.qmax(9, oracle.SIGNED) == -1


# ----------------------------------------------------- O2/O3 signed codes
@pytest.mark.parametrize("bits", [2, 3, 4, 5, 6, 7, 8])
def test_signed_codes_match_brute_force_argmin(bits):
    rng = np.random.default_rng(bits)
    N, K = 64, 257
    W = (rng.standard_normal((N, K)) * rng.uniform(1e-3, 10, (N, 1))).astype(np.float32)
    q, s = oracle.quantize_weights(W, np.full(N, bits, np.uint8))
    Q = 2 ** (bits - 1) - 1
    m = np.abs(W).max(axis=1)
    np.testing.assert_array_equal(s, m / np.float32(Q))            # fp32 IEEE division
    r = (W / s[:, None]).astype(np.float32)
    ref = brute_code(r.ravel(), -Q, Q).reshape(N, K)
    np.testing.assert_array_equal(q, ref)
    # the max-abs element lands on +-Q
    am = np.abs(W).argmax(axis=1)
    np.testing.assert_array_equal(np.abs(q[np.arange(N), am]), Q)
    # symmetric grid: q(-x) = -q(x)
    q2, _ = oracle.quantize_weights(-W, np.full(N, bits, np.uint8))
    np.testing.assert_array_equal(q2, -q)


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_error_bound_of_rounding(bits):
    """Sec. 2.3: Q(x) = round(x/D) D = x + e with |e| <= D/2."""
    rng = np.random.default_rng(100 + bits)
    W = rng.standard_normal((32, 500)).astype(np.float32)
    q, s = oracle.quantize_weights(W, np.full(32, bits, np.uint8))
    err = np.abs(W.astype(np.float64) - q * s[:, None].astype(np.float64))
    bound = s[:, None].astype(np.float64) / 2 * (1 + 1e-6) + 1e-12
    assert (err <= bound).all()


def test_ties_round_to_even():
    s = np.float32(0.25)   # power of two: x/s is exact
    cases = {0.375: 2, 0.625: 2, 0.125: 0, -0.375: -2, -0.125: 0, 0.875: 4, 1.125: 4}
    for x, want in cases.items():
        assert oracle.code(x, s, 8, oracle.SIGNED) == want, x
    # clamp at the grid edge
    assert oracle.code(100.0, s, 4, oracle.SIGNED) == 7
    assert oracle.code(-100.0, s, 4, oracle.SIGNED) == -7


def test_sign_mode_one_bit():
    """1-bit channels are +-1 (XNOR/popcount semantics, Sec. 4.2), scale = max-abs."""
    W = np.array([[0.5, -0.25, 0.0, -0.0, 2.0]], np.float32)
    q, s = oracle.quantize_weights(W, np.array([1], np.uint8))
    np.testing.assert_array_equal(q, [[1, -1, 1, 1, 1]])
    assert s[0] == np.float32(2.0)


def test_zero_group():
    W = np.zeros((3, 8), np.float32)
    q, s = oracle.quantize_weights(W, np.array([1, 4, 8], np.uint8))
    np.testing.assert_array_equal(s, 0)
    np.testing.assert_array_equal(q[0], 1)     # sign mode of +0
    np.testing.assert_array_equal(q[1:], 0)


# ------------------------------------------------------- O5 unsigned codes
@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_unsigned_codes_match_brute_force(bits):
    rng = np.random.default_rng(7 + bits)
    A = rng.standard_normal((40, 300)).astype(np.float32)
    q, s, sb, so = oracle.quantize_act(A, np.full(300, bits, np.uint8), a_signed=False)
    Q = 2 ** bits - 1
    assert s[0] == np.abs(A).max() / np.float32(Q)
    r = (A / s[0]).astype(np.float32)
    ref = brute_code(r.ravel(), 0, Q).reshape(A.shape)
    np.testing.assert_array_equal(q, ref)
    assert (q[A < 0] == 0).all()                 # clip of the negative side


def test_unsigned_golden():
    rows = [l.split() for l in open(os.path.join(GOLD, "unsigned_codec_n4.txt"))
            if l.strip() and not l.startswith("#")]
    a = np.array([float(r[0]) for r in rows], np.float32)[None, :]
    want = np.array([int(r[1]) for r in rows])
    q, s, _, _ = oracle.quantize_act(a, np.full(a.shape[1], 4, np.uint8), a_signed=False)
    assert s[0] == np.float32(0.5)
    np.testing.assert_array_equal(q[0], want)


# -------------------------------------------- Eq. (1) two's-complement grid
def eq1_value(bits_lsb_first, n):
    """Eq. (1): q(b) = -b_{n-1} + sum_{i=0}^{n-2} b_i 2^-(i+1)."""
    v = -float(bits_lsb_first[n - 1])
    for i in range(n - 1):
        v += bits_lsb_first[i] * 2.0 ** -(i + 1)
    return v


def test_eq1_table_golden():
    rows = [l.split() for l in open(os.path.join(GOLD, "eq1_table_n3.txt"))
            if l.strip() and not l.startswith("#")]
    for b2, b1, b0, q in rows:
        assert eq1_value([int(b0), int(b1), int(b2)], 3) == float(q)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 8])
def test_eq1_mode_is_the_argmin_over_all_bit_patterns(n):
    values = sorted({eq1_value(bs, n) for bs in itertools.product([0, 1], repeat=n)})
    # the value set of Eq. (1) is k / 2^(n-1), k in [-2^(n-1), 2^(n-1) - 1]
    assert values == [k / 2 ** (n - 1) for k in range(-2 ** (n - 1), 2 ** (n - 1))]
    rng = np.random.default_rng(n)
    W = rng.standard_normal((16, 200)).astype(np.float32)
    q, s = oracle.quantize_weights(W, np.full(16, n, np.uint8), mode=oracle.TWOS_FRACTION)
    m = np.abs(W).max(axis=1)
    np.testing.assert_array_equal(s, m / np.float32(2 ** (n - 1)))
    wn = (W / m[:, None]).astype(np.float32).astype(np.float64)     # w' = w / s_g
    vals = np.array(values)
    d = np.abs(wn.ravel()[:, None] - vals[None, :])
    best = d.min(axis=1, keepdims=True)
    cand = d == best
    ks = np.arange(-2 ** (n - 1), 2 ** (n - 1))
    even = (ks % 2 == 0)[None, :]
    pe = cand & even
    idx = np.where(pe.any(axis=1), pe.argmax(axis=1), cand.argmax(axis=1))
    np.testing.assert_array_equal(q.ravel(), ks[idx])
    # decode is s_g * q(b*): the reconstructed weight is m * value
    np.testing.assert_allclose(q * s[:, None], m[:, None] * vals[idx].reshape(q.shape), rtol=0, atol=0)


# ------------------------------------------------------------ O4 segments
def test_segments():
    S, sb, so = oracle.segments(np.array([8, 4, 4, 8, 4], np.uint8))
    assert S == 2 and list(sb) == [4, 8] and list(so) == [1, 0, 0, 1, 0]
    S, sb, so = oracle.segments(np.array([3, 3], np.uint8))
    assert S == 1 and list(sb) == [3] and list(so) == [0, 0]
    for bad in ([1, 2, 4], [0, 4], [9, 4]):
        with pytest.raises(ValueError):
            oracle.segments(np.array(bad, np.uint8))


def test_activation_group_scale_is_shared():
    """C2: one scale per activation precision group, from the group max-abs."""
    rng = np.random.default_rng(3)
    A = rng.standard_normal((8, 50)).astype(np.float32)
    ab = np.where(rng.random(50) < 0.3, 8, 2).astype(np.uint8)
    q, s, sb, so = oracle.quantize_act(A, ab, a_signed=True)
    for g, b in enumerate(sb):
        m = np.abs(A[:, ab == b]).max()
        assert s[g] == m / np.float32(2 ** (b - 1) - 1)


# --------------------------------------------------------------- O6 MAC
def test_all_8bit_reduces_to_int8_gemm():
    rng = np.random.default_rng(11)
    A = rng.standard_normal((37, 129)).astype(np.float32)
    W = rng.standard_normal((23, 129)).astype(np.float32)
    r = oracle.run(A, W, np.full(129, 8, np.uint8), np.full(23, 8, np.uint8), a_signed=True)
    assert r["S"] == 1
    assert r["q_a"].min() >= -127 and r["q_a"].max() <= 127
    ref = r["q_a"].astype(np.int8).astype(np.int64) @ r["q_w"].astype(np.int8).astype(np.int64).T
    np.testing.assert_array_equal(r["acc"][0], ref)


def test_acc_equals_fp64_blas_per_group():
    rng = np.random.default_rng(12)
    M, N, K = 33, 41, 300
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    ab = np.where(rng.random(K) < 0.6, 4, 8).astype(np.uint8)
    wb = np.where(rng.random(N) < 0.5, 2, 8).astype(np.uint8)
    r = oracle.run(A, W, ab, wb, a_signed=True)
    for g, b in enumerate(r["seg_bits"]):
        cols = ab == b
        ref = r["q_a"][:, cols].astype(np.float64) @ r["q_w"][:, cols].astype(np.float64).T
        np.testing.assert_array_equal(r["acc"][g], ref.astype(np.int64))


@pytest.mark.parametrize("S", [1, 2, 5])
def test_sampled_mac_equals_integer_products(S):
    """The sampled MAC (one output's sums at given (m, n) pairs, used to check
    outputs one by one at sizes the full MAC cannot reach) against numpy
    int64 products over each scale group's channels, and against the pinned
    full MAC: corners, repeated pairs, a group with no channel, and a pair
    whose row and column indices differ (catches swapped m and n)."""
    rng = np.random.default_rng(40 + S)
    M, N, K = 23, 37, 301
    q_a = rng.integers(-128, 128, (M, K)).astype(np.int32)
    q_w = rng.integers(-128, 128, (N, K)).astype(np.int32)
    # scale group of each channel: S groups in a shuffled order, the last
    # one empty when S > 2 (its sums must be 0)
    used = max(1, S - 1) if S > 2 else S
    grp = rng.integers(0, used, K).astype(np.int32)
    ms = np.concatenate([rng.integers(0, M, 200), [0, 0, M - 1, M - 1, 3, 3]])
    ns = np.concatenate([rng.integers(0, N, 200), [0, N - 1, 0, N - 1, 30, 30]])
    got = oracle.mac_at(q_a, q_w, grp, S, ms, ns)
    assert got.shape == (ms.shape[0], S)
    for i, (m, n) in enumerate(zip(ms, ns)):
        for g in range(S):
            cols = grp == g
            want = int(q_a[m, cols].astype(np.int64) @ q_w[n, cols].astype(np.int64))
            assert got[i, g] == want, (i, g)
    full = oracle.mac(q_a, q_w, grp, S)
    np.testing.assert_array_equal(got, full[:, ms, ns].T.astype(np.int64))
    if S > 2:
        assert (got[:, S - 1] == 0).all()


def _bit_extract(words, j, c):
    per = 32 // c
    return (int(words[j // per]) >> ((j % per) * c)) & ((1 << c) - 1)


def _decode_field(f, bits, mode, c):
    if mode == oracle.SIGNED and bits == 1:
        return -1 if f else 1
    if mode == oracle.UNSIGNED:
        return f
    return f - (1 << c) if f >> (c - 1) else f


@pytest.mark.parametrize("wa,ww", list(itertools.product([1, 2, 4, 8], repeat=2)))
def test_tiny_brute_force_through_independent_bit_extraction(wa, ww):
    rng = np.random.default_rng(wa * 10 + ww)
    for M, N, K in [(1, 1, 1), (2, 3, 4), (4, 4, 3), (3, 2, 4)]:
        A = rng.standard_normal((M, K)).astype(np.float32)
        W = rng.standard_normal((N, K)).astype(np.float32)
        r = oracle.run(A, W, np.full(K, wa, np.uint8), np.full(N, ww, np.uint8), a_signed=True)
        ca, cw = oracle.container(wa), oracle.container(ww)
        ma = oracle.SIGNED
        qa = [[_decode_field(_bit_extract(oracle.pack(r["q_a"][m], wa, ma), k, ca), wa, ma, ca)
               for k in range(K)] for m in range(M)]
        qw = [[_decode_field(_bit_extract(oracle.pack(r["q_w"][n], ww, ma), k, cw), ww, ma, cw)
               for k in range(K)] for n in range(N)]
        for m in range(M):
            for n in range(N):
                assert r["acc"][0, m, n] == sum(qa[m][k] * qw[n][k] for k in range(K))


def test_permutation_and_zero_padding_invariance():
    """Reordering channels only clusters them (Alg. 1 permute); padding with
    zero channels leaves results unchanged (Fig. "normalization")."""
    rng = np.random.default_rng(21)
    M, N, K = 17, 19, 90
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((N, K)).astype(np.float32)
    ab = np.where(rng.random(K) < 0.5, 4, 8).astype(np.uint8)
    wb = np.where(rng.random(N) < 0.5, 2, 4).astype(np.uint8)
    base = oracle.run(A, W, ab, wb, a_signed=True)
    p = rng.permutation(K)
    r = oracle.run(A[:, p], W[:, p], ab[p], wb, a_signed=True)
    np.testing.assert_array_equal(r["acc"], base["acc"])
    np.testing.assert_array_equal(r["y_ref"], base["y_ref"])
    pn = rng.permutation(N)
    r = oracle.run(A, W[pn], ab, wb[pn], a_signed=True)
    np.testing.assert_array_equal(r["acc"], base["acc"][:, :, pn])
    pad = 13
    A2 = np.concatenate([A, np.zeros((M, pad), np.float32)], axis=1)
    W2 = np.concatenate([W, np.zeros((N, pad), np.float32)], axis=1)
    ab2 = np.concatenate([ab, np.full(pad, 4, np.uint8)])
    r = oracle.run(A2, W2, ab2, wb, a_signed=True)
    np.testing.assert_array_equal(r["acc"], base["acc"])
    np.testing.assert_array_equal(r["y_ref"], base["y_ref"])


# --------------------------------------------------------- O8 packing
@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("mode", [oracle.SIGNED, oracle.UNSIGNED, oracle.TWOS_FRACTION])
def test_pack_roundtrip_and_byte_count(bits, mode):
    if mode == oracle.UNSIGNED:
        codes = np.arange(0, 2 ** bits)
    elif mode == oracle.TWOS_FRACTION:
        codes = np.arange(-2 ** (bits - 1), 2 ** (bits - 1))
    elif bits == 1:
        codes = np.array([-1, 1])
    else:
        q = 2 ** (bits - 1) - 1
        codes = np.arange(-q, q + 1)
    codes = np.tile(codes, 7)[: 5 * 64 + 3]
    words = oracle.pack(codes, bits, mode)
    c = oracle.container(bits)
    assert c in (1, 2, 4, 8) and c >= bits and c < 2 * bits + (bits == 1)
    assert words.nbytes == 4 * -(-codes.size * c // 32)
    np.testing.assert_array_equal(oracle.unpack(words, codes.size, bits, mode), codes)


def test_bits_per_parameter_arithmetic():
    """Compression = 32 / bits-per-parameter (Sec. 6: 2.23 bpp ~ 14x)."""
    assert round(32 / 2.23) == 14
    # packed bytes of a two-level row set = sum of width * count / 8
    wb = np.array([2] * 3 + [4], np.uint8)
    K = 64
    total = sum(oracle.pack(np.zeros(K, np.int32), int(b), oracle.SIGNED).nbytes for b in wb)
    assert total == (3 * 2 + 4) * K // 8


# ------------------------------------------------------------ O7 bf16
def test_bf16_from_f32_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    ties = ((rng.integers(0, 2 ** 16, 4000, dtype=np.uint32) << 16) | 0x8000).view(np.float32)
    ties = ties[np.isfinite(ties)]           # exact ties: low 16 bits are 0x8000
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * np.float32(1e3),
                        ties]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    got = np.array([oracle.bf16_from_f32(v) for v in x], np.uint16)
    np.testing.assert_array_equal(got, ref)


def test_bf16_from_f64_is_nearest_even():
    rng = np.random.default_rng(6)
    vals = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-30, 30, 3000),
                           [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 1e-40, 3e-41]])
    for v in vals:
        b = oracle.bf16_from_f64(v)
        y = float(oracle.bf16_to_f32(np.array([b], np.uint16))[0])
        # neighbours of y in bf16
        lo = float(oracle.bf16_to_f32(np.array([b - 1 if b & 0x7FFF else b], np.uint16))[0])
        hi = float(oracle.bf16_to_f32(np.array([b + 1], np.uint16))[0])
        d = abs(y - v)
        assert d <= abs(lo - v) and d <= abs(hi - v), v
        if d == abs(lo - v) and lo != y or d == abs(hi - v) and hi != y:
            assert b % 2 == 0, v   # tie -> even mantissa


def test_epilogue_replay_matches_ref_within_rounding():
    rng = np.random.default_rng(8)
    acc = rng.integers(-2 ** 20, 2 ** 20, (2, 30, 40)).astype(np.int32)
    s_a = np.array([0.013, 0.0007], np.float32)
    s_w = rng.uniform(1e-3, 1.0, 40).astype(np.float32)
    yr = oracle.bf16_to_f32(oracle.epilogue_ref(acc, s_a, s_w)).astype(np.float64)
    yp = oracle.bf16_to_f32(oracle.epilogue_replay(acc, s_a, s_w)).astype(np.float64)
    exact = s_w[None, :].astype(np.float64) * (s_a[0] * acc[0].astype(np.float64) + s_a[1] * acc[1])
    assert (np.abs(yr - exact) <= np.abs(exact) * 2.0 ** -8 + 1e-30).all()
    assert (np.abs(yp - yr) <= np.abs(yr) * 2.0 ** -7 + 1e-30).all()


# ------------------------------------------------------ golden whole path
def test_hand_worked_example():
    sec = read_sections(os.path.join(GOLD, "hand_example.txt"))
    ab = np.array(sec["a_bits"][0], np.uint8)
    wb = np.array(sec["w_bits"][0], np.uint8)
    A = np.array(sec["A"], np.float32)
    W = np.array(sec["W"], np.float32)
    r = oracle.run(A, W, ab, wb, a_signed=True)
    np.testing.assert_array_equal(r["q_a"], np.array(sec["q_a"], np.int64))
    np.testing.assert_array_equal(r["q_w"], np.array(sec["q_w"], np.int64))
    np.testing.assert_array_equal(r["s_a"], np.array(sec["s_a"][0], np.float32))
    assert r["s_w"][0] == np.float32(0.4) and r["s_w"][1] == np.float32(0.125)
    np.testing.assert_array_equal(r["acc"][0], np.array(sec["acc0"], np.int64))
    np.testing.assert_array_equal(r["acc"][1], np.array(sec["acc1"], np.int64))
    want = np.array([[int(h, 16) for h in row] for row in sec["y_bf16_hex"]], np.uint16)
    np.testing.assert_array_equal(r["y_ref"], want)
    np.testing.assert_array_equal(r["y_replay"], want)


# ------------------------------------------- whole pipeline noise sanity
@pytest.mark.parametrize("ab,wb", [(4, 2), (8, 4), (4, 8)])
def test_uniform_noise_model_variance(ab, wb):
    """Sec. 2.3: quantization adds e ~ U[-D/2, D/2]; the error of y = A W^T
    must have the variance the model predicts (within a factor of 2)."""
    rng = np.random.default_rng(ab * 100 + wb)
    M, N, K = 64, 64, 512
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    r = oracle.run(A, W, np.full(K, ab, np.uint8), np.full(N, wb, np.uint8), a_signed=True)
    y_hat = r["s_w"][None, :].astype(np.float64) * r["s_a"][0] * r["acc"][0].astype(np.float64)
    y = A.astype(np.float64) @ W.astype(np.float64).T
    da = float(r["s_a"][0])
    dw = r["s_w"].astype(np.float64)
    pred = ((A.astype(np.float64) ** 2).sum(1)[:, None] * dw[None, :] ** 2 / 12
            + (W.astype(np.float64) ** 2).sum(1)[None, :] * da ** 2 / 12
            + K * da ** 2 * dw[None, :] ** 2 / 144)
    ratio = ((y_hat - y) ** 2).mean() / pred.mean()
    assert 0.5 < ratio < 2.0, ratio


def test_im2col_lowering_is_the_convolution():
    """The 3x3 stride-1 pad-1 lowering the convolution path is defined by:
    the lowered matrix times the flattened filters equals a convolution
    computed by direct loops over output pixels, channels and taps (fp64),
    on shapes with borders on every side and a 1x1 image."""
    import workloads
    rng = np.random.default_rng(11)
    for (B, C, H, W, N) in [(2, 3, 4, 5, 4), (1, 2, 1, 1, 3), (1, 1, 3, 1, 2)]:
        X = rng.standard_normal((B, C, H, W)).astype(np.float32)
        F = rng.standard_normal((N, C, 3, 3))
        direct = np.zeros((B, H, W, N))
        for b in range(B):
            for y in range(H):
                for x in range(W):
                    for n in range(N):
                        v = 0.0
                        for c in range(C):
                            for kh in range(3):
                                for kw in range(3):
                                    yy, xx = y + kh - 1, x + kw - 1
                                    if 0 <= yy < H and 0 <= xx < W:
                                        v += float(X[b, c, yy, xx]) * F[n, c, kh, kw]
                        direct[b, y, x, n] = v
        A = workloads.im2col_3x3(X).astype(np.float64)
        got = A @ F.reshape(N, C * 9).T
        np.testing.assert_allclose(got, direct.reshape(B * H * W, N), rtol=1e-12, atol=1e-12)


# ------------------------------------------------- sub-group activation scales
def test_grouped_without_blocks_is_the_precision_group_case():
    """GroupSize_act large enough for a whole precision group (or 0) gives
    one block per group: exactly the pinned per-group quantizer."""
    rng = np.random.default_rng(21)
    M, K = 9, 700
    A = rng.standard_normal((M, K)).astype(np.float32)
    ab = np.where(rng.random(K) < 0.6, 4, 8).astype(np.uint8)
    q0, s0, sb0, so0 = oracle.quantize_act(A, ab, True)
    for gb in (0, 8 * 1024):
        q, s, sb, so = oracle.quantize_act_grouped(A, ab, True, gb)
        np.testing.assert_array_equal(q, q0)
        np.testing.assert_array_equal(s, s0)
        np.testing.assert_array_equal(sb, sb0)
        np.testing.assert_array_equal(so, so0.astype(np.int32))


@pytest.mark.parametrize("signed", [True, False])
def test_grouped_blocks_are_independent_quantizations(signed):
    """With the narrow channels first in index order, the Alg. 1 order is
    the identity and every block is a contiguous column range: quantizing
    each range alone with the (pinned) per-group quantizer must give the
    block's codes and scale.  512-bit blocks: 128 channels at 4 bits, 64 at
    8 bits (widths 3 and 5 share containers 4 and 8)."""
    rng = np.random.default_rng(22 + signed)
    M = 7
    for lo, hi in ((4, 8), (3, 5)):
        n_lo, n_hi = 300, 150
        K = n_lo + n_hi
        A = (rng.standard_normal((M, K)) * rng.uniform(0.1, 10, K)).astype(np.float32)
        ab = np.array([lo] * n_lo + [hi] * n_hi, np.uint8)
        q, s, sb, so = oracle.quantize_act_grouped(A, ab, signed, 512)
        c_lo, c_hi = (4, 8)
        edges = []
        for start, n, c in ((0, n_lo, c_lo), (n_lo, n_hi, c_hi)):
            per = 512 // c
            edges += [(b, min(b + per, start + n)) for b in range(start, start + n, per)]
        assert len(s) == len(edges)
        for j, (b, e) in enumerate(edges):
            qj, sj, _, _ = oracle.quantize_act(A[:, b:e], ab[b:e], signed)
            np.testing.assert_array_equal(q[:, b:e], qj)
            assert s[j] == sj[0]
            assert (so[b:e] == j).all()
            assert sb[j] == ab[b]


def test_grouped_block_scale_is_equivariant():
    """Doubling every input of one block doubles that block's scale exactly
    and leaves all codes and every other scale unchanged; a channel put in
    the wrong block breaks this."""
    rng = np.random.default_rng(24)
    M, K = 6, 520
    A = rng.standard_normal((M, K)).astype(np.float32)
    ab = np.where(rng.random(K) < 0.7, 4, 8).astype(np.uint8)
    q, s, sb, so = oracle.quantize_act_grouped(A, ab, True, 512)
    for j in range(len(s)):
        B = A.copy()
        B[:, so == j] *= 2
        q2, s2, _, so2 = oracle.quantize_act_grouped(B, ab, True, 512)
        np.testing.assert_array_equal(q2, q)
        np.testing.assert_array_equal(so2, so)
        want = s.copy()
        want[j] *= 2
        np.testing.assert_array_equal(s2, want)


def test_grouped_block_maximum_maps_to_the_top_code():
    rng = np.random.default_rng(25)
    M, K = 5, 400
    A = rng.standard_normal((M, K)).astype(np.float32)
    ab = np.where(rng.random(K) < 0.5, 4, 8).astype(np.uint8)
    q, s, sb, so = oracle.quantize_act_grouped(A, ab, True, 512)
    for j in range(len(s)):
        cols = so == j
        blk = A[:, cols]
        i = np.unravel_index(np.argmax(np.abs(blk)), blk.shape)
        top = 2 ** (int(sb[j]) - 1) - 1
        assert abs(q[:, cols][i]) == top
        assert (np.abs(q[:, cols]) <= top).all()


def test_grouped_mac_is_the_blockwise_product():
    """ACC of block j is the integer product over the block's channels
    alone (numpy int64 matmul), and the blocks of a precision group add up
    to that group's accumulator."""
    rng = np.random.default_rng(26)
    M, N, K = 8, 12, 600
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    ab = np.where(rng.random(K) < 0.6, 4, 8).astype(np.uint8)
    wb = np.where(rng.random(N) < 0.5, 2, 8).astype(np.uint8)
    q_w, s_w = oracle.quantize_weights(W, wb)
    q, s, sb, so = oracle.quantize_act_grouped(A, ab, True, 512)
    acc = oracle.mac(q, q_w, so, len(s))
    for j in range(len(s)):
        cols = so == j
        want = q[:, cols].astype(np.int64) @ q_w[:, cols].astype(np.int64).T
        np.testing.assert_array_equal(acc[j], want)
    # the same codes summed per precision group instead of per block
    _, _, seg_bits, seg_of = oracle.quantize_act(A, ab, True)
    acc_seg = oracle.mac(q, q_w, seg_of, len(seg_bits))
    for g in range(len(seg_bits)):
        np.testing.assert_array_equal(acc[sb == seg_bits[g]].sum(0), acc_seg[g])


def test_grouped_epilogue_replay_matches_ref_within_rounding():
    """Many groups: the fixed-order fp32 replay stays within the bf16
    rounding of the fp64 reference (each product and sum adds at most
    2^-24 relative to the running magnitude)."""
    rng = np.random.default_rng(27)
    S = 25
    acc = rng.integers(-2 ** 18, 2 ** 18, (S, 20, 30)).astype(np.int32)
    s_a = rng.uniform(1e-3, 1e-1, S).astype(np.float32)
    s_w = rng.uniform(1e-3, 1.0, 30).astype(np.float32)
    yr = oracle.bf16_to_f32(oracle.epilogue_ref(acc, s_a, s_w)).astype(np.float64)
    yp = oracle.bf16_to_f32(oracle.epilogue_replay(acc, s_a, s_w)).astype(np.float64)
    terms = np.abs(s_a[:, None, None].astype(np.float64) * acc).sum(0) * s_w[None, :]
    assert (np.abs(yp - yr) <= np.abs(yr) * 2.0 ** -7 + terms * 2.0 ** -15).all()
    # two groups: the general replay is the two-group order of O7
    y2 = oracle.epilogue_replay(acc[:2], s_a[:2], s_w)
    t = (acc[0].astype(np.float32) * s_a[0]) + (acc[1].astype(np.float32) * s_a[1])
    t = t * s_w[None, :]
    np.testing.assert_array_equal(oracle.bf16_to_f32(y2), oracle.bf16_to_f32(
        np.array([[oracle.bf16_from_f32(v) for v in row] for row in t], np.uint16)))


# ------------------------------------------- static scales (quantize in a producer)
@pytest.mark.parametrize("signed", [True, False])
def test_static_scales_equal_to_the_batch_ones_give_its_codes(signed):
    """Given the scales the batch maximum produces, the static quantizer
    returns the pinned dynamic quantizer's codes; halving a scale doubles
    the pre-clamp ratio, so codes move to the clamp bound where they
    exceed it and stay within range."""
    rng = np.random.default_rng(31 + signed)
    M, K = 11, 333
    A = rng.standard_normal((M, K)).astype(np.float32)
    if not signed:
        A = np.abs(A)
    ab = np.where(rng.random(K) < 0.6, 4, 8).astype(np.uint8)
    q, s, sb, so = oracle.quantize_act(A, ab, signed)
    np.testing.assert_array_equal(oracle.quantize_act_static(A, ab, signed, s), q)
    q2 = oracle.quantize_act_static(A, ab, signed, s / 2)
    for g, b in enumerate(sb):
        top = (2 ** (int(b) - 1) - 1) if signed else (2 ** int(b) - 1)
        cols = so == g
        assert np.abs(q2[:, cols]).max() == top
        big = np.abs(A[:, cols]) / (s[g] / 2) >= top + 0.5
        assert (np.abs(q2[:, cols])[big] == top).all()


def test_replay_f32_rounds_to_the_replay():
    rng = np.random.default_rng(33)
    acc = rng.integers(-2 ** 20, 2 ** 20, (2, 17, 23)).astype(np.int32)
    s_a = np.array([0.013, 0.0007], np.float32)
    s_w = rng.uniform(1e-3, 1.0, 23).astype(np.float32)
    y32 = oracle.epilogue_replay_f32(acc, s_a, s_w)
    yb = oracle.epilogue_replay(acc, s_a, s_w)
    np.testing.assert_array_equal(
        np.array([[oracle.bf16_from_f32(v) for v in row] for row in y32], np.uint16), yb)


def test_static_block_scales_equal_to_the_batch_ones_give_its_codes():
    """Static scales per sub-group block, set to the blocks' batch scales,
    reproduce the pinned grouped quantizer's codes and blocks; doubling one
    block's static scale changes codes in that block only."""
    rng = np.random.default_rng(34)
    M, K = 9, 650
    A = (rng.standard_normal((M, K)) * rng.uniform(0.1, 10, K)).astype(np.float32)
    ab = np.where(rng.random(K) < 0.6, 4, 8).astype(np.uint8)
    q, s, sb, so = oracle.quantize_act_grouped(A, ab, True, 512)
    q2, so2 = oracle.quantize_act_static_grouped(A, ab, True, 512, s)
    np.testing.assert_array_equal(q2, q)
    np.testing.assert_array_equal(so2, so)
    s3 = s.copy()
    s3[1] *= 2
    q3, _ = oracle.quantize_act_static_grouped(A, ab, True, 512, s3)
    np.testing.assert_array_equal(q3[:, so != 1], q[:, so != 1])
    assert (q3[:, so == 1] != q[:, so == 1]).any()
