"""GPU parity of quantization fused into the producing GEMM
(soniq_mp_gemm_quantize_next; Sec. 4 fuses quantization into the operation
that produces the activations): the next layer's codes equal the oracle's
static-scale codes of this layer's fp32 outputs (before their bf16
rounding), its scales are the static ones, and the next layer's GEMM on
them matches the oracle bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu


def _bf16_bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def chain(M, K1, N1, N2, a1, w1, a2, w2, a2_signed, seed, scale_mul=1.0, with_y=True):
    l1 = workloads.generic(M, N1, K1, a_lo=a1[0], a_hi=a1[1], a_frac_lo=0.6, w_lo=w1[0],
                           w_hi=w1[1], w_frac_lo=0.7, a_signed=True, seed=seed, name="chain1")
    l2 = workloads.generic(M, N2, N1, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.7, w_lo=w2[0],
                           w_hi=w2[1], w_frac_lo=0.5, a_signed=a2_signed, seed=seed + 1,
                           name="chain2")
    print(f"[gpu] chain M={M} K1={K1} N1={N1} N2={N2} a2={a2} signed={a2_signed}", flush=True)
    # oracle: layer 1, its fp32 outputs, static-scale codes for layer 2
    r1 = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], True)
    y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])
    # calibration: the scales the batch maximum of y1 would give, scaled
    _, s_cal, _, _ = oracle.quantize_act(y1, l2["a_bits"], a2_signed)
    s2 = (s_cal * np.float32(scale_mul)).astype(np.float32)
    q2 = oracle.quantize_act_static(y1, l2["a_bits"], a2_signed, s2)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, seg_bits2, seg_of2 = oracle.segments(l2["a_bits"])
    acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
    # GPU
    W1 = torch.from_numpy(l1["W"]).cuda()
    W2 = torch.from_numpy(l2["W"]).cuda()
    A1 = torch.from_numpy(l1["A"]).cuda()
    wh1 = sq.soniq_pack_weights(W1, l1["w_bits"], l1["a_bits"], True)
    wh2 = sq.soniq_pack_weights(W2, l2["w_bits"], l2["a_bits"], a2_signed)
    act1 = sq.soniq_act_create(wh1, M)
    act2 = sq.soniq_act_create(wh2, M)
    sq.soniq_quantize_act(act1, A1)
    Y1 = torch.empty((M, N1), dtype=torch.bfloat16, device="cuda") if with_y else None
    sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, s2, out=Y1)
    acc = torch.empty((wh2.S, M, N2), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(act2, wh2, acc=acc)
    torch.cuda.synchronize()
    g_q2, g_s2 = sq.soniq_act_unpack_debug(act2)
    np.testing.assert_array_equal(g_s2, s2[:S2])
    np.testing.assert_array_equal(g_q2, q2)
    if with_y:
        np.testing.assert_array_equal(_bf16_bits(Y1), r1["y_replay"])
    np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
    np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2[:S2], s_w2))
    return dict(act1=act1, act2=act2, wh1=wh1, wh2=wh2, s2=s2, a_bits2=l2["a_bits"])


CHAINS = [  # (M, K1, N1, N2, a1, w1, a2, w2, a2_signed)
    (64, 256, 256, 128, (4, 8), (2, 4), (4, 8), (2, 8), True),
    (300, 200, 333, 70, (4, 8), (1, 4), (4, 8), (4, 8), False),   # unsigned next layer (zero point)
    (1, 128, 130, 64, (4, 8), (2, 8), (3, 6), (2, 4), True),       # one row, 4- and 8-bit containers
    (17, 96, 500, 100, (8, 8), (8, 8), (1, 8), (1, 4), True),      # 1-bit next-layer group
    (129, 300, 1000, 64, (4, 8), (2, 8), (2, 8), (2, 8), True),    # 2-bit next-layer group
    (70, 64, 5000, 16, (4, 8), (2, 4), (4, 8), (2, 4), True),      # 4-row packing (16 rows exceed 64 KB)
    # batches of at most 8 rows: the GEMV forms carry the epilogue
    (1, 4096, 1000, 300, (4, 8), (2, 4), (4, 8), (2, 4), True),    # decode row, nibble blocks
    (3, 700, 500, 100, (4, 8), (4, 8), (4, 8), (2, 8), False),     # byte blocks, unsigned next
    (8, 1000, 640, 96, (4, 8), (2, 8), (1, 8), (1, 4), True),      # 8 rows, 1-bit next group
    (1, 300, 200, 64, (4, 8), (1, 4), (4, 8), (2, 4), True),       # sign-bit producer weights
]


@pytest.mark.parametrize("c", CHAINS, ids=lambda c: f"M{c[0]}_K{c[1]}_N{c[2]}_a{c[6][0]}{c[6][1]}{'s' if c[8] else 'u'}")
def test_chain(c):
    chain(*c, seed=sum(c[:4]))


def test_chain_clamps_and_skips_y():
    """Scales below the calibrated ones clamp the largest outputs; no Y."""
    chain(200, 256, 384, 96, (4, 8), (2, 8), (4, 8), (2, 8), True, seed=5, scale_mul=0.5,
          with_y=False)


def test_chain_small_batch_skips_y():
    """A GEMV producer without Y, with scales below the calibrated ones."""
    chain(2, 640, 384, 96, (4, 8), (2, 8), (4, 8), (2, 8), True, seed=6, scale_mul=0.5,
          with_y=False)


def test_chain_repeat_and_other_producer():
    """A second call with fewer rows, then a different producer layer (other
    K, other weights) into the same next handle: its column table is
    rebuilt and the codes follow the new producer's outputs."""
    r = chain(150, 128, 256, 64, (4, 8), (2, 4), (4, 8), (2, 8), True, seed=9)
    A = torch.from_numpy(np.random.default_rng(3).standard_normal((40, 128)).astype(np.float32)).cuda()
    sq.soniq_quantize_act(r["act1"], A)
    sq.soniq_mp_gemm_quantize_next(r["act1"], r["wh1"], r["act2"], r["s2"])
    torch.cuda.synchronize()
    assert r["act2"].M == 40
    # another producer: K=96, N=256 (the next layer's K)
    pb = workloads.generic(33, 256, 96, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.6, a_signed=True, seed=44, name="producer_b")
    rb = oracle.run(pb["A"], pb["W"], pb["a_bits"], pb["w_bits"], True)
    yb = oracle.epilogue_replay_f32(rb["acc"], rb["s_a"], rb["s_w"])
    a_bits2 = r["a_bits2"]
    qb = oracle.quantize_act_static(yb, a_bits2, True, r["s2"])
    whb = sq.soniq_pack_weights(torch.from_numpy(pb["W"]).cuda(), pb["w_bits"], pb["a_bits"], True)
    actb = sq.soniq_act_create(whb, 33)
    sq.soniq_quantize_act(actb, torch.from_numpy(pb["A"]).cuda())
    sq.soniq_mp_gemm_quantize_next(actb, whb, r["act2"], r["s2"])
    torch.cuda.synchronize()
    g_q, _ = sq.soniq_act_unpack_debug(r["act2"])
    np.testing.assert_array_equal(g_q, qb)


def test_chain_tiles_and_gemv_forms_share_next():
    """One (producer, next) pair fed by the GEMM tiles (more than 8 rows) and
    by the GEMV forms (8 or fewer) in turn: the two write their codes in
    different layouts, and neither may leave a code where the other's
    layout keeps padding.  The next layer has a sign group, 1-bit weights
    and padded groups (K = 100), so a stray padding code would change its
    accumulators."""
    Mmax, K1, N1, N2 = 64, 192, 100, 48
    l1 = workloads.generic(Mmax, N1, K1, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.7, a_signed=True, seed=71, name="share1")
    l2 = workloads.generic(Mmax, N2, N1, a_lo=1, a_hi=8, a_frac_lo=0.7, w_lo=1, w_hi=4,
                           w_frac_lo=0.5, a_signed=True, seed=72, name="share2")
    r_all = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], True)
    y_all = oracle.epilogue_replay_f32(r_all["acc"], r_all["s_a"], r_all["s_w"])
    _, s2, _, _ = oracle.quantize_act(y_all, l2["a_bits"], True)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, _, seg_of2 = oracle.segments(l2["a_bits"])
    wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], True)
    act1 = sq.soniq_act_create(wh1, Mmax)
    act2 = sq.soniq_act_create(wh2, Mmax)
    for M in (64, 5, 40, 1, 64):
        print(f"[gpu] shared next handle, M={M}", flush=True)
        A = np.ascontiguousarray(l1["A"][:M])
        r1 = oracle.run(A, l1["W"], l1["a_bits"], l1["w_bits"], True)
        y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])
        q2 = oracle.quantize_act_static(y1, l2["a_bits"], True, s2)
        acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
        sq.soniq_quantize_act(act1, torch.from_numpy(A).cuda())
        sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, s2)
        acc = torch.empty((S2, M, N2), dtype=torch.int32, device="cuda")
        Y2 = sq.soniq_mp_gemm(act2, wh2, acc=acc)
        torch.cuda.synchronize()
        g_q, _ = sq.soniq_act_unpack_debug(act2)
        np.testing.assert_array_equal(g_q, q2)
        np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
        np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2, s_w2))


def test_chain_at_benchmark_size():
    """The two transformer linears bench.py --chain times (FFN up 4096 x 3072
    x 768, then FFN down 4096 x 768 x 3072), in its launch configuration:
    the layer-2 codes, scales, accumulators and outputs, bit for bit."""
    up, down = workloads.xfmr_ffn_up(), workloads.xfmr_ffn_down()
    M = up["M"]
    print(f"[gpu] chain at benchmark size M={M}", flush=True)
    r1 = oracle.run(up["A"], up["W"], up["a_bits"], up["w_bits"], True)
    y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])
    _, s2, _, _ = oracle.quantize_act(y1, down["a_bits"], down["a_signed"])
    q2 = oracle.quantize_act_static(y1, down["a_bits"], down["a_signed"], s2)
    q_w2, s_w2 = oracle.quantize_weights(down["W"], down["w_bits"])
    S2, _, seg_of2 = oracle.segments(down["a_bits"])
    acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
    wh1 = sq.soniq_pack_weights(torch.from_numpy(up["W"]).cuda(), up["w_bits"], up["a_bits"], True)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(down["W"]).cuda(), down["w_bits"], down["a_bits"],
                                down["a_signed"])
    a1, a2 = sq.soniq_act_create(wh1, M), sq.soniq_act_create(wh2, M)
    sq.soniq_quantize_act(a1, torch.from_numpy(up["A"]).cuda())
    sq.soniq_mp_gemm_quantize_next(a1, wh1, a2, s2)
    acc = torch.empty((S2, M, down["N"]), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(a2, wh2, acc=acc)
    torch.cuda.synchronize()
    g_q, g_s = sq.soniq_act_unpack_debug(a2)
    np.testing.assert_array_equal(g_s, s2)
    np.testing.assert_array_equal(g_q, q2)
    np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
    np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2, s_w2))


@pytest.mark.parametrize("c", [
    (64, 256, 768, 128, (4, 8), True, 512),
    (300, 200, 1000, 70, (3, 6), False, 1024),   # unsigned widths below their containers
    (5, 128, 600, 96, (4, 8), True, 512),
    (33, 96, 4000, 40, (2, 8), True, 512),       # 2-bit blocks of 256 channels; 1-row packing
    (1, 512, 900, 64, (4, 8), True, 512),        # one row through the GEMV into blocks
], ids=lambda c: f"M{c[0]}_N{c[2]}_a{c[4][0]}{c[4][1]}_g{c[6]}")
def test_chain_into_sub_group_scales(c):
    """The next layer packed with sub-group scales: one static scale per
    block; its codes, accumulators per block and outputs match the oracle."""
    M, K1, N1, N2, a2, signed2, gbits = c
    l1 = workloads.generic(M, N1, K1, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.7, a_signed=True, seed=M + N1, name="c1")
    l2 = workloads.generic(M, N2, N1, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.7, w_lo=2, w_hi=4,
                           w_frac_lo=0.5, a_signed=signed2, seed=M + N2, name="c2")
    print(f"[gpu] chain into blocks M={M} N1={N1} N2={N2} a2={a2} signed={signed2} g={gbits}", flush=True)
    r1 = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], True)
    y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])
    _, s_cal, _, _ = oracle.quantize_act_grouped(y1, l2["a_bits"], signed2, gbits)
    s2 = (s_cal * np.float32(0.8)).astype(np.float32)
    q2, sub_of = oracle.quantize_act_static_grouped(y1, l2["a_bits"], signed2, gbits, s2)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    acc2 = oracle.mac(q2, q_w2, sub_of, len(s2))
    wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], signed2,
                                act_group_bits=gbits)
    assert wh2.S == len(s2)
    a1, a2h = sq.soniq_act_create(wh1, M), sq.soniq_act_create(wh2, M)
    sq.soniq_quantize_act(a1, torch.from_numpy(l1["A"]).cuda())
    sq.soniq_mp_gemm_quantize_next(a1, wh1, a2h, s2)
    acc = torch.empty((wh2.S, M, N2), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(a2h, wh2, acc=acc)
    torch.cuda.synchronize()
    g_q, g_s = sq.soniq_act_unpack_debug(a2h)
    np.testing.assert_array_equal(g_s, s2)
    np.testing.assert_array_equal(g_q, q2)
    np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
    np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2, s_w2))


@pytest.mark.parametrize("c", [
    (64, 512, 256, 128, 512, 0, (4, 8), True),
    (300, 1000, 333, 70, 512, 0, (4, 8), False),     # unsigned next layer (zero point)
    (1, 768, 130, 64, 1024, 0, (2, 8), True),         # one row; 2-bit next-layer group
    (129, 768, 768, 96, 512, 512, (4, 8), True),      # blocks on both sides
    (33, 3072, 1000, 40, 512, 1024, (3, 6), False),   # 25 producer blocks; wide next blocks
    (6, 1024, 700, 80, 512, 512, (4, 8), True),       # block-sum GEMV producer into blocks
], ids=lambda c: f"M{c[0]}_K{c[1]}_N{c[2]}_g{c[4]}_next{c[5]}")
def test_chain_from_sub_group_scales(c):
    """The producing layer packed with sub-group scales (its per-block
    tiles carry the epilogue): the next layer's codes come from the fp32
    value (sum over blocks of f(ACC_j) s_a[j]) s_w, and its GEMM matches the
    oracle; Y and the producer's per-block sums match too."""
    M, K1, N1, N2, g1, g2, a2, signed2 = c
    l1 = workloads.generic(M, N1, K1, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.7, a_signed=True, seed=M + K1, name="gp1")
    l2 = workloads.generic(M, N2, N1, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.7, w_lo=2, w_hi=4,
                           w_frac_lo=0.5, a_signed=signed2, seed=M + N2, name="gp2")
    print(f"[gpu] chain from blocks M={M} K1={K1} N1={N1} N2={N2} g1={g1} g2={g2}", flush=True)
    # oracle: the grouped producer, its fp32 outputs, then the next layer
    q_a1, s_a1, _, sub1 = oracle.quantize_act_grouped(l1["A"], l1["a_bits"], True, g1)
    q_w1, s_w1 = oracle.quantize_weights(l1["W"], l1["w_bits"])
    acc1 = oracle.mac(q_a1, q_w1, sub1, len(s_a1))
    y1 = oracle.epilogue_replay_f32(acc1, s_a1, s_w1)
    if g2:
        _, s_cal, _, _ = oracle.quantize_act_grouped(y1, l2["a_bits"], signed2, g2)
        s2 = (s_cal * np.float32(0.8)).astype(np.float32)
        q2, sub2 = oracle.quantize_act_static_grouped(y1, l2["a_bits"], signed2, g2, s2)
    else:
        _, s_cal, _, _ = oracle.quantize_act(y1, l2["a_bits"], signed2)
        s2 = (s_cal * np.float32(0.8)).astype(np.float32)
        q2 = oracle.quantize_act_static(y1, l2["a_bits"], signed2, s2)
        S2, _, sub2 = oracle.segments(l2["a_bits"])
        s2 = s2[:S2]
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    acc2 = oracle.mac(q2, q_w2, sub2, len(s2))
    # GPU
    wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True,
                                act_group_bits=g1)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], signed2,
                                act_group_bits=g2)
    assert wh1.S == len(s_a1) and wh2.S == len(s2)
    h1, h2 = sq.soniq_act_create(wh1, M), sq.soniq_act_create(wh2, M)
    sq.soniq_quantize_act(h1, torch.from_numpy(l1["A"]).cuda())
    Y1 = torch.empty((M, N1), dtype=torch.bfloat16, device="cuda")
    acc1_g = torch.empty((wh1.S, M, N1), dtype=torch.int32, device="cuda")
    sq.soniq_mp_gemm_quantize_next(h1, wh1, h2, s2, out=Y1, acc=acc1_g)
    acc2_g = torch.empty((wh2.S, M, N2), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(h2, wh2, acc=acc2_g)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(acc1_g.cpu().numpy(), acc1)
    np.testing.assert_array_equal(_bf16_bits(Y1), oracle.epilogue_replay(acc1, s_a1, s_w1))
    g_q, g_s = sq.soniq_act_unpack_debug(h2)
    np.testing.assert_array_equal(g_s, s2)
    np.testing.assert_array_equal(g_q, q2)
    np.testing.assert_array_equal(acc2_g.cpu().numpy(), acc2)
    np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2, s_w2))


def test_graph_replay_after_another_producer():
    """A graph captured with producer A into a next handle, then an eager
    call from producer B into the same handle, then replays of A's graph:
    each replay's codes follow A's outputs (A's column table is still the
    one the graph holds), and a later eager call from B still follows B."""
    M, K1, N1, N2 = 96, 128, 256, 64
    la = workloads.generic(M, N1, K1, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.7, a_signed=True, seed=71, name="prod_a")
    lb = workloads.generic(M, N1, 96, a_lo=4, a_hi=8, a_frac_lo=0.5, w_lo=2, w_hi=4,
                           w_frac_lo=0.4, a_signed=True, seed=72, name="prod_b")
    l2 = workloads.generic(M, N2, N1, a_lo=4, a_hi=8, a_frac_lo=0.7, w_lo=2, w_hi=8,
                           w_frac_lo=0.5, a_signed=True, seed=73, name="next")
    print(f"[gpu] producer switch then replay M={M} N1={N1}", flush=True)

    def static_codes(l):
        r = oracle.run(l["A"], l["W"], l["a_bits"], l["w_bits"], True)
        return oracle.epilogue_replay_f32(r["acc"], r["s_a"], r["s_w"])

    ya, yb = static_codes(la), static_codes(lb)
    _, s2, _, _ = oracle.quantize_act(ya, l2["a_bits"], True)
    qa = oracle.quantize_act_static(ya, l2["a_bits"], True, s2)
    qb = oracle.quantize_act_static(yb, l2["a_bits"], True, s2)
    assert not np.array_equal(qa, qb)
    wa = sq.soniq_pack_weights(torch.from_numpy(la["W"]).cuda(), la["w_bits"], la["a_bits"], True)
    wb = sq.soniq_pack_weights(torch.from_numpy(lb["W"]).cuda(), lb["w_bits"], lb["a_bits"], True)
    w2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], True)
    ha, hb, h2 = sq.soniq_act_create(wa, M), sq.soniq_act_create(wb, M), sq.soniq_act_create(w2, M)
    Aa, Ab = torch.from_numpy(la["A"]).cuda(), torch.from_numpy(lb["A"]).cuda()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm: builds A's table outside the capture
        sq.soniq_quantize_act(ha, Aa)
        sq.soniq_mp_gemm_quantize_next(ha, wa, h2, s2)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        sq.soniq_quantize_act(ha, Aa)
        sq.soniq_mp_gemm_quantize_next(ha, wa, h2, s2)
    torch.cuda.synchronize()
    for r in range(3):
        sq.soniq_quantize_act(hb, Ab)
        sq.soniq_mp_gemm_quantize_next(hb, wb, h2, s2)   # eager, producer B
        torch.cuda.synchronize()
        np.testing.assert_array_equal(sq.soniq_act_unpack_debug(h2)[0], qb, err_msg=f"eager B {r}")
        g.replay()                                        # producer A, captured
        torch.cuda.synchronize()
        np.testing.assert_array_equal(sq.soniq_act_unpack_debug(h2)[0], qa, err_msg=f"replay A {r}")


def test_next_must_not_be_the_producers_handle():
    """A square layer fed back into its own activation handle would have its
    scales overwritten before the GEMM reads them: rejected, nothing run."""
    l = workloads.generic(64, 256, 256, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                          w_frac_lo=0.7, a_signed=True, seed=74, name="square")
    w = sq.soniq_pack_weights(torch.from_numpy(l["W"]).cuda(), l["w_bits"], l["a_bits"], True)
    h = sq.soniq_act_create(w, 64)
    sq.soniq_quantize_act(h, torch.from_numpy(l["A"]).cuda())
    with pytest.raises(sq.SoniqError) as e:
        sq.soniq_mp_gemm_quantize_next(h, w, h, np.ones(w.S, np.float32))
    assert e.value.status == sq.SONIQ_ERR_INVALID_ARGUMENT


def conv_chain(B, C1, H, W, N1, N2, a1, w1, a2, w2, a2_signed, implicit1, seed, with_y=False):
    """Conv -> conv (Sec. 4 fuses quantization into the convolution that
    produces the next one's input): layer 1 (implicit, or as a GEMM on its
    lowered matrix) quantizes its fp32 outputs with static scales straight
    into layer 2's haloed code image; layer 2 then runs as an implicit
    convolution.  Against the oracle: layer 2's lowered codes (the halo and
    border taps hold the code of 0.0), accumulators and outputs."""
    l1 = workloads.conv3x3(B, C1, H, W, N1, a_lo=a1[0], a_hi=a1[1], a_frac_lo=0.6, w_lo=w1[0],
                           w_hi=w1[1], w_frac_lo=0.7, a_signed=False, seed=seed)
    l2 = workloads.conv3x3(B, N1, H, W, N2, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.6, w_lo=w2[0],
                           w_hi=w2[1], w_frac_lo=0.5, a_signed=a2_signed, seed=seed + 1)
    M = B * H * W
    print(f"[gpu] conv chain B={B} C1={C1} {H}x{W} N1={N1} N2={N2} a2={a2} "
          f"signed={a2_signed} implicit={implicit1}", flush=True)
    r1 = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], False)
    y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])  # [M, N1], rows (b, y, x)
    X2 = np.ascontiguousarray(y1.reshape(B, H, W, N1).transpose(0, 3, 1, 2))
    A2 = workloads.im2col_3x3(X2)
    _, s2, _, _ = oracle.quantize_act(A2, l2["a_bits"], a2_signed)
    q2 = oracle.quantize_act_static(A2, l2["a_bits"], a2_signed, s2)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, _, seg_of2 = oracle.segments(l2["a_bits"])
    acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
    if implicit1:
        W1 = torch.from_numpy(np.ascontiguousarray(l1["W"].reshape(N1, C1, 3, 3))).cuda()
        wh1 = sq.soniq_pack_weights_conv3x3(W1, l1["w_bits"], l1["a_bits"][::9], False)
        act1 = sq.soniq_act_create_conv3x3(wh1, B, H, W)
        sq.soniq_quantize_act_conv3x3(act1, torch.from_numpy(l1["X"]).cuda())
    else:
        wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], False)
        act1 = sq.soniq_act_create(wh1, M)
        sq.soniq_quantize_act(act1, torch.from_numpy(l1["A"]).cuda())
    W2 = torch.from_numpy(np.ascontiguousarray(l2["W"].reshape(N2, N1, 3, 3))).cuda()
    wh2 = sq.soniq_pack_weights_conv3x3(W2, l2["w_bits"], l2["a_bits"][::9], a2_signed)
    act2 = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    Y1 = torch.empty((M, N1), dtype=torch.bfloat16, device="cuda") if with_y else None
    sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, s2, out=Y1)
    acc = torch.empty((S2, M, N2), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(act2, wh2, acc=acc)
    torch.cuda.synchronize()
    g_q2, g_s2 = sq.soniq_act_unpack_debug(act2)
    np.testing.assert_array_equal(g_s2, s2[:S2])
    np.testing.assert_array_equal(g_q2, q2)
    if with_y:
        np.testing.assert_array_equal(_bf16_bits(Y1), r1["y_replay"])
    np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
    np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2[:S2], s_w2))


CONV_CHAINS = [  # (B, C1, H, W, N1, N2, a1, w1, a2, w2, a2_signed, implicit1)
    (2, 16, 5, 7, 32, 24, (4, 8), (1, 4), (4, 8), (2, 4), False, True),   # implicit -> implicit
    (2, 16, 5, 7, 32, 24, (4, 8), (1, 4), (4, 8), (2, 4), False, False),  # lowered GEMM -> implicit
    (1, 20, 6, 9, 40, 130, (4, 8), (2, 8), (3, 6), (4, 8), True, True),   # signed 3/6-bit next
    (3, 8, 4, 4, 48, 16, (4, 8), (4, 8), (4, 8), (1, 4), False, True),    # 16 channels past a group
    (1, 12, 2, 2, 24, 16, (4, 8), (2, 4), (4, 8), (2, 4), False, False),  # 4 pixels: a GEMV producer
    (2, 16, 5, 7, 32, 24, (4, 8), (5, 8), (4, 8), (1, 8), True, True),    # 8/8 producer, 1/8 next
    (2, 16, 5, 7, 32, 24, (4, 8), (2, 4), (6, 6), (2, 8), True, True),    # one-width next (S = 1)
]


@pytest.mark.parametrize("c", CONV_CHAINS,
                         ids=lambda c: f"B{c[0]}_C{c[1]}_{c[2]}x{c[3]}_N{c[4]}_{'impl' if c[11] else 'gemm'}")
def test_conv_chain(c):
    conv_chain(*c, seed=sum(c[:6]))


def test_conv_chain_with_y():
    """The producer's Y as well as the next layer's codes."""
    conv_chain(3, 16, 6, 6, 32, 32, (4, 8), (1, 4), (4, 8), (2, 4), False, True, seed=5, with_y=True)


def test_conv_chain_smaller_batch_same_handles():
    """Three images, then one new image through the same producer and next
    handles: the second call's codes cover its one image (interior and
    halo) and its next-layer GEMM matches the oracle."""
    B, C1, H, W, N1, N2 = 3, 16, 5, 6, 32, 24
    l1 = workloads.conv3x3(B, C1, H, W, N1, w_lo=1, w_hi=4, seed=31)
    l2 = workloads.conv3x3(B, N1, H, W, N2, w_lo=2, w_hi=4, seed=77)
    W1 = torch.from_numpy(np.ascontiguousarray(l1["W"].reshape(N1, C1, 3, 3))).cuda()
    wh1 = sq.soniq_pack_weights_conv3x3(W1, l1["w_bits"], l1["a_bits"][::9], False)
    act1 = sq.soniq_act_create_conv3x3(wh1, B, H, W)
    W2 = torch.from_numpy(np.ascontiguousarray(l2["W"].reshape(N2, N1, 3, 3))).cuda()
    wh2 = sq.soniq_pack_weights_conv3x3(W2, l2["w_bits"], l2["a_bits"][::9], False)
    act2 = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, _, seg_of2 = oracle.segments(l2["a_bits"])
    s2 = np.array([0.05, 0.4], np.float32)
    X_one = np.abs(np.random.default_rng(5).standard_normal((1, C1, H, W)).astype(np.float32))
    for X in (l1["X"], X_one):
        b = X.shape[0]
        print(f"[gpu] conv chain on shared handles, {b} image(s)", flush=True)
        A1 = workloads.im2col_3x3(X)
        r1 = oracle.run(A1, l1["W"], l1["a_bits"], l1["w_bits"], False)
        y1 = oracle.epilogue_replay_f32(r1["acc"], r1["s_a"], r1["s_w"])
        A2 = workloads.im2col_3x3(np.ascontiguousarray(y1.reshape(b, H, W, N1).transpose(0, 3, 1, 2)))
        q2 = oracle.quantize_act_static(A2, l2["a_bits"], False, s2)
        acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
        sq.soniq_quantize_act_conv3x3(act1, torch.from_numpy(X).cuda())
        sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, s2)
        acc = torch.empty((S2, b * H * W, N2), dtype=torch.int32, device="cuda")
        Y2 = sq.soniq_mp_gemm(act2, wh2, acc=acc)
        torch.cuda.synchronize()
        g_q2, _ = sq.soniq_act_unpack_debug(act2)
        np.testing.assert_array_equal(g_q2, q2)
        np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
        np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2[:S2], s_w2))


def test_conv_chain_rejects_bad_batches():
    """A producer whose rows are not whole images of the next handle, or more
    images than it holds."""
    l1 = workloads.conv3x3(2, 8, 4, 4, 16, seed=3)
    l2 = workloads.conv3x3(1, 16, 4, 4, 16, seed=4)
    wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], False)
    W2 = torch.from_numpy(np.ascontiguousarray(l2["W"].reshape(16, 16, 3, 3))).cuda()
    wh2 = sq.soniq_pack_weights_conv3x3(W2, l2["w_bits"], l2["a_bits"][::9], False)
    act2 = sq.soniq_act_create_conv3x3(wh2, 1, 4, 4)
    act1 = sq.soniq_act_create(wh1, 32)
    for rows in (20, 32):  # not whole 4x4 images; two images into a one-image handle
        sq.soniq_quantize_act(act1, torch.from_numpy(l1["A"][:rows].copy()).cuda())
        with pytest.raises(sq.SoniqError) as e:
            sq.soniq_mp_gemm_quantize_next(act1, wh1, act2, [0.1, 0.2])
        assert e.value.status == sq.SONIQ_ERR_INVALID_ARGUMENT


def test_conv_chain_at_workload_size():
    """Two 256 -> 256 3x3 layers at 14x14, batch 32 (the CNN workload's
    shape), the first quantizing the second's input in its epilogue."""
    conv_chain(32, 256, 14, 14, 256, 256, (4, 8), (1, 4), (4, 8), (1, 4), False, True, seed=11)


def bf16_to_f32(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


MAX_CHAINS = [  # (M, K1, N1, N2, a1, w1, a2, w2, a2_signed)
    (300, 256, 384, 96, (4, 8), (2, 8), (4, 8), (2, 8), True),    # tiles, a partial last tile
    (64, 200, 130, 70, (4, 8), (1, 4), (4, 8), (4, 8), False),    # unsigned next; K2 % 4 != 0
    (129, 128, 256, 64, (4, 8), (2, 4), (1, 8), (1, 4), True),    # 1-bit next group
    (1, 512, 300, 64, (4, 8), (2, 4), (4, 8), (2, 4), True),      # one row: the GEMV form
    (8, 640, 384, 96, (4, 8), (2, 8), (3, 6), (2, 8), False),     # 8 rows, 3/6-bit next
]


@pytest.mark.parametrize("c", MAX_CHAINS, ids=lambda c: f"M{c[0]}_N{c[2]}_a{c[6][0]}{c[6][1]}{'s' if c[8] else 'u'}")
def test_chain_batch_max(c):
    """The two-pass form (soniq_mp_gemm_quantize_next_max): Y as
    soniq_mp_gemm stores it, and the next handle exactly as
    soniq_quantize_act would leave it for float(Y), against the oracle's
    quantize_act on the stored values (codec items 1-2 with the batch
    maximum), and the next layer's GEMM on them."""
    M, K1, N1, N2, a1, w1, a2, w2, a2_signed = c
    l1 = workloads.generic(M, N1, K1, a_lo=a1[0], a_hi=a1[1], a_frac_lo=0.6, w_lo=w1[0],
                           w_hi=w1[1], w_frac_lo=0.7, a_signed=True, seed=sum(c[:4]), name="max1")
    l2 = workloads.generic(M, N2, N1, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.7, w_lo=w2[0],
                           w_hi=w2[1], w_frac_lo=0.5, a_signed=a2_signed, seed=sum(c[:4]) + 1,
                           name="max2")
    print(f"[gpu] batch-max chain M={M} K1={K1} N1={N1} N2={N2} a2={a2}", flush=True)
    r1 = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], True)
    Y1f = bf16_to_f32(r1["y_replay"])
    q2, s2, _, _ = oracle.quantize_act(Y1f, l2["a_bits"], a2_signed)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, _, seg_of2 = oracle.segments(l2["a_bits"])
    acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
    wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], a2_signed)
    act1, act2, ref = sq.soniq_act_create(wh1, M), sq.soniq_act_create(wh2, M), sq.soniq_act_create(wh2, M)
    sq.soniq_quantize_act(act1, torch.from_numpy(l1["A"]).cuda())
    Y1 = sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2)
    acc = torch.empty((S2, M, N2), dtype=torch.int32, device="cuda")
    Y2 = sq.soniq_mp_gemm(act2, wh2, acc=acc)
    sq.soniq_quantize_act(ref, Y1.float())  # the unfused form on the same GPU
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bf16_bits(Y1), r1["y_replay"])
    g_q2, g_s2 = sq.soniq_act_unpack_debug(act2)
    r_q2, r_s2 = sq.soniq_act_unpack_debug(ref)
    np.testing.assert_array_equal(g_s2, s2)
    np.testing.assert_array_equal(g_q2, q2)
    np.testing.assert_array_equal(g_s2, r_s2)
    np.testing.assert_array_equal(g_q2, r_q2)
    np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
    np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2, s_w2))


def conv_chain_max(B, C1, H, W, N1, N2, a1, w1, a2, w2, a2_signed, implicit1, seed):
    """The two-pass form into a next convolution: layer 1 (implicit, or a
    GEMM on its lowered matrix) stores Y and folds its tiles' maxima, then
    layer 2's haloed code image is quantized from the stored bf16 Y with the
    batch maximum.  Against the oracle's quantize_act of the lowering of
    float(Y) (the lowering's zeros change no maximum), layer 2's
    accumulators and outputs, and the unfused form on the GPU
    (soniq_quantize_act_conv3x3 of float(Y) as NCHW)."""
    l1 = workloads.conv3x3(B, C1, H, W, N1, a_lo=a1[0], a_hi=a1[1], a_frac_lo=0.6, w_lo=w1[0],
                           w_hi=w1[1], w_frac_lo=0.7, a_signed=False, seed=seed)
    l2 = workloads.conv3x3(B, N1, H, W, N2, a_lo=a2[0], a_hi=a2[1], a_frac_lo=0.6, w_lo=w2[0],
                           w_hi=w2[1], w_frac_lo=0.5, a_signed=a2_signed, seed=seed + 1)
    M = B * H * W
    print(f"[gpu] conv batch-max chain B={B} C1={C1} {H}x{W} N1={N1} N2={N2} a2={a2} "
          f"signed={a2_signed} implicit={implicit1}", flush=True)
    r1 = oracle.run(l1["A"], l1["W"], l1["a_bits"], l1["w_bits"], False)
    Y1f = bf16_to_f32(r1["y_replay"])  # [M, N1], rows (b, y, x)
    X2 = np.ascontiguousarray(Y1f.reshape(B, H, W, N1).transpose(0, 3, 1, 2))
    A2 = workloads.im2col_3x3(X2)
    q2, s2, _, _ = oracle.quantize_act(A2, l2["a_bits"], a2_signed)
    q_w2, s_w2 = oracle.quantize_weights(l2["W"], l2["w_bits"])
    S2, _, seg_of2 = oracle.segments(l2["a_bits"])
    acc2 = oracle.mac(q2, q_w2, seg_of2, S2)
    if implicit1:
        W1 = torch.from_numpy(np.ascontiguousarray(l1["W"].reshape(N1, C1, 3, 3))).cuda()
        wh1 = sq.soniq_pack_weights_conv3x3(W1, l1["w_bits"], l1["a_bits"][::9], False)
        act1 = sq.soniq_act_create_conv3x3(wh1, B, H, W)
        sq.soniq_quantize_act_conv3x3(act1, torch.from_numpy(l1["X"]).cuda())
    else:
        wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], False)
        act1 = sq.soniq_act_create(wh1, M)
        sq.soniq_quantize_act(act1, torch.from_numpy(l1["A"]).cuda())
    W2 = torch.from_numpy(np.ascontiguousarray(l2["W"].reshape(N2, N1, 3, 3))).cuda()
    wh2 = sq.soniq_pack_weights_conv3x3(W2, l2["w_bits"], l2["a_bits"][::9], a2_signed)
    act2 = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    ref = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    for _ in range(2):  # the second call reuses the pair's table and image
        Y1 = sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2)
        acc = torch.empty((S2, M, N2), dtype=torch.int32, device="cuda")
        Y2 = sq.soniq_mp_gemm(act2, wh2, acc=acc)
        Xg = Y1.float().reshape(B, H, W, N1).permute(0, 3, 1, 2).contiguous()
        sq.soniq_quantize_act_conv3x3(ref, Xg)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bf16_bits(Y1), r1["y_replay"])
        g_q2, g_s2 = sq.soniq_act_unpack_debug(act2)
        r_q2, r_s2 = sq.soniq_act_unpack_debug(ref)
        np.testing.assert_array_equal(g_s2, s2[:S2])
        np.testing.assert_array_equal(g_q2, q2)
        np.testing.assert_array_equal(g_s2, r_s2)
        np.testing.assert_array_equal(g_q2, r_q2)
        np.testing.assert_array_equal(acc.cpu().numpy(), acc2)
        np.testing.assert_array_equal(_bf16_bits(Y2), oracle.epilogue_replay(acc2, s2[:S2], s_w2))


@pytest.mark.parametrize("c", CONV_CHAINS,
                         ids=lambda c: f"B{c[0]}_C{c[1]}_{c[2]}x{c[3]}_N{c[4]}_{'impl' if c[11] else 'gemm'}")
def test_conv_chain_batch_max(c):
    conv_chain_max(*c, seed=sum(c[:6]) + 11)


def test_chain_batch_max_repeats_and_graph():
    """Repeated calls (the slots are cleared each time, a smaller batch
    second), then the call captured in a HIP graph and replayed three times
    with eager work between the replays, each against the eager result."""
    l1 = workloads.generic(200, 256, 192, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.7, a_signed=True, seed=91, name="maxg1")
    l2 = workloads.generic(200, 64, 256, a_lo=4, a_hi=8, a_frac_lo=0.7, w_lo=2, w_hi=4,
                           w_frac_lo=0.5, a_signed=True, seed=92, name="maxg2")
    wh1 = sq.soniq_pack_weights(torch.from_numpy(l1["W"]).cuda(), l1["w_bits"], l1["a_bits"], True)
    wh2 = sq.soniq_pack_weights(torch.from_numpy(l2["W"]).cuda(), l2["w_bits"], l2["a_bits"], True)
    act1, act2, ref = sq.soniq_act_create(wh1, 200), sq.soniq_act_create(wh2, 200), sq.soniq_act_create(wh2, 200)
    A = torch.from_numpy(l1["A"]).cuda()
    for rows in (200, 70):
        sq.soniq_quantize_act(act1, A[:rows].contiguous())
        Y1 = sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2)
        sq.soniq_quantize_act(ref, Y1.float())
        torch.cuda.synchronize()
        np.testing.assert_array_equal(sq.soniq_act_unpack_debug(act2)[0], sq.soniq_act_unpack_debug(ref)[0])
        np.testing.assert_array_equal(sq.soniq_act_unpack_debug(act2)[1], sq.soniq_act_unpack_debug(ref)[1])
    Ag = A[:150].contiguous()
    Yg = torch.empty((150, 256), dtype=torch.bfloat16, device="cuda")
    Y2 = torch.empty((150, 64), dtype=torch.bfloat16, device="cuda")
    sq.soniq_quantize_act(act1, Ag)
    sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2, out=Yg)
    sq.soniq_mp_gemm(act2, wh2, out=Y2)
    torch.cuda.synchronize()
    eager = _bf16_bits(Y2).copy()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        sq.soniq_quantize_act(act1, Ag, stream=s.cuda_stream)
        sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2, out=Yg, stream=s.cuda_stream)
        sq.soniq_mp_gemm(act2, wh2, out=Y2, stream=s.cuda_stream)
    for _ in range(3):
        Y2.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bf16_bits(Y2), eager)


def test_conv_chain_batch_max_smaller_batch_and_graph():
    """The two-pass form into a next convolution on handles made for three
    images, called with three then two (the unfused form on the same
    stored Y as reference), then captured in a HIP graph and replayed three
    times with eager work between the replays, each against the eager
    result."""
    B, C1, H, W, N1, N2 = 3, 16, 6, 7, 32, 24
    l1 = workloads.conv3x3(B, C1, H, W, N1, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=1, w_hi=4,
                           w_frac_lo=0.7, a_signed=False, seed=301)
    l2 = workloads.conv3x3(B, N1, H, W, N2, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                           w_frac_lo=0.5, a_signed=True, seed=302)
    W1 = torch.from_numpy(np.ascontiguousarray(l1["W"].reshape(N1, C1, 3, 3))).cuda()
    wh1 = sq.soniq_pack_weights_conv3x3(W1, l1["w_bits"], l1["a_bits"][::9], False)
    W2 = torch.from_numpy(np.ascontiguousarray(l2["W"].reshape(N2, N1, 3, 3))).cuda()
    wh2 = sq.soniq_pack_weights_conv3x3(W2, l2["w_bits"], l2["a_bits"][::9], True)
    act1 = sq.soniq_act_create_conv3x3(wh1, B, H, W)
    act2 = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    ref = sq.soniq_act_create_conv3x3(wh2, B, H, W)
    X = torch.from_numpy(l1["X"]).cuda()
    for nb in (3, 2):
        print(f"[gpu] conv batch-max on {nb} of {B} images", flush=True)
        sq.soniq_quantize_act_conv3x3(act1, X[:nb].contiguous())
        Y1 = sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2)
        sq.soniq_quantize_act_conv3x3(ref, Y1.float().reshape(nb, H, W, N1).permute(0, 3, 1, 2).contiguous())
        torch.cuda.synchronize()
        g_q, g_s = sq.soniq_act_unpack_debug(act2)
        r_q, r_s = sq.soniq_act_unpack_debug(ref)
        np.testing.assert_array_equal(g_s, r_s)
        np.testing.assert_array_equal(g_q, r_q)
    Xg = X[:2].contiguous()
    M = 2 * H * W
    Yg = torch.empty((M, N1), dtype=torch.bfloat16, device="cuda")
    Y2 = torch.empty((M, N2), dtype=torch.bfloat16, device="cuda")
    sq.soniq_quantize_act_conv3x3(act1, Xg)
    sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2, out=Yg)
    sq.soniq_mp_gemm(act2, wh2, out=Y2)
    torch.cuda.synchronize()
    eager = _bf16_bits(Y2).copy()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=s):
        sq.soniq_quantize_act_conv3x3(act1, Xg, stream=s.cuda_stream)
        sq.soniq_mp_gemm_quantize_next_max(act1, wh1, act2, out=Yg, stream=s.cuda_stream)
        sq.soniq_mp_gemm(act2, wh2, out=Y2, stream=s.cuda_stream)
    for _ in range(3):
        Y2.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(_bf16_bits(Y2), eager)
