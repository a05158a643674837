"""GPU parity of sub-group activation scales (GroupSize_act blocks, the
design-space parameter of Sec. 3; Sec. 5 uses 512-bit activation groups):
codes, block scales and every per-block int32 accumulator bit-exact against
the oracle; bf16 outputs equal its fixed-order fp32 replay over the blocks
and lie within the fp64 reference's tolerance."""
import numpy as np
import pytest
import torch

import oracle
import paper_2311_14114_amd as sq
import workloads

pytestmark = pytest.mark.gpu


def _bf16_bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def gpu_run(case, group_bits):
    M, N, K = case["M"], case["N"], case["K"]
    print(f"[gpu] grouped {case['name']} M={M} N={N} K={K} bits={group_bits}", flush=True)
    W = torch.from_numpy(case["W"]).cuda()
    A = torch.from_numpy(case["A"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], case["a_signed"],
                              act_group_bits=group_bits)
    act = sq.soniq_act_create(w, M)
    acc = torch.empty((w.S, M, N), dtype=torch.int32, device="cuda")
    Y = sq.soniq_quantize_mp_gemm(act, w, A, acc=acc)
    torch.cuda.synchronize()
    q_a, s_a = sq.soniq_act_unpack_debug(act)
    return dict(S=w.S, info=w.info, y=_bf16_bits(Y), acc=acc.cpu().numpy(), q_a=q_a, s_a=s_a,
                w=w, act=act, Y=Y)


def oracle_run(case, group_bits):
    q_w, s_w = oracle.quantize_weights(case["W"], case["w_bits"])
    q_a, s_a, sub_bits, sub_of = oracle.quantize_act_grouped(case["A"], case["a_bits"],
                                                             case["a_signed"], group_bits)
    acc = oracle.mac(q_a, q_w, sub_of, len(s_a))
    return dict(S=len(s_a), q_a=q_a, s_a=s_a, s_w=s_w, acc=acc,
                y_ref=oracle.epilogue_ref(acc, s_a, s_w),
                y_replay=oracle.epilogue_replay(acc, s_a, s_w))


def compare(g, r):
    assert g["S"] == r["S"]
    np.testing.assert_array_equal(g["s_a"], r["s_a"])
    np.testing.assert_array_equal(g["q_a"], r["q_a"])
    np.testing.assert_array_equal(g["acc"], r["acc"])
    np.testing.assert_array_equal(g["y"], r["y_replay"])
    yg = oracle.bf16_to_f32(g["y"]).astype(np.float64)
    yr = oracle.bf16_to_f32(r["y_ref"]).astype(np.float64)
    T = np.abs(r["s_w"].astype(np.float64))[None, :] * sum(
        np.abs(float(r["s_a"][j]) * r["acc"][j].astype(np.float64)) for j in range(r["S"]))
    bad = np.abs(yg - yr) > np.maximum(1e-2 * np.abs(yr), 2.0 ** -15 * T)
    assert not bad.any(), f"{bad.sum()} outputs outside tolerance"


SHAPES = [  # (M, N, K, a_lo, a_hi, w_lo, w_hi, a_signed, group_bits)
    (64, 256, 768, 4, 8, 2, 8, True, 512),
    (37, 130, 600, 4, 8, 1, 4, True, 512),      # ragged rows, 1-bit weights
    (300, 200, 1000, 3, 5, 2, 4, False, 512),   # unsigned widths below their containers
    (5, 70, 129, 4, 8, 4, 8, True, 1024),       # a few rows: the block-sum GEMV
    (129, 300, 2000, 2, 8, 2, 8, True, 512),    # 2-bit activations: 256-channel blocks
    (260, 128, 4096, 4, 8, 2, 4, True, 512),    # 4-row quantizer (16 code rows exceed 64 KB)
    (1, 64, 64, 8, 8, 8, 8, True, 512),         # one block
    (1030, 70, 333, 4, 7, 2, 8, True, 1536),    # blocks of 3 granules, ragged 16-row block
    (20, 64, 15000, 8, 8, 4, 4, True, 512),     # 235 blocks
    (24, 130, 16384, 8, 8, 2, 8, True, 512),    # 256 blocks: the most a handle takes
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s[:3])) + f"_a{s[3]}{s[4]}w{s[5]}{s[6]}{'s' if s[7] else 'u'}_g{s[8]}")
def test_grouped_shapes(shape):
    M, N, K, alo, ahi, wlo, whi, sgn, gb = shape
    case = workloads.generic(M, N, K, a_lo=alo, a_hi=ahi, a_frac_lo=0.6, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.7, a_signed=sgn, seed=M * 7 + N + K, a_abs=not sgn,
                             name="grouped")
    # spread the channel magnitudes so that block scales differ widely
    rng = np.random.default_rng(K)
    case["A"] = (case["A"] * rng.uniform(0.05, 20.0, K).astype(np.float32)).astype(np.float32)
    compare(gpu_run(case, gb), oracle_run(case, gb))


def test_grouped_zero_block():
    """A block whose inputs are all zero has scale 0 and codes 0."""
    case = workloads.generic(70, 96, 700, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                             w_frac_lo=0.5, a_signed=True, seed=5, name="zero_block")
    _, _, _, sub_of = oracle.quantize_act_grouped(case["A"], case["a_bits"], True, 512)
    case["A"][:, sub_of == 1] = 0.0
    g, r = gpu_run(case, 512), oracle_run(case, 512)
    assert r["s_a"][1] == 0.0
    compare(g, r)


GEMV_SHAPES = [  # (M, N, K, w_lo, w_hi, group_bits): batches of up to 8 rows
    (1, 200, 1000, 2, 4, 512),
    (1, 130, 4100, 2, 8, 512),
    (1, 96, 2000, 4, 8, 1024),
    (1, 64, 700, 8, 8, 512),
    (1, 70, 20000, 2, 4, 512),     # several staging rounds, 157 blocks
    (2, 150, 1500, 2, 8, 512),
    (3, 100, 900, 4, 8, 1536),     # blocks of three granules
    (5, 333, 1200, 2, 4, 512),
    (8, 128, 3000, 2, 8, 512),
]


@pytest.mark.parametrize("shape", GEMV_SHAPES, ids=lambda s: "x".join(map(str, s[:3])) + f"_w{s[3]}{s[4]}_g{s[5]}")
def test_grouped_gemv(shape, monkeypatch):
    """Batches of at most 8 rows take the block-sum GEMV: every per-block
    accumulator and output against the oracle, and bit for bit against the
    MFMA tiles on the same handles."""
    M, N, K, wlo, whi, gb = shape
    case = workloads.generic(M, N, K, a_lo=4, a_hi=8, a_frac_lo=0.7, w_lo=wlo, w_hi=whi,
                             w_frac_lo=0.6, a_signed=True, seed=M * 13 + N + K, name="grouped_gemv")
    rng = np.random.default_rng(K + M)
    case["A"] = (case["A"] * rng.uniform(0.05, 20.0, K).astype(np.float32)).astype(np.float32)
    g = gpu_run(case, gb)
    compare(g, oracle_run(case, gb))
    monkeypatch.setenv("SONIQ_GROUPED_MFMA", "1")
    acc = torch.empty_like(torch.from_numpy(g["acc"])).cuda()
    Y = sq.soniq_mp_gemm(g["act"], g["w"], acc=acc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_bf16_bits(Y), g["y"])
    np.testing.assert_array_equal(acc.cpu().numpy(), g["acc"])


@pytest.mark.parametrize("name", ["xfmr_qkv_g512", "xfmr_ffn_down_g512", "decode_11008_m1_g512",
                                  "decode_11008_m8_g512"])
def test_grouped_workload_parity(name):
    case = workloads.make(name)
    compare(gpu_run(case, case["act_group_bits"]), oracle_run(case, case["act_group_bits"]))


def test_blocks_spanning_whole_groups_match_the_plain_path():
    """Blocks as large as the precision groups: the grouped kernels give
    the plain path's output bits and accumulators."""
    case = workloads.generic(200, 192, 900, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=4,
                             w_frac_lo=0.6, a_signed=True, seed=11, name="whole")
    g = gpu_run(case, 8192)
    assert g["S"] == 2
    W = torch.from_numpy(case["W"]).cuda()
    A = torch.from_numpy(case["A"]).cuda()
    w = sq.soniq_pack_weights(W, case["w_bits"], case["a_bits"], True)
    act = sq.soniq_act_create(w, case["M"])
    acc = torch.empty((2, case["M"], case["N"]), dtype=torch.int32, device="cuda")
    Y = sq.soniq_quantize_mp_gemm(act, w, A, acc=acc)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(g["y"], _bf16_bits(Y))
    np.testing.assert_array_equal(g["acc"], acc.cpu().numpy())


def test_grouped_repeat_calls_and_rejections():
    """Second call with fewer rows reuses the handle; the conv entry point
    refuses grouped weights."""
    case = workloads.generic(300, 130, 520, a_lo=4, a_hi=8, a_frac_lo=0.6, w_lo=2, w_hi=8,
                             w_frac_lo=0.5, a_signed=True, seed=12, name="repeat")
    g = gpu_run(case, 512)
    small = dict(case)
    small["M"], small["A"] = 33, np.ascontiguousarray(case["A"][:33] * np.float32(3.0))
    A = torch.from_numpy(small["A"]).cuda()
    acc = torch.empty((g["S"], 33, case["N"]), dtype=torch.int32, device="cuda")
    Y = sq.soniq_quantize_mp_gemm(g["act"], g["w"], A, acc=acc)
    torch.cuda.synchronize()
    q_a, s_a = sq.soniq_act_unpack_debug(g["act"])
    r = oracle_run(small, 512)
    compare(dict(S=g["S"], y=_bf16_bits(Y), acc=acc.cpu().numpy(), q_a=q_a, s_a=s_a), r)
    X = torch.zeros((1, 4, 4, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(sq.SoniqError):
        sq.soniq_quantize_act_conv3x3(g["act"], X)


@pytest.mark.parametrize("mode", ["single_pass", "two_pass", "wait_timeout"])
def test_grouped_quantizer_paths(mode, monkeypatch):
    """A batch large enough for the single pass (M*K >= 2^20), through the
    single pass, the two-pass form, and the single pass whose grid wait
    gives up at once (every workgroup then takes the block maxima itself):
    the same codes, scales and outputs as the oracle."""
    if mode == "two_pass":
        monkeypatch.setenv("SONIQ_ACT_COOP", "0")
    if mode == "wait_timeout":
        monkeypatch.setenv("SONIQ_COOP_SPINS", "0")
    case = workloads.generic(1536, 256, 1024, a_lo=4, a_hi=8, a_frac_lo=0.7, w_lo=2, w_hi=8,
                             w_frac_lo=0.7, a_signed=True, seed=31, name="grouped_paths")
    rng = np.random.default_rng(1024)
    case["A"] = (case["A"] * rng.uniform(0.05, 20.0, 1024).astype(np.float32)).astype(np.float32)
    g = gpu_run(case, 512)
    compare(g, oracle_run(case, 512))
    stalls = sq.soniq_act_wait_timeouts(g["act"])
    assert stalls >= 1 if mode == "wait_timeout" else stalls == 0
    if mode == "single_pass":
        # unsigned widths below their containers, and a second call
        case2 = dict(case)
        case2["A"] = np.abs(case["A"])
        case2["a_bits"] = np.where(case["a_bits"] == 4, 3, 6).astype(np.uint8)
        case2["a_signed"] = False
        compare(gpu_run(case2, 1024), oracle_run(case2, 1024))
