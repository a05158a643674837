"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/soniq.h declares, validates arguments before touching the device,
and plans input channels on the host (Alg. 1 permutation, Fig.
"normalization" padding)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2311_14114_amd as sq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sq.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return sq.lib()


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "soniq.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(soniq_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    decl = declared_symbols()
    assert len(decl) >= 12
    assert sorted(sq.EXPORTED) == decl
    for name in decl:
        assert hasattr(L, name), name


def test_stream_read_validation(L):
    fake = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first
    for src, n, sink in ((None, 64, fake), (fake, 64, None), (fake, 0, fake), (fake, 24, fake),
                         (ctypes.c_void_p(0x1008), 64, fake), (fake, 1 << 31, fake)):
        assert L.soniq_debug_stream_read(src, n, sink, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert b"soniq_debug_stream_read" in L.soniq_last_error()


def _pack(L, W, N, K, ldw, wb, ab, a_signed=1, mode=0):
    h = ctypes.c_void_p()
    rc = L.soniq_pack_weights_ex(W, N, K, ldw, wb, ab, a_signed, mode, None, ctypes.byref(h))
    return rc, h


def test_validation_before_any_device_work(L):
    fake = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first
    wb = np.full(4, 4, np.uint8)
    ab = np.full(4, 8, np.uint8)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    assert _pack(L, None, 4, 4, 4, p(wb), p(ab))[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert b"null" in L.soniq_last_error()
    assert _pack(L, fake, 0, 4, 4, p(wb), p(ab))[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert _pack(L, fake, 4, 4, 3, p(wb), p(ab))[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert b"ldw" in L.soniq_last_error()
    for bad in ([0, 4, 4, 4], [9, 4, 4, 4], [1, 2, 4, 4]):
        b = np.array(bad, np.uint8)
        assert _pack(L, fake, 4, 4, 4, p(b), p(ab))[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
        assert _pack(L, fake, 4, 4, 4, p(wb), p(b))[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert _pack(L, fake, 4, 4, 4, p(wb), p(ab), a_signed=2)[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert _pack(L, fake, 4, 4, 4, p(wb), p(ab), mode=7)[0] == sq.SONIQ_ERR_INVALID_ARGUMENT
    # accumulator-exactness limit on the padded channel count
    K = sq.SONIQ_MAX_K + 1
    abig = np.full(K, 4, np.uint8)
    assert _pack(L, fake, 4, K, K, p(wb), p(abig))[0] == sq.SONIQ_ERR_UNSUPPORTED
    K = sq.SONIQ_MAX_K - 10             # fits alone, but two padded groups do not
    abig = np.full(K, 4, np.uint8)
    abig[:40] = 8
    assert _pack(L, fake, 4, K, K, p(wb), p(abig))[0] == sq.SONIQ_ERR_UNSUPPORTED


def test_null_handles_are_rejected(L):
    h = ctypes.c_void_p()
    assert L.soniq_act_create(None, 4, ctypes.byref(h)) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert L.soniq_quantize_act(None, ctypes.c_void_p(0x1000), 1, 1, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert L.soniq_quantize_act_conv3x3(None, ctypes.c_void_p(0x1000), 1, 1, 1, 1, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert L.soniq_mp_gemm(None, None, ctypes.c_void_p(0x1000), 1, None, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert L.soniq_weights_info(None, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert L.soniq_weights_unpack_debug(None, None, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert L.soniq_act_unpack_debug(None, None, None) == sq.SONIQ_ERR_INVALID_ARGUMENT
    L.soniq_weights_destroy(None)
    L.soniq_act_destroy(None)


@pytest.mark.parametrize("seed", range(6))
def test_input_channel_plan_matches_definition(L, seed):
    rng = np.random.default_rng(seed)
    K = int(rng.integers(1, 700))
    lo, hi = sorted(rng.choice(np.arange(1, 9), 2, replace=False))
    ab = np.where(rng.random(K) < rng.random(), lo, hi).astype(np.uint8)
    pos, seg_len, seg_pad, S = sq.soniq_plan_input_channels(ab)
    widths = sorted(set(ab.tolist()))
    assert S == len(widths)
    # definition: narrow group first, original order inside a group, each
    # group padded with zero channels to a multiple of 64
    order = [k for k in range(K) if ab[k] == widths[0]] + [k for k in range(K) if S == 2 and ab[k] == widths[1]]
    n0 = int((ab == widths[0]).sum())
    pad0 = -(-n0 // 64) * 64
    want = np.empty(K, np.int64)
    for r, k in enumerate(order):
        want[k] = r if r < n0 else pad0 + (r - n0)
    np.testing.assert_array_equal(pos, want)
    assert seg_len[0] == n0 and seg_pad[0] == pad0
    assert seg_len[1] == K - n0 and seg_pad[1] == -(-(K - n0) // 64) * 64
    assert len(set(pos.tolist())) == K


def test_grouped_pack_validation(L):
    """Sub-group scale requests are checked before any device work."""
    fake = ctypes.c_void_p(0x1000)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    wb = np.full(4, 4, np.uint8)

    def pack(ab, signed, bits):
        h = ctypes.c_void_p()
        K = ab.shape[0]
        return L.soniq_pack_weights_grouped(fake, 4, K, K, p(wb), p(ab), signed, 0, bits, None,
                                            ctypes.byref(h))
    ab4 = np.full(256, 4, np.uint8)
    assert pack(ab4, 1, 100) == sq.SONIQ_ERR_INVALID_ARGUMENT
    assert b"512" in L.soniq_last_error()
    assert pack(ab4, 1, -512) == sq.SONIQ_ERR_INVALID_ARGUMENT
    # unsigned 4-bit codes fill their container: zero point, not supported
    assert pack(ab4, 0, 512) == sq.SONIQ_ERR_UNSUPPORTED
    assert b"zero point" in L.soniq_last_error()
    assert pack(np.full(256, 1, np.uint8), 1, 512) == sq.SONIQ_ERR_UNSUPPORTED
    # 300 blocks of 64 8-bit channels
    assert pack(np.full(64 * 300, 8, np.uint8), 1, 512) == sq.SONIQ_ERR_UNSUPPORTED
    assert b"blocks" in L.soniq_last_error()
