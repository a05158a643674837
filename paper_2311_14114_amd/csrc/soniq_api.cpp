// Host side of libsoniq: argument validation, the input-channel and
// output-channel plans, device buffers, dispatch and debug readback.
//
// Input-channel plan (Alg. 1 channel permutation; Fig. "normalization"):
// the activation widths define at most two groups (C3), ordered narrow then
// wide; within a group channels keep their original order; each group is
// padded with zero channels to a multiple of 64 (one MFMA k-step) so every
// group starts on a fresh granule of every packed row.
//
// Output-channel plan (C1: one width per 16-row block): the channels of
// each weight width, in original order, are cut into blocks of 16 (the
// last block of a width padded with empty rows); all blocks of the narrow
// width come first, padded with empty blocks to a multiple of 8 (one
// 128-column GEMM tile), then those of the wide width, padded the same way.
// So every GEMM tile holds one width, and since blocks are contiguous a
// kernel derives any block's container and byte offset from the plan alone
// (WPlan::nlo, c_lo, c_hi, ngt) without reading a table.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "soniq.h"
#include "soniq_internal.h"

using namespace soniq;

namespace {

thread_local std::string g_err;

soniq_status fail(soniq_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

soniq_status fail_hip(hipError_t e, const char* what) {
  return fail(e == hipErrorOutOfMemory ? SONIQ_ERR_OUT_OF_MEMORY : SONIQ_ERR_HIP,
              "%s failed: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr)                                   \
  do {                                                  \
    hipError_t e_ = (expr);                             \
    if (e_ != hipSuccess) return fail_hip(e_, #expr);   \
  } while (0)

constexpr uint32_t kMagicW = 0x57514E53u;  // live weights handle
constexpr uint32_t kMagicA = 0x41514E53u;  // live activation handle
std::atomic<uint64_t> g_serial{1};          // weights handles, in creation order
constexpr uint32_t kDead = 0xDEADBEEFu;

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

int pow2_container(int b) { return b <= 1 ? 1 : b <= 2 ? 2 : b <= 4 ? 4 : 8; }

// Weight container: 1-bit symmetric channels are sign bits; the Eq. (1)
// 1-bit grid {-1, 0} is two's complement and needs two bits.
// 1-bit sign channels go in bits, or in nibbles when the handle asks for
// SONIQ_WPACK_SIGN_NIBBLES (cheaper to widen for the MFMA GEMM).
int w_container(int b, int wq_mode, bool sign_nibbles = false) {
  if (b == 1) return wq_mode == SONIQ_WQ_TWOS_FRACTION ? 2 : sign_nibbles ? 4 : 1;
  return pow2_container(b);
}

// Activation container: unsigned 1-bit codes {0, 1} go in a 2-bit field.
int a_container(int b, int is_signed) {
  if (b == 1) return is_signed ? 1 : 2;
  return pow2_container(b);
}

int unpack_shift(int c) { return c == 8 ? 0 : c == 4 ? 4 : 6; }

QParam w_qparam(int b, int wq_mode) {
  QParam q{};
  if (wq_mode == SONIQ_WQ_TWOS_FRACTION) {
    q.qdiv = (float)(1 << (b - 1));
    q.lo = -(1 << (b - 1));
    q.hi = (1 << (b - 1)) - 1;
  } else if (b == 1) {
    q.sign1 = 1;
    q.qdiv = 1.0f;
    q.lo = -1;
    q.hi = 1;
  } else {
    const int Q = (1 << (b - 1)) - 1;
    q.qdiv = (float)Q;
    q.lo = -Q;
    q.hi = Q;
  }
  return q;
}

QParam a_qparam(int b, int is_signed) {
  if (is_signed) return w_qparam(b, SONIQ_WQ_SYMMETRIC);
  QParam q{};
  q.qdiv = (float)((1 << b) - 1);
  q.lo = 0;
  q.hi = (1 << b) - 1;
  return q;
}

// Unsigned codes that fill their container are stored shifted by 2^(c-1).
int a_zero_point(int b, int is_signed, int c) {
  return (!is_signed && b == c) ? (1 << (c - 1)) : 0;
}

struct KPlan {
  int S = 0;
  int bits[2] = {0, 0};
  int64_t len[2] = {0, 0}, pad[2] = {0, 0};
  int64_t Kp = 0;
  std::vector<int32_t> pos;
  std::vector<uint8_t> seg;
};

// Distinct widths (ascending) of a bit vector; false if a width is outside
// 1..8 or there are more than two.
bool distinct_widths(const uint8_t* bits, int64_t n, int out[2], int* count) {
  bool seen[9] = {false};
  for (int64_t i = 0; i < n; ++i) {
    if (bits[i] < 1 || bits[i] > 8) return false;
    seen[bits[i]] = true;
  }
  int c = 0;
  out[0] = out[1] = 0;
  for (int b = 1; b <= 8; ++b)
    if (seen[b]) {
      if (c == 2) return false;
      out[c++] = b;
    }
  *count = c;
  return true;
}

bool plan_k(const uint8_t* a_bits, int64_t K, KPlan& kp) {
  if (!distinct_widths(a_bits, K, kp.bits, &kp.S)) return false;
  kp.pos.resize(K);
  kp.seg.resize(K);
  kp.len[0] = kp.len[1] = 0;
  for (int64_t k = 0; k < K; ++k) kp.len[a_bits[k] == kp.bits[0] ? 0 : 1]++;
  kp.pad[0] = round_up(kp.len[0], kGran);
  kp.pad[1] = round_up(kp.len[1], kGran);
  kp.Kp = kp.pad[0] + kp.pad[1];
  int64_t r0 = 0, r1 = 0;
  for (int64_t k = 0; k < K; ++k) {
    if (a_bits[k] == kp.bits[0]) {
      kp.seg[k] = 0;
      kp.pos[k] = (int32_t)r0++;
    } else {
      kp.seg[k] = 1;
      kp.pos[k] = (int32_t)(kp.pad[0] + r1++);
    }
  }
  return true;
}

// Input-channel plan of a 3x3 convolution computed as an implicit GEMM:
// column k = c*9 + t of the lowered matrix (t = kh*3 + kw) goes to tap-major
// order inside its precision group: position t*cpad_g + rank of c in the
// group, each tap's run padded to a multiple of 16 channels (one MFMA
// fragment unit) and the group to a multiple of 64 (a granule).  The GEMM
// then finds every 16-channel unit of a tap as one run of a pixel's codes.
bool plan_k_conv(const uint8_t* c_bits, int64_t C, KPlan& kp, int64_t cpad[2]) {
  if (!distinct_widths(c_bits, C, kp.bits, &kp.S)) return false;
  int64_t cnt[2] = {0, 0};
  std::vector<int64_t> rank(C);
  for (int64_t c = 0; c < C; ++c) {
    const int g = c_bits[c] == kp.bits[0] ? 0 : 1;
    rank[c] = cnt[g]++;
  }
  for (int g = 0; g < 2; ++g) {
    cpad[g] = round_up(cnt[g], 16);
    kp.len[g] = 9 * cnt[g];
    kp.pad[g] = round_up(9 * cpad[g], kGran);
  }
  kp.Kp = kp.pad[0] + kp.pad[1];
  kp.pos.resize(9 * C);
  kp.seg.resize(9 * C);
  for (int64_t c = 0; c < C; ++c) {
    const int g = c_bits[c] == kp.bits[0] ? 0 : 1;
    for (int t = 0; t < 9; ++t) {
      kp.seg[9 * c + t] = (uint8_t)g;
      kp.pos[9 * c + t] = (int32_t)((g ? kp.pad[0] : 0) + t * cpad[g] + rank[c]);
    }
  }
  return true;
}

template <class T>
hipError_t dev_alloc(T** p, size_t count) {
  *p = nullptr;
  if (count == 0) count = 1;
  return hipMalloc(reinterpret_cast<void**>(p), count * sizeof(T));
}

}  // namespace

struct soniq_weights_s {
  uint32_t magic = 0;
  int refs = 1;          // 1 for the owner + 1 per live activation handle
  bool released = false;  // soniq_weights_destroy was called
  int64_t N = 0, K = 0;
  int a_signed = 1, wq_mode = SONIQ_WQ_SYMMETRIC;
  KPlan kp;
  int nw = 0;
  int wb[2] = {0, 0};
  int64_t w_cnt[2] = {0, 0};
  WPlan wp{};
  std::vector<uint64_t> blk_off_h;
  std::vector<uint8_t> blk_c_h;
  std::vector<int32_t> phys_h;
  int64_t packed_bytes = 0;
  uint8_t* packed = nullptr;
  uint64_t* blk_off = nullptr;
  uint8_t* blk_c = nullptr;
  ColInfo* colinfo = nullptr;
  uint8_t* shw = nullptr;
  int32_t* tile_cols = nullptr;
  uint8_t* colrank = nullptr;
  int32_t* pos = nullptr;
  uint16_t* pos16 = nullptr;  // the same positions in 16 bits (planned K <= 65536)
  uint8_t* seg = nullptr;
  // sub-group activation scales (0 bits: one scale per precision group)
  uint64_t serial = 0;  // unique per handle (tables built for it are keyed by it)
  int act_group_bits = 0;
  int gsub[2] = {0, 0};   // granules per block
  int nsub[2] = {0, 0};   // blocks per precision group
  int32_t* grp = nullptr;  // block of each original input channel
  int32_t* posg = nullptr;  // planned position | block << 16
  std::vector<int32_t> grp_h;  // host copy of grp
  // MFMA-native copies (SONIQ_WPACK_F8F6F4): the weight side of the plan
  // (formats, fgranule counts, region offsets) and the weight copy
  bool f8f6f4 = false;
  FPlan fplan{};
  uint8_t* fw = nullptr;
  // dense copy (SONIQ_WPACK_DENSE): every code in its width, for the GEMV
  uint8_t* dense = nullptr;
  int64_t dense_bytes = 0;
  // 3x3 convolution packed for the implicit GEMM (tap-major channel plan)
  bool conv = false;
  int64_t C = 0;
  int64_t cpad[2] = {0, 0};
  int32_t* chan = nullptr;  // [2][max group size]: original channel of each rank

  int scales() const { return act_group_bits ? nsub[0] + nsub[1] : kp.S; }
  WDev dev() const { return WDev{packed, blk_off, blk_c, colinfo, shw, tile_cols, colrank}; }
};

struct soniq_act_s {
  uint32_t magic = 0;
  soniq_weights w = nullptr;
  int64_t max_M = 0, M_alloc = 0, M = 0;
  ActPlan ap{};
  int64_t packed_bytes = 0;
  uint8_t* packed = nullptr;
  float* partial = nullptr;
  unsigned int* counter = nullptr;  // kActStateWords words: the single-pass quantizer's grid state
  float* s_a = nullptr;
  // filled by soniq_mp_gemm_quantize_next from the producing layer: its
  // outputs' codes as bytes: M_alloc * Kp in 16-row blocks of 16-byte
  // columns from the GEMM tiles, then 8 * Kp row-major from the GEMV forms
  // (padding positions stay 0), and
  // the producer's per-physical-column table (position | group << 16)
  uint8_t* qn_img = nullptr;
  float* qn_brs = nullptr;  // reciprocals of static block scales (sub-group weights)
  // MFMA-native copy of the narrow activation groups (weights packed with
  // SONIQ_WPACK_F8F6F4), refreshed from the units before each MFMA GEMM;
  // fplan = the weights' plan with this buffer's offsets
  uint8_t* fa = nullptr;
  FPlan fplan{};
  // weights of an implicit 3x3 convolution: the haloed code image of its
  // input, per precision group [B][H+2][W+2][cpad_g channels], for up to
  // cg.B images of H x W
  ConvGeo cg{};
  uint8_t* img = nullptr;
  // a single row's contiguous image for the batch-1 GEMV (plans with a
  // 4-bit group 0 and an 8-bit or no group 1), and whether the last
  // quantization into this handle left it (one row, by a path that writes
  // it); the GEMV of one row reads it instead of the spread-out units
  uint8_t* ximg = nullptr;
  bool ximg_ok = false;
  // one column table per producer weights handle (keyed by its serial),
  // kept until this handle is destroyed: a captured graph may still hold a
  // table's address after another producer has fed this handle
  std::vector<std::pair<uint64_t, int32_t*>> qn_tabs;
  int32_t* qn_table(uint64_t serial) const {
    for (const auto& t : qn_tabs)
      if (t.first == serial) return t.second;
    return nullptr;
  }
};

namespace {

void free_weights(soniq_weights w) {
  (void)hipDeviceSynchronize();
  (void)hipFree(w->packed);
  (void)hipFree(w->blk_off);
  (void)hipFree(w->blk_c);
  (void)hipFree(w->colinfo);
  (void)hipFree(w->shw);
  (void)hipFree(w->tile_cols);
  (void)hipFree(w->colrank);
  (void)hipFree(w->pos);
  (void)hipFree(w->pos16);
  (void)hipFree(w->seg);
  (void)hipFree(w->grp);
  (void)hipFree(w->posg);
  (void)hipFree(w->fw);
  (void)hipFree(w->dense);
  (void)hipFree(w->chan);
  w->magic = kDead;
  delete w;
}

void release_weights(soniq_weights w) {
  if (--w->refs == 0) free_weights(w);
}

bool live_w(soniq_weights w) { return w && w->magic == kMagicW && !w->released; }
bool live_a(soniq_act a) { return a && a->magic == kMagicA; }

ActPlan make_act_plan(const soniq_weights_s& w, int64_t M_alloc) {
  ActPlan ap{};
  ap.S = w.kp.S;
  int64_t off = 0;
  for (int g = 0; g < 2; ++g) {
    if (g < ap.S) {
      const int b = w.kp.bits[g];
      ap.c[g] = a_container(b, w.a_signed);
      ap.sh[g] = unpack_shift(ap.c[g]);
      ap.zp[g] = a_zero_point(b, w.a_signed, ap.c[g]);
      ap.kpad[g] = (int)w.kp.pad[g];
      ap.ng[g] = (int)(w.kp.pad[g] / kGran);
      ap.padcnt[g] = (int)(w.kp.pad[g] - w.kp.len[g]);
      ap.mblk_bytes[g] = (int64_t)ap.ng[g] * 128 * ap.c[g];
      ap.seg_off[g] = off;
      off = round_up(off + (M_alloc / kBlk) * ap.mblk_bytes[g], 256);
      ap.q[g] = a_qparam(b, w.a_signed);
    } else {
      ap.c[g] = 8;
      ap.q[g] = a_qparam(8, 1);
    }
  }
  ap.Kp = (int)w.kp.Kp;
  for (int g = 0; g < 2; ++g) {
    ap.gsub[g] = w.gsub[g];
    ap.nsub[g] = w.nsub[g];
  }
  return ap;
}

int64_t act_bytes(const ActPlan& ap, int64_t M_alloc) {
  int64_t off = 0;
  for (int g = 0; g < ap.S; ++g) off = round_up(off + (M_alloc / kBlk) * ap.mblk_bytes[g], 256);
  return off;
}

// The activation side of an MFMA-native plan for M_alloc rows: each narrow
// group's region in the activation copy; returns the copy's bytes.
int64_t act_fplan(FPlan& fp, int64_t M_alloc) {
  int64_t off = 0;
  for (int g = 0; g < 2; ++g) {
    fp.fa_off[g] = off;
    fp.fa_mblk[g] = fp.fa[g] ? (int64_t)fp.nfg[g] * f_block_bytes(fp.fa[g]) : 0;
    off = round_up(off + (M_alloc / kBlk) * fp.fa_mblk[g], 256);
  }
  return off;
}

// Field of element e (0..15) of a unit of container c at p.
uint32_t unit_field(const uint8_t* p, int e, int c) {
  const int j = e / 4, b = e % 4;
  if (c == 8) return p[e];
  if (c == 1) {
    const uint32_t h = (uint32_t)p[0] | ((uint32_t)p[1] << 8);
    return (h >> (4 * b + j)) & 1u;
  }
  uint32_t word;
  if (c == 4) {
    memcpy(&word, p + 4 * (e / 8), 4);
    const int jj = (e % 8) / 4;
    return (word >> (8 * b + 4 * jj)) & 0xFu;
  }
  // c = 2: elements 4j+b with j = 0, 1 sit in the top two bits of nibble
  // 2b+j, those with j = 2, 3 in the bottom two bits of nibble 2b+j-2.
  memcpy(&word, p, 4);
  return (word >> (8 * b + 4 * (j & 1) + ((j >> 1) ? 0 : 2))) & 0x3u;
}

// Field of row r, channel position e (in the group-ordered padded axis of
// one group) of a fragment-major region whose block-granules are `gstride`
// = 128*c bytes apart.
uint32_t block_field(const uint8_t* blk, int r, int64_t e, int c) {
  const int64_t q = e / kGran;
  const int within = (int)(e % kGran);
  const int kg = within / 16, el = within % 16;
  return unit_field(blk + q * 128 * c + (kg * 16 + r) * 2 * c, el, c);
}

int decode_signed(uint32_t f, int c) {
  if (c == 1) return f ? -1 : 1;
  return (f >> (c - 1)) ? (int)f - (1 << c) : (int)f;
}

// The launches behind the entry points, on validated arguments: an
// activation handle's buffers (or their stand-ins in the device scratch).
soniq_status run_quantize(soniq_act_s& act, const float* A_dev, int64_t M, int64_t lda,
                          hipStream_t st) {
  const soniq_weights w = act.w;
  if (w->act_group_bits)
    HIP_TRY(launch_act_quant_grouped(A_dev, M, w->K, lda, act.ap, w->pos, w->grp, w->posg,
                                     act.partial, act.counter, act.s_a, act.packed, st));
  bool ximg = false;
  if (!w->act_group_bits)
    HIP_TRY(launch_act_quant(A_dev, M, w->K, lda, act.ap, w->pos, w->seg, act.partial, act.counter,
                             act.s_a, act.packed, st, act.ximg, &ximg));
  act.ximg_ok = ximg;
  act.M = M;
  return SONIQ_OK;
}

soniq_status run_gemm(soniq_act_s& act, uint16_t* Y_dev, int64_t ldy, int32_t* acc_dev,
                      hipStream_t st) {
  const soniq_weights w = act.w;
  const int64_t M = act.M;
  if (w->conv) {
    HIP_TRY(launch_mp_gemm_conv(act.img, act.cg, act.s_a, act.ap, w->dev(), w->wp, M, w->N, Y_dev,
                                ldy, acc_dev, st));
    return SONIQ_OK;
  }
  const bool gemv = !w->act_group_bits && gemv_fits(M, act.ap, w->wp);
  if (!gemv && ((M + 63) / 64) * (w->wp.Np / kGemmBN) > 0x7FFFFFFFLL)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_mp_gemm: problem too large for one launch");
  if (w->act_group_bits && gemv_g_fits(M, act.ap, w->wp) && !getenv("SONIQ_GROUPED_MFMA"))
    HIP_TRY(launch_mp_gemv_grouped(act.packed, act.s_a, act.ap, w->dev(), w->wp, M, w->N, Y_dev,
                                   ldy, acc_dev, st));
  else if (w->act_group_bits)
    HIP_TRY(launch_mp_gemm_grouped(act.packed, act.s_a, act.ap, w->dev(), w->wp, M, w->N, Y_dev, ldy,
                                   acc_dev, st));
  else if (w->dense && gemv_dense_fits(M, act.ap))
    HIP_TRY(launch_mp_gemv_dense(act.packed, act.s_a, act.ap, w->dev(), w->wp, w->dense, w->wb[0],
                                 w->nw == 2 ? w->wb[1] : w->wb[0], M, w->N, Y_dev, ldy, acc_dev, st));
  else if (gemv)
    HIP_TRY(launch_mp_gemv(act.packed, act.s_a, act.ap, w->dev(), w->wp, M, w->N, Y_dev, ldy,
                           acc_dev, st, act.ximg_ok ? act.ximg : nullptr));
  else if (act.fa) {
    // refresh the MFMA-native copy of the narrow groups from the units the
    // producer left, then the GEMM with both forms
    const FPlan& fp = act.fplan;
    for (int g = 0; g < act.ap.S; ++g)
      if (fp.fa[g])
        HIP_TRY(launch_to_fp(act.packed + act.ap.seg_off[g], act.ap.mblk_bytes[g], act.ap.c[g],
                             act.ap.ng[g], (M + kBlk - 1) / kBlk, act.fa + fp.fa_off[g],
                             fp.fa_mblk[g], fp.fa[g], st));
    HIP_TRY(launch_mp_gemm(act.packed, act.s_a, act.ap, w->dev(), w->wp, M, w->N, Y_dev, ldy,
                           acc_dev, st, &fp, act.fa, w->fw));
  } else
    HIP_TRY(launch_mp_gemm(act.packed, act.s_a, act.ap, w->dev(), w->wp, M, w->N, Y_dev, ldy,
                           acc_dev, st));
  return SONIQ_OK;
}

soniq_status run_quantize_gemm(soniq_act_s& act, const float* A_dev, int64_t M, int64_t lda,
                               uint16_t* Y_dev, int64_t ldy, int32_t* acc_dev, hipStream_t st) {
  const soniq_weights w = act.w;
  if (M == 1 && !w->act_group_bits && !w->dense && gemv_fused_fits(A_dev, w->K, act.ap, w->wp)) {
    HIP_TRY(launch_gemv_fused(A_dev, w->K, w->pos16, act.packed, act.s_a, act.ap, w->dev(), w->wp,
                              w->N, Y_dev, acc_dev, st, act.ximg));
    act.ximg_ok = act.ximg != nullptr;
    act.M = 1;
    return SONIQ_OK;
  }
  const soniq_status q = run_quantize(act, A_dev, M, lda, st);
  if (q != SONIQ_OK) return q;
  return run_gemm(act, Y_dev, ldy, acc_dev, st);
}

}  // namespace

extern "C" {

const char* soniq_last_error(void) { return g_err.c_str(); }

soniq_status soniq_plan_input_channels(const uint8_t* a_bits, int64_t K, int64_t* pos,
                                       int64_t seg_len[2], int64_t seg_pad[2], int32_t* S) {
  if (!a_bits || !pos || !seg_len || !seg_pad || !S)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_plan_input_channels: null pointer");
  if (K < 1) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_plan_input_channels: K < 1");
  KPlan kp;
  if (!plan_k(a_bits, K, kp))
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_plan_input_channels: widths must be 1..8 with at most two values");
  for (int64_t k = 0; k < K; ++k) pos[k] = kp.pos[k];
  for (int g = 0; g < 2; ++g) {
    seg_len[g] = kp.len[g];
    seg_pad[g] = kp.pad[g];
  }
  *S = kp.S;
  return SONIQ_OK;
}

}  // extern "C"

namespace {
// Packing behind the entry points; c_bits (host, C widths) selects the
// tap-major plan of a 3x3 convolution (K = 9*C), else a_bits gives the
// plain plan.
soniq_status pack_impl(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                       const uint8_t* w_bits, const uint8_t* a_bits, int a_signed, int wq_mode,
                       int act_group_bits, void* stream, soniq_weights* out,
                       const uint8_t* c_bits = nullptr, int64_t C = 0) {
  if (!W_dev || !w_bits || (!a_bits && !c_bits) || !out)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights: null pointer");
  if (N < 1 || K < 1) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights: N, K must be >= 1");
  if (ldw < K) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights: ldw < K");
  if (a_signed != 0 && a_signed != 1)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights: a_signed must be 0 or 1");
  const bool sign_nibbles = (wq_mode & SONIQ_WPACK_SIGN_NIBBLES) != 0;
  const bool f8f6f4 = (wq_mode & SONIQ_WPACK_F8F6F4) != 0;
  const bool dense = (wq_mode & SONIQ_WPACK_DENSE) != 0;
  wq_mode &= ~(SONIQ_WPACK_SIGN_NIBBLES | SONIQ_WPACK_F8F6F4 | SONIQ_WPACK_DENSE);
  if (f8f6f4 && act_group_bits > 0)
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_pack_weights: SONIQ_WPACK_F8F6F4 with sub-group activation scales");
  if (dense && (f8f6f4 || act_group_bits > 0 || c_bits))
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_pack_weights: SONIQ_WPACK_DENSE with f8f6f4 copies, sub-group scales or a "
                "convolution");
  if (wq_mode != SONIQ_WQ_SYMMETRIC && wq_mode != SONIQ_WQ_TWOS_FRACTION)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights: unknown wq_mode %d", wq_mode);
  int wb[2], nw = 0;
  if (!distinct_widths(w_bits, N, wb, &nw))
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_pack_weights: w_bits must be 1..8 with at most two distinct values");
  KPlan kp;
  int64_t cpad[2] = {0, 0};
  if (c_bits ? !plan_k_conv(c_bits, C, kp, cpad) : !plan_k(a_bits, K, kp))
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_pack_weights: activation widths must be 1..8 with at most two distinct values");
  if (c_bits && (f8f6f4 || act_group_bits))
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_pack_weights_conv3x3: SONIQ_WPACK_F8F6F4 and sub-group scales are not "
                "available for the implicit convolution");
  if (kp.Kp > SONIQ_MAX_K)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_pack_weights: padded K %lld exceeds %d",
                (long long)kp.Kp, SONIQ_MAX_K);
  if (N > (int64_t)1 << 24)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_pack_weights: N %lld exceeds 2^24", (long long)N);
  if (act_group_bits < 0 || act_group_bits % 512 != 0)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_pack_weights: act_group_bits %d is not 0 or a positive multiple of 512",
                act_group_bits);
  int gsub[2] = {0, 0}, nsub[2] = {0, 0};
  if (act_group_bits > 0) {
    for (int g = 0; g < kp.S; ++g) {
      const int b = kp.bits[g];
      const int c = a_container(b, a_signed);
      if (a_qparam(b, a_signed).sign1 || a_zero_point(b, a_signed, c) != 0)
        return fail(SONIQ_ERR_UNSUPPORTED,
                    "soniq_pack_weights: sub-group scales need a zero point of 0 and no 1-bit "
                    "group (activation width %d, %s)", b, a_signed ? "signed" : "unsigned");
      const int per = act_group_bits / c;  // channels per block, a multiple of 64
      gsub[g] = per / kGran;
      nsub[g] = (int)((kp.len[g] + per - 1) / per);
    }
    if (nsub[0] + nsub[1] > kGSubMax)
      return fail(SONIQ_ERR_UNSUPPORTED, "soniq_pack_weights: %d activation blocks exceed %d",
                  nsub[0] + nsub[1], kGSubMax);
    // one code row and the block scales must fit a workgroup's 64 KB
    if (kp.Kp + 8 * (int64_t)(nsub[0] + nsub[1]) > 64 * 1024)
      return fail(SONIQ_ERR_UNSUPPORTED,
                  "soniq_pack_weights: padded K %lld too large for sub-group scales",
                  (long long)kp.Kp);
  }

  soniq_weights w = new (std::nothrow) soniq_weights_s();
  if (!w) return fail(SONIQ_ERR_OUT_OF_MEMORY, "soniq_pack_weights: host allocation");
  w->N = N;
  w->K = K;
  w->a_signed = a_signed;
  w->wq_mode = wq_mode;
  w->kp = std::move(kp);
  w->nw = nw;
  w->act_group_bits = act_group_bits;
  for (int g = 0; g < 2; ++g) {
    w->gsub[g] = gsub[g];
    w->nsub[g] = nsub[g];
  }
  w->wb[0] = wb[0];
  w->wb[1] = nw == 2 ? wb[1] : 0;

  // Output-channel plan.
  const int b_lo = wb[0], b_hi = nw == 2 ? wb[1] : wb[0];
  WPlan& wp = w->wp;
  wp.c_lo = w_container(b_lo, wq_mode, sign_nibbles);
  wp.c_hi = w_container(b_hi, wq_mode, sign_nibbles);
  wp.ngt = (int)(w->kp.Kp / kGran);
  std::vector<int32_t> rows_lo, rows_hi;
  for (int64_t n = 0; n < N; ++n) (w_bits[n] == b_lo ? rows_lo : rows_hi).push_back((int32_t)n);
  w->w_cnt[0] = (int64_t)rows_lo.size();
  w->w_cnt[1] = (int64_t)rows_hi.size();
  const int64_t nb_lo = (w->w_cnt[0] + kBlk - 1) / kBlk, nb_hi = (w->w_cnt[1] + kBlk - 1) / kBlk;
  // With two containers the narrow blocks are padded to whole tiles, so that
  // a tile holds one container.  Two widths in one container (1-bit channels
  // in nibbles beside 3- or 4-bit ones, or 5..8 bits) need no such padding:
  // the columns run on, narrow first, and a block may hold both widths (a
  // block needs one container; codes and scales are per column).
  const bool one_container = nw == 2 && wp.c_lo == wp.c_hi && !f8f6f4 && !dense;
  const int64_t nb_all = (N + kBlk - 1) / kBlk;
  const int64_t nlo = one_container ? round_up(nb_all, kGemmBN / kBlk)
                      : nw == 2    ? round_up(nb_lo, kGemmBN / kBlk)
                                   : nb_lo;
  const int64_t nblk = one_container ? nlo : round_up(nlo + nb_hi, kGemmBN / kBlk);
  wp.nblk = (int)nblk;
  wp.nlo = (int)nlo;
  wp.Np = (int)(nblk * kBlk);
  w->blk_off_h.assign(nblk, 0);
  w->blk_c_h.assign(nblk, (uint8_t)wp.c_lo);
  w->phys_h.assign(N, 0);
  std::vector<ColInfo> colinfo_h(wp.Np, ColInfo{-1, 0.0f, {0, 0}});
  std::vector<uint8_t> shw_h(wp.Np, 0);
  {
    int64_t il = 0, ih = 0, b = 0;
    uint64_t off = 0;
    auto place = [&](const std::vector<int32_t>& rows, int64_t blk_in_width, int c) {
      for (int r = 0; r < kBlk; ++r) {
        const int64_t idx = blk_in_width * kBlk + r;
        if (idx >= (int64_t)rows.size()) break;
        const int32_t n = rows[idx];
        const int32_t p = (int32_t)(b * kBlk + r);
        w->phys_h[n] = p;
        colinfo_h[p].n = n;
        shw_h[p] = (uint8_t)(unpack_shift(c) | (c == 1 ? kShwSign : 0));
      }
      w->blk_c_h[b] = (uint8_t)c;
      w->blk_off_h[b] = off;
      off += (uint64_t)wp.ngt * 128 * c;  // blocks are contiguous (the GEMM relies on it)
      ++b;
    };
    static const std::vector<int32_t> none;
    if (one_container) {
      std::vector<int32_t> rows_all(rows_lo);
      rows_all.insert(rows_all.end(), rows_hi.begin(), rows_hi.end());
      while (il < nb_all) place(rows_all, il++, wp.c_lo);
      while (b < nblk) place(none, 0, wp.c_lo);
    } else {
      while (il < nb_lo) place(rows_lo, il++, wp.c_lo);
      while (b < nlo) place(none, 0, wp.c_lo);
      while (ih < nb_hi) place(rows_hi, ih++, wp.c_hi);
      while (b < nblk) place(none, 0, wp.c_hi);
    }
    w->packed_bytes = (int64_t)off;
    // Kernels derive block offsets from the plan; the table must agree.
    for (int64_t i = 0; i < nblk; ++i)
      if (w->blk_off_h[i] != wblk_off(wp, (int)i) || w->blk_c_h[i] != wblk_c(wp, (int)i)) {
        free_weights(w);
        return fail(SONIQ_ERR_UNSUPPORTED, "soniq_pack_weights: block plan mismatch");
      }
  }
  // Output order inside each 128-column tile, for coalesced stores.
  const int ntile = wp.Np / kGemmBN;
  std::vector<int32_t> tile_cols_h((size_t)wp.Np, -1);
  std::vector<uint8_t> colrank_h((size_t)wp.Np, 255);
  for (int t = 0; t < ntile; ++t) {
    std::vector<std::pair<int32_t, int32_t>> cols;  // (n, physical position)
    for (int j = 0; j < kGemmBN; ++j) {
      const int32_t p = t * kGemmBN + j;
      if (colinfo_h[p].n >= 0) cols.emplace_back(colinfo_h[p].n, p);
    }
    std::sort(cols.begin(), cols.end());
    for (size_t r = 0; r < cols.size(); ++r) {
      tile_cols_h[(size_t)t * kGemmBN + r] = cols[r].first;
      colrank_h[cols[r].second] = (uint8_t)r;
    }
  }

  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  soniq_status rc = SONIQ_OK;
  uint8_t* wbits_dev = nullptr;
  int32_t* phys_dev = nullptr;
  hipError_t e = hipSuccess;
#define STEP(expr)                              \
  if (e == hipSuccess) {                        \
    e = (expr);                                 \
    if (e != hipSuccess) rc = fail_hip(e, #expr); \
  }
  STEP(dev_alloc(&w->packed, (size_t)w->packed_bytes));
  STEP(dev_alloc(&w->blk_off, (size_t)wp.nblk));
  STEP(dev_alloc(&w->blk_c, (size_t)wp.nblk));
  STEP(dev_alloc(&w->colinfo, (size_t)wp.Np));
  STEP(dev_alloc(&w->shw, (size_t)wp.Np));
  STEP(dev_alloc(&w->tile_cols, (size_t)wp.Np));
  STEP(dev_alloc(&w->colrank, (size_t)wp.Np));
  STEP(dev_alloc(&w->pos, (size_t)K));
  STEP(dev_alloc(&w->pos16, (size_t)K));
  STEP(dev_alloc(&w->seg, (size_t)K));
  const std::vector<uint16_t> pos16_h(w->kp.pos.begin(), w->kp.pos.end());
  std::vector<int32_t> grp_h, posg_h;
  if (act_group_bits > 0) {
    // block of channel k: its rank inside its precision group over the
    // channels per block, after the blocks of group 0
    grp_h.resize(K);
    for (int64_t k = 0; k < K; ++k) {
      const int g = w->kp.seg[k];
      const int64_t rank = w->kp.pos[k] - (g ? w->kp.pad[0] : 0);
      grp_h[k] = (g ? nsub[0] : 0) + (int32_t)(rank / ((int64_t)gsub[g] * kGran));
    }
    STEP(dev_alloc(&w->grp, (size_t)K));
    STEP(hipMemcpyAsync(w->grp, grp_h.data(), K * sizeof(int32_t), hipMemcpyHostToDevice, st));
    posg_h.resize(K);
    for (int64_t k = 0; k < K; ++k) posg_h[k] = w->kp.pos[k] | (grp_h[k] << 16);
    STEP(dev_alloc(&w->posg, (size_t)K));
    STEP(hipMemcpyAsync(w->posg, posg_h.data(), K * sizeof(int32_t), hipMemcpyHostToDevice, st));
  }
  STEP(dev_alloc(&wbits_dev, (size_t)N));
  STEP(dev_alloc(&phys_dev, (size_t)N));
  STEP(hipMemsetAsync(w->packed, 0, (size_t)w->packed_bytes, st));
  STEP(hipMemcpyAsync(w->blk_off, w->blk_off_h.data(), wp.nblk * sizeof(uint64_t), hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->blk_c, w->blk_c_h.data(), wp.nblk, hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->colinfo, colinfo_h.data(), wp.Np * sizeof(ColInfo), hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->shw, shw_h.data(), wp.Np, hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->tile_cols, tile_cols_h.data(), wp.Np * sizeof(int32_t), hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->colrank, colrank_h.data(), wp.Np, hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->pos, w->kp.pos.data(), K * sizeof(int32_t), hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->pos16, pos16_h.data(), K * sizeof(uint16_t), hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(w->seg, w->kp.seg.data(), K, hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(wbits_dev, w_bits, N, hipMemcpyHostToDevice, st));
  STEP(hipMemcpyAsync(phys_dev, w->phys_h.data(), N * sizeof(int32_t), hipMemcpyHostToDevice, st));
  STEP(launch_wpack(W_dev, N, K, ldw, wbits_dev, w->pos, w->seg, phys_dev, w->blk_off, w->blk_c,
                    w_qparam(b_lo, wq_mode), w_qparam(b_hi, wq_mode), b_lo, (int)w->kp.Kp,
                    w->packed, w->colinfo, st));
  if (dense && e == hipSuccess) {
    // the dense copy, converted from the units just packed
    w->dense_bytes = (int64_t)dense_off(wp, wp.nblk, b_lo, b_hi);
    STEP(dev_alloc(&w->dense, (size_t)w->dense_bytes));
    STEP(launch_dense_pack(w->packed, wp, b_lo, b_hi, w->dense, st));
  }
  if (f8f6f4 && e == hipSuccess) {
    // The MFMA-native copy of every (narrow activation group, narrow weight
    // class) pair, converted from the units just packed.
    FPlan& fp = w->fplan;
    w->f8f6f4 = true;
    const int ngr[2] = {(int)(w->kp.pad[0] / kGran), (int)(w->kp.pad[1] / kGran)};
    for (int g = 0; g < 2; ++g) {
      fp.fa[g] = g < w->kp.S ? f_fmt(a_container(w->kp.bits[g], a_signed)) : 0;
      fp.nfg[g] = (ngr[g] + 1) / 2;
    }
    fp.fw[0] = f_fmt(wp.c_lo);
    fp.fw[1] = f_fmt(wp.c_hi);
    const int64_t cls_blocks[2] = {wp.nlo, wp.nblk - wp.nlo};
    int64_t off = 0;
    for (int g = 0; g < 2; ++g)
      for (int k = 0; k < 2; ++k) {
        fp.fw_off[g][k] = -1;
        if (!fp.fa[g] || !fp.fw[k] || !cls_blocks[k]) continue;
        fp.fw_off[g][k] = off;
        off = round_up(off + cls_blocks[k] * fp.nfg[g] * f_block_bytes(fp.fw[k]), 256);
      }
    STEP(dev_alloc(&w->fw, (size_t)off));
    for (int g = 0; g < 2; ++g)
      for (int k = 0; k < 2; ++k) {
        if (fp.fw_off[g][k] < 0 || e != hipSuccess) continue;
        const int first = k ? wp.nlo : 0;
        const int c = k ? wp.c_hi : wp.c_lo;
        const int64_t qbase = g ? ngr[0] : 0;  // the group's first granule in a block
        STEP(launch_to_fp(w->packed + wblk_off(wp, first) + qbase * 128 * c,
                          (int64_t)wp.ngt * 128 * c, c, ngr[g], cls_blocks[k],
                          w->fw + fp.fw_off[g][k], (int64_t)fp.nfg[g] * f_block_bytes(fp.fw[k]),
                          fp.fw[k], st));
      }
  }
  STEP(hipStreamSynchronize(st));
#undef STEP
  (void)hipFree(wbits_dev);
  (void)hipFree(phys_dev);
  if (rc != SONIQ_OK) {
    free_weights(w);
    return rc;
  }
  w->grp_h = std::move(grp_h);
  if (c_bits) {
    if (!conv_gemm_supported(make_act_plan(*w, kMAlign), w->wp)) {
      free_weights(w);
      return fail(SONIQ_ERR_UNSUPPORTED,
                  "soniq_pack_weights_conv3x3: the implicit convolution takes activation "
                  "widths in 4- and 8-bit containers (two widths, or one of 3 to 8 bits)");
    }
    // rank -> original channel, per group (the image quantizer's gather)
    w->conv = true;
    w->C = C;
    w->cpad[0] = cpad[0];
    w->cpad[1] = cpad[1];
    const int64_t mx = std::max(cpad[0], cpad[1]);
    std::vector<int32_t> chan(2 * (size_t)mx, -1);
    int64_t cnt[2] = {0, 0};
    for (int64_t c = 0; c < C; ++c) {
      const int g = w->kp.seg[9 * c];
      chan[g * mx + cnt[g]++] = (int32_t)c;
    }
    hipError_t e2 = dev_alloc(&w->chan, chan.size());
    if (e2 == hipSuccess)
      e2 = hipMemcpy(w->chan, chan.data(), chan.size() * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e2 != hipSuccess) {
      free_weights(w);
      return fail_hip(e2, "soniq_pack_weights_conv3x3");
    }
  }
  w->serial = g_serial.fetch_add(1);
  w->magic = kMagicW;
  *out = w;
  return SONIQ_OK;
}
}  // namespace

extern "C" {

soniq_status soniq_pack_weights_grouped(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                                        const uint8_t* w_bits, const uint8_t* a_bits,
                                        int a_signed, int wq_mode, int act_group_bits,
                                        void* stream, soniq_weights* out) {
  return pack_impl(W_dev, N, K, ldw, w_bits, a_bits, a_signed, wq_mode, act_group_bits, stream, out);
}

soniq_status soniq_pack_weights_conv3x3(const float* W_dev, int64_t N, int64_t C,
                                        const uint8_t* w_bits, const uint8_t* c_bits,
                                        int a_signed, int wq_mode, void* stream,
                                        soniq_weights* out) {
  if (!c_bits) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights_conv3x3: null pointer");
  if (C < 1 || C > SONIQ_MAX_K / 9)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_pack_weights_conv3x3: C=%lld out of range",
                (long long)C);
  return pack_impl(W_dev, N, 9 * C, 9 * C, w_bits, nullptr, a_signed, wq_mode, 0, stream, out,
                   c_bits, C);
}

soniq_status soniq_pack_weights_ex(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                                   const uint8_t* w_bits, const uint8_t* a_bits,
                                   int a_signed, int wq_mode, void* stream,
                                   soniq_weights* out) {
  return soniq_pack_weights_grouped(W_dev, N, K, ldw, w_bits, a_bits, a_signed, wq_mode, 0,
                                    stream, out);
}

soniq_status soniq_pack_weights(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                                const uint8_t* w_bits, const uint8_t* a_bits, int a_signed,
                                void* stream, soniq_weights* out) {
  return soniq_pack_weights_ex(W_dev, N, K, ldw, w_bits, a_bits, a_signed,
                               SONIQ_WQ_SYMMETRIC, stream, out);
}

soniq_status soniq_weights_info(soniq_weights w, soniq_weights_info_t* out) {
  if (!live_w(w) || !out) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_weights_info: bad handle or null");
  memset(out, 0, sizeof *out);
  out->N = w->N;
  out->K = w->K;
  out->S = w->kp.S;
  out->a_signed = w->a_signed;
  out->wq_mode = w->wq_mode;
  for (int g = 0; g < 2; ++g) {
    out->a_bits[g] = (uint8_t)w->kp.bits[g];
    out->a_count[g] = w->kp.len[g];
    out->a_count_padded[g] = w->kp.pad[g];
    out->w_bits[g] = (uint8_t)w->wb[g];
    out->w_count[g] = w->w_cnt[g];
  }
  out->packed_w_bytes = w->packed_bytes;
  out->packed_w_bytes_algorithmic =
      (w->w_cnt[0] * w->wp.c_lo + w->w_cnt[1] * w->wp.c_hi) * w->K / 8;
  out->act_group_bits = w->act_group_bits;
  out->act_scales = w->scales();
  out->f8f6f4 = w->f8f6f4 ? 1 : 0;
  out->dense_w_bytes = w->dense_bytes;
  return SONIQ_OK;
}

soniq_status soniq_act_create_conv3x3(soniq_weights w, int64_t B, int64_t H, int64_t W,
                                      soniq_act* out) {
  if (!live_w(w) || !out)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_create_conv3x3: bad handle or null");
  if (!w->conv)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_act_create_conv3x3: weights not packed with soniq_pack_weights_conv3x3");
  if (B < 1 || H < 1 || W < 1 || B * H * W > ((int64_t)1 << 31) - kMAlign ||
      B * (H + 2) * (W + 2) >= ((int64_t)1 << 31) / 256 || B * w->C * H * W >= ((int64_t)1 << 31))
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_create_conv3x3: B, H, W out of range");
  soniq_act a = new (std::nothrow) soniq_act_s();
  if (!a) return fail(SONIQ_ERR_OUT_OF_MEMORY, "soniq_act_create_conv3x3: host allocation");
  a->w = w;
  a->max_M = B * H * W;
  a->M_alloc = round_up(a->max_M, kMAlign);
  a->ap = make_act_plan(*w, a->M_alloc);
  ConvGeo& cg = a->cg;
  cg.B = (int)B;
  cg.H = (int)H;
  cg.W = (int)W;
  int64_t off = 0;
  for (int g = 0; g < 2; ++g) {
    cg.cpad[g] = (int)w->cpad[g];
    cg.rowbytes[g] = g < w->kp.S ? (int)(w->cpad[g] * a->ap.c[g] / 8) : 0;
    cg.img_off[g] = off;
    off = round_up(off + B * (H + 2) * (W + 2) * (int64_t)cg.rowbytes[g], 256);
  }
  cg.chan_ld = (int)std::max(w->cpad[0], w->cpad[1]);
  hipError_t e = dev_alloc(&a->img, (size_t)off);
  if (e == hipSuccess) e = dev_alloc(&a->partial, (size_t)2 * kAbsmaxBlocks);
  if (e == hipSuccess) e = dev_alloc(&a->s_a, 2);
  if (e == hipSuccess) e = hipMemset(a->s_a, 0, 2 * sizeof(float));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    soniq_status rc = fail_hip(e, "soniq_act_create_conv3x3");
    (void)hipFree(a->img);
    (void)hipFree(a->partial);
    (void)hipFree(a->s_a);
    delete a;
    return rc;
  }
  w->refs++;
  a->magic = kMagicA;
  *out = a;
  return SONIQ_OK;
}

soniq_status soniq_act_create(soniq_weights w, int64_t max_M, soniq_act* out) {
  if (!live_w(w) || !out) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_create: bad handle or null");
  if (w->conv)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_act_create: convolution weights take soniq_act_create_conv3x3");
  if (max_M < 1 || max_M > ((int64_t)1 << 31) - kMAlign)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_create: max_M out of range");
  soniq_act a = new (std::nothrow) soniq_act_s();
  if (!a) return fail(SONIQ_ERR_OUT_OF_MEMORY, "soniq_act_create: host allocation");
  a->w = w;
  a->max_M = max_M;
  a->M_alloc = round_up(max_M, kMAlign);
  a->ap = make_act_plan(*w, a->M_alloc);
  a->packed_bytes = act_bytes(a->ap, a->M_alloc);
  hipError_t e = dev_alloc(&a->packed, (size_t)a->packed_bytes);
  const size_t nscale = (size_t)std::max(2, w->scales());
  const size_t npart = std::max((size_t)2 * kAbsmaxBlocks,
                                w->act_group_bits ? (size_t)kGAbsParts * nscale : 0);
  if (e == hipSuccess) e = dev_alloc(&a->partial, npart);
  if (e == hipSuccess) e = dev_alloc(&a->counter, kActStateWords);
  if (e == hipSuccess) e = dev_alloc(&a->s_a, nscale);
  if (e == hipSuccess) e = hipMemset(a->counter, 0, kActStateWords * sizeof(unsigned int));
  if (e == hipSuccess) e = hipMemset(a->s_a, 0, nscale * sizeof(float));
  if (e == hipSuccess) e = hipMemset(a->packed, 0, (size_t)a->packed_bytes);
  if (e == hipSuccess && w->f8f6f4) {
    a->fplan = w->fplan;
    e = dev_alloc(&a->fa, (size_t)act_fplan(a->fplan, a->M_alloc));
  }
  const ActPlan& ap = a->ap;
  if (e == hipSuccess && !w->act_group_bits && ap.c[0] == 4 && (ap.S == 1 || ap.c[1] == 8))
    e = dev_alloc(&a->ximg, (size_t)round_up(32 * (int64_t)ap.ng[0] + 64 * (int64_t)ap.ng[1], 256));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    soniq_status rc = fail_hip(e, "soniq_act_create");
    (void)hipFree(a->ximg);
    (void)hipFree(a->fa);
    (void)hipFree(a->packed);
    (void)hipFree(a->partial);
    (void)hipFree(a->counter);
    (void)hipFree(a->s_a);
    delete a;
    return rc;
  }
  w->refs++;
  a->magic = kMagicA;
  *out = a;
  return SONIQ_OK;
}

soniq_status soniq_quantize_act(soniq_act act, const float* A_dev, int64_t M, int64_t lda,
                                void* stream) {
  if (!live_a(act) || !A_dev) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act: bad handle or null");
  const soniq_weights w = act->w;
  if (M < 1 || M > act->max_M)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act: M=%lld outside [1, %lld]",
                (long long)M, (long long)act->max_M);
  if (lda < w->K) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act: lda < K");
  if (w->conv)
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_quantize_act: implicit-convolution weights quantize with soniq_quantize_act_conv3x3");
  return run_quantize(*act, A_dev, M, lda, reinterpret_cast<hipStream_t>(stream));
}

soniq_status soniq_quantize_act_conv3x3(soniq_act act, const float* X_dev, int64_t B, int64_t C,
                                        int64_t H, int64_t W, void* stream) {
  if (!live_a(act) || !X_dev)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act_conv3x3: bad handle or null");
  const soniq_weights w = act->w;
  if (B < 1 || C < 1 || H < 1 || W < 1)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act_conv3x3: B, C, H, W must be >= 1");
  if (9 * C != w->K)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act_conv3x3: 9*C=%lld != K=%lld",
                (long long)(9 * C), (long long)w->K);
  if (B * C * H * W >= ((int64_t)1 << 31))
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act_conv3x3: input has 2^31 elements or more");
  if (w->act_group_bits)
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_quantize_act_conv3x3: weights packed with sub-group activation scales");
  const int64_t M = B * H * W;
  if (w->conv) {
    const ConvGeo& cg = act->cg;
    if (H != cg.H || W != cg.W || B > cg.B)
      return fail(SONIQ_ERR_INVALID_ARGUMENT,
                  "soniq_quantize_act_conv3x3: B=%lld H=%lld W=%lld do not fit the handle (B<=%d, "
                  "H=%d, W=%d)", (long long)B, (long long)H, (long long)W, cg.B, cg.H, cg.W);
    HIP_TRY(launch_conv_img(X_dev, B, C, H, W, act->ap, cg, w->seg, w->chan, act->partial, act->s_a,
                            act->img, reinterpret_cast<hipStream_t>(stream)));
    act->ximg_ok = false;
    act->M = M;
    return SONIQ_OK;
  }
  if (M > act->max_M)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_act_conv3x3: B*H*W=%lld > max_M=%lld",
                (long long)M, (long long)act->max_M);
  for (int64_t c = 0; c < C; ++c)
    for (int t = 1; t < 9; ++t)
      if (w->kp.seg[9 * c + t] != w->kp.seg[9 * c])
        return fail(SONIQ_ERR_UNSUPPORTED,
                    "soniq_quantize_act_conv3x3: the taps of channel %lld have different widths",
                    (long long)c);
  if (!conv_quant_fits(act->ap))
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_quantize_act_conv3x3: K=%lld too large for one block",
                (long long)w->K);
  HIP_TRY(launch_conv_quant(X_dev, B, C, H, W, act->ap, w->pos, w->seg, act->partial, act->s_a,
                            act->packed, reinterpret_cast<hipStream_t>(stream)));
  act->ximg_ok = false;
  act->M = M;
  return SONIQ_OK;
}

soniq_status soniq_mp_gemm(soniq_act act, soniq_weights w, uint16_t* Y_dev, int64_t ldy,
                           int32_t* acc_dev, void* stream) {
  if (!live_a(act) || !live_w(w) || !Y_dev)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm: bad handle or null");
  if (act->w != w)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm: activation handle belongs to other weights");
  if (act->M < 1)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm: no activations quantized yet");
  if (ldy < w->N) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm: ldy < N");
  return run_gemm(*act, Y_dev, ldy, acc_dev, reinterpret_cast<hipStream_t>(stream));
}

soniq_status soniq_quantize_mp_gemm(soniq_act act, soniq_weights w, const float* A_dev, int64_t M,
                                    int64_t lda, uint16_t* Y_dev, int64_t ldy, int32_t* acc_dev,
                                    void* stream) {
  if (!live_a(act) || !live_w(w) || !A_dev || !Y_dev)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm: bad handle or null");
  if (act->w != w)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_quantize_mp_gemm: activation handle belongs to other weights");
  if (M < 1 || M > act->max_M)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm: M=%lld outside [1, %lld]",
                (long long)M, (long long)act->max_M);
  if (lda < w->K) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm: lda < K");
  if (ldy < w->N) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm: ldy < N");
  if (w->conv)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_quantize_mp_gemm: implicit-convolution weights");
  return run_quantize_gemm(*act, A_dev, M, lda, Y_dev, ldy, acc_dev,
                           reinterpret_cast<hipStream_t>(stream));
}

soniq_status soniq_quantize_mp_gemm_scratch(soniq_weights w, const float* A_dev, int64_t M,
                                            int64_t lda, uint16_t* Y_dev, int64_t ldy,
                                            int32_t* acc_dev, void* stream) {
  if (!live_w(w) || !A_dev || !Y_dev)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm_scratch: bad handle or null");
  if (M < 1) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm_scratch: M < 1");
  if (lda < w->K) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm_scratch: lda < K");
  if (ldy < w->N) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_quantize_mp_gemm_scratch: ldy < N");
  if (w->conv)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_quantize_mp_gemm_scratch: implicit-convolution weights");
  // The activation buffers an activation handle for M rows would own, laid
  // out in the device's scratch: grid state, scales, partial maxima, packed
  // rows.
  if (M > ((int64_t)1 << 31) - kMAlign)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_quantize_mp_gemm_scratch: M=%lld too large",
                (long long)M);
  const int64_t M_alloc = round_up(M, kMAlign);
  const ActPlan ap = make_act_plan(*w, M_alloc);
  const size_t nscale = (size_t)std::max(2, w->scales());
  const size_t npart = std::max((size_t)2 * kAbsmaxBlocks,
                                w->act_group_bits ? (size_t)kGAbsParts * nscale : 0);
  const size_t packed_off = (size_t)round_up((int64_t)(kScratchPartialOff + 4 * npart), 256);
  FPlan fplan = w->fplan;
  const size_t fa_off = packed_off + (size_t)round_up(act_bytes(ap, M_alloc), 256);
  const size_t need = w->f8f6f4 ? fa_off + (size_t)act_fplan(fplan, M_alloc)
                                : packed_off + (size_t)act_bytes(ap, M_alloc);
  if (4 * nscale > kScratchPartialOff - kScratchScalesOff || need > kScratchBytes)
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_quantize_mp_gemm_scratch: M=%lld needs %zu bytes of scratch, more than its "
                "%zu (use an activation handle)",
                (long long)M, need, kScratchBytes);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  uint8_t* base = nullptr;
  HIP_TRY(scratch_device_ptr(st, &base));
  soniq_act_s a;
  a.w = w;
  a.max_M = M;
  a.M_alloc = M_alloc;
  a.ap = ap;
  a.packed_bytes = act_bytes(ap, M_alloc);
  a.counter = reinterpret_cast<unsigned int*>(base);
  a.s_a = reinterpret_cast<float*>(base + kScratchScalesOff);
  a.partial = reinterpret_cast<float*>(base + kScratchPartialOff);
  a.packed = base + packed_off;
  if (w->f8f6f4) {
    a.fplan = fplan;
    a.fa = base + fa_off;
  }
  return run_quantize_gemm(a, A_dev, M, lda, Y_dev, ldy, acc_dev, st);
}

// Positions of one row of a handle's next-layer byte image: its plan's
// padded K, or for an implicit convolution the channel ranks of its groups.
static int64_t qn_cols(const soniq_act_s& a) {
  return a.w->conv ? a.cg.cpad[0] + (a.ap.S == 2 ? a.cg.cpad[1] : 0) : a.ap.Kp;
}

// Words of a pair's table taken by the tiles' maxima of a full batch.
static size_t qn_ymax_words(const soniq_act_s& next, const soniq_weights_s& w) {
  return 2 * (size_t)((next.M_alloc + 63) / 64) * (size_t)(w.wp.Np / kGemmBN);
}

// The next-convolution description of a producer's M output pixels.
static QnConv qn_conv(const soniq_act_s& next, const soniq_weights_s& w, int64_t M) {
  QnConv qc{};
  const soniq_weights w2 = next.w;
  qc.cg = next.cg;
  qc.img = next.img;
  qc.B = (int)(M / ((int64_t)next.cg.H * next.cg.W));
  for (int64_t n = 0; n < w.N; ++n) qc.cnt[w2->kp.seg[9 * n]]++;
  for (int g = 0; g < 2; ++g) {
    // the stored code of 0.0: +1 in a sign group, else 0, less the zero point
    const int code0 = next.ap.q[g].sign1 ? 1 : 0;
    qc.halo[g] = code0 - next.ap.zp[g];
  }
  return qc;
}

// First use of a (producer weights, next) pair: next's code image and the
// producer's column table, built synchronously (later calls find both).
static soniq_status qn_prepare(soniq_act next, soniq_weights w, const char* who, int32_t** out) {
  int32_t* qn_tab = next->qn_table(w->serial);
  if (!next->qn_img || !qn_tab) {
    const soniq_weights w2 = next->w;
    const bool conv_next = w2->conv;
    // first use of this (producer, next) pair: the code image and the
    // producer's column table, built synchronously
    if (!next->qn_img) {
      uint8_t* img = nullptr;
      const size_t bytes = (size_t)((next->M_alloc + 8) * qn_cols(*next));
      HIP_TRY(dev_alloc(&img, bytes));
      const hipError_t e = hipMemset(img, 0, bytes);
      if (e != hipSuccess) {
        (void)hipFree(img);
        return fail_hip(e, (std::string(who) + ": hipMemset").c_str());
      }
      next->qn_img = img;
    }
    if (w2->act_group_bits && !next->qn_brs)
      HIP_TRY(dev_alloc(&next->qn_brs, (size_t)w2->scales()));
    // [0, Np): next-layer group of each physical column's channel;
    // [Np, 2 Np): next-layer position of each tile's r-th column in
    // ascending original order (the order the GEMM stages its outputs in);
    // [2 Np, 3 Np): next-layer position of each physical column (the GEMV)
    const int Np = w->wp.Np;
    std::vector<int32_t> tab(3 * (size_t)Np, -1);
    std::vector<std::vector<int64_t>> cols(Np / kGemmBN);
    // next-layer position of input channel n: its planned position, or for a
    // next convolution its rank within its group (group 1 after cpad[0])
    std::vector<int32_t> npos(w->N), ngrp(w->N);
    if (conv_next) {
      int64_t cnt[2] = {0, 0};
      for (int64_t n = 0; n < w->N; ++n) {
        const int g = w2->kp.seg[9 * n];
        ngrp[n] = g;
        npos[n] = (int32_t)((g ? w2->cpad[0] : 0) + cnt[g]++);
      }
    } else {
      for (int64_t n = 0; n < w->N; ++n) {
        ngrp[n] = w2->act_group_bits ? w2->grp_h[n] : w2->kp.seg[n];  // block, or group
        npos[n] = w2->kp.pos[n];
      }
    }
    for (int64_t n = 0; n < w->N; ++n) {
      const int32_t p = w->phys_h[n];
      tab[p] = ngrp[n];
      tab[2 * (size_t)Np + p] = npos[n];  // [2 Np, 3 Np): position by physical column
      cols[p / kGemmBN].push_back(n);
    }
    for (size_t t = 0; t < cols.size(); ++t) {
      std::sort(cols[t].begin(), cols[t].end());
      for (size_t r = 0; r < cols[t].size(); ++r) tab[Np + t * kGemmBN + r] = npos[cols[t][r]];
    }
    // followed by one pair of floats per GEMM tile of a full batch: the
    // tiles' maxima of the two-pass form (soniq_mp_gemm_quantize_next_max),
    // then the next-layer position of each input channel n (npos)
    const size_t ymax_words = qn_ymax_words(*next, *w);
    int32_t* t = nullptr;
    HIP_TRY(dev_alloc(&t, tab.size() + ymax_words + (size_t)w->N));
    hipError_t e = hipMemcpy(t, tab.data(), tab.size() * sizeof(int32_t), hipMemcpyHostToDevice);
    if (e == hipSuccess)
      e = hipMemcpy(t + tab.size() + ymax_words, npos.data(), npos.size() * sizeof(int32_t),
                    hipMemcpyHostToDevice);
    if (e != hipSuccess) {
      (void)hipFree(t);
      return fail_hip(e, (std::string(who) + ": hipMemcpy").c_str());
    }
    next->qn_tabs.emplace_back(w->serial, t);
    qn_tab = t;
  }
  *out = qn_tab;
  return SONIQ_OK;
}

soniq_status soniq_mp_gemm_quantize_next(soniq_act act, soniq_weights w, soniq_act next,
                                         const float* s_next, uint16_t* Y_dev, int64_t ldy,
                                         int32_t* acc_dev, void* stream) {
  if (!live_a(act) || !live_w(w) || !live_a(next) || !s_next)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm_quantize_next: bad handle or null");
  if (act->w != w)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_mp_gemm_quantize_next: activation handle belongs to other weights");
  if (act->M < 1)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm_quantize_next: no activations quantized yet");
  if (next == act)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_mp_gemm_quantize_next: next is the producer's own activation handle");
  const soniq_weights w2 = next->w;
  // an implicit convolution as the next layer: its input channels are this
  // layer's outputs, and this layer's rows its output pixels
  const bool conv_next = w2->conv;
  if (w->conv && !conv_gemm_qn_supported(act->ap, w->wp))
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_mp_gemm_quantize_next: no implicit-convolution kernel for these widths");
  if (w->conv && w2->act_group_bits)
    return fail(SONIQ_ERR_UNSUPPORTED,
                "soniq_mp_gemm_quantize_next: an implicit convolution into sub-group scales");
  const int64_t K2 = conv_next ? w2->C : w2->K;
  if (K2 != w->N)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_mp_gemm_quantize_next: next layer has %lld input channels, this layer N=%lld",
                (long long)K2, (long long)w->N);
  const int64_t M = act->M;
  if (conv_next) {
    const ConvGeo& cg2 = next->cg;
    const int64_t hw = (int64_t)cg2.H * cg2.W;
    if (M % hw != 0 || M / hw > cg2.B)
      return fail(SONIQ_ERR_INVALID_ARGUMENT,
                  "soniq_mp_gemm_quantize_next: M=%lld is not a batch of at most %d images of %dx%d",
                  (long long)M, cg2.B, cg2.H, cg2.W);
  } else if (M > next->max_M) {
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm_quantize_next: M=%lld > next max_M=%lld",
                (long long)M, (long long)next->max_M);
  }
  if (Y_dev && ldy < w->N)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_mp_gemm_quantize_next: ldy < N");
  for (int g = 0; g < w2->scales(); ++g)
    if (!(s_next[g] >= 0.0f) || !std::isfinite(s_next[g]))
      return fail(SONIQ_ERR_INVALID_ARGUMENT,
                  "soniq_mp_gemm_quantize_next: static scale %d is negative or not finite", g);
  const int64_t tiles = ((M + 63) / 64) * (w->wp.Np / kGemmBN);
  if (tiles > 0x7FFFFFFFLL)
    return fail(SONIQ_ERR_UNSUPPORTED, "soniq_mp_gemm_quantize_next: problem too large for one launch");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  int32_t* qn_tab = nullptr;
  {
    const soniq_status rc = qn_prepare(next, w, "soniq_mp_gemm_quantize_next", &qn_tab);
    if (rc != SONIQ_OK) return rc;
  }
  float s2[2] = {s_next[0], w2->kp.S == 2 ? s_next[1] : 0.0f};
  QnConv qc{};
  if (conv_next) qc = qn_conv(*next, *w, M);
  HIP_TRY(launch_mp_gemm_qnext(w->conv ? nullptr : act->packed, act->s_a, act->ap, w->dev(), w->wp,
                               M, w->N, Y_dev, ldy, acc_dev, next->qn_img, next->M_alloc, qn_tab,
                               next->ap, w2->act_group_bits ? s_next : s2, next->s_a, next->qn_brs,
                               next->packed, st, next->ximg, act->ximg_ok ? act->ximg : nullptr,
                               w->conv ? act->img : nullptr, w->conv ? &act->cg : nullptr,
                               conv_next ? &qc : nullptr));
  next->ximg_ok = !conv_next && M == 1 && next->ximg != nullptr;
  next->M = M;
  return SONIQ_OK;
}

soniq_status soniq_mp_gemm_quantize_next_max(soniq_act act, soniq_weights w, soniq_act next,
                                             uint16_t* Y_dev, int64_t ldy, int32_t* acc_dev,
                                             void* stream) {
  const char* who = "soniq_mp_gemm_quantize_next_max";
  if (!live_a(act) || !live_w(w) || !live_a(next) || !Y_dev)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: bad handle or null", who);
  if (act->w != w)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: activation handle belongs to other weights", who);
  if (act->M < 1) return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: no activations quantized yet", who);
  if (next == act)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: next is the producer's own activation handle", who);
  const soniq_weights w2 = next->w;
  const bool conv_next = w2->conv;
  if (w->conv && !conv_gemm_qn_supported(act->ap, w->wp))
    return fail(SONIQ_ERR_UNSUPPORTED, "%s: no implicit-convolution kernel for these widths", who);
  if (w->act_group_bits || w2->act_group_bits)
    return fail(SONIQ_ERR_UNSUPPORTED, "%s: weights packed with sub-group activation scales", who);
  const int64_t K2 = conv_next ? w2->C : w2->K;
  if (K2 != w->N)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: next layer has %lld input channels, this layer N=%lld",
                who, (long long)K2, (long long)w->N);
  const int64_t M = act->M;
  if (conv_next) {
    const int64_t hw = (int64_t)next->cg.H * next->cg.W;
    if (M % hw != 0 || M / hw > next->cg.B)
      return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: M=%lld is not a batch of at most %d images of %dx%d",
                  who, (long long)M, next->cg.B, next->cg.H, next->cg.W);
  } else if (M > next->max_M) {
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: M=%lld > next max_M=%lld", who, (long long)M,
                (long long)next->max_M);
  }
  if (ldy < w->N) return fail(SONIQ_ERR_INVALID_ARGUMENT, "%s: ldy < N", who);
  if (((M + 63) / 64) * (w->wp.Np / kGemmBN) > 0x7FFFFFFFLL)
    return fail(SONIQ_ERR_UNSUPPORTED, "%s: problem too large for one launch", who);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  int32_t* qn_tab = nullptr;
  {
    const soniq_status rc = qn_prepare(next, w, who, &qn_tab);
    if (rc != SONIQ_OK) return rc;
  }
  // the tiles' maxima, after the pair's column table
  float* ymax = reinterpret_cast<float*>(qn_tab + 3 * (size_t)w->wp.Np);
  const int32_t* posn = qn_tab + 3 * (size_t)w->wp.Np + qn_ymax_words(*next, *w);
  int nslot = 0;
  if (M <= 8 && !w->conv) {
    // the GEMV forms store Y; the quantizer reduces the small batch's maxima
    const soniq_status rc = run_gemm(*act, Y_dev, ldy, acc_dev, st);
    if (rc != SONIQ_OK) return rc;
  } else {
    HIP_TRY(launch_mp_gemm_ymax(w->conv ? nullptr : act->packed, act->s_a, act->ap, w->dev(), w->wp,
                                M, w->N, Y_dev, ldy, acc_dev, qn_tab, ymax, st,
                                w->conv ? act->img : nullptr, w->conv ? &act->cg : nullptr));
    nslot = (int)(((M + 63) / 64) * (w->wp.Np / kGemmBN));
  }
  if (conv_next) {
    // the blocked byte image the tiles' epilogue would write, then the
    // convolution's haloed code image
    HIP_TRY(launch_img_bf16(Y_dev, M, (int)w->N, ldy, posn, next->ap, qn_conv(*next, *w, M), ymax,
                            nslot, next->s_a, next->qn_img, st));
    next->ximg_ok = false;
  } else {
    HIP_TRY(launch_act_bf16(Y_dev, M, w2->K, ldy, next->ap, w2->pos, w2->seg, ymax, nslot,
                            next->s_a, next->packed, next->ximg, st));
    next->ximg_ok = M == 1 && next->ximg != nullptr;
  }
  next->M = M;
  return SONIQ_OK;
}

soniq_status soniq_weights_unpack_debug(soniq_weights w, int32_t* codes, float* s_w) {
  if (!live_w(w)) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_weights_unpack_debug: bad handle");
  HIP_TRY(hipDeviceSynchronize());
  std::vector<uint8_t> packed(w->packed_bytes);
  std::vector<ColInfo> ci(w->wp.Np);
  HIP_TRY(hipMemcpy(packed.data(), w->packed, w->packed_bytes, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(ci.data(), w->colinfo, ci.size() * sizeof(ColInfo), hipMemcpyDeviceToHost));
  for (int64_t n = 0; n < w->N; ++n) {
    const int32_t p = w->phys_h[n];
    const int b = p / kBlk, r = p % kBlk;
    const int c = w->blk_c_h[b];
    const uint8_t* blk = packed.data() + w->blk_off_h[b];
    if (codes)
      for (int64_t k = 0; k < w->K; ++k)
        codes[n * w->K + k] = decode_signed(block_field(blk, r, w->kp.pos[k], c), c);
    if (s_w) s_w[n] = ci[p].s_w;
  }
  return SONIQ_OK;
}

soniq_status soniq_act_unpack_debug(soniq_act act, int32_t* codes, float* s_a) {
  if (!live_a(act)) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_unpack_debug: bad handle");
  if (act->M < 1) return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_unpack_debug: nothing quantized");
  HIP_TRY(hipDeviceSynchronize());
  const ActPlan& ap = act->ap;
  const soniq_weights w = act->w;
  if (w->conv) {
    // codes of the lowered matrix, read back from the haloed image: column
    // k = c*9 + t of row m = (b*H + y)*W + x is channel c of pixel
    // (y + t/3 - 1, x + t%3 - 1), the halo holding the code of 0
    const ConvGeo& cg = act->cg;
    const int64_t Wp = cg.W + 2, Hp = cg.H + 2;
    size_t bytes = 0;
    for (int g = 0; g < ap.S; ++g)
      bytes = std::max(bytes, (size_t)(cg.img_off[g] + cg.B * Hp * Wp * (int64_t)cg.rowbytes[g]));
    std::vector<uint8_t> img(bytes);
    float sa[2] = {0.0f, 0.0f};
    HIP_TRY(hipMemcpy(img.data(), act->img, bytes, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(sa, act->s_a, sizeof sa, hipMemcpyDeviceToHost));
    if (codes) {
      std::vector<int64_t> rank(w->C);
      int64_t cnt[2] = {0, 0};
      for (int64_t c = 0; c < w->C; ++c) rank[c] = cnt[w->kp.seg[9 * c]]++;
      for (int64_t m = 0; m < act->M; ++m) {
        const int64_t b = m / (cg.H * cg.W), y = (m / cg.W) % cg.H, x = m % cg.W;
        for (int64_t c = 0; c < w->C; ++c) {
          const int g = w->kp.seg[9 * c];
          const int cc = ap.c[g];
          for (int t = 0; t < 9; ++t) {
            const int64_t hp = (b * Hp + y + 1 + t / 3 - 1) * Wp + x + 1 + t % 3 - 1;
            const uint8_t* unit =
                img.data() + cg.img_off[g] + hp * cg.rowbytes[g] + (rank[c] / 16) * 2 * cc;
            codes[m * w->K + 9 * c + t] =
                decode_signed(unit_field(unit, (int)(rank[c] % 16), cc), cc) + ap.zp[g];
          }
        }
      }
    }
    if (s_a)
      for (int g = 0; g < w->kp.S; ++g) s_a[g] = sa[g];
    return SONIQ_OK;
  }
  std::vector<uint8_t> packed(act->packed_bytes);
  std::vector<float> sa((size_t)std::max(2, w->scales()), 0.0f);
  HIP_TRY(hipMemcpy(packed.data(), act->packed, act->packed_bytes, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(sa.data(), act->s_a, sa.size() * sizeof(float), hipMemcpyDeviceToHost));
  if (codes)
    for (int64_t m = 0; m < act->M; ++m)
      for (int64_t k = 0; k < w->K; ++k) {
        const int g = w->kp.seg[k];
        const int64_t e = w->kp.pos[k] - (g ? ap.kpad[0] : 0);
        const uint8_t* blk = packed.data() + ap.seg_off[g] + (m / kBlk) * ap.mblk_bytes[g];
        codes[m * w->K + k] = decode_signed(block_field(blk, (int)(m % kBlk), e, ap.c[g]), ap.c[g]) + ap.zp[g];
      }
  if (s_a)
    for (int g = 0; g < w->scales(); ++g) s_a[g] = sa[g];
  return SONIQ_OK;
}

soniq_status soniq_act_wait_timeouts(soniq_act act, uint64_t* count) {
  if (!live_a(act) || !count)
    return fail(SONIQ_ERR_INVALID_ARGUMENT, "soniq_act_wait_timeouts: bad handle or null");
  HIP_TRY(hipDeviceSynchronize());
  unsigned int v = 0;
  HIP_TRY(hipMemcpy(&v, act->counter + kActStallWord, sizeof v, hipMemcpyDeviceToHost));
  *count = v;
  return SONIQ_OK;
}

soniq_status soniq_debug_stream_read(const void* src_dev, int64_t bytes, uint32_t* sink_dev,
                                     void* stream) {
  if (!src_dev || !sink_dev || bytes < 16 || bytes % 16 != 0 || bytes >= ((int64_t)1 << 31) ||
      reinterpret_cast<uintptr_t>(src_dev) % 16 != 0)
    return fail(SONIQ_ERR_INVALID_ARGUMENT,
                "soniq_debug_stream_read: null pointer, unaligned source or bad byte count");
  HIP_TRY(launch_stream_read(src_dev, bytes, sink_dev, reinterpret_cast<hipStream_t>(stream)));
  return SONIQ_OK;
}

void soniq_weights_destroy(soniq_weights w) {
  if (!live_w(w)) return;
  w->released = true;
  release_weights(w);
}

void soniq_act_destroy(soniq_act act) {
  if (!live_a(act)) return;
  (void)hipDeviceSynchronize();
  (void)hipFree(act->packed);
  (void)hipFree(act->partial);
  (void)hipFree(act->counter);
  (void)hipFree(act->s_a);
  (void)hipFree(act->qn_img);
  for (const auto& t : act->qn_tabs) (void)hipFree(t.second);
  (void)hipFree(act->qn_brs);
  (void)hipFree(act->fa);
  (void)hipFree(act->img);
  (void)hipFree(act->ximg);
  act->magic = kDead;
  soniq_weights w = act->w;
  delete act;
  release_weights(w);
}

}  // extern "C"
