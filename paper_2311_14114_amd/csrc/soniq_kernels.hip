// gfx950 (CDNA4) kernels of the SONIQ inference hot path.
//
//   k_wpack         quantize one output channel, place its codes on the
//                   group-ordered padded channel axis and write its units
//                   into its 16-row block; record scale and code sums
//   k_act_coop      activation quantize in one pass over HBM: a resident
//                   grid holds its rows in registers, folds the group
//                   maxima at a grid barrier, quantizes and packs
//   k_absmax_*      two-pass form, pass 1: per-workgroup partial maxima
//   k_act_blk16,    two-pass form, pass 2: reduce the partials, quantize,
//   k_act_rows      pack 16- or 8-row slices (or rows)
//   k_act_small     small batches in one launch (max, quantize, pack)
//   k_act_row1      batches of up to 8 rows, from registers after one load
//   k_gemm          int8 MFMA GEMM on packed operands: an LDS ring filled by
//                   direct global->LDS buffer loads, units widened to int8
//                   in registers right before v_mfma_i32_16x16x64_i8, one
//                   int32 accumulator set per activation group, fixed-order
//                   fp32 epilogue to bf16
//   k_gemv          batch <= 8 without matrix cores: one workgroup streams
//                   one 16-row weight block, v_dot8_i32_i4 on nibbles or
//                   v_dot4_i32_i8 on bytes against activations in LDS
//   k_gemv_mfma     batch 2..8: one workgroup per weight block, the batch
//                   rows as the MFMA A operand, straight from global memory
//
// Paper passages: Sec. 2.4 C1/C2/C5; Sec. 3 codec (group max-abs scale,
// unsigned codes, Eq. 1 weight codes); Alg. 1 channel permutation and Phase
// II integer MAC; Fig. "normalization" (group by width, pad to the vector
// width).
#include "soniq_internal.h"

#include <hip/hip_bf16.h>

#include <type_traits>
#include <utility>

#include <algorithm>
#include <cstdlib>
#include <mutex>

namespace soniq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- codec --
// Code of x under step s.  The quotient is taken as one IEEE fp32 division
// rounded to nearest even.  When `fast` (s normal and not tiny) the
// quotient is first estimated with a reciprocal; the estimate is within
// 2^-14 of the true quotient (|x/s| <= 256), so rint of the estimate equals
// rint of the correctly rounded quotient unless the estimate lies within
// 2^-9 of a half-integer, where the exact division decides.
__device__ __forceinline__ int quant_code(float x, float s, float rs, bool fast,
                                          const QParam& q) {
  if (q.sign1) return x < 0.0f ? -1 : 1;
  if (s == 0.0f) return 0;
  float t;
  if (fast) {
    const float e = x * rs;
    t = __builtin_rintf(e);
    if (fabsf(fabsf(e - t) - 0.5f) <= 0x1p-9f) t = __builtin_rintf(__fdiv_rn(x, s));
  } else {
    t = __builtin_rintf(__fdiv_rn(x, s));
  }
  t = fminf(fmaxf(t, (float)q.lo), (float)q.hi);
  return (int)t;
}

__device__ __forceinline__ bool fast_ok(float s) { return s >= 0x1p-100f && s <= 0x1p100f; }

__device__ __forceinline__ float group_scale(float maxabs, const QParam& q) {
  return q.sign1 ? maxabs : __fdiv_rn(maxabs, q.qdiv);
}

__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Fixed-order epilogue: t = f(ACC0)*s_a0; t = t + f(ACC1)*s_a1; t = t*s_w.
__device__ __forceinline__ float epilogue(int t0, int t1, int S, float sa0, float sa1,
                                          float sw) {
  float t = __fmul_rn((float)t0, sa0);
  if (S == 2) t = __fadd_rn(t, __fmul_rn((float)t1, sa1));
  return __fmul_rn(t, sw);
}

// Exact accumulator of one activation group from the raw dot product of
// unpacked bytes: remove the products of padding channels (only sign-bit x
// sign-bit padding is nonzero: both decode to +1, each product 64*64), undo
// the unpack scales, add the unsigned zero point times the code sum.
__device__ __forceinline__ int true_acc(int raw, int sha, int ca, int padcnt, int zp,
                                        uint8_t shw, int colsum) {
  if (ca == 1 && (shw & kShwSign)) raw -= padcnt << 12;
  return (raw >> (sha + (shw & 0x7F))) + zp * colsum;
}

// ------------------------------------------------------ unit pack/unpack --
// Pack 16 stored int8 codes (4 dwords, natural order) into one unit.
// Returns the unit's words; the unit occupies 2*c bytes.
__device__ __forceinline__ uint4 pack_unit(uint32_t d0, uint32_t d1, uint32_t d2, uint32_t d3,
                                           int c) {
  if (c == 8) return make_uint4(d0, d1, d2, d3);
  if (c == 4)
    return make_uint4((d0 & 0x0F0F0F0Fu) | ((d1 & 0x0F0F0F0Fu) << 4),
                      (d2 & 0x0F0F0F0Fu) | ((d3 & 0x0F0F0F0Fu) << 4), 0u, 0u);
  if (c == 2)
    return make_uint4(((d0 & 0x03030303u) << 2) | ((d1 & 0x03030303u) << 6) |
                          (d2 & 0x03030303u) | ((d3 & 0x03030303u) << 4),
                      0u, 0u, 0u);
  const uint32_t y = ((d0 >> 7) & 0x01010101u) | (((d1 >> 7) & 0x01010101u) << 1) |
                     (((d2 >> 7) & 0x01010101u) << 2) | (((d3 >> 7) & 0x01010101u) << 3);
  const uint32_t h = (y & 0xFu) | ((y >> 4) & 0xF0u) | ((y >> 8) & 0xF00u) | ((y >> 12) & 0xF000u);
  return make_uint4(h, 0u, 0u, 0u);
}

__device__ __forceinline__ void store_unit(uint8_t* p, uint4 u, int c) {
  if (c == 8) *reinterpret_cast<uint4*>(p) = u;
  else if (c == 4) *reinterpret_cast<uint2*>(p) = make_uint2(u.x, u.y);
  else if (c == 2) *reinterpret_cast<uint32_t*>(p) = u.x;
  else *reinterpret_cast<uint16_t*>(p) = (uint16_t)u.x;
}

__device__ __forceinline__ uint4 load_unit(const uint8_t* p, int c) {
  if (c == 8) return *reinterpret_cast<const uint4*>(p);
  if (c == 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    return make_uint4(v.x, v.y, 0u, 0u);
  }
  if (c == 2) return make_uint4(*reinterpret_cast<const uint32_t*>(p), 0u, 0u, 0u);
  return make_uint4(*reinterpret_cast<const uint16_t*>(p), 0u, 0u, 0u);
}

__device__ __forceinline__ uint4 unpack4(uint32_t w0, uint32_t w1) {
  return make_uint4((w0 << 4) & 0xF0F0F0F0u, w0 & 0xF0F0F0F0u, (w1 << 4) & 0xF0F0F0F0u,
                    w1 & 0xF0F0F0F0u);
}
__device__ __forceinline__ uint4 unpack2(uint32_t w) {
  return make_uint4((w << 4) & 0xC0C0C0C0u, w & 0xC0C0C0C0u, (w << 6) & 0xC0C0C0C0u,
                    (w << 2) & 0xC0C0C0C0u);
}
__device__ __forceinline__ uint32_t sgn1(uint32_t y, int j) {
  return ((y << (7 - j)) & 0x80808080u) | 0x40404040u;
}
__device__ __forceinline__ uint4 unpack1(uint32_t h) {
  uint32_t x = (h | (h << 8)) & 0x00FF00FFu;
  const uint32_t y = (x | (x << 4)) & 0x0F0F0F0Fu;  // byte b = nibble b of h
  return make_uint4(sgn1(y, 0), sgn1(y, 1), sgn1(y, 2), sgn1(y, 3));
}

// Unit (raw, low 2*c bytes valid) -> 16 scaled int8 elements.
template <int C>
__device__ __forceinline__ uint4 unpack_unit(uint4 raw) {
  if constexpr (C == 8) return raw;
  else if constexpr (C == 4) return unpack4(raw.x, raw.y);
  else if constexpr (C == 2) return unpack2(raw.x);
  else return unpack1(raw.x & 0xFFFFu);
}
__device__ __forceinline__ uint4 unpack_unit_rt(uint4 raw, int c) {
  if (c == 8) return raw;
  if (c == 4) return unpack4(raw.x, raw.y);
  if (c == 2) return unpack2(raw.x);
  return unpack1(raw.x & 0xFFFFu);
}

// ------------------------------------------------------------ reductions --
__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wid] = v;
  __syncthreads();
  float r = red[0];
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) r = fmaxf(r, red[i]);
  return r;
}

// Maxima of two values over the workgroup (one pair of barriers).
__device__ __forceinline__ float2 block_max2(float2 v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    v.x = fmaxf(v.x, __shfl_xor(v.x, o, 64));
    v.y = fmaxf(v.y, __shfl_xor(v.y, o, 64));
  }
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) {
    red[2 * wid] = v.x;
    red[2 * wid + 1] = v.y;
  }
  __syncthreads();
  float2 r = make_float2(red[0], red[1]);
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) {
    r.x = fmaxf(r.x, red[2 * i]);
    r.y = fmaxf(r.y, red[2 * i + 1]);
  }
  return r;
}

__device__ __forceinline__ int block_sum(int v, int* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wid] = v;
  __syncthreads();
  int r = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) r += red[i];
  return r;
}

// --------------------------------------------------------------- k_wpack --
// One workgroup per original output channel n.  Dynamic LDS: Kp bytes.
__global__ __launch_bounds__(256) void k_wpack(
    const float* __restrict__ W, int64_t K, int64_t ldw, const uint8_t* __restrict__ w_bits,
    const int32_t* __restrict__ pos, const uint8_t* __restrict__ seg,
    const int32_t* __restrict__ phys, const uint64_t* __restrict__ blk_off,
    const uint8_t* __restrict__ blk_c, QParam q_lo, QParam q_hi, int b_lo, int Kp,
    uint8_t* __restrict__ packed, ColInfo* __restrict__ colinfo) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float redf[4];
  __shared__ int redi[4];
  const int64_t n = blockIdx.x;
  const float* row = W + n * ldw;
  const int tid = threadIdx.x;

  float m = 0.0f;
  for (int64_t k = tid; k < K; k += blockDim.x) m = fmaxf(m, fabsf(row[k]));
  m = block_max(m, redf);

  const QParam q = w_bits[n] == b_lo ? q_lo : q_hi;
  const float s = group_scale(m, q);
  const bool fast = fast_ok(s);
  const float rs = fast ? __builtin_amdgcn_rcpf(s) : 0.0f;

  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < Kp / 4; i += blockDim.x) codes32[i] = 0;
  __syncthreads();
  int cs0 = 0, cs1 = 0;
  for (int64_t k = tid; k < K; k += blockDim.x) {
    const int code = quant_code(row[k], s, rs, fast, q);
    codes[pos[k]] = (uint8_t)(int8_t)code;
    if (seg[k] == 0) cs0 += code; else cs1 += code;
  }
  cs0 = block_sum(cs0, redi);
  cs1 = block_sum(cs1, redi);  // block_sum syncs, so the code writes are visible

  const int p = phys[n];
  const int blk = p / kBlk, r = p % kBlk;
  const int c = blk_c[blk];
  uint8_t* dst = packed + blk_off[blk];
  const int nunits = (Kp / kGran) * 4;
  for (int u = tid; u < nunits; u += blockDim.x) {
    const int qg = u >> 2, kg = u & 3;
    const uint4 d = *reinterpret_cast<const uint4*>(codes + qg * kGran + kg * 16);
    store_unit(dst + (int64_t)qg * 128 * c + (kg * 16 + r) * 2 * c, pack_unit(d.x, d.y, d.z, d.w, c), c);
  }
  if (tid == 0) {
    ColInfo ci;
    ci.n = (int32_t)n;
    ci.s_w = s;
    ci.colsum[0] = cs0;
    ci.colsum[1] = cs1;
    colinfo[p] = ci;
  }
}

// -------------------------------------------------------------- k_absmax --
// Max-abs of every activation group over all M rows, in two launches: each
// workgroup here writes its partial maxima (no atomics, no fences: a
// per-workgroup device-scope fence costs tens of nanoseconds each on a chip
// with per-XCD L2s); the pack kernel that follows reduces the partials.

__device__ __forceinline__ void max4(float4 v, uchar4 g, float& mx0, float& mx1) {
  const float a0 = fabsf(v.x), a1 = fabsf(v.y), a2 = fabsf(v.z), a3 = fabsf(v.w);
  mx0 = fmaxf(mx0, fmaxf(fmaxf(g.x ? 0.0f : a0, g.y ? 0.0f : a1), fmaxf(g.z ? 0.0f : a2, g.w ? 0.0f : a3)));
  mx1 = fmaxf(mx1, fmaxf(fmaxf(g.x ? a0 : 0.0f, g.y ? a1 : 0.0f), fmaxf(g.z ? a2 : 0.0f, g.w ? a3 : 0.0f)));
}

__device__ __forceinline__ void write_partial(float mx0, float mx1, float* red,
                                              float* __restrict__ partial) {
  const float2 m = block_max2(make_float2(mx0, mx1), red);
  if (threadIdx.x == 0) {
    partial[2 * blockIdx.x] = m.x;
    partial[2 * blockIdx.x + 1] = m.y;
  }
}

// Rows with K % 4 == 0, lda % 4 == 0, 16-byte aligned.  Workgroup b takes
// RB consecutive rows; thread tid owns float4 positions k4 = base + 256*j
// of every row, loads all RB rows of them at once, keeps their |max| over
// the rows (one v_max per element) and folds them into the two group
// maxima once per position batch.  Clamped rows and positions re-read
// in-bounds data already counted, which a max ignores.
template <int J, int RB>
__global__ __launch_bounds__(256) void k_absmax_blk(const float4* __restrict__ A, int64_t M,
                                                    int K4, int64_t lda4,
                                                    const uchar4* __restrict__ seg4,
                                                    float* __restrict__ partial) {
  __shared__ float red[8];
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blockIdx.x * RB;
  const int rows = (int)min((int64_t)RB, M - m0);
  float mx0 = 0.0f, mx1 = 0.0f;
  for (int base = 0; base < K4; base += 256 * J) {
    int k4[J];
#pragma unroll
    for (int j = 0; j < J; ++j) k4[j] = min(base + 256 * j + tid, K4 - 1);
    float4 v[RB][J];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const float4* row = A + (m0 + min(r, rows - 1)) * lda4;
#pragma unroll
      for (int j = 0; j < J; ++j) v[r][j] = row[k4[j]];
    }
    float4 mx[J];
#pragma unroll
    for (int j = 0; j < J; ++j) mx[j] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int j = 0; j < J; ++j) {
        mx[j].x = fmaxf(mx[j].x, fabsf(v[r][j].x));
        mx[j].y = fmaxf(mx[j].y, fabsf(v[r][j].y));
        mx[j].z = fmaxf(mx[j].z, fabsf(v[r][j].z));
        mx[j].w = fmaxf(mx[j].w, fabsf(v[r][j].w));
      }
#pragma unroll
    for (int j = 0; j < J; ++j) max4(mx[j], seg4[k4[j]], mx0, mx1);
  }
  write_partial(mx0, mx1, red, partial);
}

// Any stride or width: one row at a time, scalar loads.
__global__ __launch_bounds__(256) void k_absmax_rows(const float* __restrict__ A, int64_t M,
                                                     int64_t K, int64_t lda,
                                                     const uint8_t* __restrict__ seg,
                                                     float* __restrict__ partial) {
  __shared__ float red[8];
  float mx0 = 0.0f, mx1 = 0.0f;
  for (int64_t m = blockIdx.x; m < M; m += gridDim.x) {
    const float* row = A + m * lda;
    for (int64_t k = threadIdx.x; k < K; k += 256) {
      const float a = fabsf(row[k]);
      if (seg[k]) mx1 = fmaxf(mx1, a); else mx0 = fmaxf(mx0, a);
    }
  }
  write_partial(mx0, mx1, red, partial);
}

// Group scales from the partial maxima (every pack workgroup computes the
// same values; workgroup 0 also stores them for the GEMM epilogue).
__device__ __forceinline__ void scales_from_partials(const float* __restrict__ partial, int nparts,
                                                     const ActPlan& ap, float* red, float& s0,
                                                     float& s1, float* __restrict__ s_a_out) {
  float r0 = 0.0f, r1 = 0.0f;
  for (int b = threadIdx.x; b < nparts; b += blockDim.x) {
    const float2 v = reinterpret_cast<const float2*>(partial)[b];
    r0 = fmaxf(r0, v.x);
    r1 = fmaxf(r1, v.y);
  }
  const float2 rr = block_max2(make_float2(r0, r1), red);
  r0 = rr.x;
  r1 = rr.y;
  s0 = group_scale(r0, ap.q[0]);
  s1 = ap.S == 2 ? group_scale(r1, ap.q[1]) : 0.0f;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
}

// Quantizer state of both activation groups.
struct ActQ {
  float s[2], rs[2], lo[2], hi[2];
  int zp[2];
  bool fast[2], sign1[2];
};

__device__ __forceinline__ ActQ make_actq(const ActPlan& ap, float s0, float s1) {
  ActQ a;
  const float sv[2] = {s0, s1};
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const QParam& q = g ? ap.q[1] : ap.q[0];
    a.s[g] = sv[g];
    a.fast[g] = fast_ok(sv[g]);
    a.rs[g] = a.fast[g] ? __builtin_amdgcn_rcpf(sv[g]) : 0.0f;
    a.lo[g] = (float)q.lo;
    a.hi[g] = (float)q.hi;
    a.zp[g] = g ? ap.zp[1] : ap.zp[0];
    a.sign1[g] = q.sign1 != 0;
  }
  return a;
}

// Stored activation code of x in group g (code minus the group zero
// point): the group's parameters are selected first, then one quantizer
// runs (see quant_code for the reciprocal fast path).
__device__ __forceinline__ uint8_t store_code(float x, int g, const ActQ& a) {
  const float s = g ? a.s[1] : a.s[0];
  const float rs = g ? a.rs[1] : a.rs[0];
  const bool fast = g ? a.fast[1] : a.fast[0];
  int code;
  if (g ? a.sign1[1] : a.sign1[0]) {
    code = x < 0.0f ? -1 : 1;
  } else if (s == 0.0f) {
    code = 0;
  } else {
    const float e = x * rs;
    float t = __builtin_rintf(e);
    if (!fast || fabsf(fabsf(e - t) - 0.5f) <= 0x1p-9f) t = __builtin_rintf(__fdiv_rn(x, s));
    t = fminf(fmaxf(t, g ? a.lo[1] : a.lo[0]), g ? a.hi[1] : a.hi[0]);
    code = (int)t;
  }
  return (uint8_t)(int8_t)(code - (g ? a.zp[1] : a.zp[0]));
}

// Write the units of `nrows` rows whose stored codes sit in LDS (row r at
// codes + r*Kp) to rows m0.. of the packed activation buffer, one 2*c-byte
// unit per store.  Used when a workgroup holds fewer than 16 rows.  Row 0
// of the batch also goes, unit after unit, to xdst when that is given (the
// batch-1 GEMV's contiguous row image).
template <int C>
__device__ __forceinline__ void write_group_units(const uint8_t* codes, int nrows, int64_t m0,
                                                  int Kp, int ng, int gbase, int64_t mblk,
                                                  uint8_t* __restrict__ dst0,
                                                  uint8_t* __restrict__ xdst) {
  const int per_row = ng * 4;
  for (int r = 0; r < nrows; ++r) {
    const int64_t m = m0 + r;
    uint8_t* dst = dst0 + (m / kBlk) * mblk + (int)(m % kBlk) * 2 * C;
    const uint8_t* src = codes + r * Kp + gbase;
    for (int rest = threadIdx.x; rest < per_row; rest += blockDim.x) {
      const int qg = rest >> 2, kg = rest & 3;
      const uint4 d = *reinterpret_cast<const uint4*>(src + rest * 16);
      const uint4 u = pack_unit(d.x, d.y, d.z, d.w, C);
      store_unit(dst + qg * 128 * C + kg * 32 * C, u, C);
      if (xdst != nullptr && m == 0) store_unit(xdst + rest * 2 * C, u, C);
    }
  }
}

// ximg (null: none): the batch-1 GEMV's image of row 0, written beside the
// units when the plan has the 4-bit group 0 and 8-bit group 1 that the
// GEMV stages: group 0's 8-byte units in planned order, then group 1's
// 16-byte units (at 32 bytes per granule of group 0).
__device__ __forceinline__ void write_act_units(const uint8_t* codes, int nrows, int64_t m0,
                                                const ActPlan& ap, uint8_t* __restrict__ packed,
                                                uint8_t* __restrict__ ximg = nullptr) {
  for (int g = 0; g < ap.S; ++g) {
    const int c = g ? ap.c[1] : ap.c[0];
    const int ng = g ? ap.ng[1] : ap.ng[0];
    const int gbase = g ? ap.kpad[0] : 0;
    const int64_t mblk = g ? ap.mblk_bytes[1] : ap.mblk_bytes[0];
    uint8_t* dst0 = packed + (g ? ap.seg_off[1] : ap.seg_off[0]);
    uint8_t* xdst = ximg != nullptr && c == (g ? 8 : 4) ? ximg + (g ? ap.ng[0] * 32 : 0) : nullptr;
    if (c == 8) write_group_units<8>(codes, nrows, m0, ap.Kp, ng, gbase, mblk, dst0, xdst);
    else if (c == 4) write_group_units<4>(codes, nrows, m0, ap.Kp, ng, gbase, mblk, dst0, xdst);
    else if (c == 2) write_group_units<2>(codes, nrows, m0, ap.Kp, ng, gbase, mblk, dst0, nullptr);
    else write_group_units<1>(codes, nrows, m0, ap.Kp, ng, gbase, mblk, dst0, nullptr);
  }
}

// Per-element quantizer parameters of one group, arranged so that the
// common case needs no branch: code = clamp(rint(x*rs) - zp, lo - zp,
// hi - zp).  rs is NaN where the reciprocal shortcut is not exact enough
// (scale outside [2^-100, 2^100]), which sends every element of the group
// through the exact division; a zero scale has rs = 0 and gives code 0.
struct QElem {
  float rs, lo, hi, zp, s;
};

__device__ __forceinline__ QElem qelem(float s, const QParam& q, int zp) {
  QElem e;
  e.s = s;
  e.rs = s == 0.0f ? 0.0f : fast_ok(s) ? __builtin_amdgcn_rcpf(s) : __builtin_nanf("");
  e.zp = (float)zp;
  e.lo = (float)(q.lo - zp);
  e.hi = (float)(q.hi - zp);
  return e;
}

// Stored code (code - zp) of x.  The shortcut rint(x * rcp(s)) equals
// rint(x / s) unless x/s lies near a rounding tie: v_rcp_f32 is within 1 ulp
// and the product adds half an ulp, so for |x/s| <= 256 the two quotients
// differ by less than 256 * 2^-22 = 2^-14; inside a band of 2^-12 around a
// tie (or when the shortcut is off, rs NaN) the exact IEEE quotient decides.
constexpr float kTieBand = 0x1p-12f;

// Shortcut code (stored code = code - zp) and whether x/s lies in the band.
__device__ __forceinline__ int qfast(float x, float rs, float lo, float hi, float zp, bool& near) {
  const float e = x * rs;
  const float t = __builtin_rintf(e);
  near = !(fabsf(fabsf(e - t) - 0.5f) > kTieBand);
  return (int)__builtin_amdgcn_fmed3f(t - zp, lo, hi);
}

__device__ __forceinline__ int qexact(float x, float lo, float hi, float zp, float s) {
  const float t = s == 0.0f ? 0.0f : __builtin_rintf(__fdiv_rn(x, s));
  return (int)__builtin_amdgcn_fmed3f(t - zp, lo, hi);
}

__device__ __forceinline__ int qstore(float x, float rs, float lo, float hi, float zp, float s) {
  bool near;
  const int c = qfast(x, rs, lo, hi, zp, near);
  return near ? qexact(x, lo, hi, zp, s) : c;
}

// Four elements sharing one branch for the rare exact path.
struct QE4 {
  float rs[4], lo[4], hi[4], zp[4], s[4];
};

__device__ __forceinline__ void qstore4(const float4& v, const QE4& q, uint8_t* row, int4 p) {
  bool n0, n1, n2, n3;
  int c0 = qfast(v.x, q.rs[0], q.lo[0], q.hi[0], q.zp[0], n0);
  int c1 = qfast(v.y, q.rs[1], q.lo[1], q.hi[1], q.zp[1], n1);
  int c2 = qfast(v.z, q.rs[2], q.lo[2], q.hi[2], q.zp[2], n2);
  int c3 = qfast(v.w, q.rs[3], q.lo[3], q.hi[3], q.zp[3], n3);
  if ((n0 | n1 | n2 | n3)) [[unlikely]] {
    if (n0) c0 = qexact(v.x, q.lo[0], q.hi[0], q.zp[0], q.s[0]);
    if (n1) c1 = qexact(v.y, q.lo[1], q.hi[1], q.zp[1], q.s[1]);
    if (n2) c2 = qexact(v.z, q.lo[2], q.hi[2], q.zp[2], q.s[2]);
    if (n3) c3 = qexact(v.w, q.lo[3], q.hi[3], q.zp[3], q.s[3]);
  }
  row[p.x] = (uint8_t)c0;
  row[p.y] = (uint8_t)c1;
  row[p.z] = (uint8_t)c2;
  row[p.w] = (uint8_t)c3;
}

// ------------------------------------------------------------ k_act_rows --
// R activation rows per workgroup: reduce the partial maxima, quantize the
// rows into LDS at their group-ordered positions, write their units.
// Thread tid owns float4 positions base + tid + 256*j (j < J) of every row;
// their LDS positions and group parameters are looked up once for all R
// rows.  The first batch of rows is loaded before the partial maxima are
// reduced, so the two latencies overlap.  Groups of 1-bit sign codes, and
// unaligned rows, take the generic per-element quantizer (J = 0).
// Dynamic LDS: R*Kp bytes.
template <int R, int J>
__device__ __forceinline__ void act_rows_load(const float* __restrict__ A, int64_t m0, int rows,
                                              int64_t lda, int K4, int base,
                                              const int32_t* __restrict__ pos,
                                              const uint8_t* __restrict__ seg, int4 (&p)[J],
                                              uchar4 (&g)[J], float4 (&v)[R][J]) {
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int k4 = min(base + 256 * j, K4 - 1);
    p[j] = reinterpret_cast<const int4*>(pos)[k4];
    g[j] = reinterpret_cast<const uchar4*>(seg)[k4];
#pragma unroll
    for (int r = 0; r < R; ++r)
      v[r][j] = *reinterpret_cast<const float4*>(A + (m0 + min(r, rows - 1)) * lda + 4 * k4);
  }
}

template <int R, int J>
__device__ __forceinline__ void act_rows_quant(uint8_t* codes, int Kp, int rows, int K4, int base,
                                               const int4 (&p)[J], const uchar4 (&g)[J],
                                               const float4 (&v)[R][J], const QElem& q0,
                                               const QElem& q1) {
#pragma unroll
  for (int j = 0; j < J; ++j) {
    if (base + 256 * j < K4) {
      const uchar4 h = g[j];
      QE4 q;
      const bool hv[4] = {h.x != 0, h.y != 0, h.z != 0, h.w != 0};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        q.rs[e] = hv[e] ? q1.rs : q0.rs;
        q.lo[e] = hv[e] ? q1.lo : q0.lo;
        q.hi[e] = hv[e] ? q1.hi : q0.hi;
        q.zp[e] = hv[e] ? q1.zp : q0.zp;
        q.s[e] = hv[e] ? q1.s : q0.s;
      }
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (r < rows) qstore4(v[r][j], q, codes + r * Kp, p[j]);
    }
  }
}

template <int R, int J>
__global__ __launch_bounds__(256) void k_act_rows(const float* __restrict__ A, int64_t M,
                                                  int64_t K, int64_t lda,
                                                  const int32_t* __restrict__ pos,
                                                  const uint8_t* __restrict__ seg, ActPlan ap,
                                                  const float* __restrict__ partial, int nparts,
                                                  float* __restrict__ s_a_out,
                                                  uint8_t* __restrict__ packed,
                                                  uint8_t* __restrict__ ximg) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  // R = 4: the four workgroups of one 16-row block run on one XCD
  // (workgroup i goes to XCD i mod 8), so its L2 joins their partial unit
  // lines before they reach HBM; the grid is a multiple of 32 workgroups
  int64_t wg = blockIdx.x;
  if constexpr (R == 4) {
    const int64_t x = wg & 7, j = wg >> 3;
    wg = 4 * ((j >> 2) * 8 + x) + (j & 3);
  }
  const int64_t m0 = wg * R;
  if (m0 >= M) return;
  const int rows = (int)min((int64_t)R, M - m0);
  const int tid = threadIdx.x;
  if constexpr (J > 0) {
    const int K4 = (int)(K / 4);
    int4 p[J];
    uchar4 g[J];
    float4 v[R][J];
    act_rows_load<R, J>(A, m0, rows, lda, K4, tid, pos, seg, p, g, v);
    uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
    for (int i = tid; i < rows * ap.Kp / 4; i += blockDim.x) codes32[i] = 0;
    float s0, s1;
    scales_from_partials(partial, nparts, ap, red, s0, s1, s_a_out);  // syncs
    const QElem q0 = qelem(s0, ap.q[0], ap.zp[0]), q1 = qelem(s1, ap.q[1], ap.zp[1]);
    act_rows_quant<R, J>(codes, ap.Kp, rows, K4, tid, p, g, v, q0, q1);
    for (int base = tid + 256 * J; base < K4; base += 256 * J) {
      act_rows_load<R, J>(A, m0, rows, lda, K4, base, pos, seg, p, g, v);
      act_rows_quant<R, J>(codes, ap.Kp, rows, K4, base, p, g, v, q0, q1);
    }
  } else {
    uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
    for (int i = tid; i < rows * ap.Kp / 4; i += blockDim.x) codes32[i] = 0;
    float s0, s1;
    scales_from_partials(partial, nparts, ap, red, s0, s1, s_a_out);  // syncs
    const ActQ aq = make_actq(ap, s0, s1);
    for (int r = 0; r < rows; ++r)
      for (int64_t k = tid; k < K; k += blockDim.x)
        codes[(int64_t)r * ap.Kp + pos[k]] = store_code(A[(m0 + r) * lda + k], seg[k], aq);
  }
  __syncthreads();
  write_act_units(codes, rows, m0, ap, packed, ximg);
}

// ------------------------------------------------------------ k_act_bf16 --
// Activations of the next layer from a producer's stored bf16 outputs Y
// with the batch maximum (the two-pass form of quantization fused into the
// producer): each group's maximum |Y| is the largest over nslot pairs
// (one per producer tile, written by its epilogue), or with
// nslot = 0 every workgroup reduces it from the whole batch itself (small
// batches).  R rows per workgroup are then quantized exactly as k_act_rows
// quantizes float rows (the bf16 values widened, which is exact), and
// written as units.  J > 0: rows with K % 4 == 0 and ldy % 4 == 0, Y 8-byte
// aligned, J bf16 quadruples per thread per pass; J = 0: any layout, one
// element at a time.  Dynamic LDS: R*Kp bytes.
__device__ __forceinline__ float4 bf16x4(const uint16_t* p) {
  const uint2 w = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u),
                     __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xFFFF0000u));
}

template <int R, int J>
__global__ __launch_bounds__(256) void k_act_bf16(const uint16_t* __restrict__ Y, int64_t M,
                                                  int64_t K, int64_t ldy,
                                                  const int32_t* __restrict__ pos,
                                                  const uint8_t* __restrict__ seg, ActPlan ap,
                                                  const float* __restrict__ slots, int nslot,
                                                  float* __restrict__ s_a_out,
                                                  uint8_t* __restrict__ packed,
                                                  uint8_t* __restrict__ ximg) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int64_t m0 = (int64_t)blockIdx.x * R;
  const int rows = (int)min((int64_t)R, M - m0);
  const int tid = threadIdx.x;
  // the first batch of the rows' values is loaded before the maxima are
  // reduced, so the two latencies overlap
  constexpr int JJ = J > 0 ? J : 1;
  const int K4 = (int)(K / 4);
  int4 p[JJ];
  uchar4 g[JJ];
  float4 v[R][JJ];
  auto load = [&](int base) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < JJ; ++j) {
      const int k4 = min(base + 256 * j, K4 - 1);
      p[j] = reinterpret_cast<const int4*>(pos)[k4];
      g[j] = reinterpret_cast<const uchar4*>(seg)[k4];
#pragma unroll
      for (int r = 0; r < R; ++r) v[r][j] = bf16x4(Y + (m0 + min(r, rows - 1)) * ldy + 4 * k4);
    }
  };
  if constexpr (J > 0) load(tid);
  float r0 = 0.0f, r1 = 0.0f;
  if (nslot > 0) {
    for (int b = tid; b < nslot; b += 256) {
      const float2 sv = reinterpret_cast<const float2*>(slots)[b];
      r0 = fmaxf(r0, sv.x);
      r1 = fmaxf(r1, sv.y);
    }
  } else if (J > 0) {
    // the whole (small) batch: eight loads in flight per thread, then their
    // maxima (a clamped repeat changes no maximum)
    const uchar4* s4 = reinterpret_cast<const uchar4*>(seg);
    const int64_t tot = M * K4;
    for (int64_t f0 = tid; f0 < tot; f0 += 256 * 8) {
      float4 yv[8];
      uchar4 sv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int64_t f = min(f0 + 256 * u, tot - 1);
        const int64_t m = f / K4;
        const int k4 = (int)(f - m * K4);
        yv[u] = bf16x4(Y + m * ldy + 4 * k4);
        sv[u] = s4[k4];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) max4(yv[u], sv[u], r0, r1);
    }
  } else {
    for (int64_t m = 0; m < M; ++m)
      for (int64_t k = tid; k < K; k += 256) {
        const float a = fabsf(__uint_as_float((uint32_t)Y[m * ldy + k] << 16));
        if (seg[k]) r1 = fmaxf(r1, a); else r0 = fmaxf(r0, a);
      }
  }
  const float2 rr = block_max2(make_float2(r0, r1), red);
  const float s0 = group_scale(rr.x, ap.q[0]);
  const float s1 = ap.S == 2 ? group_scale(rr.y, ap.q[1]) : 0.0f;
  if (blockIdx.x == 0 && tid == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < rows * ap.Kp / 4; i += 256) codes32[i] = 0;
  __syncthreads();
  if constexpr (J > 0) {
    const QElem q0 = qelem(s0, ap.q[0], ap.zp[0]), q1 = qelem(s1, ap.q[1], ap.zp[1]);
    for (int base = tid; base < K4; base += 256 * J) {
      if (base != tid) load(base);
      act_rows_quant<R, J>(codes, ap.Kp, rows, K4, base, p, g, v, q0, q1);
    }
  } else {
    const ActQ aq = make_actq(ap, s0, s1);
    for (int r = 0; r < rows; ++r)
      for (int64_t k = tid; k < K; k += 256)
        codes[(int64_t)r * ap.Kp + pos[k]] =
            store_code(__uint_as_float((uint32_t)Y[(m0 + r) * ldy + k] << 16), seg[k], aq);
  }
  __syncthreads();
  write_act_units(codes, rows, m0, ap, packed, ximg);
}

// The two-pass form into a next convolution: its byte image (blocked: row
// m, rank-space position p at (m/16)*16*Cp + 16p + m%16, as the GEMM tiles'
// epilogue writes it) from the stored bf16 Y, with each group's maximum
// from nslot tile pairs (nslot = 0: reduced from the whole batch).  posn
// gives each producer column's position in rank space (group 1 from
// cpad0).  Workgroup b quantizes 16-row block b into LDS (rank-major, 16
// rows a position: one thread a channel) with the arithmetic of
// soniq_quantize_act, then writes the block's 16*Cp bytes; workgroup 0
// also stores the scales.  Dynamic
// LDS: 16 * Cp bytes.
__global__ __launch_bounds__(256) void k_img_bf16(const uint16_t* __restrict__ Y, int64_t M, int N,
                                                  int64_t ldy, const int32_t* __restrict__ posn,
                                                  int cpad0, int Cp, ActPlan ap,
                                                  const float* __restrict__ slots, int nslot,
                                                  float* __restrict__ s_a_out,
                                                  uint8_t* __restrict__ bimg) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int64_t m0 = (int64_t)blockIdx.x * kBlk;
  const int rows = (int)min((int64_t)kBlk, M - m0);
  const int tid = threadIdx.x;
  float r0 = 0.0f, r1 = 0.0f;
  if (nslot > 0) {
    for (int b = tid; b < nslot; b += 256) {
      const float2 v = reinterpret_cast<const float2*>(slots)[b];
      r0 = fmaxf(r0, v.x);
      r1 = fmaxf(r1, v.y);
    }
  } else {
    for (int64_t i = tid; i < M * N; i += 256) {
      const int64_t m = i / N;
      const int n = (int)(i - m * N);
      const float a = fabsf(__uint_as_float((uint32_t)Y[m * ldy + n] << 16));
      if (posn[n] >= cpad0) r1 = fmaxf(r1, a); else r0 = fmaxf(r0, a);
    }
  }
  const float2 rr = block_max2(make_float2(r0, r1), red);
  const float s0 = group_scale(rr.x, ap.q[0]);
  const float s1 = ap.S == 2 ? group_scale(rr.y, ap.q[1]) : 0.0f;
  if (blockIdx.x == 0 && tid == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
  const ActQ aq = make_actq(ap, s0, s1);
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < 4 * Cp; i += 256) codes32[i] = 0;
  __syncthreads();
  // thread n takes channel n: its 16 rows' values (each row's loads
  // coalesced across the threads), their codes as one 16-byte position
  for (int n = tid; n < N; n += 256) {
    const int p = posn[n];
    const int g = p >= cpad0 ? 1 : 0;
    uint32_t yv[kBlk];
#pragma unroll
    for (int r = 0; r < kBlk; ++r) yv[r] = Y[(m0 + min(r, rows - 1)) * ldy + n];
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int r = 0; r < kBlk; ++r) {
      const uint32_t c = r < rows ? store_code(__uint_as_float(yv[r] << 16), g, aq) : 0u;
      w[r >> 2] |= c << (8 * (r & 3));
    }
    *reinterpret_cast<uint4*>(codes + 16 * p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
  __syncthreads();
  uint4* dst = reinterpret_cast<uint4*>(bimg + (m0 / kBlk) * (int64_t)kBlk * Cp);
  for (int i = tid; i < Cp; i += 256) dst[i] = reinterpret_cast<const uint4*>(codes)[i];
}

// One group's units of a 16-row block whose stored codes sit in LDS (row r
// at codes + r*ldc + gbase): granule q holds units l = kg*16 + r of 2C bytes
// (128C contiguous bytes); 16-byte piece w holds units w*U .. w*U+U-1
// (U = 8/C), i.e. rows of one 16-channel group.  zx (a byte replicated)
// is XORed into every code byte first: codes held without their zero
// point get it applied here.
template <int C, int RB>
__device__ __forceinline__ void write_block_pieces(const uint8_t* codes, int ldc, int gbase, int ng,
                                                   int r0, uint8_t* __restrict__ dst,
                                                   uint32_t zx = 0u) {
  constexpr int U = 8 / C;            // units per piece
  constexpr int PK = RB / U > 0 ? RB / U : 1;  // pieces per 16-channel group
  static_assert(RB % U == 0, "row range covers whole pieces");
  const int npieces = ng * 4 * PK;
  for (int i = threadIdx.x; i < npieces; i += blockDim.x) {
    const int q = i / (4 * PK), rem = i - q * 4 * PK;
    const int kg = rem / PK, pr = rem - kg * PK;
    const int w = (kg * 16 + r0) / U + pr;  // piece within the granule
    uint32_t wd[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int l = w * U + u, r = (l & 15) - r0;
      const uint4 d = *reinterpret_cast<const uint4*>(codes + r * ldc + gbase + q * kGran + kg * 16);
      const uint4 pk = pack_unit(d.x ^ zx, d.y ^ zx, d.z ^ zx, d.w ^ zx, C);
      if constexpr (C == 8) {
        wd[0] = pk.x; wd[1] = pk.y; wd[2] = pk.z; wd[3] = pk.w;
      } else if constexpr (C == 4) {
        wd[2 * u] = pk.x; wd[2 * u + 1] = pk.y;
      } else if constexpr (C == 2) {
        wd[u] = pk.x;
      } else {
        wd[u >> 1] |= (pk.x & 0xFFFFu) << (16 * (u & 1));
      }
    }
    *reinterpret_cast<uint4*>(dst + (int64_t)(q * 8 * C + w) * 16) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
  }
}

// ----------------------------------------------------------- k_act_blk16 --
// RB rows (8 or 16, aligned to a 16-row block) per workgroup, aligned rows,
// no sign-code group: the rows go through in batches of four, the next
// batch's loads in flight while the current one is quantized into LDS; the
// partial maxima are reduced once; the rows' packed units are then written
// as whole 16-byte pieces (each 16-channel group's units of these rows are
// contiguous).  Rows past M are clamped to row M-1 (in bounds) and their
// units land in padding rows, which no consumer reads.
// Dynamic LDS: RB*Kp bytes.
template <int J, int RB>
__global__ __launch_bounds__(256) void k_act_blk16(const float* __restrict__ A, int64_t M,
                                                   int64_t K, int64_t lda,
                                                   const int32_t* __restrict__ pos,
                                                   const uint8_t* __restrict__ seg, ActPlan ap,
                                                   const float* __restrict__ partial, int nparts,
                                                   float* __restrict__ s_a_out,
                                                   uint8_t* __restrict__ packed) {
  static_assert(RB == 8 || RB == 16, "row batch");
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int64_t m0 = (int64_t)blockIdx.x * RB;
  const int rows = (int)min((int64_t)RB, M - m0);
  const int tid = threadIdx.x;
  const int K4 = (int)(K / 4);
  int4 p[J];
  uchar4 g[J];
  float4 va[4][J], vb[4][J];
  // batch b holds rows 4b..4b+3 (clamped into the valid rows)
  auto load = [&](float4 (&v)[4][J], int b) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int k4 = min(tid + 256 * j, K4 - 1);
#pragma unroll
      for (int r = 0; r < 4; ++r)
        v[r][j] = *reinterpret_cast<const float4*>(A + (m0 + min(4 * b + r, rows - 1)) * lda + 4 * k4);
    }
  };
  load(va, 0);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int k4 = min(tid + 256 * j, K4 - 1);
    p[j] = reinterpret_cast<const int4*>(pos)[k4];
    g[j] = reinterpret_cast<const uchar4*>(seg)[k4];
  }
  load(vb, 1);
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < RB * ap.Kp / 4; i += 256) codes32[i] = 0;
  float s0, s1;
  scales_from_partials(partial, nparts, ap, red, s0, s1, s_a_out);  // syncs
  const QElem q0 = qelem(s0, ap.q[0], ap.zp[0]), q1 = qelem(s1, ap.q[1], ap.zp[1]);
  act_rows_quant<4, J>(codes, ap.Kp, 4, K4, tid, p, g, va, q0, q1);
  if constexpr (RB == 16) load(va, 2);
  act_rows_quant<4, J>(codes + 4 * ap.Kp, ap.Kp, 4, K4, tid, p, g, vb, q0, q1);
  if constexpr (RB == 16) {
    load(vb, 3);
    act_rows_quant<4, J>(codes + 8 * ap.Kp, ap.Kp, 4, K4, tid, p, g, va, q0, q1);
    act_rows_quant<4, J>(codes + 12 * ap.Kp, ap.Kp, 4, K4, tid, p, g, vb, q0, q1);
  }
  __syncthreads();
  const int r0 = (int)(m0 % kBlk);
  for (int gi = 0; gi < ap.S; ++gi) {
    const int c = gi ? ap.c[1] : ap.c[0];
    const int ng = gi ? ap.ng[1] : ap.ng[0];
    const int gbase = gi ? ap.kpad[0] : 0;
    uint8_t* dst = packed + (gi ? ap.seg_off[1] : ap.seg_off[0]) +
                   (m0 / kBlk) * (gi ? ap.mblk_bytes[1] : ap.mblk_bytes[0]);
    if (c == 8) write_block_pieces<8, RB>(codes, ap.Kp, gbase, ng, r0, dst);
    else if (c == 4) write_block_pieces<4, RB>(codes, ap.Kp, gbase, ng, r0, dst);
    else if (c == 2) write_block_pieces<2, RB>(codes, ap.Kp, gbase, ng, r0, dst);
    else write_block_pieces<1, RB>(codes, ap.Kp, gbase, ng, r0, dst);
  }
}

// ------------------------------------------------- wait and LDS helpers --
// s_waitcnt immediate for vmcnt(n) (gfx9 encoding), expcnt/lgkmcnt untouched.
#define SONIQ_VMCNT_IMM(n) (((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))
// s_waitcnt immediate for lgkmcnt(0) alone (vmcnt and expcnt at their maxima).
#define SONIQ_LGKMCNT0_IMM (0xF | (3 << 14) | (0x7 << 4))

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(SONIQ_VMCNT_IMM(N));
}

// Workgroup barrier without a memory fence, for LDS filled by direct
// loads whose completion each wave has already awaited with wait_vm; the
// compiler fences keep LDS accesses on their side.
__device__ __forceinline__ void bar_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// block_max2 with fence-free barriers, for workgroups whose global loads
// must stay in flight across it; red is used once.
__device__ __forceinline__ float2 block_max2_nofence(float2 v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    v.x = fmaxf(v.x, __shfl_xor(v.x, o, 64));
    v.y = fmaxf(v.y, __shfl_xor(v.y, o, 64));
  }
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) {
    red[2 * wid] = v.x;
    red[2 * wid + 1] = v.y;
  }
  __builtin_amdgcn_s_waitcnt(SONIQ_LGKMCNT0_IMM);
  bar_nofence();
  float2 r = make_float2(red[0], red[1]);
  for (int i = 1; i < (int)(blockDim.x >> 6); ++i) {
    r.x = fmaxf(r.x, red[2 * i]);
    r.y = fmaxf(r.y, red[2 * i + 1]);
  }
  return r;
}

// All but the last N loads of this wave have landed, direct-to-LDS ones
// included; LDS reads stay after it.
template <int N>
__device__ __forceinline__ void lds_dma_wait() {
  wait_vm<N>();
  asm volatile("" ::: "memory");
}

// Buffer-resource offset past any buffer: the load returns zero without
// touching memory.
constexpr uint32_t kOOB = 0x7FFFFFF0u;

// LDS byte address of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_off(const uint8_t* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) uint8_t*)p);
}

// ------------------------------------------------------------ k_act_coop --
// One pass over HBM for batches that fit in the registers of the chip.
// The grid is no larger than the number of workgroups that can be resident
// at once, so every workgroup holds its rows while the group maxima meet.
// Workgroup b holds the RB rows m0 = RB*b .. of one 16-row block
// (RB = 4, 8 or 16): its RB*K4 float4 are spread evenly over the 256
// threads, thread tid taking flat positions f = tid + 256*i (i < T) with
// row f / K4 and position f % K4.  It folds its group maxima into the
// grid's, waits until every workgroup has done so, quantizes the rows it
// still holds into LDS and writes their units as whole pieces.  Rows past
// M are clamped to row M-1 for the loads and left as zero codes, which
// land in padding rows.  Dynamic LDS: RB*Kp code bytes, then the K
// planned positions (group 1 starts at planned position kpad[0]), padded
// to a multiple of 256, then TL*4 KB of row data.
//
// Grid state (zero when the handle is made, and left that way between
// calls), in 32-bit words, each counter on a 128-byte line of its own:
//   sub[x]     at 32*x          arrivals of workgroups b with b % 8 == x
//   top        at kBarTop       groups x complete
//   gen[x]     at kBarGen+32*x  generation, one copy per group (equal)
//   max[p][x][g] at kBarMax+32*(8p+x)+g  group maxima (float bits) of
//                               the call with generation parity p
// Only relaxed agent-scope atomics touch this state, and each step waits
// for the previous one's returned value before it issues, so a workgroup
// that sees the generation move also sees every folded maximum.  No L2
// write-back or invalidate is needed (the rows stay in registers).  The
// last arrival of a group resets its sub counter, the last group resets
// top and the other parity's maxima, then advances every gen copy.
constexpr int kBarTop = 256, kBarGen = 288, kBarMax = 544;
constexpr int kBarWords = kBarMax + 32 * 16;
static_assert(kBarWords <= kActStateWords, "grid state fits the handle's words");
// Sub-group scales: block maxima maxg[p][x][j] at kBarMaxG + kGSubMax*(8p + x)
// + j (the same counters and generation words as above).
constexpr int kBarMaxG = 1088;
static_assert(kBarMaxG >= kBarWords && kBarMaxG + 16 * kGSubMax <= kActStateWords,
              "block maxima fit the handle's words");

// Spin limit of the wait: far beyond any real wait (a few tenths of a
// second).  A workgroup that times out (its grid was not resident after
// all) computes the maxima itself from the whole batch, so the result is
// the same, only slower.  SONIQ_COOP_SPINS overrides the limit (tests set
// it to 0 to run that path).
constexpr unsigned kBarrierSpins = 1u << 18;
// Count of workgroups whose wait timed out, kept for the handle's lifetime
// (the barrier protocol never touches it): a grid that was not resident
// after all is slow, not wrong, and this word makes that visible.
static_assert(kBarMaxG + 16 * kGSubMax <= kActStallWord && kActStallWord < kActStateWords,
              "the stall count has a word of its own");

__device__ __forceinline__ unsigned bar_load(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned bar_add(unsigned* p, unsigned v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void bar_store(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Make the following atomics wait for v (an atomic's returned value).
__device__ __forceinline__ void bar_after(unsigned v) {
  asm volatile("" ::"v"(v) : "memory");
}

// This workgroup's generation word; thread 0 reads it before arriving (it
// cannot move before every workgroup has arrived).
__device__ __forceinline__ unsigned* grid_gen_word(unsigned* st) {
  return st + kBarGen + 32 * (blockIdx.x & 7);
}

// Fold (mx0, mx1) into the grid maxima and wait for every workgroup.
// Thread 0 only, gen = this call's generation; returns false when the
// wait timed out.
__device__ __forceinline__ bool grid_fold_max(unsigned* st, unsigned gen, unsigned spins,
                                              float mx0, float mx1, float& g0, float& g1) {
  const unsigned x = blockIdx.x & 7;
  const unsigned ngroups = gridDim.x < 8 ? gridDim.x : 8;
  const unsigned nx = (gridDim.x - x + 7) / 8;  // workgroups in group x
  unsigned* genx = st + kBarGen + 32 * x;
  bar_after(gen);
  unsigned* mp = st + kBarMax + 32 * (8 * (gen & 1));
  const unsigned o0 = __hip_atomic_fetch_max(mp + 32 * x, __float_as_uint(mx0), __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
  const unsigned o1 = __hip_atomic_fetch_max(mp + 32 * x + 1, __float_as_uint(mx1),
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  bar_after(o0 | o1);
  bool ok = true, last = false;
  const unsigned a1 = bar_add(st + 32 * x, 1u);
  bar_after(a1);
  if (a1 == nx - 1) {
    bar_store(st + 32 * x, 0u);
    const unsigned a2 = bar_add(st + kBarTop, 1u);
    bar_after(a2);
    if (a2 == ngroups - 1) {
      bar_store(st + kBarTop, 0u);
      unsigned* other = st + kBarMax + 32 * (8 * ((gen & 1) ^ 1));
      for (int i = 0; i < 8; ++i) {
        bar_store(other + 32 * i, 0u);
        bar_store(other + 32 * i + 1, 0u);
      }
      // the maxima were folded before every arrival, so the copies can go
      // out together
      for (int i = 0; i < 8; ++i) bar_add(st + kBarGen + 32 * i, 1u);
      last = true;
    }
  }
  if (!last) {
    unsigned n = 0;
    unsigned now;
    while ((now = bar_load(genx)) == gen) {
      if (++n > spins) {
        ok = false;
        break;
      }
      __builtin_amdgcn_s_sleep(20);
    }
    bar_after(now);
  }
  unsigned m0 = 0, m1 = 0;
  for (int i = 0; i < 8; ++i) {
    m0 = max(m0, bar_load(mp + 32 * i));
    m1 = max(m1, bar_load(mp + 32 * i + 1));
  }
  g0 = __uint_as_float(m0);
  g1 = __uint_as_float(m1);
  return ok;
}

// Fold n block maxima (LDS words mx[0..n), n <= kGSubMax, non-negative
// floats as bits) into the grid's and wait for every workgroup: run by all
// of wave 0, gen = this call's generation in lane 0.  The same protocol as
// grid_fold_max with the maxima spread over the wave's lanes; the last
// arrival's whole wave clears the other parity's maxima.  On return mx[j]
// holds the grid maximum of block j; false (every lane) when the wait
// timed out.
__device__ __forceinline__ bool grid_fold_max_n(unsigned* st, unsigned gen, unsigned spins,
                                                unsigned* mx, int n) {
  const int lane = threadIdx.x & 63;
  gen = __builtin_amdgcn_readfirstlane(gen);
  const unsigned x = blockIdx.x & 7;
  const unsigned ngroups = gridDim.x < 8 ? gridDim.x : 8;
  const unsigned nx = (gridDim.x - x + 7) / 8;
  unsigned* cur = st + kBarMaxG + 8 * kGSubMax * (gen & 1);
  unsigned done = gen;
  for (int j = lane; j < n; j += 64)
    done |= __hip_atomic_fetch_max(cur + x * kGSubMax + j, mx[j], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
  bar_after(done);
  int last = 0, ok = 1;
  if (lane == 0) {
    const unsigned a1 = bar_add(st + 32 * x, 1u);
    bar_after(a1);
    if (a1 == nx - 1) {
      bar_store(st + 32 * x, 0u);
      const unsigned a2 = bar_add(st + kBarTop, 1u);
      bar_after(a2);
      if (a2 == ngroups - 1) {
        bar_store(st + kBarTop, 0u);
        last = 1;
      }
    }
  }
  last = __shfl(last, 0, 64);
  if (last) {
    // every fold came before its arrival: the other parity's maxima can be
    // cleared for the next call, then the generation advances
    unsigned* other = st + kBarMaxG + 8 * kGSubMax * ((gen & 1) ^ 1);
    for (int xx = 0; xx < 8; ++xx)
      for (int j = lane; j < n; j += 64) bar_store(other + xx * kGSubMax + j, 0u);
    if (lane == 0)
      for (int i = 0; i < 8; ++i) bar_add(st + kBarGen + 32 * i, 1u);
  } else if (lane == 0) {
    unsigned* genx = st + kBarGen + 32 * x;
    unsigned c = 0, now;
    while ((now = bar_load(genx)) == gen) {
      if (++c > spins) {
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(20);
    }
    bar_after(now);
  }
  ok = __shfl(ok, 0, 64);
  for (int j = lane; j < n; j += 64) {
    unsigned m = 0;
    for (int xx = 0; xx < 8; ++xx) m = max(m, bar_load(cur + xx * kGSubMax + j));
    mx[j] = m;
  }
  return ok != 0;
}

// Block maxima of the whole batch, by this workgroup alone (the timed-out
// wait only): block index in bits 16.. of the planned-position table.
__device__ __forceinline__ void absmax_all_blocks(const float* __restrict__ A, int64_t M, int K4,
                                                  int64_t lda, const int4* pos4, unsigned* mx,
                                                  int n) {
  for (int j = threadIdx.x; j < n; j += 256) mx[j] = 0u;
  __syncthreads();
  for (int64_t m = 0; m < M; ++m)
    for (int k = threadIdx.x; k < K4; k += 256) {
      const int4 p = pos4[k];
      const float4 v = *reinterpret_cast<const float4*>(A + m * lda + 4 * k);
      atomicMax(&mx[p.x >> 16], __float_as_uint(fabsf(v.x)));
      atomicMax(&mx[p.y >> 16], __float_as_uint(fabsf(v.y)));
      atomicMax(&mx[p.z >> 16], __float_as_uint(fabsf(v.z)));
      atomicMax(&mx[p.w >> 16], __float_as_uint(fabsf(v.w)));
    }
  __syncthreads();
}

// Group maxima of the whole batch, by this workgroup alone (the timed-out
// wait only).  pos4: LDS copy of the planned positions; group 1 starts at
// planned position kp0.
__device__ __forceinline__ void absmax_all(const float* __restrict__ A, int64_t M, int K4,
                                           int64_t lda, const int4* pos4, int kp0, float* red,
                                           float& g0, float& g1) {
  float mx0 = 0.0f, mx1 = 0.0f;
  for (int64_t m = 0; m < M; ++m)
    for (int k = threadIdx.x; k < K4; k += 256) {
      const int4 p = pos4[k];
      max4(*reinterpret_cast<const float4*>(A + m * lda + 4 * k),
           make_uchar4(p.x >= kp0, p.y >= kp0, p.z >= kp0, p.w >= kp0), mx0, mx1);
    }
  const float2 r = block_max2(make_float2(mx0, mx1), red);
  g0 = r.x;
  g1 = r.y;
}

// Step from flat position (r, k) to (r, k) + 256 within rows of K4 float4:
// 256 = q256*K4 + r256.
__device__ __forceinline__ void coop_step(int& r, int& k, int K4, int q256, int r256) {
  k += r256;
  r += q256;
  if (k >= K4) {
    k -= K4;
    ++r;
  }
}

__device__ __forceinline__ void coop_first(int& r, int& k, int K4) {
  r = 0;
  k = threadIdx.x;
  if (k >= K4) {
    r = k / K4;
    k -= r * K4;
  }
}

// Rounding by the 1.5*2^23 shift: for |e| < 2^22, e + (kShift - zp)
// rounds to the integer kShift + rint(e) - zp, whose float bits are
// kShiftBits + rint(e) - zp; it is clamped between kShift + the
// stored-code bounds (exact integers too) and the low byte of its bits is
// the stored code (no conversion, no zero-point subtraction).  Outside a rounding tie the sum
// rounds to the nearest integer exactly as rint does; the tie band sends
// ties to the exact division anyway.  Every element of a group has
// |x * rcp(s)| <= qmax + 1 < 2^22.
constexpr float kShift = 12582912.0f;  // 1.5 * 2^23

// Both groups' quantizer parameters held in VGPRs, so that an element's
// set costs one select per parameter (the empty asm keeps the compiler
// from re-deriving them per element).
struct QPair {
  float rs0, rs1, mz0, mz1;  // reciprocal scale; kShift - zp
  float lb0, lb1, hb0, hb1;  // kShift + stored-code bounds
  float s0, s1, zp0, zp1;
};

__device__ __forceinline__ QPair qpair(const QElem& a, const QElem& b) {
  QPair p{a.rs, b.rs, kShift - a.zp, kShift - b.zp, kShift + a.lo, kShift + b.lo,
          kShift + a.hi, kShift + b.hi, a.s, b.s, a.zp, b.zp};
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(p.rs0), "+v"(p.rs1), "+v"(p.mz0), "+v"(p.mz1), "+v"(p.lb0), "+v"(p.lb1),
               "+v"(p.hb0), "+v"(p.hb1));
#endif
  return p;
}

// Stored code of x (low byte of the result), and whether x/s lies in the
// tie band (then the caller takes the exact division).
__device__ __forceinline__ int qshift(float x, float rs, float mz, float lb, float hb, bool& near) {
  const float e = x * rs;
  const float t = e + mz;
  near = !(fabsf(fabsf(e - (t - mz)) - 0.5f) > kTieBand);
  return __float_as_int(__builtin_amdgcn_fmed3f(t, lb, hb));
}

// Stored codes of four elements whose groups are h (true: group 1) into
// row[p.*] (same codes as qstore4).
__device__ __forceinline__ void qstore4g(const float4& v, const bool (&h)[4], const QPair& q,
                                         uint8_t* row, int4 p) {
  const float xs[4] = {v.x, v.y, v.z, v.w};
  int c[4];
  bool n[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    c[e] = qshift(xs[e], h[e] ? q.rs1 : q.rs0, h[e] ? q.mz1 : q.mz0, h[e] ? q.lb1 : q.lb0,
                  h[e] ? q.hb1 : q.hb0, n[e]);
  if (n[0] | n[1] | n[2] | n[3]) [[unlikely]] {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (n[e])
        c[e] = qexact(xs[e], (h[e] ? q.lb1 : q.lb0) - kShift, (h[e] ? q.hb1 : q.hb0) - kShift,
                      h[e] ? q.zp1 : q.zp0, h[e] ? q.s1 : q.s0);
  }
  row[p.x] = (uint8_t)c[0];
  row[p.y] = (uint8_t)c[1];
  row[p.z] = (uint8_t)c[2];
  row[p.w] = (uint8_t)c[3];
}

// Codes without the zero point, for the single pass: a group's zero point
// (0 or 2^(c-1) there, c >= 2) is applied as an XOR of each code byte when
// its units are packed.  Unsigned codes lie in [0, hi], signed ones in
// [-hi, hi]; the single pass never has a sign (1-bit) group.
//
// The shortcut: t = fma(x, rcp(s), kShift) rounds the exact product
// x * rcp(s) to the nearest integer n, held as kShift + n, and the low
// byte of t's bits is the code (clamped below at kShift, i.e. code 0, when
// unsigned).  No upper clamp is needed: |x| is at most the group's
// maximum m, s = m / hi rounded, and rcp(s) is within an ulp, so
// |x * rcp(s)| <= hi * (1 + 2^-22) < hi + 1/2.  The product differs from
// x/s by at most 2^-15 (|x/s| <= 256); its residue d = x * rcp(s) - n
// (|d| <= 1/2, one more fma) is checked for the four elements together:
// any one within kTieBand of a tie sends that element to the exact
// division.
template <bool SIGNED>
__device__ __forceinline__ void qcodes4(const float4& v, int4 p, int kp0, float rs0, float rs1,
                                        float s0, float s1, float hi0, float hi1, uint8_t* row) {
  const float xs[4] = {v.x, v.y, v.z, v.w};
  const int pp[4] = {p.x, p.y, p.z, p.w};
  int c[4];
  float d[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float rs = pp[e] >= kp0 ? rs1 : rs0;
    const float t = __builtin_fmaf(xs[e], rs, kShift);
    c[e] = __float_as_int(SIGNED ? t : fmaxf(t, kShift));
    d[e] = __builtin_fmaf(xs[e], rs, kShift - t);
  }
  const float dm = fmaxf(fmaxf(fabsf(d[0]), fabsf(d[1])), fmaxf(fabsf(d[2]), fabsf(d[3])));
  if (dm >= 0.5f - kTieBand) [[unlikely]] {
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (fabsf(d[e]) >= 0.5f - kTieBand) {
        const bool g1 = pp[e] >= kp0;
        const float hi = g1 ? hi1 : hi0;
        c[e] = qexact(xs[e], SIGNED ? -hi : 0.0f, hi, 0.0f, g1 ? s1 : s0);
      }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) row[pp[e]] = (uint8_t)c[e];
}

// The same codes by exact division alone (a scale outside the shortcut's
// range).
__device__ __forceinline__ void qcodes4_exact(const float4& v, int4 p, int kp0, float s0, float s1,
                                              float lo0, float lo1, float hi0, float hi1,
                                              uint8_t* row) {
  const float xs[4] = {v.x, v.y, v.z, v.w};
  const int pp[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bool g1 = pp[e] >= kp0;
    row[pp[e]] = (uint8_t)qexact(xs[e], g1 ? lo1 : lo0, g1 ? hi1 : hi0, 0.0f, g1 ? s1 : s0);
  }
}

// The shortcut codes of qcodes4 with sub-group scales: element e's block
// (bits 16.. of its table entry) selects its reciprocal from rtab (0 for a
// scale outside the shortcut's range, which sends the element to the exact
// division like a tie); hi per precision group (blocks >= nsub0 are group
// 1's).  The block maximum bounds |x|, so the shortcut needs no upper
// clamp, as in qcodes4.
template <bool SIGNED>
__device__ __forceinline__ void qcodes4g(const float4& v, int4 p, const float* stab,
                                         const float* rtab, int nsub0, float hi0, float hi1,
                                         uint8_t* row) {
  const float xs[4] = {v.x, v.y, v.z, v.w};
  const int pp[4] = {p.x, p.y, p.z, p.w};
  int c[4];
  float d[4];
  bool slow = false;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float rs = rtab[pp[e] >> 16];
    const float t = __builtin_fmaf(xs[e], rs, kShift);
    c[e] = __float_as_int(SIGNED ? t : fmaxf(t, kShift));
    d[e] = __builtin_fmaf(xs[e], rs, kShift - t);
    slow |= rs == 0.0f;
  }
  const float dm = fmaxf(fmaxf(fabsf(d[0]), fabsf(d[1])), fmaxf(fabsf(d[2]), fabsf(d[3])));
  if (slow || dm >= 0.5f - kTieBand) [[unlikely]] {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int b = pp[e] >> 16;
      if (rtab[b] == 0.0f || fabsf(d[e]) >= 0.5f - kTieBand) {
        const float hi = b >= nsub0 ? hi1 : hi0;
        c[e] = qexact(xs[e], SIGNED ? -hi : 0.0f, hi, 0.0f, stab[b]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) row[pp[e] & 0xFFFF] = (uint8_t)c[e];
}

// Waves per SIMD the register budget must allow: T <= 9 keeps seven
// workgroups per CU resident (1568 four-row workgroups on 256 CUs), more
// float4 per thread four.  TL of the T float4 per thread wait in LDS.
// GRP: sub-group scales (the planned-position table carries each
// element's block in bits 16..; block maxima, scales and reciprocals sit in
// LDS after the row slots: 3*nsub words).
template <int T, int TL, bool GRP = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(T <= 9 ? 7 : 4)))
void k_act_coop(const float* __restrict__ A, int64_t M, int K4, int64_t lda, int RB,
                const int32_t* __restrict__ pos, ActPlan ap, unsigned* __restrict__ st,
                unsigned spins, float* __restrict__ s_a_out, uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  __shared__ float gmax[2];
  __shared__ int flag;
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blockIdx.x * RB;
  const int rows = (int)min((int64_t)RB, M - m0);
  const int nf = RB * K4;  // flat positions of this workgroup (T*256 >= nf)
  // uniform: kept in SGPRs (the division runs on the vector unit)
  const int q256 = __builtin_amdgcn_readfirstlane(256 / K4);
  const int r256 = 256 - q256 * K4;
  const int kp0 = ap.kpad[0];  // planned positions >= kp0 belong to group 1
  // The generation word first (thread 0 of wave 0): its wait then rides on
  // the table's, long before the maxima are folded.
  unsigned gen = 0;
  if (tid == 0) gen = bar_load(grid_gen_word(st));
  const float* A0 = A + m0 * lda;
  int4* pos4 = reinterpret_cast<int4*>(codes + RB * ap.Kp);
  // The position table goes global -> LDS directly (no registers), ahead
  // of the row loads: entry k of wave wid's chunk j (k = 256j + 64wid +
  // lane) lands at pos4[k]; lanes past K4 read zeros into the padding of
  // the table's region (K4 rounded up to 64 entries).  RB >= 4 gives
  // K4 <= 64*T <= 256*TJ.
  constexpr int TJ = (T + 3) / 4;
  {
    const __amdgpu_buffer_rsrc_t pr =
        __builtin_amdgcn_make_buffer_rsrc((void*)pos, (short)0, K4 * 16, 0x00020000);
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t base = lds_off(codes) + (uint32_t)(RB * ap.Kp);
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int k0 = 256 * j + 64 * wid;
      const int k = k0 + (tid & 63);
      if (k0 < K4)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            pr, (__attribute__((address_space(3))) void*)(uintptr_t)(base + 16 * k0), 16,
            k < K4 ? 16u * k : kOOB, 0, 0, 0);
    }
    asm volatile("" ::: "memory");
  }
  // The first TL slots go global -> LDS (lane l of wave w: vlds + i*4096 +
  // (64w + l)*16) where the register budget cannot hold them, slots
  // i >= TL to registers.  Issued first, the LDS slots are what the first
  // LDS read after the barrier waits for (any LDS read waits for the
  // direct loads before it), and slot 0 is the first one the maxima need.
  constexpr int TV = T - TL;
  float4 v[TV];
  float4* vlds = reinterpret_cast<float4*>(codes + RB * ap.Kp + 16 * ((K4 + 63) / 64 * 64));
  {
    // rows through a buffer resource based at row m0: 32-bit offsets
    const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
        (void*)A0, (short)0, (int)(((int64_t)(rows - 1) * lda + 4 * K4) * 4), 0x00020000);
    const uint32_t ld4 = (uint32_t)lda * 4u;
    const uint32_t vb = lds_off(reinterpret_cast<uint8_t*>(vlds)) +
                        (uint32_t)__builtin_amdgcn_readfirstlane(tid >> 6) * 1024u;
    int r, k;
    coop_first(r, k, K4);
#pragma unroll
    for (int i = 0; i < T; ++i) {
      // positions past nf re-read this workgroup's last element
      const bool in = tid + 256 * i < nf;
      const int rc = in ? min(r, rows - 1) : rows - 1;
      const int kc = in ? k : K4 - 1;
      const uint32_t off = (uint32_t)rc * ld4 + 16u * (uint32_t)kc;
      if (i >= TL)
        v[i >= TL ? i - TL : 0] =
            __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(ar, off, 0, 0));
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            ar, (__attribute__((address_space(3))) void*)(uintptr_t)(vb + i * 4096), 16, off, 0, 0,
            0);
      coop_step(r, k, K4, q256, r256);
    }
  }
  // Codes start as each group's zero point, which packs to a stored zero
  // (the padding channels and rows no element writes).
  {
    uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
    const int kw = ap.Kp / 4, kw0 = kp0 / 4;
    const uint32_t z0 = 0x01010101u * (uint32_t)ap.zp[0], z1 = 0x01010101u * (uint32_t)ap.zp[1];
    for (int r = 0; r < RB; ++r)
      for (int i = tid; i < kw; i += 256) codes32[r * kw + i] = i < kw0 ? z0 : z1;
  }
  const int nsub = GRP ? ap.nsub[0] + (ap.S == 2 ? ap.nsub[1] : 0) : 0;
  unsigned* bmax = reinterpret_cast<unsigned*>(vlds + TL * 256);
  float* stab = reinterpret_cast<float*>(bmax + nsub);
  float* rtab = stab + nsub;
  if constexpr (GRP)
    for (int j = tid; j < nsub; j += 256) bmax[j] = 0u;
  // This wave's generation read and table chunks (issued before the T row
  // loads) have landed; a barrier without a fence, so the row loads stay
  // in flight and the maxima below fold each slot as it arrives.
  wait_vm<T>();
  bar_nofence();
  // slot i's float4 (the LDS ones are read where they are used)
  auto val = [&](int i) __attribute__((always_inline)) {
    return i < TL ? vlds[i * 256 + tid] : v[i >= TL ? i - TL : 0];
  };
  float mx0 = 0.0f, mx1 = 0.0f;
  {
    int r, k;
    coop_first(r, k, K4);
#pragma unroll
    for (int i = 0; i < T; ++i) {
      if (i == 0 && TL > 0) lds_dma_wait<TV>();  // the LDS slots, issued before the TV others
      const int4 p = pos4[tid + 256 * i < nf ? k : K4 - 1];
      if constexpr (GRP) {
        // each element's |x| into its block's word; one atomic when the
        // four share a block (the usual case)
        const float4 x = val(i);
        const float a0 = fabsf(x.x), a1 = fabsf(x.y), a2 = fabsf(x.z), a3 = fabsf(x.w);
        const int b0 = p.x >> 16, b1 = p.y >> 16, b2 = p.z >> 16, b3 = p.w >> 16;
        if (b0 == b1 && b0 == b2 && b0 == b3) {
          atomicMax(&bmax[b0], __float_as_uint(fmaxf(fmaxf(a0, a1), fmaxf(a2, a3))));
        } else {
          atomicMax(&bmax[b0], __float_as_uint(a0));
          atomicMax(&bmax[b1], __float_as_uint(a1));
          atomicMax(&bmax[b2], __float_as_uint(a2));
          atomicMax(&bmax[b3], __float_as_uint(a3));
        }
      } else {
        max4(val(i), make_uchar4(p.x >= kp0, p.y >= kp0, p.z >= kp0, p.w >= kp0), mx0, mx1);
      }
      coop_step(r, k, K4, q256, r256);
    }
  }
  if constexpr (GRP) {
    __syncthreads();
    if (tid < 64) {
      const bool ok = grid_fold_max_n(st, gen, spins, bmax, nsub);
      if (tid == 0) flag = ok;
    }
    __syncthreads();
    if (!flag && tid == 0) bar_add(st + kActStallWord, 1u);
    if (!flag) absmax_all_blocks(A, M, K4, lda, pos4, bmax, nsub);
    for (int j = tid; j < nsub; j += 256) {
      const float sc = group_scale(__uint_as_float(bmax[j]), j < ap.nsub[0] ? ap.q[0] : ap.q[1]);
      stab[j] = sc;
      rtab[j] = fast_ok(sc) ? __builtin_amdgcn_rcpf(sc) : 0.0f;
      if (blockIdx.x == 0) s_a_out[j] = sc;
    }
    __syncthreads();
  } else {
    const float2 m = block_max2(make_float2(mx0, mx1), red);
    if (tid == 0) {
      float g0, g1;
      flag = grid_fold_max(st, gen, spins, m.x, m.y, g0, g1);
      gmax[0] = g0;
      gmax[1] = g1;
      if (!flag) bar_add(st + kActStallWord, 1u);
    }
    __syncthreads();
  }
  float g0 = gmax[0], g1 = gmax[1];
  if (!GRP && !flag) absmax_all(A, M, K4, lda, pos4, kp0, red, g0, g1);
  const float s0 = group_scale(g0, ap.q[0]);
  const float s1 = ap.S == 2 ? group_scale(g1, ap.q[1]) : 0.0f;
  if (!GRP && blockIdx.x == 0 && tid == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
  {
    const float hi0 = (float)ap.q[0].hi, hi1 = (float)ap.q[1].hi;
    const float lo0 = (float)ap.q[0].lo, lo1 = (float)ap.q[1].lo;
    const bool fast = GRP || (fast_ok(s0) && (ap.S == 1 || fast_ok(s1)));
    float rs0 = fast ? __builtin_amdgcn_rcpf(s0) : 0.0f;
    float rs1 = fast && ap.S == 2 ? __builtin_amdgcn_rcpf(s1) : 0.0f;
    auto each = [&](auto&& f) __attribute__((always_inline)) {
      int r, k;
      coop_first(r, k, K4);
      int ro = r * ap.Kp;  // row r's codes; the row is stepped through ro alone
      const int qk = __builtin_amdgcn_readfirstlane(q256 * ap.Kp);
      const int lim = __builtin_amdgcn_readfirstlane(rows * ap.Kp);
#pragma unroll
      for (int i = 0; i < T; ++i) {
        if (tid + 256 * i < nf && ro < lim) f(val(i), pos4[k], codes + ro);
        k += r256;
        ro += qk;
        if (k >= K4) {
          k -= K4;
          ro += ap.Kp;
        }
      }
    };
    if constexpr (GRP) {
      if (ap.q[0].lo < 0)
        each([&](const float4& x, int4 p, uint8_t* row) __attribute__((always_inline)) {
          qcodes4g<true>(x, p, stab, rtab, ap.nsub[0], hi0, hi1, row);
        });
      else
        each([&](const float4& x, int4 p, uint8_t* row) __attribute__((always_inline)) {
          qcodes4g<false>(x, p, stab, rtab, ap.nsub[0], hi0, hi1, row);
        });
    } else if (!fast) {
      each([&](const float4& x, int4 p, uint8_t* row) __attribute__((always_inline)) {
        qcodes4_exact(x, p, kp0, s0, s1, lo0, lo1, hi0, hi1, row);
      });
    } else if (ap.q[0].lo < 0) {
      each([&](const float4& x, int4 p, uint8_t* row) __attribute__((always_inline)) {
        qcodes4<true>(x, p, kp0, rs0, rs1, s0, s1, hi0, hi1, row);
      });
    } else {
      each([&](const float4& x, int4 p, uint8_t* row) __attribute__((always_inline)) {
        qcodes4<false>(x, p, kp0, rs0, rs1, s0, s1, hi0, hi1, row);
      });
    }
  }
  __syncthreads();
  const int r0 = (int)(m0 % kBlk);
  for (int gi = 0; gi < ap.S; ++gi) {
    const int c = gi ? ap.c[1] : ap.c[0];
    const int ng = gi ? ap.ng[1] : ap.ng[0];
    const int gbase = gi ? ap.kpad[0] : 0;
    uint8_t* dst = packed + (gi ? ap.seg_off[1] : ap.seg_off[0]) +
                   (m0 / kBlk) * (gi ? ap.mblk_bytes[1] : ap.mblk_bytes[0]);
    const uint32_t zx = 0x01010101u * (uint32_t)(gi ? ap.zp[1] : ap.zp[0]);
#define SONIQ_PIECES(RB_)                                                             \
  if (c == 8) write_block_pieces<8, RB_>(codes, ap.Kp, gbase, ng, r0, dst, zx);        \
  else if (c == 4) write_block_pieces<4, RB_>(codes, ap.Kp, gbase, ng, r0, dst, zx);   \
  else write_block_pieces<2, RB_>(codes, ap.Kp, gbase, ng, r0, dst, zx)
    if (RB == 4) { SONIQ_PIECES(4); }
    else if (RB == 8) { SONIQ_PIECES(8); }
    else { SONIQ_PIECES(16); }
#undef SONIQ_PIECES
  }
}

// ----------------------------------------------------------- k_act_small --
// Small batches (M <= 64, M*K <= kSmallElems, contiguous aligned rows): one
// launch.  Every workgroup reduces the group maxima of the whole batch
// itself (at most 256 KB, L2-resident after the first pass), then
// quantizes and packs its own row.  Dynamic LDS: Kp bytes.
constexpr int kSmallElems = 65536;
constexpr int kSmallU = 4;

__global__ __launch_bounds__(256) void k_act_small(const float* __restrict__ A, int M, int K,
                                                   int64_t lda, const int32_t* __restrict__ pos,
                                                   const uint8_t* __restrict__ seg, ActPlan ap,
                                                   float* __restrict__ s_a_out,
                                                   uint8_t* __restrict__ packed,
                                                   uint8_t* __restrict__ ximg) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int tid = threadIdx.x;
  const int K4 = K / 4;
  const int total4 = M * K4;
  float mx0 = 0.0f, mx1 = 0.0f;
  for (int base = tid; base < total4; base += 256 * kSmallU) {
    float4 v[kSmallU];
    uchar4 g[kSmallU];
#pragma unroll
    for (int j = 0; j < kSmallU; ++j) {
      const int i = min(base + 256 * j, total4 - 1);  // repeats change no max
      const int m = i / K4, k4 = i - m * K4;
      v[j] = *reinterpret_cast<const float4*>(A + (int64_t)m * lda + 4 * k4);
      g[j] = reinterpret_cast<const uchar4*>(seg)[k4];
    }
#pragma unroll
    for (int j = 0; j < kSmallU; ++j) max4(v[j], g[j], mx0, mx1);
  }
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < ap.Kp / 4; i += 256) codes32[i] = 0;
  mx0 = block_max(mx0, red);
  mx1 = block_max(mx1, red);
  const float s0 = group_scale(mx0, ap.q[0]);
  const float s1 = ap.S == 2 ? group_scale(mx1, ap.q[1]) : 0.0f;
  if (blockIdx.x == 0 && tid == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
  const ActQ aq = make_actq(ap, s0, s1);
  const int m = blockIdx.x;
  const float* row = A + (int64_t)m * lda;
  for (int base = tid; base < K4; base += 256 * kSmallU) {
    float4 v[kSmallU];
    int4 p[kSmallU];
    uchar4 g[kSmallU];
#pragma unroll
    for (int j = 0; j < kSmallU; ++j) {
      const int k4 = min(base + 256 * j, K4 - 1);
      v[j] = reinterpret_cast<const float4*>(row)[k4];
      p[j] = reinterpret_cast<const int4*>(pos)[k4];
      g[j] = reinterpret_cast<const uchar4*>(seg)[k4];
    }
#pragma unroll
    for (int j = 0; j < kSmallU; ++j) {
      if (base + 256 * j < K4) {
        codes[p[j].x] = store_code(v[j].x, g[j].x, aq);
        codes[p[j].y] = store_code(v[j].y, g[j].y, aq);
        codes[p[j].z] = store_code(v[j].z, g[j].z, aq);
        codes[p[j].w] = store_code(v[j].w, g[j].w, aq);
      }
    }
  }
  __syncthreads();
  write_act_units(codes, 1, m, ap, packed, ximg);
}

// ------------------------------------------------------------ k_act_row1 --
// Batches of at most MT rows (decode steps), aligned, no sign-code group:
// workgroup m loads every row of the batch and the planned positions once
// (thread tid owns float4 positions tid + 256*j, j < J, of every row),
// reduces the group maxima of the batch from registers, then quantizes
// its own row m (group 1 starts at planned position kpad[0]) into LDS and
// writes the row's units.  One HBM round trip instead of two; every
// workgroup computes the same maxima from the same data.
// Dynamic LDS: Kp bytes.
template <int J, int MT>
__global__ __launch_bounds__(256) void k_act_row1(const float* __restrict__ A, int M, int K4,
                                                  int64_t lda, const int32_t* __restrict__ pos,
                                                  ActPlan ap, float* __restrict__ s_a_out,
                                                  uint8_t* __restrict__ packed,
                                                  uint8_t* __restrict__ ximg) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int tid = threadIdx.x;
  const int m = blockIdx.x;
  const int kp0 = ap.kpad[0];
  float4 v[MT][J];
  int4 p[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int k4 = min(tid + 256 * j, K4 - 1);  // repeats change no max
    p[j] = reinterpret_cast<const int4*>(pos)[k4];
#pragma unroll
    for (int r = 0; r < MT; ++r)
      v[r][j] = reinterpret_cast<const float4*>(A + (int64_t)min(r, M - 1) * lda)[k4];
  }
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < ap.Kp / 4; i += 256) codes32[i] = 0;
  float mx0 = 0.0f, mx1 = 0.0f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const uchar4 g = make_uchar4(p[j].x >= kp0, p[j].y >= kp0, p[j].z >= kp0, p[j].w >= kp0);
#pragma unroll
    for (int r = 0; r < MT; ++r) max4(v[r][j], g, mx0, mx1);
  }
  const float2 mm = block_max2(make_float2(mx0, mx1), red);  // syncs
  const float s0 = group_scale(mm.x, ap.q[0]);
  const float s1 = ap.S == 2 ? group_scale(mm.y, ap.q[1]) : 0.0f;
  if (m == 0 && tid == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
  const QPair q = qpair(qelem(s0, ap.q[0], ap.zp[0]), qelem(s1, ap.q[1], ap.zp[1]));
#pragma unroll
  for (int j = 0; j < J; ++j)
    if (tid + 256 * j < K4) {
      const bool h[4] = {p[j].x >= kp0, p[j].y >= kp0, p[j].z >= kp0, p[j].w >= kp0};
      float4 x = v[0][j];
#pragma unroll
      for (int r = 1; r < MT; ++r)
        if (r == m) x = v[r][j];
      qstore4g(x, h, q, codes, p[j]);
    }
  __syncthreads();
  write_act_units(codes, 1, m, ap, packed, ximg);
}

// ------------------------------------------------------------ GEMM/GEMV --
// Quantizer of the next layer's activation groups with static scales.
struct QNext {
  float s[2], rs[2];  // scale; its reciprocal, or 0 where the exact division decides
  float lo[2], hi[2];
  int zp[2], sign1[2];
};

// The quantizer of one output column (its next-layer group's), selected
// once per column; codes by the reciprocal shortcut, with `near` set where
// the exact division must decide (near a tie, or a scale outside the
// shortcut's range).
struct QCol {
  float sc, rs, lo, hi;
  int zp;
  bool sign1;
};

__device__ __forceinline__ QCol qnext_col(int g, const QNext& q) {
  QCol c;
  c.sc = g ? q.s[1] : q.s[0];
  c.rs = g ? q.rs[1] : q.rs[0];
  c.lo = g ? q.lo[1] : q.lo[0];
  c.hi = g ? q.hi[1] : q.hi[0];
  c.zp = g ? q.zp[1] : q.zp[0];
  c.sign1 = (g ? q.sign1[1] : q.sign1[0]) != 0;
  return c;
}

// rs is the correctly rounded reciprocal (0 outside [2^-100, 2^100]), so
// y * rs lies within 2^-22.4 |y/s| of the exact quotient: kTieBand's
// argument holds wherever the code is not clamped (|y/s| <= 256), and
// beyond that both quotients clamp to the same bound.
__device__ __forceinline__ int qnext_fast(float y, const QCol& c, bool& near) {
  const float e = y * c.rs;
  const float t = __builtin_rintf(e);
  const bool plain = !c.sign1 && c.sc != 0.0f;
  near = plain && (c.rs == 0.0f || !(fabsf(fabsf(e - t) - 0.5f) > kTieBand));
  const int code = c.sign1 ? (y < 0.0f ? -1 : 1)
                           : plain ? (int)__builtin_amdgcn_fmed3f(t, c.lo, c.hi) : 0;
  return code - c.zp;
}

__device__ __forceinline__ int qnext_exact(float y, const QCol& c) {
  const float t = __builtin_rintf(__fdiv_rn(y, c.sc));
  return (int)__builtin_amdgcn_fmed3f(t, c.lo, c.hi) - c.zp;
}

// Stored codes of four outputs of one column as the bytes of a word (byte
// h: output h), by the shifted form of the quantizer (as qshift): y*rs +
// (kShift - zp) rounds to kShift + rint(y*rs) - zp, clamped between
// kShift + the stored-code bounds, whose low byte is the stored code.
// Outputs within the tie band (or all, for a scale outside the shortcut's
// range) take the exact division; the branch is taken by the wave.
__device__ __forceinline__ uint32_t qnext4(const float (&y)[4], const QCol& c) {
  const bool plain = !c.sign1 && c.sc != 0.0f;
  const float zf = (float)c.zp;
  const float mz = kShift - zf, lb = kShift + (c.lo - zf), hb = kShift + (c.hi - zf);
  uint32_t b[4];
  bool nr[4];
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const float e = y[h] * c.rs;
    const float t = e + mz;
    nr[h] = plain && (c.rs == 0.0f || !(fabsf(e - (t - mz)) < 0.5f - kTieBand));
    b[h] = __float_as_uint(__builtin_amdgcn_fmed3f(t, lb, hb));
    if (c.sign1) b[h] = (uint32_t)((y[h] < 0.0f ? -1 : 1) - c.zp);
  }
  uint32_t w = __builtin_amdgcn_perm(b[1], b[0], 0x0C0C0400u) |
               __builtin_amdgcn_perm(b[3], b[2], 0x04000C0Cu);
  if (__builtin_amdgcn_ballot_w64(nr[0] || nr[1] || nr[2] || nr[3]) != 0) [[unlikely]] {
#pragma unroll
    for (int h = 0; h < 4; ++h)
      if (nr[h])
        w = (w & ~(0xFFu << (8 * h))) | (((uint32_t)qnext_exact(y[h], c) & 0xFFu) << (8 * h));
  }
  return w;
}

struct GemmArgs {
  const uint8_t* act;
  const float* s_a;
  ActPlan ap;
  WDev wd;
  WPlan wp;
  int64_t M, N;
  uint16_t* Y;
  int64_t ldy;
  int32_t* acc;
  int xcd_tiles;  // GEMM: give each XCD a contiguous range of tiles
  // the dense weight copy (k_gemv_dense) and its two widths
  const uint8_t* dense;
  int db_lo, db_hi;
  // fused batch-1 path (k_gemv_fused): the fp32 row, its planned
  // positions, where the handle's scales and packed row go, the row's
  // length in float4 and the staging bytes ahead of the code row in LDS
  const float* a32;
  const uint16_t* apos16;  // planned positions, 16 bits each
  float* s_a_out;
  uint8_t* act_out;
  int K4, xs_bytes;
  // batch-1 GEMV: the activation row's contiguous image (null: stage the
  // row from the units); the fused form writes it
  uint8_t* ximg;
  // quantization of the outputs for the next layer (k_gemm<..., true>):
  // the next layer's stored codes as bytes; from the GEMM tiles in 16-row
  // blocks of 16-byte columns, row m and position p at
  // qn_img[(m/16)*qn_ld + 16*p + m%16] (qn_ld = 16 * the next plan's Kp),
  // from the GEMV forms row-major at qn_img[m*qn_ld + p] (qn_ld = Kp);
  // qn_tab[physical column] = the next-layer group of its channel, and
  // qn_tab[Np + 128*tile + r] = the next-layer position of the tile's r-th
  // column in ascending original order (-1 past the last); the quantizer
  // of each next-layer group with its static scale
  uint8_t* qn_img;
  const int32_t* qn_tab;
  int64_t qn_ld;
  // QN = 3 (batch maximum): per next-layer group the largest |Y| the tile
  // stores, as pair qn_max[2*tile], qn_max[2*tile + 1]
  float* qn_max;
  QNext qn;
  // a next layer with sub-group scales: qn_tab holds each column's block,
  // whose static scale and reciprocal are qn_bs[b], qn_brs[b] (blocks
  // >= qn_nsub0 belong to its group 1); null otherwise
  const float* qn_bs;
  const float* qn_brs;
  int qn_nsub0;
  // MFMA-native copies of the narrow operands (null: none), and their plan
  const uint8_t* fa;
  const uint8_t* fw;
  FPlan fp;
  // implicit 3x3 convolution: the input's haloed code image and geometry
  const uint8_t* img;
  ConvGeo cg;
};

// 16 bytes per lane, global -> LDS; lane l lands at lds_dst + 16*l.
__device__ __forceinline__ void load_lds16(const uint8_t* src, uint8_t* lds_dst_uniform) {
  __builtin_amdgcn_global_load_lds(
      reinterpret_cast<const void*>(src),
      reinterpret_cast<__attribute__((address_space(3))) void*>(
          reinterpret_cast<uintptr_t>(lds_dst_uniform)),
      16, 0, 0);
}

template <int C>
__device__ __forceinline__ v4i read_frag(const uint8_t* p, int lane) {
  uint4 raw;
  if constexpr (C == 8) {
    raw = *reinterpret_cast<const uint4*>(p + lane * 16);
  } else if constexpr (C == 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(p + lane * 8);
    raw = make_uint4(v.x, v.y, 0u, 0u);
  } else if constexpr (C == 2) {
    raw = make_uint4(*reinterpret_cast<const uint32_t*>(p + lane * 4), 0u, 0u, 0u);
  } else {
    raw = make_uint4(*reinterpret_cast<const uint16_t*>(p + lane * 2), 0u, 0u, 0u);
  }
  const uint4 d = unpack_unit<C>(raw);
  return v4i{(int)d.x, (int)d.y, (int)d.z, (int)d.w};
}

__device__ __forceinline__ v4i read_frag_rt(const uint8_t* p, int lane, int c) {
  if (c == 8) return read_frag<8>(p, lane);
  if (c == 4) return read_frag<4>(p, lane);
  if (c == 2) return read_frag<2>(p, lane);
  return read_frag<1>(p, lane);
}

template <int CA>
__device__ __forceinline__ v4i read_frag_a(const uint8_t* p, int lane, int c) {
  if constexpr (CA != 0) return read_frag<CA>(p, lane);
  else return read_frag_rt(p, lane, c);
}

// Weight-block fragment: the container is one of two per handle; CBL/CBH
// fix them at compile time (0 = decided at run time).
template <int CBL, int CBH>
__device__ __forceinline__ v4i read_frag_w(const uint8_t* p, int lane, int c) {
  if constexpr (CBL != 0 && CBL == CBH) {
    return read_frag<CBL>(p, lane);
  } else if constexpr (CBL != 0 && CBH != 0) {
    if (c == CBL) return read_frag<CBL>(p, lane);
    return read_frag<CBH>(p, lane);
  } else {
    return read_frag_rt(p, lane, c);
  }
}

constexpr int kBSlot = 128 * 16 * 8;  // B stage bytes at c = 8 (8 blocks, 2 granules)
constexpr int kLB = 4;                // B loads per stage (kBSlot / 4 KB)

// Ring slot of a (32*WFM) x 128 tile: the A stage at the larger activation
// container, then the B stage at the larger weight container (8-bit where
// the containers are only known at run time).
constexpr int gemm_aslot(int S, int CA0, int CA1, int CBL, int CBH, int WFM) {
  return (CA0 == 0 || (S == 2 && CA1 == 0) || CBL == 0 || CBH == 0)
             ? 32 * WFM * 16 * 8
             : 32 * WFM * 16 * (S == 2 && CA1 > CA0 ? CA1 : CA0);
}
constexpr int gemm_slot(int S, int CA0, int CA1, int CBL, int CBH, int WFM) {
  return gemm_aslot(S, CA0, CA1, CBL, CBH, WFM) +
         ((CA0 == 0 || (S == 2 && CA1 == 0) || CBL == 0 || CBH == 0)
              ? kBSlot
              : 128 * 16 * (CBH > CBL ? CBH : CBL));
}

// Fragment reads from the LDS ring are issued as inline asm.  The ring is
// filled by direct global->LDS loads whose completion each wave awaits with
// an explicit vmcnt wait and a barrier; through plain C++ loads the
// compiler cannot tell the ring slots apart and drains every in-flight
// load (vmcnt(0)) before each read, which serializes the pipeline.
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));


// Packed unit (2*C bytes) at LDS byte address a + OFF, in a register type
// of its size.
template <int C>
struct RawT { using type = uint32_t; };
template <>
struct RawT<4> { using type = u32x2v; };
template <>
struct RawT<8> { using type = u32x4v; };
template <int C>
using raw_t = typename RawT<C>::type;

template <int C, int OFF>
__device__ __forceinline__ raw_t<C> lds_unit(uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
  raw_t<C> r{};
#if defined(__HIP_DEVICE_COMPILE__)  // GPU asm; the host pass never runs it
  if constexpr (C == 8) asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
  else if constexpr (C == 4) asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
  else if constexpr (C == 2) asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
  else asm volatile("ds_read_u16 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
#else
  (void)a;
#endif
  return r;
}

// Waits for every LDS read in flight; each fragment is then passed through
// an empty asm so that nothing using it can be scheduled above the wait.
__device__ __forceinline__ void lds_wait() {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#endif
}
// Waits until at most N LDS reads (or scalar loads) are in flight; LDS
// reads complete in order, so the earliest ones have landed.  A scalar
// load still in flight only makes the wait longer.
template <int N>
__device__ __forceinline__ void lds_wait_n() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
#endif
}
template <typename T>
__device__ __forceinline__ void lds_touch(T& r) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("" : "+v"(r));
#else
  (void)r;
#endif
}

__device__ __forceinline__ v4i frag_of(uint4 d) { return v4i{(int)d.x, (int)d.y, (int)d.z, (int)d.w}; }

template <int C>
__device__ __forceinline__ v4i unpack_frag(raw_t<C> r) {
  if constexpr (C == 8) return frag_of(make_uint4(r.x, r.y, r.z, r.w));
  else if constexpr (C == 4) return frag_of(unpack4(r.x, r.y));
  else if constexpr (C == 2) return frag_of(unpack2(r));
  else return frag_of(unpack1(r & 0xFFFFu));
}

template <int CA, int KK, int WFM, int... I>
__device__ __forceinline__ void read_a_units(raw_t<CA> (&ra)[WFM], uint32_t a,
                                             std::integer_sequence<int, I...>) {
  ((ra[I] = lds_unit<CA, (I * 2 + KK) * 128 * CA>(a)), ...);
}

// B fragment jj of a granule: the block's container is CBL or CBH.
template <int CBL, int CBH, int KK>
__device__ __forceinline__ v4i b_frag(uint32_t addr, int c, bool) {
  if constexpr (CBL == CBH) {
    raw_t<CBL> r = lds_unit<CBL, KK * 128 * CBL>(addr);
    lds_wait();
    lds_touch(r);
    return unpack_frag<CBL>(r);
  } else {
    if (c == CBL) {
      raw_t<CBL> r = lds_unit<CBL, KK * 128 * CBL>(addr);
      lds_wait();
      lds_touch(r);
      return unpack_frag<CBL>(r);
    }
    raw_t<CBH> r = lds_unit<CBH, KK * 128 * CBH>(addr);
    lds_wait();
    lds_touch(r);
    return unpack_frag<CBH>(r);
  }
}

// Granule KK of a stage for containers fixed at compile time: read and
// widen the wave's 4 B units, then read its WFM A units and per A fragment
// widen and issue its 4 MFMAs (two waits keep fewer raw units live).
template <int CA, int CBL, int CBH, int WFM, int KK>
__device__ __forceinline__ void mma_granule(v4i (&acc)[WFM][4], uint32_t a_addr,
                                            const uint32_t (&b_addr)[4], const int (&wcj)[4],
                                            bool) {
  v4i bf[4];
  if constexpr (CBL == CBH) {
    raw_t<CBL> rb[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) rb[jj] = lds_unit<CBL, KK * 128 * CBL>(b_addr[jj]);
    lds_wait();
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      lds_touch(rb[jj]);
      bf[jj] = unpack_frag<CBL>(rb[jj]);
    }
  } else {
    // the mixed-width tile: one wait per fragment (rare)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) bf[jj] = b_frag<CBL, CBH, KK>(b_addr[jj], wcj[jj], false);
  }
  raw_t<CA> ra[WFM];
  read_a_units<CA, KK>(ra, a_addr, std::make_integer_sequence<int, WFM>{});
  lds_wait();
#pragma unroll
  for (int i = 0; i < WFM; ++i) {
    lds_touch(ra[i]);
    const v4i af = unpack_frag<CA>(ra[i]);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf[jj], acc[i][jj], 0, 0, 0);
  }
}

// The hook run after each granule's products, given the accumulators and
// the granule's index in its group (see k_gemm_g); the plain GEMM passes
// this one, which does nothing.
struct NoGranuleHook {
  template <class T>
  __device__ __forceinline__ void operator()(T&, int) const {}
};

// Both granules of a stage on a tile of one weight width CB: every unit
// read of the stage is issued first; granule 0 is widened and multiplied
// once its reads have landed (the 4 + WFM reads of granule 1 may still be
// in flight), then granule 1.  q0: index of granule 0 for the hook.
template <int CA, int CB, int WFM, class Hook = NoGranuleHook>
__device__ __forceinline__ void mma_stage(v4i (&acc)[WFM][4], uint32_t a_addr,
                                          const uint32_t (&b_addr)[4], Hook&& hook = Hook{},
                                          int q0 = 0) {
  raw_t<CB> rb0[4], rb1[4];
  raw_t<CA> ra0[WFM], ra1[WFM];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) rb0[jj] = lds_unit<CB, 0>(b_addr[jj]);
  read_a_units<CA, 0>(ra0, a_addr, std::make_integer_sequence<int, WFM>{});
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) rb1[jj] = lds_unit<CB, 128 * CB>(b_addr[jj]);
  read_a_units<CA, 1>(ra1, a_addr, std::make_integer_sequence<int, WFM>{});
  auto granule = [&](raw_t<CB> (&rb)[4], raw_t<CA> (&ra)[WFM]) __attribute__((always_inline)) {
    v4i bf[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      lds_touch(rb[jj]);
      bf[jj] = unpack_frag<CB>(rb[jj]);
    }
#pragma unroll
    for (int i = 0; i < WFM; ++i) {
      lds_touch(ra[i]);
      const v4i af = unpack_frag<CA>(ra[i]);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf[jj], acc[i][jj], 0, 0, 0);
    }
  };
  lds_wait_n<4 + WFM>();
  granule(rb0, ra0);
  hook(acc, q0);
#if defined(__HIP_DEVICE_COMPILE__)
  // keep granule 0's products ahead of the wait (MFMAs are not memory
  // operations, so the wait's memory clobber alone does not order them)
  __builtin_amdgcn_sched_barrier(0);
#endif
  lds_wait();
  granule(rb1, ra1);
  hook(acc, q0 + 1);
}

// One activation group's K loop for containers fixed at compile time (A in
// CA, the tile's weight blocks in CBL or CBH; CBL == CBH for tiles of one
// width).  Tile BM x 128 (BM = 32*WFM), waves 2x2, wave tile (16*WFM) x 64,
// NST-deep LDS ring, stage = 2 granules, same LDS stage layout as the
// generic loop.  Loads go through buffer resources: each lane's offsets are
// fixed for the group and a scalar stage offset advances them (per lane on
// the mixed-width tile); chunks past the data read as zero, which also
// zeroes the second granule of a final half stage, so its products vanish.
template <int CA, int CBL, int CBH, int WFM, int NST, int ASLOT, int SLOT,
          class Hook = NoGranuleHook>
__device__ __forceinline__ void gemm_group_fast(uint8_t* lds, const uint8_t* abase,
                                                int64_t mstride, int ng, const uint8_t* wtile,
                                                int wbytes, int ngt, const int (&bc)[8],
                                                const int (&bpre)[9], int qbase,
                                                v4i (&acc)[WFM][4], int tid, int lane, int wid,
                                                int wm, int wn, Hook&& hook = Hook{}) {
#if defined(__HIP_DEVICE_COMPILE__)  // GPU builtins; the host pass never runs it
  static_assert(CA == 4 || CA == 8, "activation container");
  constexpr int BM = 32 * WFM;
  static_assert(ASLOT >= BM * 16 * CA && SLOT - ASLOT >= 128 * 16 * CBH, "ring slot holds a stage");
  constexpr int LA = BM * CA / 256;                      // A loads per stage
  constexpr int LB = CBH >= 2 ? CBH / 2 : 1;             // B loads per stage
  constexpr int L = LA + LB;
  constexpr bool UNI = CBL == CBH;
  const int nst = (ng + 1) >> 1;
  const int TB = bpre[8];  // B chunks per full stage

  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      (void*)abase, (short)0, (int)min((int64_t)0x7FFFFFF0, (int64_t)(BM / kBlk) * mstride), 0x00020000);
  const __amdgpu_buffer_rsrc_t br =
      __builtin_amdgcn_make_buffer_rsrc((void*)wtile, (short)0, wbytes, 0x00020000);

  // A chunk ci = i*256 + tid of a stage: m-block ci / (16*CA), byte
  // (ci mod 16*CA)*16 of the stage's 256*CA bytes; second granule when that
  // byte is >= 128*CA.
  uint32_t aoff[LA];
  bool asec[LA];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int ci = i * 256 + tid;
    const int mb = ci / (16 * CA), w = ci - mb * 16 * CA;
    aoff[i] = (uint32_t)(mb * mstride + w * 16);
    asec[i] = w >= 8 * CA;
  }
  // B chunk ci: block j (bpre[j] <= ci < bpre[j+1]), container c_j.
  uint32_t boff[LB];
  uint32_t bstep[LB];
  bool bsec[LB], bval[LB];
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int ci = i * 256 + tid;
    int pj = 0, cj = bc[0];
#pragma unroll
    for (int t = 1; t < 8; ++t) {
      const bool in = ci >= bpre[t];
      pj += in ? bpre[t] - bpre[t - 1] : 0;
      cj += in ? bc[t] - bc[t - 1] : 0;
    }
    // block j starts ngt*128*(sum of earlier c) = ngt*8*pj bytes in
    boff[i] = (uint32_t)(ngt * 8 * pj + qbase * 128 * cj + (ci - pj) * 16);
    bstep[i] = 256 * cj;
    bsec[i] = ci - pj >= 8 * cj;
    bval[i] = ci < TB;
  }

  auto issue = [&](int st, int slot) __attribute__((always_inline)) {
    const bool half = 2 * st + 1 >= ng;  // final stage holds one granule
    const uint32_t ldsb = lds_off(lds) + (uint32_t)(slot * SLOT);
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ar, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + (i * 256 + wid * 64) * 16), 16,
          half && asec[i] ? kOOB : aoff[i], st * 256 * CA, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const bool skip = !bval[i] || (half && bsec[i]);
      const uint32_t vo = UNI ? boff[i] : boff[i] + (uint32_t)st * bstep[i];
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          br, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + ASLOT + (i * 256 + wid * 64) * 16), 16,
          skip ? kOOB : vo, UNI ? st * 256 * CBL : 0, 0, 0);
    }
  };

  // The wave's four weight blocks: container (wave-uniform) and this lane's
  // unit address in granule 0 of slot 0.
  int wcj[4];
  uint32_t b_lds[4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    wcj[jj] = UNI ? CBL : __builtin_amdgcn_readfirstlane(wn ? bc[4 + jj] : bc[jj]);
    b_lds[jj] = lds_off(lds) + (uint32_t)(ASLOT + (wn ? bpre[4 + jj] : bpre[jj]) * 16 + lane * 2 * wcj[jj]);
  }
  const uint32_t a_lds = lds_off(lds) + (uint32_t)(lane * 2 * CA + wm * WFM * 2 * 128 * CA);

  int issued = 0;
  for (; issued < NST - 1 && issued < nst; ++issued) issue(issued, issued);
  for (int st = 0; st < nst; ++st) {
    // Stages issued after st: at most NST - 2.
    const int later = issued - st - 1;
    if (NST >= 6 && later >= 4) wait_vm<(NST >= 6 ? 4 * L : 0)>();
    else if (NST >= 5 && later == 3) wait_vm<(NST >= 5 ? 3 * L : 0)>();
    else if (NST >= 4 && later == 2) wait_vm<(NST >= 4 ? 2 * L : 0)>();
    else if (NST >= 3 && later == 1) wait_vm<(NST >= 3 ? L : 0)>();
    else wait_vm<0>();
    bar_nofence();
    if (issued < nst) {
      issue(issued, issued % NST);
      ++issued;
    }
    const uint32_t soff = (uint32_t)((st % NST) * SLOT);
    const uint32_t b_addr[4] = {b_lds[0] + soff, b_lds[1] + soff, b_lds[2] + soff, b_lds[3] + soff};
    if constexpr (UNI) {
      mma_stage<CA, CBL, WFM>(acc, a_lds + soff, b_addr, hook, 2 * st);
    } else {
      mma_granule<CA, CBL, CBH, WFM, 0>(acc, a_lds + soff, b_addr, wcj, false);
      hook(acc, 2 * st);
      mma_granule<CA, CBL, CBH, WFM, 1>(acc, a_lds + soff, b_addr, wcj, false);
      hook(acc, 2 * st + 1);
    }
  }
  // Everyone is done reading the ring before the next group refills it.
  bar_nofence();
#endif
}

// ----------------------------------------------------------- wide stages --
// A stage of a tile of one weight width holds as many granules as its two
// containers allow in the ring slot, so narrow operands (4-bit activations
// against 2-bit weights, say) fill a slot with 4 or 6 granules instead of
// 2: fewer stages per group, so fewer memory round trips and barriers on
// short K.  A granule of a BM x 128 tile holds BM*8*CA activation bytes and
// 1024*CB weight bytes; each side's stage region is a whole number of
// 4 KB load rounds (256 lanes x 16 bytes).
constexpr int wide_loads(int chunks) { return (chunks + 255) / 256; }
constexpr int wide_bytes(int WFM, int CA, int CB, int g) {
  return 4096 * (wide_loads(16 * WFM * g * CA) + wide_loads(64 * g * CB));
}
constexpr int wide_gps(int WFM, int CA, int CB, int slot) {
  int best = 2;
  for (int g = 4; g <= 8; g += 2)
    if (wide_bytes(WFM, CA, CB, g) <= slot) best = g;
  return best;
}

// Granule KK of a wide stage: B fragments of the wave's four blocks (block
// jj at jj*GPS*128*CB from b_addr), A fragments of its WFM m-blocks (m-block
// i at i*GPS*128*CA from a_addr), both at granule offset KK*128*C.
template <int C, int GPS, int KK, int N, int... I>
__device__ __forceinline__ void wide_units(raw_t<C> (&r)[N], uint32_t addr,
                                           std::integer_sequence<int, I...>) {
  ((r[I] = lds_unit<C, (I * GPS + KK) * 128 * C>(addr)), ...);
}

template <int CA, int CB, int WFM, int GPS, int KK>
__device__ __forceinline__ void wide_read(raw_t<CB> (&rb)[4], raw_t<CA> (&ra)[WFM], uint32_t a_addr,
                                          uint32_t b_addr) {
  wide_units<CB, GPS, KK>(rb, b_addr, std::make_integer_sequence<int, 4>{});
  wide_units<CA, GPS, KK>(ra, a_addr, std::make_integer_sequence<int, WFM>{});
}

template <int CA, int CB, int WFM>
__device__ __forceinline__ void wide_mma(v4i (&acc)[WFM][4], raw_t<CB> (&rb)[4], raw_t<CA> (&ra)[WFM]) {
  v4i bf[4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    lds_touch(rb[jj]);
    bf[jj] = unpack_frag<CB>(rb[jj]);
  }
#pragma unroll
  for (int i = 0; i < WFM; ++i) {
    lds_touch(ra[i]);
    const v4i af = unpack_frag<CA>(ra[i]);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf[jj], acc[i][jj], 0, 0, 0);
  }
}

// R granules of one wide stage, straight-line: granule KK+1's reads are
// issued before granule KK is widened and multiplied, so an LDS round trip
// hides behind the products of the granule before.  The two register sets
// alternate at compile time and no branch joins values of reads still in
// flight (a join would let the register allocator copy such a register
// before its wait).
template <int CA, int CB, int WFM, int GPS, int R, int KK>
__device__ __forceinline__ void wide_granules(v4i (&acc)[WFM][4], raw_t<CB> (&b0)[4],
                                              raw_t<CA> (&a0)[WFM], raw_t<CB> (&b1)[4],
                                              raw_t<CA> (&a1)[WFM], uint32_t a_addr,
                                              uint32_t b_addr) {
  if constexpr (KK < R) {
    constexpr bool odd = (KK & 1) != 0;
    if constexpr (KK + 1 < R) {
      if constexpr (odd) wide_read<CA, CB, WFM, GPS, KK + 1>(b0, a0, a_addr, b_addr);
      else wide_read<CA, CB, WFM, GPS, KK + 1>(b1, a1, a_addr, b_addr);
      lds_wait_n<4 + WFM>();
    } else {
      lds_wait();
    }
    if constexpr (odd) wide_mma<CA, CB, WFM>(acc, b1, a1);
    else wide_mma<CA, CB, WFM>(acc, b0, a0);
#if defined(__HIP_DEVICE_COMPILE__)
    // keep these products ahead of the next granule's wait
    __builtin_amdgcn_sched_barrier(0);
#endif
    wide_granules<CA, CB, WFM, GPS, R, KK + 1>(acc, b0, a0, b1, a1, a_addr, b_addr);
  }
}

template <int CA, int CB, int WFM, int GPS, int R>
__device__ __forceinline__ void wide_stage(v4i (&acc)[WFM][4], uint32_t a_addr, uint32_t b_addr) {
  raw_t<CB> b0[4], b1[4];
  raw_t<CA> a0[WFM], a1[WFM];
  wide_read<CA, CB, WFM, GPS, 0>(b0, a0, a_addr, b_addr);
  wide_granules<CA, CB, WFM, GPS, R, 0>(acc, b0, a0, b1, a1, a_addr, b_addr);
}

// A stage with rem valid granules (rem >= GPS: a full one); each count is
// its own straight-line body.
template <int CA, int CB, int WFM, int GPS, int R = GPS>
__device__ __forceinline__ void wide_stage_rem(v4i (&acc)[WFM][4], uint32_t a_addr, uint32_t b_addr,
                                               int rem) {
  if constexpr (R >= 1) {
    if (rem >= R) wide_stage<CA, CB, WFM, GPS, R>(acc, a_addr, b_addr);
    else wide_stage_rem<CA, CB, WFM, GPS, R - 1>(acc, a_addr, b_addr, rem);
  }
}

// One activation group's K loop on a tile of one weight width (CA, CB
// fixed), BM x 128 (BM = 32*WFM), waves 2 x 2, through an NST-deep ring of
// SLOT-byte slots, GPS granules per stage (wide_gps).  Slot layout: the A
// stage (m-block i, granule kk at (i*GPS + kk)*128*CA), then at ABYTES the
// B stage (block j, granule kk at (j*GPS + kk)*128*CB).  Loads go through
// buffer resources; chunks past the group's data, and lanes past a stage's
// chunks, read as zero (their products vanish).
template <int CA, int CB, int WFM, int NST, int SLOT>
__device__ __forceinline__ void gemm_group_wide(uint8_t* lds, const uint8_t* abase, int64_t mstride,
                                                int ng, const uint8_t* wtile, int wbytes, int ngt,
                                                int qbase, v4i (&acc)[WFM][4], int tid, int lane,
                                                int wid, int wm, int wn) {
#if defined(__HIP_DEVICE_COMPILE__)  // GPU builtins; the host pass never runs it
  constexpr int BM = 32 * WFM;
  constexpr int GPS = wide_gps(WFM, CA, CB, SLOT);
  constexpr int CHA = 16 * WFM * GPS * CA;  // A chunks per stage
  constexpr int CHB = 64 * GPS * CB;        // B chunks per stage
  constexpr int LA = wide_loads(CHA), LB = wide_loads(CHB);
  constexpr int L = LA + LB;
  constexpr int ABYTES = 4096 * LA;
  static_assert(4096 * (LA + LB) <= SLOT, "a wide stage fits its slot");
  static_assert((GPS - 1 + 3 * GPS) * 128 * CB + ABYTES < 65536 && (WFM * GPS) * 128 * CA < 65536,
                "ds offsets");
  const int nst = (ng + GPS - 1) / GPS;

  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      (void*)abase, (short)0, (int)min((int64_t)0x7FFFFFF0, (int64_t)(BM / kBlk) * mstride), 0x00020000);
  const __amdgpu_buffer_rsrc_t br =
      __builtin_amdgcn_make_buffer_rsrc((void*)wtile, (short)0, wbytes, 0x00020000);

  // A chunk ci of a stage: m-block ci / (GPS*8*CA), granule-in-stage
  // (ci mod GPS*8*CA) / (8*CA); B chunk ci: block ci / (GPS*8*CB).
  // Lanes past a stage's chunks read zeros (kOOB) into the region's tail.
  uint32_t aoff[LA], boff[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int ci = i * 256 + tid;
    const int mb = ci / (GPS * 8 * CA), w = ci - mb * (GPS * 8 * CA);
    aoff[i] = ci < CHA ? (uint32_t)(mb * mstride + w * 16) : kOOB;
  }
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int ci = i * 256 + tid;
    const int j = ci / (GPS * 8 * CB), w = ci - j * (GPS * 8 * CB);
    boff[i] = ci < CHB ? (uint32_t)(j * ngt * 128 * CB + qbase * 128 * CB + w * 16) : kOOB;
  }

  // Stage st into ring slot `slot`; in a final partial stage (rem < GPS
  // valid granules) the chunks of the missing granules read zeros, so
  // their products vanish.
  auto issue = [&](int st, int slot) __attribute__((always_inline)) {
    const int rem = ng - st * GPS;
    const uint32_t ldsb = lds_off(lds) + (uint32_t)(slot * SLOT);
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      const int q = ((i * 256 + tid) % (GPS * 8 * CA)) / (8 * CA);  // granule in the stage
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ar, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + (i * 256 + wid * 64) * 16), 16,
          rem >= GPS || q < rem ? aoff[i] : kOOB, st * GPS * 128 * CA, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const int q = ((i * 256 + tid) % (GPS * 8 * CB)) / (8 * CB);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          br, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + ABYTES + (i * 256 + wid * 64) * 16),
          16, rem >= GPS || q < rem ? boff[i] : kOOB, st * GPS * 128 * CB, 0, 0);
    }
  };

  const uint32_t b_lds = lds_off(lds) + (uint32_t)(ABYTES + wn * 4 * GPS * 128 * CB + lane * 2 * CB);
  const uint32_t a_lds = lds_off(lds) + (uint32_t)(wm * WFM * GPS * 128 * CA + lane * 2 * CA);

  int issued = 0;
  for (; issued < NST - 1 && issued < nst; ++issued) issue(issued, issued);
  // Stage st's loads have landed for every wave, and the next stage's
  // loads are in flight.
  auto ready = [&](int st) __attribute__((always_inline)) {
    const int later = issued - st - 1;
    if (NST >= 4 && later == 2) wait_vm<(NST >= 4 ? 2 * L : 0)>();
    else if (NST >= 3 && later == 1) wait_vm<(NST >= 3 ? L : 0)>();
    else wait_vm<0>();
    bar_nofence();
    if (issued < nst) {
      issue(issued, issued % NST);
      ++issued;
    }
    return (uint32_t)((st % NST) * SLOT);
  };
  // Full stages share one loop body (one path, so the accumulators stay
  // in place); a final partial stage runs once after it.
  const int nfull = ng / GPS;
  for (int st = 0; st < nfull; ++st) {
    const uint32_t soff = ready(st);
    wide_stage<CA, CB, WFM, GPS, GPS>(acc, a_lds + soff, b_lds + soff);
  }
  if (nfull < nst) {
    const uint32_t soff = ready(nfull);
    wide_stage_rem<CA, CB, WFM, GPS, GPS - 1>(acc, a_lds + soff, b_lds + soff, ng - nfull * GPS);
  }
  // Everyone is done reading the ring before the next group refills it.
  bar_nofence();
#endif
}

// One activation group's K loop of a BM x 128 tile (BM = 32*WFM; waves 2x2,
// wave tile (16*WFM) x 64), through an NST-deep LDS ring.  Stage = 2
// granules.  A stage in LDS: m-block i granule kk at (2i + kk)*128*ca; B
// stage: block j at bpre[j]*16, granule kk at +kk*128*c_j.  Every wave
// issues exactly WFM + kLB direct loads per stage (lanes past the data
// re-load one valid chunk into an unused slot), so each wait is a
// compile-time vmcnt.
template <int CA, int CBL, int CBH, int WFM, int NST, int ASLOT, int SLOT,
          class Hook = NoGranuleHook>
__device__ __forceinline__ void gemm_group_any(uint8_t* lds, const uint8_t* abase, int64_t mstride,
                                           int ca_rt, int ng, const uint8_t* wtile, int ngt,
                                           const int (&bc)[8], const int (&bpre)[9], int qbase,
                                           v4i (&acc)[WFM][4], int tid, int lane, int wid,
                                           int wm, int wn, Hook&& hook = Hook{}) {
  constexpr int BM = 32 * WFM;
  static_assert(ASLOT == BM * 16 * 8 && SLOT == ASLOT + kBSlot, "runtime containers: 8-bit slots");
  constexpr int L = WFM + kLB;
  const int ca = CA ? CA : ca_rt;
  const int ach = BM * ca;  // A chunks (16 B) per full stage
  const int TB = bpre[8];
  const int nst = (ng + 1) >> 1;

  // Per-lane source offsets, fixed for the whole group: stage st adds
  // st*256*ca (A, uniform) or st*256*c_j (B, per lane).
  uint32_t aoff[WFM];
#pragma unroll
  for (int i = 0; i < WFM; ++i) {
    const int ci = min(i * 256 + tid, ach - 1);
    const int mb = ci / (16 * ca);
    aoff[i] = (uint32_t)(mb * mstride + (ci - mb * 16 * ca) * 16);
  }
  uint32_t boffs[kLB], bstr[kLB];
#pragma unroll
  for (int i = 0; i < kLB; ++i) {
    const int ci = min(i * 256 + tid, TB - 1);
    int pj = 0, cj = bc[0];
#pragma unroll
    for (int t = 1; t < 8; ++t) {
      const bool in = ci >= bpre[t];
      pj += in ? bpre[t] - bpre[t - 1] : 0;
      cj += in ? bc[t] - bc[t - 1] : 0;
    }
    // Blocks are contiguous: block j starts ngt*128*(sum of earlier c) bytes in.
    boffs[i] = (uint32_t)(ngt * 8 * pj + qbase * 128 * cj + (ci - pj) * 16);
    bstr[i] = 256 * cj;
  }

  auto issue = [&](int st, int slot) {
    uint8_t* As = lds + slot * SLOT;
    uint8_t* Bs = As + ASLOT;
    const uint8_t* ast = abase + (int64_t)st * 256 * ca;
    if (2 * st + 1 < ng) {
#pragma unroll
      for (int i = 0; i < WFM; ++i) load_lds16(ast + aoff[i], As + (i * 256 + wid * 64) * 16);
#pragma unroll
      for (int i = 0; i < kLB; ++i)
        load_lds16(wtile + boffs[i] + (uint32_t)st * bstr[i], Bs + (i * 256 + wid * 64) * 16);
    } else {
      // Final half stage: second-granule chunks re-load a first-granule chunk
      // (same slot layout; those slots are never read as data).
#pragma unroll
      for (int i = 0; i < WFM; ++i) {
        const int ci = min(i * 256 + tid, ach - 1);
        const int mb = ci / (16 * ca);
        const int off = ci - mb * 16 * ca;
        load_lds16(ast + aoff[i] - (off >= 8 * ca ? 8 * ca * 16 : 0), As + (i * 256 + wid * 64) * 16);
      }
#pragma unroll
      for (int i = 0; i < kLB; ++i) {
        const uint32_t cj = bstr[i] >> 8;
        const int ci = min(i * 256 + tid, TB - 1);
        int pj = 0;
#pragma unroll
        for (int t = 1; t < 8; ++t) pj += ci >= bpre[t] ? bpre[t] - bpre[t - 1] : 0;
        const int off = ci - pj;
        load_lds16(wtile + boffs[i] + (uint32_t)st * bstr[i] - (off >= 8 * (int)cj ? 8 * cj * 16 : 0),
                   Bs + (i * 256 + wid * 64) * 16);
      }
    }
  };

  // The wave's four weight blocks: LDS offset of this lane's unit in
  // granule 0 of the stage, and the block's container (wave-uniform).
  int wcj[4], wlo[4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    wcj[jj] = __builtin_amdgcn_readfirstlane(wn ? bc[4 + jj] : bc[jj]);
    wlo[jj] = (wn ? bpre[4 + jj] : bpre[jj]) * 16 + lane * 2 * wcj[jj];
  }

  int issued = 0;
  for (; issued < NST - 1 && issued < nst; ++issued) issue(issued, issued);
  for (int st = 0; st < nst; ++st) {
    // Stages issued after st: at most NST - 2.
    const int later = issued - st - 1;
    if (NST >= 6 && later >= 4) wait_vm<(NST >= 6 ? 4 * L : 0)>();
    else if (NST >= 5 && later == 3) wait_vm<(NST >= 5 ? 3 * L : 0)>();
    else if (NST >= 4 && later == 2) wait_vm<(NST >= 4 ? 2 * L : 0)>();
    else if (NST >= 3 && later == 1) wait_vm<(NST >= 3 ? L : 0)>();
    else wait_vm<0>();
    bar_nofence();
    if (issued < nst) {
      issue(issued, issued % NST);
      ++issued;
    }
    const int slot = st % NST;
    // Both granules of the stage run unconditionally; in a final half stage
    // the second granule's A fragments are zeroed, so its products vanish
    // whatever its slot holds.
    const bool second = 2 * st + 1 < ng;
    {
      const uint8_t* As = lds + slot * SLOT + lane * 2 * ca;
      const uint8_t* Bs = lds + slot * SLOT + ASLOT;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        v4i af[WFM], bf[4];
#pragma unroll
        for (int i = 0; i < WFM; ++i) {
          const v4i f = read_frag_a<CA>(As + ((wm * WFM + i) * 2 + kk) * 128 * ca, 0, ca);
          af[i] = (kk == 0 || second) ? f : v4i{0, 0, 0, 0};
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          bf[jj] = read_frag_w<CBL, CBH>(Bs + wlo[jj] + kk * 128 * wcj[jj], 0, wcj[jj]);
#pragma unroll
        for (int i = 0; i < WFM; ++i)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[jj], acc[i][jj], 0, 0, 0);
        hook(acc, 2 * st + kk);
      }
    }
  }
  // Everyone is done reading the ring before the next group refills it.
  bar_nofence();
}

// ---------------------------------------------------- implicit conv 3x3 --
// One activation group's K loop of a 64 x 128 tile of an implicit 3x3
// convolution: the weights as in gemm_group_wide (direct loads into the
// ring); the activation units gathered from the haloed code image.  The
// group's tap-major axis puts unit (granule q, 16-channel column kg) of an
// output pixel at tap t = K'/cpad, channels K' mod cpad .. +16 (K' = 64q +
// 16kg; past 9*cpad: padding, zero), which is one 2*CA-byte run of the
// image at the pixel shifted by the tap.  Thread (wave kg, m-block
// (tid/16)%4, row tid%16) loads its unit of every granule of a stage into
// registers while the previous stage is multiplied, then writes them into
// the stage's ring slot in the fragment-major layout the products read.
template <int CA, int CB, int NST, int SLOT>
__device__ __forceinline__ void gemm_group_conv(uint8_t* lds, const uint8_t* img, int rowbytes,
                                                int cpad, int H, int W, int64_t M, int64_t m0,
                                                int ng, const uint8_t* wtile, int wbytes, int ngt,
                                                int qbase, v4i (&acc)[2][4], int tid, int lane,
                                                int wid, int wm, int wn) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int WFM = 2;
  constexpr int GPS = wide_gps(WFM, CA, CB, SLOT);
  constexpr int CHB = 64 * GPS * CB;
  constexpr int LA = wide_loads(16 * WFM * GPS * CA), LB = wide_loads(CHB);
  constexpr int ABYTES = 4096 * LA;
  static_assert(NST == 2, "two ring slots");
  static_assert(4096 * (LA + LB) <= SLOT, "a stage fits its slot");
  const int nst = (ng + GPS - 1) / GPS;

  const __amdgpu_buffer_rsrc_t br =
      __builtin_amdgcn_make_buffer_rsrc((void*)wtile, (short)0, wbytes, 0x00020000);
  uint32_t boff[LB];
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int ci = i * 256 + tid;
    const int j = ci / (GPS * 8 * CB), w = ci - j * (GPS * 8 * CB);
    boff[i] = ci < CHB ? (uint32_t)(j * ngt * 128 * CB + qbase * 128 * CB + w * 16) : kOOB;
  }
  auto issue_b = [&](int st, int slot) __attribute__((always_inline)) {
    const int rem = ng - st * GPS;
    const uint32_t ldsb = lds_off(lds) + (uint32_t)(slot * SLOT) + ABYTES;
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const int q = ((i * 256 + tid) % (GPS * 8 * CB)) / (8 * CB);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          br, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + (i * 256 + wid * 64) * 16),
          16, rem >= GPS || q < rem ? boff[i] : kOOB, st * GPS * 128 * CB, 0, 0);
    }
  };

  // this thread's output pixel (rows past M repeat the last one; their
  // sums are never stored) and its haloed center
  const int mb = (tid >> 4) & 3, r = tid & 15, kg = wid;
  const int64_t P = min(m0 + 16 * mb + r, M - 1);
  const int HW = H * W;
  const int b = (int)(P / HW), rem0 = (int)(P - (int64_t)b * HW);
  const int y = rem0 / W, x = rem0 - y * W;
  const int Wp = W + 2;
  const int hp0 = (b * (H + 2) + y + 1) * Wp + x + 1;
  const int kend = 9 * cpad;
  raw_t<CA> ua[GPS];
  auto load_a = [&](int st) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < GPS; ++q) {
      const int gq = st * GPS + q;
      const int kq = gq * 64 + 16 * kg;
      raw_t<CA> v{};
      if (gq < ng && kq < kend) {
        const int t = kq / cpad, c16 = (kq - t * cpad) >> 4;
        const int tr = t / 3;
        const int hp = hp0 + (tr - 1) * Wp + (t - 3 * tr - 1);
        v = *reinterpret_cast<const raw_t<CA>*>(img + (int64_t)hp * rowbytes + c16 * 2 * CA);
      }
      ua[q] = v;
    }
  };
  const int aw = (mb * GPS) * 128 * CA + (kg * 16 + r) * 2 * CA;
  auto write_a = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < GPS; ++q)
      *reinterpret_cast<raw_t<CA>*>(lds + slot * SLOT + aw + q * 128 * CA) = ua[q];
  };

  const uint32_t b_lds = lds_off(lds) + (uint32_t)(ABYTES + wn * 4 * GPS * 128 * CB + lane * 2 * CB);
  const uint32_t a_lds = lds_off(lds) + (uint32_t)(wm * WFM * GPS * 128 * CA + lane * 2 * CA);

  issue_b(0, 0);
  load_a(0);
  write_a(0);
  auto ready = [&](int st) __attribute__((always_inline)) {
    // this thread's unit writes and every wave's weight loads have landed
    __builtin_amdgcn_s_waitcnt(0);
    bar_nofence();
    if (st + 1 < nst) {
      issue_b(st + 1, (st + 1) & 1);
      load_a(st + 1);
    }
    return (uint32_t)((st & 1) * SLOT);
  };
  const int nfull = ng / GPS;
  for (int st = 0; st < nfull; ++st) {
    const uint32_t soff = ready(st);
    wide_stage<CA, CB, WFM, GPS, GPS>(acc, a_lds + soff, b_lds + soff);
    if (st + 1 < nst) write_a((st + 1) & 1);
  }
  if (nfull < nst) {
    const uint32_t soff = ready(nfull);
    wide_stage_rem<CA, CB, WFM, GPS, GPS - 1>(acc, a_lds + soff, b_lds + soff, ng - nfull * GPS);
  }
  // Everyone is done reading the ring before the next group refills it.
  bar_nofence();
#endif
}

// ------------------------------------------------------ f8f6f4 tiles --
// One unit of an MFMA-native copy in LDS, as the raw registers of its reads:
// the lane's first 16 bytes at a + OFF, and for fp6 its last 8 bytes at
// a8 + OFF (a8 = this lane's address in the fp6 tail region).  The operand
// (8-dword type of the instruction; the unused dwords are never read by it)
// is assembled only after the reads have landed (f_operand), so that no
// register move can read a destination still in flight.
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

struct FRaw {
  u32x4v lo;
  u32x2v hi;
};

template <int FMT, int OFF>
__device__ __forceinline__ FRaw lds_funit(uint32_t a, uint32_t a8) {
  static_assert(OFF >= 0 && OFF + 1024 < 65536, "ds offset range");
  FRaw r{};
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r.lo) : "v"(a), "i"(OFF));
  if constexpr (FMT == kFmtFp6) asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(r.hi) : "v"(a8), "i"(OFF));
#else
  (void)a;
  (void)a8;
#endif
  return r;
}

template <int FMT, int STRIDE, int N, int... I>
__device__ __forceinline__ void lds_funits(FRaw (&r)[N], uint32_t a, uint32_t a8,
                                           std::integer_sequence<int, I...>) {
  ((r[I] = lds_funit<FMT, I * STRIDE>(a, a8)), ...);
}

// After the wait: pin the raw registers below it, then form the operand.
template <int FMT>
__device__ __forceinline__ v8i f_operand(FRaw& r) {
  lds_touch(r.lo);
  if constexpr (FMT == kFmtFp6) lds_touch(r.hi);
  v8i o{};
  o[0] = (int)r.lo.x;
  o[1] = (int)r.lo.y;
  o[2] = (int)r.lo.z;
  o[3] = (int)r.lo.w;
  if constexpr (FMT == kFmtFp6) {
    o[4] = (int)r.hi.x;
    o[5] = (int)r.hi.y;
  }
  return o;
}

constexpr int f_rounds(int bytes) { return (bytes / 16 + 255) / 256; }

// One activation group's K loop on the MFMA-native copies: A (format FA)
// against a tile of narrow weights (format FB), one fgranule (128
// channels) per stage, through as deep a ring as LDSB bytes hold (at most
// four).  Each wave multiplies its (16*WFM) x 64 block with
// v_mfma_scale_f32_16x16x128_f8f6f4, block scales 2^sha and 2^shw (the
// unpack exponents of the integer path, so each fp32 sum is that path's raw
// integer sum exactly), and converts the sums to int32 at the end.
// fa_tile: the group's copy at the tile's first row block (block stride
// fa_mblk); fw_tile: the tile's first weight block (block stride
// nfg*block bytes).
template <int FA, int FB, int WFM, int LDSB>
__device__ __forceinline__ void gemm_group_f(uint8_t* lds, const uint8_t* fa_tile, int64_t fa_mblk,
                                             const uint8_t* fw_tile, int wblocks, int nfg, int sha,
                                             int shw,
                                             v4i (&acc)[WFM][4], int tid, int lane, int wid, int wm,
                                             int wn) {
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int BM = 32 * WFM;
  constexpr int FBA = f_block_bytes(FA), FBB = f_block_bytes(FB);
  constexpr int CHA = (BM / kBlk) * FBA / 16, CHB = 8 * FBB / 16;  // chunks per stage
  constexpr int LA = f_rounds((BM / kBlk) * FBA), LB = f_rounds(8 * FBB);
  constexpr int L = LA + LB;
  constexpr int ABYTES = 4096 * LA, SLOTF = 4096 * (LA + LB);
  constexpr int NSTF = LDSB / SLOTF >= 4 ? 4 : LDSB / SLOTF;
  static_assert(NSTF >= 2, "at least a double ring");

  const __amdgpu_buffer_rsrc_t ar = __builtin_amdgcn_make_buffer_rsrc(
      (void*)fa_tile, (short)0, (int)min((int64_t)0x7FFFFFF0, (int64_t)(BM / kBlk) * fa_mblk), 0x00020000);
  // the weight region ends after `wblocks` of the tile's blocks (a tile of
  // a single-width handle may run past its class); beyond reads zeros
  const int64_t wbytes = (int64_t)min(8, wblocks) * nfg * FBB;
  const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc(
      (void*)fw_tile, (short)0, (int)min((int64_t)0x7FFFFFF0, wbytes), 0x00020000);
  uint32_t aoff[LA], boff[LB];
#pragma unroll
  for (int i = 0; i < LA; ++i) {
    const int ci = i * 256 + tid;
    const int mb = ci / (FBA / 16), w = ci - mb * (FBA / 16);
    aoff[i] = ci < CHA ? (uint32_t)(mb * fa_mblk + w * 16) : kOOB;
  }
#pragma unroll
  for (int i = 0; i < LB; ++i) {
    const int ci = i * 256 + tid;
    const int j = ci / (FBB / 16), w = ci - j * (FBB / 16);
    boff[i] = ci < CHB ? (uint32_t)(j * nfg * FBB + w * 16) : kOOB;
  }
  auto issue = [&](int f, int slot) __attribute__((always_inline)) {
    const uint32_t ldsb = lds_off(lds) + (uint32_t)(slot * SLOTF);
#pragma unroll
    for (int i = 0; i < LA; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ar, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + (i * 256 + wid * 64) * 16), 16,
          aoff[i], f * FBA, 0, 0);
#pragma unroll
    for (int i = 0; i < LB; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          br, (__attribute__((address_space(3))) void*)(uintptr_t)(ldsb + ABYTES + (i * 256 + wid * 64) * 16),
          16, boff[i], f * FBB, 0, 0);
  };

  const uint32_t base = lds_off(lds);
  const uint32_t a_lds = base + (uint32_t)(wm * WFM * FBA + 16 * lane);
  const uint32_t a8_lds = base + (uint32_t)(wm * WFM * FBA + 1024 + 8 * lane);
  const uint32_t b_lds = base + (uint32_t)(ABYTES + wn * 4 * FBB + 16 * lane);
  const uint32_t b8_lds = base + (uint32_t)(ABYTES + wn * 4 * FBB + 1024 + 8 * lane);
  const int sa = 127 + sha, sb = 127 + shw;  // E8M0 block scales 2^sha, 2^shw

  v4f accf[WFM][4];
#pragma unroll
  for (int i = 0; i < WFM; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) accf[i][jj] = v4f{0.0f, 0.0f, 0.0f, 0.0f};

  int issued = 0;
  for (; issued < NSTF - 1 && issued < nfg; ++issued) issue(issued, issued);
  for (int f = 0; f < nfg; ++f) {
    const int later = issued - f - 1;
    if (NSTF >= 4 && later == 2) wait_vm<(NSTF >= 4 ? 2 * L : 0)>();
    else if (NSTF >= 3 && later == 1) wait_vm<(NSTF >= 3 ? L : 0)>();
    else wait_vm<0>();
    bar_nofence();
    if (issued < nfg) {
      issue(issued, issued % NSTF);
      ++issued;
    }
    const uint32_t soff = (uint32_t)((f % NSTF) * SLOTF);
    FRaw rb[4], ra[WFM];
    lds_funits<FB, FBB>(rb, b_lds + soff, b8_lds + soff, std::make_integer_sequence<int, 4>{});
    lds_funits<FA, FBA>(ra, a_lds + soff, a8_lds + soff, std::make_integer_sequence<int, WFM>{});
    lds_wait();
    v8i bf[4];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) bf[jj] = f_operand<FB>(rb[jj]);
#pragma unroll
    for (int i = 0; i < WFM; ++i) {
      const v8i af = f_operand<FA>(ra[i]);
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        accf[i][jj] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf[jj], accf[i][jj], FA,
                                                                      FB, 0, sa, 0, sb);
    }
  }
  // Everyone is done reading the ring before it is reused.
  bar_nofence();
  // exact: integer multiples of 2^(sha+shw), below 2^24 of it
#pragma unroll
  for (int i = 0; i < WFM; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][jj][r] = (int)accf[i][jj][r];
#endif
}


// Next-layer codes of a tile, staged column-major in LDS: column rank c at
// c * (BM + 16), its BM rows in order, four rows (a qnext4 word) per write.
template <int BM>
__device__ __forceinline__ void qn_stage4(uint8_t* qs, int rank, int row0, uint32_t w) {
  *reinterpret_cast<uint32_t*>(qs + rank * (BM + 16) + row0) = w;
}

// The staged codes to the image: the thread of column rank c (next-layer
// position qpos, -1 for none) writes each 16-row block's 16 codes of its
// position as one 16-byte store (rows past M land in the image's padding
// rows, which nothing packs).
template <int BM>
__device__ __forceinline__ void qn_store(const GemmArgs& a, const uint8_t* qs, int qpos, int64_t m0,
                                         int tid) {
  const int c = tid & (kGemmBN - 1);
  if (qpos < 0) return;
  uint8_t* out = a.qn_img + (m0 / kBlk) * a.qn_ld + (int64_t)qpos * 16;
  for (int ch = tid / kGemmBN; ch < BM / 16; ch += 256 / kGemmBN)
    *reinterpret_cast<uint4*>(out + ch * a.qn_ld) =
        *reinterpret_cast<const uint4*>(qs + c * (BM + 16) + ch * 16);
}

// (32*WFM) x 128 output tile per workgroup of four waves (2 x 2).  QN > 0:
// the epilogue also quantizes every output for the next layer into qn_img
// (and stores Y only when a.Y is set), with one static scale per
// next-layer group (QN = 1) or per block of a next layer with sub-group
// scales (QN = 2, asked to keep three waves per SIMD).
template <int S, int CA0, int CA1, int CBL, int CBH, int WFM, int NST, int QN = 0, bool F = false,
          bool CV = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(
    QN == 2 ? 3 : WFM == 2 ? 3 : 2)))
void k_gemm(GemmArgs a) {
  constexpr int BM = 32 * WFM;
  // Instances whose containers are all known take at least 24 KB slots at
  // 64-row tiles (three workgroups per CU still fit LDS), so narrow
  // operands get wide stages (gemm_group_wide).
  constexpr bool KNOWN = CA0 != 0 && (S == 1 || CA1 != 0) && CBL != 0 && CBH != 0;
  constexpr int SLOT0 = gemm_slot(S, CA0, CA1, CBL, CBH, WFM);
  constexpr int SLOT = KNOWN && WFM == 2 && SLOT0 < 24576 ? 24576 : SLOT0;
  constexpr int ASLOT = gemm_aslot(S, CA0, CA1, CBL, CBH, WFM);
  __shared__ __align__(16) uint8_t lds[NST * SLOT];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const ActPlan& ap = a.ap;
  const int ntn = a.wp.Np / kGemmBN;
  // Workgroups go round-robin to the 8 XCDs (b mod 8), each with its own
  // L2.  On grids of a few rounds XCD x takes a contiguous range of tiles,
  // so the N tiles of one row block share that L2 for their activation
  // reads and for the partial output lines they write (a tile's output
  // columns are scattered); longer grids keep the launch order, whose
  // concurrent tiles share weight tiles across XCDs.
  const int G = (int)gridDim.x, x = (int)(blockIdx.x & 7), l = (int)(blockIdx.x >> 3);
  const int tile = a.xcd_tiles ? x * (G >> 3) + min(x, G & 7) + l : (int)blockIdx.x;
  const int mt = tile / ntn, nt = tile - mt * ntn;
  const int64_t m0 = (int64_t)mt * BM;
  const int jb0 = nt * 8;

  int bc[8], bpre[9];
  bpre[0] = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    bc[j] = wblk_c(a.wp, jb0 + j);
    bpre[j + 1] = bpre[j] + 16 * bc[j];
  }
  const uint8_t* wtile = a.wd.packed + wblk_off(a.wp, jb0);

  // The activation scales (written by the quantize launch just before) and,
  // on 64-row tiles, the wave's four columns of epilogue data are requested
  // now, so that they have arrived when the epilogue needs them (the
  // 128-row tiles have no registers to spare for the latter: two waves per
  // SIMD need at most 256).
  const float sa0 = a.s_a[0];
  const float sa1 = S == 2 ? a.s_a[1] : 0.0f;
  ColInfo cinf[4];
  uint8_t cshw[4], crank[4];
  int cqg[4] = {0, 0, 0, 0};  // next-layer group (or block) of each column (QN)
  if constexpr (WFM <= 2) {
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int pc = (jb0 + wn * 4 + jj) * kBlk + (lane & 15);
      cinf[jj] = a.wd.colinfo[pc];
      cshw[jj] = a.wd.shw[pc];
      crank[jj] = a.wd.colrank[pc];
      if constexpr (QN > 0) cqg[jj] = a.qn_tab[pc];
    }
  }
  // The store phase's column of this thread (its next-layer position when
  // the tile stores codes, else its original column), requested now rather
  // than after the epilogue's barrier, where its latency would hold back
  // every store of the tile.
  const int st_col = QN == 1 || QN == 2 ? a.qn_tab[a.wp.Np + nt * kGemmBN + (tid & (kGemmBN - 1))]
                                        : a.wd.tile_cols[nt * kGemmBN + (tid & (kGemmBN - 1))];

  v4i acc0[WFM][4];
#pragma unroll
  for (int i = 0; i < WFM; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) acc0[i][jj] = v4i{0, 0, 0, 0};
  // Every tile holds one weight width (the plan pads the narrow blocks to
  // whole tiles), so the loop runs with that container fixed.
  const int wbytes = (int)(wblk_off(a.wp, jb0 + 8) - wblk_off(a.wp, jb0));
  const bool tile_lo = jb0 < a.wp.nlo;
  auto run_group = [&](auto ca_tag, const uint8_t* abase, int64_t mstride, int ca_rt, int ng,
                       int qbase, v4i (&acc)[WFM][4]) __attribute__((always_inline)) {
    constexpr int CA = decltype(ca_tag)::value;
    if constexpr (CV) {
      static_assert(WFM == 2 && CA != 0 && CBL != 0 && CBH != 0, "implicit conv instances");
      const int g = qbase ? 1 : 0;
      const uint8_t* img = a.img + a.cg.img_off[g];
      if (CBL == CBH || tile_lo)
        gemm_group_conv<CA, CBL, NST, SLOT>(lds, img, a.cg.rowbytes[g], a.cg.cpad[g], a.cg.H,
                                            a.cg.W, a.M, m0, ng, wtile, wbytes, a.wp.ngt, qbase,
                                            acc, tid, lane, wid, wm, wn);
      else
        gemm_group_conv<CA, CBH, NST, SLOT>(lds, img, a.cg.rowbytes[g], a.cg.cpad[g], a.cg.H,
                                            a.cg.W, a.M, m0, ng, wtile, wbytes, a.wp.ngt, qbase,
                                            acc, tid, lane, wid, wm, wn);
      return;
    }
    if constexpr (F && CA != 0 && CBL != 0 && CBH != 0) {
      // narrow x narrow: the MFMA-native copies, when the handle has them
      const int g = qbase ? 1 : 0;
      const int k = tile_lo ? 0 : 1;
      if (a.fa && a.fp.fa[g] && a.fp.fw_off[g][k] >= 0) {
        constexpr int FA = f_fmt(CA);
        constexpr int FBL = f_fmt(CBL), FBH = f_fmt(CBH);
        const int nfg = a.fp.nfg[g];
        const uint8_t* fat = a.fa + a.fp.fa_off[g] + (m0 / kBlk) * a.fp.fa_mblk[g];
        const int first = k ? a.wp.nlo : 0;
        const int wblocks = (k ? a.wp.nblk - a.wp.nlo : a.wp.nlo) - (jb0 - first);
        const uint8_t* fwt = a.fw + a.fp.fw_off[g][k] +
                             (int64_t)(jb0 - first) * nfg * f_block_bytes(k ? FBH : FBL);
        const int sha = ap.sh[g];
        if constexpr (FA != 0 && FBL != 0) {
          if (k == 0) {
            gemm_group_f<FA, FBL, WFM, NST * SLOT>(lds, fat, a.fp.fa_mblk[g], fwt, wblocks, nfg, sha,
                                                   CBL == 8 ? 0 : CBL == 4 ? 4 : 6, acc, tid, lane,
                                                   wid, wm, wn);
            return;
          }
        }
        if constexpr (FA != 0 && FBH != 0 && CBH != CBL) {
          if (k == 1) {
            gemm_group_f<FA, FBH, WFM, NST * SLOT>(lds, fat, a.fp.fa_mblk[g], fwt, wblocks, nfg, sha,
                                                   CBH == 8 ? 0 : CBH == 4 ? 4 : 6, acc, tid, lane,
                                                   wid, wm, wn);
            return;
          }
        }
      }
    }
    if constexpr (CA != 0 && CBL != 0 && CBH != 0) {
      if (CBL == CBH || tile_lo)
        gemm_group_wide<CA, CBL, WFM, NST, SLOT>(lds, abase, mstride, ng, wtile, wbytes, a.wp.ngt,
                                                 qbase, acc, tid, lane, wid, wm, wn);
      else
        gemm_group_wide<CA, CBH, WFM, NST, SLOT>(lds, abase, mstride, ng, wtile, wbytes, a.wp.ngt,
                                                 qbase, acc, tid, lane, wid, wm, wn);
    } else {
      gemm_group_any<CA, CBL, CBH, WFM, NST, ASLOT, SLOT>(lds, abase, mstride, ca_rt, ng, wtile,
                                                          a.wp.ngt, bc, bpre, qbase, acc, tid,
                                                          lane, wid, wm, wn);
    }
  };
  run_group(std::integral_constant<int, CA0>{}, a.act + ap.seg_off[0] + (m0 / kBlk) * ap.mblk_bytes[0],
            ap.mblk_bytes[0], ap.c[0], ap.ng[0], 0, acc0);
  v4i acc1[WFM][4];
#pragma unroll
  for (int i = 0; i < WFM; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) acc1[i][jj] = v4i{0, 0, 0, 0};
  if constexpr (S == 2)
    run_group(std::integral_constant<int, CA1>{}, a.act + ap.seg_off[1] + (m0 / kBlk) * ap.mblk_bytes[1],
              ap.mblk_bytes[1], ap.c[1], ap.ng[1], ap.ng[0], acc1);

  // Epilogue: exact int32 per group, fixed-order fp32 scaling, bf16.  The
  // tile is staged in LDS (the ring is free: gemm_group ended with a
  // barrier) with its columns in ascending original order, then stored so
  // that consecutive lanes write consecutive output columns.  Staging rows
  // are padded by 8 halfwords so the four row quads of a wave's store land
  // in different banks.
  constexpr int YS = kGemmBN + 8;
  uint16_t* ys = reinterpret_cast<uint16_t*>(lds);
  static_assert(BM * YS * 2 <= NST * SLOT, "output staging fits the ring");
  if constexpr (QN == 0 || QN == 3) {
    // QN = 3: the largest |y| per next-layer group over the tile's rows
    // below M (the bf16 of the largest |y| is the largest |bf16(y)|, since
    // rounding is monotonic and symmetric)
    float ymax[2] = {0.0f, 0.0f};
    const bool full_rows = m0 + BM <= a.M;
    // Staged column-major (column rank c, row r at c*YT + r; YT odd in
    // dwords, so consecutive ranks of one row sit in different banks): a
    // lane's two pairs of rows go out as two 4-byte writes, and the stores
    // read two rows of a column at once.  The raw sum is corrected in
    // place, v = raw + add * 2^sh = (exact sum) * 2^sh, and scaled by
    // s_a * 2^-sh: f(v) * (s_a 2^-sh) is exactly f(sum) * s_a, since a
    // power of two changes no rounding (unless s_a 2^-sh is not a normal
    // number: then the shifted sum is used).
    constexpr int YT = BM + 2;
    static_assert(kGemmBN * YT * 2 <= NST * SLOT, "output staging fits the ring");
    static_assert(YT % 4 == 2, "odd dword stride");
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int pc = (jb0 + wn * 4 + jj) * kBlk + (lane & 15);
      const ColInfo ci = WFM <= 2 ? cinf[jj] : a.wd.colinfo[pc];
      if (ci.n < 0) continue;
      const uint8_t shw = WFM <= 2 ? cshw[jj] : a.wd.shw[pc];
      const bool sgn = (shw & kShwSign) != 0;
      const int sh0 = ap.sh[0] + (shw & 0x7F);
      const int add0 = ap.zp[0] * ci.colsum[0] - (ap.c[0] == 1 && sgn ? ap.padcnt[0] : 0);
      const int sh1 = ap.sh[1] + (shw & 0x7F);
      const int add1 = ap.zp[1] * ci.colsum[1] - (ap.c[1] == 1 && sgn ? ap.padcnt[1] : 0);
      const float sa0s = __builtin_ldexpf(sa0, -sh0);
      const float sa1s = S == 2 ? __builtin_ldexpf(sa1, -sh1) : 0.0f;
      const bool scaled = (sa0s == 0.0f || fabsf(sa0s) >= 0x1p-126f) &&
                          (S == 1 || sa1s == 0.0f || fabsf(sa1s) >= 0x1p-126f);
      const int add0s = add0 * (1 << sh0), add1s = S == 2 ? add1 * (1 << sh1) : 0;
      uint32_t* ycol = reinterpret_cast<uint32_t*>(ys + (WFM <= 2 ? crank[jj] : a.wd.colrank[pc]) * YT);
#pragma unroll
      for (int i = 0; i < WFM; ++i) {
        const int row0 = (wm * WFM + i) * 16 + (lane >> 4) * 4;
        float y[4];
        if (scaled) [[likely]] {
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            float t = __fmul_rn((float)(acc0[i][jj][h] + add0s), sa0s);
            if (S == 2) t = __fadd_rn(t, __fmul_rn((float)(acc1[i][jj][h] + add1s), sa1s));
            y[h] = __fmul_rn(t, ci.s_w);
          }
        } else {
#pragma unroll
          for (int h = 0; h < 4; ++h)
            y[h] = epilogue((acc0[i][jj][h] >> sh0) + add0,
                            S == 2 ? (acc1[i][jj][h] >> sh1) + add1 : 0, S, sa0, sa1, ci.s_w);
        }
        // v_cvt_pk_bf16_f32: round to nearest even, as bf16_rne.
        const __hip_bfloat162 p01 = __float22bfloat162_rn(make_float2(y[0], y[1]));
        const __hip_bfloat162 p23 = __float22bfloat162_rn(make_float2(y[2], y[3]));
        const uint32_t w01 = (uint32_t)__builtin_bit_cast(uint16_t, p01.x) |
                             ((uint32_t)__builtin_bit_cast(uint16_t, p01.y) << 16);
        const uint32_t w23 = (uint32_t)__builtin_bit_cast(uint16_t, p23.x) |
                             ((uint32_t)__builtin_bit_cast(uint16_t, p23.y) << 16);
        ycol[row0 / 2] = w01;
        ycol[row0 / 2 + 1] = w23;
        if constexpr (QN == 3) {
          float m4 = 0.0f;
          if (full_rows) [[likely]] {
#pragma unroll
            for (int h = 0; h < 4; ++h) m4 = fmaxf(m4, fabsf(y[h]));
          } else {
#pragma unroll
            for (int h = 0; h < 4; ++h)
              if (m0 + row0 + h < a.M) m4 = fmaxf(m4, fabsf(y[h]));
          }
          if (cqg[jj]) ymax[1] = fmaxf(ymax[1], m4);
          else ymax[0] = fmaxf(ymax[0], m4);
        }
        if (a.acc) {
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            const int64_t m = m0 + row0 + h;
            if (m < a.M) {
              a.acc[m * a.N + ci.n] = (acc0[i][jj][h] >> sh0) + add0;
              if (S == 2) a.acc[(a.M + m) * a.N + ci.n] = (acc1[i][jj][h] >> sh1) + add1;
            }
          }
        }
      }
    }
    if constexpr (QN == 3) {
      // the tile's maxima (over the wave, then the workgroup), rounded to
      // bf16 as Y is, into the tile's own pair: no atomics, nothing to clear
      __shared__ float qred[8];
      const float2 mx = block_max2(make_float2(ymax[0], ymax[1]), qred);
      if (tid == 0) {
        // the same rounding as the stores' (v_cvt_pk_bf16_f32), widened back
        const __hip_bfloat162 pm = __float22bfloat162_rn(mx);
        a.qn_max[2 * blockIdx.x] = __uint_as_float((uint32_t)__builtin_bit_cast(uint16_t, pm.x) << 16);
        a.qn_max[2 * blockIdx.x + 1] = __uint_as_float((uint32_t)__builtin_bit_cast(uint16_t, pm.y) << 16);
      }
    }
    __syncthreads();
    // thread: column rank tid % 128, rows 2*(tid / 128) + 4k and the next
    const int n = st_col;
    if (n >= 0) {
      const int mrem = (int)min((int64_t)BM, a.M - m0);
      uint16_t* yout = a.Y + m0 * a.ldy + n;
      const uint32_t* yc = reinterpret_cast<const uint32_t*>(ys + (tid & (kGemmBN - 1)) * YT);
      for (int row = 2 * (tid / kGemmBN); row < mrem; row += 512 / kGemmBN) {
        const uint32_t v = yc[row / 2];
        yout[(int64_t)row * a.ldy] = (uint16_t)(v & 0xFFFFu);
        if (row + 1 < mrem) yout[(int64_t)(row + 1) * a.ldy] = (uint16_t)(v >> 16);
      }
    }
    return;
  }
  // QN > 0: the same scaling as above, Y staged row-major (when asked
  // for), and each output's next-layer code staged column-major.
  uint8_t* qs = reinterpret_cast<uint8_t*>(lds) + BM * YS * 2;
  static_assert(QN == 0 || BM * YS * 2 + kGemmBN * (BM + 16) <= NST * SLOT,
                "code staging fits the ring");
  const bool want_y = a.Y != nullptr;
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    const int pc = (jb0 + wn * 4 + jj) * kBlk + (lane & 15);
    const ColInfo ci = WFM <= 2 ? cinf[jj] : a.wd.colinfo[pc];
    if (ci.n < 0) continue;
    // Exact accumulator of group g: (raw >> sh_g) + add_g, where add_g folds
    // the zero-point term and the sign x sign padding products (padcnt
    // products of +1 each, exact multiples of 2^sh_g in the raw sum); the
    // scaled form is the one above.
    const uint8_t shw = WFM <= 2 ? cshw[jj] : a.wd.shw[pc];
    const bool sgn = (shw & kShwSign) != 0;
    const int sh0 = ap.sh[0] + (shw & 0x7F);
    const int add0 = ap.zp[0] * ci.colsum[0] - (ap.c[0] == 1 && sgn ? ap.padcnt[0] : 0);
    const int sh1 = ap.sh[1] + (shw & 0x7F);
    const int add1 = ap.zp[1] * ci.colsum[1] - (ap.c[1] == 1 && sgn ? ap.padcnt[1] : 0);
    const float sa0s = __builtin_ldexpf(sa0, -sh0);
    const float sa1s = S == 2 ? __builtin_ldexpf(sa1, -sh1) : 0.0f;
    const bool scaled = (sa0s == 0.0f || fabsf(sa0s) >= 0x1p-126f) &&
                        (S == 1 || sa1s == 0.0f || fabsf(sa1s) >= 0x1p-126f);
    const int add0s = add0 * (1 << sh0), add1s = S == 2 ? add1 * (1 << sh1) : 0;
    const int rank = WFM <= 2 ? crank[jj] : a.wd.colrank[pc];
    uint16_t* ycol = ys + rank;
    QCol qc;
    if constexpr (QN == 2) {
      // sub-group scales: the block's static scale, its group's range
      const int b = WFM <= 2 ? cqg[jj] : a.qn_tab[pc];
      const bool g1 = b >= a.qn_nsub0;
      // (read here, not held through the K loop: registers decide
      // this kernel's occupancy)
      qc.sc = a.qn_bs[b];
      qc.rs = a.qn_brs[b];
      qc.lo = g1 ? a.qn.lo[1] : a.qn.lo[0];
      qc.hi = g1 ? a.qn.hi[1] : a.qn.hi[0];
      qc.zp = 0;
      qc.sign1 = false;
    } else {
      qc = qnext_col(WFM <= 2 ? cqg[jj] : a.qn_tab[pc], a.qn);
    }
#pragma unroll
    for (int i = 0; i < WFM; ++i) {
      const int row0 = (wm * WFM + i) * 16 + (lane >> 4) * 4;
      float y[4];
      if (scaled) [[likely]] {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          float t = __fmul_rn((float)(acc0[i][jj][h] + add0s), sa0s);
          if (S == 2) t = __fadd_rn(t, __fmul_rn((float)(acc1[i][jj][h] + add1s), sa1s));
          y[h] = __fmul_rn(t, ci.s_w);
        }
      } else {
#pragma unroll
        for (int h = 0; h < 4; ++h)
          y[h] = epilogue((acc0[i][jj][h] >> sh0) + add0,
                          S == 2 ? (acc1[i][jj][h] >> sh1) + add1 : 0, S, sa0, sa1, ci.s_w);
      }
      if (want_y) {
#pragma unroll
        for (int h = 0; h < 4; h += 2) {
          // v_cvt_pk_bf16_f32: round to nearest even, as bf16_rne.
          const __hip_bfloat162 pr = __float22bfloat162_rn(make_float2(y[h], y[h + 1]));
          ycol[(row0 + h) * YS] = __builtin_bit_cast(uint16_t, pr.x);
          ycol[(row0 + h + 1) * YS] = __builtin_bit_cast(uint16_t, pr.y);
        }
      }
      if (a.acc) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const int64_t m = m0 + row0 + h;
          if (m < a.M) {
            a.acc[m * a.N + ci.n] = (acc0[i][jj][h] >> sh0) + add0;
            if (S == 2) a.acc[(a.M + m) * a.N + ci.n] = (acc1[i][jj][h] >> sh1) + add1;
          }
        }
      }
      qn_stage4<BM>(qs, rank, row0, qnext4(y, qc));
    }
  }
  __syncthreads();
  qn_store<BM>(a, qs, st_col, m0, tid);
  if (!want_y) return;
  const int n = a.wd.tile_cols[nt * kGemmBN + (tid & (kGemmBN - 1))];
  if (n >= 0) {
    const int mrem = (int)min((int64_t)BM, a.M - m0);
    uint16_t* yout = a.Y + m0 * a.ldy + n;
    for (int row = tid / kGemmBN; row < mrem; row += 256 / kGemmBN)
      yout[(int64_t)row * a.ldy] = ys[row * YS + (tid & (kGemmBN - 1))];
  }
}

// ------------------------------------------------------------ k_gemv_any --
// Generic batch <= 8 path for any activation containers.
// One workgroup (4 waves) per 16-row weight block.  The block's bytes are a
// contiguous run of 16-byte chunks; wave w takes chunk rows i = w, w+4, ...
// (64 chunks each).  A chunk of container C holds U = 8/C units that share
// one granule and one 16-channel group and belong to U different rows, so
// each lane keeps U row accumulators per activation group and row.
constexpr int kGemvB = 8;  // chunk rows in flight per wave

__device__ __forceinline__ int dot16(uint4 d, uint4 x, int v) {
  v = __builtin_amdgcn_sdot4((int)d.x, (int)x.x, v, false);
  v = __builtin_amdgcn_sdot4((int)d.y, (int)x.y, v, false);
  v = __builtin_amdgcn_sdot4((int)d.z, (int)x.z, v, false);
  return __builtin_amdgcn_sdot4((int)d.w, (int)x.w, v, false);
}

template <int C>
__device__ __forceinline__ uint4 chunk_unit(uint4 raw, int u) {
  if constexpr (C == 8) return raw;
  else if constexpr (C == 4) return u == 0 ? unpack4(raw.x, raw.y) : unpack4(raw.z, raw.w);
  else if constexpr (C == 2) {
    const uint32_t w = u == 0 ? raw.x : u == 1 ? raw.y : u == 2 ? raw.z : raw.w;
    return unpack2(w);
  } else {
    const uint32_t w = (u >> 1) == 0 ? raw.x : (u >> 1) == 1 ? raw.y : (u >> 1) == 2 ? raw.z : raw.w;
    return unpack1((w >> (16 * (u & 1))) & 0xFFFFu);
  }
}

// Unpack the activation rows (block 0 of the packed buffer) into LDS.
__device__ __forceinline__ void gemv_stage_x(const GemmArgs& a, uint8_t* xs) {
  const ActPlan& ap = a.ap;
  const int M = (int)a.M, ngt = a.wp.ngt, ng0 = ap.ng[0];
  for (int u = threadIdx.x; u < M * ngt * 4; u += blockDim.x) {
    const int m = u / (ngt * 4), rest = u - m * ngt * 4;
    const int q = rest >> 2, kg = rest & 3;
    const bool g1 = q >= ng0;
    const int qq = g1 ? q - ng0 : q;
    const int c = g1 ? ap.c[1] : ap.c[0];
    const uint8_t* src = a.act + (g1 ? ap.seg_off[1] : ap.seg_off[0]) + (int64_t)qq * 128 * c +
                         (kg * 16 + m) * 2 * c;
    *reinterpret_cast<uint4*>(xs + m * ap.Kp + q * kGran + kg * 16) =
        unpack_unit_rt(load_unit(src, c), c);
  }
}

// Bytes of the activation buffer up to the end of the last group's first
// 16-row block (what a GEMV reads).
__host__ __device__ inline int64_t gemv_dense_xbytes64(const ActPlan& ap) {
  const int64_t e0 = ap.seg_off[0] + ap.mblk_bytes[0];
  const int64_t e1 = ap.S == 2 ? ap.seg_off[1] + ap.mblk_bytes[1] : 0;
  return e0 > e1 ? e0 : e1;
}
__device__ __forceinline__ int gemv_dense_xbytes(const ActPlan& ap) { return (int)gemv_dense_xbytes64(ap); }

template <int MT, int C>
__device__ __forceinline__ void gemv_block(const GemmArgs& a, uint8_t* xs, int blk,
                                           int (&red)[4][kBlk][2][8]) {
  constexpr int U = 8 / C;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const ActPlan& ap = a.ap;
  const int M = (int)a.M, Kp = ap.Kp, ng0 = ap.ng[0];
  const uint8_t* base = a.wd.packed + wblk_off(a.wp, blk);
  const int nchunks = a.wp.ngt * 8 * C;
  const int NI = (nchunks + 63) >> 6;
  const int kg = ((U * lane) & 63) >> 4;
  const int qoff = (U * lane) >> 6;

  int acc0[U][MT], acc1[U][MT];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) {
      acc0[u][mm] = 0;
      acc1[u][mm] = 0;
    }

  // The first batch of weight chunks is in flight while the activations are
  // unpacked into LDS.
  uint4 raw[kGemvB];
  int i0 = wid;
#pragma unroll
  for (int b = 0; b < kGemvB; ++b) {
    const int ci = min((i0 + 4 * b) * 64 + lane, nchunks - 1);
    raw[b] = *reinterpret_cast<const uint4*>(base + (int64_t)ci * 16);
  }
  gemv_stage_x(a, xs);
  __syncthreads();

  for (; i0 < NI; i0 += 4 * kGemvB) {
    if (i0 != wid) {
#pragma unroll
      for (int b = 0; b < kGemvB; ++b) {
        const int ci = min((i0 + 4 * b) * 64 + lane, nchunks - 1);
        raw[b] = *reinterpret_cast<const uint4*>(base + (int64_t)ci * 16);
      }
    }
#pragma unroll
    for (int b = 0; b < kGemvB; ++b) {
      const int i = i0 + 4 * b;
      if (i * 64 + lane < nchunks) {
        const int q = U * i + qoff;
        const int k0 = q * kGran + 16 * kg;
        const bool g1 = q >= ng0;
#pragma unroll
        for (int mm = 0; mm < MT; ++mm) {
          if (mm < M) {
            const uint4 x = *reinterpret_cast<const uint4*>(xs + mm * Kp + k0);
#pragma unroll
            for (int u = 0; u < U; ++u) {
              const int v = dot16(chunk_unit<C>(raw[b], u), x, 0);
              if (g1) acc1[u][mm] += v; else acc0[u][mm] += v;
            }
          }
        }
      }
    }
  }

  // Lanes that share rows: equal lane mod (16/U).
#pragma unroll
  for (int o = 16 / U; o < 64; o <<= 1)
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) {
        acc0[u][mm] += __shfl_xor(acc0[u][mm], o, 64);
        acc1[u][mm] += __shfl_xor(acc1[u][mm], o, 64);
      }

  // Across the four waves, through LDS; then one thread per (row, m).
  if (lane < 16 / U) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) {
        red[wid][U * lane + u][0][mm] = acc0[u][mm];
        red[wid][U * lane + u][1][mm] = acc1[u][mm];
      }
  }
  __syncthreads();
  if (tid < kBlk * M) {
    const int r = tid / M, m = tid - r * M;
    int s0 = 0, s1 = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      s0 += red[w][r][0][m];
      s1 += red[w][r][1][m];
    }
    const int p = blk * kBlk + r;
    const ColInfo ci = a.wd.colinfo[p];
    if (ci.n >= 0) {
      const uint8_t shw = a.wd.shw[p];
      const int S = ap.S;
      const int t0 = true_acc(s0, ap.sh[0], ap.c[0], ap.padcnt[0], ap.zp[0], shw, ci.colsum[0]);
      const int t1 = S == 2 ? true_acc(s1, ap.sh[1], ap.c[1], ap.padcnt[1], ap.zp[1], shw, ci.colsum[1])
                            : 0;
      const float sa0 = a.s_a[0], sa1 = S == 2 ? a.s_a[1] : 0.0f;
      a.Y[(int64_t)m * a.ldy + ci.n] = bf16_rne(epilogue(t0, t1, S, sa0, sa1, ci.s_w));
      if (a.acc) {
        a.acc[(int64_t)m * a.N + ci.n] = t0;
        if (S == 2) a.acc[(a.M + m) * a.N + ci.n] = t1;
      }
    }
  }
}

// Dynamic LDS: M * Kp bytes of unpacked activations.
template <int MT>
__global__ __launch_bounds__(256) void k_gemv_any(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];
  __shared__ int red[4][kBlk][2][8];
  const int blk = blockIdx.x;
  const int c = wblk_c(a.wp, blk);
  if (c == 2) gemv_block<MT, 2>(a, xs, blk, red);
  else if (c == 4) gemv_block<MT, 4>(a, xs, blk, red);
  else if (c == 8) gemv_block<MT, 8>(a, xs, blk, red);
  else gemv_block<MT, 1>(a, xs, blk, red);
}



// ---------------------------------------------------------------- k_gemv --
// Batch <= 8 decode with the first activation group in 4-bit containers and
// the second (if any) in bytes.  One workgroup (256 threads) per 16-row
// weight block.  A block is ngt granules of 8*CW 16-byte chunks; the first
// ng0 granules meet activation group 0, the rest group 1.  Load slot b of
// thread tid holds chunk tid + 256*b of group 0 for b < NB0, else chunk
// tid + 256*(b - NB0) of group 1, so a slot's group is fixed at compile
// time and the thread's place inside a granule is fixed too:
// t = tid mod 8*CW, i.e. rows r0 .. r0+U-1 (U = 8/CW) of 16-channel group
// kg.  Loads are raw buffer loads; chunks past a group's end read as zero
// without touching memory, so all of a thread's loads are issued at once
// and zero chunks add nothing (except 1-bit blocks, where they are masked).
//   - group 0 x 2- or 4-bit weights: v_dot8_i32_i4 on packed nibbles (a
//     2-bit word becomes two nibble words with two masks);
//   - otherwise bytes and v_dot4_i32_i8.
// Lanes of a 16-lane DPP row that share output rows are summed with
// row_ror; the four rows of a wave and the four waves meet in LDS.

__device__ __forceinline__ int dot16n(uint32_t w0, uint32_t w1, uint2 x, int v) {
  v = __builtin_amdgcn_sdot8((int)w0, (int)x.x, v, false);
  return __builtin_amdgcn_sdot8((int)w1, (int)x.y, v, false);
}

template <int CW>
__device__ __forceinline__ uint4 chunk_bytes(uint4 raw, int u) {
  if constexpr (CW == 8) return raw;
  else if constexpr (CW == 4) return u == 0 ? unpack4(raw.x, raw.y) : unpack4(raw.z, raw.w);
  else if constexpr (CW == 2) {
    const uint32_t w = u == 0 ? raw.x : u == 1 ? raw.y : u == 2 ? raw.z : raw.w;
    return unpack2(w);
  } else {
    const uint32_t w = (u >> 1) == 0 ? raw.x : (u >> 1) == 1 ? raw.y : (u >> 1) == 2 ? raw.z : raw.w;
    return unpack1((w >> (16 * (u & 1))) & 0xFFFFu);
  }
}

// Nibble words (elements 0-7, 8-15 in the 4-bit unit arrangement) of unit u.
template <int CW>
__device__ __forceinline__ uint2 chunk_nibbles(uint4 raw, int u) {
  if constexpr (CW == 4) {
    return u == 0 ? make_uint2(raw.x, raw.y) : make_uint2(raw.z, raw.w);
  } else {
    const uint32_t w = u == 0 ? raw.x : u == 1 ? raw.y : u == 2 ? raw.z : raw.w;
    return make_uint2(w & 0xCCCCCCCCu, (w << 2) & 0xCCCCCCCCu);
  }
}

template <int CW>
__device__ __forceinline__ int dpp_row_sum(int v) {
  // lanes of a 16-lane row with equal index mod 2*CW hold the same rows
  if constexpr (2 * CW <= 8) v += __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);
  if constexpr (2 * CW <= 4) v += __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false);
  if constexpr (2 * CW <= 2) v += __builtin_amdgcn_update_dpp(0, v, 0x122, 0xF, 0xF, false);
  return v;
}

// Batch row of flattened unit index u (rows of d units), M <= MT <= 8.
template <int MT>
__device__ __forceinline__ int gemv_row_of(int u, int d) {
  int m = 0;
#pragma unroll
  for (int j = 1; j < MT; ++j) m += u >= j * d ? 1 : 0;
  return m;
}

// Activation staging: rows 0..M-1 of block 0 of both groups go to LDS.
// For a nibble-path block (NIB): group 0 as packed 8-byte nibble units
// [m][q][kg], group 1 as bytes [m][q - ng0][kg] at nbase = M*ng0*32.
// Otherwise every unit as bytes [m][q][kg] (group 0 widened).  A unit is
// loaded as 16 bytes through a buffer resource over the activation buffer
// (group 0 units use the first half); indexes past the last unit read as
// zero.  A single row whose quantizer also left its contiguous image (the
// nibble-path layout itself) loads 16-byte pieces of that instead: a
// fraction of the cache lines the row's units are spread over.
template <int MT>
constexpr int gemv_xr() { return MT == 1 ? 2 : MT == 2 ? 3 : MT <= 4 ? 5 : 9; }

template <int MT, bool NIB>
__device__ __forceinline__ void gemv_store_x(const GemmArgs& a, int u0,
                                             const uint4 (&xl)[gemv_xr<MT>()], uint8_t* xs,
                                             int nbase) {
  const int d = a.wp.ngt * 4, d0 = a.ap.ng[0] * 4;
  const int total = (int)a.M * d;
#pragma unroll
  for (int i = 0; i < gemv_xr<MT>(); ++i) {
    const int u = u0 + i * 256 + (int)threadIdx.x;
    if (u < total) {
      const int m = gemv_row_of<MT>(u, d), rest = u - m * d;
      if (rest < d0 && NIB) {
        *reinterpret_cast<uint2*>(xs + m * d0 * 8 + rest * 8) = make_uint2(xl[i].x, xl[i].y);
      } else if (NIB) {
        *reinterpret_cast<uint4*>(xs + nbase + (m * (d - d0) + rest - d0) * 16) = xl[i];
      } else {
        const uint4 v = rest < d0 ? unpack4(xl[i].x, xl[i].y) : xl[i];
        *reinterpret_cast<uint4*>(xs + (m * d + rest) * 16) = v;
      }
    }
  }
}

// One output of a GEMV workgroup: physical column p, batch row m, fp32
// value v (what the epilogue rounds to bf16).  Y only where it is asked
// for; with a next layer (qn_img) also its code, by the quantizer of the
// column's next-layer group (or block, with sub-group scales), written at
// the column's planned position in the next layer's byte image.
__device__ __forceinline__ void gemv_store_out(const GemmArgs& a, int p, int64_t m, int n, float v) {
  if (a.Y) a.Y[m * a.ldy + n] = bf16_rne(v);
  if (a.qn_img) {
    const int qg = a.qn_tab[p];
    const int qpos = a.qn_tab[2 * a.wp.Np + p];
    QCol qc;
    if (a.qn_bs) {
      const bool g1 = qg >= a.qn_nsub0;
      qc.sc = a.qn_bs[qg];
      qc.rs = a.qn_brs[qg];
      qc.lo = g1 ? a.qn.lo[1] : a.qn.lo[0];
      qc.hi = g1 ? a.qn.hi[1] : a.qn.hi[0];
      qc.zp = 0;
      qc.sign1 = false;
    } else {
      // each field through readfirstlane, so the choice of group is a
      // select between registers (selecting the fields' addresses instead
      // made the compiler copy the kernel-argument quantizer to scratch in
      // every thread)
      const bool g1 = qg != 0;
      auto rf = [](float x) { return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x))); };
      auto ri = [](int x) { return __builtin_amdgcn_readfirstlane(x); };
      qc.sc = g1 ? rf(a.qn.s[1]) : rf(a.qn.s[0]);
      qc.rs = g1 ? rf(a.qn.rs[1]) : rf(a.qn.rs[0]);
      qc.lo = g1 ? rf(a.qn.lo[1]) : rf(a.qn.lo[0]);
      qc.hi = g1 ? rf(a.qn.hi[1]) : rf(a.qn.hi[0]);
      qc.zp = g1 ? ri(a.qn.zp[1]) : ri(a.qn.zp[0]);
      qc.sign1 = (g1 ? ri(a.qn.sign1[1]) : ri(a.qn.sign1[0])) != 0;
    }
    bool near;
    int c = qnext_fast(v, qc, near);
    if (near) c = qnext_exact(v, qc);
    if (qpos >= 0) a.qn_img[m * a.qn_ld + qpos] = (uint8_t)(int8_t)c;
  }
}

// FJ > 0 (batch of one row only): the fused form, which quantizes the fp32
// row itself (FJ float4 per thread) instead of staging packed units.
// GB: sub-group activation scales (zero points 0, no 1-bit weights): each
// slot's products are summed over the lanes of its rows and added into one
// exact int32 sum per activation block in LDS (after the staged rows), and
// the epilogue folds the blocks in order as the MFMA GEMM does.
template <int MT, int CW, bool NIB, int FJ = 0, bool GB = false>
__device__ __forceinline__ void gemv4_block(const GemmArgs& a, uint8_t* xs, int blk,
                                            int (&red)[4][4][kBlk][2][MT]) {
  static_assert(FJ == 0 || MT == 1, "the fused form takes one row");
  static_assert(!GB || (FJ == 0 && CW != 1), "block sums: no fused form, no sign-bit weights");
  constexpr int U = 8 / CW;
  constexpr int CPG = 8 * CW;    // chunks per granule
  constexpr int QS = 256 / CPG;  // granules per slot of the workgroup
  // load slots per batch for the two activation groups (sized so a 4096-
  // channel row with a dominant narrow group needs one batch)
  constexpr int NB0 = CW == 1 ? 2 : CW == 2 ? 4 : CW == 4 ? 8 : 8;
  constexpr int NB1 = CW == 1 ? 1 : CW == 2 ? 2 : CW == 4 ? 4 : 4;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const ActPlan& ap = a.ap;
  const int M = (int)a.M, ngt = a.wp.ngt, ng0 = ap.ng[0], ng1 = ngt - ng0;
  const int nbase = NIB ? M * ng0 * 32 : 0;
  const int nch0 = ng0 * CPG, nch1 = ng1 * CPG;
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.wd.packed + wblk_off(a.wp, blk)), (short)0, (nch0 + nch1) * 16, 0x00020000);
  const int t = tid & (CPG - 1);
  const int kg = (U * t) >> 4;
  const int q0 = tid / CPG;
  // Epilogue inputs of this thread's output (block row er, batch row em),
  // fetched together with the first loads rather than after the reduction.
  const int er = tid & (kBlk - 1), em = tid >> 4;
  const int ep = blk * kBlk + er;
  const ColInfo eci = a.wd.colinfo[ep];
  const uint8_t eshw = a.wd.shw[ep];
  float sa0 = 0.0f, sa1 = 0.0f;
  if constexpr (FJ == 0) {
    sa0 = a.s_a[0];
    sa1 = ap.S == 2 ? a.s_a[1] : 0.0f;
  }

  int acc0[U][MT], acc1[U][MT];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) acc0[u][mm] = acc1[u][mm] = 0;

  // Group-0 slot b of batch i holds chunk tid + 256*(i*NB0 + b), group-1
  // slot b of batch i chunk tid + 256*(i*NB1 + b) past the group-0 chunks.
  auto issue0 = [&](int s0, uint4 (&raw)[NB0]) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < NB0; ++b) {
      const int c = tid + 256 * (s0 + b);
      raw[b] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                             wr, c < nch0 ? (uint32_t)c * 16 : kOOB, 0, 0));
    }
  };
  auto issue1 = [&](int s0, uint4 (&raw)[NB1]) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < NB1; ++b) {
      const int c = tid + 256 * (s0 + b);
      raw[b] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                             wr, c < nch1 ? (uint32_t)(nch0 + c) * 16 : kOOB, 0, 0));
    }
  };
  // Byte-path products of one chunk (zero chunks add nothing; 1-bit
  // chunks, whose zero bits decode to +1, are masked).
  auto bytes_into = [&](int (&acc)[U][MT], uint4 raw, int xq, bool ok) __attribute__((always_inline)) {
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) {
      if (mm < M) {
        // NIB blocks read group 1 only, staged from granule ng0 on
        const uint4 x = *reinterpret_cast<const uint4*>(
            NIB ? xs + nbase + (mm * (ngt - ng0) + xq - ng0) * 64 + kg * 16
                : xs + (mm * ngt + xq) * 64 + kg * 16);
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int v = dot16(chunk_bytes<CW>(raw, u), x, 0);
          acc[u][mm] += (CW != 1 || ok) ? v : 0;
        }
      }
    }
  };
  // GB: exact per-block sums in LDS, [block][batch row][block row]
  int* gacc = reinterpret_cast<int*>(xs + a.xs_bytes);
  const int gl16 = lane & 15;
  auto gadd = [&](int j, int (&v)[U][MT]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) v[u][mm] = dpp_row_sum<CW>(v[u][mm]);
    if (gl16 < 2 * CW) {
#pragma unroll
      for (int mm = 0; mm < MT; ++mm)
        if (mm < M)
#pragma unroll
          for (int u = 0; u < U; ++u) atomicAdd(&gacc[(j * MT + mm) * kBlk + U * gl16 + u], v[u][mm]);
    }
  };
  auto consume0 = [&](int s0, const uint4 (&raw)[NB0]) __attribute__((always_inline)) {
    if constexpr (GB) {
      // one slot's granule lies in one block; a 16-lane row of lanes never
      // spans two granules (CW >= 2)
      const int gpg = ap.gsub[0];
#pragma unroll
      for (int b = 0; b < NB0; ++b) {
        if (256 * (s0 + b) >= nch0) break;  // the same for the whole workgroup
        const int q = q0 + QS * (s0 + b);
        int v[U][MT];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int mm = 0; mm < MT; ++mm) v[u][mm] = 0;
        if constexpr (NIB) {
#pragma unroll
          for (int mm = 0; mm < MT; ++mm) {
            if (mm < M) {
              const uint2 xq = *reinterpret_cast<const uint2*>(
                  xs + (mm * ng0 + min(q, ng0 - 1)) * 32 + kg * 8);
#pragma unroll
              for (int u = 0; u < U; ++u) {
                const uint2 w = chunk_nibbles<CW>(raw[b], u);
                v[u][mm] = dot16n(w.x, w.y, xq, 0);
              }
            }
          }
        } else {
          bytes_into(v, raw[b], min(q, ng0 - 1), true);
        }
        if (q < ng0) gadd(q / gpg, v);
      }
      return;
    }
    if constexpr (NIB) {
      // every slot's staged activations first (one LDS round trip), then
      // the products slot by slot as the chunks land
      uint2 xv[NB0][MT];
#pragma unroll
      for (int b = 0; b < NB0; ++b) {
        const int q = min(q0 + QS * (s0 + b), ng0 - 1);
#pragma unroll
        for (int mm = 0; mm < MT; ++mm)
          xv[b][mm] = *reinterpret_cast<const uint2*>(xs + (min(mm, M - 1) * ng0 + q) * 32 + kg * 8);
      }
#pragma unroll
      for (int b = 0; b < NB0; ++b) {
        if (256 * (s0 + b) >= nch0) break;  // the same for the whole workgroup
#pragma unroll
        for (int mm = 0; mm < MT; ++mm) {
          if (mm < M) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
              const uint2 w = chunk_nibbles<CW>(raw[b], u);
              acc0[u][mm] = dot16n(w.x, w.y, xv[b][mm], acc0[u][mm]);
            }
          }
        }
      }
    } else {
#pragma unroll
      for (int b = 0; b < NB0; ++b) {
        if (256 * (s0 + b) >= nch0) break;  // the same for the whole workgroup
        bytes_into(acc0, raw[b], min(q0 + QS * (s0 + b), ng0 - 1), tid + 256 * (s0 + b) < nch0);
      }
    }
  };
  auto consume1 = [&](int s0, const uint4 (&raw)[NB1]) __attribute__((always_inline)) {
    if constexpr (GB) {
      const int gpg = ap.gsub[1];
#pragma unroll
      for (int b = 0; b < NB1; ++b) {
        if (256 * (s0 + b) >= nch1) break;  // the same for the whole workgroup
        const int q = q0 + QS * (s0 + b);
        int v[U][MT];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int mm = 0; mm < MT; ++mm) v[u][mm] = 0;
        bytes_into(v, raw[b], ng0 + min(q, ng1 - 1), true);
        if (q < ng1) gadd(ap.nsub[0] + q / gpg, v);
      }
      return;
    }
#pragma unroll
    for (int b = 0; b < NB1; ++b) {
      if (256 * (s0 + b) >= nch1) break;  // the same for the whole workgroup
      bytes_into(acc1, raw[b], ng0 + min(q0 + QS * (s0 + b), ng1 - 1), tid + 256 * (s0 + b) < nch1);
    }
  };

  // The activation loads go first (they hit L2), then the first batch of
  // both groups' chunks; staging waits only for the former.
  if constexpr (FJ > 0) {
    // Fused: the row's float4 and planned positions first, then the
    // chunks; the group maxima (every workgroup computes the same ones
    // from the same row), codes and staged units are done while the chunks
    // are in flight (fence-free barriers), with the arithmetic of the
    // one-row quantizer, so the codes are those of soniq_quantize_act.
    const int K4 = a.K4, kp0 = ap.kpad[0];
    float4 v[FJ];
    int4 p[FJ];
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int k4 = min(tid + 256 * j, K4 - 1);  // repeats change no max
      const uint2 pq = reinterpret_cast<const uint2*>(a.apos16)[k4];  // half the bytes of int32
      p[j] = make_int4((int)(pq.x & 0xFFFFu), (int)(pq.x >> 16), (int)(pq.y & 0xFFFFu), (int)(pq.y >> 16));
      v[j] = reinterpret_cast<const float4*>(a.a32)[k4];
    }
    uint4 raw0[NB0], raw1[NB1];
    issue0(0, raw0);
    issue1(0, raw1);
    uint8_t* codes = xs + a.xs_bytes;
    uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
    for (int i = tid; i < ap.Kp / 4; i += 256) codes32[i] = 0;
    float mx0 = 0.0f, mx1 = 0.0f;
#pragma unroll
    for (int j = 0; j < FJ; ++j)
      max4(v[j], make_uchar4(p[j].x >= kp0, p[j].y >= kp0, p[j].z >= kp0, p[j].w >= kp0), mx0, mx1);
    const float2 mm = block_max2_nofence(make_float2(mx0, mx1),
                                         reinterpret_cast<float*>(&red[0][0][0][0][0]));
    const float s0 = group_scale(mm.x, ap.q[0]);
    const float s1 = ap.S == 2 ? group_scale(mm.y, ap.q[1]) : 0.0f;
    sa0 = s0;
    sa1 = s1;
    if (blk == 0 && tid == 0) {
      a.s_a_out[0] = s0;
      a.s_a_out[1] = s1;
    }
    const QPair q = qpair(qelem(s0, ap.q[0], ap.zp[0]), qelem(s1, ap.q[1], ap.zp[1]));
#pragma unroll
    for (int j = 0; j < FJ; ++j)
      if (tid + 256 * j < K4) {
        const bool h[4] = {p[j].x >= kp0, p[j].y >= kp0, p[j].z >= kp0, p[j].w >= kp0};
        qstore4g(v[j], h, q, codes, p[j]);
      }
    __builtin_amdgcn_s_waitcnt(SONIQ_LGKMCNT0_IMM);
    bar_nofence();
    // unit u = planned positions 16u .. 16u + 15 (granule u / 4, group u % 4
    // of 16), staged as gemv_store_x stages the packed unit
    for (int u = tid; u < 4 * ngt; u += 256) {
      const uint4 d = *reinterpret_cast<const uint4*>(codes + 16 * u);
      const bool g0 = u < 4 * ng0;
      const uint4 pk = pack_unit(d.x, d.y, d.z, d.w, 4);
      if constexpr (NIB) {
        if (g0) *reinterpret_cast<uint2*>(xs + 8 * u) = make_uint2(pk.x, pk.y);
        else *reinterpret_cast<uint4*>(xs + nbase + 16 * (u - 4 * ng0)) = d;
      } else {
        *reinterpret_cast<uint4*>(xs + 16 * u) = g0 ? unpack4(pk.x, pk.y) : d;
      }
    }
    // the handle's packed row and scales, as soniq_quantize_act leaves them
    if (blk == 0) write_act_units(codes, 1, 0, ap, a.act_out, a.ximg);
    __builtin_amdgcn_s_waitcnt(SONIQ_LGKMCNT0_IMM);
    bar_nofence();
    consume0(0, raw0);
    if (nch1 > 0) consume1(0, raw1);
  } else {
    // A single row with its contiguous image (cx): 16-byte pieces of it, as
    // many as the row's units take at 8 (group 0) and 16 bytes (group 1).
    // Otherwise the units of the batch's rows from the packed buffer.
    const bool cx = MT == 1 && a.ximg != nullptr;
    const int total_x = cx ? 2 * ng0 + 4 * ng1 : M * ngt * 4;
    const __amdgpu_buffer_rsrc_t xr =
        cx ? __builtin_amdgcn_make_buffer_rsrc((void*)a.ximg, (short)0, total_x * 16, 0x00020000)
           : __builtin_amdgcn_make_buffer_rsrc(
                 (void*)a.act, (short)0,
                 (int)(ap.S == 2 ? ap.seg_off[1] + ap.mblk_bytes[1]
                                 : ap.seg_off[0] + ap.mblk_bytes[0]),
                 0x00020000);
    uint4 xl[gemv_xr<MT>()];
    // one load per piece whichever the source (loads on both sides of a
    // branch would be joined by copies that wait for them)
    const int d = ngt * 4, d0 = ng0 * 4;
    const uint32_t o0 = (uint32_t)ap.seg_off[0], o1 = (uint32_t)ap.seg_off[1];
    auto load_x = [&](int u0) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < gemv_xr<MT>(); ++i) {
        const int u = u0 + i * 256 + tid;
        uint32_t off = (uint32_t)u * 16;
        if (!cx) {
          // unit rest = 4q + kg of row m: at rest*128 + 8m (4-bit group) or
          // (rest - 4*ng0)*256 + 16m (byte group) from the group's base
          const int m = gemv_row_of<MT>(u, d), rest = u - m * d;
          off = rest < d0 ? o0 + (uint32_t)(rest * 128 + m * 8)
                          : o1 + (uint32_t)((rest - d0) * 256 + m * 16);
        }
        xl[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                              xr, u < total_x ? off : kOOB, 0, 0));
      }
    };
    // the image is the staged layout of a nibble-path block; other blocks
    // widen group 0's units to bytes
    auto store_x = [&](int u0) __attribute__((always_inline)) {
      if (cx) {
#pragma unroll
        for (int i = 0; i < gemv_xr<MT>(); ++i) {
          const int c = u0 + i * 256 + tid;
          if (c < total_x) {
            if (NIB) {
              *reinterpret_cast<uint4*>(xs + 16 * c) = xl[i];
            } else if (c < 2 * ng0) {
              *reinterpret_cast<uint4*>(xs + 32 * c) = unpack4(xl[i].x, xl[i].y);
              *reinterpret_cast<uint4*>(xs + 32 * c + 16) = unpack4(xl[i].z, xl[i].w);
            } else {
              *reinterpret_cast<uint4*>(xs + 16 * (c + 2 * ng0)) = xl[i];
            }
          }
        }
      } else {
        gemv_store_x<MT, NIB>(a, u0, xl, xs, nbase);
      }
    };
    load_x(0);
    uint4 raw0[NB0], raw1[NB1];
    const bool more_x = total_x > 256 * gemv_xr<MT>();
    if (more_x) {
      // rows too long for one round: stage them all before the chunk loads
      // (waits inside the staging loop would otherwise drain the chunks)
      store_x(0);
      for (int u0 = 256 * gemv_xr<MT>(); u0 < total_x; u0 += 256 * gemv_xr<MT>()) {
        load_x(u0);
        store_x(u0);
      }
    }
    // one place for the chunk loads: their registers need no copies at a join
    issue0(0, raw0);
    issue1(0, raw1);
    if (!more_x) store_x(0);
    if constexpr (GB) {
      const int nsub = ap.nsub[0] + (ap.S == 2 ? ap.nsub[1] : 0);
      for (int i = tid; i < nsub * MT * kBlk; i += 256) gacc[i] = 0;
    }
    // The staged rows must be visible to every wave, but the weight chunks
    // may still be in flight: wait for LDS writes only, then a plain
    // barrier (a full __syncthreads would also drain every chunk load).
    __builtin_amdgcn_s_waitcnt(SONIQ_LGKMCNT0_IMM);
    bar_nofence();
    consume0(0, raw0);
    if (nch1 > 0) consume1(0, raw1);
  }
  for (int s0 = NB0; 256 * s0 < nch0; s0 += NB0) {
    uint4 raw[NB0];
    issue0(s0, raw);
    consume0(s0, raw);
  }
  for (int s0 = NB1; 256 * s0 < nch1; s0 += NB1) {
    uint4 raw[NB1];
    issue1(s0, raw);
    consume1(s0, raw);
  }

  if constexpr (GB) {
    // every block sum is in LDS: fold the blocks in order, multiply then
    // add (y = sum_j f(ACC_j) * s_a[j]), then scale by s_w
    __syncthreads();
    if (tid < kBlk * M && eci.n >= 0) {
      const int nsub0 = ap.nsub[0], nsub = nsub0 + (ap.S == 2 ? ap.nsub[1] : 0);
      const int shb0 = NIB ? (CW == 2 ? 2 : 0) : ap.sh[0] + (eshw & 0x7F);
      const int shb1 = ap.sh[1] + (eshw & 0x7F);
      float y = 0.0f;
      for (int j = 0; j < nsub; ++j) {
        const int t = gacc[(j * MT + em) * kBlk + er] >> (j < nsub0 ? shb0 : shb1);
        y = __fadd_rn(y, __fmul_rn((float)t, a.s_a[j]));
        if (a.acc) a.acc[((int64_t)j * a.M + em) * a.N + eci.n] = t;
      }
      gemv_store_out(a, ep, em, eci.n, __fmul_rn(y, eci.s_w));
    }
    return;
  }
  // Within each 16-lane row, then rows and waves through LDS.
  const int row16 = lane >> 4, l16 = lane & 15;
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) {
      acc0[u][mm] = dpp_row_sum<CW>(acc0[u][mm]);
      acc1[u][mm] = dpp_row_sum<CW>(acc1[u][mm]);
    }
  if (l16 < 2 * CW) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm) {
        red[wid][row16][U * l16 + u][0][mm] = acc0[u][mm];
        red[wid][row16][U * l16 + u][1][mm] = acc1[u][mm];
      }
  }
  __syncthreads();
  if (tid < kBlk * M && eci.n >= 0) {
    int s0 = 0, s1 = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        s0 += red[w][h][er][0][em];
        s1 += red[w][h][er][1][em];
      }
    const int S = ap.S;
    // group 0 sums are in units of 2^2 (2-bit nibbles) or 1 on the nibble
    // path; byte-path sums carry both unpack scales
    const int t0 = NIB ? (s0 >> (CW == 2 ? 2 : 0)) + ap.zp[0] * eci.colsum[0]
                       : true_acc(s0, ap.sh[0], ap.c[0], ap.padcnt[0], ap.zp[0], eshw, eci.colsum[0]);
    const int t1 = S == 2 ? true_acc(s1, ap.sh[1], ap.c[1], ap.padcnt[1], ap.zp[1], eshw, eci.colsum[1])
                          : 0;
    gemv_store_out(a, ep, em, eci.n, epilogue(t0, t1, S, sa0, sa1, eci.s_w));
    if (a.acc) {
      a.acc[(int64_t)em * a.N + eci.n] = t0;
      if (S == 2) a.acc[(a.M + em) * a.N + eci.n] = t1;
    }
  }
}

// Dynamic LDS: the staged rows (see gemv_lds).
template <int MT>
__global__ __launch_bounds__(256) void k_gemv(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];
  __shared__ int red[4][4][kBlk][2][MT];
  const int blk = blockIdx.x;
  const int c = wblk_c(a.wp, blk);
  if (c == 2) gemv4_block<MT, 2, true>(a, xs, blk, red);
  else if (c == 4) gemv4_block<MT, 4, true>(a, xs, blk, red);
  else if (c == 8) gemv4_block<MT, 8, false>(a, xs, blk, red);
  // 1-bit blocks keep eight row accumulators per lane and batch row; the
  // host sends them here only for batches of at most 4 rows, so larger
  // instances are compiled without that path (and its registers)
  else if constexpr (MT <= 4) gemv4_block<MT, 1, false>(a, xs, blk, red);
}


// Batches of at most 8 rows whose activations have sub-group scales: the
// GEMV with one exact int32 sum per activation block.  Dynamic LDS: the
// staged rows (xs_bytes), then the block sums [nsub][MT][16].
template <int MT>
__global__ __launch_bounds__(256) void k_gemv_g(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];
  __shared__ int red[4][4][kBlk][2][MT];
  const int blk = blockIdx.x;
  const int c = wblk_c(a.wp, blk);
  if (c == 2) gemv4_block<MT, 2, true, 0, true>(a, xs, blk, red);
  else if (c == 4) gemv4_block<MT, 4, true, 0, true>(a, xs, blk, red);
  else gemv4_block<MT, 8, false, 0, true>(a, xs, blk, red);
}

// Batch of one row, quantized inside the GEMV: every workgroup computes
// the row's group maxima and codes (J float4 per thread) while its weight
// chunks stream in; workgroup 0 also leaves the packed row, its image and
// the scales in the handle.  Dynamic LDS: the staged row (xs_bytes), then
// Kp code bytes.
template <int J>
__global__ __launch_bounds__(256) void k_gemv_fused(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];
  __shared__ int red[4][4][kBlk][2][1];
  const int blk = blockIdx.x;
  const int c = wblk_c(a.wp, blk);
  if (c == 2) gemv4_block<1, 2, true, J>(a, xs, blk, red);
  else if (c == 4) gemv4_block<1, 4, true, J>(a, xs, blk, red);
  else if (c == 8) gemv4_block<1, 8, false, J>(a, xs, blk, red);
  else gemv4_block<1, 1, false, J>(a, xs, blk, red);
}

// ----------------------------------------------------------- k_gemv_mfma --
// Batches of 2..8 rows with activation containers 4 (group 0) and 8
// (group 1): one workgroup per 16-row weight block, as in k_gemv, but the
// products run on v_mfma_i32_16x16x64_i8 with the batch rows as the A
// operand (rows past M are never read out) and the block's 16 weight rows
// as B.  The block's bytes go global -> LDS in 16-byte chunks, all in
// flight at once; both buffers are fragment-major, so lane l reads unit l
// of a granule as its operand (the activations straight from global
// memory, where every workgroup finds them in L2).  Wave w takes granules
// w, w + 4, ... of each group in batches of kMB; the four partial 16x16
// sums per group meet in LDS and the block's 16 columns get the GEMM's
// exact epilogue.  Dynamic LDS: the largest block (ngt * 128 * c_hi bytes)
// rounded up to 1 KB.
constexpr int kMB = 4;

template <int CW>
__device__ __forceinline__ void gemv_mfma_block(const GemmArgs& a, int blk, uint8_t* wl,
                                                int (&red)[4][2][4][64]) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const ActPlan& ap = a.ap;
  const int ngt = a.wp.ngt, ng0 = ap.ng[0], ng1 = ngt - ng0;
  {
    const int nch = ngt * 8 * CW;  // 16-byte chunks of the block
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.wd.packed + wblk_off(a.wp, blk)), (short)0, nch * 16, 0x00020000);
    const uint32_t base = lds_off(wl);
    // a wave's 64 chunks land at base + 16 * (256i + 64 wid + lane); waves
    // wholly past the block skip, the last partial one writes zeros up to
    // the next 64-chunk boundary (the allocation covers it)
    for (int i = 0; 256 * i < nch; ++i) {
      const int ch = 256 * i + tid;
      if (256 * i + 64 * wid < nch)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            wr, (__attribute__((address_space(3))) void*)(uintptr_t)(base + (256 * i + 64 * wid) * 16),
            16, ch < nch ? (uint32_t)ch * 16 : kOOB, 0, 0, 0);
    }
  }
  const uint8_t* x0 = a.act + ap.seg_off[0] + lane * 8;
  const uint8_t* x1 = a.act + (ap.S == 2 ? ap.seg_off[1] : 0) + lane * 16;
  // epilogue inputs, requested before the stream lands
  const int pc = blk * kBlk + (lane & 15);
  const ColInfo ci = a.wd.colinfo[pc];
  const uint8_t shw = a.wd.shw[pc];
  const float sa0 = a.s_a[0], sa1 = ap.S == 2 ? a.s_a[1] : 0.0f;
  wait_vm<0>();
  __syncthreads();

  auto wunit = [&](int q) __attribute__((always_inline)) {
    uint4 r = make_uint4(0u, 0u, 0u, 0u);
    const uint8_t* p = wl + (q * 64 + lane) * 2 * CW;
    if constexpr (CW == 8) r = *reinterpret_cast<const uint4*>(p);
    else if constexpr (CW == 4) { const uint2 v = *reinterpret_cast<const uint2*>(p); r.x = v.x; r.y = v.y; }
    else if constexpr (CW == 2) r.x = *reinterpret_cast<const uint32_t*>(p);
    else r.x = *reinterpret_cast<const uint16_t*>(p);
    return r;
  };
  v4i acc0 = v4i{0, 0, 0, 0}, acc1 = v4i{0, 0, 0, 0};
  for (int q = wid; q < ng0; q += 4 * kMB) {
    uint2 xa[kMB];
#pragma unroll
    for (int i = 0; i < kMB; ++i) xa[i] = *reinterpret_cast<const uint2*>(x0 + min(q + 4 * i, ng0 - 1) * 512);
#pragma unroll
    for (int i = 0; i < kMB; ++i)
      if (q + 4 * i < ng0)
        acc0 = __builtin_amdgcn_mfma_i32_16x16x64_i8(frag_of(unpack4(xa[i].x, xa[i].y)),
                                                     frag_of(unpack_unit<CW>(wunit(q + 4 * i))),
                                                     acc0, 0, 0, 0);
  }
  for (int q = wid; q < ng1; q += 4 * kMB) {
    uint4 xa[kMB];
#pragma unroll
    for (int i = 0; i < kMB; ++i) xa[i] = *reinterpret_cast<const uint4*>(x1 + min(q + 4 * i, ng1 - 1) * 1024);
#pragma unroll
    for (int i = 0; i < kMB; ++i)
      if (q + 4 * i < ng1)
        acc1 = __builtin_amdgcn_mfma_i32_16x16x64_i8(frag_of(xa[i]),
                                                     frag_of(unpack_unit<CW>(wunit(ng0 + q + 4 * i))),
                                                     acc1, 0, 0, 0);
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    red[wid][0][e][lane] = acc0[e];
    red[wid][1][e][lane] = acc1[e];
  }
  __syncthreads();
  if (wid == 0 && ci.n >= 0) {
    const int sh0 = ap.sh[0] + (shw & 0x7F), sh1 = ap.sh[1] + (shw & 0x7F);
    const int add0 = ap.zp[0] * ci.colsum[0], add1 = ap.zp[1] * ci.colsum[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = (lane >> 4) * 4 + e;  // batch row of this lane's sum e
      if (m < a.M) {
        const int r0 = red[0][0][e][lane] + red[1][0][e][lane] + red[2][0][e][lane] + red[3][0][e][lane];
        const int r1 = red[0][1][e][lane] + red[1][1][e][lane] + red[2][1][e][lane] + red[3][1][e][lane];
        const int t0 = (r0 >> sh0) + add0;
        const int t1 = ap.S == 2 ? (r1 >> sh1) + add1 : 0;
        gemv_store_out(a, pc, m, ci.n, epilogue(t0, t1, ap.S, sa0, sa1, ci.s_w));
        if (a.acc) {
          a.acc[(int64_t)m * a.N + ci.n] = t0;
          if (ap.S == 2) a.acc[(a.M + m) * a.N + ci.n] = t1;
        }
      }
    }
  }
}

__global__ __launch_bounds__(256) void k_gemv_mfma(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t wl[];
  __shared__ int red[4][2][4][64];
  const int blk = blockIdx.x;
  const int c = wblk_c(a.wp, blk);
  if (c == 2) gemv_mfma_block<2>(a, blk, wl, red);
  else if (c == 4) gemv_mfma_block<4>(a, blk, wl, red);
  else if (c == 8) gemv_mfma_block<8>(a, blk, wl, red);
  else gemv_mfma_block<1>(a, blk, wl, red);
}

// ------------------------------------------------- single-pass quantize --
// Batches of at least kCoopMinElems elements whose rows fit the registers
// of one resident grid take k_act_coop: RB rows per workgroup (4, 8 or 16,
// the choice wasting the fewest register slots), T float4 per thread, and
// at most as many workgroups as can be resident at once (by the occupancy
// of k_act_coop<T> with this LDS size, times the CU count).
// SONIQ_ACT_COOP=0 turns the path off for measurement; results do not
// depend on it.
constexpr int64_t kCoopMinElems = (int64_t)1 << 20;

template <int T, int TL, bool GRP>
int coop_capacity(size_t lds) {
  // resident workgroups per CU for this T and LDS size, cached per device
  struct Entry {
    int dev = -1;
    size_t lds = 0;
    int per_cu = 0, cus = 0;
  };
  static thread_local Entry cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (cache.dev != dev || cache.lds != lds) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_act_coop<T, TL, GRP>, 256, lds) != hipSuccess)
      return 0;
    cache.dev = dev;
    cache.lds = lds;
    cache.per_cu = per_cu;
    cache.cus = cus;
  }
  return cache.per_cu * cache.cus;
}

template <int T, int TL, bool GRP>
bool coop_launch(const float* A, int64_t M, int64_t K, int64_t lda, int RB, const ActPlan& ap,
                 const int32_t* pos_dev, unsigned* bar, float* s_a,
                 uint8_t* packed, hipStream_t stream, hipError_t& e) {
  const int nsub = GRP ? ap.nsub[0] + (ap.S == 2 ? ap.nsub[1] : 0) : 0;
  const size_t lds = (size_t)RB * ap.Kp + 16 * (size_t)((K / 4 + 63) / 64 * 64) + 4096 * TL +
                     (size_t)(12 * nsub + 15) / 16 * 16;
  const int64_t blocks = (M + RB - 1) / RB;
  // a workgroup's rows are addressed with 32-bit byte offsets
  if ((int64_t)(RB - 1) * lda * 4 + K * 4 >= ((int64_t)1 << 31)) return false;
  if (lds > 64 * 1024 || blocks > coop_capacity<T, TL, GRP>(lds)) return false;
  unsigned spins = kBarrierSpins;
  if (const char* env = getenv("SONIQ_COOP_SPINS")) spins = (unsigned)strtoul(env, nullptr, 10);
  hipLaunchKernelGGL((k_act_coop<T, TL, GRP>), dim3((unsigned)blocks), dim3(256), lds, stream, A, M,
                     (int)(K / 4), lda, RB, pos_dev, ap, bar, spins, s_a, packed);
  e = hipGetLastError();
  return true;
}

// grp: sub-group scales (pos_dev then holds position | block << 16).
bool launch_act_coop(const float* A, int64_t M, int64_t K, int64_t lda, const ActPlan& ap,
                     const int32_t* pos_dev, unsigned* bar, float* s_a,
                     uint8_t* packed, hipStream_t stream, hipError_t& e, bool grp = false) {
  if (const char* env = getenv("SONIQ_ACT_COOP"))
    if (atoi(env) == 0) return false;
  const int64_t K4 = K / 4;
  // candidates (RB, T) ordered by wasted register slots, more workgroups
  // first (they spread the quantize work more evenly over the CUs)
  struct Cand {
    int rb, t;
    int64_t waste;
  } cand[3];
  int nc = 0;
  for (int rb : {4, 8, 16}) {
    const int64_t need = (rb * K4 + 255) / 256;
    const int t = need <= 6 ? 6 : need <= 9 ? 9 : need <= 12 ? 12 : need <= 18 ? 18 : 0;
    if (t == 0) continue;
    cand[nc++] = {rb, t, 256 * (int64_t)t - rb * K4};
  }
  for (int i = 1; i < nc; ++i)
    for (int j = i; j > 0 && cand[j].waste < cand[j - 1].waste; --j) std::swap(cand[j], cand[j - 1]);
  for (int i = 0; i < nc; ++i) {
    const Cand& c = cand[i];
    bool done = false;
#define SONIQ_COOP(T_, TL_)                                                                         \
  (grp ? coop_launch<T_, TL_, true>(A, M, K, lda, c.rb, ap, pos_dev, bar, s_a, packed, stream, e)  \
       : coop_launch<T_, TL_, false>(A, M, K, lda, c.rb, ap, pos_dev, bar, s_a, packed, stream, e))
    if (c.t == 6) done = SONIQ_COOP(6, 0);
    else if (c.t == 9) done = SONIQ_COOP(9, 1);
    else if (c.t == 12) done = SONIQ_COOP(12, 0);
    else done = SONIQ_COOP(18, 0);
#undef SONIQ_COOP
    if (done) return true;
  }
  return false;
}

// Static scales of a next layer with sub-group blocks, passed by value (so
// that a captured launch carries them): the handle's s_a and the
// reciprocals the GEMM's epilogue uses (0 outside the shortcut's range).
struct BlockScales {
  float s[kGSubMax];
  int n;
};

__global__ __launch_bounds__(256) void k_set_scales(BlockScales b, float* __restrict__ s_a,
                                                    float* __restrict__ brs) {
  for (int j = threadIdx.x; j < b.n; j += 256) {
    const float sc = b.s[j];
    s_a[j] = sc;
    brs[j] = (sc >= 0x1p-100f && sc <= 0x1p100f) ? __fdiv_rn(1.0f, sc) : 0.0f;
  }
}

// ------------------------------------------------------------ k_pack_img --
// The next layer's packed rows from the byte image the producer's epilogue
// wrote (stored codes; padding positions stay 0): in 16-row blocks of
// 16-byte columns (row m, position p at img[(m/16)*ld + 16*p + m%16]) from
// the GEMM tiles, row-major (img[m*ld + p]) from the GEMV forms.

// Positions [p0, p0 + 4*n4) of a 16-row block of the blocked image into LDS
// as rows of pitch 4*n4: thread = four positions, 16 rows each (16-byte
// loads), turned into four-position words of each row by byte permutes.
__device__ __forceinline__ void img_block_rows(const uint8_t* __restrict__ blk, int p0, int n4,
                                               uint8_t* codes) {
  const uint4* src = reinterpret_cast<const uint4*>(blk) + p0;
  for (int p4 = threadIdx.x; p4 < n4; p4 += 256) {
    uint4 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = src[4 * p4 + j];
    const uint32_t w[4][4] = {{v[0].x, v[0].y, v[0].z, v[0].w}, {v[1].x, v[1].y, v[1].z, v[1].w},
                              {v[2].x, v[2].y, v[2].z, v[2].w}, {v[3].x, v[3].y, v[3].z, v[3].w}};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      // rows 4q .. 4q+3: bytes of positions 0,1 (x01) and 2,3 (x23)
      const uint32_t x01lo = __builtin_amdgcn_perm(w[1][q], w[0][q], 0x05010400u);
      const uint32_t x01hi = __builtin_amdgcn_perm(w[1][q], w[0][q], 0x07030602u);
      const uint32_t x23lo = __builtin_amdgcn_perm(w[3][q], w[2][q], 0x05010400u);
      const uint32_t x23hi = __builtin_amdgcn_perm(w[3][q], w[2][q], 0x07030602u);
      uint32_t* c32 = reinterpret_cast<uint32_t*>(codes) + p4;
      c32[(4 * q + 0) * n4] = __builtin_amdgcn_perm(x23lo, x01lo, 0x05040100u);
      c32[(4 * q + 1) * n4] = __builtin_amdgcn_perm(x23lo, x01lo, 0x07060302u);
      c32[(4 * q + 2) * n4] = __builtin_amdgcn_perm(x23hi, x01hi, 0x05040100u);
      c32[(4 * q + 3) * n4] = __builtin_amdgcn_perm(x23hi, x01hi, 0x07060302u);
    }
  }
}

// Full 16-row blocks of the blocked image, no 1-bit group: workgroup
// (b, j) packs granules [j*ngr/P, (j+1)*ngr/P) of block b (P = gridDim.y),
// so a batch's blocks spread over about a thousand workgroups.  Workgroup
// (0, 0) also stores the static scales.  Dynamic LDS: 16 * 64 *
// ceil(ngr/P) bytes.
__global__ __launch_bounds__(256) void k_pack_img_split(const uint8_t* __restrict__ img, int64_t ld,
                                                        ActPlan ap, float s0, float s1,
                                                        float* __restrict__ s_a,
                                                        uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  const int64_t b = blockIdx.x;
  const int ngr = ap.Kp / kGran;
  const int q0 = (int)((int64_t)blockIdx.y * ngr / gridDim.y);
  const int q1 = (int)((int64_t)(blockIdx.y + 1) * ngr / gridDim.y);
  if (s_a && b == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
    s_a[0] = s0;
    s_a[1] = s1;
  }
  if (q1 <= q0) return;
  const int W = (q1 - q0) * kGran;
  img_block_rows(img + b * ld, q0 * kGran, W / 4, codes);
  __syncthreads();
  for (int gi = 0; gi < ap.S; ++gi) {
    const int c = gi ? ap.c[1] : ap.c[0];
    const int gs = gi ? ap.ng[0] : 0;  // the group's first granule
    const int g0 = max(q0, gs), g1 = min(q1, gs + (gi ? ap.ng[1] : ap.ng[0]));
    if (g1 <= g0) continue;
    uint8_t* dst = packed + (gi ? ap.seg_off[1] : ap.seg_off[0]) +
                   b * (gi ? ap.mblk_bytes[1] : ap.mblk_bytes[0]) + (int64_t)(g0 - gs) * 128 * c;
    const int lb = (g0 - q0) * kGran;
    if (c == 8) write_block_pieces<8, kBlk>(codes, W, lb, g1 - g0, 0, dst);
    else if (c == 4) write_block_pieces<4, kBlk>(codes, W, lb, g1 - g0, 0, dst);
    else write_block_pieces<2, kBlk>(codes, W, lb, g1 - g0, 0, dst);
  }
}

// Every other case (the GEMV forms' row-major image, a 1-bit group, the
// last block of a batch): R rows per workgroup from block row blk0*R on go
// to LDS as rows of planned positions and out as units.  Workgroup 0 also
// stores the static scales (when s_a is set).  Dynamic LDS: R*Kp bytes.
template <int R>
__global__ __launch_bounds__(256) void k_pack_img(const uint8_t* __restrict__ img, int64_t ld,
                                                  bool blocked, int64_t blk0, int64_t M, ActPlan ap,
                                                  float s0, float s1, float* __restrict__ s_a,
                                                  uint8_t* __restrict__ packed,
                                                  uint8_t* __restrict__ ximg) {
  extern __shared__ __align__(16) uint8_t codes[];
  const int64_t m0 = (blk0 + blockIdx.x) * R;
  const int rows = (int)min((int64_t)R, M - m0);
  if (!blocked) {
    for (int r = 0; r < rows; ++r) {
      const uint4* src = reinterpret_cast<const uint4*>(img + (m0 + r) * ld);
      for (int i = threadIdx.x; i < ap.Kp / 16; i += 256)
        reinterpret_cast<uint4*>(codes + r * ap.Kp)[i] = src[i];
    }
  } else if (R == kBlk && rows == kBlk) {
    img_block_rows(img + (m0 / kBlk) * ld, 0, ap.Kp / 4, codes);
  } else {
    // the last block of a batch, or one row: only its rows' bytes
    const uint8_t* blk = img + (m0 / kBlk) * ld + m0 % kBlk;
    for (int r = 0; r < rows; ++r)
      for (int p = threadIdx.x; p < ap.Kp; p += 256) codes[r * ap.Kp + p] = blk[16 * p + r];
  }
  if (s_a && blockIdx.x == 0 && threadIdx.x == 0) {
    s_a[0] = s0;
    s_a[1] = s1;
  }
  __syncthreads();
  write_act_units(codes, rows, m0, ap, packed, ximg);
}

// The next layer's haloed code image (an implicit 3x3 convolution's input,
// geometry cg) from the byte image its producer's epilogue wrote: positions
// are ranks within the precision groups (rank r of group g at
// g ? cpad[0] + r : r, Cp positions a row), blocked from the GEMM tiles,
// row-major from the GEMV forms, as for k_pack_img.  Output pixel m of the
// producer is pixel (y, x) = ((m / W) % H, m % W) of image m / (H*W).
// Workgroup b packs 16-row block b into its interior pixels, one unit
// (16 ranks) per thread; every workgroup then takes a share of the halo
// pixels, whose units hold the stored code of 0.0 (halo[g]) at the group's
// ranks and the stored 0 of padding past them.  Workgroup 0 also stores
// the static scales.  Dynamic LDS: 16 * Cp bytes.
__global__ __launch_bounds__(256) void k_pack_conv_img(const uint8_t* __restrict__ bimg, int64_t ld,
                                                       bool blocked, int64_t M, int nimg, int cnt0,
                                                       int cnt1, int halo0, int halo1, ActPlan ap,
                                                       ConvGeo cg, float s0, float s1,
                                                       float* __restrict__ s_a,
                                                       uint8_t* __restrict__ img) {
  extern __shared__ __align__(16) uint8_t codes[];
  const int Cp = cg.cpad[0] + (ap.S == 2 ? cg.cpad[1] : 0);
  const int U0 = cg.cpad[0] / 16, U = U0 + (ap.S == 2 ? cg.cpad[1] / 16 : 0);
  const int Wp = cg.W + 2, Hp = cg.H + 2, HW = cg.H * cg.W;
  const int64_t m0 = (int64_t)blockIdx.x * kBlk;
  const int rows = (int)min((int64_t)kBlk, M - m0);
  if (s_a && blockIdx.x == 0 && threadIdx.x == 0) {
    s_a[0] = s0;
    s_a[1] = s1;
  }
  if (blocked) {
    img_block_rows(bimg + (m0 / kBlk) * ld, 0, Cp / 4, codes);
  } else {
    for (int r = 0; r < rows; ++r)
      for (int i = threadIdx.x; i < Cp / 16; i += 256)
        reinterpret_cast<uint4*>(codes + r * Cp)[i] = reinterpret_cast<const uint4*>(bimg + (m0 + r) * ld)[i];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < rows * U; i += 256) {
    const int r = i / U, u = i - r * U;
    const int g = u >= U0 ? 1 : 0, uu = g ? u - U0 : u;
    const uint4 d = *reinterpret_cast<const uint4*>(codes + r * Cp + 16 * u);
    const int64_t m = m0 + r;
    const int b = (int)(m / HW), rem = (int)(m - (int64_t)b * HW);
    const int y = rem / cg.W, x = rem - y * cg.W;
    const int64_t hp = ((int64_t)b * Hp + y + 1) * Wp + x + 1;
    const int c = ap.c[g];
    store_unit(img + cg.img_off[g] + hp * cg.rowbytes[g] + uu * 2 * c, pack_unit(d.x, d.y, d.z, d.w, c), c);
  }
  // halo pixels: the top and bottom rows, then the left and right columns
  const int nh = 2 * Wp + 2 * cg.H;
  const int64_t hitems = (int64_t)nimg * nh * U;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < hitems; i += (int64_t)gridDim.x * 256) {
    const int u = (int)(i % U);
    const int64_t q = i / U;
    const int b = (int)(q / nh), h = (int)(q - (int64_t)b * nh);
    int yh, xh;
    if (h < 2 * Wp) {
      yh = h < Wp ? 0 : Hp - 1;
      xh = h < Wp ? h : h - Wp;
    } else {
      const int v = h - 2 * Wp;
      yh = 1 + (v >> 1);
      xh = (v & 1) ? Wp - 1 : 0;
    }
    const int g = u >= U0 ? 1 : 0, uu = g ? u - U0 : u;
    const int cnt = g ? cnt1 : cnt0;
    const uint32_t hb = (uint32_t)(g ? halo1 : halo0) & 0xFFu;
    uint32_t dw[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      dw[j] = 0u;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (16 * uu + 4 * j + e < cnt) dw[j] |= hb << (8 * e);
    }
    const int64_t hp = ((int64_t)b * Hp + yh) * Wp + xh;
    const int c = ap.c[g];
    store_unit(img + cg.img_off[g] + hp * cg.rowbytes[g] + uu * 2 * c, pack_unit(dw[0], dw[1], dw[2], dw[3], c), c);
  }
}

// ------------------------------------------------------ sub-group scales --
// GroupSize_act blocks (the design-space parameters of Sec. 3; Sec. 5 uses
// 512-bit activation groups for transformers): each precision group is cut
// into blocks of gsub granules (64 channels each) in the planned order,
// and each block has its own scale, the max-abs over the batch and the
// block's channels.  Quantizing takes three launches (partial block maxima
// per row range, block scales, codes); the GEMM folds each block's exact
// int32 sum into fp32 as soon as the block ends.  grp[k] is the block of
// original channel k; blocks of group 0 come first.  These paths run only
// with a zero point of 0 in both groups (signed codes, or unsigned widths
// below their container) and no 1-bit sign group.

// Workgroup b takes rows [b*rpb, min(M, (b+1)*rpb)): each column's max-abs
// over them goes into its block's LDS word (non-negative floats order as
// their bits), then the block maxima go to part[b*nsub + j].  Dynamic LDS:
// nsub words.
__global__ __launch_bounds__(256) void k_gabsmax(const float* __restrict__ A, int64_t M, int64_t K,
                                                 int64_t lda, int64_t rpb,
                                                 const int32_t* __restrict__ grp, int nsub,
                                                 float* __restrict__ part) {
  extern __shared__ unsigned smax[];
  const int tid = threadIdx.x;
  for (int j = tid; j < nsub; j += 256) smax[j] = 0u;
  __syncthreads();
  const int64_t m0 = (int64_t)blockIdx.x * rpb;
  const int64_t n = min(M, m0 + rpb) - m0;
  for (int64_t k = tid; k < K; k += 256) {
    const float* col = A + m0 * lda + k;
    float m = 0.0f;
    int64_t r = 0;
    for (; r + 8 <= n; r += 8) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = fabsf(col[(r + i) * lda]);
      m = fmaxf(m, fmaxf(fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])),
                         fmaxf(fmaxf(v[4], v[5]), fmaxf(v[6], v[7]))));
    }
    for (; r < n; ++r) m = fmaxf(m, fabsf(col[r * lda]));
    atomicMax(&smax[grp[k]], __float_as_uint(m));
  }
  __syncthreads();
  for (int j = tid; j < nsub; j += 256) part[(int64_t)blockIdx.x * nsub + j] = __uint_as_float(smax[j]);
}

// Scale of block j (one workgroup per block) from the partial maxima.
__global__ __launch_bounds__(256) void k_gscales(const float* __restrict__ part, int nparts,
                                                 int nsub, ActPlan ap, float* __restrict__ s_a) {
  __shared__ float red[8];
  const int j = blockIdx.x;
  float m = 0.0f;
  for (int b = threadIdx.x; b < nparts; b += 256) m = fmaxf(m, part[(int64_t)b * nsub + j]);
  m = block_max(m, red);
  if (threadIdx.x == 0) s_a[j] = group_scale(m, j < ap.nsub[0] ? ap.q[0] : ap.q[1]);
}

// R rows per workgroup: each element's code with its block's scale goes to
// LDS at its planned position, then the rows' units are written.  Codes
// follow the per-group quantizer (reciprocal shortcut, exact division near
// a tie or for scales outside the shortcut's range).  Dynamic LDS: R*Kp
// code bytes, then nsub scales and nsub reciprocals.
template <int R>
__global__ __launch_bounds__(256) void k_gquant(const float* __restrict__ A, int64_t M, int64_t K,
                                                int64_t lda, const int32_t* __restrict__ pos,
                                                const int32_t* __restrict__ grp, ActPlan ap,
                                                int nsub, const float* __restrict__ s_a,
                                                uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  float* stab = reinterpret_cast<float*>(codes + R * ap.Kp);
  float* rtab = stab + nsub;
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blockIdx.x * R;
  const int rows = (int)min((int64_t)R, M - m0);
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < rows * ap.Kp / 4; i += 256) codes32[i] = 0u;
  for (int j = tid; j < nsub; j += 256) {
    const float sc = s_a[j];
    stab[j] = sc;
    rtab[j] = fast_ok(sc) ? __builtin_amdgcn_rcpf(sc) : 0.0f;
  }
  __syncthreads();
  const float lo0 = (float)ap.q[0].lo, hi0 = (float)ap.q[0].hi;
  const float lo1 = (float)ap.q[1].lo, hi1 = (float)ap.q[1].hi;
  for (int64_t k = tid; k < K; k += 256) {
    const int j = grp[k], p = pos[k];
    const bool g1 = j >= ap.nsub[0];
    const float sc = stab[j], rs = rtab[j];
    const float lo = g1 ? lo1 : lo0, hi = g1 ? hi1 : hi0;
    float x[R];
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = r < rows ? A[(m0 + r) * lda + k] : 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float t = 0.0f;
      if (sc != 0.0f) {
        const float e = x[r] * rs;
        t = __builtin_rintf(e);
        if (rs == 0.0f || fabsf(fabsf(e - t) - 0.5f) <= 0x1p-9f) t = __builtin_rintf(__fdiv_rn(x[r], sc));
        t = fminf(fmaxf(t, lo), hi);
      }
      if (r < rows) codes[r * ap.Kp + p] = (uint8_t)(int8_t)(int)t;
    }
  }
  __syncthreads();
  write_act_units(codes, rows, m0, ap, packed);
}

// float4 forms of the two passes above (K % 4 == 0, lda % 4 == 0, A
// 16-byte aligned, K <= 1024*J): thread tid owns float4 columns
// k4 = tid + 256*j (j < J) of every row; rows are loaded four at a time
// for all its columns together.  Clamped rows and columns re-read data
// already counted (a max ignores them; the quantizer skips them).
template <int J>
__global__ __launch_bounds__(256) void k_gabsmax4(const float4* __restrict__ A, int64_t M, int K4,
                                                  int64_t lda4, int64_t rpb,
                                                  const int4* __restrict__ grp4, int nsub,
                                                  float* __restrict__ part) {
  extern __shared__ unsigned smax[];
  const int tid = threadIdx.x;
  for (int j = tid; j < nsub; j += 256) smax[j] = 0u;
  const int64_t m0 = (int64_t)blockIdx.x * rpb;
  const int n = (int)(min(M, m0 + rpb) - m0);
  float4 mx[J];
#pragma unroll
  for (int j = 0; j < J; ++j) mx[j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int r = 0; r < n; r += 4) {
    float4 v[4][J];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
#pragma unroll
      for (int j = 0; j < J; ++j)
        v[rr][j] = A[(m0 + min(r + rr, n - 1)) * lda4 + min(tid + 256 * j, K4 - 1)];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
#pragma unroll
      for (int j = 0; j < J; ++j) {
        mx[j].x = fmaxf(mx[j].x, fabsf(v[rr][j].x));
        mx[j].y = fmaxf(mx[j].y, fabsf(v[rr][j].y));
        mx[j].z = fmaxf(mx[j].z, fabsf(v[rr][j].z));
        mx[j].w = fmaxf(mx[j].w, fabsf(v[rr][j].w));
      }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int k4 = tid + 256 * j;
    if (k4 < K4) {
      const int4 g = grp4[k4];
      atomicMax(&smax[g.x], __float_as_uint(mx[j].x));
      atomicMax(&smax[g.y], __float_as_uint(mx[j].y));
      atomicMax(&smax[g.z], __float_as_uint(mx[j].z));
      atomicMax(&smax[g.w], __float_as_uint(mx[j].w));
    }
  }
  __syncthreads();
  for (int j = tid; j < nsub; j += 256) part[(int64_t)blockIdx.x * nsub + j] = __uint_as_float(smax[j]);
}

// Sub-group scales for batches of at most MT <= 8 rows in one launch:
// workgroup m loads every row of the batch once (J float4 per thread and
// row), folds their block maxima into LDS, turns them into the block
// scales, and quantizes its own row m with them, with the arithmetic of
// k_gabsmax4, k_gscales and k_gquant4 (so the codes and scales are
// theirs).  Workgroup 0 stores the scales.  Dynamic LDS: Kp code bytes,
// then nsub maxima, scales and reciprocals.
template <int J, int MT>
__global__ __launch_bounds__(256) void k_gact_rows(const float4* __restrict__ A, int M, int K4,
                                                   int64_t lda4, const int4* __restrict__ pos4,
                                                   const int4* __restrict__ grp4, ActPlan ap,
                                                   int nsub, float* __restrict__ s_a,
                                                   uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  unsigned* smax = reinterpret_cast<unsigned*>(codes + ap.Kp);
  float* stab = reinterpret_cast<float*>(smax + nsub);
  float* rtab = stab + nsub;
  const int tid = threadIdx.x;
  const int m = blockIdx.x;
  float4 v[MT][J];
  int4 p[J], gb[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int k4 = min(tid + 256 * j, K4 - 1);  // repeats change no max
    p[j] = pos4[k4];
    gb[j] = grp4[k4];
#pragma unroll
    for (int r = 0; r < MT; ++r) v[r][j] = A[(int64_t)min(r, M - 1) * lda4 + k4];
  }
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < ap.Kp / 4; i += 256) codes32[i] = 0u;
  for (int j = tid; j < nsub; j += 256) smax[j] = 0u;
  __syncthreads();
#pragma unroll
  for (int j = 0; j < J; ++j) {
    float4 mx = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
    for (int r = 0; r < MT; ++r) {
      mx.x = fmaxf(mx.x, fabsf(v[r][j].x));
      mx.y = fmaxf(mx.y, fabsf(v[r][j].y));
      mx.z = fmaxf(mx.z, fabsf(v[r][j].z));
      mx.w = fmaxf(mx.w, fabsf(v[r][j].w));
    }
    atomicMax(&smax[gb[j].x], __float_as_uint(mx.x));
    atomicMax(&smax[gb[j].y], __float_as_uint(mx.y));
    atomicMax(&smax[gb[j].z], __float_as_uint(mx.z));
    atomicMax(&smax[gb[j].w], __float_as_uint(mx.w));
  }
  __syncthreads();
  for (int j = tid; j < nsub; j += 256) {
    const float sc = group_scale(__uint_as_float(smax[j]), j < ap.nsub[0] ? ap.q[0] : ap.q[1]);
    stab[j] = sc;
    rtab[j] = fast_ok(sc) ? __builtin_amdgcn_rcpf(sc) : 0.0f;
    if (m == 0) s_a[j] = sc;
  }
  __syncthreads();
  const float lo0 = (float)ap.q[0].lo, hi0 = (float)ap.q[0].hi;
  const float lo1 = (float)ap.q[1].lo, hi1 = (float)ap.q[1].hi;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    if (tid + 256 * j >= K4) break;
    float4 x = v[0][j];
#pragma unroll
    for (int r = 1; r < MT; ++r)
      if (r == m) x = v[r][j];
    const float xs[4] = {x.x, x.y, x.z, x.w};
    const int pp[4] = {p[j].x, p[j].y, p[j].z, p[j].w};
    const int gg[4] = {gb[j].x, gb[j].y, gb[j].z, gb[j].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float sc = stab[gg[e]], rs = rtab[gg[e]];
      const bool g1 = gg[e] >= ap.nsub[0];
      float t = 0.0f;
      if (sc != 0.0f) {
        const float ex = xs[e] * rs;
        t = __builtin_rintf(ex);
        if (rs == 0.0f || fabsf(fabsf(ex - t) - 0.5f) <= 0x1p-9f) t = __builtin_rintf(__fdiv_rn(xs[e], sc));
        t = fminf(fmaxf(t, g1 ? lo1 : lo0), g1 ? hi1 : hi0);
      }
      codes[pp[e]] = (uint8_t)(int8_t)(int)t;
    }
  }
  __syncthreads();
  write_act_units(codes, 1, m, ap, packed);
}

template <int R, int J>
__global__ __launch_bounds__(256) void k_gquant4(const float4* __restrict__ A, int64_t M, int K4,
                                                 int64_t lda4, const int4* __restrict__ pos4,
                                                 const int4* __restrict__ grp4, ActPlan ap,
                                                 int nsub, const float* __restrict__ s_a,
                                                 uint8_t* __restrict__ packed) {
  static_assert(R % 4 == 0, "rows go four at a time");
  extern __shared__ __align__(16) uint8_t codes[];
  float* stab = reinterpret_cast<float*>(codes + R * ap.Kp);
  float* rtab = stab + nsub;
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blockIdx.x * R;
  const int rows = (int)min((int64_t)R, M - m0);
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < rows * ap.Kp / 4; i += 256) codes32[i] = 0u;
  for (int j = tid; j < nsub; j += 256) {
    const float sc = s_a[j];
    stab[j] = sc;
    rtab[j] = fast_ok(sc) ? __builtin_amdgcn_rcpf(sc) : 0.0f;
  }
  int4 p[J], gb[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int k4 = min(tid + 256 * j, K4 - 1);
    p[j] = pos4[k4];
    gb[j] = grp4[k4];
  }
  __syncthreads();
  const float lo0 = (float)ap.q[0].lo, hi0 = (float)ap.q[0].hi;
  const float lo1 = (float)ap.q[1].lo, hi1 = (float)ap.q[1].hi;
  float sc[J][4], rs[J][4];
  bool g1[J][4];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int gg[4] = {gb[j].x, gb[j].y, gb[j].z, gb[j].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      sc[j][e] = stab[gg[e]];
      rs[j][e] = rtab[gg[e]];
      g1[j][e] = gg[e] >= ap.nsub[0];
    }
  }
  for (int r = 0; r < rows; r += 4) {
    float4 v[4][J];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr)
#pragma unroll
      for (int j = 0; j < J; ++j)
        v[rr][j] = A[(m0 + min(r + rr, rows - 1)) * lda4 + min(tid + 256 * j, K4 - 1)];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      if (r + rr >= rows) break;
      uint8_t* row = codes + (r + rr) * ap.Kp;
#pragma unroll
      for (int j = 0; j < J; ++j) {
        if (tid + 256 * j >= K4) break;
        const float xs[4] = {v[rr][j].x, v[rr][j].y, v[rr][j].z, v[rr][j].w};
        const int pp[4] = {p[j].x, p[j].y, p[j].z, p[j].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float t = 0.0f;
          if (sc[j][e] != 0.0f) {
            const float ex = xs[e] * rs[j][e];
            t = __builtin_rintf(ex);
            if (rs[j][e] == 0.0f || fabsf(fabsf(ex - t) - 0.5f) <= 0x1p-9f)
              t = __builtin_rintf(__fdiv_rn(xs[e], sc[j][e]));
            t = fminf(fmaxf(t, g1[j][e] ? lo1 : lo0), g1[j][e] ? hi1 : hi0);
          }
          row[pp[e]] = (uint8_t)(int8_t)(int)t;
        }
      }
    }
  }
  __syncthreads();
  write_act_units(codes, rows, m0, ap, packed);
}

// Block scales a wave keeps in registers: lane l holds s_a[l + 64*i].
constexpr int kGSubRegs = 4;
static_assert(kGSubMax <= 64 * kGSubRegs, "every block scale has a lane");

// The 64 x 128 tile of k_gemm with sub-group scales.  After the last
// granule of each block the tile folds its int32 sums into fp32,
// y = y + f(acc >> sh) * s_a[j] (multiply, then add, in block order), and
// restarts them at 0; the epilogue scales by s_w and rounds to bf16.  With
// a zero point of 0, acc >> sh is the block's exact sum (the unpack scales
// removed), which the optional int32 dump receives as [block][M][N].
// QN > 0 quantizes each fp32 output for the next layer as k_gemm does (one
// static scale per next-layer group, QN = 1, or per block, QN = 2).
template <int S, int CA0, int CA1, int CBL, int CBH, int QN = 0>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
void k_gemm_g(GemmArgs a) {
  constexpr int WFM = 2, NST = 2, BM = 32 * WFM;
  constexpr int SLOT = gemm_slot(S, CA0, CA1, CBL, CBH, WFM);
  constexpr int ASLOT = gemm_aslot(S, CA0, CA1, CBL, CBH, WFM);
  __shared__ __align__(16) uint8_t lds[NST * SLOT];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 1, wn = wid & 1;
  const ActPlan& ap = a.ap;
  const int ntn = a.wp.Np / kGemmBN;
  const int G = (int)gridDim.x, x = (int)(blockIdx.x & 7), l = (int)(blockIdx.x >> 3);
  const int tile = a.xcd_tiles ? x * (G >> 3) + min(x, G & 7) + l : (int)blockIdx.x;
  const int mt = tile / ntn, nt = tile - mt * ntn;
  const int64_t m0 = (int64_t)mt * BM;
  const int jb0 = nt * 8;

  int bc[8], bpre[9];
  bpre[0] = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    bc[j] = wblk_c(a.wp, jb0 + j);
    bpre[j + 1] = bpre[j] + 16 * bc[j];
  }
  const uint8_t* wtile = a.wd.packed + wblk_off(a.wp, jb0);
  const int wbytes = (int)(wblk_off(a.wp, jb0 + 8) - wblk_off(a.wp, jb0));
  const bool tile_lo = jb0 < a.wp.nlo;

  const int nsub = ap.nsub[0] + (S == 2 ? ap.nsub[1] : 0);
  float sreg[kGSubRegs];
#pragma unroll
  for (int i = 0; i < kGSubRegs; ++i) sreg[i] = lane + 64 * i < nsub ? a.s_a[lane + 64 * i] : 0.0f;
  ColInfo cinf[4];
  uint8_t cshw[4], crank[4];
  int cqg[4] = {0, 0, 0, 0};  // next-layer group (or block) of each column (QN)
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    const int pc = (jb0 + wn * 4 + jj) * kBlk + (lane & 15);
    cinf[jj] = a.wd.colinfo[pc];
    cshw[jj] = a.wd.shw[pc];
    crank[jj] = a.wd.colrank[pc];
    if constexpr (QN > 0) cqg[jj] = a.qn_tab[pc];
  }
  // the store phase's column of this thread, requested early (as k_gemm)
  const int st_col = QN > 0 ? a.qn_tab[a.wp.Np + nt * kGemmBN + (tid & (kGemmBN - 1))]
                            : a.wd.tile_cols[nt * kGemmBN + (tid & (kGemmBN - 1))];

  v4i acc[WFM][4];
  float yf[WFM][4][4];
#pragma unroll
  for (int i = 0; i < WFM; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      acc[i][jj] = v4i{0, 0, 0, 0};
#pragma unroll
      for (int r = 0; r < 4; ++r) yf[i][jj][r] = 0.0f;
    }

  // Fold block j of group g.
  auto fold = [&](v4i (&ac)[WFM][4], int g, int j) __attribute__((always_inline)) {
    const int jr = j >> 6;
    const float sv = jr == 0 ? sreg[0] : jr == 1 ? sreg[1] : jr == 2 ? sreg[2] : sreg[3];
    const float sj = __builtin_bit_cast(
        float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, sv), j & 63));
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int sh = ap.sh[g] + (cshw[jj] & 0x7F);
#pragma unroll
      for (int i = 0; i < WFM; ++i) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          yf[i][jj][r] = __fadd_rn(yf[i][jj][r], __fmul_rn((float)(ac[i][jj][r] >> sh), sj));
        if (a.acc) {
          const int row0 = (wm * WFM + i) * 16 + (lane >> 4) * 4;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int64_t m = m0 + row0 + r;
            if (m < a.M && cinf[jj].n >= 0)
              a.acc[((int64_t)j * a.M + m) * a.N + cinf[jj].n] = ac[i][jj][r] >> sh;
          }
        }
        ac[i][jj] = v4i{0, 0, 0, 0};
      }
    }
  };
  auto run_group = [&](auto ca_tag, int g) __attribute__((always_inline)) {
    constexpr int CA = decltype(ca_tag)::value;
    const int ng = g ? ap.ng[1] : ap.ng[0];
    const int gpg = g ? ap.gsub[1] : ap.gsub[0];
    const int j0 = g ? ap.nsub[0] : 0;
    auto hook = [&](v4i (&ac)[WFM][4], int q) __attribute__((always_inline)) {
      if (q < ng && ((q + 1) % gpg == 0 || q == ng - 1)) fold(ac, g, j0 + q / gpg);
    };
    const int64_t mstride = g ? ap.mblk_bytes[1] : ap.mblk_bytes[0];
    const uint8_t* abase = a.act + (g ? ap.seg_off[1] : ap.seg_off[0]) + (m0 / kBlk) * mstride;
    const int qbase = g ? ap.ng[0] : 0;
    if constexpr (CA != 0 && CBL != 0 && CBH != 0) {
      if (CBL == CBH || tile_lo)
        gemm_group_fast<CA, CBL, CBL, WFM, NST, ASLOT, SLOT>(lds, abase, mstride, ng, wtile, wbytes,
                                                             a.wp.ngt, bc, bpre, qbase, acc, tid,
                                                             lane, wid, wm, wn, hook);
      else
        gemm_group_fast<CA, CBH, CBH, WFM, NST, ASLOT, SLOT>(lds, abase, mstride, ng, wtile, wbytes,
                                                             a.wp.ngt, bc, bpre, qbase, acc, tid,
                                                             lane, wid, wm, wn, hook);
    } else {
      gemm_group_any<CA, CBL, CBH, WFM, NST, ASLOT, SLOT>(lds, abase, mstride,
                                                          g ? ap.c[1] : ap.c[0], ng, wtile,
                                                          a.wp.ngt, bc, bpre, qbase, acc, tid,
                                                          lane, wid, wm, wn, hook);
    }
  };
  run_group(std::integral_constant<int, CA0>{}, 0);
  if constexpr (S == 2) run_group(std::integral_constant<int, CA1>{}, 1);

  // Epilogue: y * s_w, bf16, staged in LDS in ascending original column
  // order (as in k_gemm), then stored row by row.
  constexpr int YS = kGemmBN + 8;
  uint16_t* ys = reinterpret_cast<uint16_t*>(lds);
  static_assert(BM * YS * 2 <= NST * SLOT, "output staging fits the ring");
  // QN > 0: each output's next-layer code, staged column-major as in k_gemm
  uint8_t* qs = reinterpret_cast<uint8_t*>(lds) + BM * YS * 2;
  static_assert(QN == 0 || BM * YS * 2 + kGemmBN * (BM + 16) <= NST * SLOT,
                "code staging fits the ring");
  const bool want_y = QN == 0 || a.Y != nullptr;
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    const ColInfo ci = cinf[jj];
    if (ci.n < 0) continue;
    uint16_t* ycol = ys + crank[jj];
#pragma unroll
    for (int i = 0; i < WFM; ++i) {
      const int row0 = (wm * WFM + i) * 16 + (lane >> 4) * 4;
      float y[4];
#pragma unroll
      for (int h = 0; h < 4; ++h) y[h] = __fmul_rn(yf[i][jj][h], ci.s_w);
      if (want_y) {
#pragma unroll
        for (int h = 0; h < 4; h += 2) {
          const __hip_bfloat162 pr = __float22bfloat162_rn(make_float2(y[h], y[h + 1]));
          ycol[(row0 + h) * YS] = __builtin_bit_cast(uint16_t, pr.x);
          ycol[(row0 + h + 1) * YS] = __builtin_bit_cast(uint16_t, pr.y);
        }
      }
      if constexpr (QN > 0) {
        QCol qc;
        if constexpr (QN == 2) {
          const int b = cqg[jj];
          const bool g1 = b >= a.qn_nsub0;
          qc.sc = a.qn_bs[b];
          qc.rs = a.qn_brs[b];
          qc.lo = g1 ? a.qn.lo[1] : a.qn.lo[0];
          qc.hi = g1 ? a.qn.hi[1] : a.qn.hi[0];
          qc.zp = 0;
          qc.sign1 = false;
        } else {
          qc = qnext_col(cqg[jj], a.qn);
        }
        qn_stage4<BM>(qs, crank[jj], row0, qnext4(y, qc));
      }
    }
  }
  __syncthreads();
  if constexpr (QN > 0) {
    qn_store<BM>(a, qs, st_col, m0, tid);
    if (!want_y) return;
  }
  const int n = QN > 0 ? a.wd.tile_cols[nt * kGemmBN + (tid & (kGemmBN - 1))] : st_col;
  if (n >= 0) {
    const int mrem = (int)min((int64_t)BM, a.M - m0);
    uint16_t* yout = a.Y + m0 * a.ldy + n;
    for (int row = tid / kGemmBN; row < mrem; row += 256 / kGemmBN)
      yout[(int64_t)row * a.ldy] = ys[row * YS + (tid & (kGemmBN - 1))];
  }
}

}  // namespace

// ------------------------------------------------------------- launchers --
hipError_t launch_wpack(const float* W, int64_t N, int64_t K, int64_t ldw,
                        const uint8_t* w_bits_dev, const int32_t* pos_dev,
                        const uint8_t* seg_dev, const int32_t* phys_dev,
                        const uint64_t* blk_off, const uint8_t* blk_c, QParam q_lo,
                        QParam q_hi, int b_lo, int Kp, uint8_t* packed, ColInfo* colinfo,
                        hipStream_t stream) {
  hipLaunchKernelGGL(k_wpack, dim3((unsigned)N), dim3(256), (size_t)Kp, stream, W, K, ldw,
                     w_bits_dev, pos_dev, seg_dev, phys_dev, blk_off, blk_c, q_lo, q_hi, b_lo,
                     Kp, packed, colinfo);
  return hipGetLastError();
}

// ------------------------------------------------------------ conv 3x3 --
// Activations of a stride-1, pad-1 3x3 convolution taken straight from its
// input X[B][C][H][W] (fp32, contiguous), with no lowered fp32 matrix: row
// m = (b*H + y)*W + x of the lowered matrix holds, at column
// k = c*9 + kh*3 + kw, the value X[b][c][y+kh-1][x+kw-1] (zero outside the
// image), the column order of a 3x3 unfold.  The host requires the nine
// columns of a channel to share one width, so the group maxima are maxima
// over X's channels, and (the plan keeps original order within a group)
// channel c's nine columns sit at the consecutive planned positions
// pos[9c] .. pos[9c] + 8.

// The conv kernels run a few waves per SIMD (a grid of a few hundred
// workgroups) and need their loads in flight together: the waves-per-EU
// bound lets the compiler keep a batch in registers rather than trade it
// for an occupancy the grid never reaches.
// Group maxima of X, one partial pair per workgroup.  Wave w of workgroup
// b takes the kAbsR rows (b*4 + w)*kAbsR .. of the [B*C][H*W] view (then
// every 4*kAbsR*grid rows on), kAbsJ 64-column strips per row at once: all
// of a batch's loads are in flight together.
constexpr int kAbsR = 8, kAbsJ = 4;

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 4))) void k_conv_absmax(const float* __restrict__ X, int BC, int C,
                                                     int HW, const uint8_t* __restrict__ seg,
                                                     float* __restrict__ partial) {
  __shared__ float red[8];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  float m0 = 0.0f, m1 = 0.0f;
  for (int rb = ((int)blockIdx.x * 4 + wid) * kAbsR; rb < BC; rb += (int)gridDim.x * 4 * kAbsR) {
    // the batch's channels (row = b*C + c), stepped from one division
    int cr[kAbsR];
    cr[0] = rb % C;
#pragma unroll
    for (int rr = 1; rr < kAbsR; ++rr) cr[rr] = cr[rr - 1] + 1 == C ? 0 : cr[rr - 1] + 1;
    uint8_t g[kAbsR];
#pragma unroll
    for (int rr = 0; rr < kAbsR; ++rr) g[rr] = seg[9 * cr[rr]];
    for (int j0 = 0; j0 < HW; j0 += 64 * kAbsJ) {
      float v[kAbsR][kAbsJ];
#pragma unroll
      for (int rr = 0; rr < kAbsR; ++rr)
#pragma unroll
        for (int jj = 0; jj < kAbsJ; ++jj) {
          // clamped indices stay in bounds; what they add is masked out
          const int row = rb + rr < BC ? rb + rr : BC - 1;
          const int col = j0 + jj * 64 + lane;
          const float x = X[(int64_t)row * HW + (col < HW ? col : HW - 1)];
          v[rr][jj] = rb + rr < BC && col < HW ? fabsf(x) : 0.0f;
        }
#pragma unroll
      for (int rr = 0; rr < kAbsR; ++rr) {
        const float m = fmaxf(fmaxf(v[rr][0], v[rr][1]), fmaxf(v[rr][2], v[rr][3]));
        if (g[rr] != 0) m1 = fmaxf(m1, m);
        else m0 = fmaxf(m0, m);
      }
    }
  }
  const float2 r = block_max2(make_float2(m0, m1), red);
  if (threadIdx.x == 0) reinterpret_cast<float2*>(partial)[blockIdx.x] = r;
}

// RB = 8 rows of the lowered matrix per workgroup (half a 16-row block).
// Thread t takes row r = t % 8 and channels c = t / 8 + 32j: batches of
// kConvCB channels, each batch's nine taps per channel (and the channels'
// planned positions and groups) all loaded before any is quantized, the
// 8 rows of a tap being neighbouring pixels.  FAST (no sign group): codes
// without the zero point (the shortcut of qcodes4 with a per-tap tie
// check), applied as a byte XOR when the units are packed; otherwise the
// generic stored codes.  Dynamic LDS: 8 rows of ldc bytes (ldc = Kp + 16
// keeps the rows' byte writes in different banks).
constexpr int kConvRB = 8, kConvCB = 8;

template <bool FAST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_conv_quant(const float* __restrict__ X, int B, int C, int H,
                                                    int W, const int32_t* __restrict__ pos,
                                                    const uint8_t* __restrict__ seg,
                                                    const float* __restrict__ partial, int nparts,
                                                    ActPlan ap, int ldc, float* __restrict__ s_a_out,
                                                    uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int tid = threadIdx.x;
  const int HW = H * W;
  const int64_t M = (int64_t)B * HW;
  const int64_t m0 = (int64_t)blockIdx.x * kConvRB;
  {
    // each group's zero point (FAST) or zero: the padding packs to zeros
    uint32_t* c32 = reinterpret_cast<uint32_t*>(codes);
    const int kw = ldc / 4, kw0 = ap.kpad[0] / 4;
    const uint32_t z0 = FAST ? 0x01010101u * (uint32_t)ap.zp[0] : 0u;
    const uint32_t z1 = FAST ? 0x01010101u * (uint32_t)ap.zp[1] : 0u;
    for (int r = 0; r < kConvRB; ++r)
      for (int j = tid; j < kw; j += 256) c32[r * kw + j] = j < kw0 ? z0 : z1;
  }
  float s0, s1;
  scales_from_partials(partial, nparts, ap, red, s0, s1, s_a_out);  // syncs
  const int r = tid % kConvRB, cl = tid / kConvRB;
  constexpr int kLanes = 256 / kConvRB;  // channel lanes
  const int64_t m = m0 + r;
  if (m < M) {
    const int b = (int)(m / HW), yx = (int)(m - (int64_t)b * HW);
    const int y = yx / W, x = yx - y * W;
    // tap t reads xc[off[t]]; a tap outside the image reads xc[0] (always
    // in bounds) and takes zero instead
    int off[9];
    unsigned valid = 0;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int dy = t / 3 - 1, dx = t % 3 - 1;
      const bool in = y + dy >= 0 && y + dy < H && x + dx >= 0 && x + dx < W;
      off[t] = in ? dy * W + dx : 0;
      valid |= in ? 1u << t : 0u;
    }
    const float* xb = X + (int64_t)b * C * HW + (int64_t)y * W + x;
    uint8_t* crow = codes + r * ldc;
    const bool sgn = ap.q[0].lo < 0;
    const bool fast = fast_ok(s0) && (ap.S == 1 || fast_ok(s1));
    const float rs0 = fast ? __builtin_amdgcn_rcpf(s0) : 0.0f;
    const float rs1 = fast && ap.S == 2 ? __builtin_amdgcn_rcpf(s1) : 0.0f;
    const float hi0 = (float)ap.q[0].hi, hi1 = (float)ap.q[1].hi;
    const ActQ aq = make_actq(ap, s0, s1);
    for (int c0 = cl; c0 < C; c0 += kLanes * kConvCB) {
      float v[kConvCB][9];
      int pj[kConvCB];
      uint8_t gj[kConvCB];
#pragma unroll
      for (int j = 0; j < kConvCB; ++j) {
        const int c = c0 + kLanes * j;
        const int cc = c < C ? c : C - 1;  // in bounds; its codes are not stored
        const float* xc = xb + (int64_t)cc * HW;
#pragma unroll
        for (int t = 0; t < 9; ++t) v[j][t] = xc[off[t]];
        pj[j] = pos[9 * cc];
        gj[j] = seg[9 * cc];
      }
#pragma unroll
      for (int j = 0; j < kConvCB; ++j) {
        if (c0 + kLanes * j >= C) break;
        uint8_t* dst = crow + pj[j];
        const bool g1 = gj[j] != 0;
        if constexpr (FAST) {
          const float rs = g1 ? rs1 : rs0, sc = g1 ? s1 : s0, hi = g1 ? hi1 : hi0;
          const float lo = sgn ? -hi : 0.0f;
#pragma unroll
          for (int t = 0; t < 9; ++t) {
            const float xv = (valid >> t) & 1u ? v[j][t] : 0.0f;
            int code;
            if (fast) {
              const float tt = __builtin_fmaf(xv, rs, kShift);
              code = __float_as_int(sgn ? tt : fmaxf(tt, kShift));
              const float d = __builtin_fmaf(xv, rs, kShift - tt);
              if (fabsf(d) >= 0.5f - kTieBand) [[unlikely]]
                code = qexact(xv, lo, hi, 0.0f, sc);
            } else {
              code = qexact(xv, lo, hi, 0.0f, sc);
            }
            dst[t] = (uint8_t)code;
          }
        } else {
#pragma unroll
          for (int t = 0; t < 9; ++t)
            dst[t] = store_code((valid >> t) & 1u ? v[j][t] : 0.0f, g1 ? 1 : 0, aq);
        }
      }
    }
  }
  __syncthreads();
  const int r0 = (int)(m0 % kBlk);
  for (int gi = 0; gi < ap.S; ++gi) {
    const int c = gi ? ap.c[1] : ap.c[0];
    const int ng = gi ? ap.ng[1] : ap.ng[0];
    const int gbase = gi ? ap.kpad[0] : 0;
    const uint32_t zx = FAST ? 0x01010101u * (uint32_t)(gi ? ap.zp[1] : ap.zp[0]) : 0u;
    uint8_t* dst = packed + (gi ? ap.seg_off[1] : ap.seg_off[0]) +
                   (m0 / kBlk) * (gi ? ap.mblk_bytes[1] : ap.mblk_bytes[0]);
    if (c == 8) write_block_pieces<8, kConvRB>(codes, ldc, gbase, ng, r0, dst, zx);
    else if (c == 4) write_block_pieces<4, kConvRB>(codes, ldc, gbase, ng, r0, dst, zx);
    else if (c == 2) write_block_pieces<2, kConvRB>(codes, ldc, gbase, ng, r0, dst, zx);
    else write_block_pieces<1, kConvRB>(codes, ldc, gbase, ng, r0, dst, zx);
  }
}

// The same result from an LDS window: workgroup b takes the 16 rows of
// block b (pixels m0 .. m0 + 15, global image rows R = b*H + y from
// m0 / W to (m0 + 15) / W) and first quantizes, once each, every input
// value of the global image rows R0 - 1 .. R1 + 1 (all channels) into
// win[row][c][x] (one code byte each), with coalesced loads.  A pixel's
// nine taps are then byte copies out of the window into its code row
// (taps outside the image take the code of 0.0).  Dynamic LDS: 16 code
// rows of ldc bytes, then the window (nr * C * W bytes, nr <= 19).
template <bool FAST>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 2))) void k_conv_quant_win(const float* __restrict__ X, int B, int C,
                                                        int H, int W, const int32_t* __restrict__ pos,
                                                        const uint8_t* __restrict__ seg,
                                                        const float* __restrict__ partial, int nparts,
                                                        ActPlan ap, int ldc, float* __restrict__ s_a_out,
                                                        uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[8];
  const int tid = threadIdx.x;
  const int HW = H * W;
  const int64_t M = (int64_t)B * HW;
  const int64_t m0 = (int64_t)blockIdx.x * kBlk;
  const int64_t mlast = min(m0 + kBlk, M) - 1;
  const int R0 = (int)(m0 / W), R1 = (int)(mlast / W);
  const int wr0 = max(R0 - 1, 0), wr1 = min(R1 + 1, B * H - 1);
  const int nr = wr1 - wr0 + 1;
  uint8_t* win = codes + kBlk * ldc;
  {
    uint32_t* c32 = reinterpret_cast<uint32_t*>(codes);
    const int kw = ldc / 4, kw0 = ap.kpad[0] / 4;
    const uint32_t z0 = FAST ? 0x01010101u * (uint32_t)ap.zp[0] : 0u;
    const uint32_t z1 = FAST ? 0x01010101u * (uint32_t)ap.zp[1] : 0u;
    for (int r = 0; r < kBlk; ++r)
      for (int j = tid; j < kw; j += 256) c32[r * kw + j] = j < kw0 ? z0 : z1;
  }
  // Each channel's group and planned run start, in LDS.
  uint8_t* cg = win + ((conv_win_rows(W) * C * W + 15) & ~(int64_t)15);
  int32_t* cp = reinterpret_cast<int32_t*>(cg + ((C + 15) & ~15));
  for (int c = tid; c < C; c += 256) {
    cg[c] = seg[9 * c];
    cp[c] = pos[9 * c];
  }
  __syncthreads();
  // Window row rc = c*nr + i is X[b][c][y][:] for the global image row
  // wr0 + i = b*H + y (a channel's rows are neighbours in memory within an
  // image): its start index (group of c in bit 31), in LDS.
  int32_t* rbase = cp + C;
  for (int rc = tid; rc < nr * C; rc += 256) {
    const int c = rc / nr, i = rc - c * nr;
    const int gr = wr0 + i, b = gr / H, y = gr - b * H;
    rbase[rc] = (((b * C + c) * H + y) * W) | (cg[c] != 0 ? (int)0x80000000u : 0);
  }
  __syncthreads();
  // Window element rc*W + x: thread t keeps column x = t % W and takes rows
  // t / W + P*j (P = 256 / W rows per pass; the last 256 - P*W threads
  // idle), kWinU loads at a time.  The first batch is issued before the
  // scales are reduced, so that both wait together.
  constexpr int kWinU = 64;
  const int P = 256 / W, nrc = nr * C;
  const int wx = tid % W, rq = tid / W;
  const bool active = rq < P;
  float xv[kWinU];
  int meta[kWinU];
  auto issue = [&](int j0) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < kWinU; ++u) {
      const int rc = rq + P * (j0 + u);
      const bool ok = active && rc < nrc;
      const int m = rbase[ok ? rc : 0];  // row 0 keeps the load in bounds
      meta[u] = m;
      xv[u] = X[(m & 0x7FFFFFFF) + (ok ? wx : 0)];
    }
  };
  issue(0);
  float s0, s1;
  scales_from_partials(partial, nparts, ap, red, s0, s1, s_a_out);  // syncs
  const ActQ aq = make_actq(ap, s0, s1);
  const bool sgn = ap.q[0].lo < 0;
  const bool fast = fast_ok(s0) && (ap.S == 1 || fast_ok(s1));
  const float rs0 = fast ? __builtin_amdgcn_rcpf(s0) : 0.0f;
  const float rs1 = fast && ap.S == 2 ? __builtin_amdgcn_rcpf(s1) : 0.0f;
  const float hi0 = (float)ap.q[0].hi, hi1 = (float)ap.q[1].hi;
  auto code_of = [&](float xv, bool g1) __attribute__((always_inline)) -> uint8_t {
    if constexpr (FAST) {
      const float rs = g1 ? rs1 : rs0, hi = g1 ? hi1 : hi0;
      const float lo = sgn ? -hi : 0.0f;
      if (fast) {
        const float tt = __builtin_fmaf(xv, rs, kShift);
        const int code = __float_as_int(sgn ? tt : fmaxf(tt, kShift));
        const float d = __builtin_fmaf(xv, rs, kShift - tt);
        if (fabsf(d) < 0.5f - kTieBand) [[likely]]
          return (uint8_t)code;
      }
      return (uint8_t)qexact(xv, lo, hi, 0.0f, g1 ? s1 : s0);
    } else {
      return store_code(xv, g1 ? 1 : 0, aq);
    }
  };
  for (int j0 = 0;;) {
#pragma unroll
    for (int u = 0; u < kWinU; ++u) {
      const int rc = rq + P * (j0 + u);
      if (active && rc < nrc) win[rc * W + wx] = code_of(xv[u], meta[u] < 0);
    }
    j0 += kWinU;
    if (rq + P * j0 >= nrc) break;
    issue(j0);
  }
  __syncthreads();
  // Taps: thread t takes pixel r = t % 16 and channels t / 16 + 16j.
  {
    const int r = tid & 15, cl = tid >> 4;
    const int64_t m = m0 + r;
    if (m < M) {
      const int R = (int)(m / W), x = (int)(m - (int64_t)R * W);
      const int y = R % H;
      int off[9];
      unsigned valid = 0;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int dy = t / 3 - 1, dx = t % 3 - 1;
        const bool in = y + dy >= 0 && y + dy < H && x + dx >= 0 && x + dx < W;
        // window row R + dy - wr0 of the channel, column x + dx
        off[t] = in ? (R + dy - wr0) * W + x + dx : 0;
        valid |= in ? 1u << t : 0u;
      }
      const uint8_t zc0 = code_of(0.0f, false), zc1 = code_of(0.0f, true);
      uint8_t* crow = codes + r * ldc;
      // kTapCB channels at a time: their table entries, then all their
      // window bytes, then all their code bytes
      constexpr int kTapCB = 4;
      for (int c0 = cl; c0 < C; c0 += 16 * kTapCB) {
        int pj[kTapCB];
        uint8_t gj[kTapCB], bj[kTapCB][9];
#pragma unroll
        for (int j = 0; j < kTapCB; ++j) {
          const int c = min(c0 + 16 * j, C - 1);
          pj[j] = cp[c];
          gj[j] = cg[c];
          const uint8_t* wc = win + c * nr * W;
#pragma unroll
          for (int t = 0; t < 9; ++t) bj[j][t] = wc[off[t]];
        }
#pragma unroll
        for (int j = 0; j < kTapCB; ++j) {
          if (c0 + 16 * j >= C) break;
          const uint8_t zc = gj[j] != 0 ? zc1 : zc0;
          uint8_t* dst = crow + pj[j];
#pragma unroll
          for (int t = 0; t < 9; ++t) dst[t] = (valid >> t) & 1u ? bj[j][t] : zc;
        }
      }
    }
  }
  __syncthreads();
  for (int gi = 0; gi < ap.S; ++gi) {
    const int c = gi ? ap.c[1] : ap.c[0];
    const int ng = gi ? ap.ng[1] : ap.ng[0];
    const int gbase = gi ? ap.kpad[0] : 0;
    const uint32_t zx = FAST ? 0x01010101u * (uint32_t)(gi ? ap.zp[1] : ap.zp[0]) : 0u;
    uint8_t* dst = packed + (gi ? ap.seg_off[1] : ap.seg_off[0]) +
                   (m0 / kBlk) * (gi ? ap.mblk_bytes[1] : ap.mblk_bytes[0]);
    if (c == 8) write_block_pieces<8, kBlk>(codes, ldc, gbase, ng, 0, dst, zx);
    else if (c == 4) write_block_pieces<4, kBlk>(codes, ldc, gbase, ng, 0, dst, zx);
    else if (c == 2) write_block_pieces<2, kBlk>(codes, ldc, gbase, ng, 0, dst, zx);
    else write_block_pieces<1, kBlk>(codes, ldc, gbase, ng, 0, dst, zx);
  }
}

hipError_t launch_conv_quant(const float* X, int64_t B, int64_t C, int64_t H, int64_t W,
                             const ActPlan& ap, const int32_t* pos_dev, const uint8_t* seg_dev,
                             float* partial, float* s_a, uint8_t* packed, hipStream_t stream) {
  const int64_t BC = B * C;
  const int64_t rows_per_block = 4 * kAbsR;
  const int64_t nparts = (BC + rows_per_block - 1) / rows_per_block < kAbsmaxBlocks
                             ? (BC + rows_per_block - 1) / rows_per_block
                             : kAbsmaxBlocks;
  hipLaunchKernelGGL(k_conv_absmax, dim3((unsigned)nparts), dim3(256), 0, stream, X, (int)BC, (int)C,
                     (int)(H * W), seg_dev, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool sign = ap.q[0].sign1 || (ap.S == 2 && ap.q[1].sign1);
  const int ldc = conv_quant_ldc(ap);
  const size_t wlds = conv_win_lds(ap, C, W);
  if (W <= 256 && wlds <= 64 * 1024) {
    const int64_t wblocks = (B * H * W + kBlk - 1) / kBlk;
    if (!sign)
      hipLaunchKernelGGL(k_conv_quant_win<true>, dim3((unsigned)wblocks), dim3(256), wlds, stream, X,
                         (int)B, (int)C, (int)H, (int)W, pos_dev, seg_dev, partial, (int)nparts, ap,
                         ldc, s_a, packed);
    else
      hipLaunchKernelGGL(k_conv_quant_win<false>, dim3((unsigned)wblocks), dim3(256), wlds, stream, X,
                         (int)B, (int)C, (int)H, (int)W, pos_dev, seg_dev, partial, (int)nparts, ap,
                         ldc, s_a, packed);
    return hipGetLastError();
  }
  const int64_t blocks = (B * H * W + kConvRB - 1) / kConvRB;
  if (!sign)
    hipLaunchKernelGGL(k_conv_quant<true>, dim3((unsigned)blocks), dim3(256), (size_t)(kConvRB * ldc),
                       stream, X, (int)B, (int)C, (int)H, (int)W, pos_dev, seg_dev, partial,
                       (int)nparts, ap, ldc, s_a, packed);
  else
    hipLaunchKernelGGL(k_conv_quant<false>, dim3((unsigned)blocks), dim3(256), (size_t)(kConvRB * ldc),
                       stream, X, (int)B, (int)C, (int)H, (int)W, pos_dev, seg_dev, partial,
                       (int)nparts, ap, ldc, s_a, packed);
  return hipGetLastError();
}

hipError_t launch_act_quant(const float* A, int64_t M, int64_t K, int64_t lda,
                            const ActPlan& ap, const int32_t* pos_dev,
                            const uint8_t* seg_dev, float* partial,
                            unsigned int* counter, float* s_a, uint8_t* packed,
                            hipStream_t stream, uint8_t* ximg, bool* ximg_done) {
  // the row image is written by the per-row quantizers below, for one row
  if (M != 1) ximg = nullptr;
  if (ximg_done) *ximg_done = false;
  const bool aligned = (K % 4 == 0) && (lda % 4 == 0) &&
                       (reinterpret_cast<uintptr_t>(A) % 16 == 0);
  const bool sign = ap.q[0].sign1 || (ap.S == 2 && ap.q[1].sign1);
  // batches of one row (up to 16 float4 per thread) or up to 8 rows (up
  // to 4 float4 per thread and row): every row loaded once
  if (aligned && !sign && ((M == 1 && K / 4 <= 256 * 16) || (M <= 8 && K / 4 <= 256 * 4))) {
    const int K4 = (int)(K / 4);
    const int J = (K4 + 255) / 256;
#define SONIQ_ROWS(J_, MT_)                                                                       \
  hipLaunchKernelGGL((k_act_row1<J_, MT_>), dim3((unsigned)M), dim3(256), (size_t)ap.Kp, stream, A, \
                     (int)M, K4, lda, pos_dev, ap, s_a, packed, ximg)
    if (M == 1) {
      if (J <= 1) SONIQ_ROWS(1, 1);
      else if (J <= 2) SONIQ_ROWS(2, 1);
      else if (J <= 4) SONIQ_ROWS(4, 1);
      else if (J <= 8) SONIQ_ROWS(8, 1);
      else SONIQ_ROWS(16, 1);
    } else if (M <= 2) {
      if (J <= 2) SONIQ_ROWS(2, 2); else SONIQ_ROWS(4, 2);
    } else if (M <= 4) {
      if (J <= 2) SONIQ_ROWS(2, 4); else SONIQ_ROWS(4, 4);
    } else {
      if (J <= 2) SONIQ_ROWS(2, 8); else SONIQ_ROWS(4, 8);
    }
#undef SONIQ_ROWS
    if (ximg_done) *ximg_done = ximg != nullptr;
    return hipGetLastError();
  }
  if (aligned && M <= 64 && M * K <= kSmallElems) {
    hipLaunchKernelGGL(k_act_small, dim3((unsigned)M), dim3(256), (size_t)ap.Kp, stream, A,
                       (int)M, (int)K, lda, pos_dev, seg_dev, ap, s_a, packed, ximg);
    if (ximg_done) *ximg_done = ximg != nullptr;
    return hipGetLastError();
  }
  if (aligned && !sign && M * K >= kCoopMinElems) {
    hipError_t e = hipSuccess;
    if (launch_act_coop(A, M, K, lda, ap, pos_dev, counter, s_a, packed, stream, e))
      return e;
  }
  int nparts;
  if (aligned && M <= 16 * (int64_t)kAbsmaxBlocks) {
    // 8 (or 16) rows per workgroup keep the grid within the partial buffer
    const int K4 = (int)(K / 4);
    const int RB = M <= 8 * (int64_t)kAbsmaxBlocks ? 8 : 16;
    const int64_t blocks = (M + RB - 1) / RB;
    nparts = (int)blocks;
    const int J = K4 <= 256 ? 1 : K4 <= 512 ? 2 : K4 <= 768 ? 3 : 4;
    const float4* A4 = reinterpret_cast<const float4*>(A);
    const uchar4* s4 = reinterpret_cast<const uchar4*>(seg_dev);
#define SONIQ_ABSMAX(J_, RB_)                                                                   \
  hipLaunchKernelGGL((k_absmax_blk<J_, RB_>), dim3((unsigned)blocks), dim3(256), 0, stream, A4, M, \
                     K4, lda / 4, s4, partial)
    if (RB == 8) {
      if (J == 1) SONIQ_ABSMAX(1, 8); else if (J == 2) SONIQ_ABSMAX(2, 8);
      else if (J == 3) SONIQ_ABSMAX(3, 8); else SONIQ_ABSMAX(4, 8);
    } else {
      if (J == 1) SONIQ_ABSMAX(1, 16); else if (J == 2) SONIQ_ABSMAX(2, 16);
      else SONIQ_ABSMAX(2, 16);
    }
#undef SONIQ_ABSMAX
  } else {
    const int64_t blocks = M < kAbsmaxBlocks ? M : kAbsmaxBlocks;
    nparts = (int)blocks;
    hipLaunchKernelGGL(k_absmax_rows, dim3((unsigned)blocks), dim3(256), 0, stream, A, M, K, lda,
                       seg_dev, partial);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // groups of 1-bit sign codes, and unaligned rows, take the generic
  // per-element quantizer (J = 0); otherwise J float4 positions per thread
  const int K4 = (int)(K / 4);
  const int J = (sign || !aligned) ? 0 : K4 <= 256 ? 1 : K4 <= 512 ? 2 : K4 <= 768 ? 3 : 4;
#define SONIQ_ACT_ROWS(R_, J_)                                                                  \
  hipLaunchKernelGGL((k_act_rows<R_, J_>),                                                      \
                     dim3((unsigned)(R_ == 4 ? ((M + 127) / 128) * 32 : (M + R_ - 1) / R_)),    \
                     dim3(256),                                                                 \
                     (size_t)R_ * ap.Kp, stream, A, M, K, lda, pos_dev, seg_dev, ap, partial,    \
                     nparts, s_a, packed, ximg)
  // whole 8- or 16-row block slices per workgroup for larger batches
  // 16 rows per workgroup once that still gives ~1.5 workgroups per CU,
  // else 8 (more workgroups in flight)
  const int rbk = M >= 6144 ? 16 : 8;
  if (J > 0 && J <= 3 && M >= 1024 && rbk * (int64_t)ap.Kp <= 64 * 1024) {
    const size_t lds = (size_t)rbk * ap.Kp;
#define SONIQ_BLK(J_, RB_)                                                                       \
  hipLaunchKernelGGL((k_act_blk16<J_, RB_>), dim3((unsigned)((M + RB_ - 1) / RB_)), dim3(256), lds, \
                     stream, A, M, K, lda, pos_dev, seg_dev, ap, partial, nparts, s_a, packed)
    if (rbk == 8) {
      if (J == 1) SONIQ_BLK(1, 8); else if (J == 2) SONIQ_BLK(2, 8); else SONIQ_BLK(3, 8);
    } else {
      if (J == 1) SONIQ_BLK(1, 16); else if (J == 2) SONIQ_BLK(2, 16); else SONIQ_BLK(3, 16);
    }
#undef SONIQ_BLK
  } else if (4 * (int64_t)ap.Kp <= 64 * 1024) {
    switch (J) {
      case 0: SONIQ_ACT_ROWS(4, 0); break;
      case 1: SONIQ_ACT_ROWS(4, 1); break;
      case 2: SONIQ_ACT_ROWS(4, 2); break;
      case 3: SONIQ_ACT_ROWS(4, 3); break;
      default: SONIQ_ACT_ROWS(4, 4); break;
    }
  } else {
    switch (J) {
      case 0: SONIQ_ACT_ROWS(1, 0); break;
      default: SONIQ_ACT_ROWS(1, 4); break;
    }
  }
#undef SONIQ_ACT_ROWS
  // a single row never takes the block form (M >= 1024)
  if (ximg_done) *ximg_done = ximg != nullptr;
  return hipGetLastError();
}

static GemmArgs make_args(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const WDev& wd, const WPlan& wp, int64_t M, int64_t N, uint16_t* Y,
                          int64_t ldy, int32_t* acc) {
  GemmArgs a;
  a.act = act_packed;
  a.s_a = s_a;
  a.ap = ap;
  a.wd = wd;
  a.wp = wp;
  a.M = M;
  a.N = N;
  a.Y = Y;
  a.ldy = ldy;
  a.acc = acc;
  a.xcd_tiles = 0;
  a.dense = nullptr;
  a.db_lo = a.db_hi = 0;
  a.a32 = nullptr;
  a.apos16 = nullptr;
  a.s_a_out = nullptr;
  a.act_out = nullptr;
  a.ximg = nullptr;
  a.K4 = 0;
  a.xs_bytes = 0;
  a.qn_img = nullptr;
  a.qn_max = nullptr;
  a.qn_tab = nullptr;
  a.qn_ld = 0;
  a.qn = QNext{};
  a.qn_bs = nullptr;
  a.qn_brs = nullptr;
  a.qn_nsub0 = 0;
  a.fa = nullptr;
  a.fw = nullptr;
  a.fp = FPlan{};
  a.img = nullptr;
  a.cg = ConvGeo{};
  return a;
}

// Tile shapes: 3 = 128x128 (WFM 4, 2-deep ring, two workgroups per CU),
// 7 = 64x128 (WFM 2, 2-deep, three per CU), 2 = 64x128 (WFM 2, 3-deep).
template <int S, int CA0, int CA1, int CBL, int CBH>
static void launch_gemm_t(const GemmArgs& a, int64_t M, int shape, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  const dim3 blk(256);
  constexpr bool FOK = CA0 != 0 && CBL != 0 && CBH != 0;
  if (FOK && a.fa && shape != 2) {
    // tiles with MFMA-native copies of the narrow operands
    if (shape == 3)
      hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 4, 2, 0, FOK>),
                         dim3((unsigned)(((M + 127) / 128) * ntn)), blk, 0, stream, a);
    else
      hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 2, 2, 0, FOK>),
                         dim3((unsigned)(((M + 63) / 64) * ntn)), blk, 0, stream, a);
    return;
  }
  switch (shape) {
    case 3:
      hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 4, 2>), dim3((unsigned)(((M + 127) / 128) * ntn)), blk, 0, stream, a);
      break;
    case 2:
      hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 2, 3>), dim3((unsigned)(((M + 63) / 64) * ntn)), blk, 0, stream, a);
      break;
    default:
      hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 2, 2>), dim3((unsigned)(((M + 63) / 64) * ntn)), blk, 0, stream, a);
      break;
  }
}

// 128x128 tiles when there are enough of them to keep every CU busy for
// several rounds; otherwise 64x128 tiles through a 2-deep ring, which hide
// latency better on smaller problems.  SONIQ_GEMM_SHAPE (2, 3 or 7)
// overrides the choice for measurement; results do not depend on it.
static int gemm_shape(int64_t M, int ntn) {
  if (const char* e = getenv("SONIQ_GEMM_SHAPE")) return atoi(e);
  if (((M + 127) / 128) * ntn >= 1024) return 3;
  return 7;
}

hipError_t launch_mp_gemm(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                          uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream,
                          const FPlan* fp, const uint8_t* fa, const uint8_t* fw) {
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  if (fp && fa && fw) {
    a.fp = *fp;
    a.fa = fa;
    a.fw = fw;
  }
  const int ca0 = ap.c[0], ca1 = ap.S == 2 ? ap.c[1] : 0;
  const int cl = wp.c_lo, ch = wp.c_hi;
  const int shape = gemm_shape(M, wp.Np / kGemmBN);
  const int64_t tiles = (shape == 3 ? (M + 127) / 128 : (M + 63) / 64) * (wp.Np / kGemmBN);
  a.xcd_tiles = tiles <= 2048;  // a few rounds of two workgroups per CU
  if (ap.S == 2 && ca0 == 4 && ca1 == 8) {
    if (cl == 4 && ch == 8) launch_gemm_t<2, 4, 8, 4, 8>(a, M, shape, stream);
    else if (cl == 4 && ch == 4) launch_gemm_t<2, 4, 8, 4, 4>(a, M, shape, stream);
    else if (cl == 2 && ch == 8) launch_gemm_t<2, 4, 8, 2, 8>(a, M, shape, stream);
    else if (cl == 1 && ch == 4) launch_gemm_t<2, 4, 8, 1, 4>(a, M, shape, stream);
    else if (cl == 2 && ch == 4) launch_gemm_t<2, 4, 8, 2, 4>(a, M, shape, stream);
    else launch_gemm_t<2, 4, 8, 0, 0>(a, M, shape, stream);
  } else if (ap.S == 2) {
    launch_gemm_t<2, 0, 0, 0, 0>(a, M, shape, stream);
  } else {
    launch_gemm_t<1, 0, 0, 0, 0>(a, M, shape, stream);
  }
  return hipGetLastError();
}

// The GEMM with the next layer's quantization in its epilogue (64 x 128
// tiles at every batch size; k_gemm_g when the producer's activations have
// sub-group scales), then the packing of that layer's rows.
static size_t gemv_lds(int64_t M, const ActPlan& ap, const WPlan& wp);
static size_t gemv_g_lds(int64_t M, const ActPlan& ap, const WPlan& wp);
static bool gemv_nibble_plan(const ActPlan& ap);

// k_gemv_mfma's dynamic LDS: the largest weight block in whole 64-chunk
// (1 KB) wave batches; it applies when that and the static reduction
// buffer (8 KB) fit in 64 KB.
static size_t gemv_mfma_lds(const WPlan& wp) {
  return (size_t)(wp.ngt * 8 * wp.c_hi + 63) / 64 * 1024;
}
static bool gemv_mfma_fits(const WPlan& wp) {
  return gemv_mfma_lds(wp) + sizeof(int) * 2048 <= 64 * 1024;
}

template <int S, int CA0, int CA1, int CBL, int CBH>
static void launch_gemm_qn_t(const GemmArgs& a, int64_t M, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  const dim3 grid((unsigned)(((M + 63) / 64) * ntn));
  if (a.ap.gsub[0] > 0) {  // the producer's own activations have blocks
    if (a.qn_bs)
      hipLaunchKernelGGL((k_gemm_g<S, CA0, CA1, CBL, CBH, 2>), grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL((k_gemm_g<S, CA0, CA1, CBL, CBH, 1>), grid, dim3(256), 0, stream, a);
  } else if (a.qn_bs)
    hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 2, 2, 2>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 2, 2, 1>), grid, dim3(256), 0, stream, a);
}

// The implicit convolution's tiles with the next layer's quantization.
template <int CBL, int CBH>
static void launch_gemm_qn_conv_t(const GemmArgs& a, int64_t M, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  hipLaunchKernelGGL((k_gemm<2, 4, 8, CBL, CBH, 2, 2, 1, false, true>),
                     dim3((unsigned)(((M + 63) / 64) * ntn)), dim3(256), 0, stream, a);
}

hipError_t launch_mp_gemm_qnext(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                const WDev& wd, const WPlan& wp, int64_t M, int64_t N, uint16_t* Y,
                                int64_t ldy, int32_t* acc, uint8_t* img, int64_t img_rows,
                                const int32_t* qtab, const ActPlan& ap2, const float* s_next,
                                float* s_a2, float* brs2, uint8_t* packed2, hipStream_t stream,
                                uint8_t* ximg2, const uint8_t* ximg, const uint8_t* pimg,
                                const ConvGeo* pcg, const QnConv* conv) {
  if (pimg && (!conv_gemm_qn_supported(ap, wp) || ap2.gsub[0] > 0)) return hipErrorInvalidValue;
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  if (pimg) {
    a.img = pimg;
    a.cg = *pcg;
  }
  // positions of one row of the byte image: the next plan's, or the ranks
  // of a next convolution's two groups
  const int64_t qcols = conv ? (int64_t)conv->cg.cpad[0] + (ap2.S == 2 ? conv->cg.cpad[1] : 0)
                             : (int64_t)ap2.Kp;
  const bool blocks = ap2.gsub[0] > 0;
  if (blocks) {
    BlockScales b{};
    b.n = ap2.nsub[0] + (ap2.S == 2 ? ap2.nsub[1] : 0);
    for (int j = 0; j < b.n; ++j) b.s[j] = s_next[j];
    hipLaunchKernelGGL(k_set_scales, dim3(1), dim3(256), 0, stream, b, s_a2, brs2);
    a.qn_bs = s_a2;
    a.qn_brs = brs2;
    a.qn_nsub0 = ap2.nsub[0];
  }
  const int64_t tiles = ((M + 63) / 64) * (wp.Np / kGemmBN);
  a.xcd_tiles = tiles <= 2048;
  a.qn_img = img;
  a.qn_tab = qtab;
  a.qn_ld = 0;  // set below with the producer's form
  for (int g = 0; g < 2; ++g) {
    const float sc = !blocks && g < ap2.S ? s_next[g] : 0.0f;
    a.qn.s[g] = sc;
    // the reciprocal shortcut under the same range rule as the device
    // quantizers; IEEE division is within half an ulp of 1/s
    a.qn.rs[g] = (sc >= 0x1p-100f && sc <= 0x1p100f) ? 1.0f / sc : 0.0f;
    a.qn.lo[g] = (float)ap2.q[g].lo;
    a.qn.hi[g] = (float)ap2.q[g].hi;
    a.qn.zp[g] = ap2.zp[g];
    a.qn.sign1[g] = ap2.q[g].sign1;
  }
  // batches of at most 8 rows: the GEMV forms, whose epilogue quantizes
  // each output the same way
  const bool gv_g = !pimg && ap.gsub[0] > 0 && gemv_g_fits(M, ap, wp);
  const bool gv = !pimg && ap.gsub[0] == 0 && gemv_nibble_plan(ap) && gemv_fits(M, ap, wp);
  // The two forms keep separate images, so that neither writes a position
  // that is padding in the other's layout (padding bytes stay 0).
  const bool gemv_form = gv || gv_g;
  a.qn_ld = gemv_form ? qcols : 16 * qcols;
  if (gemv_form) {
    img += img_rows * qcols;
    a.qn_img = img;
  }
  const int cl = wp.c_lo, ch = wp.c_hi;
  if (pimg) {
    if (cl == 4 && ch == 4) launch_gemm_qn_conv_t<4, 4>(a, M, stream);
    else if (cl == 1 && ch == 4) launch_gemm_qn_conv_t<1, 4>(a, M, stream);
    else if (cl == 2 && ch == 4) launch_gemm_qn_conv_t<2, 4>(a, M, stream);
    else if (cl == 2 && ch == 8) launch_gemm_qn_conv_t<2, 8>(a, M, stream);
    else if (cl == 8 && ch == 8) launch_gemm_qn_conv_t<8, 8>(a, M, stream);
    else if (cl == 1 && ch == 8) launch_gemm_qn_conv_t<1, 8>(a, M, stream);
    else if (cl == 2 && ch == 2) launch_gemm_qn_conv_t<2, 2>(a, M, stream);
    else if (cl == 1 && ch == 2) launch_gemm_qn_conv_t<1, 2>(a, M, stream);
    else if (cl == 1 && ch == 1) launch_gemm_qn_conv_t<1, 1>(a, M, stream);
    else launch_gemm_qn_conv_t<4, 8>(a, M, stream);
  } else if (gemv_form) {
    a.xs_bytes = (int)((gemv_lds(M, ap, wp) + 15) / 16 * 16);
    if (M == 1 && gv) a.ximg = const_cast<uint8_t*>(ximg);
    const dim3 grid((unsigned)wp.nblk);
    if (gv_g) {
      const size_t lds = gemv_g_lds(M, ap, wp);
      if (M == 1) hipLaunchKernelGGL(k_gemv_g<1>, grid, dim3(256), lds, stream, a);
      else if (M == 2) hipLaunchKernelGGL(k_gemv_g<2>, grid, dim3(256), lds, stream, a);
      else if (M <= 4) hipLaunchKernelGGL(k_gemv_g<4>, grid, dim3(256), lds, stream, a);
      else hipLaunchKernelGGL(k_gemv_g<8>, grid, dim3(256), lds, stream, a);
    } else if (M >= 2 && gemv_mfma_fits(wp)) {
      hipLaunchKernelGGL(k_gemv_mfma, grid, dim3(256), gemv_mfma_lds(wp), stream, a);
    } else {
      const size_t lds = gemv_lds(M, ap, wp);
      if (M == 1) hipLaunchKernelGGL(k_gemv<1>, grid, dim3(256), lds, stream, a);
      else if (M == 2) hipLaunchKernelGGL(k_gemv<2>, grid, dim3(256), lds, stream, a);
      else if (M <= 4) hipLaunchKernelGGL(k_gemv<4>, grid, dim3(256), lds, stream, a);
      else hipLaunchKernelGGL(k_gemv<8>, grid, dim3(256), lds, stream, a);
    }
  } else if (ap.S == 2 && ap.c[0] == 4 && ap.c[1] == 8) {
    if (cl == 4 && ch == 8) launch_gemm_qn_t<2, 4, 8, 4, 8>(a, M, stream);
    else if (cl == 2 && ch == 8) launch_gemm_qn_t<2, 4, 8, 2, 8>(a, M, stream);
    else if (cl == 1 && ch == 4) launch_gemm_qn_t<2, 4, 8, 1, 4>(a, M, stream);
    else if (cl == 2 && ch == 4) launch_gemm_qn_t<2, 4, 8, 2, 4>(a, M, stream);
    else launch_gemm_qn_t<2, 4, 8, 0, 0>(a, M, stream);
  } else if (ap.S == 2) {
    launch_gemm_qn_t<2, 0, 0, 0, 0>(a, M, stream);
  } else {
    launch_gemm_qn_t<1, 0, 0, 0, 0>(a, M, stream);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const float s0 = blocks ? 0.0f : s_next[0];
  const float s1 = !blocks && ap2.S == 2 ? s_next[1] : 0.0f;
  float* s_out = blocks ? nullptr : s_a2;  // block scales were stored above
  if (conv) {
    // a next convolution: its haloed image, interior and halo
    hipLaunchKernelGGL(k_pack_conv_img, dim3((unsigned)((M + kBlk - 1) / kBlk)), dim3(256),
                       (size_t)kBlk * qcols, stream, img, a.qn_ld, !gemv_form, M, conv->B,
                       conv->cnt[0], conv->cnt[1], conv->halo[0], conv->halo[1], ap2, conv->cg, s0,
                       s1, s_out, conv->img);
    return hipGetLastError();
  }
  // Full 16-row blocks of the GEMM tiles' image (no 1-bit group) spread
  // over about a thousand workgroups; the rest (the GEMV forms' rows, a
  // 1-bit group, a last partial block) one block (or row) per workgroup.
  const bool one_bit = ap2.c[0] == 1 || (ap2.S == 2 && ap2.c[1] == 1);
  const int64_t nfull = !gemv_form && !one_bit ? M / kBlk : 0;
  if (nfull > 0) {
    const int ngr = ap2.Kp / kGran;
    // at least enough parts to keep a part's LDS within 64 KB (64 granules)
    const int parts = (int)std::max<int64_t>((ngr + 63) / 64,
                                             std::min<int64_t>(ngr, (1024 + nfull - 1) / nfull));
    const size_t lds = (size_t)kBlk * kGran * ((ngr + parts - 1) / parts);
    hipLaunchKernelGGL(k_pack_img_split, dim3((unsigned)nfull, (unsigned)parts), dim3(256), lds,
                       stream, img, a.qn_ld, ap2, s0, s1, s_out, packed2);
    s_out = nullptr;  // stored
  }
  const int64_t rest = M - nfull * kBlk;
  if (rest > 0) {
    if (kBlk * (size_t)ap2.Kp <= 64 * 1024)
      hipLaunchKernelGGL(k_pack_img<kBlk>, dim3((unsigned)((rest + kBlk - 1) / kBlk)), dim3(256),
                         kBlk * (size_t)ap2.Kp, stream, img, a.qn_ld, !gemv_form, nfull, M, ap2, s0,
                         s1, s_out, packed2, M == 1 ? ximg2 : nullptr);
    else
      hipLaunchKernelGGL(k_pack_img<1>, dim3((unsigned)rest), dim3(256), (size_t)ap2.Kp, stream, img,
                         a.qn_ld, !gemv_form, nfull * kBlk, M, ap2, s0, s1, s_out, packed2,
                         M == 1 ? ximg2 : nullptr);
  }
  return hipGetLastError();
}

// The GEMM tiles storing Y and folding each next-layer group's largest |Y|
// into the slots (cleared first), for the two-pass fused quantization.
template <int S, int CA0, int CA1, int CBL, int CBH>
static void launch_gemm_ymax_t(const GemmArgs& a, int64_t M, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  hipLaunchKernelGGL((k_gemm<S, CA0, CA1, CBL, CBH, 2, 2, 3>), dim3((unsigned)(((M + 63) / 64) * ntn)),
                     dim3(256), 0, stream, a);
}

// The same for the implicit convolution's tiles.
template <int CBL, int CBH>
static void launch_gemm_ymax_conv_t(const GemmArgs& a, int64_t M, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  hipLaunchKernelGGL((k_gemm<2, 4, 8, CBL, CBH, 2, 2, 3, false, true>),
                     dim3((unsigned)(((M + 63) / 64) * ntn)), dim3(256), 0, stream, a);
}

hipError_t launch_mp_gemm_ymax(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                               const WDev& wd, const WPlan& wp, int64_t M, int64_t N, uint16_t* Y,
                               int64_t ldy, int32_t* acc, const int32_t* qtab, float* slots,
                               hipStream_t stream, const uint8_t* pimg, const ConvGeo* pcg) {
  if (ap.gsub[0] > 0) return hipErrorInvalidValue;
  if (pimg && !conv_gemm_qn_supported(ap, wp)) return hipErrorInvalidValue;
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  const int64_t tiles = ((M + 63) / 64) * (wp.Np / kGemmBN);
  a.qn_tab = qtab;
  a.qn_max = slots;
  const int cl = wp.c_lo, ch = wp.c_hi;
  if (pimg) {
    a.img = pimg;
    a.cg = *pcg;
    if (cl == 4 && ch == 4) launch_gemm_ymax_conv_t<4, 4>(a, M, stream);
    else if (cl == 1 && ch == 4) launch_gemm_ymax_conv_t<1, 4>(a, M, stream);
    else if (cl == 2 && ch == 4) launch_gemm_ymax_conv_t<2, 4>(a, M, stream);
    else if (cl == 2 && ch == 8) launch_gemm_ymax_conv_t<2, 8>(a, M, stream);
    else if (cl == 8 && ch == 8) launch_gemm_ymax_conv_t<8, 8>(a, M, stream);
    else if (cl == 1 && ch == 8) launch_gemm_ymax_conv_t<1, 8>(a, M, stream);
    else if (cl == 2 && ch == 2) launch_gemm_ymax_conv_t<2, 2>(a, M, stream);
    else if (cl == 1 && ch == 2) launch_gemm_ymax_conv_t<1, 2>(a, M, stream);
    else if (cl == 1 && ch == 1) launch_gemm_ymax_conv_t<1, 1>(a, M, stream);
    else launch_gemm_ymax_conv_t<4, 8>(a, M, stream);
    return hipGetLastError();
  }
  a.xcd_tiles = tiles <= 2048;
  if (ap.S == 2 && ap.c[0] == 4 && ap.c[1] == 8) {
    if (cl == 4 && ch == 8) launch_gemm_ymax_t<2, 4, 8, 4, 8>(a, M, stream);
    else if (cl == 2 && ch == 8) launch_gemm_ymax_t<2, 4, 8, 2, 8>(a, M, stream);
    else if (cl == 1 && ch == 4) launch_gemm_ymax_t<2, 4, 8, 1, 4>(a, M, stream);
    else if (cl == 2 && ch == 4) launch_gemm_ymax_t<2, 4, 8, 2, 4>(a, M, stream);
    else launch_gemm_ymax_t<2, 4, 8, 0, 0>(a, M, stream);
  } else if (ap.S == 2) {
    launch_gemm_ymax_t<2, 0, 0, 0, 0>(a, M, stream);
  } else {
    launch_gemm_ymax_t<1, 0, 0, 0, 0>(a, M, stream);
  }
  return hipGetLastError();
}

hipError_t launch_img_bf16(const uint16_t* Y, int64_t M, int N, int64_t ldy, const int32_t* posn,
                           const ActPlan& ap, const QnConv& conv, const float* slots, int nslot,
                           float* s_a, uint8_t* bimg, hipStream_t stream) {
  const int cpad0 = conv.cg.cpad[0];
  const int Cp = cpad0 + (ap.S == 2 ? conv.cg.cpad[1] : 0);
  if (M < 1) return hipSuccess;
  hipLaunchKernelGGL(k_img_bf16, dim3((unsigned)((M + kBlk - 1) / kBlk)), dim3(256), (size_t)kBlk * Cp,
                     stream, Y, M, N, ldy, posn, cpad0, Cp, ap, slots, nslot, s_a, bimg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // then the convolution's haloed image from the blocked byte image (the
  // scales are stored above)
  hipLaunchKernelGGL(k_pack_conv_img, dim3((unsigned)((M + kBlk - 1) / kBlk)), dim3(256),
                     (size_t)kBlk * Cp, stream, bimg, (int64_t)kBlk * Cp, true, M, conv.B, conv.cnt[0],
                     conv.cnt[1], conv.halo[0], conv.halo[1], ap, conv.cg, 0.0f, 0.0f, nullptr,
                     conv.img);
  return hipGetLastError();
}

hipError_t launch_act_bf16(const uint16_t* Y, int64_t M, int64_t K, int64_t ldy, const ActPlan& ap,
                           const int32_t* pos_dev, const uint8_t* seg_dev, const float* slots,
                           int nslot, float* s_a, uint8_t* packed, uint8_t* ximg,
                           hipStream_t stream) {
  const bool aligned = K % 4 == 0 && ldy % 4 == 0 && (reinterpret_cast<uintptr_t>(Y) & 7) == 0;
  // groups of 1-bit sign codes take the per-element quantizer, as in
  // launch_act_quant
  const bool sign = ap.q[0].sign1 || (ap.S == 2 && ap.q[1].sign1);
  const int64_t K4 = K / 4;
  const int J = (sign || !aligned) ? 0 : K4 <= 256 ? 1 : K4 <= 512 ? 2 : K4 <= 768 ? 3 : 4;
  // four rows per workgroup, or one row (small batches, whose workgroups
  // each reduce the whole batch's maxima; or rows too long for four)
  const bool four = M > 8 && 4 * (int64_t)ap.Kp <= 64 * 1024;
  uint8_t* xi = M == 1 ? ximg : nullptr;
#define SONIQ_BF16(R_, J_)                                                                          \
  hipLaunchKernelGGL((k_act_bf16<R_, J_>), dim3((unsigned)((M + R_ - 1) / R_)), dim3(256),          \
                     (size_t)R_ * ap.Kp, stream, Y, M, K, ldy, pos_dev, seg_dev, ap, slots, nslot, s_a, \
                     packed, xi)
  if (four) {
    switch (J) {
      case 0: SONIQ_BF16(4, 0); break;
      case 1: SONIQ_BF16(4, 1); break;
      case 2: SONIQ_BF16(4, 2); break;
      case 3: SONIQ_BF16(4, 3); break;
      default: SONIQ_BF16(4, 4); break;
    }
  } else {
    switch (J) {
      case 0: SONIQ_BF16(1, 0); break;
      case 1: SONIQ_BF16(1, 1); break;
      case 2: SONIQ_BF16(1, 2); break;
      case 3: SONIQ_BF16(1, 3); break;
      default: SONIQ_BF16(1, 4); break;
    }
  }
#undef SONIQ_BF16
  return hipGetLastError();
}

bool gemv_fits(int64_t M, const ActPlan& ap, const WPlan& wp) {
  if (M < 1 || M > 8) return false;
  // dynamic LDS (activation rows) plus the static reduction buffer
  if (gemv_lds(M, ap, wp) + (size_t)2048 * 8 > 64 * 1024) return false;
  // 1-bit weight blocks keep 8 rows per lane: at most 4 activation rows.
  if ((wp.c_lo == 1 || wp.c_hi == 1) && M > 4) return false;
  // buffer-resource offsets into the activation and weight buffers are 32-bit
  const int64_t act_end = ap.S == 2 ? ap.seg_off[1] + ap.mblk_bytes[1] : ap.seg_off[0] + ap.mblk_bytes[0];
  if (act_end >= ((int64_t)1 << 31) || (int64_t)wp.ngt * 128 * 8 * 16 >= ((int64_t)1 << 31))
    return false;
  return true;
}

// The nibble GEMV needs the first activation group in 4-bit containers and
// the second (if any) in bytes.
static bool gemv_nibble_plan(const ActPlan& ap) {
  return ap.c[0] == 4 && (ap.S == 1 || ap.c[1] == 8);
}

// Staged rows: M*Kp bytes as bytes; a nibble-path block needs
// M*(32*ng0 + 64*ng1) <= M*Kp, which is all a launch needs when every
// weight block takes the nibble path (2- and 4-bit containers).
static size_t gemv_lds(int64_t M, const ActPlan& ap, const WPlan& wp) {
  const bool all_nib = gemv_nibble_plan(ap) && (wp.c_lo == 2 || wp.c_lo == 4) &&
                       (wp.c_hi == 2 || wp.c_hi == 4);
  const int ng1 = ap.S == 2 ? ap.ng[1] : 0;
  return all_nib ? (size_t)M * (32 * ap.ng[0] + 64 * ng1) : (size_t)M * ap.Kp;
}

bool gemv_fused_fits(const float* A, int64_t K, const ActPlan& ap, const WPlan& wp) {
  const bool sign = ap.q[0].sign1 || (ap.S == 2 && ap.q[1].sign1);
  return gemv_nibble_plan(ap) && !sign && K % 4 == 0 && K / 4 <= 4 * 256 &&
         reinterpret_cast<uintptr_t>(A) % 16 == 0 && gemv_fits(1, ap, wp) &&
         gemv_fused_lds(ap, wp) + (size_t)2048 * 8 <= 64 * 1024;
}

size_t gemv_fused_lds(const ActPlan& ap, const WPlan& wp) {
  return (gemv_lds(1, ap, wp) + 15) / 16 * 16 + (size_t)ap.Kp;
}

hipError_t launch_gemv_fused(const float* A, int64_t K, const uint16_t* pos16_dev, uint8_t* act_packed,
                             float* s_a, const ActPlan& ap, const WDev& wd, const WPlan& wp,
                             int64_t N, uint16_t* Y, int32_t* acc, hipStream_t stream,
                             uint8_t* ximg) {
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, 1, N, Y, N, acc);
  a.ximg = ximg;
  a.a32 = A;
  a.apos16 = pos16_dev;
  a.s_a_out = s_a;
  a.act_out = act_packed;
  a.K4 = (int)(K / 4);
  a.xs_bytes = (int)((gemv_lds(1, ap, wp) + 15) / 16 * 16);
  const dim3 grid((unsigned)wp.nblk);
  const size_t lds = gemv_fused_lds(ap, wp);
  if (a.K4 <= 256) hipLaunchKernelGGL(k_gemv_fused<1>, grid, dim3(256), lds, stream, a);
  else if (a.K4 <= 512) hipLaunchKernelGGL(k_gemv_fused<2>, grid, dim3(256), lds, stream, a);
  else hipLaunchKernelGGL(k_gemv_fused<4>, grid, dim3(256), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_mp_gemv(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                          uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream,
                          const uint8_t* ximg) {
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  if (M == 1) a.ximg = const_cast<uint8_t*>(ximg);
  dim3 grid((unsigned)wp.nblk);
  const size_t lds = gemv_lds(M, ap, wp);
  // Batches of 2..8 rows: the products on matrix cores.  SONIQ_GEMV_MFMA
  // (0: never, 2: for single rows too) overrides the choice for
  // measurement; results are the same.
  bool mfma = M >= 2;
  if (const char* env = getenv("SONIQ_GEMV_MFMA")) mfma = atoi(env) == 2 || (mfma && atoi(env) != 0);
  if (gemv_nibble_plan(ap) && mfma && gemv_mfma_fits(wp)) {
    hipLaunchKernelGGL(k_gemv_mfma, grid, dim3(256), gemv_mfma_lds(wp), stream, a);
  } else if (gemv_nibble_plan(ap)) {
    if (M == 1) hipLaunchKernelGGL(k_gemv<1>, grid, dim3(256), lds, stream, a);
    else if (M == 2) hipLaunchKernelGGL(k_gemv<2>, grid, dim3(256), lds, stream, a);
    else if (M <= 4) hipLaunchKernelGGL(k_gemv<4>, grid, dim3(256), lds, stream, a);
    else hipLaunchKernelGGL(k_gemv<8>, grid, dim3(256), lds, stream, a);
  } else {
    if (M == 1) hipLaunchKernelGGL(k_gemv_any<1>, grid, dim3(256), lds, stream, a);
    else if (M == 2) hipLaunchKernelGGL(k_gemv_any<2>, grid, dim3(256), lds, stream, a);
    else if (M <= 4) hipLaunchKernelGGL(k_gemv_any<4>, grid, dim3(256), lds, stream, a);
    else hipLaunchKernelGGL(k_gemv_any<8>, grid, dim3(256), lds, stream, a);
  }
  return hipGetLastError();
}

// The block-sum GEMV (sub-group scales, batches of at most 8 rows): a
// 4-bit group 0 and an 8-bit group 1, weight containers 2, 4 or 8, and
// the staged rows plus the block sums within 64 KB of LDS.
static size_t gemv_g_lds(int64_t M, const ActPlan& ap, const WPlan& wp) {
  const int64_t MT = M == 1 ? 1 : M == 2 ? 2 : M <= 4 ? 4 : 8;
  const int nsub = ap.nsub[0] + (ap.S == 2 ? ap.nsub[1] : 0);
  return (gemv_lds(M, ap, wp) + 15) / 16 * 16 + (size_t)nsub * MT * kBlk * 4;
}

bool gemv_g_fits(int64_t M, const ActPlan& ap, const WPlan& wp) {
  return gemv_fits(M, ap, wp) && gemv_nibble_plan(ap) && ap.zp[0] == 0 &&
         (ap.S == 1 || ap.zp[1] == 0) && wp.c_lo != 1 && wp.c_hi != 1 &&
         gemv_g_lds(M, ap, wp) + (size_t)2048 * 8 <= 64 * 1024;
}

hipError_t launch_mp_gemv_grouped(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                  const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                                  uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream) {
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  a.xs_bytes = (int)((gemv_lds(M, ap, wp) + 15) / 16 * 16);
  const dim3 grid((unsigned)wp.nblk);
  const size_t lds = gemv_g_lds(M, ap, wp);
  if (M == 1) hipLaunchKernelGGL(k_gemv_g<1>, grid, dim3(256), lds, stream, a);
  else if (M == 2) hipLaunchKernelGGL(k_gemv_g<2>, grid, dim3(256), lds, stream, a);
  else if (M <= 4) hipLaunchKernelGGL(k_gemv_g<4>, grid, dim3(256), lds, stream, a);
  else hipLaunchKernelGGL(k_gemv_g<8>, grid, dim3(256), lds, stream, a);
  return hipGetLastError();
}

// Sub-group scales: partial block maxima over row ranges of at least 8
// rows (at most kGAbsParts of them), block scales, then codes.
hipError_t launch_act_quant_grouped(const float* A, int64_t M, int64_t K, int64_t lda,
                                    const ActPlan& ap, const int32_t* pos_dev,
                                    const int32_t* grp_dev, const int32_t* posg_dev,
                                    float* partial, unsigned int* counter, float* s_a,
                                    uint8_t* packed, hipStream_t stream) {
  const int nsub = ap.nsub[0] + (ap.S == 2 ? ap.nsub[1] : 0);
  const size_t tab = (size_t)nsub * 8;
  const bool aligned = (K % 4 == 0) && (lda % 4 == 0) && (reinterpret_cast<uintptr_t>(A) % 16 == 0);
  // one pass over the rows when the batch fits one resident grid
  if (aligned && M * K >= kCoopMinElems) {
    hipError_t e = hipSuccess;
    if (launch_act_coop(A, M, K, lda, ap, posg_dev, counter, s_a, packed, stream, e, true)) return e;
  }
  const int K4 = (int)(K / 4);
  const int J = (K4 + 255) / 256;
  if (aligned && J <= 4 && M <= 8 && (size_t)ap.Kp + 3 * tab / 2 <= 64 * 1024) {
    // decode batches: one launch, every row loaded once per workgroup
    const size_t lds = (size_t)ap.Kp + (size_t)nsub * 12;
    const float4* A4 = reinterpret_cast<const float4*>(A);
    const int4* g4 = reinterpret_cast<const int4*>(grp_dev);
    const int4* p4 = reinterpret_cast<const int4*>(pos_dev);
#define SONIQ_GR(J_, MT_)                                                                      \
  hipLaunchKernelGGL((k_gact_rows<J_, MT_>), dim3((unsigned)M), dim3(256), lds, stream, A4, (int)M, \
                     K4, lda / 4, p4, g4, ap, nsub, s_a, packed)
#define SONIQ_GR_J(MT_)                                                                     \
  if (J == 1) SONIQ_GR(1, MT_); else if (J == 2) SONIQ_GR(2, MT_); else if (J == 3) SONIQ_GR(3, MT_); \
  else SONIQ_GR(4, MT_)
    if (M == 1) { SONIQ_GR_J(1); }
    else if (M == 2) { SONIQ_GR_J(2); }
    else if (M <= 4) { SONIQ_GR_J(4); }
    else { SONIQ_GR_J(8); }
#undef SONIQ_GR_J
#undef SONIQ_GR
    return hipGetLastError();
  }
  if (aligned && J <= 4) {
    // four rows per workgroup at least, else up to kGAbsParts row ranges
    const int64_t rpb = std::max<int64_t>(4, (M + kGAbsParts - 1) / kGAbsParts);
    const int nparts = (int)((M + rpb - 1) / rpb);
    const float4* A4 = reinterpret_cast<const float4*>(A);
    const int4* g4 = reinterpret_cast<const int4*>(grp_dev);
    const int4* p4 = reinterpret_cast<const int4*>(pos_dev);
#define SONIQ_GABS(J_)                                                                              \
  hipLaunchKernelGGL(k_gabsmax4<J_>, dim3((unsigned)nparts), dim3(256), (size_t)nsub * 4, stream, A4, \
                     M, K4, lda / 4, rpb, g4, nsub, partial)
    if (J == 1) SONIQ_GABS(1); else if (J == 2) SONIQ_GABS(2); else if (J == 3) SONIQ_GABS(3); else SONIQ_GABS(4);
#undef SONIQ_GABS
    hipLaunchKernelGGL(k_gscales, dim3((unsigned)nsub), dim3(256), 0, stream, partial, nparts, nsub,
                       ap, s_a);
    const int R = 8 * (size_t)ap.Kp + tab <= 64 * 1024 ? 8 : 4;
    if (R * (size_t)ap.Kp + tab <= 64 * 1024) {
      const size_t lds = R * (size_t)ap.Kp + tab;
      const dim3 grid((unsigned)((M + R - 1) / R));
#define SONIQ_GQ(R_, J_) \
  hipLaunchKernelGGL((k_gquant4<R_, J_>), grid, dim3(256), lds, stream, A4, M, K4, lda / 4, p4, g4, ap, nsub, s_a, packed)
      if (R == 8) {
        if (J == 1) SONIQ_GQ(8, 1); else if (J == 2) SONIQ_GQ(8, 2); else if (J == 3) SONIQ_GQ(8, 3); else SONIQ_GQ(8, 4);
      } else {
        if (J == 1) SONIQ_GQ(4, 1); else if (J == 2) SONIQ_GQ(4, 2); else if (J == 3) SONIQ_GQ(4, 3); else SONIQ_GQ(4, 4);
      }
#undef SONIQ_GQ
      return hipGetLastError();
    }
    hipLaunchKernelGGL(k_gquant<1>, dim3((unsigned)M), dim3(256), (size_t)ap.Kp + tab, stream, A, M,
                       K, lda, pos_dev, grp_dev, ap, nsub, s_a, packed);
    return hipGetLastError();
  }
  const int64_t rpb = std::max<int64_t>(8, (M + kGAbsParts - 1) / kGAbsParts);
  const int nparts = (int)((M + rpb - 1) / rpb);
  hipLaunchKernelGGL(k_gabsmax, dim3((unsigned)nparts), dim3(256), (size_t)nsub * 4, stream, A, M, K,
                     lda, rpb, grp_dev, nsub, partial);
  hipLaunchKernelGGL(k_gscales, dim3((unsigned)nsub), dim3(256), 0, stream, partial, nparts, nsub, ap,
                     s_a);
  if (kBlk * (size_t)ap.Kp + tab <= 64 * 1024)
    hipLaunchKernelGGL(k_gquant<kBlk>, dim3((unsigned)((M + kBlk - 1) / kBlk)), dim3(256),
                       kBlk * (size_t)ap.Kp + tab, stream, A, M, K, lda, pos_dev, grp_dev, ap, nsub,
                       s_a, packed);
  else if (4 * (size_t)ap.Kp + tab <= 64 * 1024)
    hipLaunchKernelGGL(k_gquant<4>, dim3((unsigned)((M + 3) / 4)), dim3(256), 4 * (size_t)ap.Kp + tab,
                       stream, A, M, K, lda, pos_dev, grp_dev, ap, nsub, s_a, packed);
  else
    hipLaunchKernelGGL(k_gquant<1>, dim3((unsigned)M), dim3(256), (size_t)ap.Kp + tab, stream, A, M,
                       K, lda, pos_dev, grp_dev, ap, nsub, s_a, packed);
  return hipGetLastError();
}

hipError_t launch_mp_gemm_grouped(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                  const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                                  uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream) {
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  const int64_t tiles = ((M + 63) / 64) * (wp.Np / kGemmBN);
  a.xcd_tiles = tiles <= 2048;
  const dim3 grid((unsigned)tiles), blk(256);
  const int cl = wp.c_lo, ch = wp.c_hi;
  if (ap.S == 2 && ap.c[0] == 4 && ap.c[1] == 8) {
    if (cl == 4 && ch == 8) hipLaunchKernelGGL((k_gemm_g<2, 4, 8, 4, 8>), grid, blk, 0, stream, a);
    else if (cl == 2 && ch == 8) hipLaunchKernelGGL((k_gemm_g<2, 4, 8, 2, 8>), grid, blk, 0, stream, a);
    else if (cl == 1 && ch == 4) hipLaunchKernelGGL((k_gemm_g<2, 4, 8, 1, 4>), grid, blk, 0, stream, a);
    else if (cl == 2 && ch == 4) hipLaunchKernelGGL((k_gemm_g<2, 4, 8, 2, 4>), grid, blk, 0, stream, a);
    else hipLaunchKernelGGL((k_gemm_g<2, 4, 8, 0, 0>), grid, blk, 0, stream, a);
  } else if (ap.S == 2) {
    hipLaunchKernelGGL((k_gemm_g<2, 0, 0, 0, 0>), grid, blk, 0, stream, a);
  } else {
    hipLaunchKernelGGL((k_gemm_g<1, 0, 0, 0, 0>), grid, blk, 0, stream, a);
  }
  return hipGetLastError();
}

// ----------------------------------------------------------- k_conv_img --
// Haloed code image of a convolution input X[B][C][H][W] (implicit GEMM):
// item j of group g is unit u = j / HP (channels of rank 16u .. 16u+15) of
// haloed pixel hp = j % HP, so consecutive threads take consecutive pixels
// and each of the 16 channel loads coalesces.  Halo pixels hold the stored
// code of 0.0 and ranks past the group the stored 0 of padding; every code
// is the group quantizer's (store_code) with the group scale reduced from
// the partial maxima.
__global__ __launch_bounds__(256) void k_conv_img(const float* __restrict__ X, int C, int H, int W,
                                                  int HP, const int32_t* __restrict__ chan,
                                                  const float* __restrict__ partial, int nparts,
                                                  ActPlan ap, ConvGeo cg, uint8_t* __restrict__ img,
                                                  float* __restrict__ s_a_out) {
  __shared__ float red[8];
  float s0, s1;
  scales_from_partials(partial, nparts, ap, red, s0, s1, s_a_out);  // syncs
  const ActQ aq = make_actq(ap, s0, s1);
  const int u0 = cg.cpad[0] / 16, u1 = ap.S == 2 ? cg.cpad[1] / 16 : 0;
  const int n0 = HP * u0, total = n0 + HP * u1;
  const int Wp = W + 2, HPi = (H + 2) * Wp;
  for (int i = (int)(blockIdx.x * 256 + threadIdx.x); i < total; i += (int)(gridDim.x * 256)) {
    const int g = i >= n0 ? 1 : 0;
    const int j = g ? i - n0 : i;
    const int u = j / HP, hp = j - u * HP;
    const int b = hp / HPi, rem = hp - b * HPi;
    const int yh = rem / Wp, xh = rem - yh * Wp;
    const bool halo = yh == 0 || yh == H + 1 || xh == 0 || xh == W + 1;
    // every load unconditional and in bounds (a halo pixel or a padding
    // rank reads pixel (0, 0) of channel 0 and discards it), so all 16 are
    // in flight at once
    const int64_t pix = halo ? 0 : (int64_t)(yh - 1) * W + (xh - 1);
    int cc[16];
    float xv[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) cc[e] = chan[g * cg.chan_ld + 16 * u + e];
#pragma unroll
    for (int e = 0; e < 16; ++e) xv[e] = X[((int64_t)b * C + max(cc[e], 0)) * H * W + pix];
    uint32_t d[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      // padding rank: stored 0; halo: the code of 0.0
      const uint32_t byte = cc[e] < 0 ? 0u : store_code(halo ? 0.0f : xv[e], g, aq);
      d[e >> 2] |= byte << (8 * (e & 3));
    }
    const int c = ap.c[g];
    uint8_t* dst = img + cg.img_off[g] + (int64_t)hp * cg.rowbytes[g] + u * 2 * c;
    store_unit(dst, pack_unit(d[0], d[1], d[2], d[3], c), c);
  }
}

hipError_t launch_conv_img(const float* X, int64_t B, int64_t C, int64_t H, int64_t W,
                           const ActPlan& ap, const ConvGeo& cg, const uint8_t* seg_dev,
                           const int32_t* chan_dev, float* partial, float* s_a, uint8_t* img,
                           hipStream_t stream) {
  const int64_t BC = B * C;
  const int64_t rows_per_block = 4 * kAbsR;
  const int64_t nparts = (BC + rows_per_block - 1) / rows_per_block < kAbsmaxBlocks
                             ? (BC + rows_per_block - 1) / rows_per_block
                             : kAbsmaxBlocks;
  hipLaunchKernelGGL(k_conv_absmax, dim3((unsigned)nparts), dim3(256), 0, stream, X, (int)BC, (int)C,
                     (int)(H * W), seg_dev, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t HP = B * (H + 2) * (W + 2);
  const int64_t units = cg.cpad[0] / 16 + (ap.S == 2 ? cg.cpad[1] / 16 : 0);
  const int64_t total = HP * units;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_conv_img, dim3((unsigned)blocks), dim3(256), 0, stream, X, (int)C, (int)H,
                     (int)W, (int)HP, chan_dev, partial, (int)nparts, ap, cg, img, s_a);
  return hipGetLastError();
}

template <int CBL, int CBH>
static void launch_gemm_conv_t(const GemmArgs& a, int64_t M, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  hipLaunchKernelGGL((k_gemm<2, 4, 8, CBL, CBH, 2, 2, 0, false, true>),
                     dim3((unsigned)(((M + 63) / 64) * ntn)), dim3(256), 0, stream, a);
}

// One activation width in 4- or 8-bit containers: the tiles with S = 1.
template <int CA>
static void launch_gemm_conv1(const GemmArgs& a, int64_t M, hipStream_t stream) {
  const int ntn = a.wp.Np / kGemmBN;
  const dim3 grid((unsigned)(((M + 63) / 64) * ntn));
  const int cl = a.wp.c_lo, ch = a.wp.c_hi;
#define SONIQ_CONV1(L_, H_) hipLaunchKernelGGL((k_gemm<1, CA, 0, L_, H_, 2, 2, 0, false, true>), grid, dim3(256), 0, stream, a)
  if (cl == 4 && ch == 4) SONIQ_CONV1(4, 4);
  else if (cl == 1 && ch == 4) SONIQ_CONV1(1, 4);
  else if (cl == 2 && ch == 4) SONIQ_CONV1(2, 4);
  else if (cl == 2 && ch == 8) SONIQ_CONV1(2, 8);
  else if (cl == 8 && ch == 8) SONIQ_CONV1(8, 8);
  else if (cl == 1 && ch == 8) SONIQ_CONV1(1, 8);
  else if (cl == 2 && ch == 2) SONIQ_CONV1(2, 2);
  else if (cl == 1 && ch == 2) SONIQ_CONV1(1, 2);
  else if (cl == 1 && ch == 1) SONIQ_CONV1(1, 1);
  else SONIQ_CONV1(4, 8);
#undef SONIQ_CONV1
}

// Every pair of weight containers (c_lo <= c_hi, powers of two up to 8).
static bool conv_wpair_ok(const WPlan& wp) {
  const int cl = wp.c_lo, ch = wp.c_hi;
  return cl >= 1 && ch >= cl && ch <= 8 && (cl & (cl - 1)) == 0 && (ch & (ch - 1)) == 0;
}

bool conv_gemm_qn_supported(const ActPlan& ap, const WPlan& wp) {
  return ap.S == 2 && ap.c[0] == 4 && ap.c[1] == 8 && conv_wpair_ok(wp);
}

bool conv_gemm_supported(const ActPlan& ap, const WPlan& wp) {
  return conv_gemm_qn_supported(ap, wp) ||
         (ap.S == 1 && (ap.c[0] == 4 || ap.c[0] == 8) && conv_wpair_ok(wp));
}

hipError_t launch_mp_gemm_conv(const uint8_t* img, const ConvGeo& cg, const float* s_a,
                               const ActPlan& ap, const WDev& wd, const WPlan& wp, int64_t M,
                               int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc,
                               hipStream_t stream) {
  if (!conv_gemm_supported(ap, wp)) return hipErrorInvalidValue;
  GemmArgs a = make_args(nullptr, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  a.img = img;
  a.cg = cg;
  const int64_t tiles = ((M + 63) / 64) * (wp.Np / kGemmBN);
  a.xcd_tiles = tiles <= 2048;
  if (ap.S == 1) {
    if (ap.c[0] == 4) launch_gemm_conv1<4>(a, M, stream);
    else launch_gemm_conv1<8>(a, M, stream);
    return hipGetLastError();
  }
  const int cl = wp.c_lo, ch = wp.c_hi;
  if (cl == 4 && ch == 4) launch_gemm_conv_t<4, 4>(a, M, stream);
  else if (cl == 1 && ch == 4) launch_gemm_conv_t<1, 4>(a, M, stream);
  else if (cl == 2 && ch == 4) launch_gemm_conv_t<2, 4>(a, M, stream);
  else if (cl == 2 && ch == 8) launch_gemm_conv_t<2, 8>(a, M, stream);
  else if (cl == 8 && ch == 8) launch_gemm_conv_t<8, 8>(a, M, stream);
  else if (cl == 1 && ch == 8) launch_gemm_conv_t<1, 8>(a, M, stream);
  else if (cl == 2 && ch == 2) launch_gemm_conv_t<2, 2>(a, M, stream);
  else if (cl == 1 && ch == 2) launch_gemm_conv_t<1, 2>(a, M, stream);
  else if (cl == 1 && ch == 1) launch_gemm_conv_t<1, 1>(a, M, stream);
  else launch_gemm_conv_t<4, 8>(a, M, stream);
  return hipGetLastError();
}

// ------------------------------------------------------------ k_to_fp --
// Integer units -> MFMA-native copy.  One thread per (block, fgranule,
// lane): lane l = q*16 + r takes row r, channels [32q, 32q + 32) of the
// fgranule, which are elements of two units of granule 2f + q/2 (16-channel
// groups 2(q%2) and 2(q%2) + 1); it decodes the 32 stored codes exactly as
// the GEMM widens them (two's complement fields, or sign bits +-1) and
// encodes each in fp4 (e2m1) or fp6 (e3m2).  Channels past the group's last
// granule (half of a final fgranule) encode 0.
__device__ __forceinline__ int unit_code(const uint32_t (&w)[2], int e, int c) {
  if (c == 4) {
    const int v = (int)((w[e >> 3] >> (8 * (e & 3) + 4 * ((e >> 2) & 1))) & 0xFu);
    return v >= 8 ? v - 16 : v;
  }
  if (c == 2) {
    const int j = e >> 2;
    const int v = (int)((w[0] >> (8 * (e & 3) + 4 * (j & 1) + (j < 2 ? 2 : 0))) & 0x3u);
    return v >= 2 ? v - 4 : v;
  }
  return ((w[0] >> (4 * (e & 3) + (e >> 2))) & 1u) ? -1 : 1;  // c == 1: sign bits
}

// e2m1: 0, 1 = 1.0 (exponent 1), 2 = 2.0 (exponent 2); bit 3 is the sign.
__device__ __forceinline__ uint32_t enc_fp4(int v) {
  const int m = v < 0 ? -v : v;
  return (m == 0 ? 0u : m == 1 ? 0x2u : 0x4u) | (v < 0 ? 0x8u : 0u);
}
// e3m2 (exponent bias 3): |v| = 2^(E-3) * (1 + M/4) for |v| in 1..8; bit 5 is
// the sign.
__device__ __forceinline__ uint32_t enc_fp6(int v) {
  const int m = v < 0 ? -v : v;
  uint32_t code = 0;
  if (m > 0) {
    const int e = 31 - __builtin_clz((unsigned)m);     // 2^e <= m < 2^(e+1)
    const int mant = ((m << 2) >> e) & 3;              // exact for m <= 8
    code = (uint32_t)((e + 3) << 2 | mant);
  }
  return code | (v < 0 ? 0x20u : 0u);
}

// Four (block, fgranule) pairs per workgroup, one per wave; containers and
// formats fixed at compile time, so each lane's 32 elements are a
// straight-line sequence of shifts and masks.
template <int C, int FMT>
__global__ __launch_bounds__(256) void k_to_fp(const uint8_t* __restrict__ src, int64_t src_bstride,
                                               int ng, int npairs, uint8_t* __restrict__ dst,
                                               int64_t dst_bstride) {
  const int nfg = (ng + 1) / 2;
  const int p = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6);
  if (p >= npairs) return;
  const int lane = threadIdx.x & 63;
  const int b = p / nfg, f = p - b * nfg;
  const int q = lane >> 4, r = lane & 15;
  const int gi = 2 * f + (q >> 1);
  uint32_t d[6] = {0u, 0u, 0u, 0u, 0u, 0u};
  if (gi < ng) {
    const uint8_t* gbase = src + b * src_bstride + (int64_t)gi * 128 * C;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint8_t* u = gbase + ((2 * (q & 1) + h) * 16 + r) * 2 * C;
      uint32_t w[2] = {0u, 0u};
      if constexpr (C == 4) {
        const uint2 v = *reinterpret_cast<const uint2*>(u);
        w[0] = v.x;
        w[1] = v.y;
      } else if constexpr (C == 2) {
        w[0] = *reinterpret_cast<const uint32_t*>(u);
      } else {
        w[0] = *reinterpret_cast<const uint16_t*>(u);
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int v = unit_code(w, e, C);
        const int el = 16 * h + e;  // element of the lane's 32
        if constexpr (FMT == kFmtFp4) {
          d[el >> 3] |= enc_fp4(v) << (4 * (el & 7));
        } else {
          const uint32_t code = enc_fp6(v);
          const int pos = 6 * el, wd = pos >> 5, sh = pos & 31;
          d[wd] |= code << sh;
          if (sh > 26) d[wd + 1] |= code >> (32 - sh);
        }
      }
    }
  }
  uint8_t* o = dst + b * dst_bstride + (int64_t)f * f_block_bytes(FMT);
  *reinterpret_cast<uint4*>(o + 16 * lane) = make_uint4(d[0], d[1], d[2], d[3]);
  if constexpr (FMT == kFmtFp6) *reinterpret_cast<uint2*>(o + 1024 + 8 * lane) = make_uint2(d[4], d[5]);
}

// ---------------------------------------------------------- dense weights --
// The dense copy (layout in soniq_internal.h): thread (block, run u, row r)
// reads the two 16-channel units of its run from the block's units, decodes
// their 32 codes, slices their b-bit fields into the four byte lanes and
// writes the run's b words into its record's chunks.  Runs past the planned
// K (the half of a last 128-channel quad-run) are written as zeros.
__global__ __launch_bounds__(256) void k_dense_pack(const uint8_t* __restrict__ packed, WPlan wp,
                                                    int b_lo, int b_hi, uint8_t* __restrict__ dense) {
  const int nrun = wp.ngt * 2, nquad = dense_nquad(wp), nru = 4 * nquad;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)nru * kBlk * wp.nblk) return;
  const int blk = (int)(i / ((int64_t)nru * kBlk));
  const int rem = (int)(i - (int64_t)blk * nru * kBlk);
  const int u = rem / kBlk, r = rem - u * kBlk;
  const int c = wblk_c(wp, blk), b = dense_b(wp, blk, b_lo, b_hi);
  int code[32];
  for (int e = 0; e < 32; ++e) code[e] = 0;
  if (u < nrun) {
    const uint8_t* gran = packed + wblk_off(wp, blk) + (int64_t)(u >> 1) * 128 * c;
    for (int h = 0; h < 2; ++h) {
      const uint8_t* unit = gran + ((u & 1) * 32 + h * 16 + r) * 2 * c;  // 16-channel group 2(u&1)+h
      uint32_t w2[2] = {0u, 0u};
      uint4 w8 = make_uint4(0u, 0u, 0u, 0u);
      if (c == 8) w8 = *reinterpret_cast<const uint4*>(unit);
      else if (c == 4) { const uint2 t = *reinterpret_cast<const uint2*>(unit); w2[0] = t.x; w2[1] = t.y; }
      else if (c == 2) w2[0] = *reinterpret_cast<const uint32_t*>(unit);
      else w2[0] = *reinterpret_cast<const uint16_t*>(unit);
      const uint32_t w8a[4] = {w8.x, w8.y, w8.z, w8.w};
      for (int e = 0; e < 16; ++e)
        code[16 * h + e] = c == 8 ? (int)(int8_t)(w8a[e >> 2] >> (8 * (e & 3))) : unit_code(w2, e, c);
    }
  }
  // field 4q + e is field q of byte lane e; lane e's 8 fields form a string
  // of 8b bits whose byte k goes to byte e of word k
  uint32_t out[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
  const uint32_t mask = (1u << b) - 1u;
  if (u < nrun) {
    for (int e = 0; e < 4; ++e)
      for (int q = 0; q < 8; ++q) {
        const int cd = code[4 * q + e];
        const uint32_t f = b == 1 ? (cd < 0 ? 1u : 0u) : ((uint32_t)cd & mask);
        const int bit = q * b, k = bit >> 3, off = bit & 7;
        out[k] |= ((f << off) & 0xFFu) << (8 * e);
        if (off + b > 8) out[k + 1] |= (f >> (8 - off)) << (8 * e);
      }
  }
  // record (quad-run v, row r): word w = (u % 4) * b + j of its 4b words
  const int v = u >> 2, bi = v >> 4, vl = v & 15, ni = min(16, nquad - 16 * bi);
  uint8_t* base = dense + dense_off(wp, blk, b_lo, b_hi);
  for (int j = 0; j < b; ++j) {
    const int w = (u & 3) * b + j;
    const int64_t chunk = (int64_t)256 * b * bi + 16 * ni * (w >> 2) + 16 * vl + r;
    *reinterpret_cast<uint32_t*>(base + chunk * 16 + (w & 3) * 4) = out[j];
  }
}

hipError_t launch_dense_pack(const uint8_t* packed, const WPlan& wp, int b_lo, int b_hi,
                             uint8_t* dense, hipStream_t stream) {
  const int64_t n = (int64_t)4 * dense_nquad(wp) * kBlk * wp.nblk;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_dense_pack, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, packed, wp,
                     b_lo, b_hi, dense);
  return hipGetLastError();
}

// Bits lo .. hi-1 of every byte.
__host__ __device__ constexpr uint32_t byte_bits(int lo, int hi) {
  return ((((1u << hi) - 1u) & ~((1u << lo) - 1u)) & 0xFFu) * 0x01010101u;
}

// Exponent of the scale the dense products carry: every field sits in the
// top bits of its byte (b = 1 as the two-bit string 01 or 11, i.e. +1 or -1
// times 64), so a dot4 product is 2^dense_wsh times the true one.
__host__ __device__ constexpr int dense_wsh(int b) { return b == 1 ? 6 : 8 - b; }

// A run's 32 fields (b words w, byte-sliced) as 8 words of four int8 values
// for v_dot4_i32_i8, word q holding fields 4q .. 4q+3: one shift and mask
// for a field that lies in one byte of its lane's string, two of each for
// one that straddles two bytes; the byte lanes never mix.
template <int B>
__device__ __forceinline__ void dense_top(const uint32_t* w, uint32_t (&o)[8]) {
  if constexpr (B == 8) {
#pragma unroll
    for (int q = 0; q < 8; ++q) o[q] = w[q];
  } else if constexpr (B == 1) {
#pragma unroll
    for (int q = 0; q < 8; ++q) o[q] = ((w[0] << (7 - q)) & 0x80808080u) | 0x40404040u;
  } else {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int bit = q * B, k = bit >> 3, off = bit & 7;
      if (off + B <= 8) {
        o[q] = (w[k] << (8 - B - off)) & byte_bits(8 - B, 8);
      } else {
        const int s1 = off + B - 8, s2 = 16 - B - off;
        o[q] = ((w[k] >> s1) & byte_bits(8 - B, s2)) | ((w[k + 1] << s2) & byte_bits(s2, 8));
      }
    }
  }
}

// One block of width B.  Thread t takes row t % 16 and quad-run t / 16 of
// each batch of 16 quad-runs (its b 16-byte chunks, coalesced across the
// workgroup).  The activation units are loaded first, then the first two
// batches of chunks, so staging the units (rows xld bytes apart, then 32
// zero bytes) waits for the units only; later batches are issued as a
// batch's registers free up.  Products run on v_mfma_i32_16x16x64_i8 with
// the block's decoded rows as B (lane l: row l % 16, its run of lane group
// g = l / 16) and as A row c = 2m + j the staged channels of batch row m
// that lie in activation group j, zeros elsewhere: lane l reads the run's
// bytes of batch row (l % 16) / 2 where the run is in group (l % 16) % 2,
// else the zero bytes.  So one accumulator holds both groups' sums and
// every lane group contributes its own run.
// Sign weights (B = 1) against a sign activation group: the run's product
// is 32 - 2 popcount(X ^ W), X and W the runs' 32 sign bits (set for -1)
// in the same byte-sliced order, summed per thread in xacc (true units);
// those lanes feed zeros to the matrix product.  X is staged beside the
// byte rows as two words per run and batch row (one per 16-channel unit:
// its nibbles spread to the low halves of four bytes, shifted by 4 for
// the run's second unit), at xbits.
template <int MT, int B>
__device__ __forceinline__ void gemv_dense_block(const GemmArgs& a, uint8_t* xs, int xld, int blk,
                                                 int xbits, v4i& acc, int (&xacc)[MT]) {
  const int tid = threadIdx.x, lane = tid & 63, vl = tid >> 4;
  const int nrun = a.ap.Kp >> 5, kp0 = a.ap.kpad[0];
  const int nquad = dense_nquad(a.wp), nbat = (nquad + 15) >> 4;
  const int M = (int)a.M;
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(a.dense + dense_off(a.wp, blk, a.db_lo, a.db_hi)), (short)0, 256 * B * nquad, 0x00020000);
  auto issue = [&](int i, uint4 (&c)[B]) __attribute__((always_inline)) {
    const int ni = i < nbat ? min(16, nquad - 16 * i) : 0;
    const bool ok = vl < ni;
#pragma unroll
    for (int j = 0; j < B; ++j)
      c[j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                           wr, ok ? (uint32_t)(256 * B * i + 16 * ni * j + tid) * 16 : kOOB,
                                           0, 0));
  };
  const int xm = (lane & 15) >> 1, xg = lane & 1;
  const int xrow = xm < M ? xm * xld : -1;
  const int xzero = M * xld;
  // the sign activation group, if any (XNOR runs need B = 1 weights)
  const int sgrp = B != 1 ? -1 : a.ap.c[0] == 1 ? 0 : a.ap.S == 2 && a.ap.c[1] == 1 ? 1 : -1;
  const uint2* xb2 = reinterpret_cast<const uint2*>(xs + xbits);
  auto consume = [&](int i, const uint4 (&c)[B]) __attribute__((always_inline)) {
    uint32_t w[4 * B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      w[4 * j] = c[j].x;
      w[4 * j + 1] = c[j].y;
      w[4 * j + 2] = c[j].z;
      w[4 * j + 3] = c[j].w;
    }
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int u = 4 * (16 * i + vl) + q4;
      const int ug = 32 * u >= kp0 ? 1 : 0;
      const bool xn = B == 1 && u < nrun && ug == sgrp;
      if constexpr (B == 1) {
        if (xn) {
#pragma unroll
          for (int mm = 0; mm < MT; ++mm) {
            if (mm < M) {
              const uint2 xw = xb2[mm * nrun + u];
              xacc[mm] += 32 - 2 * (int)__popc((xw.x | xw.y) ^ w[q4]);
            }
          }
        }
      }
      // runs past the planned K, rows past the batch, the other group's
      // lanes and the sign runs read the zero bytes
      const bool on = u < nrun && xrow >= 0 && ug == xg && !xn;
      const int xoff = on ? xrow + 32 * u : xzero;
      uint32_t o[8];
      dense_top<B>(w + q4 * B, o);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 x = *reinterpret_cast<const uint4*>(xs + xoff + 16 * h);
        const v4i wf = v4i{(int)o[4 * h], (int)o[4 * h + 1], (int)o[4 * h + 2], (int)o[4 * h + 3]};
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(frag_of(x), wf, acc, 0, 0, 0);
      }
    }
  };
  // Every unit is read as 16 bytes (its 2c bytes used) through a buffer
  // over both groups' first 16-row blocks: one load per unit whatever its
  // container, past the end read as zero.
  constexpr int XR = gemv_xr<MT>();
  const int ngt = a.wp.ngt, xd = ngt * 4, xtotal = M * xd, ng0 = a.ap.ng[0];
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)a.act, (short)0, gemv_dense_xbytes(a.ap), 0x00020000);
  // unit u (< xtotal): batch row m, granule q, 16-channel group kg; its
  // byte offset in the activation buffer, container and staged offset
  // and, for sign runs, the offset of its bit word
  auto xunit = [&](int u, uint32_t& off, int& c, int& dst, int& bdst) __attribute__((always_inline)) {
    const int m = MT == 1 ? 0 : gemv_row_of<MT>(u, xd);
    const int rest = u - m * xd, q = rest >> 2, kg = rest & 3;
    const bool g1 = q >= ng0;
    c = g1 ? a.ap.c[1] : a.ap.c[0];
    off = (uint32_t)((g1 ? a.ap.seg_off[1] : a.ap.seg_off[0]) + (g1 ? q - ng0 : q) * 128 * c +
                     (kg * 16 + m) * 2 * c);
    dst = m * xld + q * kGran + kg * 16;
    bdst = xbits + 8 * (m * nrun + 2 * q + (kg >> 1)) + 4 * (kg & 1);
  };
  auto stage = [&](uint4 raw, int c, int dst, int bdst) __attribute__((always_inline)) {
    *reinterpret_cast<uint4*>(xs + dst) = unpack_unit_rt(raw, c);
    if (B == 1 && c == 1 && sgrp >= 0) {
      const uint32_t h = raw.x & 0xFFFFu;
      const uint32_t t = (h | (h << 8)) & 0x00FF00FFu;
      const uint32_t y = (t | (t << 4)) & 0x0F0F0F0Fu;  // byte b = nibble b of the unit
      *reinterpret_cast<uint32_t*>(xs + bdst) = (bdst & 4) ? y << 4 : y;
    }
  };
  uint4 xr[XR];
  int xc[XR], xdst[XR], xbd[XR];
#pragma unroll
  for (int k = 0; k < XR; ++k) {
    const int u = tid + 256 * k;
    uint32_t off = 0;
    xunit(min(u, xtotal - 1), off, xc[k], xdst[k], xbd[k]);
    xr[k] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xrs, u < xtotal ? off : kOOB, 0, 0));
  }
  // keep the units' loads ahead of the weights' in the issue order
  __builtin_amdgcn_sched_barrier(0);
  uint4 c0[B], c1[B];
  issue(0, c0);
  issue(1, c1);
  __builtin_amdgcn_sched_barrier(0);
  if (tid < 2) *reinterpret_cast<uint4*>(xs + xzero + 16 * tid) = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
  for (int k = 0; k < XR; ++k)
    if (tid + 256 * k < xtotal) stage(xr[k], xc[k], xdst[k], xbd[k]);
  for (int u = tid + 256 * XR; u < xtotal; u += 256) {
    uint32_t off = 0;
    int c = 0, dst = 0, bdst = 0;
    xunit(u, off, c, dst, bdst);
    stage(load_unit(a.act + off, c), c, dst, bdst);
  }
  __syncthreads();
  for (int i = 0; i < nbat; i += 2) {
    consume(i, c0);
    if (i + 2 < nbat) issue(i + 2, c0);
    if (i + 1 < nbat) {
      consume(i + 1, c1);
      if (i + 3 < nbat) issue(i + 3, c1);
    }
  }
}

// The GEMV on the dense copy: one workgroup per 16-row block, batches of
// up to 8 rows; the block's quad-runs as above, the four waves' 16x16 sums
// met in LDS (sum row 2m + j: batch row m, activation group j) and the
// epilogue of k_gemv (the field scale 2^dense_wsh taken out with the
// activations' unpack shift).  Dynamic LDS: M rows of Kp + 16 bytes (the
// pad spreads the rows over the banks) and 32 zero bytes.
template <int MT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(MT >= 4 ? 3 : 4))) void k_gemv_dense(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];
  __shared__ int red[4][4][64];
  __shared__ int redx[4][MT][kBlk];
  const int blk = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const ActPlan& ap = a.ap;
  const int xld = ap.Kp + 16;
  const int xbits = (int)a.M * xld + 32;
  // the epilogue's column, fetched before the weights arrive
  const int pc = blk * kBlk + (lane & 15);
  const ColInfo ci = a.wd.colinfo[pc];
  v4i acc = v4i{0, 0, 0, 0};
  int xacc[MT];
#pragma unroll
  for (int mm = 0; mm < MT; ++mm) xacc[mm] = 0;
  const int b = dense_b(a.wp, blk, a.db_lo, a.db_hi);
  switch (b) {
    case 1: gemv_dense_block<MT, 1>(a, xs, xld, blk, xbits, acc, xacc); break;
    case 2: gemv_dense_block<MT, 2>(a, xs, xld, blk, xbits, acc, xacc); break;
    case 3: gemv_dense_block<MT, 3>(a, xs, xld, blk, xbits, acc, xacc); break;
    case 4: gemv_dense_block<MT, 4>(a, xs, xld, blk, xbits, acc, xacc); break;
    case 5: gemv_dense_block<MT, 5>(a, xs, xld, blk, xbits, acc, xacc); break;
    case 6: gemv_dense_block<MT, 6>(a, xs, xld, blk, xbits, acc, xacc); break;
    case 7: gemv_dense_block<MT, 7>(a, xs, xld, blk, xbits, acc, xacc); break;
    default: gemv_dense_block<MT, 8>(a, xs, xld, blk, xbits, acc, xacc); break;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) red[wid][e][lane] = acc[e];
  // the sign runs' sums: the lanes of one row (l, l^16, l^32, l^48), then
  // the waves in the epilogue
  const int sgrp = b != 1 ? -1 : ap.c[0] == 1 ? 0 : ap.S == 2 && ap.c[1] == 1 ? 1 : -1;
  if (sgrp >= 0) {
#pragma unroll
    for (int mm = 0; mm < MT; ++mm) {
      xacc[mm] += __shfl_xor(xacc[mm], 16, 64);
      xacc[mm] += __shfl_xor(xacc[mm], 32, 64);
      if (lane < kBlk) redx[wid][mm][lane] = xacc[mm];
    }
  }
  __syncthreads();
  if (wid == 0 && ci.n >= 0) {
    const bool sgn = b == 1;
    const int S = ap.S, ws = dense_wsh(b);
    const int sh0 = ap.sh[0] + ws, sh1 = ap.sh[1] + ws;
    const int add0 = ap.zp[0] * ci.colsum[0] - (ap.c[0] == 1 && sgn ? ap.padcnt[0] : 0);
    const int add1 = ap.zp[1] * ci.colsum[1] - (ap.c[1] == 1 && sgn ? ap.padcnt[1] : 0);
    const float sa0 = a.s_a[0], sa1 = S == 2 ? a.s_a[1] : 0.0f;
#pragma unroll
    for (int e = 0; e < 4; e += 2) {
      const int m = (lane >> 4) * 2 + (e >> 1);  // sums e, e + 1: batch row m, groups 0 and 1
      if (m < a.M) {
        const int r0 = red[0][e][lane] + red[1][e][lane] + red[2][e][lane] + red[3][e][lane];
        const int r1 = red[0][e + 1][lane] + red[1][e + 1][lane] + red[2][e + 1][lane] + red[3][e + 1][lane];
        int xsum = 0;
        if (sgrp >= 0) {
          const int r = lane & 15;
          xsum = redx[0][m][r] + redx[1][m][r] + redx[2][m][r] + redx[3][m][r];
        }
        const int t0 = (r0 >> sh0) + add0 + (sgrp == 0 ? xsum : 0);
        const int t1 = S == 2 ? (r1 >> sh1) + add1 + (sgrp == 1 ? xsum : 0) : 0;
        if (a.acc) {
          a.acc[(int64_t)m * a.N + ci.n] = t0;
          if (S == 2) a.acc[(a.M + m) * a.N + ci.n] = t1;
        }
        gemv_store_out(a, pc, m, ci.n, epilogue(t0, t1, S, sa0, sa1, ci.s_w));
      }
    }
  }
}

bool gemv_dense_fits(int64_t M, const ActPlan& ap) {
  const int64_t lds = M * (ap.Kp + 16) + 32 + M * (ap.Kp / 32) * 8;
  return M >= 1 && M <= 8 && lds <= 64 * 1024 && gemv_dense_xbytes64(ap) < ((int64_t)1 << 31);
}

hipError_t launch_mp_gemv_dense(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                const WDev& wd, const WPlan& wp, const uint8_t* dense, int b_lo,
                                int b_hi, int64_t M, int64_t N, uint16_t* Y, int64_t ldy,
                                int32_t* acc, hipStream_t stream) {
  if (!gemv_dense_fits(M, ap)) return hipErrorInvalidValue;
  GemmArgs a = make_args(act_packed, s_a, ap, wd, wp, M, N, Y, ldy, acc);
  a.dense = dense;
  a.db_lo = b_lo;
  a.db_hi = b_hi;
  // byte rows, 32 zero bytes, then two sign words per run and row
  const size_t lds = (size_t)M * (ap.Kp + 16) + 32 + (size_t)M * (ap.Kp / 32) * 8;
  const dim3 grid((unsigned)wp.nblk);
  if (M == 1) hipLaunchKernelGGL(k_gemv_dense<1>, grid, dim3(256), lds, stream, a);
  else if (M == 2) hipLaunchKernelGGL(k_gemv_dense<2>, grid, dim3(256), lds, stream, a);
  else if (M <= 4) hipLaunchKernelGGL(k_gemv_dense<4>, grid, dim3(256), lds, stream, a);
  else hipLaunchKernelGGL(k_gemv_dense<8>, grid, dim3(256), lds, stream, a);
  return hipGetLastError();
}

hipError_t launch_to_fp(const uint8_t* src, int64_t src_bstride, int c, int ng, int64_t nblk,
                        uint8_t* dst, int64_t dst_bstride, int fmt, hipStream_t stream) {
  const int64_t pairs = nblk * ((ng + 1) / 2);
  if (pairs == 0) return hipSuccess;
  if (pairs >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((pairs + 3) / 4)), blk(256);
  if (c == 4 && fmt == kFmtFp6)
    hipLaunchKernelGGL((k_to_fp<4, kFmtFp6>), grid, blk, 0, stream, src, src_bstride, ng, (int)pairs, dst, dst_bstride);
  else if (c == 2 && fmt == kFmtFp4)
    hipLaunchKernelGGL((k_to_fp<2, kFmtFp4>), grid, blk, 0, stream, src, src_bstride, ng, (int)pairs, dst, dst_bstride);
  else if (c == 1 && fmt == kFmtFp4)
    hipLaunchKernelGGL((k_to_fp<1, kFmtFp4>), grid, blk, 0, stream, src, src_bstride, ng, (int)pairs, dst, dst_bstride);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ------------------------------------------------------- scratch memory --
// Working memory of the allocation-free entry point
// (soniq_quantize_mp_gemm_scratch): the grid state, partial maxima, scales
// and packed activations that an activation handle would own.  Each device
// the library runs on holds its own copy until the process ends.  In host
// code `scratch` names a host-side stand-in, not device memory: kernels get
// the per-device address that hipGetSymbolAddress returns.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

__global__ __launch_bounds__(256) void k_fill_u32(uint32_t* __restrict__ p, int n, uint32_t v) {
  for (int i = (int)(blockIdx.x * 256 + threadIdx.x); i < n; i += (int)(gridDim.x * 256)) p[i] = v;
}

// ---------------------------------------------------------- k_stream_read --
// A plain read, the ceiling a bandwidth-bound kernel is measured against:
// 8 KB per workgroup in two 16-byte loads per thread, both issued before
// either is used; the XOR of the workgroup's words is its one output.
__global__ __launch_bounds__(256) void k_stream_read(const uint8_t* __restrict__ src, int bytes,
                                                     uint32_t* __restrict__ sink) {
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc((void*)src, (short)0, bytes, 0x00020000);
  const uint32_t base = blockIdx.x * 8192u + threadIdx.x * 16u;
  const uint4 v0 = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, base, 0, 0));
  const uint4 v1 =
      __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, base + 4096u, 0, 0));
  uint32_t x = v0.x ^ v0.y ^ v0.z ^ v0.w ^ v1.x ^ v1.y ^ v1.z ^ v1.w;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x ^= (uint32_t)__shfl_xor((int)x, o, 64);
  __shared__ uint32_t red[4];
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

hipError_t launch_stream_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  const unsigned grid = (unsigned)((bytes + 8191) / 8192);
  hipLaunchKernelGGL(k_stream_read, dim3(grid), dim3(256), 0, stream,
                     static_cast<const uint8_t*>(src), (int)bytes, sink);
  return hipGetLastError();
}

hipError_t scratch_device_ptr(hipStream_t stream, uint8_t** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static uint8_t* ptr[kMaxDevices] = {};
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    // The grid-state words must start at zero; the barrier protocol leaves
    // them at zero after every call, so they are cleared once, on the
    // caller's stream ahead of the first call's kernels (a fill kernel, not
    // a memset node, in case that call is being captured).
    hipLaunchKernelGGL(k_fill_u32, dim3(8), dim3(256), 0, stream, reinterpret_cast<uint32_t*>(p),
                       kActStateWords, 0u);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    ptr[dev] = static_cast<uint8_t*>(p);
  }
  *out = ptr[dev];
  return hipSuccess;
}

}  // namespace soniq
