// gfx950 (CDNA4) kernels of the SONIQ inference hot path.
//
//   k_wpack      quantize one output channel, place its codes on the
//                group-ordered, padded channel axis, bit-pack it and record
//                its scale and per-group code sums            (once per layer)
//   k_absmax     per-activation-group max-abs over all rows, finished by the
//                last workgroup, which also writes the group scales
//   k_act_pack   quantize, re-order and bit-pack activation rows
//   k_gemm<S>    int8 MFMA GEMM on the packed operands: 128x128 block tile,
//                LDS double buffer filled through a register stage that
//                unpacks 1/2/4-bit fields to int8, one int32 accumulator set
//                per activation group, fixed-order fp32 epilogue to bf16
//   k_gemv<MT>   batch <= 8 decode without matrix cores: the activation rows
//                are unpacked once per workgroup into LDS, 16 lanes stream
//                one packed weight row with 128-bit loads and v_dot4_i32_i8
//
// Paper passages: Sec. 2.4 C1/C2/C5; Sec. 3 codec (scale, unsigned codes,
// Eq. 1 weight codes); Alg. 1 channel permutation and Phase II integer MAC;
// Fig. "normalization" (group by width, pad to the vector width).
#include "soniq_internal.h"

namespace soniq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- codec --
__device__ __forceinline__ int quant_code(float x, float s, const QParam& q) {
  if (q.sign1) return x < 0.0f ? -1 : 1;
  if (s == 0.0f) return 0;
  float t = __builtin_rintf(__fdiv_rn(x, s));
  t = fminf(fmaxf(t, (float)q.lo), (float)q.hi);
  return (int)t;
}

__device__ __forceinline__ float group_scale(float maxabs, const QParam& q) {
  return q.sign1 ? maxabs : __fdiv_rn(maxabs, q.qdiv);
}

// One packed word from E = 32/c stored int8 codes (E/4 dwords, natural order).
__device__ __forceinline__ uint32_t pack_word(const uint32_t* d, int c) {
  if (c == 8) return d[0];
  if (c == 4) return (d[0] & 0x0F0F0F0Fu) | ((d[1] & 0x0F0F0F0Fu) << 4);
  if (c == 2)
    return (d[0] & 0x03030303u) | ((d[1] & 0x03030303u) << 2) |
           ((d[2] & 0x03030303u) << 4) | ((d[3] & 0x03030303u) << 6);
  uint32_t w = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) w |= ((d[j] >> 7) & 0x01010101u) << j;
  return w;
}

// A "unit" is 64 consecutive elements of one row: 8*c packed bytes, or 64
// unpacked int8.  Held in four 128-bit registers (no arrays, so it stays in
// VGPRs whatever the container).
struct Unit {
  uint4 v0, v1, v2, v3;
};

__device__ __forceinline__ uint4 u4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return make_uint4(a, b, c, d);
}

// Load a unit (8-byte aligned for c = 1, 16-byte aligned otherwise).
__device__ __forceinline__ Unit load_unit(const uint8_t* p, int c) {
  Unit u;
  const uint4 z = u4(0, 0, 0, 0);
  u.v0 = z; u.v1 = z; u.v2 = z; u.v3 = z;
  const uint4* q = reinterpret_cast<const uint4*>(p);
  if (c == 1) {
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    u.v0.x = t.x;
    u.v0.y = t.y;
  } else {
    u.v0 = q[0];
    if (c >= 4) u.v1 = q[1];
    if (c == 8) {
      u.v2 = q[2];
      u.v3 = q[3];
    }
  }
  return u;
}

// Four consecutive elements per output dword, see unpack_word.
__device__ __forceinline__ uint4 unpack2(uint32_t w) {
  return u4((w << 6) & 0xC0C0C0C0u, (w << 4) & 0xC0C0C0C0u, (w << 2) & 0xC0C0C0C0u,
            w & 0xC0C0C0C0u);
}
__device__ __forceinline__ uint4 unpack4(uint32_t w0, uint32_t w1) {
  return u4((w0 << 4) & 0xF0F0F0F0u, w0 & 0xF0F0F0F0u, (w1 << 4) & 0xF0F0F0F0u,
            w1 & 0xF0F0F0F0u);
}
__device__ __forceinline__ uint32_t sgn1(uint32_t w, int j) {
  return ((w << (7 - j)) & 0x80808080u) | 0x40404040u;
}
__device__ __forceinline__ uint4 unpack1_lo(uint32_t w) {
  return u4(sgn1(w, 0), sgn1(w, 1), sgn1(w, 2), sgn1(w, 3));
}
__device__ __forceinline__ uint4 unpack1_hi(uint32_t w) {
  return u4(sgn1(w, 4), sgn1(w, 5), sgn1(w, 6), sgn1(w, 7));
}

// Unpack a loaded unit to 64 scaled int8 elements; zeros when !valid.
__device__ __forceinline__ Unit unpack_unit(const Unit& w, int c, bool valid) {
  Unit d;
  if (!valid) {
    const uint4 z = u4(0, 0, 0, 0);
    d.v0 = z; d.v1 = z; d.v2 = z; d.v3 = z;
  } else if (c == 8) {
    d = w;
  } else if (c == 4) {
    d.v0 = unpack4(w.v0.x, w.v0.y);
    d.v1 = unpack4(w.v0.z, w.v0.w);
    d.v2 = unpack4(w.v1.x, w.v1.y);
    d.v3 = unpack4(w.v1.z, w.v1.w);
  } else if (c == 2) {
    d.v0 = unpack2(w.v0.x);
    d.v1 = unpack2(w.v0.y);
    d.v2 = unpack2(w.v0.z);
    d.v3 = unpack2(w.v0.w);
  } else {
    d.v0 = unpack1_lo(w.v0.x);
    d.v1 = unpack1_hi(w.v0.x);
    d.v2 = unpack1_lo(w.v0.y);
    d.v3 = unpack1_hi(w.v0.y);
  }
  return d;
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
// unpacked bytes: undo the unpack scales, remove the products of padding
// channels (only sign-bit x sign-bit padding is nonzero: both decode to +1,
// each product 64*64), add the unsigned zero point times the code sum.
__device__ __forceinline__ int true_acc(int raw, int sha, int ca, int padcnt, int zp,
                                        uint8_t shw, int colsum) {
  if (ca == 1 && (shw & kShwSign)) raw -= padcnt << 12;
  return (raw >> (sha + (shw & 0x7F))) + zp * colsum;
}

// Stored activation code of x in group g (code minus the group zero point).
__device__ __forceinline__ uint8_t store_code(float x, int g, float s0, float s1,
                                              const QParam& q0, const QParam& q1, int zp0,
                                              int zp1) {
  const int code = g ? quant_code(x, s1, q1) - zp1 : quant_code(x, s0, q0) - zp0;
  return (uint8_t)(int8_t)code;
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
    const int64_t* __restrict__ row_off, const int32_t* __restrict__ phys, QParam q_lo,
    QParam q_hi, int b_lo, int c_lo, int c_hi, int Kp, int64_t rb_lo, int64_t rb_hi,
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

  const bool lo = w_bits[n] == b_lo;
  const QParam q = lo ? q_lo : q_hi;
  const int c = lo ? c_lo : c_hi;
  const float s = group_scale(m, q);

  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < Kp / 4; i += blockDim.x) codes32[i] = 0;
  __syncthreads();
  int cs0 = 0, cs1 = 0;
  for (int64_t k = tid; k < K; k += blockDim.x) {
    int code = quant_code(row[k], s, q);
    codes[pos[k]] = (uint8_t)(int8_t)code;
    if (seg[k] == 0) cs0 += code; else cs1 += code;
  }
  cs0 = block_sum(cs0, redi);
  cs1 = block_sum(cs1, redi);  // block_sum syncs, so the code writes are visible

  const int per = 32 / c;
  const int nwords = Kp / per;
  const int rwords = (int)((lo ? rb_lo : rb_hi) >> 2);
  uint32_t* dst = reinterpret_cast<uint32_t*>(packed + row_off[n]);
  for (int w = tid; w < rwords; w += blockDim.x) {
    uint32_t word = 0;
    if (w < nwords) word = pack_word(codes32 + w * (per / 4), c);
    dst[w] = word;
  }
  if (tid == 0) {
    ColInfo ci;
    ci.n = (int32_t)n;
    ci.s_w = s;
    ci.colsum[0] = cs0;
    ci.colsum[1] = cs1;
    colinfo[phys[n]] = ci;
  }
}

// -------------------------------------------------------------- k_absmax --
// Max-abs of every activation group over all M rows.  Each workgroup
// writes its partial maxima; the last one to finish reduces them, writes
// the group scales s_a[g] and re-arms the counter for the next call.
// Contiguous rows (lda == K, K % 4 == 0, 16-byte aligned) are read as one
// flat float4 stream with kAbsU loads in flight per thread.
constexpr int kAbsU = 8;

__device__ __forceinline__ void absmax_finish(float mx0, float mx1, const ActPlan& ap,
                                              float* __restrict__ partial,
                                              unsigned int* __restrict__ counter,
                                              float* __restrict__ s_a, float* red,
                                              int* is_last) {
  const int tid = threadIdx.x;
  mx0 = block_max(mx0, red);
  mx1 = block_max(mx1, red);
  if (tid == 0) {
    partial[2 * blockIdx.x] = mx0;
    partial[2 * blockIdx.x + 1] = mx1;
    __threadfence();
    unsigned int ticket = atomicAdd(counter, 1u);
    *is_last = (ticket == gridDim.x - 1);
  }
  __syncthreads();
  if (!*is_last) return;
  __threadfence();
  float r0 = 0.0f, r1 = 0.0f;
  for (int b = tid; b < (int)gridDim.x; b += blockDim.x) {
    r0 = fmaxf(r0, __hip_atomic_load(&partial[2 * b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    r1 = fmaxf(r1, __hip_atomic_load(&partial[2 * b + 1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  }
  r0 = block_max(r0, red);
  r1 = block_max(r1, red);
  if (tid == 0) {
    s_a[0] = group_scale(r0, ap.q[0]);
    s_a[1] = ap.S == 2 ? group_scale(r1, ap.q[1]) : 0.0f;
    *counter = 0u;
  }
}

__device__ __forceinline__ void max4(float4 v, uchar4 g, float& mx0, float& mx1) {
  const float a0 = fabsf(v.x), a1 = fabsf(v.y), a2 = fabsf(v.z), a3 = fabsf(v.w);
  mx0 = fmaxf(mx0, fmaxf(fmaxf(g.x ? 0.0f : a0, g.y ? 0.0f : a1), fmaxf(g.z ? 0.0f : a2, g.w ? 0.0f : a3)));
  mx1 = fmaxf(mx1, fmaxf(fmaxf(g.x ? a0 : 0.0f, g.y ? a1 : 0.0f), fmaxf(g.z ? a2 : 0.0f, g.w ? a3 : 0.0f)));
}

__global__ __launch_bounds__(256) void k_absmax_flat(const float4* __restrict__ A, uint32_t total4,
                                                     uint32_t K4, const uchar4* __restrict__ seg4,
                                                     ActPlan ap, float* __restrict__ partial,
                                                     unsigned int* __restrict__ counter,
                                                     float* __restrict__ s_a) {
  __shared__ float red[4];
  __shared__ int is_last;
  float mx0 = 0.0f, mx1 = 0.0f;
  const uint32_t step = gridDim.x * 256u * kAbsU;
  for (uint32_t base = blockIdx.x * 256u * kAbsU + threadIdx.x; base < total4; base += step) {
    float4 v[kAbsU];
    uchar4 g[kAbsU];
#pragma unroll
    for (int j = 0; j < kAbsU; ++j) {
      const uint32_t i = base + 256u * j;
      if (i < total4) {
        v[j] = A[i];
        g[j] = seg4[i % K4];
      } else {
        v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        g[j] = make_uchar4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int j = 0; j < kAbsU; ++j) max4(v[j], g[j], mx0, mx1);
  }
  absmax_finish(mx0, mx1, ap, partial, counter, s_a, red, &is_last);
}

// Any stride or width: one row at a time, scalar loads.
__global__ __launch_bounds__(256) void k_absmax_rows(const float* __restrict__ A, int64_t M,
                                                     int64_t K, int64_t lda,
                                                     const uint8_t* __restrict__ seg, ActPlan ap,
                                                     float* __restrict__ partial,
                                                     unsigned int* __restrict__ counter,
                                                     float* __restrict__ s_a) {
  __shared__ float red[4];
  __shared__ int is_last;
  float mx0 = 0.0f, mx1 = 0.0f;
  for (int64_t m = blockIdx.x; m < M; m += gridDim.x) {
    const float* row = A + m * lda;
    for (int64_t k = threadIdx.x; k < K; k += 256) {
      const float a = fabsf(row[k]);
      if (seg[k]) mx1 = fmaxf(mx1, a); else mx0 = fmaxf(mx0, a);
    }
  }
  absmax_finish(mx0, mx1, ap, partial, counter, s_a, red, &is_last);
}

// ------------------------------------------------------------ k_act_pack --
// Codes of a block of rows, scattered to their group-ordered positions in
// LDS, then assembled into packed words and stored 16 bytes at a time.
__device__ __forceinline__ void pack_rows_from_lds(const uint32_t* codes32, int nrows,
                                                   int64_t m0, const ActPlan& ap,
                                                   uint8_t* __restrict__ packed) {
  const int Kp4 = ap.Kp / 4;
  for (int g = 0; g < ap.S; ++g) {
    const int c = g ? ap.c[1] : ap.c[0];
    const int per = 32 / c;
    const int nwords = (g ? ap.kpad[1] : ap.kpad[0]) / per;
    const int64_t rb = g ? ap.row_bytes[1] : ap.row_bytes[0];
    const int rquads = (int)(rb >> 4);
    const int gbase = g ? ap.kpad[0] / 4 : 0;
    uint8_t* dst0 = packed + (g ? ap.seg_off[1] : ap.seg_off[0]);
    for (int u = threadIdx.x; u < nrows * rquads; u += blockDim.x) {
      const int r = u / rquads, q = u - r * rquads;
      const uint32_t* src = codes32 + r * Kp4 + gbase;
      uint32_t w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int wi = 4 * q + i;
        w[i] = wi < nwords ? pack_word(src + wi * (per / 4), c) : 0u;
      }
      *reinterpret_cast<uint4*>(dst0 + (m0 + r) * rb + (int64_t)q * 16) =
          make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// One workgroup per activation row.  Dynamic LDS: Kp bytes of stored codes.
constexpr int kPackU = 4;
__global__ __launch_bounds__(256) void k_act_pack(const float* __restrict__ A, int64_t K,
                                                  int64_t lda, const int32_t* __restrict__ pos,
                                                  const uint8_t* __restrict__ seg, ActPlan ap,
                                                  const float* __restrict__ s_a,
                                                  uint8_t* __restrict__ packed, int vec4) {
  extern __shared__ __align__(16) uint8_t codes[];
  const int64_t m = blockIdx.x;
  const int tid = threadIdx.x;
  const float* row = A + m * lda;
  const float s0 = s_a[0], s1 = s_a[1];
  const QParam q0 = ap.q[0], q1 = ap.q[1];
  const int zp0 = ap.zp[0], zp1 = ap.zp[1];
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < ap.Kp / 4; i += blockDim.x) codes32[i] = 0;
  __syncthreads();
  if (vec4) {
    const int K4 = (int)(K / 4);
    const float4* row4 = reinterpret_cast<const float4*>(row);
    for (int base = tid; base < K4; base += 256 * kPackU) {
      float4 v[kPackU];
      int4 p[kPackU];
      uchar4 g[kPackU];
#pragma unroll
      for (int j = 0; j < kPackU; ++j) {
        const int i = base + 256 * j;
        if (i < K4) {
          v[j] = row4[i];
          p[j] = reinterpret_cast<const int4*>(pos)[i];
          g[j] = reinterpret_cast<const uchar4*>(seg)[i];
        }
      }
#pragma unroll
      for (int j = 0; j < kPackU; ++j) {
        if (base + 256 * j < K4) {
          codes[p[j].x] = store_code(v[j].x, g[j].x, s0, s1, q0, q1, zp0, zp1);
          codes[p[j].y] = store_code(v[j].y, g[j].y, s0, s1, q0, q1, zp0, zp1);
          codes[p[j].z] = store_code(v[j].z, g[j].z, s0, s1, q0, q1, zp0, zp1);
          codes[p[j].w] = store_code(v[j].w, g[j].w, s0, s1, q0, q1, zp0, zp1);
        }
      }
    }
  } else {
    for (int64_t k = tid; k < K; k += blockDim.x)
      codes[pos[k]] = store_code(row[k], seg[k], s0, s1, q0, q1, zp0, zp1);
  }
  __syncthreads();
  pack_rows_from_lds(codes32, 1, m, ap, packed);
}

// ----------------------------------------------------------- k_act_small --
// Small batches (M * K <= kSmallElems, M * Kp <= 64 KB): one workgroup of
// 1024 threads holds the whole batch in registers, reduces the group
// maxima, quantizes and packs -- one pass over A, one launch.
constexpr int kSmallU = 8;
constexpr int kSmallThreads = 1024;
constexpr int kSmallElems = kSmallThreads * kSmallU * 4;

__global__ __launch_bounds__(1024) void k_act_small(const float* __restrict__ A, int M, int K,
                                                    int64_t lda, const int32_t* __restrict__ pos,
                                                    const uint8_t* __restrict__ seg, ActPlan ap,
                                                    float* __restrict__ s_a_out,
                                                    uint8_t* __restrict__ packed) {
  extern __shared__ __align__(16) uint8_t codes[];
  __shared__ float red[16];
  const int tid = threadIdx.x;
  const int K4 = K / 4;
  const int total4 = M * K4;
  float4 v[kSmallU];
  int4 p[kSmallU];
  uchar4 g[kSmallU];
  float mx0 = 0.0f, mx1 = 0.0f;
#pragma unroll
  for (int j = 0; j < kSmallU; ++j) {
    const int i = tid + kSmallThreads * j;
    if (i < total4) {
      const int m = i / K4, k4 = i - m * K4;
      v[j] = *reinterpret_cast<const float4*>(A + (int64_t)m * lda + 4 * k4);
      p[j] = reinterpret_cast<const int4*>(pos)[k4];
      g[j] = reinterpret_cast<const uchar4*>(seg)[k4];
      max4(v[j], g[j], mx0, mx1);
    }
  }
  uint32_t* codes32 = reinterpret_cast<uint32_t*>(codes);
  for (int i = tid; i < M * ap.Kp / 4; i += kSmallThreads) codes32[i] = 0;
  mx0 = block_max(mx0, red);
  mx1 = block_max(mx1, red);
  const float s0 = group_scale(mx0, ap.q[0]);
  const float s1 = ap.S == 2 ? group_scale(mx1, ap.q[1]) : 0.0f;
  if (tid == 0) {
    s_a_out[0] = s0;
    s_a_out[1] = s1;
  }
  const QParam q0 = ap.q[0], q1 = ap.q[1];
  const int zp0 = ap.zp[0], zp1 = ap.zp[1];
#pragma unroll
  for (int j = 0; j < kSmallU; ++j) {
    const int i = tid + kSmallThreads * j;
    if (i < total4) {
      uint8_t* row = codes + (i / K4) * ap.Kp;
      row[p[j].x] = store_code(v[j].x, g[j].x, s0, s1, q0, q1, zp0, zp1);
      row[p[j].y] = store_code(v[j].y, g[j].y, s0, s1, q0, q1, zp0, zp1);
      row[p[j].z] = store_code(v[j].z, g[j].z, s0, s1, q0, q1, zp0, zp1);
      row[p[j].w] = store_code(v[j].w, g[j].w, s0, s1, q0, q1, zp0, zp1);
    }
  }
  __syncthreads();
  pack_rows_from_lds(codes32, M, 0, ap, packed);
}

// ---------------------------------------------------------------- k_gemm --
struct GemmArgs {
  const uint8_t* act;
  const float* s_a;
  ActPlan ap;
  const uint8_t* w;
  const TileDesc* tiles;
  const ColInfo* colinfo;
  const uint8_t* shw;
  WPlan wp;
  int64_t M, N;
  uint16_t* Y;
  int64_t ldy;
  int32_t* acc;
};

constexpr int kTK = 128;            // channels per LDS stage (two units)
constexpr int kRowB = kTK;          // LDS bytes per tile row (int8)
constexpr int kTileB = 128 * kRowB; // bytes of one operand tile in LDS

// 16-byte chunk `ch` of LDS row r, XOR-swizzled so that the 16 rows read by
// one MFMA fragment spread over all banks.
__device__ __forceinline__ int lds_off(int r, int ch) {
  return r * kRowB + ((ch ^ ((r >> 1) & 7)) << 4);
}

template <int S>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  __shared__ __align__(16) uint8_t lds[2][2][kTileB];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int64_t m0 = (int64_t)blockIdx.y * 128;
  const int n0 = blockIdx.x * 128;
  const ActPlan& ap = a.ap;
  const WPlan& wp = a.wp;

  // Stage list: group 0 stages, then group 1 stages.
  const int ng0 = ap.kpad[0] / kGran;
  const int ng1 = S == 2 ? ap.kpad[1] / kGran : 0;
  const int ns0 = (ng0 + 1) / 2;
  const int ns1 = (ng1 + 1) / 2;
  const int nst = ns0 + ns1;

  // Loader roles: thread -> (tile row, unit within the stage).
  const int lrow = tid >> 1, lq = tid & 1;
  // Activation row pointer per group.
  const uint8_t* arow0 = a.act + ap.seg_off[0] + (m0 + lrow) * ap.row_bytes[0];
  const uint8_t* arow1 = a.act + ap.seg_off[1] + (m0 + lrow) * ap.row_bytes[1];
  // Weight row pointer and container.
  const int p = n0 + lrow;
  const int t = p >> 6, j = p & 63;
  bool wvalid = false;
  int wc = 8;
  const uint8_t* wrow = a.w;
  if (t < wp.ntiles) {
    TileDesc td = a.tiles[t];
    if (j < td.n_rows) {
      wvalid = true;
      const bool lo = j < td.n_lo;
      wc = lo ? wp.c_lo : wp.c_hi;
      wrow = a.w + td.base +
             (lo ? (int64_t)j * wp.rb_lo : (int64_t)td.n_lo * wp.rb_lo + (int64_t)(j - td.n_lo) * wp.rb_hi);
    }
  }

  Unit ra, rb;
  bool va = false, vb = false;
  int ca = 8;

  auto stage_info = [&](int st, int& g, int& gi0, int& ngv) {
    if (st < ns0) { g = 0; gi0 = 2 * st; ngv = min(2, ng0 - gi0); }
    else { g = 1; gi0 = 2 * (st - ns0); ngv = min(2, ng1 - gi0); }
  };
  const int ca0 = ap.c[0], ca1 = ap.c[1], kp0 = ap.kpad[0];
  auto gload = [&](int st) {
    int g, gi0, ngv;
    stage_info(st, g, gi0, ngv);
    const int gi = gi0 + lq;
    ca = g ? ca1 : ca0;
    va = lq < ngv;
    if (va) ra = load_unit((g ? arow1 : arow0) + (int64_t)gi * 8 * ca, ca);
    vb = wvalid && lq < ngv;
    if (vb) {
      const int64_t e0 = (int64_t)(g ? kp0 : 0) + (int64_t)gi * kGran;
      rb = load_unit(wrow + e0 * wc / 8, wc);
    }
  };
  auto lwrite = [&](int buf) {
    const Unit da = unpack_unit(ra, ca, va);
    uint8_t* la = lds[buf][0];
    *reinterpret_cast<uint4*>(la + lds_off(lrow, lq * 4 + 0)) = da.v0;
    *reinterpret_cast<uint4*>(la + lds_off(lrow, lq * 4 + 1)) = da.v1;
    *reinterpret_cast<uint4*>(la + lds_off(lrow, lq * 4 + 2)) = da.v2;
    *reinterpret_cast<uint4*>(la + lds_off(lrow, lq * 4 + 3)) = da.v3;
    const Unit db = unpack_unit(rb, wc, vb);
    uint8_t* lb = lds[buf][1];
    *reinterpret_cast<uint4*>(lb + lds_off(lrow, lq * 4 + 0)) = db.v0;
    *reinterpret_cast<uint4*>(lb + lds_off(lrow, lq * 4 + 1)) = db.v1;
    *reinterpret_cast<uint4*>(lb + lds_off(lrow, lq * 4 + 2)) = db.v2;
    *reinterpret_cast<uint4*>(lb + lds_off(lrow, lq * 4 + 3)) = db.v3;
  };

  v4i acc0[4][4], acc1[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      acc0[i][jj] = v4i{0, 0, 0, 0};
      acc1[i][jj] = v4i{0, 0, 0, 0};
    }

  auto compute = [&](int buf, int ngv, v4i (&acc)[4][4]) {
    const uint8_t* la = lds[buf][0];
    const uint8_t* lb = lds[buf][1];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      if (kk < ngv) {
        v4i af[4], bf[4];
        const int ch = kk * 4 + (lane >> 4);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          af[i] = *reinterpret_cast<const v4i*>(la + lds_off(wm * 64 + i * 16 + (lane & 15), ch));
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          bf[jj] = *reinterpret_cast<const v4i*>(lb + lds_off(wn * 64 + jj * 16 + (lane & 15), ch));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            acc[i][jj] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[jj], acc[i][jj], 0, 0, 0);
      }
    }
  };

  if (nst > 0) {
    gload(0);
    lwrite(0);
  }
  __syncthreads();
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) gload(st + 1);
    int g, gi0, ngv;
    stage_info(st, g, gi0, ngv);
    if (S == 1 || g == 0) compute(st & 1, ngv, acc0);
    else compute(st & 1, ngv, acc1);
    if (st + 1 < nst) lwrite((st + 1) & 1);
    __syncthreads();
  }

  // Epilogue: exact int32 per group, fixed-order fp32 scaling, bf16.
  const float sa0 = a.s_a[0];
  const float sa1 = S == 2 ? a.s_a[1] : 0.0f;
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    const int pc = n0 + wn * 64 + jj * 16 + (lane & 15);
    if (pc >= wp.Np) continue;
    const ColInfo ci = a.colinfo[pc];
    if (ci.n < 0) continue;
    const uint8_t shw = a.shw[pc];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
        if (m >= a.M) continue;
        const int t0 = true_acc(acc0[i][jj][r], ap.sh[0], ap.c[0], ap.padcnt[0], ap.zp[0], shw,
                                ci.colsum[0]);
        const int t1 = S == 2 ? true_acc(acc1[i][jj][r], ap.sh[1], ap.c[1], ap.padcnt[1],
                                         ap.zp[1], shw, ci.colsum[1])
                              : 0;
        a.Y[m * a.ldy + ci.n] = bf16_rne(epilogue(t0, t1, S, sa0, sa1, ci.s_w));
        if (a.acc) {
          a.acc[m * a.N + ci.n] = t0;
          if (S == 2) a.acc[(a.M + m) * a.N + ci.n] = t1;
        }
      }
  }
}

// ---------------------------------------------------------------- k_gemv --
// Dot of NV*16 unpacked elements (k0 .. k0 + 16*NV) with every staged
// activation row; the sum goes to the accumulator of the group of k0.
__device__ __forceinline__ int dot16(uint4 d, uint4 x, int v) {
  v = __builtin_amdgcn_sdot4((int)d.x, (int)x.x, v, false);
  v = __builtin_amdgcn_sdot4((int)d.y, (int)x.y, v, false);
  v = __builtin_amdgcn_sdot4((int)d.z, (int)x.z, v, false);
  return __builtin_amdgcn_sdot4((int)d.w, (int)x.w, v, false);
}

template <int NV, int MT>
__device__ __forceinline__ void dot_rows(const Unit& d, int k0, const uint8_t* xs, int Kp,
                                         int kp0, int M, int (&acc0)[MT], int (&acc1)[MT]) {
  if (k0 >= Kp) return;
  const bool g1 = k0 >= kp0;
#pragma unroll
  for (int mm = 0; mm < MT; ++mm) {
    if (mm < M) {
      const uint4* x = reinterpret_cast<const uint4*>(xs + (int64_t)mm * Kp + k0);
      int v = dot16(d.v0, x[0], 0);
      if (NV > 1) v = dot16(d.v1, x[1], v);
      if (NV > 2) {
        v = dot16(d.v2, x[2], v);
        v = dot16(d.v3, x[3], v);
      }
      if (g1) acc1[mm] += v; else acc0[mm] += v;
    }
  }
}

// Workgroup = 4 waves = 16 physical output rows; each row is streamed by 16
// lanes with 128-bit loads.  Dynamic LDS: M * Kp bytes of unpacked
// activations.
constexpr int kGemvU = 8;  // weight chunks in flight per lane

template <int MT>
__global__ __launch_bounds__(256) void k_gemv(GemmArgs a) {
  extern __shared__ __align__(16) uint8_t xs[];
  const int tid = threadIdx.x;
  const ActPlan& ap = a.ap;
  const WPlan& wp = a.wp;
  const int M = (int)a.M;
  const int Kp = ap.Kp;
  const int ng0 = ap.kpad[0] / kGran;
  const int ngt = Kp / kGran;

  // This lane's weight row (16 lanes per row, 4 rows per wave).
  const int lane = tid & 63, wid = tid >> 6;
  const int s = lane & 15;
  const int p = blockIdx.x * kGemvRows + wid * 4 + (lane >> 4);
  const int t = p >> 6, j = p & 63;
  const TileDesc td = a.tiles[t];
  const bool valid = j < td.n_rows;
  const bool lo = j < td.n_lo;
  const int c = lo ? wp.c_lo : wp.c_hi;
  const uint8_t* row = a.w + td.base +
                       (lo ? (int64_t)j * wp.rb_lo : (int64_t)td.n_lo * wp.rb_lo + (int64_t)(j - td.n_lo) * wp.rb_hi);
  const int nch = valid ? (int)((lo ? wp.rb_lo : wp.rb_hi) >> 4) : 0;
  const int kp0 = ap.kpad[0];

  // First batch of weight chunks in flight before the activations are staged.
  uint4 cur[kGemvU];
#pragma unroll
  for (int u = 0; u < kGemvU; ++u) {
    const int ch = s + 16 * u;
    cur[u] = ch < nch ? *reinterpret_cast<const uint4*>(row + (int64_t)ch * 16) : make_uint4(0, 0, 0, 0);
  }

  // Stage the activation rows, unpacked, in LDS.
  for (int u = tid; u < M * ngt; u += blockDim.x) {
    const int m = u / ngt, ga = u - m * ngt;
    const bool g1 = ga >= ng0;
    const int gi = g1 ? ga - ng0 : ga;
    const int cx = g1 ? ap.c[1] : ap.c[0];
    const int64_t off = g1 ? ap.seg_off[1] + (int64_t)m * ap.row_bytes[1]
                           : ap.seg_off[0] + (int64_t)m * ap.row_bytes[0];
    const Unit d = unpack_unit(load_unit(a.act + off + (int64_t)gi * 8 * cx, cx), cx, true);
    uint4* dst = reinterpret_cast<uint4*>(xs + (int64_t)m * Kp + (int64_t)ga * kGran);
    dst[0] = d.v0;
    dst[1] = d.v1;
    dst[2] = d.v2;
    dst[3] = d.v3;
  }
  __syncthreads();

  int acc0[MT], acc1[MT];
#pragma unroll
  for (int mm = 0; mm < MT; ++mm) { acc0[mm] = 0; acc1[mm] = 0; }

  for (int base = s; base < nch; base += 16 * kGemvU) {
    uint4 nxt[kGemvU];
    const bool more = base + 16 * kGemvU < nch;
    if (more) {
#pragma unroll
      for (int u = 0; u < kGemvU; ++u) {
        const int ch = base + 16 * (kGemvU + u);
        nxt[u] = ch < nch ? *reinterpret_cast<const uint4*>(row + (int64_t)ch * 16) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < kGemvU; ++u) {
      const int ch = base + 16 * u;
      if (ch < nch) {
        const uint4 v = cur[u];
        Unit d;
        if (c == 2) {
          d.v0 = unpack2(v.x); d.v1 = unpack2(v.y); d.v2 = unpack2(v.z); d.v3 = unpack2(v.w);
          dot_rows<4, MT>(d, ch * 64, xs, Kp, kp0, M, acc0, acc1);
        } else if (c == 4) {
          d.v0 = unpack4(v.x, v.y); d.v1 = unpack4(v.z, v.w);
          dot_rows<2, MT>(d, ch * 32, xs, Kp, kp0, M, acc0, acc1);
        } else if (c == 8) {
          d.v0 = v;
          dot_rows<1, MT>(d, ch * 16, xs, Kp, kp0, M, acc0, acc1);
        } else {
          d.v0 = unpack1_lo(v.x); d.v1 = unpack1_hi(v.x); d.v2 = unpack1_lo(v.y); d.v3 = unpack1_hi(v.y);
          dot_rows<4, MT>(d, ch * 128, xs, Kp, kp0, M, acc0, acc1);
          d.v0 = unpack1_lo(v.z); d.v1 = unpack1_hi(v.z); d.v2 = unpack1_lo(v.w); d.v3 = unpack1_hi(v.w);
          dot_rows<4, MT>(d, ch * 128 + 64, xs, Kp, kp0, M, acc0, acc1);
        }
      }
    }
    if (more) {
#pragma unroll
      for (int u = 0; u < kGemvU; ++u) cur[u] = nxt[u];
    }
  }

  // Sum over the 16 lanes of the row; every lane ends with the totals.
#pragma unroll
  for (int mm = 0; mm < MT; ++mm) {
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      acc0[mm] += __shfl_xor(acc0[mm], o, 16);
      acc1[mm] += __shfl_xor(acc1[mm], o, 16);
    }
  }
  if (!valid || s >= M) return;
  const ColInfo ci = a.colinfo[p];
  if (ci.n < 0) return;
  int r0 = 0, r1 = 0;
#pragma unroll
  for (int mm = 0; mm < MT; ++mm)
    if (mm == s) { r0 = acc0[mm]; r1 = acc1[mm]; }
  const uint8_t shw = a.shw[p];
  const int S = ap.S;
  const int t0 = true_acc(r0, ap.sh[0], ap.c[0], ap.padcnt[0], ap.zp[0], shw, ci.colsum[0]);
  const int t1 = S == 2 ? true_acc(r1, ap.sh[1], ap.c[1], ap.padcnt[1], ap.zp[1], shw, ci.colsum[1])
                        : 0;
  const float sa0 = a.s_a[0], sa1 = S == 2 ? a.s_a[1] : 0.0f;
  const int64_t m = s;
  a.Y[m * a.ldy + ci.n] = bf16_rne(epilogue(t0, t1, S, sa0, sa1, ci.s_w));
  if (a.acc) {
    a.acc[m * a.N + ci.n] = t0;
    if (S == 2) a.acc[(a.M + m) * a.N + ci.n] = t1;
  }
}

}  // namespace

// ------------------------------------------------------------- launchers --
hipError_t launch_wpack(const float* W, int64_t N, int64_t K, int64_t ldw,
                        const uint8_t* w_bits_dev, const int32_t* pos_dev,
                        const uint8_t* seg_dev, const int64_t* row_off_dev,
                        const int32_t* phys_dev, QParam q_lo, QParam q_hi, int b_lo,
                        int c_lo, int c_hi, int Kp, int kpad0, int64_t rb_lo,
                        int64_t rb_hi, uint8_t* packed, ColInfo* colinfo,
                        hipStream_t stream) {
  (void)kpad0;
  hipLaunchKernelGGL(k_wpack, dim3((unsigned)N), dim3(256), (size_t)Kp, stream, W, K, ldw,
                     w_bits_dev, pos_dev, seg_dev, row_off_dev, phys_dev, q_lo, q_hi, b_lo,
                     c_lo, c_hi, Kp, rb_lo, rb_hi, packed, colinfo);
  return hipGetLastError();
}

hipError_t launch_act_quant(const float* A, int64_t M, int64_t K, int64_t lda,
                            const ActPlan& ap, const int32_t* pos_dev,
                            const uint8_t* seg_dev, float* partial,
                            unsigned int* counter, float* s_a, uint8_t* packed,
                            hipStream_t stream) {
  const bool aligned = (K % 4 == 0) && (lda % 4 == 0) &&
                       (reinterpret_cast<uintptr_t>(A) % 16 == 0);
  if (aligned && M * K <= kSmallElems && M * (int64_t)ap.Kp <= 64 * 1024) {
    hipLaunchKernelGGL(k_act_small, dim3(1), dim3(kSmallThreads), (size_t)(M * ap.Kp), stream, A,
                       (int)M, (int)K, lda, pos_dev, seg_dev, ap, s_a, packed);
    return hipGetLastError();
  }
  if (aligned && lda == K && M * K / 4 < (int64_t)UINT32_MAX) {
    const int64_t total4 = M * K / 4;
    int64_t blocks = (total4 + 256 * kAbsU - 1) / (256 * kAbsU);
    if (blocks > kAbsmaxBlocks) blocks = kAbsmaxBlocks;
    hipLaunchKernelGGL(k_absmax_flat, dim3((unsigned)blocks), dim3(256), 0, stream,
                       reinterpret_cast<const float4*>(A), (uint32_t)total4, (uint32_t)(K / 4),
                       reinterpret_cast<const uchar4*>(seg_dev), ap, partial, counter, s_a);
  } else {
    int64_t blocks = M < kAbsmaxBlocks ? M : kAbsmaxBlocks;
    hipLaunchKernelGGL(k_absmax_rows, dim3((unsigned)blocks), dim3(256), 0, stream, A, M, K, lda,
                       seg_dev, ap, partial, counter, s_a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_act_pack, dim3((unsigned)M), dim3(256), (size_t)ap.Kp, stream, A, K,
                     lda, pos_dev, seg_dev, ap, s_a, packed, aligned ? 1 : 0);
  return hipGetLastError();
}

static GemmArgs make_args(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const uint8_t* w_packed, const TileDesc* tiles,
                          const ColInfo* colinfo, const uint8_t* shw, const WPlan& wp,
                          int64_t M, int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc) {
  GemmArgs a;
  a.act = act_packed; a.s_a = s_a; a.ap = ap; a.w = w_packed; a.tiles = tiles;
  a.colinfo = colinfo; a.shw = shw; a.wp = wp; a.M = M; a.N = N; a.Y = Y; a.ldy = ldy;
  a.acc = acc;
  return a;
}

hipError_t launch_mp_gemm(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const uint8_t* w_packed, const TileDesc* tiles,
                          const ColInfo* colinfo, const uint8_t* shw, const WPlan& wp,
                          int64_t M, int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc,
                          hipStream_t stream) {
  GemmArgs a = make_args(act_packed, s_a, ap, w_packed, tiles, colinfo, shw, wp, M, N, Y, ldy, acc);
  dim3 grid((unsigned)((wp.Np + 127) / 128), (unsigned)((M + 127) / 128));
  if (ap.S == 2)
    hipLaunchKernelGGL(k_gemm<2>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(k_gemm<1>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

bool gemv_fits(int64_t M, int Kp) {
  return M >= 1 && M <= kGemvMaxM && M * (int64_t)Kp <= 64 * 1024;
}

hipError_t launch_mp_gemv(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const uint8_t* w_packed, const TileDesc* tiles,
                          const ColInfo* colinfo, const uint8_t* shw, const WPlan& wp,
                          int64_t M, int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc,
                          hipStream_t stream) {
  GemmArgs a = make_args(act_packed, s_a, ap, w_packed, tiles, colinfo, shw, wp, M, N, Y, ldy, acc);
  dim3 grid((unsigned)(wp.Np / kGemvRows));
  const size_t lds = (size_t)M * ap.Kp;
  if (M == 1)
    hipLaunchKernelGGL(k_gemv<1>, grid, dim3(256), lds, stream, a);
  else if (M == 2)
    hipLaunchKernelGGL(k_gemv<2>, grid, dim3(256), lds, stream, a);
  else if (M <= 4)
    hipLaunchKernelGGL(k_gemv<4>, grid, dim3(256), lds, stream, a);
  else
    hipLaunchKernelGGL(k_gemv<8>, grid, dim3(256), lds, stream, a);
  return hipGetLastError();
}

}  // namespace soniq
