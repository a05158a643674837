/*
 * soniq_oracle.c -- plain, slow CPU oracle for SONIQ's inference hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file: only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or constant with
 * the HIP library.
 *
 * What it computes (SONIQ, arXiv 2311.14114):
 *   - per-group max-abs scale                      (Sec. 3, "Enabling Low-Cost
 *                                                   Fixed-Point Operations", item 1)
 *   - unsigned activation codes clip(round(a/s*(2^n-1)), 0, 2^n-1)
 *                                                  (same paragraph, item 2)
 *   - signed weight codes: symmetric grid +-(2^(b-1)-1) (default), or the
 *     two's-complement fraction grid of Eq. (1)    (item 3, Eq. 1)
 *   - channels of equal precision form one group sharing one scale per fused
 *     dot product                                  (Sec. 2.4, C1 and C2)
 *   - integer multiply-accumulate of the codes, one int32 sum per activation
 *     precision group                              (Alg. 1, Phase II forward)
 *   - rescale once, round to bf16.
 *
 * Floating point: quantization decisions are taken in fp32 (IEEE division,
 * round-half-to-even rint, no FMA contraction); the MAC is exact in int64;
 * the reference epilogue is fp64, rounded once to bf16.
 *
 * Compiled with: -O2 -fopenmp -ffp-contract=off -fno-fast-math.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ O1 ---
 * Largest code magnitude for a b-bit code.
 *   mode 0 (signed symmetric):   2^(b-1)-1 for b>=2; b=1 is sign mode (+-1).
 *   mode 1 (unsigned):           2^b-1                 (item 2 of the codec)
 *   mode 2 (Eq. 1 two's-complement fraction): 2^(b-1) is the grid
 *           denominator, codes span [-2^(b-1), 2^(b-1)-1].
 */
enum { ORC_SIGNED = 0, ORC_UNSIGNED = 1, ORC_TWOS_FRACTION = 2 };

int64_t orc_qmax(int bits, int mode) {
  if (bits < 1 || bits > 8) return -1;
  if (mode == ORC_UNSIGNED) return ((int64_t)1 << bits) - 1;
  if (mode == ORC_TWOS_FRACTION) return (int64_t)1 << (bits - 1);
  if (bits == 1) return 1;
  return ((int64_t)1 << (bits - 1)) - 1;
}

/* ------------------------------------------------------------------ O2 ---
 * Scale of a group from its max-abs m (item 1: s_g = max |x|).  The code
 * step is m / Q, computed as one IEEE fp32 division.  Sign mode keeps m.
 */
float orc_scale(float maxabs, int bits, int mode) {
  if (mode == ORC_SIGNED && bits == 1) return maxabs;
  return maxabs / (float)orc_qmax(bits, mode);
}

/* ---------------------------------------------------------------- O3/O5 --
 * Code of one value x under step s.
 *   sign mode (signed, b=1): -1 if x < 0 else +1 (so -0 and +0 give +1).
 *   otherwise: if s == 0 the code is 0; else r = fp32(x / s) and the code is
 *   rint(r) (ties to even) clamped to the grid of the mode.
 */
int32_t orc_code(float x, float s, int bits, int mode) {
  if (mode == ORC_SIGNED && bits == 1) return (x < 0.0f) ? -1 : 1;
  if (s == 0.0f) return 0;
  float r = x / s;
  float q = rintf(r);
  int64_t lo, hi;
  if (mode == ORC_UNSIGNED) {
    lo = 0;
    hi = orc_qmax(bits, mode);
  } else if (mode == ORC_TWOS_FRACTION) {
    hi = orc_qmax(bits, mode) - 1;
    lo = -orc_qmax(bits, mode);
  } else {
    hi = orc_qmax(bits, mode);
    lo = -hi;
  }
  if (q < (float)lo) return (int32_t)lo;
  if (q > (float)hi) return (int32_t)hi;
  return (int32_t)q;
}

/* ------------------------------------------------------------------ O2/O3 -
 * Weights W[N,K] (row stride ldw): one scale per output channel n from the
 * max-abs of its row, codes q_w[N,K] (dense, row stride K).
 * wmode: ORC_SIGNED (symmetric grid) or ORC_TWOS_FRACTION (Eq. 1 grid).
 */
void orc_quantize_weights(const float* W, int64_t N, int64_t K, int64_t ldw,
                          const uint8_t* w_bits, int wmode, int32_t* q_w,
                          float* s_w) {
  int64_t n;
#pragma omp parallel for schedule(static)
  for (n = 0; n < N; ++n) {
    float m = 0.0f;
    for (int64_t k = 0; k < K; ++k) {
      float a = fabsf(W[n * ldw + k]);
      if (a > m) m = a;
    }
    float s = orc_scale(m, w_bits[n], wmode);
    s_w[n] = s;
    for (int64_t k = 0; k < K; ++k)
      q_w[n * K + k] = orc_code(W[n * ldw + k], s, w_bits[n], wmode);
  }
}

/* ------------------------------------------------------------------ O4 ---
 * Activation precision groups: the distinct widths of a_bits, ascending,
 * each group holding every channel of that width (Alg. 1 permutes equal
 * precisions together; C2 gives each group one scale).
 * Returns S (1 or 2), or -1 if there are more than two widths or a width is
 * outside 1..8.  seg_bits[S] = widths; seg_of[k] = group of channel k.
 */
int orc_segments(const uint8_t* a_bits, int64_t K, uint8_t* seg_bits,
                 uint8_t* seg_of) {
  int seen[9] = {0};
  for (int64_t k = 0; k < K; ++k) {
    if (a_bits[k] < 1 || a_bits[k] > 8) return -1;
    seen[a_bits[k]] = 1;
  }
  int S = 0;
  for (int b = 1; b <= 8; ++b)
    if (seen[b]) {
      if (S == 2) return -1;
      seg_bits[S++] = (uint8_t)b;
    }
  for (int64_t k = 0; k < K; ++k) seg_of[k] = (a_bits[k] == seg_bits[0]) ? 0 : 1;
  return S;
}

/* ---------------------------------------------------------------- O4/O5 --
 * Activations A[M,K] (row stride lda): per group g the scale comes from the
 * max-abs over all rows and all channels of the group; codes q_a[M,K].
 * a_signed = 1: symmetric signed grid; 0: the unsigned codec.
 * Returns S, or -1 on bad widths.
 */
int orc_quantize_act(const float* A, int64_t M, int64_t K, int64_t lda,
                     const uint8_t* a_bits, int a_signed, int32_t* q_a,
                     float* s_a, uint8_t* seg_bits, uint8_t* seg_of) {
  int S = orc_segments(a_bits, K, seg_bits, seg_of);
  if (S < 0) return -1;
  int mode = a_signed ? ORC_SIGNED : ORC_UNSIGNED;
  float mx[2] = {0.0f, 0.0f};
  for (int64_t m = 0; m < M; ++m)
    for (int64_t k = 0; k < K; ++k) {
      float a = fabsf(A[m * lda + k]);
      if (a > mx[seg_of[k]]) mx[seg_of[k]] = a;
    }
  for (int g = 0; g < S; ++g) s_a[g] = orc_scale(mx[g], seg_bits[g], mode);
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t k = 0; k < K; ++k) {
      int g = seg_of[k];
      q_a[m * K + k] = orc_code(A[m * lda + k], s_a[g], seg_bits[g], mode);
    }
  return S;
}

/* ------------------------------------------------------------- O4/O5 ---
 * Sub-group scales (GroupSize_act of the design-space parameters, Sec. 3,
 * and the group-wise activation normalization of the transformer setup,
 * Sec. 5).  Channels are put in the Alg. 1 order (narrow width first,
 * original index order inside a width); each precision group is then cut
 * into consecutive blocks of group_bits / c channels, c the container of
 * its width (the next power of two >= b), so that one block fills
 * group_bits of storage.  Each block has its own scale, from the max-abs
 * over all rows and its channels.  Blocks are numbered in that order,
 * group 0's first.  group_bits = 0 keeps one block per precision group.
 * Outputs: codes q_a[M,K], scales s_a[S] (S = number of blocks, at most
 * cap), the width of each block sub_bits[S], and the block of each channel
 * sub_of[K].  Returns S, or -1 on bad widths, a group_bits that is not a
 * positive multiple of every block's container, or more than cap blocks.
 */
static int orc_container_bits(int b) {
  int c = 1;
  while (c < b) c <<= 1;
  return c;
}

int orc_quantize_act_grouped(const float* A, int64_t M, int64_t K, int64_t lda,
                             const uint8_t* a_bits, int a_signed, int group_bits,
                             int cap, int32_t* q_a, float* s_a, uint8_t* sub_bits,
                             int32_t* sub_of) {
  uint8_t seg_bits[2];
  uint8_t* seg_of = (uint8_t*)malloc((size_t)(K > 0 ? K : 1));
  int S = orc_segments(a_bits, K, seg_bits, seg_of);
  if (S < 0 || group_bits < 0) {
    free(seg_of);
    return -1;
  }
  int64_t len[2] = {0, 0}, per[2] = {0, 0}, nsub[2] = {0, 0};
  for (int64_t k = 0; k < K; ++k) len[seg_of[k]]++;
  for (int g = 0; g < S; ++g) {
    int c = orc_container_bits(seg_bits[g]);
    if (group_bits == 0) {
      per[g] = len[g];
    } else {
      if (group_bits % c != 0) {
        free(seg_of);
        return -1;
      }
      per[g] = group_bits / c;
    }
    nsub[g] = (len[g] + per[g] - 1) / per[g];
  }
  int total = (int)(nsub[0] + (S == 2 ? nsub[1] : 0));
  if (total > cap) {
    free(seg_of);
    return -1;
  }
  /* rank of each channel inside its precision group, in index order */
  int64_t seen[2] = {0, 0};
  for (int64_t k = 0; k < K; ++k) {
    int g = seg_of[k];
    int64_t r = seen[g]++;
    sub_of[k] = (int32_t)((g == 1 ? nsub[0] : 0) + r / per[g]);
  }
  for (int j = 0; j < total; ++j) sub_bits[j] = seg_bits[j < nsub[0] ? 0 : 1];
  int mode = a_signed ? ORC_SIGNED : ORC_UNSIGNED;
  float* mx = (float*)calloc((size_t)total, sizeof(float));
  for (int64_t m = 0; m < M; ++m)
    for (int64_t k = 0; k < K; ++k) {
      float a = fabsf(A[m * lda + k]);
      if (a > mx[sub_of[k]]) mx[sub_of[k]] = a;
    }
  for (int j = 0; j < total; ++j) s_a[j] = orc_scale(mx[j], sub_bits[j], mode);
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t k = 0; k < K; ++k) {
      int j = sub_of[k];
      q_a[m * K + k] = orc_code(A[m * lda + k], s_a[j], sub_bits[j], mode);
    }
  free(mx);
  free(seg_of);
  return total;
}

/* ------------------------------------------------------------------ O6 ---
 * Integer MAC: ACC[g][m][n] = sum over channels k of group g of
 * q_a[m,k] * q_w[n,k], summed in int64.  grp_of[k] is the scale group of
 * channel k (0 .. S-1): a precision group, or a sub-group of one.  Returns
 * 0, or -1 if a sum does not fit int32 (the sums are then still stored,
 * truncated).
 */
int orc_mac(const int32_t* q_a, const int32_t* q_w, const int32_t* grp_of,
            int64_t M, int64_t N, int64_t K, int S, int32_t* acc) {
  int overflow = 0;
  int64_t m;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : overflow)
  for (m = 0; m < M; ++m) {
    int64_t* sum = (int64_t*)malloc(sizeof(int64_t) * (size_t)S);
    for (int64_t n = 0; n < N; ++n) {
      for (int g = 0; g < S; ++g) sum[g] = 0;
      for (int64_t k = 0; k < K; ++k)
        sum[grp_of[k]] += (int64_t)q_a[m * K + k] * (int64_t)q_w[n * K + k];
      for (int g = 0; g < S; ++g) {
        if (sum[g] > INT32_MAX || sum[g] < INT32_MIN) overflow = 1;
        acc[((int64_t)g * M + m) * N + n] = (int32_t)sum[g];
      }
    }
    free(sum);
  }
  return overflow ? -1 : 0;
}

/* One output's accumulators, for sampled checks at full size. */
void orc_mac_at(const int32_t* q_a, const int32_t* q_w, const int32_t* grp_of,
                int64_t K, int S, int64_t count, const int64_t* ms,
                const int64_t* ns, int64_t* out /* [count][S] */) {
  int64_t i;
#pragma omp parallel for schedule(static)
  for (i = 0; i < count; ++i) {
    int64_t* sum = out + i * S;
    for (int g = 0; g < S; ++g) sum[g] = 0;
    const int32_t* a = q_a + ms[i] * K;
    const int32_t* w = q_w + ns[i] * K;
    for (int64_t k = 0; k < K; ++k) sum[grp_of[k]] += (int64_t)a[k] * (int64_t)w[k];
  }
}

/* ------------------------------------------------------------------ O7 ---
 * bf16 from fp64, rounded once to nearest, ties to even.  bf16 keeps 8
 * significant bits and fp32's exponent range (normal >= 2^-126, subnormal
 * step 2^-133, largest finite (2 - 2^-7) * 2^127).
 */
uint16_t orc_bf16_from_f64(double v) {
  if (v == 0.0) return signbit(v) ? 0x8000u : 0x0000u;
  int ex;
  (void)frexp(fabs(v), &ex); /* |v| = f * 2^ex with f in [0.5, 1) */
  int step = ex - 8;              /* ulp exponent of an 8-significant-bit value */
  if (step < -133) step = -133;
  double q = nearbyint(ldexp(fabs(v), -step)); /* exact scaling, RNE */
  double r = ldexp(q, step);
  double maxf = ldexp(255.0, 120); /* (2 - 2^-7) * 2^127 */
  float rf;
  if (r > maxf)
    rf = INFINITY;
  else
    rf = (float)r; /* exact: r has <= 8 significant bits */
  if (v < 0) rf = -rf;
  uint32_t u;
  memcpy(&u, &rf, 4);
  return (uint16_t)(u >> 16);
}

/* bf16 from fp32 with one round to nearest even on the dropped 16 bits. */
uint16_t orc_bf16_from_f32(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  uint32_t lsb = (u >> 16) & 1u;
  return (uint16_t)((u + 0x7FFFu + lsb) >> 16);
}

/* Reference output: y = bf16( s_w[n] * sum_g s_a[g] * ACC[g][m][n] ) in fp64. */
void orc_epilogue_ref(const int32_t* acc, const float* s_a, const float* s_w,
                      int64_t M, int64_t N, int S, uint16_t* y) {
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t n = 0; n < N; ++n) {
      double t = 0.0;
      for (int g = 0; g < S; ++g)
        t += (double)s_a[g] * (double)acc[((int64_t)g * M + m) * N + n];
      y[m * N + n] = orc_bf16_from_f64(t * (double)s_w[n]);
    }
}

/* Replay output: the same value in a fixed fp32 order -- t = f(ACC0)*s_a0;
 * then for each later group g in order t = t + f(ACCg)*s_ag (separate
 * multiply and add); t = t*s_w; bf16 RNE. */
void orc_epilogue_replay(const int32_t* acc, const float* s_a, const float* s_w,
                         int64_t M, int64_t N, int S, uint16_t* y) {
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t n = 0; n < N; ++n) {
      float t = (float)acc[m * N + n] * s_a[0];
      for (int g = 1; g < S; ++g) {
        float u = (float)acc[((int64_t)g * M + m) * N + n] * s_a[g];
        t = t + u;
      }
      t = t * s_w[n];
      y[m * N + n] = orc_bf16_from_f32(t);
    }
}

/* Replay value before the bf16 rounding: the fp32 number the fixed-order
 * epilogue produces, y_f32[m,n]. */
void orc_epilogue_replay_f32(const int32_t* acc, const float* s_a, const float* s_w,
                             int64_t M, int64_t N, int S, float* y) {
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t n = 0; n < N; ++n) {
      float t = (float)acc[m * N + n] * s_a[0];
      for (int g = 1; g < S; ++g) {
        float u = (float)acc[((int64_t)g * M + m) * N + n] * s_a[g];
        t = t + u;
      }
      y[m * N + n] = t * s_w[n];
    }
}

/* --------------------------------------------------------------- O4/O5 ---
 * Activation codes with static (calibrated) group scales s_a[g] given by
 * the caller instead of the batch maximum (the quantizer a producing
 * kernel can run on its own outputs, Sec. 4's fusion of quantization into
 * the preceding operation): q_a[m,k] = code(A[m,k], s_a[seg_of[k]]),
 * clamped to the width's range.  Returns S, or -1 on bad widths.
 */
int orc_quantize_act_static(const float* A, int64_t M, int64_t K, int64_t lda,
                            const uint8_t* a_bits, int a_signed, const float* s_a,
                            int32_t* q_a) {
  uint8_t seg_bits[2];
  uint8_t* seg_of = (uint8_t*)malloc((size_t)(K > 0 ? K : 1));
  int S = orc_segments(a_bits, K, seg_bits, seg_of);
  if (S < 0) {
    free(seg_of);
    return -1;
  }
  int mode = a_signed ? ORC_SIGNED : ORC_UNSIGNED;
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t k = 0; k < K; ++k) {
      int g = seg_of[k];
      q_a[m * K + k] = orc_code(A[m * lda + k], s_a[g], seg_bits[g], mode);
    }
  free(seg_of);
  return S;
}

/* Static block scales: the codes of orc_quantize_act_grouped's blocks with
 * the caller's scale per block (s_blocks[S]) in place of the batch
 * maximum.  Fills sub_of[K]; returns S, or -1 as orc_quantize_act_grouped. */
int orc_quantize_act_static_grouped(const float* A, int64_t M, int64_t K, int64_t lda,
                                    const uint8_t* a_bits, int a_signed, int group_bits,
                                    int cap, const float* s_blocks, int32_t* q_a,
                                    int32_t* sub_of) {
  /* the block plan: run the grouped quantizer on one row of zeros */
  float* zero = (float*)calloc((size_t)(K > 0 ? K : 1), sizeof(float));
  int32_t* qz = (int32_t*)malloc(sizeof(int32_t) * (size_t)(K > 0 ? K : 1));
  float* sz = (float*)malloc(sizeof(float) * (size_t)(cap > 0 ? cap : 1));
  uint8_t* bits = (uint8_t*)malloc((size_t)(cap > 0 ? cap : 1));
  int S = orc_quantize_act_grouped(zero, 1, K, K, a_bits, a_signed, group_bits, cap, qz, sz, bits,
                                   sub_of);
  free(zero);
  free(qz);
  free(sz);
  if (S < 0) {
    free(bits);
    return -1;
  }
  int mode = a_signed ? ORC_SIGNED : ORC_UNSIGNED;
  int64_t m;
#pragma omp parallel for schedule(static)
  for (m = 0; m < M; ++m)
    for (int64_t k = 0; k < K; ++k) {
      int j = sub_of[k];
      q_a[m * K + k] = orc_code(A[m * lda + k], s_blocks[j], bits[j], mode);
    }
  free(bits);
  return S;
}

/* ------------------------------------------------------------------ O8 ---
 * Canonical dense packing of a run of codes, used to account bytes: element
 * j occupies bits [(j mod 32/c)*c, +c) of 32-bit word floor(j*c/32), with
 * container c = next power of two >= b.  Signed codes are two's complement;
 * sign mode stores 1 for -1 and 0 for +1; unsigned codes are stored as is.
 * Returns the number of 32-bit words written.
 */
int orc_container(int bits) {
  int c = 1;
  while (c < bits) c <<= 1;
  return c;
}

int64_t orc_pack(const int32_t* codes, int64_t n, int bits, int mode,
                 uint32_t* words) {
  int c = orc_container(bits);
  int per = 32 / c;
  int64_t nw = (n + per - 1) / per;
  uint32_t mask = (c == 32) ? 0xFFFFFFFFu : ((1u << c) - 1u);
  for (int64_t w = 0; w < nw; ++w) words[w] = 0;
  for (int64_t j = 0; j < n; ++j) {
    uint32_t field;
    if (mode == ORC_SIGNED && bits == 1)
      field = (codes[j] < 0) ? 1u : 0u;
    else
      field = ((uint32_t)codes[j]) & mask;
    words[j / per] |= field << ((j % per) * c);
  }
  return nw;
}

void orc_unpack(const uint32_t* words, int64_t n, int bits, int mode,
                int32_t* codes) {
  int c = orc_container(bits);
  int per = 32 / c;
  uint32_t mask = (1u << c) - 1u;
  for (int64_t j = 0; j < n; ++j) {
    uint32_t field = (words[j / per] >> ((j % per) * c)) & mask;
    if (mode == ORC_SIGNED && bits == 1)
      codes[j] = field ? -1 : 1;
    else if (mode == ORC_UNSIGNED)
      codes[j] = (int32_t)field;
    else
      codes[j] = (field & (1u << (c - 1))) ? (int32_t)field - (int32_t)(1u << c)
                                           : (int32_t)field;
  }
}

/* Threads an OpenMP region of the oracle runs on (for reporting only). */
int orc_threads(void) { return omp_get_max_threads(); }
