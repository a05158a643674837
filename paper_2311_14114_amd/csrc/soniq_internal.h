// Internal declarations shared by the host API (soniq_api.cpp) and the
// gfx950 kernels (soniq_kernels.hip).  Not part of the public ABI.
//
// Packed-field format (both operands).  A b-bit channel is stored in a
// container of c bits, c in {1, 2, 4, 8}.  A 32-bit word holds E = 32/c
// consecutive elements of one row; element e = 4*j + b (b in 0..3,
// j in 0..8/c-1) occupies bits [8*b + c*j, 8*b + c*j + c).  This order lets
// one shift and one mask move the fields of four consecutive elements into
// the top bits of four bytes, so unpacking to int8 costs two VALU ops per
// four elements and leaves the elements in their natural order:
//   c = 8: the byte itself                      (scale 1)
//   c = 4: two's complement nibble, x16         (scale 2^4)
//   c = 2: two's complement pair, x64           (scale 2^6)
//   c = 1: sign bit (1 = -1, 0 = +1) -> +-64    (scale 2^6)
// Integer dot products of unpacked bytes are therefore exact multiples of
// 2^(sh_a + sh_w) and are shifted back before the epilogue.
// Unsigned activation codes u whose width fills the container are stored as
// u - 2^(c-1) (a zero point); the epilogue adds 2^(c-1) * colsum, where
// colsum is the sum of the weight codes of that output over the group.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace soniq {

constexpr int kGran = 64;      // input-channel padding granule (elements)
constexpr int kNTile = 64;     // output-channel tile of the packed weights
constexpr int kGemmBM = 128;   // GEMM block tile rows (activation rows)
constexpr int kGemmBN = 128;   // GEMM block tile columns (output channels)
constexpr int kGemvRows = 16;  // output channels per GEMV workgroup
constexpr int kAbsmaxBlocks = 1024;

// Quantizer of one width: code = sign1 ? (x < 0 ? -1 : +1)
//                                : clamp(rint(x / s), lo, hi), s = max/qdiv.
struct QParam {
  float qdiv;
  int lo, hi;
  int sign1;
};

// One tile of kNTile output channels in the packed weight buffer.  Rows
// [0, n_lo) use the narrow container, [n_lo, n_rows) the wide one; the tile
// spans original channels [kNTile*t, kNTile*t + n_rows) in a stable
// narrow-first order.
struct TileDesc {
  uint64_t base;  // byte offset of the tile
  int32_t n_lo;
  int32_t n_rows;
};

// Per physical output position.
struct ColInfo {
  int32_t n;          // original output channel, -1 if the position is empty
  float s_w;          // weight scale of that channel
  int32_t colsum[2];  // sum of its codes over each activation group
};

// Input-channel plan as the kernels see it.
struct ActPlan {
  int S;
  int c[2];             // container per activation group
  int sh[2];            // unpack scale exponent per group
  int zp[2];            // zero point per group (unsigned codes), else 0
  int kpad[2];          // padded channels per group (multiple of kGran)
  int64_t row_bytes[2]; // bytes per row in each group's buffer
  int64_t seg_off[2];   // byte offset of each group's buffer
  int Kp;               // kpad[0] + kpad[1]
  int padcnt[2];        // zero channels added to each group by the padding
  QParam q[2];          // activation quantizer per group
};

// Per-column weight descriptor byte: unpack scale exponent, and bit 7 set
// for sign-bit (1-bit, +-1) channels.
constexpr uint8_t kShwSign = 0x80;

struct WPlan {
  int c_lo, c_hi;
  int sh_lo, sh_hi;
  int64_t rb_lo, rb_hi;  // packed row bytes for each container
  int ntiles;
  int Np;                // kNTile * ntiles physical positions
};

// ---- launchers (soniq_kernels.hip) ---------------------------------------
hipError_t launch_wpack(const float* W, int64_t N, int64_t K, int64_t ldw,
                        const uint8_t* w_bits_dev, const int32_t* pos_dev,
                        const uint8_t* seg_dev, const int64_t* row_off_dev,
                        const int32_t* phys_dev, QParam q_lo, QParam q_hi, int b_lo,
                        int c_lo, int c_hi, int Kp, int kpad0, int64_t rb_lo,
                        int64_t rb_hi, uint8_t* packed, ColInfo* colinfo,
                        hipStream_t stream);

hipError_t launch_act_quant(const float* A, int64_t M, int64_t K, int64_t lda,
                            const ActPlan& ap, const int32_t* pos_dev,
                            const uint8_t* seg_dev, float* partial,
                            unsigned int* counter, float* s_a, uint8_t* packed,
                            hipStream_t stream);

hipError_t launch_mp_gemm(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const uint8_t* w_packed, const TileDesc* tiles,
                          const ColInfo* colinfo, const uint8_t* shw, const WPlan& wp,
                          int64_t M, int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc,
                          hipStream_t stream);

hipError_t launch_mp_gemv(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const uint8_t* w_packed, const TileDesc* tiles,
                          const ColInfo* colinfo, const uint8_t* shw, const WPlan& wp,
                          int64_t M, int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc,
                          hipStream_t stream);

// Largest M handled by the GEMV kernel, and whether it fits for a plan.
constexpr int kGemvMaxM = 8;
bool gemv_fits(int64_t M, int Kp);

}  // namespace soniq
