// Internal declarations shared by the host API (soniq_api.cpp) and the
// gfx950 kernels (soniq_kernels.hip).  Not part of the public ABI.
//
// Packed layout (both operands).  A b-bit channel is stored in a container
// of c bits, c in {1, 2, 4, 8}.  The input-channel axis is cut into
// granules of 64 channels (one int8 MFMA k-step) and rows into blocks of 16
// (one MFMA fragment).  One block-granule holds 64 "units" of 2*c bytes:
// unit l = kg*16 + r carries row r, channels [16*kg, 16*kg + 16) of the
// granule, at byte offset 2*c*l -- exactly the 16 bytes lane l of a wave
// feeds to v_mfma_i32_16x16x64_i8, so fragment loads are contiguous across
// lanes.  Inside a unit, element e = 4*j + b sits where one shift and one
// mask move four consecutive elements into the top bits of four bytes:
//   c = 8: byte e                                (unpack scale 1)
//   c = 4: two words, element 4j+b of a word at bits 8b+4j  (scale 2^4)
//   c = 2: one word; element 4j+b at bits 8b+4(j&1)+2 for j < 2 and at
//          bits 8b+4(j&1) for j >= 2 (the top / bottom half of nibble
//          2b+(j&1)), so masking the word with 0xCCCCCCCC, directly and
//          shifted left by 2, gives the c = 4 nibble arrangement
//          (values x4) that v_dot8_i32_i4 consumes   (unpack scale 2^6)
//   c = 1: 16 bits, element 4j+b at bit 4b+j; bit 1 = -1,
//          bit 0 = +1, unpacked to -64 / +64                 (scale 2^6)
// Integer dot products of unpacked bytes are exact multiples of
// 2^(sh_a + sh_w) and are shifted back before the epilogue.  Unsigned
// activation codes u whose width fills the container are stored as
// u - 2^(c-1) (a zero point); the epilogue adds 2^(c-1) * colsum, the sum of
// the weight codes of that output over the group.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace soniq {

constexpr int kGran = 64;     // channels per granule
constexpr int kBlk = 16;      // rows per block
constexpr int kGemmBN = 128;  // GEMM block tile columns (8 weight blocks)
constexpr int kMAlign = 256;  // activation rows are allocated in multiples of this
constexpr int kAbsmaxBlocks = 1024;  // max partial maxima (pairs) per activation batch

// 32-bit words of device state per activation handle (the single-pass
// quantizer's grid counters and maxima); zero between calls.
constexpr int kActStateWords = 8192;
// The word of that state that counts timed-out grid waits (never reset).
constexpr int kActStallWord = kActStateWords - 32;
// Device scratch of the allocation-free entry point: one per device, held
// until the process ends.  Its layout for a call: the grid state, the
// scales, the partial maxima, then the packed activations.
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr size_t kScratchScalesOff = (size_t)kActStateWords * 4;
constexpr size_t kScratchPartialOff = kScratchScalesOff + 4096;
// Address of this device's scratch (set up on the first call per device,
// with a fill kernel on `stream` that clears its grid state).
hipError_t scratch_device_ptr(hipStream_t stream, uint8_t** out);

// Quantizer of one width: code = sign1 ? (x < 0 ? -1 : +1)
//                                : clamp(rint(x / s), lo, hi), s = max/qdiv.
struct QParam {
  float qdiv;
  int lo, hi;
  int sign1;
};

// Per physical output position.
struct ColInfo {
  int32_t n;          // original output channel, -1 if the position is empty
  float s_w;          // weight scale of that channel
  int32_t colsum[2];  // sum of its codes over each activation group
};

// Per-column weight descriptor byte: unpack scale exponent, and bit 7 set
// for sign-bit (1-bit, +-1) channels.
constexpr uint8_t kShwSign = 0x80;

// Input-channel plan as the kernels see it.
struct ActPlan {
  int S;
  int c[2];               // container per activation group
  int sh[2];              // unpack scale exponent per group
  int zp[2];              // zero point per group (unsigned codes), else 0
  int kpad[2];            // padded channels per group (multiple of kGran)
  int ng[2];              // granules per group
  int padcnt[2];          // zero channels added to each group by the padding
  int Kp;                 // kpad[0] + kpad[1]
  int64_t seg_off[2];     // byte offset of each group's buffer
  int64_t mblk_bytes[2];  // bytes of one 16-row block over the group's granules
  QParam q[2];            // activation quantizer per group
  // Sub-group scales (GroupSize_act): each group is cut into nsub blocks of
  // gsub granules, each with its own scale; gsub = 0 keeps one scale per
  // group.
  int gsub[2];
  int nsub[2];
};

struct WPlan {
  int c_lo, c_hi;
  int ngt;   // granules over both groups (Kp / kGran)
  int nblk;  // 16-row blocks, a multiple of 8
  int nlo;   // blocks [0, nlo) hold the narrow width, the rest the wide one
  int Np;    // kBlk * nblk physical output positions
};

// Container and byte offset of weight block `blk` (blocks are contiguous,
// narrow ones first).
__host__ __device__ inline int wblk_c(const WPlan& wp, int blk) {
  return blk < wp.nlo ? wp.c_lo : wp.c_hi;
}
__host__ __device__ inline uint64_t wblk_off(const WPlan& wp, int blk) {
  const int lo = blk < wp.nlo ? blk : wp.nlo;
  return ((uint64_t)lo * wp.c_lo + (uint64_t)(blk - lo) * wp.c_hi) * (uint64_t)wp.ngt * 128u;
}

// Dense copies of the weights for the GEMV forms (handles packed with
// SONIQ_WPACK_DENSE): every code in b bits, b being its block's width
// (widths 3, 5, 6 and 7 no longer take the next power-of-two container).
// Block j (width b = dense_b) spans nquad = ceil(Kp / 128) quad-runs of 128
// planned channels; quad-run v of row r is a record of 4b words, b for
// each of its four 32-channel runs.  A run's 32 fields are byte-sliced:
// field 4q + e (q = 0..7) is field q of byte lane e, and lane e's 8 fields
// form a little-endian string of 8b bits whose byte k is byte e of the
// run's word k.  A field is the code's b-bit two's complement (b = 1: the
// bit set for -1).  Records are cut into b 16-byte chunks and interleaved
// for the GEMV's loads: quad-runs go in batches of 16; in batch i, with
// n_i = min(16, nquad - 16i) quad-runs, chunk k of the record of quad-run
// 16i + w, row r, is chunk 256*b*i + 16*n_i*k + 16w + r of the block.  Runs
// past Kp (half of the last quad-run when Kp / 64 is odd) are zero.
// Blocks keep the plan's order, 256*b*nquad bytes each; each holds one
// width (the plan does not merge widths into shared blocks for these
// handles).
__host__ __device__ inline int dense_b(const WPlan& wp, int blk, int b_lo, int b_hi) {
  return blk < wp.nlo ? b_lo : b_hi;
}
__host__ __device__ inline int dense_nquad(const WPlan& wp) { return (wp.ngt + 1) / 2; }
__host__ __device__ inline uint64_t dense_off(const WPlan& wp, int blk, int b_lo, int b_hi) {
  const int lo = blk < wp.nlo ? blk : wp.nlo;
  return ((uint64_t)lo * b_lo + (uint64_t)(blk - lo) * b_hi) * (uint64_t)dense_nquad(wp) * 256u;
}

// MFMA-native copies of narrow operands (handles packed with
// SONIQ_WPACK_F8F6F4).  Beside the integer units above, a handle keeps the
// codes of its narrow weight blocks and of its narrow activation groups in
// the operand formats of v_mfma_scale_f32_16x16x128_f8f6f4, which takes
// them straight from LDS with no widening: 1- and 2-bit containers as fp4
// (e2m1), 4-bit containers as fp6 (e3m2); both hold every stored code
// exactly (|code| <= 2, resp. <= 8).  The K axis of a precision group is
// cut into "fgranules" of 128 channels (two granules; a final one of an
// odd granule count is half zeros).  A 16-row block fgranule holds one unit
// per lane: lane l = q*16 + r carries row r, channels [32q, 32q + 32), 16
// bytes in fp4 (element e at bits 4e) or 24 bytes in fp6 (element e at bits
// 6e of the 192-bit value), stored as the lane's first 16 bytes at 16*l and,
// in fp6, its last 8 bytes at 1024 + 8*l.
constexpr int kFmtFp6 = 3;  // MFMA operand format code of e3m2
constexpr int kFmtFp4 = 4;  // of e2m1
__host__ __device__ constexpr int f_fmt(int c) { return c <= 2 ? kFmtFp4 : c == 4 ? kFmtFp6 : 0; }
__host__ __device__ constexpr int f_block_bytes(int fmt) { return fmt == kFmtFp4 ? 1024 : 1536; }

struct FPlan {
  int fa[2];            // format of activation group g's copy (0: none)
  int nfg[2];           // fgranules of group g
  int fw[2];            // format of the narrow / wide weight blocks' copy (0: none)
  int64_t fw_off[2][2];  // [group][class] byte offset of that region in the weight copy
  int64_t fa_off[2];     // byte offset of group g's region in the activation copy
  int64_t fa_mblk[2];    // bytes of one 16-row block of that region
};

// Geometry of the code image of a 3x3 convolution's input (implicit GEMM):
// per precision group g, B images of (H+2) x (W+2) pixels (a one-pixel halo
// holding the code of 0), each pixel cpad[g] channels (the group's channels
// in rank order, padded to 16) as rowbytes[g] bytes of 16-channel units in
// the unit encoding above, at byte img_off[g] of the image buffer.
// chan_ld: row length of the weights' rank -> channel table.
struct ConvGeo {
  int B, H, W;
  int cpad[2];
  int rowbytes[2];
  int64_t img_off[2];
  int chan_ld;
};

// A next layer that is an implicit 3x3 convolution (quantization fused into
// its producer): its code image and geometry, the channels of each
// precision group (ranks past them are padding), the images in the batch,
// and the stored code of 0.0 in each group (the halo's).
struct QnConv {
  ConvGeo cg;
  uint8_t* img;
  int cnt[2];
  int B;
  int halo[2];
};

struct WDev {
  const uint8_t* packed;
  const uint64_t* blk_off;  // byte offset of each block
  const uint8_t* blk_c;     // container of each block
  const ColInfo* colinfo;
  const uint8_t* shw;
  // Per 128-column GEMM tile: the original channels of its columns in
  // ascending order (-1 past the last), and each column's rank in that list.
  const int32_t* tile_cols;  // [Np / 128][128]
  const uint8_t* colrank;    // [Np]
};

// ---- launchers (soniq_kernels.hip) ---------------------------------------
hipError_t launch_wpack(const float* W, int64_t N, int64_t K, int64_t ldw,
                        const uint8_t* w_bits_dev, const int32_t* pos_dev,
                        const uint8_t* seg_dev, const int32_t* phys_dev,
                        const uint64_t* blk_off, const uint8_t* blk_c, QParam q_lo,
                        QParam q_hi, int b_lo, int Kp, uint8_t* packed, ColInfo* colinfo,
                        hipStream_t stream);

// Row stride (bytes) of the conv quantizer's LDS code rows, and whether a
// 16-row block of them fits the 64 KB a workgroup may hold.
inline int conv_quant_ldc(const ActPlan& ap) { return ap.Kp + 16; }
inline bool conv_quant_fits(const ActPlan& ap) { return kBlk * (int64_t)conv_quant_ldc(ap) <= 64 * 1024; }
// LDS of the window form: 16 code rows, the input rows a 16-pixel block
// touches (at most (15 + W - 1) / W + 1 image rows, one above, one below),
// then each channel's group byte and planned run start, then each window
// row's start index.  The form takes images at most 256 wide.
__host__ __device__ inline int64_t conv_win_rows(int64_t W) { return (15 + W - 1) / W + 1 + 2; }
inline size_t conv_win_lds(const ActPlan& ap, int64_t C, int64_t W) {
  return (size_t)(kBlk * (int64_t)conv_quant_ldc(ap) + ((conv_win_rows(W) * C * W + 15) & ~(int64_t)15) +
                  ((C + 15) & ~(int64_t)15) + 4 * C + 4 * conv_win_rows(W) * C);
}
hipError_t launch_conv_quant(const float* X, int64_t B, int64_t C, int64_t H, int64_t W,
                             const ActPlan& ap, const int32_t* pos_dev, const uint8_t* seg_dev,
                             float* partial, float* s_a, uint8_t* packed, hipStream_t stream);
// Batch of one row quantized inside the GEMV (soniq_quantize_mp_gemm): when
// it applies, its LDS, and the launch (ximg: the handle's row image).
size_t gemv_fused_lds(const ActPlan& ap, const WPlan& wp);
bool gemv_fused_fits(const float* A, int64_t K, const ActPlan& ap, const WPlan& wp);
hipError_t launch_gemv_fused(const float* A, int64_t K, const uint16_t* pos16_dev, uint8_t* act_packed,
                             float* s_a, const ActPlan& ap, const WDev& wd, const WPlan& wp,
                             int64_t N, uint16_t* Y, int32_t* acc, hipStream_t stream,
                             uint8_t* ximg);
// ximg (null: none): where a batch of one row also leaves its contiguous
// image for the batch-1 GEMV (a plan with a 4-bit group 0 and an 8-bit
// group 1 only); *ximg_done tells whether the launched path wrote it.
hipError_t launch_act_quant(const float* A, int64_t M, int64_t K, int64_t lda,
                            const ActPlan& ap, const int32_t* pos_dev,
                            const uint8_t* seg_dev, float* partial,
                            unsigned int* counter, float* s_a, uint8_t* packed,
                            hipStream_t stream, uint8_t* ximg = nullptr,
                            bool* ximg_done = nullptr);

// Sub-group scales: block scales in s_a[block], blocks of group 0 first;
// grp_dev[k] = block of original channel k.  At most kGAbsParts partial
// rows of block maxima (the handle's partial buffer holds that many), and
// at most kGSubMax blocks.
constexpr int kGAbsParts = 1024;
constexpr int kGSubMax = 256;
// posg_dev[k] = pos_dev[k] | grp_dev[k] << 16 (the single pass's table);
// counter: the handle's grid state.
hipError_t launch_act_quant_grouped(const float* A, int64_t M, int64_t K, int64_t lda,
                                    const ActPlan& ap, const int32_t* pos_dev,
                                    const int32_t* grp_dev, const int32_t* posg_dev,
                                    float* partial, unsigned int* counter, float* s_a,
                                    uint8_t* packed, hipStream_t stream);
hipError_t launch_mp_gemm_grouped(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                  const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                                  uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream);
// The same for batches of at most 8 rows without matrix cores: one exact
// int32 sum per activation block and output, folded in block order; where
// it applies (activation containers 4 and 8, weight containers 2, 4, 8).
bool gemv_g_fits(int64_t M, const ActPlan& ap, const WPlan& wp);
hipError_t launch_mp_gemv_grouped(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                  const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                                  uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream);

// The GEMM whose epilogue also quantizes its outputs for the next layer
// with static scales s_next (host, one per next-layer group): codes go to
// the byte image img ((img_rows + 8) * ap2.Kp bytes: from the GEMM tiles
// in 16-row blocks of 16-byte columns, row m and position p at
// img[(m/16)*16*ap2.Kp + 16*p + m%16]; from the GEMV forms row-major after
// those img_rows rows, img[(img_rows + m)*ap2.Kp + p]; qtab: [Np] next-layer
// group per
// physical column, then [Np] next-layer position per tile column in
// ascending original order), then k_pack_img writes them as the next
// handle's packed rows and its scales.  Y may be null.
// A next layer with sub-group scales takes one static scale per block
// (s_next[nsub], qtab's groups are then blocks), stored with their
// reciprocals (brs2, nsub floats) by a small launch before the GEMM.
// Batches of at most 8 rows run the GEMV forms with the same epilogue
// (qtab then also holds, at [2 Np, 3 Np), the next-layer position of each
// physical column); ximg2 receives the next layer's row image for one row,
// ximg is this layer's (or null).  pimg/pcg: this layer is an implicit
// convolution reading that code image (its tiles then carry the epilogue).
// conv: the next layer is an implicit convolution, whose positions are its
// channel ranks (qtab as above in that space) and whose haloed image
// k_pack_conv_img writes instead of packed rows.
hipError_t launch_mp_gemm_qnext(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                const WDev& wd, const WPlan& wp, int64_t M, int64_t N, uint16_t* Y,
                                int64_t ldy, int32_t* acc, uint8_t* img, int64_t img_rows,
                                const int32_t* qtab, const ActPlan& ap2, const float* s_next,
                                float* s_a2, float* brs2, uint8_t* packed2, hipStream_t stream,
                                uint8_t* ximg2, const uint8_t* ximg, const uint8_t* pimg = nullptr,
                                const ConvGeo* pcg = nullptr, const QnConv* conv = nullptr);

hipError_t launch_mp_gemm(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                          uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream,
                          const FPlan* fp = nullptr, const uint8_t* fa = nullptr,
                          const uint8_t* fw = nullptr);

// Implicit 3x3 convolution: the group maxima of X and its haloed code image
// (seg[9c] = group of channel c; chan[g*cg.chan_ld + rank] = channel), then
// the GEMM that gathers each tap's units from the image.
hipError_t launch_conv_img(const float* X, int64_t B, int64_t C, int64_t H, int64_t W,
                           const ActPlan& ap, const ConvGeo& cg, const uint8_t* seg_dev,
                           const int32_t* chan_dev, float* partial, float* s_a, uint8_t* img,
                           hipStream_t stream);
// Whether the implicit-convolution GEMM has an instance for these
// containers (activations 4 + 8 bits; weights 4/4, 1/4, 2/4, 2/8 or 4/8).
// The two-pass form of the fused quantization (batch maximum): the GEMM
// tiles store Y and write each next-layer group's largest |Y| (qtab's
// groups, as above) as one float pair per tile into slots; then
// launch_act_bf16 quantizes the next layer's activations from the stored
// bf16 Y exactly as launch_act_quant would from float(Y), with the maxima
// of nslot pairs (nslot = 0: reduced from the batch itself).
// (pimg, pcg: an implicit convolution's code image and geometry as the
// producer's input.)
hipError_t launch_mp_gemm_ymax(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                               const WDev& wd, const WPlan& wp, int64_t M, int64_t N, uint16_t* Y,
                               int64_t ldy, int32_t* acc, const int32_t* qtab, float* slots,
                               hipStream_t stream, const uint8_t* pimg = nullptr,
                               const ConvGeo* pcg = nullptr);
hipError_t launch_act_bf16(const uint16_t* Y, int64_t M, int64_t K, int64_t ldy, const ActPlan& ap,
                           const int32_t* pos_dev, const uint8_t* seg_dev, const float* slots,
                           int nslot, float* s_a, uint8_t* packed, uint8_t* ximg,
                           hipStream_t stream);
// The same into a next implicit convolution (ap and conv describe it): the
// blocked byte image bimg from Y with posn (each of the N producer
// columns' rank-space position), then its haloed code image conv.img.
hipError_t launch_img_bf16(const uint16_t* Y, int64_t M, int N, int64_t ldy, const int32_t* posn,
                           const ActPlan& ap, const QnConv& conv, const float* slots, int nslot,
                           float* s_a, uint8_t* bimg, hipStream_t stream);

// The implicit convolution's tiles: two activation widths in 4- and 8-bit
// containers, or one width in a 4- or 8-bit container; any pair of weight
// containers.  The next-layer and batch-maximum epilogues from a
// convolution take the two-width plans only (conv_gemm_qn_supported).
bool conv_gemm_supported(const ActPlan& ap, const WPlan& wp);
bool conv_gemm_qn_supported(const ActPlan& ap, const WPlan& wp);
hipError_t launch_mp_gemm_conv(const uint8_t* img, const ConvGeo& cg, const float* s_a,
                               const ActPlan& ap, const WDev& wd, const WPlan& wp, int64_t M,
                               int64_t N, uint16_t* Y, int64_t ldy, int32_t* acc,
                               hipStream_t stream);

// Converts integer units to their MFMA-native copy: `nblk` 16-row blocks,
// block b's units at src + b*src_bstride (ng granules of container c),
// its copy (fmt) at dst + b*dst_bstride.
// The dense copy of a handle's weights (layout above) from its units.
hipError_t launch_dense_pack(const uint8_t* packed, const WPlan& wp, int b_lo, int b_hi,
                             uint8_t* dense, hipStream_t stream);
// The GEMV forms on the dense copy: batches of at most 8 rows (when
// gemv_dense_fits), results as launch_mp_gemv's.
bool gemv_dense_fits(int64_t M, const ActPlan& ap);
hipError_t launch_mp_gemv_dense(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                                const WDev& wd, const WPlan& wp, const uint8_t* dense, int b_lo,
                                int b_hi, int64_t M, int64_t N, uint16_t* Y, int64_t ldy,
                                int32_t* acc, hipStream_t stream);
hipError_t launch_to_fp(const uint8_t* src, int64_t src_bstride, int c, int ng, int64_t nblk,
                        uint8_t* dst, int64_t dst_bstride, int fmt, hipStream_t stream);

// ximg: a single row's contiguous image (see launch_act_quant), or null.
hipError_t launch_mp_gemv(const uint8_t* act_packed, const float* s_a, const ActPlan& ap,
                          const WDev& wd, const WPlan& wp, int64_t M, int64_t N,
                          uint16_t* Y, int64_t ldy, int32_t* acc, hipStream_t stream,
                          const uint8_t* ximg = nullptr);

// One plain read of `bytes` (a multiple of 16) at src: 8 KB per workgroup,
// the XOR of its words to sink[workgroup] (a measurement aid).
hipError_t launch_stream_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream);

// Whether the GEMV kernel handles M rows for this plan.
bool gemv_fits(int64_t M, const ActPlan& ap, const WPlan& wp);

}  // namespace soniq
