/*
 * soniq.h -- C ABI of libsoniq, a gfx950 (MI355X) implementation of the
 * inference hot path of SONIQ (arXiv 2311.14114): a per-channel two-level
 * mixed-precision integer matrix multiply
 *
 *     Y[m, n] = bf16( s_w[n] * sum_g s_a[g] * ACC[g][m][n] ),
 *     ACC[g][m][n] = sum over input channels k of precision group g of
 *                    q_a[m, k] * q_w[n, k]                   (exact, int32)
 *
 * used for linear layers and for convolutions lowered to a GEMM (im2col).
 *
 * Paper passages the calls implement:
 *   - Sec. 2.4, constraints C1 (one precision per SIMD/tile block), C2 (one
 *     scale per fused dot product), C3 (few precision levels: at most two
 *     widths per operand here), C5 (coalesced channel-packed layout);
 *   - Sec. 3, Phase I "Dynamic channel re-ordering" and Alg. 1 (channels of
 *     equal precision made contiguous), Fig. "normalization" (each
 *     equal-precision block padded to the vector width without changing
 *     results);
 *   - Sec. 3, "Enabling Low-Cost Fixed-Point Operations": group max-abs scale
 *     (item 1), unsigned activation codes (item 2), signed two's-complement
 *     weight codes (item 3, Eq. 1);
 *   - Alg. 1 Phase II: the forward pass as integer MAC execution.
 *
 * Conventions for every call:
 *   - "device" pointers are HIP device allocations on the current device;
 *     "host" pointers are ordinary host memory.  All matrices are row-major
 *     with the given leading dimension in elements.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued on it asynchronously unless stated otherwise.
 *   - Arguments are validated synchronously before anything is enqueued; on
 *     a non-OK status nothing was enqueued and outputs are untouched.  The
 *     message of the last failure on this thread is soniq_last_error().
 *   - No call throws; HIP errors are returned as SONIQ_ERR_HIP, and faults of
 *     earlier asynchronous work may be reported by a later call.
 */
#ifndef SONIQ_H_
#define SONIQ_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SONIQ_OK = 0,
  SONIQ_ERR_INVALID_ARGUMENT = 1, /* bad pointer, size, width or handle */
  SONIQ_ERR_UNSUPPORTED = 2,      /* valid but outside this build's limits */
  SONIQ_ERR_OUT_OF_MEMORY = 3,    /* a device or host allocation failed */
  SONIQ_ERR_HIP = 4               /* a HIP runtime call failed */
} soniq_status;

/* Opaque handles.  A weights handle owns the packed weights, their scales
 * and the channel plans; it is immutable after packing and may be shared by
 * streams and threads.  An activation handle owns one packed activation
 * buffer and its group scales; use it from one stream at a time. */
typedef struct soniq_weights_s* soniq_weights;
typedef struct soniq_act_s* soniq_act;

/* Weight code grid (Sec. 3 codec, item 3).
 *   SONIQ_WQ_SYMMETRIC: codes in [-(2^(b-1)-1), 2^(b-1)-1], step
 *       max-abs/(2^(b-1)-1); 1-bit channels are sign x max-abs (codes +-1,
 *       the XNOR/popcount semantics of Sec. 4.2).
 *   SONIQ_WQ_TWOS_FRACTION: the two's-complement fraction grid of Eq. (1):
 *       codes in [-2^(b-1), 2^(b-1)-1], step max-abs/2^(b-1). */
enum { SONIQ_WQ_SYMMETRIC = 0, SONIQ_WQ_TWOS_FRACTION = 1 };

/* Packing flag, OR-ed into wq_mode: store 1-bit (sign, +-1) weight channels
 * in 4-bit containers instead of single bits.  Same codes and results;
 * four times those channels' bytes, but on gfx950 a nibble widens to the
 * int8 MFMA operand in a shift and a mask where a bit takes a dozen
 * instructions, so batches on the MFMA GEMM (more than 8 rows) run faster.
 * The batch-1 GEMV, which is bound by weight bytes, is better served by
 * the default bits. */
#define SONIQ_WPACK_SIGN_NIBBLES 0x100

/* Packing flag, OR-ed into wq_mode: also keep the narrow operands in the
 * fp4 / fp6 operand formats of gfx950's v_mfma_scale_f32_16x16x128_f8f6f4,
 * so tiles of narrow weights against narrow activations run on that
 * instruction (128 channels per step, no widening to bytes) instead of the
 * int8 MFMA.  1- and 2-bit containers map to fp4 (e2m1), 4-bit containers
 * to fp6 (e3m2): every stored code is exactly representable, and with
 * power-of-two block scales the fp32 sums equal the integer sums exactly
 * (each partial sum is an integer multiple of the scale below 2^24 of it),
 * so results are bit-identical to the integer path.  The low-precision MAC
 * of the paper's hardware study (App. C; Sec. 7 findings on two-level
 * palettes) is served by gfx950's narrow-float matrix instruction here.
 * Costs a second copy of the narrow weights (fp4 or fp6 per element) and,
 * per activation handle, of the narrow activation groups, refreshed before
 * each MFMA GEMM.  Not combined with sub-group activation scales
 * (UNSUPPORTED). */
#define SONIQ_WPACK_F8F6F4 0x200

/* Packing flag, OR-ed into wq_mode: also keep a dense copy of the weights,
 * every code in exactly its channel's width (3, 5, 6 and 7 bits no longer
 * take the next power-of-two container; 1, 2, 4 and 8 as before), which
 * the GEMV forms (batches of at most 8 rows with M * (1.25 * padded K +
 * 16) + 32 <= 64 KiB, i.e. M * padded K up to about 52 K; larger batches
 * read the units) read instead of the units: fewer bytes for the
 * weight-bound decode path.  Sign (1-bit) weights against a sign
 * activation group take XNOR-popcount products there (Sec. 4.2, Hardware
 * Support).  The channels of each 16-row block share one width (two widths
 * in one container are not merged into shared blocks).  Same codes and
 * results.
 * Costs the dense copy's bytes beside the units.  Not combined with
 * sub-group activation scales or the f8f6f4 copies (UNSUPPORTED). */
#define SONIQ_WPACK_DENSE 0x400

/* Largest supported input-channel count (padded): keeps every int32
 * accumulator exact. */
#define SONIQ_MAX_K 65536

/*
 * soniq_pack_weights -- quantize, re-order and bit-pack one layer's weights.
 * Passages: codec items 1 and 3 (scale and codes per output channel), Alg. 1
 * channel permutation and Fig. "normalization" (grouping and padding),
 * Sec. 2.4 C5 (packed layout).
 *
 *   W_dev      device, float32 [N, ldw]; row n holds output channel n over
 *              the K input channels (the nn.Linear / im2col weight layout).
 *   N, K       output and input channel counts, N >= 1, 1 <= K and the
 *              padded K <= SONIQ_MAX_K.
 *   ldw        row stride of W in elements, ldw >= K.
 *   w_bits     host, uint8 [N]: width of each output channel, 1..8, at most
 *              two distinct values.  Copied during the call.
 *   a_bits     host, uint8 [K]: width of each input (activation) channel,
 *              1..8, at most two distinct values.  Fixes the activation
 *              precision groups used by every activation handle created
 *              from these weights.  Copied during the call.
 *   a_signed   1: activations use the signed symmetric grid; 0: the unsigned
 *              codec of codec item 2 (e.g. post-ReLU inputs).
 *   stream     W is read on this stream.  The call returns after the packed
 *              weights are complete (it synchronizes this stream).
 *   out        receives the new handle; release with soniq_weights_destroy.
 *
 * Widths 3, 5, 6 and 7 are stored in the next power-of-two container.
 * Errors: INVALID_ARGUMENT (null pointer, N/K < 1, ldw < K, width outside
 * 1..8, more than two widths), UNSUPPORTED (padded K > SONIQ_MAX_K),
 * OUT_OF_MEMORY, HIP.
 */
soniq_status soniq_pack_weights(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                                const uint8_t* w_bits, const uint8_t* a_bits,
                                int a_signed, void* stream, soniq_weights* out);

/* As soniq_pack_weights, with the weight grid chosen by wq_mode
 * (SONIQ_WQ_SYMMETRIC or SONIQ_WQ_TWOS_FRACTION), optionally OR-ed with
 * SONIQ_WPACK_SIGN_NIBBLES. */
soniq_status soniq_pack_weights_ex(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                                   const uint8_t* w_bits, const uint8_t* a_bits,
                                   int a_signed, int wq_mode, void* stream,
                                   soniq_weights* out);

/*
 * soniq_pack_weights_grouped -- as soniq_pack_weights_ex, with sub-group
 * activation scales: GroupSize_act of the design-space parameters (Sec. 3;
 * Sec. 5 normalizes transformer activations in 512-bit groups).
 *
 *   act_group_bits  0: one activation scale per precision group (the
 *       other pack calls).  Otherwise a positive multiple of 512: each
 *       precision group, in the planned order (narrow width first, original
 *       channel order inside a width), is cut into consecutive blocks of
 *       act_group_bits / c channels, c the group's container (the next
 *       power of two >= its width), so a block fills act_group_bits of
 *       storage: 128 channels at 4 bits, 64 at 8 bits for 512.  Each block
 *       has its own scale, max-abs over the batch and the block's channels
 *       divided by the group's largest code; the GEMM keeps one exact int32
 *       sum per block and scales it once:
 *         Y = bf16(s_w * sum_j s_a[j] * ACC[j]),
 *       summed in fp32 in block order (multiply, then add).  Blocks are
 *       numbered group 0 first; soniq_weights_info reports their count.
 * Grouped handles need a zero point of 0 in both activation groups (signed
 * activations, or unsigned widths below their container: 3, 5, 6, 7 bits)
 * and no 1-bit activation group, and at most 256 blocks; UNSUPPORTED
 * otherwise.  Their activations are quantized from the lowered matrix only
 * (soniq_quantize_act_conv3x3 returns UNSUPPORTED) and every batch size
 * runs the MFMA GEMM.
 * Errors: those of soniq_pack_weights_ex; INVALID_ARGUMENT for an
 * act_group_bits that is negative or not a multiple of 512.
 */
soniq_status soniq_pack_weights_grouped(const float* W_dev, int64_t N, int64_t K, int64_t ldw,
                                        const uint8_t* w_bits, const uint8_t* a_bits,
                                        int a_signed, int wq_mode, int act_group_bits,
                                        void* stream, soniq_weights* out);

/*
 * soniq_pack_weights_conv3x3 -- weights of a stride-1, pad-1 3x3
 * convolution packed for the implicit GEMM (no lowered activation matrix
 * exists anywhere).  Passages: as soniq_pack_weights; Sec. 4 (software
 * optimizations for convolutions: a layout that lets the kernel read each
 * input once, and input handling fused with quantization); per-channel
 * precision (Sec. 3).
 *
 *   W_dev   device, float32 [N][C][3][3] contiguous (the filter; as a
 *           matrix it is [N][9C] in the column order of a 3x3 unfold,
 *           k = c*9 + kh*3 + kw).
 *   N, C    output and input channels (9*C padded <= SONIQ_MAX_K).
 *   w_bits  host uint8 [N] as for soniq_pack_weights.
 *   c_bits  host uint8 [C]: width of each INPUT channel (shared by its nine
 *           taps), 1..8, at most two values.
 *   a_signed, wq_mode  as for soniq_pack_weights_ex (SONIQ_WPACK_SIGN_NIBBLES
 *           allowed; SONIQ_WPACK_F8F6F4 not).
 * Inside each precision group the K axis is tap-major (all channels of tap
 * 0, then tap 1, ...), each tap's run padded to 16 channels, so that a
 * GEMM fragment of one tap is one run of a pixel's codes.  Results are
 * those of soniq_pack_weights on the lowered weights: the same codes and
 * scales (soniq_weights_unpack_debug returns them in the k = c*9 + t order)
 * and, through soniq_mp_gemm, the same accumulators and outputs.
 * The implicit convolution takes two activation widths in 4- and 8-bit
 * containers (one of at most 4 bits, one of 5 to 8) or one width of 3 to
 * 8 bits, and any pair of weight containers; UNSUPPORTED otherwise (the
 * next-layer epilogues of soniq_mp_gemm_quantize_next(_max) from a
 * convolution take the two-width plans only).  Activation handles:
 * soniq_act_create_conv3x3.
 * Errors: those of soniq_pack_weights, UNSUPPORTED.
 */
soniq_status soniq_pack_weights_conv3x3(const float* W_dev, int64_t N, int64_t C,
                                        const uint8_t* w_bits, const uint8_t* c_bits,
                                        int a_signed, int wq_mode, void* stream,
                                        soniq_weights* out);

/*
 * soniq_act_create_conv3x3 -- the activation handle of weights from
 * soniq_pack_weights_conv3x3, for inputs of up to B images of H x W.  It
 * owns the input's code image: per precision group, (H+2) x (W+2) pixels
 * per image (a one-pixel halo holding the code of 0.0), each pixel its
 * channels of that group as packed codes, about 9x fewer bytes than a
 * lowered matrix.  Quantize with soniq_quantize_act_conv3x3 (the same
 * H and W, at most B images), multiply with soniq_mp_gemm; the other
 * activation entry points return UNSUPPORTED for it.
 * Errors: INVALID_ARGUMENT (other weights, sizes), OUT_OF_MEMORY, HIP.
 */
soniq_status soniq_act_create_conv3x3(soniq_weights w, int64_t B, int64_t H, int64_t W,
                                      soniq_act* out);

/*
 * soniq_act_create -- allocate a packed activation buffer for up to max_M
 * rows, laid out for the input-channel plan of `w` (activation groups,
 * permutation and padding are fixed at weight-packing time, Alg. 1).
 * Errors: INVALID_ARGUMENT (null, max_M < 1), OUT_OF_MEMORY, HIP.
 */
soniq_status soniq_act_create(soniq_weights w, int64_t max_M, soniq_act* out);

/*
 * soniq_quantize_act -- quantize, re-order and pack M activation rows.
 * Passages: codec items 1 and 2 (group max-abs scale; unsigned codes) or the
 * symmetric signed grid; Sec. 2.4 C2 (one scale per precision group, shared
 * by all rows of the call; one per block of a group for weights packed with
 * soniq_pack_weights_grouped); Alg. 1 channel permutation.
 *
 *   A_dev   device, float32 [M, lda]; row m is one input vector over K
 *           channels in the original channel order.  Finite values only.
 *   M       1 <= M <= max_M of the handle.
 *   lda     row stride in elements, lda >= K.
 * Enqueued on `stream`; the packed codes and the group scales s_a stay in
 * the handle for the next soniq_mp_gemm on the same stream.
 * Errors: INVALID_ARGUMENT, HIP.
 */
soniq_status soniq_quantize_act(soniq_act act, const float* A_dev, int64_t M, int64_t lda,
                                void* stream);

/*
 * soniq_quantize_act_conv3x3 -- the activations of a stride-1, pad-1 3x3
 * convolution, quantized straight from its input tensor with no lowered
 * fp32 matrix.  Passages: as soniq_quantize_act; the fusion of convolution
 * input handling with quantization to cut memory traffic (Sec. 4, software
 * optimizations, CPU SIMD item 2).
 *
 * The result (packed codes and s_a) is exactly that of soniq_quantize_act
 * on the lowered matrix A[M = B*H*W, K = 9*C]: row m = (b*H + y)*W + x,
 * column k = c*9 + kh*3 + kw holding X[b][c][y+kh-1][x+kw-1], or 0 where
 * that lies outside the image (the order of a 3x3 unfold; the weights are
 * the [N][C][3][3] filter viewed as [N][9C]).
 *
 *   X_dev   device, float32 [B][C][H][W], contiguous.  Finite values only.
 *   B, C, H, W  >= 1; 9*C must equal the K of the handle's weights and
 *           B*H*W must not exceed max_M; B*C*H*W < 2^31.
 * The nine columns of every channel must share one activation width
 * (UNSUPPORTED otherwise), and 16 rows of the handle's padded channel plan
 * must fit 64 KB of LDS (K up to about 4000; UNSUPPORTED otherwise).
 * For a handle of soniq_act_create_conv3x3 (weights packed for the implicit
 * GEMM) the call instead writes the handle's code image of X (H and W as
 * created, B at most as created); codes and scales are the same as above,
 * and soniq_act_unpack_debug returns them as the lowered matrix's.
 * Enqueued on `stream`, like soniq_quantize_act; X_dev is only read.
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
soniq_status soniq_quantize_act_conv3x3(soniq_act act, const float* X_dev, int64_t B, int64_t C,
                                        int64_t H, int64_t W, void* stream);

/*
 * soniq_mp_gemm -- Y = bf16(s_w * sum_g s_a[g] * ACC[g]) for the M rows last
 * quantized into `act` (Alg. 1 Phase II integer MAC forward; C2: the scales
 * are applied once per output, after the exact integer sums).
 *
 *   act      a handle created from `w`, after soniq_quantize_act.
 *   Y_dev    device, bf16 bit patterns (uint16) [M, ldy], columns in the
 *            original output-channel order; fully overwritten.
 *   ldy      row stride in elements, ldy >= N.
 *   acc_dev  optional device int32 [S][M][N] (S = act_scales of
 *            soniq_weights_info: activation groups, or blocks for grouped
 *            weights): receives the exact accumulators ACC[g][m][n] in
 *            original order.  NULL skips the dump.
 * Enqueued on `stream`.  M <= 8 uses a bandwidth-bound kernel without matrix
 * cores; larger M uses int8 MFMA tiles.
 * Errors: INVALID_ARGUMENT (null, mismatched handles, nothing quantized),
 * HIP.
 */
soniq_status soniq_mp_gemm(soniq_act act, soniq_weights w, uint16_t* Y_dev, int64_t ldy,
                           int32_t* acc_dev, void* stream);

/*
 * soniq_quantize_mp_gemm -- soniq_quantize_act followed by soniq_mp_gemm
 * in one call, with the same results (Y, the optional accumulators, and
 * the packed rows and scales left in the handle).  Passages: those of the
 * two calls.  A batch of one row (the decode case) is quantized inside
 * the GEMV launch, with no launch of its own, when its plan allows it
 * (4-bit and 8-bit activation containers, no 1-bit sign group, K a
 * multiple of 4 up to 4096, A_dev 16-byte aligned); other batches run the
 * two calls.
 *
 *   act, w  a handle made for w, and w.
 *   A_dev   device, float32 [M, lda], as for soniq_quantize_act.
 *   Y_dev, ldy, acc_dev  as for soniq_mp_gemm.
 * Enqueued on `stream`.  Errors: INVALID_ARGUMENT, HIP.
 */
soniq_status soniq_quantize_mp_gemm(soniq_act act, soniq_weights w, const float* A_dev, int64_t M,
                                    int64_t lda, uint16_t* Y_dev, int64_t ldy, int32_t* acc_dev,
                                    void* stream);

/*
 * soniq_quantize_mp_gemm_scratch -- soniq_quantize_mp_gemm without an
 * activation handle and without allocating: for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  The packed activations, their
 * scales, the partial maxima and the single pass's grid state live in a
 * per-device scratch array of the library (64 MiB, held by every device the
 * library runs on until the process ends) instead of a handle's buffers.
 * Same results as soniq_quantize_act + soniq_mp_gemm on a handle made for w
 * (Y and the optional accumulators; the codes are not kept for a later
 * call).  No hipMalloc, hipFree or other allocation happens in the call;
 * the first call on a device looks up the scratch address and clears its
 * grid state with a small kernel on `stream`.
 *
 *   w        packed weights (any packing).
 *   A_dev    device, float32 [M, lda], as for soniq_quantize_act.
 *   M        >= 1; the packed rows (M rounded up to 256) with the handle's
 *            other buffers must fit the scratch: about M * K bytes at 8-bit
 *            activations, e.g. M = 8192 at K = 8192 fits.
 *   Y_dev, ldy, acc_dev  as for soniq_mp_gemm.
 * Every call on a device shares that device's scratch: calls that overlap
 * in time on one device (other streams, other threads) race and give wrong
 * results; serialize them.  Enqueued on `stream`.
 * Errors: INVALID_ARGUMENT (null, sizes), UNSUPPORTED (M too large for the
 * scratch), HIP.
 */
soniq_status soniq_quantize_mp_gemm_scratch(soniq_weights w, const float* A_dev, int64_t M,
                                            int64_t lda, uint16_t* Y_dev, int64_t ldy,
                                            int32_t* acc_dev, void* stream);

/* Description of a packed weights handle. */
typedef struct {
  int64_t N, K;               /* logical sizes */
  int32_t S;                  /* activation precision groups (1 or 2) */
  int32_t a_signed, wq_mode;
  uint8_t a_bits[2];          /* width of each activation group, ascending */
  uint8_t w_bits[2];          /* weight widths, ascending (w_bits[1]=0 if one) */
  int64_t a_count[2];         /* input channels per activation group */
  int64_t a_count_padded[2];  /* after padding each group to 64 channels */
  int64_t w_count[2];         /* output channels per weight width */
  int64_t packed_w_bytes;     /* bytes of the packed weight buffer */
  int64_t packed_w_bytes_algorithmic; /* sum over rows of container*K/8 */
  int32_t act_group_bits;     /* GroupSize_act in bits, 0 = one scale per group */
  int32_t act_scales;         /* activation scales: blocks, or S when ungrouped */
  int32_t f8f6f4;             /* 1: packed with SONIQ_WPACK_F8F6F4 */
  int64_t dense_w_bytes;      /* bytes of the dense copy (SONIQ_WPACK_DENSE), else 0 */
} soniq_weights_info_t;

/* Fill *out.  Errors: INVALID_ARGUMENT. */
soniq_status soniq_weights_info(soniq_weights w, soniq_weights_info_t* out);

/*
 * soniq_mp_gemm_quantize_next -- soniq_mp_gemm whose epilogue also
 * quantizes its outputs as the next layer's activations, so that layer
 * needs no soniq_quantize_act call and no fp32 (or bf16) copy of them is
 * read back.  Passages: Sec. 4 fuses quantization into the operation that
 * produces the activations (for CNNs, into the convolution), to cut memory
 * traffic; codec items 1-2 with static (calibrated) group scales in place
 * of the batch maximum.
 *
 *   act, w   as for soniq_mp_gemm (act quantized, made for w); w may be an
 *            implicit convolution's (soniq_pack_weights_conv3x3, act from
 *            soniq_act_create_conv3x3), whose GEMM then carries the epilogue.
 *   next     an activation handle of the next layer's weights, whose K
 *            equals this layer's N; act's M must not exceed its max_M.  Or
 *            a handle of soniq_act_create_conv3x3 (the next layer an
 *            implicit 3x3 convolution): its input channels C equal this
 *            layer's N, and this layer's M rows are the output pixels of
 *            M / (H*W) <= B whole images in (image, y, x) order, as a
 *            convolution's GEMM produces them (INVALID_ARGUMENT
 *            otherwise).  The codes then go straight into next's haloed
 *            code image (the halo holding the code of 0.0), as
 *            soniq_quantize_act_conv3x3 would leave it for that input.
 *   s_next   host float [act_scales of the next layer's weights]: the
 *            static scale of each next-layer activation group (narrow width
 *            first), or of each block when the next layer's weights were
 *            packed with sub-group scales (blocks in their order), finite
 *            and >= 0.  Copied during the call.
 *   Y_dev    as for soniq_mp_gemm, or NULL to skip storing Y.
 *   ldy, acc_dev  as for soniq_mp_gemm.
 * Each output's code is taken from the fp32 value the epilogue rounds to
 * bf16 (before that rounding): code = clamp(rint(y / s_next[g]), lo, hi)
 * of its next-layer group g, exactly as soniq_quantize_act would with that
 * scale.  On return (stream order) `next` holds M packed rows and its
 * scales are s_next, ready for soniq_mp_gemm(next, next's weights).
 * Batches of more than 8 rows run the MFMA tiles, smaller ones the GEMV
 * forms of soniq_mp_gemm (activation containers 4 and 8) with the same
 * quantizing epilogue; weights packed with sub-group scales produce through
 * their per-block kernels (acc_dev then holds their per-block sums, as for
 * soniq_mp_gemm).  The first call with a given
 * (weights, next) pair allocates next's code image (max_M rounded up to
 * 256, plus 8, rows of its padded K, or of its two groups' padded channel
 * counts for a convolution, bytes) and a column table, synchronously; later calls with the
 * same pair allocate nothing, so make that first call before capturing the
 * call in a HIP graph.  `next` keeps one table per producer weights handle
 * until it is destroyed: a graph captured with one producer stays valid
 * after other producers have fed the same `next`.
 * `next` must not be `act` (its scales would be overwritten before the
 * GEMM reads them).
 * Errors: INVALID_ARGUMENT (null, next == act, mismatched handles or
 * sizes, bad scales, a batch that is not whole images of a convolution
 * next), UNSUPPORTED (more tiles than one launch takes; an implicit
 * convolution whose widths have no kernel, or feeding weights packed with
 * sub-group scales), OUT_OF_MEMORY, HIP.
 */
soniq_status soniq_mp_gemm_quantize_next(soniq_act act, soniq_weights w, soniq_act next,
                                         const float* s_next, uint16_t* Y_dev, int64_t ldy,
                                         int32_t* acc_dev, void* stream);

/*
 * soniq_mp_gemm_quantize_next_max -- the two-pass form of quantization
 * fused into the producer: soniq_mp_gemm(act, w) storing Y (required),
 * whose epilogue also folds each next-layer activation group's largest |Y|
 * (of the values as stored, bf16) per output tile; one pass over Y then
 * quantizes it into `next` with the batch maxima of those.  Passages:
 * Sec. 4 (quantization fused into the producing operation); codec items
 * 1-2 (the group max-abs scale over the batch).
 *
 *   act, w, Y_dev, ldy, acc_dev  as for soniq_mp_gemm (Y_dev not NULL);
 *            w may be an implicit convolution's weights (act then its
 *            convolution handle).
 *   next     an activation handle of the next layer's weights, whose K
 *            equals this layer's N (act's M must not exceed its max_M), or
 *            of a next implicit convolution with C = N (act's M output
 *            pixels a batch of at most B of its H x W images).
 * On return (stream order) `next` holds exactly what
 * soniq_quantize_act(next, float(Y)) would leave (codes and scales; for a
 * next convolution what soniq_quantize_act_conv3x3 would leave from Y as
 * its NHWC input): no calibration, the fp32 copy of Y and the separate
 * maximum pass are what it saves.  Batches of more than 8 rows (and every
 * convolution producer) fold the maxima in the GEMM tiles; smaller ones
 * run the GEMV forms and reduce them in the quantizer.
 * The first call with a given (weights, next) pair allocates as
 * soniq_mp_gemm_quantize_next does (the same table), synchronously; make it
 * before capturing the call in a HIP graph.  The tiles' maxima sit beside
 * the pair's table, so calls with the same pair must not overlap.
 * Errors: INVALID_ARGUMENT (null, next == act, mismatched handles or
 * sizes), UNSUPPORTED (weights packed with sub-group scales on either
 * side, an implicit convolution whose widths have no kernel, more tiles
 * than one launch takes), OUT_OF_MEMORY, HIP.
 */
soniq_status soniq_mp_gemm_quantize_next_max(soniq_act act, soniq_weights w, soniq_act next,
                                             uint16_t* Y_dev, int64_t ldy, int32_t* acc_dev,
                                             void* stream);

/*
 * soniq_plan_input_channels -- the input-channel plan for a_bits, computed
 * on the host (no device needed): pos[k] receives the position of input
 * channel k in the packed, group-ordered and padded channel axis (group 0,
 * the narrower width, first; original order within a group; each group
 * padded to a multiple of 64).  seg_len[2] and seg_pad[2] receive the group
 * sizes before and after padding (second entries 0 when S = 1).
 * Returns INVALID_ARGUMENT for bad widths or pointers.
 */
soniq_status soniq_plan_input_channels(const uint8_t* a_bits, int64_t K, int64_t* pos,
                                       int64_t seg_len[2], int64_t seg_pad[2], int32_t* S);

/*
 * Debug readback (synchronous: waits for the device).  Codes are returned as
 * int32 in the original channel order; scales as float32.
 *   soniq_weights_unpack_debug: codes [N, K], s_w [N].
 *   soniq_act_unpack_debug:     codes [M, K] of the last soniq_quantize_act,
 *                               s_a [act_scales of soniq_weights_info].
 * Either output pointer may be NULL.  Errors: INVALID_ARGUMENT, HIP.
 */
soniq_status soniq_weights_unpack_debug(soniq_weights w, int32_t* codes, float* s_w);
soniq_status soniq_act_unpack_debug(soniq_act act, int32_t* codes, float* s_a);

/*
 * soniq_act_wait_timeouts -- how many workgroups of the single-pass
 * quantizer gave up waiting for the rest of their grid since `act` was
 * made (synchronous: waits for the device).  The single pass (codec item 1:
 * one max-abs per group over the whole batch, taken in the same pass that
 * quantizes) sizes its grid so that every workgroup is resident; a
 * workgroup whose wait times out anyway (e.g. other work held the compute
 * units) takes the maxima from the whole batch itself, so results are
 * unchanged but the call was slow.  A nonzero count says that happened.
 * Errors: INVALID_ARGUMENT, HIP.
 */
soniq_status soniq_act_wait_timeouts(soniq_act act, uint64_t* count);

/*
 * soniq_debug_stream_read -- a measurement aid, not part of the method:
 * reads `bytes` bytes at src_dev (device, 16-byte aligned; bytes a positive
 * multiple of 16, below 2^31) once, in 16-byte loads, two per thread and
 * 8 KB per workgroup, and writes the XOR of each workgroup's words to
 * sink_dev[workgroup] (ceil(bytes / 8192) words, device).  Its duration on
 * the packed weights of a batch-1 GEMV is the plain-read time of those
 * bytes on this device, the ceiling the GEMV is measured against.
 * Asynchronous on `stream` (NULL = default stream).
 * Errors: INVALID_ARGUMENT, HIP.
 */
soniq_status soniq_debug_stream_read(const void* src_dev, int64_t bytes, uint32_t* sink_dev,
                                     void* stream);

/* Release a handle (NULL is ignored).  Waits for the device first. */
void soniq_weights_destroy(soniq_weights w);
void soniq_act_destroy(soniq_act act);

/* Message of the last non-OK status returned on the calling thread. */
const char* soniq_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SONIQ_H_ */
