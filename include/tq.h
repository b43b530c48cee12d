/*
 * tq.h -- C ABI of the TwinQuant dual-component W4A4 linear layer for
 * AMD Instinct MI355X (gfx950).
 *
 * The layer (paper "TwinQuant: Learnable Subspace Decomposition for 4-Bit
 * LLM Quantization", Sec. 4.1 Eq. 4/6 and Sec. 4.3) is
 *
 *     Y = Q(X) [ Q(L1) Q(L2) + Q(W_res)^T ]
 *
 * X [m,k] activations, W_res [n,k] the 4-bit residual component R' (stored
 * like a PyTorch Linear weight, Y = X W_res^T), L1 = U' [k,r] and
 * L2 = V' [r,n] the low-rank factors.  Q is the symmetric 4-bit group
 * quantizer of Sec. 2 Eq. (1): codes q in [-7, 7], one fp16 scale
 * s = fp16(max|v| / 7) per group of `group` consecutive values along the
 * reduction axis (Sec. 5.1 uses groups of contiguous elements; 64 or 128
 * here, 128 being the paper's default).  The low-rank
 * branch is two integer products: H = Q(X) Q(L1) is formed on chip,
 * re-quantized per token and group of min(group, r) rank columns with an fp32
 * scale s_H, and multiplied by Q(L2); both branches are merged in one
 * epilogue with a single rounding to fp16 or bf16 (Sec. 4.3, "fused two-stage
 * low-rank pipeline" and "on-the-fly scaling with a single epilogue").
 *
 * Conventions for every entry point:
 *  - All array pointers are DEVICE pointers owned by the caller; the library
 *    never allocates, frees or synchronizes.  Its only global state is the
 *    static scratch array of tq_dual_gemm_unfused_noalloc.  Device pointers
 *    must be 16-byte aligned (TQ_ERR_ALIGN otherwise).
 *  - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *    asynchronously on it; results are visible after the stream completes.
 *  - Arguments are validated on the host before anything is launched; on any
 *    error nothing is written and the call returns the error code.  A failed
 *    launch returns TQ_ERR_HIP.  No C++ exception crosses the ABI.
 *  - Inputs must be finite; for NaN/Inf inputs results are unspecified (but
 *    every access stays in bounds).
 *  - fp16 / bf16 values are passed as their 16-bit IEEE bit patterns.
 *
 * TQ4 code word (the packed 4-bit format of activations and of exported
 * weights).  A little-endian 32-bit word holds 8 consecutive codes c0..c7
 * (consecutive along the reduction axis) in sign-magnitude form:
 *     c_i     (i < 4): |c_i| in bits 8i..8i+2,  sign in bit 8i+7
 *     c_(4+i) (i < 4): |c_(4+i)| in bits 8i+4..8i+6,
 *                      sign in bit 8*((i+1) mod 4) + 3
 * A sign bit is 1 for negative codes only (zero is never "-0").  The layout
 * lets the kernels turn 8 codes into two words of fp8 e4m3 matrix-core
 * operands with three bit operations (mask, rotate, mask).
 */
#ifndef TQ_H
#define TQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TQ_OK = 0,
    TQ_ERR_NULL = 1,    /* a required pointer is NULL                        */
    TQ_ERR_SHAPE = 2,   /* a size is out of range                            */
    TQ_ERR_GROUP = 3,   /* group size unsupported or k not a multiple of it  */
    TQ_ERR_RANK = 4,    /* rank unsupported                                  */
    TQ_ERR_DTYPE = 5,   /* unknown output dtype                              */
    TQ_ERR_ALIGN = 6,   /* a device pointer is not 16-byte aligned           */
    TQ_ERR_BUFFER = 7,  /* descriptor inconsistent / not initialised         */
    TQ_ERR_HIP = 8,     /* the HIP runtime reported an error on launch       */
    TQ_ERR_TOO_LARGE = 9 /* needs more scratch than the static buffer holds  */
} tq_status;

typedef enum { TQ_F16 = 0, TQ_BF16 = 1 } tq_dtype;

/* Geometry of one layer's packed weights.  Filled by tq_weight_desc_init;
 * treat every field as read-only. */
typedef struct {
    int32_t n, k, rank, group;   /* layer sizes; group = quantization group    */
    int32_t group_r;             /* group along the rank axis = min(group, r)  */
    int32_t n_pad;               /* n rounded up to 32                         */
    int32_t r_pad32, r_pad64;    /* r rounded up to 32 and to 64               */
    int32_t magic;               /* set by tq_weight_desc_init                 */
    int32_t reserved;
    uint64_t packed_bytes;       /* size of the packed weight buffer           */
    uint64_t off_w, off_ws, off_l1, off_l1s, off_l2, off_l2s;  /* section offsets */
} tq_weight_desc;

/* Validate a layer shape and fill `out` (host only, touches no GPU).
 *   n >= 1 output features, k input features with k % group == 0,
 *   group 64 or 128, rank r in {0, 8, 16, 32, 64, 128}.  r == 0 is the plain
 *   4-bit linear layer of Sec. 2 Eq. (2).  The packed buffer must stay below
 *   4 GiB (TQ_ERR_SHAPE otherwise).
 * Errors: TQ_ERR_NULL, TQ_ERR_SHAPE, TQ_ERR_GROUP, TQ_ERR_RANK. */
tq_status tq_weight_desc_init(int n, int k, int rank, int group, tq_weight_desc *out);

/* Quantize and pack one layer's weights (the offline fold of Sec. 4.1:
 * U', V', R' are quantized once and stored in 4 bits).
 *   w_res  [n,k] fp16 row-major   (quantized per row, groups along k)
 *   l1     [k,r] fp16 row-major   (quantized per column, groups along k)
 *   l2     [r,n] fp16 row-major   (quantized per column, groups of group_r
 *                                  along r); l1 and l2 may be NULL iff r == 0
 *   packed  device buffer of d->packed_bytes bytes, written completely; its
 *           layout is private to the library (see tq_export_weights).
 * Errors: TQ_ERR_NULL, TQ_ERR_BUFFER, TQ_ERR_ALIGN, TQ_ERR_HIP. */
tq_status tq_pack_weights(const tq_weight_desc *d, const void *w_res, const void *l1,
                          const void *l2, void *packed, void *stream);

/* Per-token, per-group activation quantizer (Sec. 2 Eq. 1; Sec. 4.3: the
 * activation is quantized once and shared by both branches).
 *   x         [m,k] fp16 row-major, 0 <= m <= 2097120 (65535 tiles of 32),
 *             k % group == 0, group 64 or 128 (the layer's group)
 *   x_codes   tq_act_codes_bytes(m, k) bytes, tile-major.  The tokens are
 *             cut into tiles of 32 (m32 = m rounded up to a multiple of 32)
 *             and K into blocks of 64 (called groups below; a 128-wide
 *             quantization group spans two blocks and has one scale).  The
 *             layout does not depend on the group.  For m <= 512 each code is a TQ4
 *             nibble (m32 * k / 2 bytes): tile t, group g is one 1 KiB block
 *             at byte (t * (k / 64) + g) * 1024, whose 16-byte lane slot
 *             32 h + i (h = 0, 1; i = 0 .. 31) holds the four TQ4 words of
 *             codes 32 h .. 32 h + 31 of the group for token 32 t + i (the
 *             order in which the matrix cores take one operand of a
 *             32 x 32 x 64 product, so each block is one coalesced load).
 *             For m > 512 each code is its fp8 e4m3 operand byte,
 *             sign << 7 | |q| (m32 * k bytes): tile t, group g is a 2 KiB
 *             block at byte (t * (k / 64) + g) * 2048 made of two 1 KiB
 *             halves p = 0, 1; lane slot 32 h + i of half p holds the bytes
 *             of codes 32 h + 16 p .. 32 h + 16 p + 15 of the group for token
 *             32 t + i.  Tokens [m, m32) get zero codes.
 *   x_scales  [k/group, m32] fp16: the scale of token i, group g is
 *             x_scales[g*m32 + i] (group-major, so one group's scales of a
 *             token tile are contiguous); entries i in [m, m32) are 0
 * m == 0 is a no-op.  Errors: TQ_ERR_NULL, TQ_ERR_SHAPE, TQ_ERR_GROUP,
 * TQ_ERR_ALIGN, TQ_ERR_HIP. */
tq_status tq_quant_act(const void *x, int m, int k, int group, void *x_codes,
                       void *x_scales, void *stream);

/* Size in bytes of the x_codes buffer of m tokens with reduction size k
 * (0 if m or k is out of range or k % 64 != 0).  Host-only. */
size_t tq_act_codes_bytes(int m, int k);

/* The fused dual-component layer: residual 4-bit GEMM, low-rank stage 1
 * (H = Q(X) Q(L1)), on-the-fly re-quantization of H, stage 2 (Q_H Q(L2)),
 * and one epilogue that sums both branches and stores Y once (Sec. 4.3).
 *   packed            buffer written by tq_pack_weights for descriptor d
 *   x_codes/x_scales  written by tq_quant_act for the same k (m tokens)
 *   y                 [m,n] output, fp16 or bf16 per y_dtype, row-major
 * One kernel launch; H, s_H and Q_H never leave the chip (registers and LDS
 * of each work-group).  No workspace and no state: calls may run
 * concurrently on any streams.  m == 0 is a no-op.  Errors: TQ_ERR_NULL,
 * TQ_ERR_SHAPE, TQ_ERR_BUFFER, TQ_ERR_DTYPE, TQ_ERR_ALIGN, TQ_ERR_HIP. */
tq_status tq_dual_gemm(const tq_weight_desc *d, const void *packed, const void *x_codes,
                       const void *x_scales, int m, void *y, tq_dtype y_dtype, void *stream);

/* The fused layer with the activation quantizer inside the same launch
 * (Sec. 4.3: the kernel quantizes the activation tile once and feeds the
 * codes to both branches): x is the fp16 activation [m,k], row-major.  Each
 * work-group quantizes X into its own LDS with the arithmetic of
 * tq_quant_act (bit-identical codes and scales), so nothing but Y is
 * written.  For decode-sized calls: 1 <= m <= 16 and the codes of m tokens
 * must fit the kernel's LDS (m = 1: k <= 114688; m = 2: k <= 57344;
 * m <= 8: k <= 28672; m <= 16: k <= 14336); TQ_ERR_SHAPE otherwise.
 * Errors as tq_dual_gemm. */
tq_status tq_dual_gemm_fused_quant(const tq_weight_desc *d, const void *packed, const void *x,
                                   int m, void *y, tq_dtype y_dtype, void *stream);

/* Kernels of tq_dual_gemm. */
typedef enum {
  TQ_KERNEL_DECODE = 0,   /* m <= 16: weight-streaming, H formed in every work-group */
  TQ_KERNEL_MID = 1,      /* 32-token blocks, K split over wavefronts */
  TQ_KERNEL_LARGE = 2,    /* 128 x 256 blocks, H in the main loop */
  TQ_KERNEL_PREFILL = 3   /* 128 x 256 blocks, H in a separate pass */
} tq_kernel;

/* The kernel tq_dual_gemm launches for descriptor d and m tokens (a tq_kernel
 * value), or -1 for a NULL or invalid descriptor or m outside [1, 2^24].
 * (Decode-sized m whose activation codes exceed the decode kernel's LDS --
 * e.g. m = 16 with k > 14336 -- run the mid kernel.)
 * Host-only; launches nothing.  Every kernel returns the same codes, H, s_H
 * and Q_H; the large and prefill kernels also sum each output in the order of
 * the fp64 definition's fp32 evaluation (ascending K-groups, then the
 * low-rank term), while the decode and mid kernels add partial sums over
 * parts of K, so their Y can differ from it in the last bits (within the
 * tolerance the fp32 accumulation allows). */
int tq_dual_gemm_kernel(const tq_weight_desc *d, int m);

/* The same computation as tq_dual_gemm, for tests and measurements:
 *   x          NULL: the activations are x_codes / x_scales as in
 *              tq_dual_gemm; otherwise (x_codes and x_scales NULL) the fp16
 *              activation [m,k] of tq_dual_gemm_fused_quant, quantized in the
 *              kernel (kernel must then be -1 or TQ_KERNEL_DECODE)
 *   kernel     -1: the kernel tq_dual_gemm would launch; otherwise the
 *              tq_kernel value to run (TQ_KERNEL_DECODE needs a decode-sized
 *              m that fits its LDS, TQ_KERNEL_LARGE / TQ_KERNEL_PREFILL need
 *              m > 512, TQ_KERNEL_MID serves any m; TQ_ERR_SHAPE otherwise)
 *   mid_tiles  0: the mid kernel's own choice of 32-column tiles per
 *              work-group; 1, 2 or 4 forces it (TQ_ERR_SHAPE otherwise)
 *   h, sh, qh  all NULL, or all set (r > 0, else TQ_ERR_RANK) to copy the
 *              low-rank intermediate of every token out of the kernel:
 *                h   [m,r] fp32     H before re-quantization
 *                sh  [m,r/group_r]  fp32 scales s_H
 *                qh  [m,r] int8     codes Q_H in [-7, 7]
 * Errors as tq_dual_gemm. */
tq_status tq_dual_gemm_debug(const tq_weight_desc *d, const void *packed, const void *x_codes,
                             const void *x_scales, const void *x, int m, void *y, tq_dtype y_dtype,
                             int kernel, int mid_tiles, void *h, void *sh, void *qh, void *stream);

/* The same layer without kernel fusion, the comparison baseline of the
 * paper's kernel profile (Appendix, Kernel Profile; Sec. 4.3 names the
 * intermediate traffic and launches that fusion removes): the residual 4-bit
 * GEMM writes Y, a second kernel writes H to global memory, a third
 * re-quantizes it to Q_H and s_H in global memory, and a fourth adds
 * Q_H Q(L2) to Y -- four launches.  H, s_H and Q_H are bit-identical to the
 * fused layer's; Y differs by the fp16 (bf16) rounding of the residual
 * before the low-rank part is added.
 *   scratch  device buffer of tq_unfused_scratch_bytes(d, m) bytes, owned by
 *            the caller, 16-byte aligned, no initial contents needed; after
 *            the call (r > 0) it holds, at 256-byte-aligned offsets in this
 *            order: H fp32 [m32][r_pad32], Q_H fp8 code bytes (sign << 7 |
 *            |q|) [m32][r_pad64], s_H fp32 [r/group_r][m32], with
 *            r_pad32 / r_pad64 the rank rounded up to 32 / 64
 *   other arguments as tq_dual_gemm
 * Errors as tq_dual_gemm (TQ_ERR_NULL for a NULL scratch). */
size_t tq_unfused_scratch_bytes(const tq_weight_desc *d, int m);
tq_status tq_dual_gemm_unfused(const tq_weight_desc *d, const void *packed, const void *x_codes,
                               const void *x_scales, int m, void *y, tq_dtype y_dtype,
                               void *scratch, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the layer
 * without fusion exactly as tq_dual_gemm_unfused computes it (same kernels,
 * same Y, H, s_H and Q_H), but its scratch is a static device array of
 * TQ_NOALLOC_SCRATCH_BYTES inside the library instead of a caller buffer.
 * Every device the library runs on holds one copy of that array until the
 * process ends; its address is looked up on the first call for a device
 * (the device of `stream`, or the current device for the NULL stream).  The
 * call allocates nothing and needs no initial contents in the array.
 *   limits  tq_unfused_scratch_bytes(d, m) <= TQ_NOALLOC_SCRATCH_BYTES (8 MiB:
 *           e.g. r = 128 up to m = 12928 tokens, r = 64 up to m = 25888),
 *           TQ_ERR_TOO_LARGE otherwise (checked before anything is launched)
 *   races   every call on one device shares that device's array: calls that
 *           may overlap in time on one device (other streams, other host
 *           threads) race and must be serialized by the caller; calls on one
 *           stream never overlap
 * Other arguments and errors as tq_dual_gemm_unfused (no scratch argument). */
#define TQ_NOALLOC_SCRATCH_BYTES (8u << 20)
tq_status tq_dual_gemm_unfused_noalloc(const tq_weight_desc *d, const void *packed,
                                       const void *x_codes, const void *x_scales, int m, void *y,
                                       tq_dtype y_dtype, void *stream);

/* Copy the packed weights out (for tests/debug), codes as TQ4 words (the
 * packed layout's sign-magnitude encoding, 8 codes per word):
 *   w_codes  [n, k/8] TQ4 words      w_scales  [n, k/group] fp16
 *   l1_codes [r, k/8] TQ4 words (row j = column j of L1, along k)
 *   l1_scales[r, k/group] fp16
 *   l2_codes [n, r/8] TQ4 words (row c = column c of L2, along r)
 *   l2_scales[n, r/group_r] fp16
 * The l1/l2 pointers may be NULL iff r == 0.
 * Errors: TQ_ERR_NULL, TQ_ERR_BUFFER, TQ_ERR_ALIGN, TQ_ERR_HIP. */
tq_status tq_export_weights(const tq_weight_desc *d, const void *packed, void *w_codes,
                            void *w_scales, void *l1_codes, void *l1_scales, void *l2_codes,
                            void *l2_scales, void *stream);

/* The same in the canonical 4-bit layout: two's-complement nibbles (codes in
 * [-7, 7]), element 2i in the low and 2i+1 in the high nibble of byte i,
 * contiguous along the reduction axis; scales as fp16 bit patterns.
 *   wq  [n, k/2]  bytes          ws  [n, k/group] fp16
 *   l1q [r, k/2]  (row j = column j of L1)   l1s [k/group, r] fp16
 *   l2q [n, r/2]  (row c = column c of L2)   l2s [r/group_r, n] fp16
 * The l1/l2 pointers may be NULL iff r == 0.
 * Errors: TQ_ERR_NULL, TQ_ERR_BUFFER, TQ_ERR_ALIGN, TQ_ERR_HIP. */
tq_status tq_export_weights_canonical(const tq_weight_desc *d, const void *packed, void *wq, void *ws,
                                      void *l1q, void *l1s, void *l2q, void *l2s, void *stream);

/* Activation codes and scales written by tq_quant_act (m tokens, reduction
 * size k, quantization group `group`) copied out in the canonical layout:
 *   codes_out  [m, k/2] bytes, two's-complement nibbles as above
 *   scales_out [m, k/group] fp16
 * Errors: TQ_ERR_NULL, TQ_ERR_SHAPE, TQ_ERR_GROUP, TQ_ERR_ALIGN, TQ_ERR_HIP. */
tq_status tq_act_codes_canonical(const void *x_codes, const void *x_scales, int m, int k, int group,
                                 void *codes_out, void *scales_out, void *stream);

/* Static description of a status code; never NULL. */
const char *tq_status_string(tq_status s);

#ifdef __cplusplus
}
#endif

#endif /* TQ_H */
