/*
 * rotate_attn.h -- C ABI of the MI355X (gfx950) INT4 RotateAttention library.
 *
 * The library implements the attention hot path of RotateAttention
 * (Liu et al., "RotateAttention: RoPE-Aware Rotation and Range Rectification
 * for INT4 Quantized Attention in Video Generation"): 3D RoPE fused with the
 * RoPE-aware Q/K rotation (Sec. 4.1.2 interleaved/merged, Sec. 4.1.3 half),
 * smoothing (Sec. 4), INT4 quantization of Q, K and V (Sec. 5.1), the INT4
 * FlashAttention forward with the Range-optimized P quantization (Sec. 4.2),
 * and the BF16/FP16 fallback attention used for accuracy-sensitive blocks and
 * denoising steps (abstract; Sec. 5.1 mixed-precision schedule).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers owned by the caller; the library
 *    never frees them.  `rot_blocks` in ra_params is a HOST pointer.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).  Every
 *    call only enqueues work on that stream and returns; results are ready when
 *    the stream reaches them.  Calls that overlap on one device must use
 *    distinct workspaces.
 *  - Inputs q, k, v have layout [B][H][N][D] (token-major rows of D elements),
 *    dtype ra_params.in_dtype (RA_BF16 or RA_FP16).  Output o has the same
 *    layout in ra_params.out_dtype (RA_BF16, RA_FP16 or RA_FP32).
 *  - q, k, v and the code buffers (q_codes, k_codes, v_codes) must be 16-byte
 *    aligned: they are read and written in 16-byte pieces (RA_ERR_INVALID
 *    otherwise).
 *  - Only D == 128 is supported (RA_ERR_UNSUPPORTED otherwise).
 *  - Every entry point validates all arguments before touching the GPU and
 *    returns RA_OK (0) or a negative RA_ERR_* code; no exception crosses the ABI.
 *    rotate_attn_last_error() returns a thread-local message for the last
 *    failure on the calling thread.
 *  - The library allocates no device memory and creates no streams or events.
 *    The RoPE/rotation tables (binary64 trigonometry rounded once to binary32)
 *    are built on the host on the first call for a geometry (grid, split,
 *    theta, rotation, blocks) and kept for the life of the process in pinned
 *    host memory (hipHostMalloc, never freed); every call that needs them
 *    copies them into its workspace with a small kernel on `stream` that reads
 *    the pinned memory through its device mapping (no copy engine, so the copy
 *    is ordered with the kernels around it at no extra latency).  Only that
 *    first call per geometry performs a host allocation.
 *  - Results are deterministic: repeated calls give identical bytes.
 *
 * Packed INT4 layouts (written by the quantize calls, read by the attention)
 * ------------------------------------------------------------------------
 *  Npad = N rounded up to a multiple of 128; tokens n >= N hold zero codes.
 *  A code is a 4-bit two's-complement nibble in [-7, 7].
 *
 *  INT4 container (code_format == RA_CODES_INT4):
 *  Q/K codes, per head (Npad * 64 bytes, heads contiguous, head bh at
 *  bh * Npad * 64): token n = 32*c + r, channel pair j (channels 2j and 2j+1)
 *  lives in byte ((c*8 + j/8)*32 + r)*8 + (j%8); channel 2j in the low nibble,
 *  channel 2j+1 in the high nibble.
 *
 *  V codes, per head (Npad * 64 bytes): token n = 32*c + kappa, channel ch.
 *  With a = kappa/16, b = (kappa/8)%2, h = (kappa/4)%2, s = kappa%4, the
 *  nibble index is np = 8a + 2s + b; the code lives in byte
 *  ((c*2 + h)*128 + ch)*8 + np/2, low nibble when np is even.
 *  (This order makes each 32-token chunk an operand of the int8 matrix core.)
 *
 *  E2M3 container (code_format == RA_CODES_E2M3), Npad * 96 bytes per head.
 *  A code c is the 6-bit E2M3 float equal to c (sign in bit 5, exponent bias 1,
 *  3 mantissa bits); 32 codes form a 24-byte record, code f at bits [6f, 6f+6)
 *  of the little-endian record.
 *   Q/K: token n = 32*c + r, channel ch: record ((c*2 + ch/64)*2 + (ch/32)%2)*32 + r,
 *        field ch%32.
 *   V:   token n = 64*g + kappa, channel ch: record ((g*4 + ch/32)*2 + (kappa/4)%2)*32
 *        + ch%32, field 8*((kappa%32)/8) + 2*(kappa%4) + kappa/32.
 *
 *  Scales are binary32.  Q scales: [B*H][Npad/q_group]; K scales:
 *  [B*H][Npad/k_group]; V scales: [B*H][ceil(N/v_group)][128].  Q/K groups
 *  that hold no valid token have scale 0.
 */
#ifndef ROTATE_ATTN_H
#define ROTATE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define RA_OK 0
#define RA_ERR_INVALID (-1)     /* bad shape, split, grid, group, null pointer */
#define RA_ERR_UNSUPPORTED (-2) /* valid request the library does not implement */
#define RA_ERR_WORKSPACE (-3)   /* workspace missing or smaller than required */
#define RA_ERR_HIP (-4)         /* a HIP runtime call failed (see last_error) */

/* rotation applied to Q and K after 3D RoPE (Sec. 4.1) */
#define RA_ROT_NONE 0
#define RA_ROT_INTERLEAVED 1 /* Sec. 4.1.2: blocks on (2i, 2i+1), merged into the RoPE table */
#define RA_ROT_HALF 2        /* Sec. 4.1.3: pairs (i, i + D_j/2) inside each RoPE segment */
#define RA_ROT_HADAMARD 3    /* "Full" rotation (Sec. 5.3 baseline): RoPE, then the orthonormal
                                128x128 Sylvester-Hadamard matrix of Sec. 4.3; rot_blocks unused */

/* V rotation (Sec. 4.3).  The paper folds the D x D Hadamard H into W_v and
 * W_o offline, so V arrives already rotated (RA_VROT_NONE).  For callers that
 * cannot change the weights, RA_VROT_HADAMARD rotates V online: quantize_v
 * takes V H (the binary32 butterflies of RA_ROT_HADAMARD) and the INT4
 * attention returns O = O' H^T, O' being the output in the rotated basis. */
#define RA_VROT_NONE 0
#define RA_VROT_HADAMARD 1

/* quantization of P (Sec. 4.2.1) */
#define RA_PQ_RANGE15 0 /* affine: fixed scale 15, zero-point -8, 16 levels */
#define RA_PQ_SYM7 1    /* symmetric baseline: round(7 P), 8 levels */

/* smoothing flags (Sec. 4: biases shared by all tokens) */
#define RA_SMOOTH_K 1 /* subtract the per-channel mean of rotated K (softmax invariant) */
#define RA_SMOOTH_V 2 /* subtract the per-channel mean of V, add it back to O */
#define RA_SMOOTH_Q 4 /* subtract the per-channel mean mu_Q of rotated Q; every key j then
                         carries the score bias b_j = mu_Q . K_j (k_bias), added to its
                         dequantized scores (Sec. 4: Q, K and V smoothing) */

/* dtypes */
#define RA_BF16 0
#define RA_FP16 1
#define RA_FP32 2

/* container of the INT4 codes (the code values are the same in both) */
#define RA_CODES_INT4 0 /* two's-complement nibbles, two per byte (int8 matrix-core kernel) */
#define RA_CODES_E2M3 1 /* each code as a 6-bit E2M3 float, the operand format of the
                           FP6 matrix core: exact for integers in [-7, 7], twice the int8 rate */

/* device scratch of rotate_attn_fwd_int4_noalloc, per GPU (128 MiB: the 32760-token,
   12-head layer fits) */
#define RA_NOALLOC_SCRATCH_BYTES (128u << 20)

/* which forward a workspace is sized for */
#define RA_PATH_INT4 0
#define RA_PATH_FP16 1

typedef struct ra_params {
  int32_t B, H, N, D;      /* batch, heads, tokens (N == T*Hg*W), head dim (128) */
  int32_t grid[3];         /* T, Hg, W: token n = (t*Hg + h)*W + w (Sec. 3) */
  int32_t rope_split[3];   /* D_t, D_h, D_w: each even and > 0, sum == D (Sec. 3) */
  float rope_theta;        /* RoPE base, e.g. 10000 or 256 */
  int32_t rotation;        /* RA_ROT_* */
  const double* rot_blocks;/* host, [D/2][2][2] row-major O(2) blocks; NULL = H_2 (Sec. 4.1).
                              Each block must be orthogonal (|R R^T - I| <= 1e-6 elementwise,
                              RA_ERR_INVALID otherwise); used by INTERLEAVED and HALF only */
  int32_t p_quant;         /* RA_PQ_* */
  int32_t smooth;          /* RA_SMOOTH_* bitmask */
  int32_t q_group;         /* tokens per Q scale: 1 (per-token) .. 128, must divide 128 */
  int32_t k_group;         /* tokens per K scale: 1, 16, 32, 64 or 128 */
  int32_t v_group;         /* tokens per V scale (per channel): a multiple of kv_block, or >= N */
  int32_t kv_block;        /* online-softmax block of both paths: 64 or 128 keys (fixes the
                              running-max granularity of Sec. 4.2 and hence the P codes, and
                              the block at whose maximum the fallback rounds P) */
  float sm_scale;          /* softmax scale; 0 = 1/sqrt(D) */
  int32_t in_dtype;        /* RA_BF16 | RA_FP16 */
  int32_t out_dtype;       /* RA_BF16 | RA_FP16 | RA_FP32 */
  int32_t code_format;     /* RA_CODES_*: container of the codes quantize_* write and attn_int4 reads */
  int32_t v_rotation;      /* RA_VROT_*: how the INT4 path treats V (the fallback takes V as given) */
  int32_t l_quant;         /* INT4 normaliser: 0 = l is the sum of the unquantized P (default);
                              1 = l is the sum of the dequantized P^ = u/15 (u/7 for SYM7), the
                              values PV uses, so every output row is a convex combination */
} ra_params;

/* Sizes of the caller-visible INT4 buffers for these parameters (the code and
 * scale layouts above; Sec. 5.1 granularities). */
typedef struct ra_layout {
  int64_t n_pad;          /* Npad */
  int64_t qk_code_bytes;  /* bytes of ONE of q_codes / k_codes (all heads) */
  int64_t q_scale_count;  /* floats in q_scale */
  int64_t k_scale_count;  /* floats in k_scale */
  int64_t v_code_bytes;   /* bytes of v_codes */
  int64_t v_scale_count;  /* floats in v_scale */
  int64_t mu_count;       /* floats in mu_q / mu_k / mu_v: B*H*D */
  int64_t k_bias_count;   /* floats in k_bias: B*H*Npad */
} ra_layout;

/* Fills *out; RA_ERR_INVALID / RA_ERR_UNSUPPORTED on bad parameters. */
int rotate_attn_layout(const ra_params* p, ra_layout* out);

/* Workspace bytes needed by the calls of `path` (RA_PATH_INT4 covers
 * quantize_qk, quantize_v, quantize_qkv, attn_int4 and fwd_int4; RA_PATH_FP16
 * covers prepare_fp16, attn_fp16 and fwd_fp16).  The workspace is device
 * memory, 256-byte aligned, owned by the caller and reused by every call; it
 * holds the RoPE tables, the smoothing sums, and (INT4 forward) the codes and
 * scales; its content between calls is irrelevant. */
int rotate_attn_workspace_size(const ra_params* p, int path, size_t* bytes);

/* Producer for Q and K (Sec. 3, 4, 4.1, 5.1): 3D RoPE and the chosen rotation,
 * K smoothing (if RA_SMOOTH_K), Q smoothing (if RA_SMOOTH_Q), per-group INT4
 * quantization, packing.
 * q, k: inputs [B][H][N][D].  q_codes/k_codes: ra_layout.qk_code_bytes each;
 * q_scale/k_scale: ra_layout.q_scale_count / k_scale_count floats.
 * mu_k, mu_q: nullable, receive the smoothing means [B*H][D] (zeros where that
 * smoothing is off).
 * k_bias: with RA_SMOOTH_Q required (RA_ERR_INVALID if NULL), receives the
 * per-key score bias b_j = mu_Q . K_j [B*H][Npad] in binary32 (K after RoPE,
 * rotation and K smoothing; pairwise sum over the channels: halves of the
 * channel range recursively; padded keys get 0); ignored otherwise. */
int rotate_attn_quantize_qk(const ra_params* p, const void* q, const void* k, uint8_t* q_codes,
                            float* q_scale, uint8_t* k_codes, float* k_scale, float* mu_k,
                            float* mu_q, float* k_bias, void* workspace, size_t workspace_bytes,
                            void* stream);

/* Producer for V (Sec. 4.3, 5.1): V is taken as given (a Hadamard rotation of
 * V is folded into W_v/W_o offline), smoothed (if RA_SMOOTH_V) and quantized
 * per (v_group tokens, channel).  mu_v: nullable, receives the V mean [B*H][D]
 * that the attention adds back (zeros if smoothing is off). */
int rotate_attn_quantize_v(const ra_params* p, const void* v, uint8_t* v_codes, float* v_scale,
                           float* mu_v, void* workspace, size_t workspace_bytes, void* stream);

/* Both producers in one call (Sec. 3, 4, 4.1, 4.3, 5.1): the same results as
 * quantize_qk followed by quantize_v, bit for bit, in fewer passes.  Arguments
 * as in the two calls; mu_k, mu_q, mu_v nullable; k_bias required with
 * RA_SMOOTH_Q. */
int rotate_attn_quantize_qkv(const ra_params* p, const void* q, const void* k, const void* v,
                             uint8_t* q_codes, float* q_scale, uint8_t* k_codes, float* k_scale,
                             uint8_t* v_codes, float* v_scale, float* mu_k, float* mu_q, float* mu_v,
                             float* k_bias, void* workspace, size_t workspace_bytes, void* stream);

/* INT4 attention on already quantized operands (Sec. 4.2, Sec. 4.2.1, Sec. 5.1):
 * S = Q~ K~^T exact, blockwise online softmax with blocks of kv_block keys in
 * ascending order, P mapped to the unsigned code u = round(15 P) in [0, 15]
 * (the affine code P~ = u - 8, Sec. 4.2.1), PV on the codes,
 * O = (sum of dequantized PV) / l + mu_v, l = sum of the unquantized P.  The
 * container selects the matrix-core path: RA_CODES_E2M3 runs the FP6 matrix
 * core (v_mfma_scale_f32_*_f8f6f4, codes as E2M3 values, binary32 sums that are
 * exact for these integers); RA_CODES_INT4 runs the int8 matrix core
 * (v_mfma_i32_32x32x32_i8 on the unpacked nibbles, int32 accumulation).  Both
 * compute the same integers.
 * mu_v: nullable (treated as zeros).  k_bias: the per-key score bias written
 * by quantize_qk, required with RA_SMOOTH_Q (RA_ERR_INVALID if NULL), ignored
 * otherwise; with it the log2e-scaled score of key j is
 * t = fma(S, c, fl(b_j * Kc)) and P = 2^(t - m).  o: [B][H][N][D] in out_dtype. */
int rotate_attn_attn_int4(const ra_params* p, const uint8_t* q_codes, const float* q_scale,
                          const uint8_t* k_codes, const float* k_scale, const uint8_t* v_codes,
                          const float* v_scale, const float* mu_v, const float* k_bias, void* o,
                          void* stream);

/* Debug variant of rotate_attn_attn_int4 (the quantities of Sec. 4.2 made
 * observable): runs the same kernel with a dump enabled for the query rows
 * [row0, row0 + rows) of head bh:
 *   s_out [rows][N] int32  exact S = Q~ . K~
 *   u_out [rows][N] uint8  P codes u in [0, 15]
 *   m_out [rows][ceil(N/kv_block)] binary32 running maximum after each block
 * (all device pointers, any may be NULL).  o receives the same output as the
 * plain call. */
int rotate_attn_attn_int4_debug(const ra_params* p, const uint8_t* q_codes, const float* q_scale,
                                const uint8_t* k_codes, const float* k_scale,
                                const uint8_t* v_codes, const float* v_scale, const float* mu_v,
                                const float* k_bias, void* o, int32_t bh, int32_t row0, int32_t rows,
                                int32_t* s_out,
                                uint8_t* u_out, float* m_out, void* stream);

/* Whole INT4 forward (Sec. 3-4.3 producers, Sec. 4.2 attention, Sec. 5.1
 * granularities): quantize_qkv + attn_int4, codes and scales kept in the
 * workspace (size RA_PATH_INT4). */
int rotate_attn_fwd_int4(const ra_params* p, const void* q, const void* k, const void* v, void* o,
                         void* workspace, size_t workspace_bytes, void* stream);

/* The whole INT4 forward of rotate_attn_fwd_int4 without a caller workspace
 * and without allocating anything on the device: for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Its workspace is a static device array of
 * RA_NOALLOC_SCRATCH_BYTES per GPU, part of the library's code object (held
 * from the first call on a device until the process ends); problems whose
 * INT4 workspace (rotate_attn_workspace_size, RA_PATH_INT4) exceeds it return
 * RA_ERR_UNSUPPORTED before any HIP call.  The RoPE tables are written into
 * that array through kernel arguments when the geometry differs from the
 * previous call's on the device (the host keeps one table per geometry).
 * Every call on a GPU shares that GPU's array and leaves its contents behind:
 * calls that overlap on one GPU (different streams or threads) race and must
 * be serialised by the caller.  Output identical to rotate_attn_fwd_int4. */
int rotate_attn_fwd_int4_noalloc(const ra_params* p, const void* q, const void* k, const void* v, void* o,
                                 void* stream);

/* Producer of the fallback (the FP16 attention the paper keeps for sensitive
 * steps and blocks, Sec. 5.1): plain 3D RoPE (Sec. 3; no rotation, which is an
 * identity in exact arithmetic, and no smoothing) of Q and K rounded to
 * in_dtype, and V re-laid out for the matrix cores, into the workspace (size
 * RA_PATH_FP16, which also holds the RoPE tables). */
int rotate_attn_prepare_fp16(const ra_params* p, const void* q, const void* k, const void* v,
                             void* workspace, size_t workspace_bytes, void* stream);

/* Fallback attention kernel alone (Sec. 5.1 FP16 attention with the blockwise
 * online softmax of Sec. 4.2) on a workspace filled by prepare_fp16: 16-bit
 * matrix cores, online softmax with blocks of kv_block (64 or 128) keys in
 * ascending order, P rounded to in_dtype before PV (at the running maximum of
 * its block), l from the unrounded P. */
int rotate_attn_attn_fp16(const ra_params* p, const void* workspace, size_t workspace_bytes, void* o,
                          void* stream);

/* Whole fallback forward (Sec. 5.1): prepare_fp16 + attn_fp16. */
int rotate_attn_fwd_fp16(const ra_params* p, const void* q, const void* k, const void* v, void* o,
                         void* workspace, size_t workspace_bytes, void* stream);

/* Mixed-precision dispatch (abstract; Sec. 5.1 schedule): fallback != 0 runs
 * fwd_fp16, otherwise fwd_int4.  The workspace must fit the chosen path. */
int rotate_attn_fwd(const ra_params* p, int fallback, const void* q, const void* k, const void* v,
                    void* o, void* workspace, size_t workspace_bytes, void* stream);

/* Status code -> static text; and the thread-local message of the last failure
 * on the calling thread (library utilities, no paper passage). */
const char* rotate_attn_error_string(int status);
const char* rotate_attn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ROTATE_ATTN_H */
