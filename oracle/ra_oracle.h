/*
 * ra_oracle.h -- plain CPU oracle for the RotateAttention INT4 attention path
 * (Liu et al., "RotateAttention: RoPE-Aware Rotation and Range Rectification for
 * INT4 Quantized Attention in Video Generation").
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  The GPU library
 * never includes, links or calls anything here, and nothing here includes or
 * calls the GPU library.
 *
 * Every routine works on ONE attention head (one (b, h) slice): token-major
 * arrays [N][D] with D == 128 channels, exactly as the paper's problem statement
 * (Sec. 3: Q, K, V in R^{N x D}).
 *
 * Two precisions appear:
 *   - "_f64" routines follow the paper's mathematics in double precision; they
 *     are the fidelity reference and the subject of the invariance pins.
 *   - "_f32" routines are the single-precision operation sequence that defines
 *     every integer the INT4 path produces (codes, scales, S tiles, running
 *     maxima); they are written op by op with fmaf/rintf so that the result is
 *     fixed by IEEE-754 binary32 arithmetic alone (build with -ffp-contract=off).
 */
#ifndef RA_ORACLE_H
#define RA_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORA_ROT_NONE = 0, ORA_ROT_INTERLEAVED = 1, ORA_ROT_HALF = 2, ORA_ROT_HADAMARD = 3 };
enum { ORA_PQ_RANGE15 = 0, ORA_PQ_SYM7 = 1, ORA_PQ_NONE = 2 };

/* Geometry of the 3D RoPE (Sec. 3): grid T x Hg x W with N = T*Hg*W tokens,
 * token n = (t*Hg + h)*W + w, head dim D = D_t + D_h + D_w (each even). */
typedef struct {
  int N, D;
  int T, Hg, W;
  int split[3];
  double theta;
  int rotation;          /* ORA_ROT_* */
  const double* rot;     /* [D/2][2][2] O(2) blocks, row-major; NULL = H_2 in every block */
  int in_fp16;           /* input bits are binary16 (else bfloat16) */
} ora_rope_cfg;

/* The 2x2 matrix that maps the channel pair p of token n, row-vector form
 * [y0 y1] = [x0 x1] * G.  For ORA_ROT_INTERLEAVED G = M * R_p (rotation merged
 * into RoPE, Sec. 4.1.2); otherwise G = M (plain 3D RoPE, Sec. 3). fp64. */
void ora_rope_block(const ora_rope_cfg* c, int n, int p, double G[4]);

/* RoPE followed by the chosen rotation, 16-bit input bits (bf16, or fp16 with
 * in_fp16) -> y [N][D].
 * ORA_ROT_HADAMARD is the "Full" rotation the paper compares against
 * (Sec. 5.3 baselines): y = RoPE(x) H_D with the orthonormal Sylvester matrix
 * H_D = H_2 (x) H_{D/2} of Sec. 4.3.  In binary32 it is
 * the Kronecker recursion taken literally -- the first factor pairs channel i
 * of the first half with channel i of the second half (sum, difference), then
 * each half recurses -- with every sum and difference unscaled and one final
 * multiply by fl32(D^-1/2) (the product of the log2(D) factors 1/sqrt 2). */
void ora_rope_rot_f32(const ora_rope_cfg* c, const uint16_t* x_bits, float* y);
void ora_rope_rot_f64(const ora_rope_cfg* c, const uint16_t* x_bits, double* y);

/* y <- y H_D in place for one row of D = 2^n values: the binary32 sequence
 * described above (sum/difference butterflies, widest stride first, then the
 * single normalising multiply). */
void ora_hadamard_f32(float* y, int D);
void ora_hadamard_f64(double* y, int D);

/* Smoothing mean (Sec. 4, QKV smoothing), order-independent definition: every
 * value is scaled by 2^20, clamped to +-2^32, rounded half-to-even to an
 * integer; the integers are summed exactly; mu = fl32(sum / (N * 2^20)). */
void ora_mean_fixed(const float* y, int N, int D, float* mu);

/* z = fl32(y - mu) for every token (mu broadcast over tokens). */
void ora_center(const float* y, const float* mu, int N, int D, float* z);

/* Q smoothing (Sec. 4): the per-key score bias b_j = mu_Q . zk_j that the
 * smoothed-away query mean contributes, binary32, pairwise summation over the
 * channels (halves recursively; D a power of two).  bias [N]. */
void ora_key_bias(const float* mu_q, const float* zk, int N, int D, float* bias);

/* Symmetric INT4 quantization of Q or K (Sec. 5.1: per-token, or per-block of
 * g tokens): scale s = amax/7, codes = clamp(rint(z * (7/amax)), -7, 7).
 * codes [N][D], scales [ceil(N/g)]. */
void ora_quant_tokens(const float* z, int N, int D, int g, int8_t* codes, float* scales);

/* INT4 quantization of V per group of g tokens and per channel (Sec. 5.1:
 * per-group V).  codes [N][D], scales [ceil(N/g)][D]. */
void ora_quant_v(const float* z, int N, int D, int g, int8_t* codes, float* scales);

typedef struct {
  int N, D;
  int q_group, k_group, v_group;
  int kv_block;          /* online-softmax block size (Sec. 4.2) */
  int p_quant;           /* ORA_PQ_*; ORA_PQ_NONE keeps P unquantized (pin only) */
  double sm_scale;       /* 0 = 1/sqrt(D) */
  int l_quant;           /* 0: l = sum of the unquantized P; 1: l = sum of the dequantized
                            P^ = u / 15 (u / 7 for SYM7), the same values PV uses */
} ora_attn_cfg;

/* Blockwise INT4 attention for query rows [row0, row0+nrows) of one head
 * (Sec. 4.2 online softmax + Range-optimized P quantization).  O [nrows][D] is
 * returned in double.  bias (NULL without Q smoothing): the per-key score
 * bias b [N]; the log2e-scaled score of key j is then
 * t = fma(S, c, fl(b_j Kc)) and x = fl(t - m), otherwise x = fma(S, c, -m)
 * with the maximum taken over fl(S c).  Optional dumps (NULL to skip):
 *   S_dump [nrows][N] int32 exact S = q_codes . k_codes
 *   u_dump [nrows][N] P codes u = P~ + 8 in [0,15] (or [0,7] for SYM7)
 *   x_dump [nrows][N] the binary32 exponent argument x of each P = 2^x
 *   m_dump [nrows][ceil(N/kv_block)] running maximum after each block
 *   l_dump [nrows] final normaliser */
void ora_attn_int4(const ora_attn_cfg* a,
                   const int8_t* qc, const float* qs,
                   const int8_t* kc, const float* ks,
                   const int8_t* vc, const float* vs, const float* mu_v, const float* bias,
                   int row0, int nrows, double* O,
                   int32_t* S_dump, uint8_t* u_dump, float* x_dump, float* m_dump,
                   double* l_dump);

/* Unquantized softmax attention in fp64 (the fidelity reference), two-pass
 * (global row max, then sum); q, k, v [N][D]; rows [row0, row0+nrows). */
void ora_attn_ref_f64(const double* q, const double* k, const double* v, int N, int D,
                      double sm_scale, int row0, int nrows, double* O);

/* 16-bit fallback attention semantics (the FP16 attention the paper keeps for
 * sensitive steps and blocks, Sec. 5.1; bf16 or fp16 with the flag): 16-bit
 * q/k/v bits, fp64 dot products, blockwise online softmax over blocks of
 * kv_block keys in ascending order with exact exp2, P rounded to binary32 and
 * then to the 16-bit type before the PV product, the normaliser l from the
 * unrounded P.  ora_attn_bf16 is the bf16 form. */
void ora_attn_fb16(const uint16_t* qb, const uint16_t* kb, const uint16_t* vb, int N, int D,
                   int kv_block, double sm_scale, int fp16, int row0, int nrows, double* O);
void ora_attn_bf16(const uint16_t* qb, const uint16_t* kb, const uint16_t* vb, int N, int D,
                   int kv_block, double sm_scale, int row0, int nrows, double* O);

/* Helpers exposed for the pins. */
float ora_bf16_to_f32(uint16_t b);
uint16_t ora_f32_to_bf16(float f);
float ora_f16_to_f32(uint16_t h);
uint16_t ora_f32_to_f16(float f);     /* round to nearest even, overflow to inf */
float ora_exp2_f32(float x);          /* exp2 in double, rounded to binary32 */
int ora_pcode(float P, int p_quant);  /* u = clamp(rint(fl(15P)), 0, 15) or SYM7 */
int ora_threads(void);                /* worker threads the parallel loops use */

#ifdef __cplusplus
}
#endif
#endif
