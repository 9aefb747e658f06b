/*
 * ra_oracle.c -- plain, slow CPU oracle of the RotateAttention INT4 attention
 * path.  TEST INFRASTRUCTURE ONLY (see ra_oracle.h): tests, the smoke check and
 * the benchmark's CPU-baseline leg are its only callers.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fopenmp -fPIC -shared
 * (-ffp-contract=off keeps every a*b+c of the binary32 sequences below as two
 * rounded operations unless fmaf is written explicitly).
 *
 * Paper references are to sections and equations of the paper:
 *   Sec. 3     3D RoPE, block-diagonal rotary matrix M of D/2 SO(2) blocks split
 *              into the temporal/height/width segments D = D_f + D_h + D_w.
 *   Sec. 4     smoothing of Q, K, V (shared biases) before quantization.
 *   Sec. 4.1   block-diagonal orthogonal rotation R, blocks initialised to H_2.
 *   Sec. 4.1.2 interleaved rotation merged into RoPE: RoPE(Q) R = Q (M R).
 *   Sec. 4.1.3 half rotation Q Pi R, pairing d_i with d_{i + D_j/2} per segment.
 *   Sec. 4.3   D x D Sylvester-Hadamard matrix (Kronecker recursion), used here
 *              as the "Full" Q/K rotation baseline of Sec. 5.3.
 *   Sec. 4.2   FlashAttention blockwise online softmax and the affine
 *              (Range-optimized) P mapping with fixed scale 15 and zero-point -8.
 *   Sec. 5.1   per-token Q/K quantization and per-group V quantization.
 */
#include "ra_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define LOG2E 1.4426950408889634074

/* binary16 bits -> binary32 (exact: every binary16 value is a binary32 value). */
float ora_f16_to_f32(uint16_t h) {
  const int e = (h >> 10) & 0x1f, m = h & 0x3ff;
  double v;
  if (e == 0) v = ldexp((double)m, -24);                       /* zero or subnormal */
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexp(1024.0 + (double)m, e - 25);                   /* (1 + m/1024) 2^(e-15) */
  return (float)((h & 0x8000) ? -v : v);
}

/* Round-to-nearest-even binary32 -> binary16.  |f| is split into a power of
 * two and a significand in double (exact), the significand is rounded to 10
 * fraction bits with rint (ties to even under the default rounding mode);
 * below 2^-14 the grid is the fixed subnormal step 2^-24; from 65520 (half way
 * between the largest finite value 65504 and 2^16) upward the result is inf. */
uint16_t ora_f32_to_f16(float f) {
  const uint16_t sign = signbit(f) ? 0x8000u : 0u;
  if (isnan(f)) return (uint16_t)(sign | 0x7e00u);
  const double a = fabs((double)f);
  if (a >= 65520.0) return (uint16_t)(sign | 0x7c00u);
  if (a < ldexp(1.0, -14)) return (uint16_t)(sign | (uint16_t)rint(ldexp(a, 24)));
  int ex;
  frexp(a, &ex);                        /* a = fr 2^ex, fr in [0.5, 1) */
  int E = ex - 1;                       /* a = s 2^E, s in [1, 2) */
  double q = rint((ldexp(a, -E) - 1.0) * 1024.0);
  if (q == 1024.0) {
    q = 0.0;
    ++E;
  }
  if (E + 15 >= 31) return (uint16_t)(sign | 0x7c00u);
  return (uint16_t)(sign | ((E + 15) << 10) | (uint16_t)q);
}

static float in16_to_f32(uint16_t b, int fp16) { return fp16 ? ora_f16_to_f32(b) : ora_bf16_to_f32(b); }
static uint16_t f32_to_16(float f, int fp16) { return fp16 ? ora_f32_to_f16(f) : ora_f32_to_bf16(f); }

float ora_bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Round-to-nearest-even binary32 -> bfloat16 (NaN kept quiet). */
uint16_t ora_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

int ora_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ---------------------------------------------------------------- 3D RoPE -- */

/* Token n -> grid coordinates (t, h, w); t-major, w fastest, 0-based. */
static void token_pos(const ora_rope_cfg* c, int n, int pos[3]) {
  pos[2] = n % c->W;
  pos[1] = (n / c->W) % c->Hg;
  pos[0] = n / (c->W * c->Hg);
}

/* Channel pair p (channels 2p, 2p+1) -> axis a and index k inside the segment. */
static void pair_axis(const ora_rope_cfg* c, int p, int* a, int* k) {
  int first = 0;
  for (int ax = 0; ax < 3; ++ax) {
    int np = c->split[ax] / 2;
    if (p < first + np) {
      *a = ax;
      *k = p - first;
      return;
    }
    first += np;
  }
  *a = 2;
  *k = p - first; /* unreachable for valid p */
}

/* The rotation block R_p in fp64 (Sec. 4.1, H_2 equation when none given). */
static void rot_block(const ora_rope_cfg* c, int p, double R[4]) {
  if (c->rot) {
    memcpy(R, c->rot + 4 * p, 4 * sizeof(double));
  } else {
    double r = 1.0 / sqrt(2.0);
    R[0] = r; R[1] = r; R[2] = r; R[3] = -r;
  }
}

/* Sec. 3: M is block diagonal with SO(2) blocks; pair k of axis a turns by
 * phi = pos_a * theta^(-2k/D_a) (RoFormer frequencies per axis).  Row-vector
 * convention [y0 y1] = [x0 x1] M with M = [[cos, sin], [-sin, cos]].
 * Sec. 4.1.2: the interleaved rotation is merged as G = M R_p. */
void ora_rope_block(const ora_rope_cfg* c, int n, int p, double G[4]) {
  int pos[3], a, k;
  token_pos(c, n, pos);
  pair_axis(c, p, &a, &k);
  double omega = pow(c->theta, -(2.0 * k) / (double)c->split[a]);
  double phi = (double)pos[a] * omega;
  double cs = cos(phi), sn = sin(phi);
  double M[4] = {cs, sn, -sn, cs};
  if (c->rotation == ORA_ROT_INTERLEAVED) {
    double R[4];
    rot_block(c, p, R);
    G[0] = M[0] * R[0] + M[1] * R[2];
    G[1] = M[0] * R[1] + M[1] * R[3];
    G[2] = M[2] * R[0] + M[3] * R[2];
    G[3] = M[2] * R[1] + M[3] * R[3];
  } else {
    memcpy(G, M, sizeof(M));
  }
}

/* The orthonormal Sylvester-Hadamard transform of one row (Sec. 4.3:
 * H_{2^n} = H_2 (x) H_{2^(n-1)}, with H_2 = [[1, 1], [1, -1]] / sqrt 2 of Sec. 4.1).
 * For a row vector x = [a b] split into halves, x (H_2 (x) H') = [(a + b) H',
 * (a - b) H'] / sqrt 2, so each level forms sums and differences of the two
 * halves and recurses into both; the 1/sqrt 2 of every level is collected into
 * one factor D^-1/2 applied at the end. */
static void hadamard_levels_f32(float* y, int D) {
  for (int len = D; len >= 2; len /= 2) {
    int h = len / 2;
    for (int base = 0; base < D; base += len)
      for (int i = 0; i < h; ++i) {
        float a = y[base + i], b = y[base + i + h];
        y[base + i] = a + b;
        y[base + i + h] = a - b;
      }
  }
}

void ora_hadamard_f32(float* y, int D) {
  hadamard_levels_f32(y, D);
  float r = (float)(1.0 / sqrt((double)D));
  for (int i = 0; i < D; ++i) y[i] = y[i] * r;
}

void ora_hadamard_f64(double* y, int D) {
  for (int len = D; len >= 2; len /= 2) {
    int h = len / 2;
    for (int base = 0; base < D; base += len)
      for (int i = 0; i < h; ++i) {
        double a = y[base + i], b = y[base + i + h];
        y[base + i] = a + b;
        y[base + i + h] = a - b;
      }
  }
  double r = 1.0 / sqrt((double)D);
  for (int i = 0; i < D; ++i) y[i] *= r;
}

void ora_rope_rot_f32(const ora_rope_cfg* c, const uint16_t* x_bits, float* y) {
  const int D = c->D, P = D / 2;
  float* tmp = (float*)malloc(sizeof(float) * D);
  for (int n = 0; n < c->N; ++n) {
    const uint16_t* x = x_bits + (size_t)n * D;
    float* yn = y + (size_t)n * D;
    for (int p = 0; p < P; ++p) {
      double G[4];
      ora_rope_block(c, n, p, G);
      float g00 = (float)G[0], g01 = (float)G[1], g10 = (float)G[2], g11 = (float)G[3];
      float x0 = in16_to_f32(x[2 * p], c->in_fp16), x1 = in16_to_f32(x[2 * p + 1], c->in_fp16);
      tmp[2 * p] = fmaf(x1, g10, x0 * g00);
      tmp[2 * p + 1] = fmaf(x1, g11, x0 * g01);
    }
    if (c->rotation == ORA_ROT_HALF) {
      /* Sec. 4.1.3: in segment j (offset o, width D_j) channel o+i pairs with
       * o+i+D_j/2; Pi places the pair at (o+2i, o+2i+1); R^j_i acts on it. */
      int o = 0;
      for (int ax = 0; ax < 3; ++ax) {
        int h = c->split[ax] / 2;
        for (int i = 0; i < h; ++i) {
          double R[4];
          rot_block(c, o / 2 + i, R);
          float r00 = (float)R[0], r01 = (float)R[1], r10 = (float)R[2], r11 = (float)R[3];
          float av = tmp[o + i], bv = tmp[o + i + h];
          yn[o + 2 * i] = fmaf(bv, r10, av * r00);
          yn[o + 2 * i + 1] = fmaf(bv, r11, av * r01);
        }
        o += c->split[ax];
      }
    } else {
      memcpy(yn, tmp, sizeof(float) * D);
      if (c->rotation == ORA_ROT_HADAMARD) ora_hadamard_f32(yn, D);
    }
  }
  free(tmp);
}

void ora_rope_rot_f64(const ora_rope_cfg* c, const uint16_t* x_bits, double* y) {
  const int D = c->D, P = D / 2;
  double* tmp = (double*)malloc(sizeof(double) * D);
  for (int n = 0; n < c->N; ++n) {
    const uint16_t* x = x_bits + (size_t)n * D;
    double* yn = y + (size_t)n * D;
    for (int p = 0; p < P; ++p) {
      double G[4];
      ora_rope_block(c, n, p, G);
      double x0 = in16_to_f32(x[2 * p], c->in_fp16), x1 = in16_to_f32(x[2 * p + 1], c->in_fp16);
      tmp[2 * p] = x0 * G[0] + x1 * G[2];
      tmp[2 * p + 1] = x0 * G[1] + x1 * G[3];
    }
    if (c->rotation == ORA_ROT_HALF) {
      int o = 0;
      for (int ax = 0; ax < 3; ++ax) {
        int h = c->split[ax] / 2;
        for (int i = 0; i < h; ++i) {
          double R[4];
          rot_block(c, o / 2 + i, R);
          double av = tmp[o + i], bv = tmp[o + i + h];
          yn[o + 2 * i] = av * R[0] + bv * R[2];
          yn[o + 2 * i + 1] = av * R[1] + bv * R[3];
        }
        o += c->split[ax];
      }
    } else {
      memcpy(yn, tmp, sizeof(double) * D);
      if (c->rotation == ORA_ROT_HADAMARD) ora_hadamard_f64(yn, D);
    }
  }
  free(tmp);
}

/* ----------------------------------------------------------- smoothing -- */

void ora_mean_fixed(const float* y, int N, int D, float* mu) {
  const float lim = 4294967296.0f; /* 2^32 */
  for (int ch = 0; ch < D; ++ch) {
    double s = 0.0; /* every partial sum is an integer below 2^53: exact */
    for (int n = 0; n < N; ++n) {
      float t = y[(size_t)n * D + ch] * 1048576.0f; /* exact scaling by 2^20 */
      if (t > lim) t = lim;
      if (t < -lim) t = -lim;
      s += (double)rintf(t);
    }
    mu[ch] = (float)(s / ((double)N * 1048576.0));
  }
}

void ora_center(const float* y, const float* mu, int N, int D, float* z) {
  for (int n = 0; n < N; ++n)
    for (int ch = 0; ch < D; ++ch) z[(size_t)n * D + ch] = y[(size_t)n * D + ch] - mu[ch];
}

/* Sec. 4 Q smoothing: with Q = Q_s + 1 mu_Q^T the scores split as
 * Q K^T = Q_s K^T + 1 (K mu_Q)^T, so every key j carries the additive score
 * bias b_j = mu_Q . K_j (K after RoPE, rotation and its own smoothing), which
 * is the same for all queries and stays in binary32 beside the INT4 scores.
 * The dot product is summed pairwise: the two halves of the channel range
 * recursively, with the products fl(mu_c k_c) at the leaves. */
static float pairwise_sum(const float* p, int n) {
  if (n == 1) return p[0];
  return pairwise_sum(p, n / 2) + pairwise_sum(p + n / 2, n / 2);
}

void ora_key_bias(const float* mu_q, const float* zk, int N, int D, float* bias) {
  float* p = (float*)malloc(sizeof(float) * D);
  for (int n = 0; n < N; ++n) {
    for (int ch = 0; ch < D; ++ch) p[ch] = mu_q[ch] * zk[(size_t)n * D + ch];
    bias[n] = pairwise_sum(p, D);
  }
  free(p);
}

/* -------------------------------------------------------- quantization -- */

static int8_t qcode(float z, float inv) {
  float t = rintf(z * inv);
  if (t > 7.0f) t = 7.0f;
  if (t < -7.0f) t = -7.0f;
  return (int8_t)t;
}

void ora_quant_tokens(const float* z, int N, int D, int g, int8_t* codes, float* scales) {
  int ng = (N + g - 1) / g;
  for (int gi = 0; gi < ng; ++gi) {
    int n0 = gi * g, n1 = n0 + g < N ? n0 + g : N;
    float amax = 0.0f;
    for (int n = n0; n < n1; ++n)
      for (int ch = 0; ch < D; ++ch) amax = fmaxf(amax, fabsf(z[(size_t)n * D + ch]));
    float s = 0.0f, inv = 0.0f;
    if (amax > 0.0f) {
      s = amax / 7.0f;
      inv = 7.0f / amax;
    }
    scales[gi] = s;
    for (int n = n0; n < n1; ++n)
      for (int ch = 0; ch < D; ++ch) codes[(size_t)n * D + ch] = qcode(z[(size_t)n * D + ch], inv);
  }
}

void ora_quant_v(const float* z, int N, int D, int g, int8_t* codes, float* scales) {
  int ng = (N + g - 1) / g;
  for (int gi = 0; gi < ng; ++gi) {
    int n0 = gi * g, n1 = n0 + g < N ? n0 + g : N;
    for (int ch = 0; ch < D; ++ch) {
      float amax = 0.0f;
      for (int n = n0; n < n1; ++n) amax = fmaxf(amax, fabsf(z[(size_t)n * D + ch]));
      float s = 0.0f, inv = 0.0f;
      if (amax > 0.0f) {
        s = amax / 7.0f;
        inv = 7.0f / amax;
      }
      scales[(size_t)gi * D + ch] = s;
      for (int n = n0; n < n1; ++n) codes[(size_t)n * D + ch] = qcode(z[(size_t)n * D + ch], inv);
    }
  }
}

/* ------------------------------------------------------------- attention -- */

float ora_exp2_f32(float x) { return (float)exp2((double)x); }

/* Sec. 4.2: P~ = (P / max P) * 15 - 8 with max P = 1 (online-softmax P lies in
 * (0, 1]); rounding to nearest, ties to even.  The stored code is u = P~ + 8.
 * The symmetric baseline rounds P * 7 onto [0, 7]. */
int ora_pcode(float P, int p_quant) {
  float t = rintf((p_quant == ORA_PQ_SYM7 ? 7.0f : 15.0f) * P);
  float hi = p_quant == ORA_PQ_SYM7 ? 7.0f : 15.0f;
  if (t > hi) t = hi;
  if (t < 0.0f) t = 0.0f;
  return (int)t;
}

static double sigma_of(double sm_scale, int D) { return sm_scale > 0.0 ? sm_scale : 1.0 / sqrt((double)D); }

void ora_attn_int4(const ora_attn_cfg* a,
                   const int8_t* qc, const float* qs,
                   const int8_t* kc, const float* ks,
                   const int8_t* vc, const float* vs, const float* mu_v, const float* bias,
                   int row0, int nrows, double* O,
                   int32_t* S_dump, uint8_t* u_dump, float* x_dump, float* m_dump,
                   double* l_dump) {
  const int N = a->N, D = a->D, kv = a->kv_block;
  const int nblocks = (N + kv - 1) / kv;
  /* log2(e) folded into the score scale so that P = 2^x (same value as e^(S/sqrt D - m)) */
  const float Kc = (float)(sigma_of(a->sm_scale, D) * LOG2E);
  const float pdiv = a->p_quant == ORA_PQ_SYM7 ? 7.0f : 15.0f;

#pragma omp parallel
  {
    int32_t* S = (int32_t*)malloc(sizeof(int32_t) * kv);
    float* cn = (float*)malloc(sizeof(float) * kv);
    float* t = (float*)malloc(sizeof(float) * kv);
    double* acc = (double*)malloc(sizeof(double) * D);
    double* part = (double*)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < nrows; ++r) {
      const int i = row0 + r;
      const int8_t* q = qc + (size_t)i * D;
      const float cq = qs[i / a->q_group] * Kc;
      float m = -INFINITY;
      double l = 0.0;
      for (int ch = 0; ch < D; ++ch) acc[ch] = 0.0;
      for (int j = 0; j < nblocks; ++j) {
        const int j0 = j * kv, j1 = j0 + kv < N ? j0 + kv : N;
        /* S_ij = Q_i K_j^T on the integer codes; block row maximum of the
         * dequantised, log2e-scaled scores. */
        float bm = -INFINITY;
        for (int n = j0; n < j1; ++n) {
          const int8_t* k = kc + (size_t)n * D;
          int32_t s = 0;
          for (int ch = 0; ch < D; ++ch) s += (int32_t)q[ch] * (int32_t)k[ch];
          S[n - j0] = s;
          cn[n - j0] = cq * ks[n / a->k_group];
          /* with Q smoothing the key's bias, on the same log2e-scaled scale,
           * joins the dequantised score in one fused step */
          t[n - j0] = bias ? fmaf((float)s, cn[n - j0], bias[n] * Kc) : (float)s * cn[n - j0];
          bm = fmaxf(bm, t[n - j0]);
          if (S_dump) S_dump[(size_t)r * N + n] = s;
        }
        /* m_ij = max(m_{i,j-1}, rowmax S_ij); rescale the running sums. */
        const float mn = fmaxf(m, bm);
        const float alpha = (m == -INFINITY) ? 0.0f : ora_exp2_f32(m - mn);
        l *= (double)alpha;
        for (int ch = 0; ch < D; ++ch) acc[ch] *= (double)alpha;
        if (m_dump) m_dump[(size_t)r * nblocks + j] = mn;
        m = mn;
        /* P_ij = exp(S_ij - m_ij), quantised; PV on the integer codes, one V
         * scale group at a time. */
        for (int ch = 0; ch < D; ++ch) part[ch] = 0.0;
        int gcur = j0 / a->v_group;
        for (int n = j0; n < j1; ++n) {
          const float x = bias ? t[n - j0] - mn : fmaf((float)S[n - j0], cn[n - j0], -mn);
          const float P = ora_exp2_f32(x);
          if (!a->l_quant || a->p_quant == ORA_PQ_NONE) l += (double)P;
          if (x_dump) x_dump[(size_t)r * N + n] = x;
          int g = n / a->v_group;
          if (g != gcur) {
            for (int ch = 0; ch < D; ++ch) {
              float dq = a->p_quant == ORA_PQ_NONE ? vs[(size_t)gcur * D + ch] : vs[(size_t)gcur * D + ch] / pdiv;
              acc[ch] += (double)dq * part[ch];
              part[ch] = 0.0;
            }
            gcur = g;
          }
          const int8_t* v = vc + (size_t)n * D;
          if (a->p_quant == ORA_PQ_NONE) {
            for (int ch = 0; ch < D; ++ch) part[ch] += (double)P * (double)v[ch];
            if (u_dump) u_dump[(size_t)r * N + n] = 0;
          } else {
            const int u = ora_pcode(P, a->p_quant);
            if (a->l_quant) l += (double)u / (double)pdiv;
            if (u_dump) u_dump[(size_t)r * N + n] = (uint8_t)u;
            for (int ch = 0; ch < D; ++ch) part[ch] += (double)(u * (int32_t)v[ch]);
          }
        }
        for (int ch = 0; ch < D; ++ch) {
          float dq = a->p_quant == ORA_PQ_NONE ? vs[(size_t)gcur * D + ch] : vs[(size_t)gcur * D + ch] / pdiv;
          acc[ch] += (double)dq * part[ch];
        }
      }
      if (l_dump) l_dump[r] = l;
      for (int ch = 0; ch < D; ++ch) O[(size_t)r * D + ch] = acc[ch] / l + (mu_v ? (double)mu_v[ch] : 0.0);
    }
    free(S);
    free(cn);
    free(t);
    free(acc);
    free(part);
  }
}

void ora_attn_ref_f64(const double* q, const double* k, const double* v, int N, int D,
                      double sm_scale, int row0, int nrows, double* O) {
  const double sg = sigma_of(sm_scale, D);
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * N);
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < nrows; ++r) {
      const double* qi = q + (size_t)(row0 + r) * D;
      double mx = -INFINITY;
      for (int n = 0; n < N; ++n) {
        double t = 0.0;
        for (int ch = 0; ch < D; ++ch) t += qi[ch] * k[(size_t)n * D + ch];
        s[n] = t * sg;
        if (s[n] > mx) mx = s[n];
      }
      double l = 0.0;
      for (int n = 0; n < N; ++n) {
        s[n] = exp(s[n] - mx);
        l += s[n];
      }
      for (int ch = 0; ch < D; ++ch) {
        double t = 0.0;
        for (int n = 0; n < N; ++n) t += s[n] * v[(size_t)n * D + ch];
        O[(size_t)r * D + ch] = t / l;
      }
    }
    free(s);
  }
}

void ora_attn_fb16(const uint16_t* qb, const uint16_t* kb, const uint16_t* vb, int N, int D,
                   int kv_block, double sm_scale, int fp16, int row0, int nrows, double* O) {
  const double c = sigma_of(sm_scale, D) * LOG2E;
  const int kv = kv_block;
#pragma omp parallel
  {
    double* t = (double*)malloc(sizeof(double) * kv);
    double* acc = (double*)malloc(sizeof(double) * D);
#pragma omp for schedule(dynamic, 1)
    for (int r = 0; r < nrows; ++r) {
      const uint16_t* qi = qb + (size_t)(row0 + r) * D;
      double m = -INFINITY, l = 0.0;
      for (int ch = 0; ch < D; ++ch) acc[ch] = 0.0;
      for (int j0 = 0; j0 < N; j0 += kv) {
        int j1 = j0 + kv < N ? j0 + kv : N;
        double bm = -INFINITY;
        for (int n = j0; n < j1; ++n) {
          double s = 0.0;
          for (int ch = 0; ch < D; ++ch)
            s += (double)in16_to_f32(qi[ch], fp16) * (double)in16_to_f32(kb[(size_t)n * D + ch], fp16);
          t[n - j0] = s * c;
          if (t[n - j0] > bm) bm = t[n - j0];
        }
        double mn = m > bm ? m : bm;
        double alpha = (m == -INFINITY) ? 0.0 : exp2(m - mn);
        l *= alpha;
        for (int ch = 0; ch < D; ++ch) acc[ch] *= alpha;
        for (int n = j0; n < j1; ++n) {
          double P = exp2(t[n - j0] - mn);
          l += P;
          /* the PV product sees P rounded to the 16-bit type (through binary32) */
          double Pr = in16_to_f32(f32_to_16((float)P, fp16), fp16);
          for (int ch = 0; ch < D; ++ch) acc[ch] += Pr * (double)in16_to_f32(vb[(size_t)n * D + ch], fp16);
        }
        m = mn;
      }
      for (int ch = 0; ch < D; ++ch) O[(size_t)r * D + ch] = acc[ch] / l;
    }
    free(t);
    free(acc);
  }
}

void ora_attn_bf16(const uint16_t* qb, const uint16_t* kb, const uint16_t* vb, int N, int D,
                   int kv_block, double sm_scale, int row0, int nrows, double* O) {
  ora_attn_fb16(qb, kb, vb, N, D, kv_block, sm_scale, 0, row0, nrows, O);
}
