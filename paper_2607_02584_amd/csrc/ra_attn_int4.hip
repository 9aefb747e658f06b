// ra_attn_int4.hip -- INT4 FlashAttention forward on the int8 matrix core (gfx950).
//
// Computes, per head and query row i, the blockwise online softmax of the
// paper's Sec. 4.2 over blocks of KV keys in ascending order:
//   S_ij   = Q~_i K~_j^T                      (exact int32 on the i8 matrix core)
//   m_ij   = max(m_i,j-1, rowmax fl(S * c)),  c = fl(fl(s_q * Kc) * s_k)
//   pscale P = 2^fma(S, c, -(m_ij - log2 pscale))   (pscale = 15, or 7 for SYM7;
//                                              Kc folds 1/sqrt(D) and log2 e)
//   u      = rint(pscale P) in [0, 15]        (Range-optimized P, Sec. 4.2.1:
//                                              P~ = u - 8, fixed scale 15)
//   l      = alpha * l + sum pscale P,  alpha = 2^(m_i,j-1 - m_ij)
//   O      = alpha * O + sum_g fl(s_v[g]/pscale) * (u . V~)
// and writes O * pscale / l + mu_v.  The P scale rides in the exponent (one
// exponential per score, no multiply); the binary32 rounding of
// m - log2 pscale perturbs pscale P by a relative ln 2 * 2^-24 (|m| + 6) at
// most.  With Q smoothing every key j carries the score bias fl(b_j Kc):
// t = fma(S, c, bias_j) replaces fl(S c) in the maximum and the exponent is
// t - (m - log2 pscale).
//
// Matrix-core mapping (v_mfma_i32_32x32x32_i8, one wave = 32 queries):
//   S^T = K Q^T : A = K tile (32 keys x 32 channels), B = Q^T, so every lane
//                 holds 16 keys of ONE query: the row max and sum need no
//                 cross-lane work except one exchange between the wave halves.
//                 The int32 scores are converted to binary32 once (exact).
//   O^T = V^T P^T: B = P^T comes straight from the S^T accumulator lanes (the
//                 P codes of a lane are the B operand of that lane), A = V^T
//                 read from LDS; the V codes are stored with the key order the
//                 accumulator layout implies, so no register shuffle is needed.
//                 A lane holds one query of the output tile, so alpha is the
//                 lane's own (applied only when some row of the wave moved its
//                 maximum); each block's int32 product is converted and scaled
//                 by its V group's per-channel factor into the binary32 O.
// K and V codes arrive packed (two per byte); a workgroup stages them in LDS,
// expanding each nibble c to the int8 value 16c with two bit operations per
// four codes (the factor 16 is folded into the scales, which is exact).  Q is
// expanded once per wave to plain int8 codes.  Two workgroups of four waves
// share a compute unit.  The next block's score products run beside this
// block's PV conversion (software pipeline), so K is staged two blocks ahead.
#include <type_traits>

#include "ra_internal.h"
#include "ra_xcd.h"

namespace ra {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBlockM = 128;  // queries per workgroup (4 waves x 32)

// nibbles at bits 0-3 of each byte, sign-extended to int8 codes
__device__ __forceinline__ uint32_t sext_lo(uint32_t w) {
  const uint32_t u = w & 0x0F0F0F0Fu;
  return u | ((u & 0x08080808u) * 30u);
}
// nibbles at bits 4-7 of each byte, sign-extended to int8 codes
__device__ __forceinline__ uint32_t sext_hi(uint32_t w) {
  const uint32_t u = (w >> 4) & 0x0F0F0F0Fu;
  return u | ((u & 0x08080808u) * 30u);
}

// 8 packed bytes -> 16 int8 values 16*code, order [lo(w0) hi(w0) lo(w1) hi(w1)]
__device__ __forceinline__ uint4 expand16(uint2 w) {
  return make_uint4((w.x << 4) & 0xF0F0F0F0u, w.x & 0xF0F0F0F0u, (w.y << 4) & 0xF0F0F0F0u, w.y & 0xF0F0F0F0u);
}

// A lane carries 8-byte pieces of the packed block (KV/32 of K, KV/32 of V):
// piece i of lane tid is packed bytes (i*256 + tid)*8 .. +7, which expand to
// the 16 int8 bytes at twice that offset, so each LDS store of a wave covers
// 1 KB contiguously (no bank conflicts).
template <int KV>
struct Stage {
  uint2 k[KV / 32];
  uint2 v[KV / 32];
};

// the packed K codes of block jk and the packed V codes of block jv
template <int KV>
__device__ __forceinline__ void stage_load(const AttnArgs& a, int bh, int jk, int jv, Stage<KV>& st) {
  const int tid = threadIdx.x;
  const uint8_t* kb = a.kc + static_cast<size_t>(bh) * a.Npad * 64 + static_cast<size_t>(jk) * KV * 64;
  const uint8_t* vb = a.vc + static_cast<size_t>(bh) * a.Npad * 64 + static_cast<size_t>(jv) * KV * 64;
#pragma unroll
  for (int i = 0; i < KV / 32; ++i) {
    st.k[i] = *reinterpret_cast<const uint2*>(kb + (i * 256 + tid) * 8);
    st.v[i] = *reinterpret_cast<const uint2*>(vb + (i * 256 + tid) * 8);
  }
}

// LDS int8 offset = 2 x packed offset (each 8-byte piece expands to 16 bytes)
template <int KV>
__device__ __forceinline__ void stage_store(const Stage<KV>& st, uint8_t* sk, uint8_t* sv) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < KV / 32; ++i) {
    const int o = (i * 256 + tid) * 16;
    *reinterpret_cast<uint4*>(sk + o) = expand16(st.k[i]);
    *reinterpret_cast<uint4*>(sv + o) = expand16(st.v[i]);
  }
}

// QB: Q smoothing, every key carries the score bias fl(b_j Kc).
// LQ: the normaliser sums the codes u (l = sum of P^) instead of pscale P.
template <int KV, bool KTOK, bool SYM7, bool DEBUG, bool QB, bool LQ>
__global__ __launch_bounds__(256, 2) void k_attn_int4(AttnArgs a) {
  constexpr int NCH = KV / 32;
  __shared__ __align__(16) uint8_t sK[2][KV * 128];
  __shared__ __align__(16) uint8_t sV[2][KV * 128];
  __shared__ __align__(16) float sDq[2][kD];
  __shared__ __align__(16) float sKs[2][KTOK ? KV : 1];
  __shared__ __align__(16) float sKc[2][NCH];          // K scale of each 32-key chunk (grouped K)
  __shared__ __align__(16) float sB[2][QB ? KV : 1];   // per-key score bias fl(b Kc)

  // the wave index is uniform: conditions on it are scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5, j = lane & 31;
  int bh, qtile;
  xcd_tile(bh, qtile);
  const int qrow = qtile * kBlockM + wave * 32 + j;
  const int N = a.N;
  const int nblocks = (N + KV - 1) / KV;
  const int kstride = a.Npad / a.k_group;
  constexpr float pscale = SYM7 ? 7.0f : 15.0f;
  // log2 of the P scale: pscale P = 2^(S c - (m - log2 pscale)), one exponential per score
  constexpr float kLog2P = SYM7 ? 2.80735492205760410f : 3.90689059560851852f;

  // ---- Q operand: plain int8 codes in the order of the K expansion ----
  v4i qop[4];
  {
    const uint8_t* qp = a.qc + static_cast<size_t>(bh) * a.Npad * 64 + static_cast<size_t>(qrow >> 5) * 2048 +
                        (qrow & 31) * 8;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const uint2 w = *reinterpret_cast<const uint2*>(qp + (2 * kc + hh) * 256);
      qop[kc] = v4i{static_cast<int>(sext_lo(w.x)), static_cast<int>(sext_hi(w.x)), static_cast<int>(sext_lo(w.y)),
                    static_cast<int>(sext_hi(w.y))};
    }
  }
  const float cq = __fmul_rn(a.qs[static_cast<size_t>(bh) * (a.Npad / a.q_group) + qrow / a.q_group], a.Kc);

  // Per-block side data in LDS: V dequantization factors fl(s_v / pscale) / 16
  // (exact /16) of the block's group, the K scales (per 32-key chunk or per
  // key) and, with Q smoothing, the per-key bias.
  // Waves 0 and 1 (thread = channel) stage the V factors; thread 128 + t
  // stages key t of the block (waves 2 and 3, or wave 2 alone for 64-key
  // blocks), or the K scale of chunk t (grouped K: k_group is 32, 64 or 128,
  // so the group index is a shift).  stage_aux runs for blocks 0, 1, 2, ... in
  // order; (vg, vgr) = (V group, block within it) of the next block it stages.
  const bool kwave = KV == 128 ? wave >= 2 : wave == 2;
  const int kgs = __builtin_ctz(static_cast<unsigned>(a.k_group));
  int vg = 0, vgr = 0;
  auto stage_aux = [&](int jb, int buf) {
    if (wave < 2) {
      const float s = a.vs[(static_cast<size_t>(bh) * a.nvgroups + vg) * kD + tid];
      sDq[buf][tid] = __fmul_rn(__fdiv_rn(s, pscale), 0.0625f);
    }
    if (++vgr == a.v_bpg) {
      vgr = 0;
      ++vg;
    }
    const int kt = tid - kD;
    if (KTOK) {
      if (kwave) sKs[buf][kt] = a.ks[static_cast<size_t>(bh) * kstride + ((jb * KV + kt) >> kgs)];
    } else if (wave == 2 && lane < NCH) {
      sKc[buf][kt] = a.ks[static_cast<size_t>(bh) * kstride + ((jb * KV + kt * 32) >> kgs)];
    }
    if (QB && kwave) sB[buf][kt] = __fmul_rn(a.kbias[static_cast<size_t>(bh) * a.Npad + jb * KV + kt], a.Kc);
  };

  float of[4][16];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) of[mt][r] = 0.f;
  // running maximum m and row sum l of pscale P (LQ: of the codes u)
  float m = -INFINITY, l = 0.f;

  // Software pipeline over blocks: a block's score products run while the
  // previous block's PV products are converted (matrix core and vector unit
  // side by side), so a block starts with its scores in registers.  K tiles
  // are therefore staged two blocks ahead and V tiles one block ahead: block
  // j + 2's K goes where block j's K was (its scores were taken during block
  // j - 1), block j + 1's V where block j - 1's V was; two LDS buffers each.
  auto blk = [&](int b) { return b < nblocks ? b : nblocks - 1; };
  Stage<KV> st;
  stage_load<KV>(a, bh, 0, 0, st);
  stage_store<KV>(st, sK[0], sV[0]);
  stage_load<KV>(a, bh, blk(1), blk(1), st);
  stage_store<KV>(st, sK[1], sV[1]);
  stage_aux(0, 0);
  __syncthreads();

  // S^T = K Q^T of one 32-key chunk of the K tile kt (int32, 16 x the exact S)
  v16i si[NCH];
  auto score_chunk = [&](const uint8_t* kt, int ch) {
    si[ch] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int kc = 0; kc < 4; ++kc) {
      const v4i A = *reinterpret_cast<const v4i*>(&kt[(((ch * 8) + 2 * kc + hh) * 32 + j) * 16]);
      si[ch] = __builtin_amdgcn_mfma_i32_32x32x32_i8(A, qop[kc], si[ch], 0, 0, 0);
    }
  };
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch) score_chunk(sK[0], ch);
  stage_load<KV>(a, bh, blk(2), blk(1), st);
  __syncthreads();   // every wave has read block 0's K before it is overwritten

  // One block of KV keys; MASKED (keys past N) only for the last block (a full
  // last block masks nothing).  MORE: a next block exists; as a template
  // argument it keeps the product phase one basic block.
  auto step = [&](int jb, auto masked_tag, auto more_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool more = decltype(more_tag)::value;
    // Issue priority: the first half of the block (scores to binary32,
    // maximum, alpha, every probability and code, the first output tile's
    // products) is a dependent chain of vector work, the rest mostly
    // matrix-core products; with the chain at the higher priority the two
    // waves of a SIMD alternate halves (4.32 -> 4.24 ms on the 32760-token
    // layer).
    __builtin_amdgcn_s_setprio(1);
    const int buf = jb & 1;
    const int key0 = jb * KV;
    // key of accumulator register r in chunk ch: key0 + ch*32 + 8*(r/4) + 4*hh + r%4
    auto is_out = [&](int ch, int r) { return MASKED && key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3) >= N; };

    // ---- the block's int32 scores, kept as binary32 (exact: |16 S| <= 16 * 6272 < 2^24) ----
    float s[NCH][16];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[ch][r] = static_cast<float>(si[ch][r]);
    if (DEBUG) {
      if (bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows && a.dbg_s) {
        const size_t rowo = static_cast<size_t>(qrow - a.dbg_row0);
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
            if (key < N) a.dbg_s[rowo * N + key] = static_cast<int32_t>(s[ch][r]) >> 4;
          }
      }
    }

    // ---- block row maximum: of fl(S c) (c >= 0: fl(max S * c)), or of
    //      t = fma(S, c, bias) with Q smoothing; 16 S * c/16 == S * c exactly ----
    float cch[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) cch[ch] = KTOK ? 0.f : __fmul_rn(__fmul_rn(cq, sKc[buf][ch]), 0.0625f);
    auto ckey = [&](int ch, int r) {
      const int kl = ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
      return KTOK ? __fmul_rn(__fmul_rn(cq, sKs[buf][kl]), 0.0625f) : cch[ch];
    };
    float tmax = -INFINITY;
    if (QB || KTOK) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kl = ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
          const float sf = s[ch][r];
          float t = QB ? __fmaf_rn(sf, ckey(ch, r), sB[buf][kl]) : __fmul_rn(sf, ckey(ch, r));
          if (is_out(ch, r)) t = -INFINITY;
          tmax = fmaxf(tmax, t);
        }
    } else {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, is_out(ch, r) ? -INFINITY : s[ch][r]);
        // a fully masked chunk gives -inf (or NaN when c == 0), which fmax ignores
        tmax = fmaxf(tmax, __fmul_rn(mx, cch[ch]));
      }
    }
    tmax = max_halves(tmax);
    const float mnew = fmaxf(m, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    const float mq = __fsub_rn(mnew, kLog2P);

    // ---- pscale P from the exponential, codes u = rint(pscale P) (the B
    //      operand of O^T = V^T P^T straight from this lane), row sums ----
    uint32_t pk[NCH][4];
    float ls[4];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t word = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int r = 4 * q + t;
          const float sf = s[ch][r];
          float x;
          if (QB) {
            const int kl = ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
            x = __fsub_rn(__fmaf_rn(sf, ckey(ch, r), sB[buf][kl]), mq);
          } else {
            x = __fmaf_rn(sf, ckey(ch, r), -mq);
          }
          float P = __builtin_amdgcn_exp2f(x);   // pscale * P
          if (is_out(ch, r)) P = 0.f;
          const float lv = LQ ? __builtin_rintf(P) : P;
          if (ch == 0 && q == 0) ls[t] = lv;
          else ls[t] += lv;
          word = __builtin_amdgcn_cvt_pk_u8_f32(P, t, word);
        }
        pk[ch][q] = word;
      }
    }
    l = __fmaf_rn(l, alpha, (ls[0] + ls[1]) + (ls[2] + ls[3]));

    if (DEBUG) {
      if (bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows) {
        const size_t rowo = static_cast<size_t>(qrow - a.dbg_row0);
        if (a.dbg_u) {
#pragma unroll
          for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
              if (key < N) a.dbg_u[rowo * N + key] = static_cast<uint8_t>((pk[ch][r >> 2] >> (8 * (r & 3))) & 0xFF);
            }
        }
        if (a.dbg_m && hh == 0) a.dbg_m[rowo * nblocks + jb] = mnew;
      }
    }

    // block j + 2's K and block j + 1's V go to LDS here, so the staging
    // registers die early
    stage_store<KV>(st, sK[buf], sV[buf ^ 1]);
    if (more) stage_aux(jb + 1, buf ^ 1);
    // ---- O^T += V^T P^T (int32 per block), then O = alpha O + acc * dq; the
    //      alpha rescale only when some row of the wave moved its maximum ----
    if (__ballot(alpha != 1.0f) != 0) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) of[mt][r] = __fmul_rn(of[mt][r], alpha);
    }
    // the products of output tile mt (and the next block's scores of chunk mt)
    // run beside the conversion of tile mt - 1 (a quarter of it after every
    // second product), all in one scheduling region
    v16i acc[2];
    auto convert_q = [&](int mt, int rq) {   // registers 4 rq .. 4 rq + 3 of tile mt
      const float4 dq = *reinterpret_cast<const float4*>(&sDq[buf][mt * 32 + 8 * rq + 4 * hh]);
      const float d4[4] = {dq.x, dq.y, dq.z, dq.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int r = 4 * rq + t;
        of[mt][r] = __fmaf_rn(static_cast<float>(acc[mt & 1][r]), d4[t], of[mt][r]);
      }
    };
    // region g = 8 mt + i: i < NCH the PV product of tile mt with chunk i;
    // 4 <= i < 8 (more, mt < NCH) the next block's score product of chunk mt,
    // channel quarter i - 4; its A operand is read from LDS two regions ahead
    const uint8_t* kn = sK[buf ^ 1];
    auto has = [&](int g) {
      const int mt = g >> 3, i = g & 7;
      return i < NCH || (more && i >= 4 && mt < NCH);
    };
    auto opA = [&](int g) {
      const int mt = g >> 3, i = g & 7;
      if (i < NCH) return *reinterpret_cast<const v4i*>(&sV[buf][((i * 2 + hh) * 128 + mt * 32 + j) * 16]);
      return *reinterpret_cast<const v4i*>(&kn[(((mt * 8) + 2 * (i - 4) + hh) * 32 + j) * 16]);
    };
    const v16i zero16 = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    v4i a0 = opA(0), a1 = opA(1);
#pragma unroll
    for (int g = 0; g < 32; ++g) {
      const int mt = g >> 3, i = g & 7;
      // the operand two products ahead
      int g2 = g + 1;
      while (g2 < 32 && !has(g2)) ++g2;
      int g3 = g2 + 1;
      while (g3 < 32 && !has(g3)) ++g3;
      if (has(g)) {
        const v4i an = g3 < 32 ? opA(g3) : a0;
        if (i < NCH) {
          const v4i B = v4i{static_cast<int>(pk[i][0]), static_cast<int>(pk[i][1]), static_cast<int>(pk[i][2]),
                            static_cast<int>(pk[i][3])};
          acc[mt & 1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, B, i == 0 ? zero16 : acc[mt & 1], 0, 0, 0);
        } else {
          const int kc = i - 4;
          si[mt] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, qop[kc], kc == 0 ? zero16 : si[mt], 0, 0, 0);
        }
        a0 = a1;
        a1 = an;
      }
      if (mt > 0 && (i & 1)) convert_q(mt - 1, i >> 1);
      if (g == 7) __builtin_amdgcn_s_setprio(0);

    }
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) convert_q(3, rq);
    if (more) stage_load<KV>(a, bh, blk(jb + 3), blk(jb + 2), st);
    __syncthreads();
  };

  using kNo = std::integral_constant<bool, false>;
  using kYes = std::integral_constant<bool, true>;
  for (int jb = 0; jb + 1 < nblocks; ++jb) step(jb, kNo(), kYes());
  step(nblocks - 1, kYes(), kNo());

  // ---- epilogue: O = O' pscale / l + mu_v (rotated back by H when V was
  //      rotated online); l is pscale * sum P, or the sum of the codes ----
  const float ltot = l + __shfl_xor(l, 32);
  {
    const float inv = pscale / ltot;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int c = mt * 32 + 8 * rq + 4 * hh + t;
          of[mt][4 * rq + t] = of[mt][4 * rq + t] * inv;
          if (a.mu_v) of[mt][4 * rq + t] += a.mu_v[bh * kD + c];
        }
  }
  if (a.vhad) {
    // O = O' H^T = O' H per query row.  Element (mt, 4 rq + t) of lane half hh is
    // channel 32 mt + 8 rq + 4 hh + t: strides 64, 32 (mt), 16, 8 (rq), 2, 1 (t)
    // stay in the thread, stride 4 pairs the two lane halves.
    float* f = &of[0][0];
    auto level = [&](int st) {
#pragma unroll
      for (int i = 0; i < 64; ++i)
        if (!(i & st)) {
          const float x0 = f[i], x1 = f[i + st];
          f[i] = x0 + x1;
          f[i + st] = x0 - x1;
        }
    };
    level(32);
    level(16);
    level(8);
    level(4);
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      const float o = __shfl_xor(f[i], 32);
      f[i] = hh ? o - f[i] : f[i] + o;
    }
    level(2);
    level(1);
#pragma unroll
    for (int i = 0; i < 64; ++i) f[i] *= kInvSqrtD;
  }
  if (qrow < N) {
    const size_t obase = (static_cast<size_t>(bh) * N + qrow) * kD;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int c0 = mt * 32 + 8 * rq + 4 * hh;
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = of[mt][4 * rq + t];
        if (a.out_dtype == 2) {
          *reinterpret_cast<float4*>(static_cast<float*>(a.o) + obase + c0) = make_float4(v[0], v[1], v[2], v[3]);
        } else if (a.out_dtype == 0) {
          uint16_t b[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) b[t] = __bfloat16_as_ushort(__float2bfloat16(v[t]));
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.o) + obase + c0) =
              make_uint2(b[0] | (static_cast<uint32_t>(b[1]) << 16), b[2] | (static_cast<uint32_t>(b[3]) << 16));
        } else {
          uint16_t b[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) b[t] = __half_as_ushort(__float2half(v[t]));
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.o) + obase + c0) =
              make_uint2(b[0] | (static_cast<uint32_t>(b[1]) << 16), b[2] | (static_cast<uint32_t>(b[3]) << 16));
        }
      }
  }
}

template <int KV, bool KTOK, bool SYM7, bool DEBUG, bool QB, bool LQ>
hipError_t launch_l(const AttnArgs& a, hipStream_t s) {
  const dim3 grid(a.Npad / kBlockM, a.BH);
  hipLaunchKernelGGL((k_attn_int4<KV, KTOK, SYM7, DEBUG, QB, LQ>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int KV, bool KTOK, bool SYM7, bool DEBUG, bool QB>
hipError_t launch_b(const AttnArgs& a, hipStream_t s) {
  return a.lq ? launch_l<KV, KTOK, SYM7, DEBUG, QB, true>(a, s) : launch_l<KV, KTOK, SYM7, DEBUG, QB, false>(a, s);
}

template <int KV, bool KTOK, bool SYM7, bool DEBUG>
hipError_t launch_t(const AttnArgs& a, hipStream_t s) {
  return a.kbias ? launch_b<KV, KTOK, SYM7, DEBUG, true>(a, s) : launch_b<KV, KTOK, SYM7, DEBUG, false>(a, s);
}

template <int KV, bool KTOK, bool SYM7>
hipError_t launch_d(const AttnArgs& a, bool debug, hipStream_t s) {
  return debug ? launch_t<KV, KTOK, SYM7, true>(a, s) : launch_t<KV, KTOK, SYM7, false>(a, s);
}

template <int KV, bool KTOK>
hipError_t launch_p(const AttnArgs& a, bool sym7, bool debug, hipStream_t s) {
  return sym7 ? launch_d<KV, KTOK, true>(a, debug, s) : launch_d<KV, KTOK, false>(a, debug, s);
}

template <int KV>
hipError_t launch_k(const AttnArgs& a, bool ktok, bool sym7, bool debug, hipStream_t s) {
  return ktok ? launch_p<KV, true>(a, sym7, debug, s) : launch_p<KV, false>(a, sym7, debug, s);
}

}  // namespace

hipError_t launch_attn_int4(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, bool debug,
                            hipStream_t s) {
  if (kv_block == 64) return launch_k<64>(a, k_per_token, sym7, debug, s);
  return launch_k<128>(a, k_per_token, sym7, debug, s);
}

}  // namespace ra
