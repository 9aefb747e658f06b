// ra_attn_e2m3.hip -- INT4 FlashAttention forward on the FP6 matrix core (gfx950).
//
// Same computation as the int8 kernel (the paper's Sec. 4.2 blockwise online
// softmax with the Range-optimized P quantization over INT4 Q, K, V codes),
// but every INT4 code is carried as the 6-bit E2M3 float of the same value.
// E2M3 represents the integers -7..7 exactly, and u/8 for u = 0..15 with a
// uniform step (the subnormals and the first binade), and the E2M3 bit pattern
// of u/8 is the integer u itself.  The products and 64-term sums of the matrix
// core stay integer multiples of 1/8 far below 2^24, so
//   S  = Q~ K~^T                         is the exact integer score, and
//   O' += V~^T (u/8)                     is exact per block,
// on v_mfma_scale_f32_32x32x64_f8f6f4, which runs at twice the int8 rate and
// accumulates in binary32: PV accumulates straight into the output tile.
//
// Per block of KV keys (ascending):
//   m_new = max(m, rowmax fl(S * c)),  x = fma(S, c, -m_new),  P = 2^x,
//   u = rint(fl(15 P)),  l = alpha l + sum P,  alpha = 2^(m - m_new),
//   O' = O' * alpha * (w_old / w_new) + V~^T (u/8)   (w = V scale of the block's group)
// and finally O = O' * 8 w / 15 / l + mu_v.  The rounding u = rint(fl(15 P)) is
// done by the packing conversion itself: it converts fl(15 P) / 8 to E2M3 with
// round-to-nearest-even, and on the uniform 1/8 grid that is rint to an integer.
//
// Matrix-core mapping (one wave = 32 queries): S^T = K Q^T (A = 32 keys x 64
// channels of K, B = Q^T), so a lane holds 16 scores of one query per 32-key
// chunk.  The P codes of two chunks (64 keys) are packed by
// v_cvt_scalef32_2xpk16_fp6_f32 (which interleaves its two 16-value sources)
// into the B operand of O^T = V^T P^T; the V records are stored in the key
// order that packing produces.
#include <type_traits>

#include "ra_internal.h"

namespace ra {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v6i __attribute__((ext_vector_type(6)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kBlockM = 128;  // queries per workgroup (4 waves x 32)
constexpr int kScaleOne = 127;  // E8M0 block scale 2^0

__device__ __forceinline__ v16f mfma6(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 2, 2, 0, kScaleOne, 0, kScaleOne);
}

// 24-byte record -> operand registers (6 used dwords)
__device__ __forceinline__ v8i load_rec(const uint8_t* p) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  const uint2 b = *reinterpret_cast<const uint2*>(p + 8);
  const uint2 c = *reinterpret_cast<const uint2*>(p + 16);
  return v8i{static_cast<int>(a.x), static_cast<int>(a.y), static_cast<int>(b.x), static_cast<int>(b.y),
             static_cast<int>(c.x), static_cast<int>(c.y), 0, 0};
}

// Copies `bytes` (a multiple of 1024) from global to LDS with the LDS-DMA path
// (global_load_lds_dwordx4: lane i of a wave moves 16 bytes to base + 16 i);
// the four waves of the workgroup take every fourth kilobyte.
__device__ __forceinline__ void dma_copy(const uint8_t* src, uint8_t* dst, int bytes, int wave, int lane) {
  for (int off = wave * 1024; off < bytes; off += 4096) {
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)(src + off + lane * 16),
                                     (void __attribute__((address_space(3)))*)(dst + off), 16, 0, 0);
  }
}

template <int KV, bool KTOK, bool SYM7, bool DEBUG>
__global__ __launch_bounds__(256, 2) void k_attn_e2m3(AttnArgs a) {
  constexpr int NCH = KV / 32;   // 32-key chunks
  constexpr int NG = KV / 64;    // 64-key groups (one PV instruction each)
  constexpr int KB = KV * 96;    // bytes of K (and of V) codes per block
  __shared__ __align__(16) uint8_t sK[2][KB];
  __shared__ __align__(16) uint8_t sV[2][KB];
  __shared__ __align__(16) float sR[2][kD];   // V scale ratio w_old / w_new for the block
  __shared__ __align__(16) float sW[kD];      // final V scale per channel
  __shared__ __align__(16) float sKs[2][KTOK ? KV : 1];
  __shared__ __align__(16) float sKc[2][NCH];  // K scale of each 32-key chunk (grouped K)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, j = lane & 31;
  const int bh = blockIdx.y;
  const int qrow = blockIdx.x * kBlockM + wave * 32 + j;
  const int N = a.N;
  const int nblocks = (N + KV - 1) / KV;
  const int kstride = a.Npad / a.k_group;
  const float pscale = SYM7 ? 7.0f : 15.0f;
  const size_t hcode = static_cast<size_t>(bh) * a.Npad * 96;
  const uint8_t* kbase = a.kc + hcode;
  const uint8_t* vbase = a.vc + hcode;
  const float* ksh = a.ks + static_cast<size_t>(bh) * kstride;

  // ---- Q operand (B of S^T = K Q^T) ----
  v8i qop[2];
#pragma unroll
  for (int kc = 0; kc < 2; ++kc) {
    const int rec = (((qrow >> 5) * 2 + kc) * 2 + hh) * 32 + (qrow & 31);
    qop[kc] = load_rec(a.qc + hcode + static_cast<size_t>(rec) * 24);
  }
  const float cq = __fmul_rn(a.qs[static_cast<size_t>(bh) * (a.Npad / a.q_group) + qrow / a.q_group], a.Kc);

  // V scale bookkeeping: thread ch < 128 owns channel ch's working scale w.
  float wcur = 1.0f;
  auto stage_aux = [&](int jb, int buf) {
    if (tid < kD) {
      int g = (jb * KV) / a.v_group;
      if (g >= a.nvgroups) g = a.nvgroups - 1;
      const float s = a.vs[(static_cast<size_t>(bh) * a.nvgroups + g) * kD + tid];
      float r = 1.0f;
      if (s > 0.0f) {
        r = (jb == 0) ? 1.0f : __fdiv_rn(wcur, s);
        wcur = s;
      }
      sR[buf][tid] = r;
    }
    if (KTOK && tid < KV) sKs[buf][tid] = ksh[jb * KV + tid];
    if (!KTOK && tid >= kD && tid < kD + NCH) sKc[buf][tid - kD] = ksh[(jb * KV + (tid - kD) * 32) / a.k_group];
  };

  v16f of[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) of[mt][r] = 0.f;
  float m = -INFINITY, l = 0.f;

  dma_copy(kbase, sK[0], KB, wave, lane);
  dma_copy(vbase, sV[0], KB, wave, lane);
  stage_aux(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // One block of KV keys.  MASKED (keys past N) only for the partial last
  // block, which runs outside the main loop so the full blocks carry no masking.
  auto step = [&](int jb, auto masked_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    const int buf = jb & 1;
    const int key0 = jb * KV;
    if (jb + 1 < nblocks) {
      dma_copy(kbase + static_cast<size_t>(jb + 1) * KB, sK[buf ^ 1], KB, wave, lane);
      dma_copy(vbase + static_cast<size_t>(jb + 1) * KB, sV[buf ^ 1], KB, wave, lane);
      stage_aux(jb + 1, buf ^ 1);
    }
    __builtin_amdgcn_sched_barrier(0);

    // ---- S^T = K Q^T: exact integer scores in binary32; the operands of
    //      chunk ch+1 are read from LDS while chunk ch is on the matrix core ----
    v16f s[NCH];
    v8i kop0 = load_rec(&sK[buf][((0 * 2 + hh) * 32 + j) * 24]);
    v8i kop1 = load_rec(&sK[buf][((1 * 2 + hh) * 32 + j) * 24]);
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      v8i n0 = kop0, n1 = kop1;
      if (ch + 1 < NCH) {
        n0 = load_rec(&sK[buf][(((((ch + 1) * 2) + 0) * 2 + hh) * 32 + j) * 24]);
        n1 = load_rec(&sK[buf][(((((ch + 1) * 2) + 1) * 2 + hh) * 32 + j) * 24]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) s[ch][r] = 0.f;
      s[ch] = mfma6(kop0, qop[0], s[ch]);
      s[ch] = mfma6(kop1, qop[1], s[ch]);
      kop0 = n0;
      kop1 = n1;
      __builtin_amdgcn_sched_barrier(0);
    }
    // key of accumulator register r in chunk ch: key0 + 32*ch + 8*(r/4) + 4*hh + r%4
    if (MASKED) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3) >= N) s[ch][r] = -INFINITY;
    }

    // ---- block row maximum of fl(S * c) (c >= 0, so it is fl(max S * c);
    //      a fully masked chunk gives -inf, or NaN when c == 0, which fmax ignores) ----
    float cch[NCH];
    float tmax = -INFINITY;
    const bool vchange = jb > 0 && a.nvgroups > 1 && ((jb * KV) % a.v_group) == 0;
    float4 rr[4][4];
    if (vchange) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) rr[mt][rq] = *reinterpret_cast<const float4*>(&sR[buf][mt * 32 + 8 * rq + 4 * hh]);
    }
    if (!KTOK && a.k_group >= KV) {
      // one K scale for the whole block: a single product after the maximum
      float cm[NCH];
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        float mx = fmaxf(fmaxf(s[ch][0], s[ch][1]), s[ch][2]);
#pragma unroll
        for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, s[ch][r]), s[ch][r + 1]);
        cm[ch] = fmaxf(mx, s[ch][15]);
      }
      float mx = cm[0];
#pragma unroll
      for (int ch = 1; ch < NCH; ++ch) mx = fmaxf(mx, cm[ch]);
      const float c0 = __fmul_rn(cq, sKc[buf][0]);
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) cch[ch] = c0;
      tmax = __fmul_rn(mx, c0);
    } else if (!KTOK) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        cch[ch] = __fmul_rn(cq, sKc[buf][ch]);
        float mx = fmaxf(fmaxf(s[ch][0], s[ch][1]), s[ch][2]);
#pragma unroll
        for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, s[ch][r]), s[ch][r + 1]);
        mx = fmaxf(mx, s[ch][15]);
        tmax = fmaxf(tmax, __fmul_rn(mx, cch[ch]));
      }
    } else {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int kl = ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
          tmax = fmaxf(tmax, __fmul_rn(s[ch][r], __fmul_rn(cq, sKs[buf][kl])));
        }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(m, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;

    // ---- rescale O' for the block's V scale and the new maximum ----
    if (vchange) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          of[mt][4 * rq + 0] = __fmul_rn(of[mt][4 * rq + 0], rr[mt][rq].x);
          of[mt][4 * rq + 1] = __fmul_rn(of[mt][4 * rq + 1], rr[mt][rq].y);
          of[mt][4 * rq + 2] = __fmul_rn(of[mt][4 * rq + 2], rr[mt][rq].z);
          of[mt][4 * rq + 3] = __fmul_rn(of[mt][4 * rq + 3], rr[mt][rq].w);
        }
    }
    if (__any(alpha != 1.0f)) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) of[mt][r] = __fmul_rn(of[mt][r], alpha);
    }
    __builtin_amdgcn_sched_barrier(0);

    // ---- P, codes u = rint(15 P) packed as E2M3 u/8, row sums, PV.  15 P
    //      overwrites the score's register, so the 32 converter
    //      inputs of a 64-key group are the two chunks' accumulators in place:
    //      element 2i + c2 of the packed operand is register i of chunk 2gg + c2. ----
    float ls[4];   // independent partial sums, started by the first four values
#pragma unroll
    for (int gg = 0; gg < NG; ++gg) {
      if (DEBUG) {
        if (bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows && a.dbg_s) {
          const size_t rowo = static_cast<size_t>(qrow - a.dbg_row0);
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = key0 + (2 * gg + c2) * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
              if (key < N) a.dbg_s[rowo * N + key] = static_cast<int32_t>(s[2 * gg + c2][r]);
            }
        }
      }
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2) {
        const int ch = 2 * gg + c2;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float c;
          if (KTOK) c = __fmul_rn(cq, sKs[buf][ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3)]);
          else c = cch[ch];
          float P = __builtin_amdgcn_exp2f(__fmaf_rn(s[ch][r], c, -mnew));
          if (MASKED && s[ch][r] == -INFINITY) P = 0.f;
          if (gg == 0 && c2 == 0 && r < 4) ls[r] = P;
          else ls[r & 3] += P;
          s[ch][r] = __fmul_rn(P, pscale);
        }
      }
      // E2M3(rint(fl(15 P)) / 8): the conversion divides by the power-of-two
      // scale exactly and rounds to nearest even on the uniform 1/8 grid
      const v6i pk6 = __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(s[2 * gg], s[2 * gg + 1], 8.0f);
      const v8i B = v8i{pk6[0], pk6[1], pk6[2], pk6[3], pk6[4], pk6[5], 0, 0};
      if (DEBUG) {
        if (bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows && a.dbg_u) {
          const size_t rowo = static_cast<size_t>(qrow - a.dbg_row0);
#pragma unroll
          for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = key0 + (2 * gg + c2) * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
              const int bit = 6 * (2 * r + c2);   // packed element 2r + c2; its E2M3 code is u
              uint32_t w = static_cast<uint32_t>(pk6[bit >> 5]) >> (bit & 31);
              if ((bit & 31) > 26) w |= static_cast<uint32_t>(pk6[(bit >> 5) + 1]) << (32 - (bit & 31));
              if (key < N) a.dbg_u[rowo * N + key] = static_cast<uint8_t>(w & 63);
            }
        }
      }
      {
        const v8i v0 = load_rec(&sV[buf][(((gg * 4 + 0) * 2 + hh) * 32 + j) * 24]);
        const v8i v1 = load_rec(&sV[buf][(((gg * 4 + 1) * 2 + hh) * 32 + j) * 24]);
        of[0] = mfma6(v0, B, of[0]);
        const v8i v2 = load_rec(&sV[buf][(((gg * 4 + 2) * 2 + hh) * 32 + j) * 24]);
        of[1] = mfma6(v1, B, of[1]);
        const v8i v3 = load_rec(&sV[buf][(((gg * 4 + 3) * 2 + hh) * 32 + j) * 24]);
        of[2] = mfma6(v2, B, of[2]);
        of[3] = mfma6(v3, B, of[3]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    l = __fmaf_rn(l, alpha, (ls[0] + ls[1]) + (ls[2] + ls[3]));
    if (DEBUG && a.dbg_m && hh == 0 && bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows)
      a.dbg_m[static_cast<size_t>(qrow - a.dbg_row0) * nblocks + jb] = mnew;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };

  const int nfull = N / KV;
  for (int jb = 0; jb < nfull; ++jb) step(jb, std::integral_constant<bool, false>());
  if (nfull < nblocks) step(nfull, std::integral_constant<bool, true>());

  if (tid < kD) sW[tid] = wcur;
  __syncthreads();

  // ---- epilogue: O = O' * 8 w / 15 / l + mu_v ----
  const float ltot = l + __shfl_xor(l, 32);
  if (qrow < N) {
    const float inv = 1.0f / ltot;
    const float k2 = 8.0f / pscale;
    const size_t obase = (static_cast<size_t>(bh) * N + qrow) * kD;
    const float* muv = a.mu_v ? a.mu_v + bh * kD : nullptr;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int c0 = mt * 32 + 8 * rq + 4 * hh;
        const float4 w4 = *reinterpret_cast<const float4*>(&sW[c0]);
        float4 mu4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (muv) mu4 = *reinterpret_cast<const float4*>(muv + c0);
        float v[4];
        v[0] = of[mt][4 * rq + 0] * (w4.x * k2) * inv + mu4.x;
        v[1] = of[mt][4 * rq + 1] * (w4.y * k2) * inv + mu4.y;
        v[2] = of[mt][4 * rq + 2] * (w4.z * k2) * inv + mu4.z;
        v[3] = of[mt][4 * rq + 3] * (w4.w * k2) * inv + mu4.w;
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

template <int KV, bool KTOK, bool SYM7, bool DEBUG>
hipError_t launch_t(const AttnArgs& a, hipStream_t s) {
  const dim3 grid(a.Npad / kBlockM, a.BH);
  hipLaunchKernelGGL((k_attn_e2m3<KV, KTOK, SYM7, DEBUG>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
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

hipError_t launch_attn_e2m3(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, bool debug,
                            hipStream_t s) {
  if (kv_block == 64) return launch_k<64>(a, k_per_token, sym7, debug, s);
  return launch_k<128>(a, k_per_token, sym7, debug, s);
}

}  // namespace ra
