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
//   O' += (u/8) V~                       is exact per block,
// on v_mfma_scale_f32_32x32x64_f8f6f4, which runs at twice the int8 rate and
// accumulates in binary32: PV accumulates straight into the output tile.
//
// Per block of KV keys (ascending):
//   m_new = max(m, rowmax fl(S * c)),  P = 2^(S c - m_new),
//   u = rint(15 P),  l = alpha l + sum P,  alpha = 2^(m - m_new),
//   O' = O' * alpha * (w_old / w_new) + (u/8) V~   (w = V scale of the block's group)
// and finally O = O' * 8 w / 15 / l + mu_v (rotated back by H when V was
// rotated online, Sec. 4.3).  With Q smoothing every key j
// carries the score bias fl(b_j Kc): the scores become t = fma(S, c, bias_j)
// before the maximum, and 15 P = 2^(t - (m_new - log2 15)).  The factor 15 rides in the
// exponent: 15 P = 2^fma(S, c, -(m_new - log2 15)), one exponential per score
// and no multiply (the binary32 roundings of log2 15 and of m_new - log2 15
// perturb 15 P by a relative ln 2 * 2^-24 (|m_new| + 6) at most); l is kept as
// the sum of 15 P.  The
// rounding u = rint(15 P) is done by the packing conversion itself: it
// converts 15 P / 8 to E2M3 with round-to-nearest-even, and on the uniform 1/8
// grid that is rint to an integer.  Rows rescale O' by alpha only in the
// registers of queries whose maximum moved.
//
// Matrix-core mapping (one wave = 32 queries): S^T = K Q^T (A = 32 keys x 64
// channels of K, B = Q^T), so a lane holds 16 scores of one query per 32-key
// chunk, and the row statistics m, l are per lane.  The P codes of two chunks
// (64 keys) are packed by v_cvt_scalef32_2xpk16_fp6_f32 (which interleaves its
// two 16-value sources) into the A operand of O = P V~ (A and B operands share
// one lane layout: lane = row or column, lane / 32 = half of the reduction),
// and the V records, read as the B operand, are stored in the key order that
// packing produces.  In the output tile a lane holds one channel of 16
// queries, so the per-channel V scale ratio is one register per tile, and
// alpha reaches the query rows by a lane permute when some row's max moved.
//
// Software pipeline over blocks: once a 64-key group's probabilities are
// packed, its two score registers take the next block's scores of the same
// chunks, and those score products run on the matrix core while the vector
// unit computes the following group's probabilities (the PV products of the
// packed group likewise), so a block starts with its scores in registers.
// Three LDS tile buffers hold blocks j, j + 1 (read by the early score
// products) and j + 2 (written during block j); one barrier per block.  The
// first half of a block (its dependent chain of vector work) runs at a raised
// issue priority, so the two waves of a SIMD settle into alternating halves.
//
// The plain kernels are built from this file; ra_attn_e2m3_debug.hip builds
// the debug-dump kernels from the same source (two translation units compile
// in parallel).
#include <type_traits>

#include "ra_internal.h"
#include "ra_xcd.h"

#ifndef RA_E2M3_DEBUG_TU
#define RA_E2M3_DEBUG_TU 0
#endif

namespace ra {
namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v6i __attribute__((ext_vector_type(6)));
typedef float v16f __attribute__((ext_vector_type(16)));

// A workgroup of 8 waves (two per SIMD) covers 256 queries and owns a compute
// unit: the K/V tiles of a block are fetched once per unit, not once per
// 128 queries.
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBlockM = 32 * kWaves;  // queries per workgroup
constexpr int kScaleOne = 127;  // E8M0 block scale 2^0

__device__ __forceinline__ v16f mfma6(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 2, 2, 0, kScaleOne, 0, kScaleOne);
}

// 32 binary32 values -> 32 E2M3 codes (value / 8, round to nearest even), the
// two sources interleaved: element 2 i + c of the result is register i of
// source c.  Written out instead of left to the builtin because of two
// properties of v_cvt_scalef32_2xpk16_fp6_f32 on gfx950, both measured on the
// device with fixed-register probes: (1) it writes its destination before it
// has read all 32 source registers, so a destination that overlaps the end of
// a source corrupts the last codes -- and the compiler does allocate such
// overlaps (the result register written over registers 14 and 15 of the
// second source gave wrong P codes in whole rows) -- hence the early-clobber
// output; (2) it reads the first register of each source one cycle too early
// for a v_exp_f32 result written by the instruction right before it, hence
// the leading wait state.  The trailing wait states cover the matrix-core
// read of the result, which the compiler cannot see through the asm.
__device__ __forceinline__ v6i pack_fp6(v16f lo, v16f hi) {
  v6i r;
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile(
      "s_nop 0\n\t"
      "v_cvt_scalef32_2xpk16_fp6_f32 %0, %1, %2, %3\n\t"
      "s_nop 1"
      : "=&v"(r)
      : "v"(lo), "v"(hi), "s"(8.0f));
#else
  (void)lo;
  (void)hi;
  r = v6i{0, 0, 0, 0, 0, 0};
#endif
  return r;
}

// Maximum of a chunk's 16 exact scores as eight three-input maxima, seeded
// with the lowest finite binary32: the seed is below every score, so the
// chain needs no quieting of its first two inputs, and a chunk whose keys
// are all masked (-inf) yields the seed, which a valid key of the block (the
// partial last block has one) outweighs.
__device__ __forceinline__ float chunk_max(const v16f& x) {
  float mx = -3.40282347e38f;
#pragma unroll
  for (int r = 0; r < 16; r += 2) mx = fmaxf(fmaxf(mx, x[r]), x[r + 1]);
  return mx;
}

// O' registers r of the four output tiles times ab of lane q0(r) = 8 (r / 4) + r % 4
// of the register's own 32-lane half (ds_swizzle in bitmask mode: and 0, or q0),
// for the registers whose row moved its maximum
template <int R>
__device__ __forceinline__ void rescale_row(v16f (&o)[4], float ab, unsigned long long moved) {
  constexpr int q0 = 8 * (R >> 2) + (R & 3);
  if ((moved >> q0) & 0x11ull) {
    const float ar = __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(ab), q0 << 5));
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) o[mt][R] = __fmul_rn(o[mt][R], ar);
  }
}
template <int G>
__device__ __forceinline__ void rescale_group(v16f (&o)[4], float ab, unsigned long long moved) {
  if (!((moved >> (8 * G)) & 0xFFull)) return;   // rows 8G .. 8G+7 kept their maximum
  rescale_row<4 * G>(o, ab, moved);
  rescale_row<4 * G + 1>(o, ab, moved);
  rescale_row<4 * G + 2>(o, ab, moved);
  rescale_row<4 * G + 3>(o, ab, moved);
}

// 24-byte record -> operand registers (6 used dwords).  The fences keep the
// three reads apart: merged into paired reads, whose offset field stops at
// 2 KiB, the records of a tile would each need an address add, while single
// reads reach every record of the tile from one base.
__device__ __forceinline__ v8i load_rec(const uint8_t* p) {
  const uint2 a = *reinterpret_cast<const uint2*>(p);
  __builtin_amdgcn_sched_barrier(0);
  const uint2 b = *reinterpret_cast<const uint2*>(p + 8);
  __builtin_amdgcn_sched_barrier(0);
  const uint2 c = *reinterpret_cast<const uint2*>(p + 16);
  return v8i{static_cast<int>(a.x), static_cast<int>(a.y), static_cast<int>(b.x), static_cast<int>(b.y),
             static_cast<int>(c.x), static_cast<int>(c.y), 0, 0};
}

// K and V code tiles of one block go global -> registers -> LDS: every thread
// moves three 8-byte (KV = 128) or 4-byte (KV = 64) pieces of each, adjacent
// threads adjacent pieces.  The global loads of block j + 3 are issued at the
// end of block j and written to LDS in block j + 1, once its first 64-key
// group is packed, so their latency overlaps the barrier, the row maxima and
// the first probabilities.
template <int KV>
struct TilePiece {
  // 8-byte (KV = 128) or 4-byte (KV = 64) pieces as 32-bit vectors, six per thread
  typedef unsigned T __attribute__((ext_vector_type(KV == 128 ? 2 : 1)));
  T k0, k1, k2, v0, v1, v2;
  __device__ __forceinline__ void load(const uint8_t* kg, const uint8_t* vg, int tid) {
    const T* K = reinterpret_cast<const T*>(kg) + tid;
    const T* V = reinterpret_cast<const T*>(vg) + tid;
    k0 = K[0];
    v0 = V[0];
    k1 = K[kThreads];
    v1 = V[kThreads];
    k2 = K[2 * kThreads];
    v2 = V[2 * kThreads];
  }
  __device__ __forceinline__ void store(uint8_t* ks, uint8_t* vs, int tid) const {
    T* K = reinterpret_cast<T*>(ks) + tid;
    T* V = reinterpret_cast<T*>(vs) + tid;
    K[0] = k0;
    V[0] = v0;
    K[kThreads] = k1;
    V[kThreads] = v1;
    K[2 * kThreads] = k2;
    V[2 * kThreads] = v2;
  }
};

// QB: Q smoothing, every key carries the score bias fl(b_j Kc), the scores
// become t = fma(S, c, bias) before the maximum and P = 2^(t - m).
// LQ: the normaliser sums the codes u = rint(pscale P) (l = sum of P^) instead of pscale P.
template <int KV, bool KTOK, bool SYM7, bool DEBUG, bool QB, bool LQ>
__global__ __launch_bounds__(kThreads, 8 / kWaves) void k_attn_e2m3(AttnArgs a) {
  constexpr int NCH = KV / 32;   // 32-key chunks
  constexpr int NG = KV / 64;    // 64-key groups (one PV instruction each)
  constexpr int KB = KV * 96;    // bytes of K (and of V) codes per block
  __shared__ __align__(16) uint8_t sK[3][KB];
  __shared__ __align__(16) uint8_t sV[3][KB];
  __shared__ __align__(16) float sR[2][kD];   // V scale ratio w_old / w_new, channel 32 mt + j at 4 j + mt
  __shared__ __align__(16) float sW[kD];      // final V scale per channel
  __shared__ __align__(16) float sKs[2][KTOK ? KV : 1];
  __shared__ __align__(16) float sKc[2][NCH];  // K scale of each 32-key chunk (grouped K)
  __shared__ __align__(16) float sB[2][QB ? KV : 1];  // per-key score bias fl(b Kc)

  // the wave index is uniform: conditions on it are scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5, j = lane & 31;
  int bh, qtile;
  xcd_tile(bh, qtile);
  const int qrow = qtile * kBlockM + wave * 32 + j;
  const int N = a.N;
  const int nblocks = (N + KV - 1) / KV;
  const int kstride = a.Npad / a.k_group;
  // log2 of the P scale (15 for the range-optimized mapping, 7 for SYM7)
  constexpr float kLog2P = SYM7 ? 2.80735492205760410f : 3.90689059560851852f;
  const size_t hcode = static_cast<size_t>(bh) * a.Npad * 96;
  const uint8_t* kbase = a.kc + hcode;
  const uint8_t* vbase = a.vc + hcode;
  const float* ksh = a.ks + static_cast<size_t>(bh) * kstride;

  // ---- Q operand (B of S^T = K Q^T) ----
  // (a wave whose 32 queries lie past the padded length, in the last
  //  workgroup, computes on zero codes and stores nothing)
  const bool qin = qrow < a.Npad;
  v8i qop[2] = {v8i{0, 0, 0, 0, 0, 0, 0, 0}, v8i{0, 0, 0, 0, 0, 0, 0, 0}};
  float cq = 0.f;
  if (qin) {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const int rec = (((qrow >> 5) * 2 + kc) * 2 + hh) * 32 + (qrow & 31);
      qop[kc] = load_rec(a.qc + hcode + static_cast<size_t>(rec) * 24);
    }
    cq = __fmul_rn(a.qs[static_cast<size_t>(bh) * (a.Npad / a.q_group) + qrow / a.q_group], a.Kc);
  }

  // Per-block side data: the V scales of the block's group (thread ch < 128
  // owns channel ch's working scale w and writes the ratio w_old / w_new) and
  // the K scales (per 32-key chunk, or per key; thread 128 + t takes scale t).
  // They are fetched from global memory one block ahead of staging, so no
  // wave waits on their latency.
  struct Aux {
    float v, k, b;
  };
  // fetch_aux runs for blocks 0, 1, 2, ... in order; (fg, fr) = (V group, block
  // within the group) of the next block it fetches
  int fg = 0, fr = 0;
  // Waves 0 and 1 (thread = channel) handle the V scales; thread 128 + t
  // handles key t of the block (waves 2 and 3, or wave 2 alone for 64-key
  // blocks), or the K scale of chunk t (t < NCH, grouped K: k_group is 32, 64
  // or 128, so the group index is a shift).
  const bool kwave = KV == 128 ? (wave == 2 || wave == 3) : wave == 2;
  const int kgs = __builtin_ctz(static_cast<unsigned>(a.k_group));
  auto fetch_aux = [&](int jb) {
    Aux f{0.f, 0.f, 0.f};
    if (wave < 2) f.v = a.vs[(static_cast<size_t>(bh) * a.nvgroups + fg) * kD + tid];
    if (++fr == a.v_bpg) {
      fr = 0;
      ++fg;
    }
    const int kt = tid - kD;
    if (KTOK) {
      if (kwave) f.k = ksh[(jb * KV + kt) >> kgs];
    } else if (wave == 2 && lane < NCH) {
      f.k = ksh[(jb * KV + kt * 32) >> kgs];
    }
    if (QB && kwave) f.b = a.kbias[static_cast<size_t>(bh) * a.Npad + jb * KV + kt];
    return f;
  };
  float wcur = 1.0f;
  auto store_aux = [&](int jb, int buf, const Aux& f) {
    if (wave < 2) {
      float r = 1.0f;
      if (f.v > 0.0f) {
        r = (jb == 0) ? 1.0f : wcur * __builtin_amdgcn_rcpf(f.v);
        wcur = f.v;
      }
      sR[buf][(tid & 31) * 4 + (tid >> 5)] = r;
    }
    const int kt = tid - kD;
    if (KTOK) {
      if (kwave) sKs[buf][kt] = f.k;
    } else if (wave == 2 && lane < NCH) {
      sKc[buf][kt] = f.k;
    }
    if (QB && kwave) sB[buf][kt] = __fmul_rn(f.b, a.Kc);
  };

  v16f of[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) of[mt][r] = 0.f;
  // running max m (on the score scale of the method) and row sum l of
  // pscale * P; vr = block index within its V group
  float m = -INFINITY, l = 0.f;
  int vr = 0;

  static_assert(KB == 3 * kThreads * static_cast<int>(sizeof(typename TilePiece<KV>::T)), "three pieces per thread");
  // Three tile buffers: block j's tiles sit in buffer j % 3; block j + 1's are
  // already in LDS while block j is processed (its score products run during
  // block j's probabilities), and block j + 2's are written during block j.
  const int t1 = nblocks > 1 ? 1 : 0, t2 = nblocks > 2 ? 2 : nblocks - 1;
  TilePiece<KV> tp;
  tp.load(kbase, vbase, tid);
  tp.store(sK[0], sV[0], tid);
  tp.load(kbase + t1 * KB, vbase + t1 * KB, tid);
  tp.store(sK[1], sV[1], tid);
  tp.load(kbase + t2 * KB, vbase + t2 * KB, tid);
  store_aux(0, 0, fetch_aux(0));
  Aux pf{0.f, 0.f, 0.f};
  if (nblocks > 1) pf = fetch_aux(1);
  __syncthreads();

  // ---- S^T = K Q^T (exact integer scores in binary32), chunks c0 and c0 + 1
  //      of the tile at kt.  s carries the scores of the next block from one
  //      block to the next. ----
  v16f s[NCH];
  auto krec = [&](const uint8_t* kt, int ch, int kc) {
    return load_rec(&kt[(((ch * 2 + kc) * 2 + hh) * 32 + j) * 24]);
  };
  auto score_pair = [&](const v8i (&kr)[4], int c0) {
    v16f z;
#pragma unroll
    for (int r = 0; r < 16; ++r) z[r] = 0.f;
    s[c0] = mfma6(kr[0], qop[0], z);
    s[c0 + 1] = mfma6(kr[1], qop[0], z);
    s[c0] = mfma6(kr[2], qop[1], s[c0]);
    s[c0 + 1] = mfma6(kr[3], qop[1], s[c0 + 1]);
  };
  // the four K records of chunks c0, c0 + 1 (channel half kc = t / 2), one
  // record per scheduling region so reads of two records are not merged
  auto read_kpair = [&](v8i (&kr)[4], const uint8_t* kt, int c0) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      kr[t] = krec(kt, c0 + (t & 1), t >> 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  {
    v8i kr[4];
#pragma unroll
    for (int c0 = 0; c0 < NCH; c0 += 2) {
      read_kpair(kr, sK[0], c0);
      score_pair(kr, c0);
    }
  }
  int tb = 0;   // buffer of the current block's tiles (block index mod 3)

  // One block of KV keys.  MASKED (keys past N) only for the partial last
  // block, which runs outside the main loop so the full blocks carry no masking.
  // MORE: a next block exists (every block but the last); as a template
  // argument it keeps the step one basic block from the probabilities on, so
  // the products stay where they are placed between them.
  auto step = [&](int jb, auto masked_tag, auto more_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool more = decltype(more_tag)::value;
    const int buf = jb & 1;   // side-data buffers
    const int key0 = jb * KV;
    const int tbn = tb == 2 ? 0 : tb + 1;   // next block's tiles
    const int tbw = tbn == 2 ? 0 : tbn + 1; // tiles written in this block (block j + 2)
    // Issue priority: the first half of the block (side data, maximum,
    // alpha, the first group's probabilities and products) is one dependent
    // chain of vector work, the second half mostly matrix-core products.
    // With the chain at the higher priority, the other wave of the SIMD in
    // its product half yields the vector unit to it, so one wave's products
    // run under the other's chain (measured: 3.05 -> 2.93 ms on the
    // 32760-token layer; the product regions at the higher priority instead
    // were slower).
    __builtin_amdgcn_s_setprio(1);
    if (more) {
      store_aux(jb + 1, buf ^ 1, pf);
      if (jb + 2 < nblocks) pf = fetch_aux(jb + 2);
    }
    __builtin_amdgcn_sched_barrier(0);

    // key of accumulator register r in chunk ch: key0 + 32*ch + 8*(r/4) + 4*hh + r%4
    if (DEBUG) {
      if (bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows && a.dbg_s) {
        const size_t rowo = static_cast<size_t>(qrow - a.dbg_row0);
#pragma unroll
        for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
            if (key < N) a.dbg_s[rowo * N + key] = static_cast<int32_t>(s[ch][r]);
          }
      }
    }
    if (MASKED) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3) >= N) s[ch][r] = -INFINITY;
    }

    // The V scale ratio of a new group rescales O' (register r of tile mt is
    // channel 32 mt + j); the multiplies do not depend on S and fill the
    // latency of the maximum's dependent chain.  They are issued
    // unconditionally (by 1 within a V group: exact); O' is rescaled by the V
    // ratio before alpha.
    const bool vchange = vr == 0 && jb > 0;   // first block of a new V group
    if (++vr == a.v_bpg) vr = 0;
    float4 rr = make_float4(1.f, 1.f, 1.f, 1.f);
    if (vchange) rr = *reinterpret_cast<const float4*>(&sR[buf][4 * j]);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      of[0][r] = __fmul_rn(of[0][r], rr.x);
      of[1][r] = __fmul_rn(of[1][r], rr.y);
      of[2][r] = __fmul_rn(of[2][r], rr.z);
      of[3][r] = __fmul_rn(of[3][r], rr.w);
    }

    // ---- block row maximum of fl(S * c) (c >= 0, so it is fl(max S * c);
    //      a fully masked chunk gives the seed of chunk_max, far below) ----
    float cch[NCH];
    float tmax = -INFINITY;
    if (QB) {
      // t = fma(S, c, bias) in place of S; the maximum is over t
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        if (!KTOK) cch[ch] = __fmul_rn(cq, sKc[buf][ch]);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int kl = ch * 32 + 8 * r4 + 4 * hh;
          const float4 b4 = *reinterpret_cast<const float4*>(&sB[buf][kl]);
          const float bb[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * r4 + e;
            const float c = KTOK ? __fmul_rn(cq, sKs[buf][kl + e]) : cch[ch];
            float t = __fmaf_rn(s[ch][r], c, bb[e]);
            if (MASKED && s[ch][r] == -INFINITY) t = -INFINITY;
            s[ch][r] = t;
            tmax = fmaxf(tmax, t);
          }
        }
      }
    } else if (!KTOK && a.k_group >= KV) {
      // one K scale for the whole block: a single product after the maximum
      float mx = chunk_max(s[0]);
#pragma unroll
      for (int ch = 1; ch < NCH; ++ch) mx = fmaxf(mx, chunk_max(s[ch]));
      const float c0 = __fmul_rn(cq, sKc[buf][0]);
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) cch[ch] = c0;
      tmax = __fmul_rn(mx, c0);
    } else if (!KTOK) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        cch[ch] = __fmul_rn(cq, sKc[buf][ch]);
        tmax = fmaxf(tmax, __fmul_rn(chunk_max(s[ch]), cch[ch]));
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
    tmax = max_halves(tmax);
    const float mnew = fmaxf(m, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    // pscale * 2^x = 2^(S c - (m - log2 pscale)): the P scale rides in the
    // exponent, so the exponential yields the packing input directly
    const float mq = __fsub_rn(mnew, kLog2P);

    // ---- rescale O' for the new maximum; register r of tile mt is channel
    //      32 mt + j of query 8 (r / 4) + 4 hh + r % 4 ----
    // only the registers whose two queries (8 (r / 4) + r % 4 in the lower
    // wave half, 4 more in the upper) moved their maximum are rescaled
    const unsigned long long moved = __ballot(alpha != 1.0f);
    if (moved) {
      // ab: lane 32 hh + i holds alpha of query i + 4 hh (a row rotation by 4
      // lanes in the upper half; the lanes read below never leave their row
      // of 16), so register r's factor is lane q0 of its own 32-lane half
      const float ab = __int_as_float(
          __builtin_amdgcn_update_dpp(__float_as_int(alpha), __float_as_int(alpha), 0x12C, 0xC, 0xF, false));
      rescale_group<0>(of, ab, moved);
      rescale_group<1>(of, ab, moved);
      rescale_group<2>(of, ab, moved);
      rescale_group<3>(of, ab, moved);
    }
    __builtin_amdgcn_sched_barrier(0);

    // ---- P, codes u = rint(15 P) packed as E2M3 u/8, row sums, PV.  15 P
    //      overwrites the score's register, so the 32 converter inputs of a
    //      64-key group are the two chunks' accumulators in place: element
    //      2i + c2 of the packed operand is register i of chunk 2gg + c2.
    //      Once a group is packed, its two score registers take the next
    //      block's scores of the same chunks; the products of group gg (PV,
    //      and the next block's scores) are interleaved with the
    //      probabilities of group gg + 1. ----
    float ls[4];   // independent partial sums, started by the first four values
    // probabilities of registers 4 q .. 4 q + 3 of chunk ch
    auto probs4 = [&](int ch, int q) {
#pragma unroll
      for (int r = 4 * q; r < 4 * q + 4; ++r) {
        float P;   // pscale * P
        if (QB) {
          P = __builtin_amdgcn_exp2f(__fsub_rn(s[ch][r], mq));
        } else {
          float c;
          if (KTOK) c = __fmul_rn(cq, sKs[buf][ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3)]);
          else c = cch[ch];
          P = __builtin_amdgcn_exp2f(__fmaf_rn(s[ch][r], c, -mq));
        }
        if (MASKED && s[ch][r] == -INFINITY) P = 0.f;
        const float lv = LQ ? __builtin_rintf(P) : P;
        if (ch == 0 && r < 4) ls[r] = lv;
        else ls[r & 3] += lv;
        s[ch][r] = P;
      }
    };
    v8i vrec[4];   // V records of the group in flight (B operands of O = P V~)
    v8i kr[4];     // K records of the next block's chunk pair
    v8i B;         // packed codes of the group in flight (A operand of O = P V~)
    auto read_vrecs = [&](int gg) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        vrec[t] = load_rec(&sV[tb][(((gg * 4 + t) * 2 + hh) * 32 + j) * 24]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    auto pack_group = [&](int gg) {
      // E2M3(rint(15 P) / 8): the conversion divides by the power-of-two
      // scale exactly and rounds to nearest even on the uniform 1/8 grid
      const v6i pk6 = pack_fp6(s[2 * gg], s[2 * gg + 1]);
      B = v8i{pk6[0], pk6[1], pk6[2], pk6[3], pk6[4], pk6[5], 0, 0};
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
    };

    read_vrecs(0);
#pragma unroll
    for (int q = 0; q < 8; ++q) probs4(q >> 2, q & 3);
    pack_group(0);
    // block j + 2's tiles into the buffer block j - 1 used
    tp.store(sK[tbw], sV[tbw], tid);
    __builtin_amdgcn_sched_barrier(0);
    if (more) read_kpair(kr, sK[tbn], 0);
#pragma unroll
    for (int gg = 1; gg < NG; ++gg) {
      // products of group gg - 1 beside the probabilities of group gg (the
      // compiler interleaves them within the region)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        of[t] = mfma6(B, vrec[t], of[t]);
        probs4(2 * gg, t);
      }
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
      read_vrecs(gg);
      if (more) {
        v16f z;
#pragma unroll
        for (int r = 0; r < 16; ++r) z[r] = 0.f;
        const int c0 = 2 * gg - 2;
        s[c0] = mfma6(kr[0], qop[0], z);
        probs4(2 * gg + 1, 0);
        s[c0 + 1] = mfma6(kr[1], qop[0], z);
        probs4(2 * gg + 1, 1);
        s[c0] = mfma6(kr[2], qop[1], s[c0]);
        probs4(2 * gg + 1, 2);
        s[c0 + 1] = mfma6(kr[3], qop[1], s[c0 + 1]);
        probs4(2 * gg + 1, 3);
        __builtin_amdgcn_sched_barrier(0);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) probs4(2 * gg + 1, q);
        __builtin_amdgcn_sched_barrier(0);
      }
      if (more) read_kpair(kr, sK[tbn], 2 * gg);
      pack_group(gg);
    }
    if (NG == 1) __builtin_amdgcn_s_setprio(0);
    // products of the last group
#pragma unroll
    for (int t = 0; t < 4; ++t) of[t] = mfma6(B, vrec[t], of[t]);
    if (more) score_pair(kr, NCH - 2);
    l = __fmaf_rn(l, alpha, (ls[0] + ls[1]) + (ls[2] + ls[3]));
    if (DEBUG && a.dbg_m && hh == 0 && bh == a.dbg_bh && qrow >= a.dbg_row0 && qrow < a.dbg_row0 + a.dbg_rows)
      a.dbg_m[static_cast<size_t>(qrow - a.dbg_row0) * nblocks + jb] = mnew;
    {
      // unconditional (the last blocks reload the final tile), so the pieces
      // are not live through the block body
      const size_t nb3 = static_cast<size_t>(jb + 3 < nblocks ? jb + 3 : nblocks - 1) * KB;
      tp.load(kbase + nb3, vbase + nb3, tid);
    }
    tb = tbn;
    __syncthreads();
  };

  // every block but the last is full; the last runs with the key checks
  // (which mask nothing when it is full)
  using kNo = std::integral_constant<bool, false>;
  using kYes = std::integral_constant<bool, true>;
  for (int jb = 0; jb + 1 < nblocks; ++jb) step(jb, kNo(), kYes());
  step(nblocks - 1, kYes(), kNo());

  if (tid < kD) sW[tid] = wcur;
  __syncthreads();

  // ---- epilogue: O = O' * 8 w / 15 / l + mu_v; lane (j, hh) holds channel
  //      32 mt + j of the wave's queries 8 (r / 4) + 4 hh + r % 4 ----
  const float ltot = l + __shfl_xor(l, 32);   // pscale * sum of P (LQ: sum of the codes u)
  const float k2 = 8.0f;
  const float* muv = a.mu_v ? a.mu_v + bh * kD : nullptr;
  float wsc[4], mu[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    wsc[mt] = sW[mt * 32 + j] * k2;
    mu[mt] = muv ? muv[mt * 32 + j] : 0.f;
  }
  const int q0 = qtile * kBlockM + wave * 32;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int qi = 8 * (r >> 2) + 4 * hh + (r & 3);
    const float inv = 1.0f / __shfl(ltot, qi);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) of[mt][r] = of[mt][r] * wsc[mt] * inv + mu[mt];
  }
  if (a.vhad) {
    // V came rotated by H: each query row goes back, O = O' H^T = O' H.  Channel
    // 32 mt + j: strides 64 and 32 pair tiles mt ^ 2 and mt ^ 1 in the thread,
    // strides 16 .. 1 pair lanes j ^ 16 .. j ^ 1 (the lane with the bit set
    // takes the difference); then the factor 1/sqrt(128).
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float t0 = of[0][r] + of[2][r], t2 = of[0][r] - of[2][r];
      const float t1 = of[1][r] + of[3][r], t3 = of[1][r] - of[3][r];
      of[0][r] = t0 + t1;
      of[1][r] = t0 - t1;
      of[2][r] = t2 + t3;
      of[3][r] = t2 - t3;
#pragma unroll
      for (int msk = 16; msk >= 1; msk >>= 1) {
        const bool upper = (j & msk) != 0;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          const float o = __shfl_xor(of[mt][r], msk);
          of[mt][r] = upper ? o - of[mt][r] : of[mt][r] + o;
        }
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) of[mt][r] *= kInvSqrtD;
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int qi = 8 * (r >> 2) + 4 * hh + (r & 3);
    if (q0 + qi < N) {
      const size_t obase = (static_cast<size_t>(bh) * N + q0 + qi) * kD + j;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const float v = of[mt][r];
        if (a.out_dtype == 2) static_cast<float*>(a.o)[obase + mt * 32] = v;
        else if (a.out_dtype == 0) static_cast<uint16_t*>(a.o)[obase + mt * 32] = __bfloat16_as_ushort(__float2bfloat16(v));
        else static_cast<uint16_t*>(a.o)[obase + mt * 32] = __half_as_ushort(__float2half(v));
      }
    }
  }
}

template <int KV, bool KTOK, bool SYM7, bool DEBUG, bool QB, bool LQ>
hipError_t launch_l(const AttnArgs& a, hipStream_t s) {
  const dim3 grid((a.Npad + kBlockM - 1) / kBlockM, a.BH);
  hipLaunchKernelGGL((k_attn_e2m3<KV, KTOK, SYM7, DEBUG, QB, LQ>), grid, dim3(kThreads), 0, s, a);
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

template <int KV, bool KTOK>
hipError_t launch_p(const AttnArgs& a, bool sym7, hipStream_t s) {
  constexpr bool kDebug = RA_E2M3_DEBUG_TU != 0;
  return sym7 ? launch_t<KV, KTOK, true, kDebug>(a, s) : launch_t<KV, KTOK, false, kDebug>(a, s);
}

template <int KV>
hipError_t launch_k(const AttnArgs& a, bool ktok, bool sym7, hipStream_t s) {
  return ktok ? launch_p<KV, true>(a, sym7, s) : launch_p<KV, false>(a, sym7, s);
}

}  // namespace

#if RA_E2M3_DEBUG_TU
hipError_t launch_attn_e2m3_debug(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, hipStream_t s) {
  if (kv_block == 64) return launch_k<64>(a, k_per_token, sym7, s);
  return launch_k<128>(a, k_per_token, sym7, s);
}
#else
hipError_t launch_attn_e2m3(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, bool debug,
                            hipStream_t s) {
  if (debug) return launch_attn_e2m3_debug(a, kv_block, k_per_token, sym7, s);
  if (kv_block == 64) return launch_k<64>(a, k_per_token, sym7, s);
  return launch_k<128>(a, k_per_token, sym7, s);
}
#endif

}  // namespace ra
