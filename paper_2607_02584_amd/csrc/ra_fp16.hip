// ra_fp16.hip -- BF16/FP16 fallback attention for gfx950 (the 16-bit path the
// paper keeps for accuracy-sensitive DiT blocks and denoising steps).
//
// Producer: plain 3D RoPE (Sec. 3) of Q and K in binary32, rounded to the
// 16-bit input type, written in a tiled layout that makes every 32-token chunk
// a ready matrix-core operand; V is re-laid out the same way, transposed.
//
// Attention: S^T = K Q^T on v_mfma_f32_32x32x16_{bf16,f16} (fp32 accumulate),
// blockwise online softmax over blocks of kv_block (64 or 128) keys in
// ascending order,
//   m = max(m, rowmax(S * Kc)),  P = 2^(S*Kc - m),  l = alpha*l + sum P,
// P rounded to the 16-bit type as the A operand of O += P V, and O = O / l.
// Each lane holds the scores of one query, so row reductions stay inside the
// lane plus one exchange between the two wave halves.
//
// 16-bit tiled layouts (elements), token n = 32*c + r:
//   Q, K: (((c*8 + ch/16)*2 + (ch/8)%2)*32 + r)*8 + ch%8
//   V:    (((c*2 + s)*2 + h)*128 + ch)*8 + e  holds V[32c + 16s + 8(e/4) + 4h + e%4][ch]
#include <type_traits>

#include "ra_internal.h"
#include "ra_xcd.h"

namespace ra {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int kBlockM = 128;  // queries per workgroup

__device__ __forceinline__ float h2f(uint16_t b, int is_fp16) {
  if (is_fp16) return __half2float(__ushort_as_half(b));
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ uint16_t f2h(float v, int is_fp16) {
  if (is_fp16) return __half_as_ushort(__float2half(v));
  return __bfloat16_as_ushort(__float2bfloat16(v));
}

__device__ __forceinline__ int fdiv(int n, int d, float inv_d) {
  int q = static_cast<int>(static_cast<float>(n) * inv_d);
  if (q * d > n) --q;
  if ((q + 1) * d <= n) ++q;
  return q;
}

// One thread per (token, 4 channels): RoPE in binary32, rounded to 16 bits,
// written to the tiled layout.  Grid: (Npad/8, BH), 256 threads = 8 tokens.
__global__ __launch_bounds__(256) void k_rope16(RopeTables t, const uint16_t* x, uint16_t* out, int N, int Npad,
                                                int is_fp16) {
  const int bh = blockIdx.y;
  const int n = blockIdx.x * 8 + (threadIdx.x >> 5);
  const int cl = threadIdx.x & 31;
  uint16_t res[4] = {0, 0, 0, 0};
  if (n < N) {
    const uint2 w = *reinterpret_cast<const uint2*>(x + (static_cast<size_t>(bh) * N + n) * kD + 4 * cl);
    const float xv[4] = {h2f(w.x & 0xffff, is_fp16), h2f(w.x >> 16, is_fp16), h2f(w.y & 0xffff, is_fp16),
                         h2f(w.y >> 16, is_fp16)};
    const int W = t.grid[2], Hg = t.grid[1];
    const int tq = fdiv(n, W * Hg, 1.0f / static_cast<float>(W * Hg));
    const int rem = n - tq * W * Hg;
    const int hq = fdiv(rem, W, 1.0f / static_cast<float>(W));
    const int pos[3] = {tq, hq, rem - hq * W};
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int p = 2 * cl + i;
      int first = 0, a = 2;
      for (int ax = 0; ax < 3; ++ax) {
        const int np = t.split[ax] / 2;
        if (p < first + np) {
          a = ax;
          break;
        }
        first += np;
      }
      const float4 g = t.axis[a][pos[a] * (t.split[a] / 2) + (p - first)];
      const float y0 = __fmaf_rn(xv[2 * i + 1], g.z, __fmul_rn(xv[2 * i], g.x));
      const float y1 = __fmaf_rn(xv[2 * i + 1], g.w, __fmul_rn(xv[2 * i], g.y));
      res[2 * i] = f2h(y0, is_fp16);
      res[2 * i + 1] = f2h(y1, is_fp16);
    }
  }
  if (n < Npad) {
    const int c = n >> 5, r = n & 31, ch = 4 * cl;
    const size_t off = static_cast<size_t>(bh) * Npad * kD +
                       ((static_cast<size_t>(c * 8 + (ch >> 4)) * 2 + ((ch >> 3) & 1)) * 32 + r) * 8 + (ch & 7);
    *reinterpret_cast<uint2*>(out + off) =
        make_uint2(res[0] | (static_cast<uint32_t>(res[1]) << 16), res[2] | (static_cast<uint32_t>(res[3]) << 16));
  }
}

// V relayout: one workgroup per 32-token chunk; the chunk goes through LDS.
__global__ __launch_bounds__(256) void k_v16_relayout(const uint16_t* v, uint16_t* out, int N, int Npad) {
  __shared__ uint16_t tile[32][kD + 2];
  const int bh = blockIdx.y, c = blockIdx.x, tid = threadIdx.x;
  for (int i = tid; i < 32 * 32; i += 256) {
    const int r = i >> 5, cl = i & 31;
    const int n = c * 32 + r;
    uint2 w = make_uint2(0u, 0u);
    if (n < N) w = *reinterpret_cast<const uint2*>(v + (static_cast<size_t>(bh) * N + n) * kD + 4 * cl);
    tile[r][4 * cl + 0] = w.x & 0xffff;
    tile[r][4 * cl + 1] = w.x >> 16;
    tile[r][4 * cl + 2] = w.y & 0xffff;
    tile[r][4 * cl + 3] = w.y >> 16;
  }
  __syncthreads();
  // 512 output vectors of 8 elements: (s, h, ch)
  for (int i = tid; i < 512; i += 256) {
    const int ch = i & 127, h = (i >> 7) & 1, s = i >> 8;
    uint32_t e[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e0 = 2 * q, e1 = 2 * q + 1;
      const int k0 = 16 * s + 8 * (e0 >> 2) + 4 * h + (e0 & 3);
      const int k1 = 16 * s + 8 * (e1 >> 2) + 4 * h + (e1 & 3);
      e[q] = tile[k0][ch] | (static_cast<uint32_t>(tile[k1][ch]) << 16);
    }
    const size_t off = static_cast<size_t>(bh) * Npad * kD + ((static_cast<size_t>(c * 2 + s) * 2 + h) * 128 + ch) * 8;
    *reinterpret_cast<uint4*>(out + off) = make_uint4(e[0], e[1], e[2], e[3]);
  }
}

template <bool F16>
struct MF;
template <>
struct MF<false> {
  typedef v8bf vec;
  typedef __bf16 v2t __attribute__((ext_vector_type(2)));
  static __device__ __forceinline__ v16f mfma(vec a, vec b, v16f c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct MF<true> {
  typedef v8h vec;
  typedef _Float16 v2t __attribute__((ext_vector_type(2)));
  static __device__ __forceinline__ v16f mfma(vec a, vec b, v16f c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

typedef float v2f __attribute__((ext_vector_type(2)));

// two binary32 values -> one dword of two 16-bit values (round to nearest even)
template <bool F16>
__device__ __forceinline__ uint32_t pack2(float x, float y) {
  const typename MF<F16>::v2t t = __builtin_convertvector(v2f{x, y}, typename MF<F16>::v2t);
  return __builtin_bit_cast(uint32_t, t);
}

template <typename V>
__device__ __forceinline__ V as_vec(uint4 u) {
  return __builtin_bit_cast(V, u);
}

// K and V tiles move global -> registers -> LDS; each thread carries KV / 16
// 16-byte pieces of each (the K and V pieces may belong to different blocks).
template <int KV>
struct Tile16 {
  typedef unsigned T __attribute__((ext_vector_type(4)));
  static constexpr int NP = KV / 16;
  static_assert(NP * 16 * 256 == KV * kD * 2, "pieces cover the tile");
  T k[NP], v[NP];
  __device__ __forceinline__ void load(const uint16_t* kg, const uint16_t* vg, int tid) {
    const T* K = reinterpret_cast<const T*>(kg) + tid;
    const T* V = reinterpret_cast<const T*>(vg) + tid;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      k[i] = K[256 * i];
      v[i] = V[256 * i];
    }
  }
  __device__ __forceinline__ void store(uint16_t* ks, uint16_t* vs, int tid) const {
    T* K = reinterpret_cast<T*>(ks) + tid;
    T* V = reinterpret_cast<T*>(vs) + tid;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      K[256 * i] = k[i];
      V[256 * i] = v[i];
    }
  }
};

// One wave = 32 queries; S^T = K Q^T puts the scores of one query in one lane
// (register r of chunk ch is key 32 ch + 8 (r / 4) + 4 hh + r % 4).  The 16-bit
// P values of register pairs are directly the A operand of O = P V (A and B
// operands share one lane layout), with V read as the B operand in the key
// order of its relayout, so a lane of the output tile holds one channel of 16
// queries (query 8 (r / 4) + 4 hh + r % 4 in register r).
//
// Software pipeline over blocks: once a 32-key chunk's probabilities are
// rounded to 16 bits, its score registers take the next block's scores of
// the same chunk; those products and the chunk's PV products run on the
// matrix core beside the next chunk's probabilities, with their LDS operands
// read two products ahead, and a block starts with its scores in registers.
// K tiles are staged two blocks ahead and V tiles one block ahead, so two LDS
// buffers of each suffice (block j + 2's K goes where block j's K was, whose
// scores were taken during block j - 1).
template <bool F16, int kKV>
__global__ __launch_bounds__(256, kKV == 64 ? 2 : 1) void k_attn16(Fp16Args a) {
  typedef typename MF<F16>::vec vec;
  constexpr int NCH = kKV / 32;
  constexpr int TILE = kKV * kD;  // elements of K (and of V) per block
  __shared__ __align__(16) uint16_t sK[2][TILE];
  __shared__ __align__(16) uint16_t sV[2][TILE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, j = lane & 31;
  int bh, qtile;
  xcd_tile(bh, qtile);
  const int q0 = qtile * kBlockM + wave * 32;
  const int qrow = q0 + j;
  const int N = a.N;
  const int nblocks = (N + kKV - 1) / kKV;
  const size_t hoff = static_cast<size_t>(bh) * a.Npad * kD;
  const uint16_t* kbase = a.k + hoff;
  const uint16_t* vbase = a.v + hoff;
  const float Kc = a.Kc;
  auto blk = [&](int b) { return static_cast<size_t>(b < nblocks ? b : nblocks - 1) * TILE; };

  vec qop[8];
  {
    const uint16_t* qp = a.q + hoff + static_cast<size_t>(qrow >> 5) * 4096 + (qrow & 31) * 8;
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) qop[kc] = as_vec<vec>(*reinterpret_cast<const uint4*>(qp + (kc * 2 + hh) * 256));
  }

  v16f of[4];
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int r = 0; r < 16; ++r) of[mt][r] = 0.f;
  float m = -INFINITY, l = 0.f;

  auto kop = [&](const uint16_t* kt, int ch, int kc) {
    return as_vec<vec>(*reinterpret_cast<const uint4*>(&kt[(((ch * 8 + kc) * 2 + hh) * 32 + j) * 8]));
  };
  v16f s[NCH];

  // prologue: K and V of block 0 and K of block 1 in LDS, block 0's scores;
  // then V of block 1 and K of block 2 staged for the first step
  Tile16<kKV> tp;
  tp.load(kbase, vbase, tid);
  tp.store(sK[0], sV[0], tid);
  tp.load(kbase + blk(1), vbase + blk(1), tid);
  tp.store(sK[1], sV[1], tid);
  __syncthreads();
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
    for (int r = 0; r < 16; ++r) s[ch][r] = 0.f;
#pragma unroll
  for (int kc = 0; kc < 8; ++kc)
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) s[ch] = MF<F16>::mfma(kop(sK[0], ch, kc), qop[kc], s[ch]);
  tp.load(kbase + blk(2), vbase + blk(1), tid);
  __syncthreads();   // every wave has read block 0's K before it is overwritten

  auto step = [&](int jb, auto masked_tag, auto more_tag) {
    constexpr bool MASKED = decltype(masked_tag)::value;
    constexpr bool more = decltype(more_tag)::value;
    // Issue priority: the block's dependent chain of vector work (maximum,
    // alpha, the first chunk's probabilities) and the first chunk's products
    // run at the higher priority, the remaining products at the lower one,
    // so the waves of a SIMD alternate halves (about 2 % faster than one
    // priority throughout).
    __builtin_amdgcn_s_setprio(1);
    const int buf = jb & 1;
    const int key0 = jb * kKV;
    if (MASKED) {
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3) >= N) s[ch][r] = -INFINITY;
    }

    // ---- row maximum of S * Kc (Kc > 0: the product of the maximum) ----
    float mx = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
#pragma unroll
    for (int r = 3; r < 15; r += 2) mx = fmaxf(fmaxf(mx, s[0][r]), s[0][r + 1]);
    mx = fmaxf(mx, s[0][15]);
#pragma unroll
    for (int ch = 1; ch < NCH; ++ch)
#pragma unroll
      for (int r = 0; r < 16; r += 2) mx = fmaxf(fmaxf(mx, s[ch][r]), s[ch][r + 1]);
    float tmax = __fmul_rn(mx, Kc);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(m, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    if (__any(alpha != 1.0f)) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float ar = __shfl(alpha, 8 * (r >> 2) + 4 * hh + (r & 3));
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) of[mt][r] = __fmul_rn(of[mt][r], ar);
      }
    }
    // block j + 2's K where block j's was, block j + 1's V where block j - 1's was
    tp.store(sK[buf], sV[buf ^ 1], tid);

    // ---- P = 2^(S Kc - m) in 16 bits, row sums of the unrounded P, O += P V ----
    float ls[4];
    uint32_t pw[NCH][8];
    auto probs = [&](int ch, int r2) {   // registers 2 r2, 2 r2 + 1 of chunk ch
      float P[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = 2 * r2 + u;
        float p = __builtin_amdgcn_exp2f(__fmaf_rn(s[ch][r], Kc, -mnew));
        if (MASKED && s[ch][r] == -INFINITY) p = 0.f;
        if (ch == 0 && r < 4) ls[r] = p;
        else ls[r & 3] += p;
        P[u] = p;
      }
      pw[ch][r2] = pack2<F16>(P[0], P[1]);
    };
    // the products of chunk c (group c): 8 PV products (k-step stp = i / 4,
    // tile mt = i % 4), then, with a next block, its 8 score products of chunk
    // c (channel step kc = i - 8); operand of product i of group c
    const uint16_t* kn = sK[buf ^ 1];
    auto opB = [&](int c, int i) {
      if (i < 8)
        return as_vec<vec>(
            *reinterpret_cast<const uint4*>(&sV[buf][(((c * 2 + (i >> 2)) * 2 + hh) * 128 + (i & 3) * 32 + j) * 8]));
      return kop(kn, c, i - 8);
    };
    constexpr int NPR = more ? 16 : 8;   // products per chunk
    auto product = [&](int c, int i, vec op) {
      if (i < 8) {
        const int stp = i >> 2, mt = i & 3;
        const vec A = as_vec<vec>(
            make_uint4(pw[c][4 * stp], pw[c][4 * stp + 1], pw[c][4 * stp + 2], pw[c][4 * stp + 3]));
        of[mt] = MF<F16>::mfma(A, op, of[mt]);
      } else {
        const int kc = i - 8;
        if (kc == 0) {
#pragma unroll
          for (int r = 0; r < 16; ++r) s[c][r] = 0.f;
        }
        s[c] = MF<F16>::mfma(op, qop[kc], s[c]);
      }
    };
#pragma unroll
    for (int r2 = 0; r2 < 8; ++r2) probs(0, r2);
    vec o0 = opB(0, 0), o1 = opB(0, 1);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      // chunk c's products, beside chunk c + 1's probabilities
#pragma unroll
      for (int i = 0; i < NPR; ++i) {
        // the operand two products ahead (into the next chunk's products)
        const int n2 = i + 2;
        const int c2 = n2 < NPR ? c : c + 1, i2 = n2 < NPR ? n2 : n2 - NPR;
        const vec on = c2 < NCH ? opB(c2, i2) : o0;
        product(c, i, o0);
        o0 = o1;
        o1 = on;
        constexpr int PER = NPR / 8;   // products per pair of probabilities
        if (c + 1 < NCH && i % PER == PER - 1) probs(c + 1, i / PER);
      }
      if (c == 0) __builtin_amdgcn_s_setprio(0);
    }
    l = __fmaf_rn(l, alpha, (ls[0] + ls[1]) + (ls[2] + ls[3]));
    tp.load(kbase + blk(jb + 3), vbase + blk(jb + 2), tid);
    __syncthreads();
  };

  using kNo = std::integral_constant<bool, false>;
  using kYes = std::integral_constant<bool, true>;
  for (int jb = 0; jb + 1 < nblocks; ++jb) step(jb, kNo(), kYes());
  step(nblocks - 1, kYes(), kNo());

  // ---- epilogue: O / l ----
  const float ltot = l + __shfl_xor(l, 32);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int qi = 8 * (r >> 2) + 4 * hh + (r & 3);
    const float inv = 1.0f / __shfl(ltot, qi);
    if (q0 + qi < N) {
      const size_t obase = (static_cast<size_t>(bh) * N + q0 + qi) * kD + j;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const float v = of[mt][r] * inv;
        if (a.out_dtype == 2) static_cast<float*>(a.o)[obase + mt * 32] = v;
        else static_cast<uint16_t*>(a.o)[obase + mt * 32] = f2h(v, a.out_dtype == 1);
      }
    }
  }
}

}  // namespace

hipError_t launch_rope16(const RopeTables& t, const uint16_t* x, uint16_t* out, int BH, int N, int Npad, int is_fp16,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_rope16, dim3(Npad / 8, BH), dim3(256), 0, s, t, x, out, N, Npad, is_fp16);
  return hipGetLastError();
}

hipError_t launch_v16_relayout(const uint16_t* v, uint16_t* out, int BH, int N, int Npad, hipStream_t s) {
  hipLaunchKernelGGL(k_v16_relayout, dim3(Npad / 32, BH), dim3(256), 0, s, v, out, N, Npad);
  return hipGetLastError();
}

hipError_t launch_attn_fp16(const Fp16Args& a, int kv_block, hipStream_t s) {
  const dim3 grid(a.Npad / kBlockM, a.BH);
  if (kv_block == 128) {
    if (a.is_fp16) hipLaunchKernelGGL((k_attn16<true, 128>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn16<false, 128>), grid, dim3(256), 0, s, a);
  } else {
    if (a.is_fp16) hipLaunchKernelGGL((k_attn16<true, 64>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_attn16<false, 64>), grid, dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace ra
