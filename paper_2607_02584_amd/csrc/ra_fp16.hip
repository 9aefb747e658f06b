// ra_fp16.hip -- BF16/FP16 fallback attention for gfx950 (the 16-bit path the
// paper keeps for accuracy-sensitive DiT blocks and denoising steps).
//
// Producer: plain 3D RoPE (Sec. 3) of Q and K in binary32, rounded to the
// 16-bit input type, written in a tiled layout that makes every 32-token chunk
// a ready matrix-core operand; V is re-laid out the same way, transposed.
//
// Attention: S^T = K Q^T on v_mfma_f32_32x32x16_{bf16,f16} (fp32 accumulate),
// blockwise online softmax over blocks of 64 keys in ascending order,
//   m = max(m, rowmax(S * Kc)),  P = 2^(S*Kc - m),  l = alpha*l + sum P,
// P rounded to the 16-bit type as the B operand of O^T += V^T P^T, and
// O = O / l.  Each lane holds the scores of one query, so row reductions stay
// inside the lane plus one exchange between the two wave halves.
//
// 16-bit tiled layouts (elements), token n = 32*c + r:
//   Q, K: (((c*8 + ch/16)*2 + (ch/8)%2)*32 + r)*8 + ch%8
//   V:    (((c*2 + s)*2 + h)*128 + ch)*8 + e  holds V[32c + 16s + 8(e/4) + 4h + e%4][ch]
#include "ra_internal.h"

namespace ra {
namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int kKV = 64;       // keys per online-softmax block of the fallback
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
  static __device__ __forceinline__ v16f mfma(vec a, vec b, v16f c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack2(float x, float y) {
    return static_cast<uint32_t>(__bfloat16_as_ushort(__float2bfloat16(x))) |
           (static_cast<uint32_t>(__bfloat16_as_ushort(__float2bfloat16(y))) << 16);
  }
};
template <>
struct MF<true> {
  typedef v8h vec;
  static __device__ __forceinline__ v16f mfma(vec a, vec b, v16f c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack2(float x, float y) {
    return static_cast<uint32_t>(__half_as_ushort(__float2half(x))) |
           (static_cast<uint32_t>(__half_as_ushort(__float2half(y))) << 16);
  }
};

template <typename V>
__device__ __forceinline__ V as_vec(uint4 u) {
  V r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}

template <bool F16>
__global__ __launch_bounds__(256, 2) void k_attn16(Fp16Args a) {
  typedef typename MF<F16>::vec vec;
  constexpr int NCH = kKV / 32;
  __shared__ __align__(16) uint16_t sK[2][kKV * kD];
  __shared__ __align__(16) uint16_t sV[2][kKV * kD];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hh = lane >> 5, j = lane & 31;
  const int bh = blockIdx.y;
  const int qrow = blockIdx.x * kBlockM + wave * 32 + j;
  const int N = a.N;
  const int nblocks = (N + kKV - 1) / kKV;
  const size_t hoff = static_cast<size_t>(bh) * a.Npad * kD;

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

  // block of 64 keys = 2 chunks = 8192 elements of K and of V: 4 x 16 B per thread each
  uint4 stk[4], stv[4];
  auto load = [&](int jb) {
    const uint16_t* kb = a.k + hoff + static_cast<size_t>(jb) * kKV * kD;
    const uint16_t* vb = a.v + hoff + static_cast<size_t>(jb) * kKV * kD;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      stk[i] = *reinterpret_cast<const uint4*>(kb + (i * 256 + tid) * 8);
      stv[i] = *reinterpret_cast<const uint4*>(vb + (i * 256 + tid) * 8);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<uint4*>(&sK[buf][(i * 256 + tid) * 8]) = stk[i];
      *reinterpret_cast<uint4*>(&sV[buf][(i * 256 + tid) * 8]) = stv[i];
    }
  };
  load(0);
  store(0);
  __syncthreads();

  for (int jb = 0; jb < nblocks; ++jb) {
    const int buf = jb & 1;
    const bool more = jb + 1 < nblocks;
    if (more) load(jb + 1);
    const int key0 = jb * kKV;
    const bool last = key0 + kKV > N;

    v16f s[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[ch][r] = 0.f;
#pragma unroll
      for (int kc = 0; kc < 8; ++kc) {
        const vec A = as_vec<vec>(*reinterpret_cast<const uint4*>(&sK[buf][(((ch * 8 + kc) * 2 + hh) * 32 + j) * 8]));
        s[ch] = MF<F16>::mfma(A, qop[kc], s[ch]);
      }
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
        if (!last || key < N) tmax = fmaxf(tmax, __fmul_rn(s[ch][r], a.Kc));
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(m, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) of[mt][r] = __fmul_rn(of[mt][r], alpha);

    float lsum = 0.f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      uint32_t pw[8];
#pragma unroll
      for (int r2 = 0; r2 < 8; ++r2) {
        float P[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int r = 2 * r2 + u;
          const int key = key0 + ch * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
          float p = __builtin_amdgcn_exp2f(__fmaf_rn(s[ch][r], a.Kc, -mnew));
          if (last && key >= N) p = 0.f;
          lsum += p;
          P[u] = p;
        }
        pw[r2] = MF<F16>::pack2(P[0], P[1]);
      }
      // step st uses accumulator registers 8*st .. 8*st+7
#pragma unroll
      for (int stp = 0; stp < 2; ++stp) {
        const vec B = as_vec<vec>(make_uint4(pw[4 * stp], pw[4 * stp + 1], pw[4 * stp + 2], pw[4 * stp + 3]));
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          const vec A =
              as_vec<vec>(*reinterpret_cast<const uint4*>(&sV[buf][(((ch * 2 + stp) * 2 + hh) * 128 + mt * 32 + j) * 8]));
          of[mt] = MF<F16>::mfma(A, B, of[mt]);
        }
      }
    }
    l = __fmaf_rn(l, alpha, lsum);
    if (more) store(buf ^ 1);
    __syncthreads();
  }

  const float ltot = l + __shfl_xor(l, 32);
  if (qrow < N) {
    const float inv = 1.0f / ltot;
    const size_t obase = (static_cast<size_t>(bh) * N + qrow) * kD;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int c0 = mt * 32 + 8 * rq + 4 * hh;
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = of[mt][4 * rq + t] * inv;
        if (a.out_dtype == 2) {
          *reinterpret_cast<float4*>(static_cast<float*>(a.o) + obase + c0) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          const int f16 = a.out_dtype == 1;
          *reinterpret_cast<uint2*>(static_cast<uint16_t*>(a.o) + obase + c0) =
              make_uint2(f2h(v[0], f16) | (static_cast<uint32_t>(f2h(v[1], f16)) << 16),
                         f2h(v[2], f16) | (static_cast<uint32_t>(f2h(v[3], f16)) << 16));
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
  (void)kv_block;
  const dim3 grid(a.Npad / kBlockM, a.BH);
  if (a.is_fp16)
    hipLaunchKernelGGL(k_attn16<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_attn16<false>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ra
