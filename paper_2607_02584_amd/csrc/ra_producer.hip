// ra_producer.hip -- element-wise producer kernels of the INT4 path (gfx950).
//
//  * 3D RoPE with the RoPE-aware rotation (Sec. 3, Sec. 4.1.2 merged
//    interleaved rotation, Sec. 4.1.3 half rotation) in binary32:
//      y0 = fma(x1, g10, x0*g00), y1 = fma(x1, g11, x0*g01)
//    and for the half rotation, on the RoPE output,
//      z(o+2i)   = fma(y(o+i+D_j/2), r10, y(o+i)*r00)
//      z(o+2i+1) = fma(y(o+i+D_j/2), r11, y(o+i)*r01).
//  * The full D x D Hadamard rotation (the "Full" baseline of Sec. 5.3, the
//    Sylvester matrix H_D = H_2 (x) H_{D/2} of Sec. 4.3) after plain RoPE: the
//    Kronecker recursion, widest stride first -- the sums and differences of
//    channels c and c + 64, then c and c + 32 inside each half, ... down to
//    adjacent channels -- unscaled, then one multiply by fl32(1/sqrt 128).
//  * Smoothing (Sec. 4): per-channel means over the tokens of a head (K, V,
//    and Q, whose mean returns as the per-key score bias mu_Q . K_j).  Each
//    value is scaled by 2^20, clamped to +-2^32 and rounded to an integer; the
//    integers are summed in binary64, which is exact (every partial sum is an
//    integer of magnitude at most 2^32 * N <= 2^53), so the sum does not depend
//    on the summation order and the tiles add theirs with atomics.  The
//    consumers derive mu = fl32(sum / (N 2^20)) themselves.
//  * Symmetric INT4 quantization (Sec. 5.1): per group of tokens (Q, K) or per
//    (group of tokens, channel) (V): s = amax/7, code = clamp(rint(z*7/amax)).
//
// Work decomposition: one workgroup of 256 threads per tile of 128 tokens of
// one head.  Thread t handles channels 4*(t%32) .. 4*(t%32)+3 of the rows
// t/32, t/32+8, ... (16 rows), so each row is read as 32 coalesced 8-byte
// pieces.  These kernels are HBM-bound.
#include "ra_internal.h"
#include "rotate_attn.h"

namespace ra {
namespace {

constexpr float kFix = 1048576.0f;     // 2^20
constexpr float kFixLim = 4294967296.0f;  // 2^32

template <bool F16>
__device__ __forceinline__ float h2f(uint16_t b) {
  if (F16) return __half2float(__ushort_as_half(b));
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// floor(n / d) for 0 <= n < 2^24, d >= 1, through binary32 with a correction.
__device__ __forceinline__ int fdiv(int n, int d, float inv_d) {
  int q = static_cast<int>(static_cast<float>(n) * inv_d);
  if (q * d > n) --q;
  if ((q + 1) * d <= n) ++q;
  return q;
}

// Per-thread RoPE setup for its two channel pairs p0 = 2*cl, p1 = 2*cl + 1:
// the axis of each pair and the table column it reads (row stride D_a / 2).
struct PairSetup {
  int axis[2];           // 0 = t, 1 = h, 2 = w
  const float4* tab[2];  // axis table offset by the pair's index in its segment
  int npair[2];          // D_a / 2 (row length of the axis table)
};

__device__ __forceinline__ PairSetup pair_setup(const RopeTables& t, int cl) {
  PairSetup s;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = 2 * cl + i;
    const int n0 = t.split[0] / 2, n1 = t.split[1] / 2;
    const int a = p < n0 ? 0 : (p < n0 + n1 ? 1 : 2);
    const int first = a == 0 ? 0 : (a == 1 ? n0 : n0 + n1);
    s.axis[i] = a;
    s.npair[i] = a == 0 ? n0 : (a == 1 ? n1 : t.split[2] / 2);
    s.tab[i] = (a == 0 ? t.axis[0] : (a == 1 ? t.axis[1] : t.axis[2])) + (p - first);
  }
  return s;
}

// Grid coordinates (t, h, w) of the tile's 128 tokens, one thread each, into
// LDS (rows past N take the last token's).
__device__ __forceinline__ void tile_positions(const RopeTables& t, int tile, int N, int (*pos)[4]) {
  const int tid = threadIdx.x;
  if (tid < kTile) {
    const int W = t.grid[2], Hg = t.grid[1];
    int n = tile * kTile + tid;
    if (n >= N) n = N - 1;
    const int tq = fdiv(n, W * Hg, 1.0f / static_cast<float>(W * Hg));
    const int rem = n - tq * W * Hg;
    const int hq = fdiv(rem, W, 1.0f / static_cast<float>(W));
    pos[tid][0] = tq;
    pos[tid][1] = hq;
    pos[tid][2] = rem - hq * W;
  }
}

// Half rotation: for output pair P the two RoPE channels it mixes.
struct HalfSetup {
  int ia[2], ib[2];
  float4 r[2];
};

__device__ __forceinline__ HalfSetup half_setup(const RopeTables& t, int cl) {
  HalfSetup s;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int P = 2 * cl + i;
    int o = 0, a = 0;
    for (int ax = 0; ax < 3; ++ax) {
      if (P >= o / 2 && P < (o + t.split[ax]) / 2) a = ax;
      o += t.split[ax];
    }
    o = 0;
    for (int ax = 0; ax < a; ++ax) o += t.split[ax];
    int ii = P - o / 2;
    s.ia[i] = o + ii;
    s.ib[i] = o + ii + t.split[a] / 2;
    s.r[i] = t.rot[P];
  }
  return s;
}

// y <- y H_128 for one row held by 32 lanes (lane cl holds channels 4cl..4cl+3):
// strides 64..4 pair lanes whose cl differs in bit 4..0 (the lane with the bit
// set takes the difference), strides 2 and 1 stay inside the thread.
__device__ __forceinline__ void hadamard_row(float y[4], int cl) {
#pragma unroll
  for (int m = 16; m >= 1; m >>= 1) {
    const bool upper = (cl & m) != 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const float o = __shfl_xor(y[c], m, 32);
      y[c] = upper ? __fsub_rn(o, y[c]) : __fadd_rn(y[c], o);
    }
  }
  const float t0 = __fadd_rn(y[0], y[2]), t2 = __fsub_rn(y[0], y[2]);
  const float t1 = __fadd_rn(y[1], y[3]), t3 = __fsub_rn(y[1], y[3]);
  y[0] = __fmul_rn(__fadd_rn(t0, t1), kInvSqrtD);
  y[1] = __fmul_rn(__fsub_rn(t0, t1), kInvSqrtD);
  y[2] = __fmul_rn(__fadd_rn(t2, t3), kInvSqrtD);
  y[3] = __fmul_rn(__fsub_rn(t2, t3), kInvSqrtD);
}

// Computes the rotated values z of the thread's 4 channels for the 16 rows of
// the tile.  Rows beyond N give zeros.  ybuf: [8][128] floats of LDS.
// ROT: RA_ROT_HALF, RA_ROT_HADAMARD, or 0 for the table-only forms (none, merged
// interleaved); F16: binary16 inputs (else bfloat16).
template <int ROT, bool F16>
__device__ __forceinline__ void rope_tile(const RopeTables& t, const QkArgs& a, int bh, int tile, float (*ybuf)[kD],
                                          float z[16][4]) {
  __shared__ int pos[kTile][4];
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
  const PairSetup ps = pair_setup(t, cl);
  constexpr bool half = ROT == RA_ROT_HALF;
  constexpr bool full = ROT == RA_ROT_HADAMARD;
  HalfSetup hs;
  if constexpr (half) hs = half_setup(t, cl);
  tile_positions(t, tile, a.N, pos);
  const uint16_t* xb = a.x + static_cast<size_t>(bh) * a.N * kD;
  // all sixteen row loads first (rows past N re-read the last row and are zeroed)
  uint2 raw[16];
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int n = tile * kTile + p * 8 + rr;
    raw[p] = *reinterpret_cast<const uint2*>(xb + static_cast<size_t>(n < a.N ? n : a.N - 1) * kD + 4 * cl);
  }
  __syncthreads();
  // without the half rotation's per-row barriers, the table entries of eight
  // rows are fetched before any of them is used, so their loads overlap
  // instead of waiting one row at a time
  float4 gt[8][2];
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int nl = p * 8 + rr, n = tile * kTile + nl;
    if (!half && (p & 7) == 0) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
#pragma unroll
        for (int i = 0; i < 2; ++i) gt[q][i] = ps.tab[i][pos[(p + q) * 8 + rr][ps.axis[i]] * ps.npair[i]];
    }
    float y[4] = {0.f, 0.f, 0.f, 0.f};
    if (n < a.N) {
      const float x[4] = {h2f<F16>(static_cast<uint16_t>(raw[p].x & 0xffff)),
                          h2f<F16>(static_cast<uint16_t>(raw[p].x >> 16)),
                          h2f<F16>(static_cast<uint16_t>(raw[p].y & 0xffff)),
                          h2f<F16>(static_cast<uint16_t>(raw[p].y >> 16))};
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const float4 g = half ? ps.tab[i][pos[nl][ps.axis[i]] * ps.npair[i]] : gt[p & 7][i];
        const float x0 = x[2 * i], x1 = x[2 * i + 1];
        y[2 * i] = __fmaf_rn(x1, g.z, __fmul_rn(x0, g.x));
        y[2 * i + 1] = __fmaf_rn(x1, g.w, __fmul_rn(x0, g.y));
      }
    }
    if constexpr (half) {
      __syncthreads();
      *reinterpret_cast<float4*>(&ybuf[rr][4 * cl]) = make_float4(y[0], y[1], y[2], y[3]);
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const float av = ybuf[rr][hs.ia[i]], bv = ybuf[rr][hs.ib[i]];
        const float4 r = hs.r[i];
        y[2 * i] = __fmaf_rn(bv, r.z, __fmul_rn(av, r.x));
        y[2 * i + 1] = __fmaf_rn(bv, r.w, __fmul_rn(av, r.y));
      }
      if (n >= a.N) y[0] = y[1] = y[2] = y[3] = 0.f;
    } else if constexpr (full) {
      hadamard_row(y, cl);  // rows past N are zero and stay zero
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) z[p][c] = y[c];
  }
}

__device__ __forceinline__ double fixq(float v) {
  float s = __fmul_rn(v, kFix);
  s = fminf(fmaxf(s, -kFixLim), kFixLim);
  return static_cast<double>(__builtin_rintf(s));
}

// Reduces the per-thread fixed-point sums over the 8 row groups and adds the
// tile's channel sums to the head's [128] (binary64 integers, exact in any order).
__device__ __forceinline__ void add_sums(double acc[4], double* out) {
  __shared__ double red[8][kD];
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
#pragma unroll
  for (int c = 0; c < 4; ++c) red[rr][4 * cl + c] = acc[c];
  __syncthreads();
  if (tid < kD) {
    double s = 0.0;
#pragma unroll
    for (int r = 0; r < 8; ++r) s += red[r][tid];
    unsafeAtomicAdd(out + tid, s);
  }
}

// mu of channels 4 cl .. 4 cl + 3 of a head from its fixed-point sums
__device__ __forceinline__ float4 mean4(const double* sums, int N, int cl) {
  const double den = static_cast<double>(N) * 1048576.0;
  return make_float4(static_cast<float>(sums[4 * cl] / den), static_cast<float>(sums[4 * cl + 1] / den),
                     static_cast<float>(sums[4 * cl + 2] / den), static_cast<float>(sums[4 * cl + 3] / den));
}

template <int ROT, bool F16>
__global__ __launch_bounds__(256) void k_qk_sums(RopeTables t, QkArgs a) {
  __shared__ float ybuf[8][kD];
  const int tile = blockIdx.x, bh = blockIdx.y;
  float z[16][4];
  rope_tile<ROT, F16>(t, a, bh, tile, ybuf, z);
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int p = 0; p < 16; ++p)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] += fixq(z[p][c]);
  add_sums(acc, a.sums + static_cast<size_t>(bh) * kD);
}

// 6-bit E2M3 float (sign bit 5, exponent bias 1, 3 mantissa bits) equal to the
// integer code c in [-7, 7]: 1 = 1.0 x 2^0, 2 = 1.0 x 2^1, 3 = 1.1b x 2^1, 4..7 = 1.xx0b x 2^2.
__device__ __forceinline__ uint32_t e2m3_of(int c) {
  const uint32_t mag = static_cast<uint32_t>(c < 0 ? -c : c);
  // magnitudes 0..7 -> 00 08 10 14 18 1A 1C 1E, packed as nibble pairs of a 64-bit table
  const uint64_t tab = 0x1E1C1A1814100800ull;
  const uint32_t v = static_cast<uint32_t>((tab >> (8 * mag)) & 0xFF);
  return c < 0 ? (v | 0x20u) : v;
}

__device__ __forceinline__ int qcode(float z, float inv) {
  float c = __builtin_rintf(__fmul_rn(z, inv));
  c = fminf(fmaxf(c, -7.0f), 7.0f);
  return static_cast<int>(c);
}

template <int ROT, bool F16>
__global__ __launch_bounds__(256) void k_qk_quant(RopeTables t, QkArgs a) {
  __shared__ float ybuf[8][kD];
  __shared__ float rowmax[kTile];
  __shared__ float ginv[kTile];
  __shared__ __align__(16) uint8_t ctile[kTile * 96];
  const int tile = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
  float z[16][4];
  rope_tile<ROT, F16>(t, a, bh, tile, ybuf, z);
  if (a.center) {
    const float4 m = mean4(a.sums + static_cast<size_t>(bh) * kD, a.N, cl);
    if (a.mu_out && tile == 0 && rr == 0) *reinterpret_cast<float4*>(a.mu_out + bh * kD + 4 * cl) = m;
    for (int p = 0; p < 16; ++p) {
      const int n = tile * kTile + p * 8 + rr;
      if (n < a.N) {
        z[p][0] = __fsub_rn(z[p][0], m.x);
        z[p][1] = __fsub_rn(z[p][1], m.y);
        z[p][2] = __fsub_rn(z[p][2], m.z);
        z[p][3] = __fsub_rn(z[p][3], m.w);
      }
    }
  }
  if (a.bias) {
    // Q smoothing: per-key score bias b = mu_Q . z (z = this K row after its
    // own smoothing), products in binary32, summed pairwise over the channel
    // range: the thread's (c0 + c1) + (c2 + c3), then lanes 1, 2, 4, 8, 16
    // apart (blocks of 8, 16, ..., 128 channels).  Padded rows give 0.
    const float4 mq = mean4(a.qsums + static_cast<size_t>(bh) * kD, a.N, cl);
    for (int p = 0; p < 16; ++p) {
      float b = __fadd_rn(__fadd_rn(__fmul_rn(mq.x, z[p][0]), __fmul_rn(mq.y, z[p][1])),
                          __fadd_rn(__fmul_rn(mq.z, z[p][2]), __fmul_rn(mq.w, z[p][3])));
#pragma unroll
      for (int off = 1; off <= 16; off <<= 1) b = __fadd_rn(b, __shfl_xor(b, off, 32));
      if (cl == 0) a.bias[static_cast<size_t>(bh) * a.Npad + tile * kTile + p * 8 + rr] = b;
    }
  }
  // row abs-max over the 128 channels (32 threads of the row)
  for (int p = 0; p < 16; ++p) {
    float v = fmaxf(fmaxf(fabsf(z[p][0]), fabsf(z[p][1])), fmaxf(fabsf(z[p][2]), fabsf(z[p][3])));
#pragma unroll
    for (int off = 16; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 32));
    if (cl == 0) rowmax[p * 8 + rr] = v;
  }
  __syncthreads();
  const int g = a.group, ng = kTile / g;
  if (tid < ng) {
    float m = 0.f;
    for (int i = 0; i < g; ++i) m = fmaxf(m, rowmax[tid * g + i]);
    float s = 0.f, inv = 0.f;
    if (m > 0.f) {
      s = __fdiv_rn(m, 7.0f);
      inv = __fdiv_rn(7.0f, m);
    }
    ginv[tid] = inv;
    a.scales[static_cast<size_t>(bh) * (a.Npad / g) + tile * ng + tid] = s;
  }
  __syncthreads();
  if (a.e2m3) {
    // record ((chunk*2 + ch/64)*2 + (ch/32)%2)*32 + row of 24 bytes; channels 4cl..4cl+3 are the
    // 6-bit fields 4*(cl%8) .. +3 of record (kc = cl/16, h = (cl/8)%2), i.e. bytes 3*(cl%8) .. +2
    for (int p = 0; p < 16; ++p) {
      const int nl = p * 8 + rr;
      const float inv = ginv[nl / g];
      const uint32_t bits = e2m3_of(qcode(z[p][0], inv)) | (e2m3_of(qcode(z[p][1], inv)) << 6) |
                            (e2m3_of(qcode(z[p][2], inv)) << 12) | (e2m3_of(qcode(z[p][3], inv)) << 18);
      const int rec = (((nl >> 5) * 2 + (cl >> 4)) * 2 + ((cl >> 3) & 1)) * 32 + (nl & 31);
      uint8_t* d = &ctile[rec * 24 + 3 * (cl & 7)];
      d[0] = static_cast<uint8_t>(bits);
      d[1] = static_cast<uint8_t>(bits >> 8);
      d[2] = static_cast<uint8_t>(bits >> 16);
    }
    __syncthreads();
    uint8_t* dst = a.codes + static_cast<size_t>(bh) * a.Npad * 96 + static_cast<size_t>(tile) * kTile * 96;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int o = (i * 256 + tid) * 16;
      *reinterpret_cast<uint4*>(dst + o) = *reinterpret_cast<const uint4*>(&ctile[o]);
    }
    return;
  }
  for (int p = 0; p < 16; ++p) {
    const int nl = p * 8 + rr;
    const float inv = ginv[nl / g];
    const int c0 = qcode(z[p][0], inv), c1 = qcode(z[p][1], inv);
    const int c2 = qcode(z[p][2], inv), c3 = qcode(z[p][3], inv);
    const uint32_t b0 = (c0 & 0xF) | ((c1 & 0xF) << 4);
    const uint32_t b1 = (c2 & 0xF) | ((c3 & 0xF) << 4);
    // tiled layout: ((chunk*8 + unit)*32 + row)*8 + byte, pair j = 2*cl -> unit cl/4, byte 2*(cl%4)
    const int off = (((nl >> 5) * 8 + (cl >> 2)) * 32 + (nl & 31)) * 8 + 2 * (cl & 3);
    *reinterpret_cast<uint16_t*>(&ctile[off]) = static_cast<uint16_t>(b0 | (b1 << 8));
  }
  __syncthreads();
  uint8_t* dst = a.codes + static_cast<size_t>(bh) * a.Npad * 64 + static_cast<size_t>(tile) * kTile * 64;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int o = (i * 256 + tid) * 16;
    *reinterpret_cast<uint4*>(dst + o) = *reinterpret_cast<const uint4*>(&ctile[o]);
  }
}

// ------------------------------------------------------------------ V --

template <bool F16, bool VHAD>
__device__ __forceinline__ void load_v_tile(const VArgs& a, int bh, int tile, float z[16][4]) {
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
  const uint16_t* xb = a.x + static_cast<size_t>(bh) * a.N * kD;
  float4 m = make_float4(0.f, 0.f, 0.f, 0.f);
  if (a.center) m = mean4(a.sums + static_cast<size_t>(bh) * kD, a.N, cl);
  uint2 raw[16];
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int n = tile * kTile + p * 8 + rr;
    raw[p] = *reinterpret_cast<const uint2*>(xb + static_cast<size_t>(n < a.N ? n : a.N - 1) * kD + 4 * cl);
  }
  for (int p = 0; p < 16; ++p) {
    const int n = tile * kTile + p * 8 + rr;
    float x[4] = {0.f, 0.f, 0.f, 0.f};
    if (n < a.N) {
      x[0] = h2f<F16>(static_cast<uint16_t>(raw[p].x & 0xffff));
      x[1] = h2f<F16>(static_cast<uint16_t>(raw[p].x >> 16));
      x[2] = h2f<F16>(static_cast<uint16_t>(raw[p].y & 0xffff));
      x[3] = h2f<F16>(static_cast<uint16_t>(raw[p].y >> 16));
    }
    // online V rotation (Sec. 4.3): the row times H, before smoothing
    if constexpr (VHAD) hadamard_row(x, cl);
    if (n < a.N && a.center) {
      x[0] = __fsub_rn(x[0], m.x);
      x[1] = __fsub_rn(x[1], m.y);
      x[2] = __fsub_rn(x[2], m.z);
      x[3] = __fsub_rn(x[3], m.w);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) z[p][c] = x[c];
  }
}

template <bool F16, bool VHAD>
__global__ __launch_bounds__(256) void k_v_sums(VArgs a) {
  const int tile = blockIdx.x, bh = blockIdx.y;
  float z[16][4];
  load_v_tile<F16, VHAD>(a, bh, tile, z);
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int p = 0; p < 16; ++p)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] += fixq(z[p][c]);
  add_sums(acc, a.sums + static_cast<size_t>(bh) * kD);
}

__device__ __forceinline__ int vgroup_of(const VArgs& a, int n) {
  int g = n / a.group;
  return g < a.ngroups ? g : a.ngroups - 1;
}

// Per (tile half, channel) abs-max, merged into the group maxima with an
// order-independent atomic max on the float bits (values are >= 0).
template <bool F16, bool VHAD>
__global__ __launch_bounds__(256) void k_v_amax(VArgs a) {
  __shared__ float red[8][2][kD];
  const int tile = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
  float z[16][4];
  load_v_tile<F16, VHAD>(a, bh, tile, z);
  float m[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  for (int p = 0; p < 16; ++p)
#pragma unroll
    for (int c = 0; c < 4; ++c) m[p >> 3][c] = fmaxf(m[p >> 3][c], fabsf(z[p][c]));
#pragma unroll
  for (int hf = 0; hf < 2; ++hf)
#pragma unroll
    for (int c = 0; c < 4; ++c) red[rr][hf][4 * cl + c] = m[hf][c];
  __syncthreads();
  const int hf = tid >> 7, ch = tid & 127;
  const int n0 = tile * kTile + hf * 64;
  if (n0 < a.N) {
    float v = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) v = fmaxf(v, red[r][hf][ch]);
    const int g = vgroup_of(a, n0);
    atomicMax(a.amax + (static_cast<size_t>(bh) * a.ngroups + g) * kD + ch, __float_as_uint(v));
  }
}

template <bool F16, bool VHAD>
__global__ __launch_bounds__(256) void k_v_quant(VArgs a) {
  __shared__ __align__(16) uint8_t ctile[kTile * 96];
  __shared__ float ginv[2][kD];
  __shared__ float red[8][2][kD];
  const int tile = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
  float z[16][4];
  if (a.local_amax) {
    // groups of 64 or 128 tokens lie inside this tile: their maxima come from
    // the tile itself, per (tile half, channel) as in k_v_amax
    load_v_tile<F16, VHAD>(a, bh, tile, z);
    float mh[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    for (int p = 0; p < 16; ++p)
#pragma unroll
      for (int c = 0; c < 4; ++c) mh[p >> 3][c] = fmaxf(mh[p >> 3][c], fabsf(z[p][c]));
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int c = 0; c < 4; ++c) red[rr][hf][4 * cl + c] = mh[hf][c];
    __syncthreads();
  }
  {
    const int hf = tid >> 7, ch = tid & 127;
    const int n0 = tile * kTile + hf * 64;
    const int g = vgroup_of(a, n0 < a.N ? n0 : a.N - 1);
    float m;
    if (a.local_amax) {
      float m0 = 0.f, m1 = 0.f;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        m0 = fmaxf(m0, red[r][0][ch]);
        m1 = fmaxf(m1, red[r][1][ch]);
      }
      m = a.group == 64 ? (hf ? m1 : m0) : fmaxf(m0, m1);
    } else {
      m = __uint_as_float(a.amax[(static_cast<size_t>(bh) * a.ngroups + g) * kD + ch]);
    }
    float s = 0.f, inv = 0.f;
    if (m > 0.f) {
      s = __fdiv_rn(m, 7.0f);
      inv = __fdiv_rn(7.0f, m);
    }
    ginv[hf][ch] = inv;
    // the tile half holding the first token of group g writes its scales
    if (n0 < a.N && g * a.group >= n0 && g * a.group < n0 + 64)
      a.scales[(static_cast<size_t>(bh) * a.ngroups + g) * kD + ch] = s;
  }
  __syncthreads();
  if (a.center && a.mu_out && tile == 0 && rr == 0)
    *reinterpret_cast<float4*>(a.mu_out + bh * kD + 4 * cl) = mean4(a.sums + static_cast<size_t>(bh) * kD, a.N, cl);
  if (!a.local_amax) load_v_tile<F16, VHAD>(a, bh, tile, z);
  if (a.e2m3) {
    // group of 64 tokens gl = p/8, kappa = (p%8)*8 + rr, half h = (rr/4)%2; token kappa of a channel is
    // field 8*((kappa%32)/8) + 2*(kappa%4) + kappa/32 of record ((gl*4 + ch/32)*2 + h)*32 + ch%32.
    // The thread's codes for passes q and q+4 (q = p%4) are the adjacent fields 8q + 2*(rr%4) and
    // +1: a 12-bit piece at bit 48q + 12*(rr%4); pieces are merged into LDS with atomic OR.
    uint32_t* cw = reinterpret_cast<uint32_t*>(ctile);
    for (int i = tid; i < kTile * 96 / 4; i += 256) cw[i] = 0u;
    __syncthreads();
    const int s4 = rr & 3, hh = (rr >> 2) & 1;
#pragma unroll
    for (int gl = 0; gl < 2; ++gl) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int ch = 4 * cl + c;
        const float inv = ginv[gl][ch];
        const int rec = ((gl * 4 + (ch >> 5)) * 2 + hh) * 32 + (ch & 31);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t piece = e2m3_of(qcode(z[gl * 8 + q][c], inv)) | (e2m3_of(qcode(z[gl * 8 + q + 4][c], inv)) << 6);
          const int b = 48 * q + 12 * s4;
          const int w = rec * 6 + (b >> 5), sh = b & 31;
          atomicOr(&cw[w], piece << sh);
          if (sh > 20) atomicOr(&cw[w + 1], piece >> (32 - sh));
        }
      }
    }
    __syncthreads();
    uint8_t* dst = a.codes + static_cast<size_t>(bh) * a.Npad * 96 + static_cast<size_t>(tile) * kTile * 96;
#pragma unroll
    for (int i = 0; i < 3; ++i) {
      const int o = (i * 256 + tid) * 16;
      *reinterpret_cast<uint4*>(dst + o) = *reinterpret_cast<const uint4*>(&ctile[o]);
    }
    return;
  }
  // token kappa = (p%4)*8 + rr inside chunk p/4; nibble np = 8*(kappa/16) + 2*(kappa%4) + (kappa/8)%2,
  // half h = (kappa/4)%2; byte ((chunk*2 + h)*128 + ch)*8 + np/2.  Passes p and p+1 (p even)
  // share every byte (np differs in its low bit only).
  for (int p = 0; p < 16; p += 2) {
    const int chunk = p >> 2;
    const int kap = (p & 3) * 8 + rr;
    const int np = 8 * (kap >> 4) + 2 * (kap & 3);  // even nibble (pass p), odd = pass p+1
    const int hh = (kap >> 2) & 1;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int ch = 4 * cl + c;
      const float inv = ginv[(p * 8) >= 64 ? 1 : 0][ch];
      const int lo = qcode(z[p][c], inv), hi = qcode(z[p + 1][c], inv);
      ctile[((chunk * 2 + hh) * kD + ch) * 8 + (np >> 1)] = static_cast<uint8_t>((lo & 0xF) | ((hi & 0xF) << 4));
    }
  }
  __syncthreads();
  uint8_t* dst = a.codes + static_cast<size_t>(bh) * a.Npad * 64 + static_cast<size_t>(tile) * kTile * 64;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int o = (i * 256 + tid) * 16;
    *reinterpret_cast<uint4*>(dst + o) = *reinterpret_cast<const uint4*>(&ctile[o]);
  }
}

// Up to kChunkFloats binary32 values carried in the kernel arguments and
// written to dst[off .. off + n): moves a host table to the device without a
// host staging buffer or a copy engine.
constexpr int kChunkFloats = 960;
struct FloatChunk {
  float v[kChunkFloats];
  int off, n;
};

__global__ __launch_bounds__(256) void k_write_floats(FloatChunk c, float* dst) {
  for (int i = threadIdx.x; i < c.n; i += 256) dst[c.off + i] = c.v[i];
}

// dst[i] = src[i] for i < n; src may be pinned host memory read through its
// device mapping, so a host table reaches the device on the kernel queue
// itself, ordered with the kernels around it and with no copy engine involved
__global__ __launch_bounds__(256) void k_copy_u32(const uint32_t* __restrict__ src, uint32_t* __restrict__ dst,
                                                  int64_t n) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    dst[i] = src[i];
}

__global__ void k_fill_zero_u32(uint32_t* p, int64_t n) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = 0u;
}

}  // namespace

// the rotation and input type as template arguments: table-only rotations share one form
#define RA_QK_DISPATCH(KERNEL)                                                                        \
  do {                                                                                                \
    const dim3 g(a.Npad / kTile, BH);                                                                 \
    const int rot = (t.rotation == RA_ROT_HALF || t.rotation == RA_ROT_HADAMARD) ? t.rotation : 0;    \
    if (rot == RA_ROT_HALF) {                                                                         \
      if (a.is_fp16) hipLaunchKernelGGL((KERNEL<RA_ROT_HALF, true>), g, dim3(256), 0, s, t, a);        \
      else hipLaunchKernelGGL((KERNEL<RA_ROT_HALF, false>), g, dim3(256), 0, s, t, a);                 \
    } else if (rot == RA_ROT_HADAMARD) {                                                              \
      if (a.is_fp16) hipLaunchKernelGGL((KERNEL<RA_ROT_HADAMARD, true>), g, dim3(256), 0, s, t, a);    \
      else hipLaunchKernelGGL((KERNEL<RA_ROT_HADAMARD, false>), g, dim3(256), 0, s, t, a);             \
    } else {                                                                                          \
      if (a.is_fp16) hipLaunchKernelGGL((KERNEL<0, true>), g, dim3(256), 0, s, t, a);                  \
      else hipLaunchKernelGGL((KERNEL<0, false>), g, dim3(256), 0, s, t, a);                           \
    }                                                                                                 \
  } while (0)

#define RA_V_DISPATCH(KERNEL)                                                                         \
  do {                                                                                                \
    const dim3 g(a.Npad / kTile, BH);                                                                 \
    if (a.is_fp16) {                                                                                  \
      if (a.vhad) hipLaunchKernelGGL((KERNEL<true, true>), g, dim3(256), 0, s, a);                     \
      else hipLaunchKernelGGL((KERNEL<true, false>), g, dim3(256), 0, s, a);                           \
    } else {                                                                                          \
      if (a.vhad) hipLaunchKernelGGL((KERNEL<false, true>), g, dim3(256), 0, s, a);                    \
      else hipLaunchKernelGGL((KERNEL<false, false>), g, dim3(256), 0, s, a);                          \
    }                                                                                                 \
  } while (0)

hipError_t launch_qk_sums(const RopeTables& t, const QkArgs& a, int BH, hipStream_t s) {
  RA_QK_DISPATCH(k_qk_sums);
  return hipGetLastError();
}

hipError_t launch_qk_quant(const RopeTables& t, const QkArgs& a, int BH, hipStream_t s) {
  RA_QK_DISPATCH(k_qk_quant);
  return hipGetLastError();
}

hipError_t launch_write_floats(const float* host, size_t n, float* dst, hipStream_t s) {
  for (size_t o = 0; o < n; o += kChunkFloats) {
    FloatChunk c;
    c.off = static_cast<int>(o);
    c.n = static_cast<int>(n - o < static_cast<size_t>(kChunkFloats) ? n - o : kChunkFloats);
    for (int i = 0; i < c.n; ++i) c.v[i] = host[o + i];
    hipLaunchKernelGGL(k_write_floats, dim3(1), dim3(256), 0, s, c, dst);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_copy_u32(const uint32_t* src, uint32_t* dst, int64_t n, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_copy_u32, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_fill_zero_u32(uint32_t* p, int64_t n, hipStream_t s) {
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_fill_zero_u32, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_v_sums(const VArgs& a, int BH, hipStream_t s) {
  RA_V_DISPATCH(k_v_sums);
  return hipGetLastError();
}

hipError_t launch_v_amax(const VArgs& a, int BH, hipStream_t s) {
  RA_V_DISPATCH(k_v_amax);
  return hipGetLastError();
}

hipError_t launch_v_quant(const VArgs& a, int BH, hipStream_t s) {
  RA_V_DISPATCH(k_v_quant);
  return hipGetLastError();
}

}  // namespace ra
