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
// one head.  Q/K: thread t handles channels 32*(t%4) .. +31 of the rows
// t/4 + 64p (p = 0, 1), each row read as four 64-byte pieces, with the RoPE
// table rows the tile needs staged in LDS.  V: thread t handles channels
// 4*(t%32) .. +3 of the rows t/32 + 8p (16 rows), each row read as 32 8-byte
// pieces.  A pass is bound by its HBM traffic and by the per-element vector
// work (RoPE, rotation, quantization, packing) together: the jobs of one
// pass share one grid, one job after another in the grid's order (one launch,
// and the end of one job overlaps the start of the next; taking the jobs in
// turn block by block was slower).
#include <type_traits>

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


__device__ __forceinline__ double fixq(float v) {
  float s = __fmul_rn(v, kFix);
  s = fminf(fmaxf(s, -kFixLim), kFixLim);
  return static_cast<double>(__builtin_rintf(s));
}

// Reduces the per-thread fixed-point sums over the 8 row groups and adds the
// tile's channel sums to the head's [128] (binary64 integers, exact in any order).
// red: 8 x 128 binary64 of LDS.
__device__ __forceinline__ void add_sums(double acc[4], double* out, double* red) {
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
#pragma unroll
  for (int c = 0; c < 4; ++c) red[rr * kD + 4 * cl + c] = acc[c];
  __syncthreads();
  if (tid < kD) {
    double s = 0.0;
#pragma unroll
    for (int r = 0; r < 8; ++r) s += red[r * kD + tid];
    unsafeAtomicAdd(out + tid, s);
  }
}

// mu of channels 4 cl .. 4 cl + 3 of a head from its fixed-point sums
__device__ __forceinline__ float4 mean4(const double* sums, int N, int cl) {
  const double den = static_cast<double>(N) * 1048576.0;
  return make_float4(static_cast<float>(sums[4 * cl] / den), static_cast<float>(sums[4 * cl + 1] / den),
                     static_cast<float>(sums[4 * cl + 2] / den), static_cast<float>(sums[4 * cl + 3] / den));
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


// ------------------------------------------------------------------ Q/K --
// Thread (r64, c4) = (tid / 4, tid % 4) holds channels 32 c4 .. 32 c4 + 31
// (pairs 16 c4 .. 16 c4 + 15) of the tile rows 64 p + r64, p = 0, 1: a row is
// read as four 64-byte pieces, its abs-max and bias sums cross 4 lanes only,
// and the thread's 32 codes of a row are one whole 24-byte E2M3 record (or two
// 8-byte units of the nibble container), written straight from registers.
constexpr int kQkPasses = 2;

// The table rows a tile reads, staged in LDS.  For axis a the tile's tokens n
// have the running index lin = n / div_a (div = W*Hg, W, 1) and the position
// lin mod extent_a; the tile's lin values are consecutive.  When there are at
// most extent_a of them, staged row lin - lin0 holds their position; otherwise
// every position occurs and staged row pos holds position pos.
struct StagePlan {
  int base[3];   // float4 index of axis a's first staged row
  int lin0[3];   // lin of the tile's first token
  int bypos[3];  // rows indexed by position
  int total;     // float4 count
};

__device__ __forceinline__ StagePlan stage_plan(const RopeTables& t, int n0, int N) {
  StagePlan s;
  const int W = t.grid[2], HW = t.grid[1] * t.grid[2];
  const int nlast = (n0 + kTile - 1 < N - 1) ? n0 + kTile - 1 : N - 1;
  int acc = 0;
#pragma unroll
  for (int ax = 0; ax < 3; ++ax) {
    const int div = ax == 0 ? HW : (ax == 1 ? W : 1);
    s.lin0[ax] = n0 / div;
    const int cnt = nlast / div - s.lin0[ax] + 1;
    s.bypos[ax] = cnt > t.grid[ax];
    s.base[ax] = acc;
    acc += (s.bypos[ax] ? t.grid[ax] : cnt) * (t.split[ax] / 2);
  }
  s.total = acc;
  return s;
}

// Upper bound of StagePlan::total over all tiles of a geometry (host side).
inline int stage_bound(const RopeTables& t) {
  const int div[3] = {t.grid[1] * t.grid[2], t.grid[2], 1};
  int acc = 0;
  for (int ax = 0; ax < 3; ++ax) {
    int rows = div[ax] == 1 ? kTile : (kTile - 1) / div[ax] + 2;
    if (rows > t.grid[ax]) rows = t.grid[ax];
    acc += rows * (t.split[ax] / 2);
  }
  return acc;
}

constexpr int kStageMaxF4 = 2560;  // 40 KB per stage buffer; larger plans read the tables in place

// 16 bytes per lane from global memory straight into LDS at m0 + 16 * lane
// (m0 = the wave-uniform LDS address of dst).  Issued from asm, so the
// compiler does not wait for it at unrelated LDS accesses; the item loop waits
// for it explicitly (vmcnt(0) and a barrier) before the rows are read.
__device__ __forceinline__ void dma16(const void* src, void* dst) {
#if defined(__HIP_DEVICE_COMPILE__)
  const unsigned lds =
      static_cast<unsigned>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) uint8_t*)(dst)));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds))
               : "m0", "memory");
#else
  (void)src;
  (void)dst;
#endif
}

// Starts the copy of the table rows of the tile at n0 into buf (stage_plan's
// layout).  The axis of an entry is a run-time value, so its fields are picked
// with selects: indexing the small arrays with it would put them in scratch.
__device__ __forceinline__ void stage_rows(const RopeTables& t, int n0, int N, float4* buf) {
  const StagePlan sp = stage_plan(t, n0, N);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int i0 = 64 * wv; i0 < sp.total; i0 += 256) {
    const int i = i0 + lane;
    if (i < sp.total) {
      const bool a2 = i >= sp.base[2], a1 = !a2 && i >= sp.base[1];
      const int np = (a2 ? t.split[2] : (a1 ? t.split[1] : t.split[0])) / 2;
      const int loc = i - (a2 ? sp.base[2] : (a1 ? sp.base[1] : sp.base[0]));
      const int s = loc / np, k = loc - s * np;
      const bool bypos = a2 ? sp.bypos[2] : (a1 ? sp.bypos[1] : sp.bypos[0]);
      const int lin0 = a2 ? sp.lin0[2] : (a1 ? sp.lin0[1] : sp.lin0[0]);
      const int extent = a2 ? t.grid[2] : (a1 ? t.grid[1] : t.grid[0]);
      const int pos = bypos ? s : (lin0 + s) % extent;
      const float4* tab = a2 ? t.axis[2] : (a1 ? t.axis[1] : t.axis[0]);
      dma16(tab + pos * np + k, buf + i0);
    }
  }
}

// Starts the loads of the thread's row pieces of the tile at n0 (rows past N
// re-read the last row; rope_item zeroes them).
__device__ __forceinline__ void load_rows(const uint16_t* xb, int n0, int N, uint4 (&raw)[kQkPasses][4]) {
  const int r64 = threadIdx.x >> 2, c4 = threadIdx.x & 3;
#pragma unroll
  for (int p = 0; p < kQkPasses; ++p) {
    const int n = n0 + 64 * p + r64;
    const uint4* src = reinterpret_cast<const uint4*>(xb + static_cast<size_t>(n < N ? n : N - 1) * kD + 32 * c4);
#pragma unroll
    for (int i = 0; i < 4; ++i) raw[p][i] = src[i];
  }
}

// v of lane ^ M (M = 1 or 2): DPP quad permutations, register moves
template <int M>
__device__ __forceinline__ float quad_xor(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), M == 1 ? 0xB1 : 0x4E, 0xF, 0xF, false));
}

// Wave-wide lane mask of the lanes with (lane mod 4) < n, n >= 0.
__device__ __forceinline__ uint64_t lanes_c4_below(int n) {
  const uint32_t nib = (1u << (n < 4 ? n : 4)) - 1u;
  const uint32_t half = nib * 0x11111111u;
  return (static_cast<uint64_t>(half) << 32) | half;
}

// The thread's two rows of the tile at n0 after RoPE and the rotation:
// z[p][c] is channel 32 c4 + c of tile row 64 p + r64 (zero for rows past N).
// STAGED: table rows from LDS (st, stage_plan's layout), else straight from the
// tables.  ROT: RA_ROT_HALF, RA_ROT_HADAMARD, or 0 for the table-only forms
// (none, merged interleaved); F16: binary16 inputs (else bfloat16).
template <int ROT, bool F16, bool STAGED>
__device__ __forceinline__ void rope_item(const RopeTables& t, int N, int n0, const uint4 (&raw)[kQkPasses][4],
                                          const float4* st, float z[kQkPasses][32]) {
  const int tid = threadIdx.x, r64 = tid >> 2, c4 = tid & 3;
  const int np0 = t.split[0] / 2, np1 = t.split[1] / 2, np2 = t.split[2] / 2;
  const int W = t.grid[2], Hg = t.grid[1], HW = Hg * W;
  StagePlan sp{};
  if (STAGED) sp = stage_plan(t, n0, N);
  // only the last tile has rows past N: the zeroing below is skipped (a
  // uniform branch) everywhere else
  const bool tail = n0 + kTile > N;
  // lanes (c4 = lane mod 4) whose pair 16 c4 + k lies before the axis
  // boundary b = 16 q + r: exactly those with c4 < q + (k < r), so per
  // boundary two wave-wide masks, chosen per k, decide the axis of every pair
  const int bnd[2] = {np0, np0 + np1};
  uint64_t below[2][2];
  int bnd_r[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = bnd[i] >> 4;
    bnd_r[i] = bnd[i] & 15;
    below[i][0] = lanes_c4_below(q + 1);
    below[i][1] = lanes_c4_below(q);
  }
#pragma unroll
  for (int p = 0; p < kQkPasses; ++p) {
    const int nl = 64 * p + r64, n = n0 + nl;
    // the row's table rows (staged or in place), per axis
    const int nn = n < N ? n : N - 1;
    const int tq = fdiv(nn, HW, 1.0f / static_cast<float>(HW));
    const int rem = nn - tq * HW;
    const int hq = fdiv(rem, W, 1.0f / static_cast<float>(W));
    const int pos[3] = {tq, hq, rem - hq * W};
    const int lin[3] = {tq, tq * Hg + hq, nn};
    int so[3];
#pragma unroll
    for (int ax = 0; ax < 3; ++ax) {
      const int row = STAGED ? (sp.bypos[ax] ? pos[ax] : lin[ax] - sp.lin0[ax]) : pos[ax];
      so[ax] = (STAGED ? sp.base[ax] : 0) + row * (t.split[ax] / 2);
    }
    // pair P of axis a sits at so[a] + P - (first pair of a).  Per axis, the
    // entry the thread's first pair (16 c4) would have on it; pair 16 c4 + k
    // is entry k from the base of its axis, so the per-pair offset is a
    // constant and only the base is chosen per pair
    const int P0 = 16 * c4;
    const float4* base[3];
    if constexpr (STAGED) {
      // byte offsets into the staged rows, kept opaque so that the compiler
      // selects the scaled offsets instead of scaling the selected index
      int bo[3] = {16 * (so[0] + P0), 16 * (so[1] + P0 - np0), 16 * (so[2] + P0 - np0 - np1)};
#pragma unroll
      for (int ax = 0; ax < 3; ++ax) {
        asm volatile("" : "+v"(bo[ax]));
        base[ax] = reinterpret_cast<const float4*>(reinterpret_cast<const uint8_t*>(st) + bo[ax]);
      }
    } else {
      base[0] = t.axis[0] + (so[0] + P0);
      base[1] = t.axis[1] + (so[1] + P0 - np0);
      base[2] = t.axis[2] + (so[2] + P0 - np0 - np1);
    }
    const uint32_t w[16] = {raw[p][0].x, raw[p][0].y, raw[p][0].z, raw[p][0].w, raw[p][1].x, raw[p][1].y,
                            raw[p][1].z, raw[p][1].w, raw[p][2].x, raw[p][2].y, raw[p][2].z, raw[p][2].w,
                            raw[p][3].x, raw[p][3].y, raw[p][3].z, raw[p][3].w};
    float y[32];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const bool ax0 = __builtin_amdgcn_inverse_ballot_w64(below[0][k < bnd_r[0] ? 0 : 1]);
      const bool ax01 = __builtin_amdgcn_inverse_ballot_w64(below[1][k < bnd_r[1] ? 0 : 1]);
      const float4 g = (ax0 ? base[0] : (ax01 ? base[1] : base[2]))[k];
      const float x0 = h2f<F16>(static_cast<uint16_t>(w[k] & 0xffff));
      const float x1 = h2f<F16>(static_cast<uint16_t>(w[k] >> 16));
      y[2 * k] = __fmaf_rn(x1, g.z, __fmul_rn(x0, g.x));
      y[2 * k + 1] = __fmaf_rn(x1, g.w, __fmul_rn(x0, g.y));
    }
    if (tail) {
      if (n >= N) {
#pragma unroll
        for (int c = 0; c < 32; ++c) y[c] = 0.f;
      }
    }
    if constexpr (ROT == RA_ROT_HALF) {
      // output pair P of axis a (first channel o_a) mixes RoPE channels
      // o_a + i and o_a + i + D_a/2, i = P - o_a/2: the row goes through LDS
      __shared__ float ybuf[64][kD];
      __syncthreads();
#pragma unroll
      for (int c = 0; c < 32; c += 4)
        *reinterpret_cast<float4*>(&ybuf[r64][32 * c4 + c]) = make_float4(y[c], y[c + 1], y[c + 2], y[c + 3]);
      __syncthreads();
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int P = 16 * c4 + k;
        const int ax = (P >= np0) + (P >= np0 + np1);
        const int oh = ax == 0 ? 0 : (ax == 1 ? np0 : np0 + np1);   // o_a / 2
        const int ia = P + oh, ib = ia + (ax == 0 ? np0 : (ax == 1 ? np1 : np2));
        const float av = ybuf[r64][ia], bv = ybuf[r64][ib];
        const float4 r = t.rot[P];
        y[2 * k] = __fmaf_rn(bv, r.z, __fmul_rn(av, r.x));
        y[2 * k + 1] = __fmaf_rn(bv, r.w, __fmul_rn(av, r.y));
      }
      if (tail) {
        if (n >= N) {
#pragma unroll
          for (int c = 0; c < 32; ++c) y[c] = 0.f;
        }
      }
    } else if constexpr (ROT == RA_ROT_HADAMARD) {
      // y <- y H_128, widest stride first: strides 64 and 32 pair the lanes
      // whose c4 differs in bit 1, 0 (the lane with the bit set takes the
      // difference), strides 16 .. 1 stay inside the thread; then 1/sqrt(128)
#pragma unroll
      for (int m = 2; m >= 1; m >>= 1) {
        const bool upper = (c4 & m) != 0;
#pragma unroll
        for (int c = 0; c < 32; ++c) {
          const float o = m == 2 ? quad_xor<2>(y[c]) : quad_xor<1>(y[c]);
          y[c] = upper ? __fsub_rn(o, y[c]) : __fadd_rn(y[c], o);
        }
      }
#pragma unroll
      for (int s = 16; s >= 1; s >>= 1)
#pragma unroll
        for (int c = 0; c < 32; ++c)
          if ((c & s) == 0) {
            const float u = y[c], v = y[c + s];
            y[c] = __fadd_rn(u, v);
            y[c + s] = __fsub_rn(u, v);
          }
#pragma unroll
      for (int c = 0; c < 32; ++c) y[c] = __fmul_rn(y[c], kInvSqrtD);   // rows past N stay zero
    }
#pragma unroll
    for (int c = 0; c < 32; ++c) z[p][c] = y[c];
  }
}

typedef float v16f_ __attribute__((ext_vector_type(16)));
typedef int v6i_ __attribute__((ext_vector_type(6)));

// E2M3 fields of 32 values (integers in [-7, 7], no negative zero): output
// field 2 i + h is element i of source h.  The instruction writes its result
// over a source register wrongly when they overlap (hence the early-clobber
// output) and reads a source written by the instruction right before it one
// cycle early (hence the leading wait state); with scale 1 the integers
// convert exactly.
__device__ __forceinline__ v6i_ pack_e2m3(v16f_ even, v16f_ odd) {
  v6i_ r;
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile(
      "s_nop 0\n\t"
      "v_cvt_scalef32_2xpk16_fp6_f32 %0, %1, %2, %3\n\t"
      "s_nop 1"
      : "=&v"(r)
      : "v"(even), "v"(odd), "s"(1.0f));
#else
  (void)even;
  (void)odd;
  r = v6i_{0, 0, 0, 0, 0, 0};
#endif
  return r;
}

// The code rint(z * inv) clamped to [-7, 7], as a float (+0 for zero)
__device__ __forceinline__ float qcode_f(float z, float inv) {
  const float c = fminf(fmaxf(__builtin_rintf(__fmul_rn(z, inv)), -7.0f), 7.0f);
  return c + 0.0f;   // -0 -> +0 (the zero code carries no sign)
}

// LDS layout of the sums pass's partial sums (in doubles): slot (row r, lane
// group c4) at r * kSumRowStride + c4 * kSumC4Stride holds 16 channels.  The
// row stride is 16 bytes past a multiple of 256, so rows of one lane group
// start in different banks.
constexpr int kSumRowStride = 66;   // 528 bytes
constexpr int kSumC4Stride = 16;    // 128 bytes
constexpr size_t kSumLdsBytes = 32 * kSumRowStride * sizeof(double);

// LDS of a Q/K workgroup: four arrays of 128 floats, then the staged table
// rows (and, in the sums pass, the partial sums in their place).
constexpr int kQkSmallBytes = 4 * kTile * 4;

// Q/K producer, one workgroup per (tile, head): the tile's rows and the table
// rows it needs are requested at once (the table rows straight into LDS),
// then RoPE and the rotation, then
//  SUMS: the fixed-point channel sums of the rotated rows (smoothing), added
//        to a.sums with atomics;
//  else: smoothing, the key bias of Q smoothing, per-group scales and codes.
template <int ROT, bool F16, bool STAGED, bool SUMS>
__device__ __forceinline__ void qk_body(const RopeTables& t, const QkArgs& a, int tile, int bh, uint8_t* lds) {
  float* rowmax = reinterpret_cast<float*>(lds);
  float* ginv = rowmax + kTile;
  float* smu = ginv + kTile;
  float* smq = smu + kD;
  float4* dyn = reinterpret_cast<float4*>(lds + kQkSmallBytes);
  const int tid = threadIdx.x, r64 = tid >> 2, c4 = tid & 3;
  const int N = a.N, n0 = tile * kTile;
  const double den = static_cast<double>(N) * 1048576.0;
  if (STAGED) stage_rows(t, n0, N, dyn);
  uint4 raw[kQkPasses][4];
  load_rows(a.x + static_cast<size_t>(bh) * N * kD, n0, N, raw);
  if (!SUMS && tid < kD) {
    if (a.center) smu[tid] = static_cast<float>(a.sums[static_cast<size_t>(bh) * kD + tid] / den);
    if (a.bias) smq[tid] = static_cast<float>(a.qsums[static_cast<size_t>(bh) * kD + tid] / den);
  }
  // the staged rows have arrived; the barrier makes them (and the means) visible
  __builtin_amdgcn_s_waitcnt(0x3F70);   // vmcnt(0)
  __syncthreads();
  float z[kQkPasses][32];
  rope_item<ROT, F16, STAGED>(t, N, n0, raw, dyn, z);

  if constexpr (SUMS) {
    // per channel: the thread's two rows, then the 64 row groups through LDS
    // (reusing the staged rows), 16 of the thread's channels at a time: rows
    // 0..31 store, rows 32..63 add theirs to the same slots, then one thread
    // per channel adds the 32 slots.  The values are integers below 2^53, so
    // every order gives the same sum.
    double* red = reinterpret_cast<double*>(dyn);
    const int slot = (r64 & 31) * kSumRowStride + c4 * kSumC4Stride;   // in doubles
    double acc[32];
#pragma unroll
    for (int c = 0; c < 32; ++c) acc[c] = fixq(z[0][c]) + fixq(z[1][c]);
    __syncthreads();   // every thread is done with the staged rows
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (r64 < 32) {
#pragma unroll
        for (int c = 0; c < 16; c += 2)
          *reinterpret_cast<double2*>(&red[slot + c]) = make_double2(acc[16 * h + c], acc[16 * h + c + 1]);
      }
      __syncthreads();
      if (r64 >= 32) {
#pragma unroll
        for (int c = 0; c < 16; c += 2) {
          double2* d = reinterpret_cast<double2*>(&red[slot + c]);
          const double2 o = *d;
          *d = make_double2(o.x + acc[16 * h + c], o.y + acc[16 * h + c + 1]);
        }
      }
      __syncthreads();
      if (tid < 64) {
        const double* col = red + (tid >> 4) * kSumC4Stride + (tid & 15);
        double sum = 0.0;
        for (int r = 0; r < 32; ++r) sum += col[r * kSumRowStride];
        unsafeAtomicAdd(a.sums + static_cast<size_t>(bh) * kD + 32 * (tid >> 4) + 16 * h + (tid & 15), sum);
      }
      if (h == 0) __syncthreads();   // read before the second half overwrites the slots
    }
  } else {
    if (a.center) {
      if (a.mu_out && tile == 0 && tid < kD) a.mu_out[bh * kD + tid] = smu[tid];
#pragma unroll
      for (int p = 0; p < kQkPasses; ++p)
        if (n0 + 64 * p + r64 < N)
#pragma unroll
          for (int c = 0; c < 32; ++c) z[p][c] = __fsub_rn(z[p][c], smu[32 * c4 + c]);
    }
    if (a.bias) {
      // Q smoothing: per-key score bias b = mu_Q . z (z = this K row after its
      // own smoothing), products in binary32 summed pairwise over the channel
      // range: inside the thread blocks of 2, 4, ..., 32 channels, then lanes
      // 1 and 2 apart (blocks of 64, 128).  Padded rows give 0.
#pragma unroll
      for (int p = 0; p < kQkPasses; ++p) {
        float bb[32];
#pragma unroll
        for (int c = 0; c < 32; ++c) bb[c] = __fmul_rn(smq[32 * c4 + c], z[p][c]);
#pragma unroll
        for (int s = 1; s < 32; s <<= 1)
#pragma unroll
          for (int c = 0; c < 32; c += 2 * s) bb[c] = __fadd_rn(bb[c], bb[c + s]);
        float v = bb[0];
        v = __fadd_rn(v, quad_xor<1>(v));
        v = __fadd_rn(v, quad_xor<2>(v));
        if (c4 == 0) a.bias[static_cast<size_t>(bh) * a.Npad + n0 + 64 * p + r64] = v;
      }
    }
    // row abs-max over the 128 channels (4 lanes of the row)
#pragma unroll
    for (int p = 0; p < kQkPasses; ++p) {
      float v = 0.f;
#pragma unroll
      for (int c = 0; c < 32; ++c) v = fmaxf(v, fabsf(z[p][c]));
      v = fmaxf(v, quad_xor<1>(v));
      v = fmaxf(v, quad_xor<2>(v));
      if (c4 == 0) rowmax[64 * p + r64] = v;
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
      // record ((chunk*2 + ch/64)*2 + (ch/32)%2)*32 + row of 24 bytes, field
      // f (channel 32 (ch/32) + f) at bit 6 f: the thread's 32 channels of a
      // row are exactly record ((chunk*2 + c4/2)*2 + c4%2)*32 + row
      uint8_t* base = a.codes + static_cast<size_t>(bh) * a.Npad * 96 + static_cast<size_t>(tile) * kTile * 96;
#pragma unroll
      for (int p = 0; p < kQkPasses; ++p) {
        const int nl = 64 * p + r64;
        const float inv = ginv[nl / g];
        v16f_ ev, od;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          ev[i] = qcode_f(z[p][2 * i], inv);
          od[i] = qcode_f(z[p][2 * i + 1], inv);
        }
        const v6i_ f = pack_e2m3(ev, od);
        const int rec = (((nl >> 5) * 2 + (c4 >> 1)) * 2 + (c4 & 1)) * 32 + (nl & 31);
        uint2* d = reinterpret_cast<uint2*>(base + rec * 24);
        d[0] = make_uint2(static_cast<uint32_t>(f[0]), static_cast<uint32_t>(f[1]));
        d[1] = make_uint2(static_cast<uint32_t>(f[2]), static_cast<uint32_t>(f[3]));
        d[2] = make_uint2(static_cast<uint32_t>(f[4]), static_cast<uint32_t>(f[5]));
      }
    } else {
      // tiled layout ((chunk*8 + unit)*32 + row)*8 + byte: the thread's 32
      // channels are units 2 c4 and 2 c4 + 1 of the row, channel pair
      // (2i, 2i+1) of a unit in byte i
      uint8_t* base = a.codes + static_cast<size_t>(bh) * a.Npad * 64 + static_cast<size_t>(tile) * kTile * 64;
#pragma unroll
      for (int p = 0; p < kQkPasses; ++p) {
        const int nl = 64 * p + r64;
        const float inv = ginv[nl / g];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          uint32_t wv[2] = {0u, 0u};
#pragma unroll
          for (int c = 0; c < 16; ++c)
            wv[c >> 3] |= static_cast<uint32_t>(qcode(z[p][16 * u + c], inv) & 0xF) << (4 * (c & 7));
          const int unit = 2 * c4 + u;
          *reinterpret_cast<uint2*>(base + (((nl >> 5) * 8 + unit) * 32 + (nl & 31)) * 8) = make_uint2(wv[0], wv[1]);
        }
      }
    }
  }
}

// ------------------------------------------------------------------ V --

template <bool F16, bool VHAD>
__device__ __forceinline__ void load_v_tile(const VArgs& a, int bh, int tile, float z[16][4]) {
  const int tid = threadIdx.x, rr = tid >> 5, cl = tid & 31;
  const uint16_t* xb = a.x + static_cast<size_t>(bh) * a.N * kD;
  // without centring the subtracted mean is 0 (x - 0 == x exactly, also for
  // -0), so the subtraction needs no per-element select
  float4 m = make_float4(0.f, 0.f, 0.f, 0.f);
  if (a.center) m = mean4(a.sums + static_cast<size_t>(bh) * kD, a.N, cl);
  uint2 raw[16];
#pragma unroll
  for (int p = 0; p < 16; ++p) {
    const int n = tile * kTile + p * 8 + rr;
    raw[p] = *reinterpret_cast<const uint2*>(xb + static_cast<size_t>(n < a.N ? n : a.N - 1) * kD + 4 * cl);
  }
  // rows past N (only in the last tile: a uniform choice between two copies
  // of the loop) are zero and not centred
  auto rows = [&](auto tail_tag) {
    constexpr bool TAIL = decltype(tail_tag)::value;
    for (int p = 0; p < 16; ++p) {
      const int n = tile * kTile + p * 8 + rr;
      const bool in = !TAIL || n < a.N;
      float x[4] = {0.f, 0.f, 0.f, 0.f};
      if (in) {
        x[0] = h2f<F16>(static_cast<uint16_t>(raw[p].x & 0xffff));
        x[1] = h2f<F16>(static_cast<uint16_t>(raw[p].x >> 16));
        x[2] = h2f<F16>(static_cast<uint16_t>(raw[p].y & 0xffff));
        x[3] = h2f<F16>(static_cast<uint16_t>(raw[p].y >> 16));
      }
      // online V rotation (Sec. 4.3): the row times H, before smoothing
      if constexpr (VHAD) hadamard_row(x, cl);
      if (in) {
        x[0] = __fsub_rn(x[0], m.x);
        x[1] = __fsub_rn(x[1], m.y);
        x[2] = __fsub_rn(x[2], m.z);
        x[3] = __fsub_rn(x[3], m.w);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) z[p][c] = x[c];
    }
  };
  if ((tile + 1) * kTile > a.N) rows(std::integral_constant<bool, true>());
  else rows(std::integral_constant<bool, false>());
}

// LDS: 8 x 128 binary64.
template <bool F16, bool VHAD>
__device__ __forceinline__ void v_sums_body(const VArgs& a, int tile, int bh, uint8_t* lds) {
  float z[16][4];
  load_v_tile<F16, VHAD>(a, bh, tile, z);
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int p = 0; p < 16; ++p)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[c] += fixq(z[p][c]);
  add_sums(acc, a.sums + static_cast<size_t>(bh) * kD, reinterpret_cast<double*>(lds));
}

__device__ __forceinline__ int vgroup_of(const VArgs& a, int n) {
  int g = n / a.group;
  return g < a.ngroups ? g : a.ngroups - 1;
}

// Per (tile half, channel) abs-max, merged into the group maxima with an
// order-independent atomic max on the float bits (values are >= 0).
// LDS: 8 x 2 x 128 floats.
template <bool F16, bool VHAD>
__device__ __forceinline__ void v_amax_body(const VArgs& a, int tile, int bh, uint8_t* lds) {
  float (*red)[2][kD] = reinterpret_cast<float (*)[2][kD]>(lds);
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

// LDS: the tile's codes (12 KB), 2 x 128 inverse scales, 8 x 2 x 128 floats.
constexpr int kVQuantLdsBytes = kTile * 96 + 2 * kD * 4 + 8 * 2 * kD * 4;

template <bool F16, bool VHAD>
__device__ __forceinline__ void v_quant_body(const VArgs& a, int tile, int bh, uint8_t* lds) {
  uint8_t* ctile = lds;
  float (*ginv)[kD] = reinterpret_cast<float (*)[kD]>(lds + kTile * 96);
  float (*red)[2][kD] = reinterpret_cast<float (*)[2][kD]>(lds + kTile * 96 + 2 * kD * 4);
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

// One producer pass: the block's job from its row of the grid.  The job's
// arguments are copied out with constant indices (indexing the argument array
// with the run-time job number would put it in scratch).
template <int ROT, bool F16, bool STAGED, bool VHAD>
__global__ __launch_bounds__(256) void k_pass(RopeTables t, PassArgs pa) {
  extern __shared__ __align__(16) uint8_t lds[];
  const int j = blockIdx.y / pa.BH, bh = blockIdx.y - j * pa.BH, tile = blockIdx.x;
  int kind;
  QkArgs qa;
  VArgs va;
  if (j == 0) {
    kind = pa.job[0].kind;
    qa = pa.job[0].qk;
    va = pa.job[0].v;
  } else if (j == 1) {
    kind = pa.job[1].kind;
    qa = pa.job[1].qk;
    va = pa.job[1].v;
  } else {
    kind = pa.job[2].kind;
    qa = pa.job[2].qk;
    va = pa.job[2].v;
  }
  switch (kind) {
    case kQkSums: qk_body<ROT, F16, STAGED, true>(t, qa, tile, bh, lds); break;
    case kQkQuant: qk_body<ROT, F16, STAGED, false>(t, qa, tile, bh, lds); break;
    case kVSums: v_sums_body<F16, VHAD>(va, tile, bh, lds); break;
    case kVAmax: v_amax_body<F16, VHAD>(va, tile, bh, lds); break;
    case kVQuant: v_quant_body<F16, VHAD>(va, tile, bh, lds); break;
    default: break;
  }
}

// The table copy and the zero fills of one producer call.
__global__ __launch_bounds__(256) void k_prologue(Prologue pr) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  const int64_t i0 = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x;
  for (int64_t i = i0; i < pr.ncopy; i += stride) pr.dst[i] = pr.src[i];
#pragma unroll
  for (int z = 0; z < 4; ++z)
    for (int64_t i = i0; i < pr.nzero[z]; i += stride) pr.zero[z][i] = 0u;
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



}  // namespace

namespace {

// LDS bytes one job of a pass needs (stage: the staged table rows, or 0).
size_t job_lds(int kind, size_t stage) {
  switch (kind) {
    case kQkSums: return kQkSmallBytes + (stage > kSumLdsBytes ? stage : kSumLdsBytes);
    case kQkQuant: return kQkSmallBytes + stage;
    case kVSums: return 8 * kD * sizeof(double);
    case kVAmax: return 8 * 2 * kD * sizeof(float);
    case kVQuant: return kVQuantLdsBytes;
    default: return 0;
  }
}

template <int ROT, bool F16>
hipError_t launch_pass_rf(const RopeTables& t, const PassArgs& pa, bool staged, bool vhad, size_t lds, hipStream_t s) {
  const dim3 g(pa.Npad / kTile, pa.njobs * pa.BH);
  if (staged) {
    if (vhad) hipLaunchKernelGGL((k_pass<ROT, F16, true, true>), g, dim3(256), lds, s, t, pa);
    else hipLaunchKernelGGL((k_pass<ROT, F16, true, false>), g, dim3(256), lds, s, t, pa);
  } else {
    if (vhad) hipLaunchKernelGGL((k_pass<ROT, F16, false, true>), g, dim3(256), lds, s, t, pa);
    else hipLaunchKernelGGL((k_pass<ROT, F16, false, false>), g, dim3(256), lds, s, t, pa);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pass(const RopeTables& t, const PassArgs& pa, hipStream_t s) {
  if (pa.njobs < 1) return hipSuccess;
  bool any_qk = false;
  for (int j = 0; j < pa.njobs; ++j) any_qk |= pa.job[j].kind == kQkSums || pa.job[j].kind == kQkQuant;
  // a pass of V jobs only carries no tables (t is empty then)
  const int bound = any_qk ? stage_bound(t) : 0;
  const bool staged = any_qk && bound <= kStageMaxF4;
  const size_t stage = staged ? static_cast<size_t>(bound) * sizeof(float4) : 0;
  size_t lds = 0;
  bool f16 = false, vhad = false;
  for (int j = 0; j < pa.njobs; ++j) {
    const size_t need = job_lds(pa.job[j].kind, stage);
    if (need > lds) lds = need;
    const int k = pa.job[j].kind;
    if (k == kQkSums || k == kQkQuant) f16 = pa.job[j].qk.is_fp16 != 0;
    else if (k != kPassNone) {
      f16 = pa.job[j].v.is_fp16 != 0;
      vhad = pa.job[j].v.vhad != 0;
    }
  }
  const int rot = (t.rotation == RA_ROT_HALF || t.rotation == RA_ROT_HADAMARD) ? t.rotation : 0;
  if (rot == RA_ROT_HALF)
    return f16 ? launch_pass_rf<RA_ROT_HALF, true>(t, pa, staged, vhad, lds, s)
               : launch_pass_rf<RA_ROT_HALF, false>(t, pa, staged, vhad, lds, s);
  if (rot == RA_ROT_HADAMARD)
    return f16 ? launch_pass_rf<RA_ROT_HADAMARD, true>(t, pa, staged, vhad, lds, s)
               : launch_pass_rf<RA_ROT_HADAMARD, false>(t, pa, staged, vhad, lds, s);
  return f16 ? launch_pass_rf<0, true>(t, pa, staged, vhad, lds, s) : launch_pass_rf<0, false>(t, pa, staged, vhad, lds, s);
}

hipError_t launch_prologue(const Prologue& pr, hipStream_t s) {
  int64_t n = pr.ncopy;
  for (int z = 0; z < 4; ++z) n = pr.nzero[z] > n ? pr.nzero[z] : n;
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_prologue, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, pr);
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





}  // namespace ra
