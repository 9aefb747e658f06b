// ra_internal.h -- declarations shared by the host side and the HIP kernels of
// librotate_attn.so (library-internal; not installed, not part of the ABI).
#pragma once
#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ra {

constexpr int kD = 128;       // head dimension
constexpr int kTile = 128;    // producer token tile; Npad is a multiple of it
constexpr float kInvSqrtD = 0.0883883476483184405501055452631f;  // fl32(1/sqrt(128))

// max(x, x of lane ^ 32) in a wave of 64: v_permlane32_swap (gfx950) exchanges
// the upper half of its first operand with the lower half of its second, so
// with x in both, the two results hold x of the lane and x of lane ^ 32 in
// every lane (a register move, no LDS round trip).
__device__ __forceinline__ float max_halves(float x) {
  const unsigned u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// RoPE/rotation tables on the device.  For axis a the table holds, for every
// position pos in [0, extent_a) and pair k in [0, D_a/2), the binary32 2x2
// block G = M (or M R for the merged interleaved rotation) as
// {g00, g01, g10, g11}, so that [y0 y1] = [x0 x1] G.  `rot` holds the 64
// binary32 rotation blocks of the half rotation.
struct RopeTables {
  const float4* axis[3];
  const float4* rot;
  int split[3];
  int grid[3];
  int rotation;
};

// Per-thread constants of the producer: which table entries the two channel
// pairs (4*cl .. 4*cl+3) of this thread read.
struct QkArgs {
  const uint16_t* x;      // [BH][N][128] bf16/fp16 bits
  uint8_t* codes;         // tiled INT4 layout, [BH][Npad*64]
  float* scales;          // [BH][Npad/group]
  double* sums;           // [BH][128] fixed-point channel sums (sums pass adds, quant pass reads)
  float* mu_out;          // [BH][128] the mean each head is centred by, or nullptr
  int center;             // quant pass: subtract the mean derived from sums
  int N, Npad, group, is_fp16;
  int e2m3;               // 1: write the E2M3 container, 0: the INT4 nibble container
  // K pass with Q smoothing: the Q fixed-point sums (mu_Q) and the per-key
  // score bias output [BH][Npad]; both nullptr otherwise
  const double* qsums;
  float* bias;
};

struct VArgs {
  const uint16_t* x;      // [BH][N][128]
  uint8_t* codes;         // tiled V layout, [BH][Npad*64]
  float* scales;          // [BH][ngroups][128]
  double* sums;           // [BH][128] fixed-point channel sums
  float* mu_out;          // [BH][128] or nullptr
  int center;             // subtract the mean derived from sums
  uint32_t* amax;         // [BH][ngroups][128] float bits (non-negative)
  int N, Npad, group, ngroups, is_fp16;
  int e2m3;
  int vhad;               // rotate each V row by the 128-point Hadamard before smoothing
  int local_amax;         // groups of 64 or 128 tokens: the quantize pass takes the group maxima
                          // from its own tile (no amax pass, amax unused)
};

struct AttnArgs {
  const uint8_t* qc;
  const float* qs;
  const uint8_t* kc;
  const float* ks;
  const uint8_t* vc;
  const float* vs;
  const float* mu_v;      // [BH][128] or nullptr
  const float* kbias;     // [BH][Npad] per-key score bias (Q smoothing) or nullptr
  void* o;
  int N, Npad, BH;
  int q_group, k_group, v_group, nvgroups;
  int v_bpg;              // KV blocks per V scale group (v_group / kv_block; nvgroups == 1: any value >= nblocks)
  float Kc;               // fl32(sm_scale * log2(e))
  int out_dtype;
  int vhad;               // V was rotated by H: rotate each output row back
  int lq;                 // l from the quantized P (sum of the codes) instead of the exact P
  // debug dump (debug kernel only)
  int32_t* dbg_s;
  uint8_t* dbg_u;
  float* dbg_m;
  int dbg_bh, dbg_row0, dbg_rows;
};

struct Fp16Args {
  const uint16_t* q;      // tiled 16-bit layout (see ra_fp16.hip)
  const uint16_t* k;
  const uint16_t* v;      // tiled transposed layout
  void* o;
  int N, Npad, BH;
  float Kc;
  int is_fp16, out_dtype;
};

// Producer passes launched together in one grid: job j of a pass covers every
// head and tile (blockIdx.y = j * BH + head, blockIdx.x = tile), and jobs of
// one pass do not depend on each other.
enum PassKind { kPassNone = 0, kQkSums = 1, kQkQuant = 2, kVSums = 3, kVAmax = 4, kVQuant = 5 };
struct PassJob {
  int kind;
  QkArgs qk;   // kQkSums, kQkQuant
  VArgs v;     // kVSums, kVAmax, kVQuant
};
struct PassArgs {
  PassJob job[3];
  int njobs, BH, Npad;
};

// The start of a producer call: the RoPE tables into the workspace (src may be
// pinned host memory read through its device mapping) and up to four zero fills.
struct Prologue {
  const uint32_t* src;
  uint32_t* dst;
  int64_t ncopy;
  uint32_t* zero[4];
  int64_t nzero[4];
};

// ---- launchers (return hipError_t) ----
hipError_t launch_pass(const RopeTables& t, const PassArgs& pa, hipStream_t s);
hipError_t launch_prologue(const Prologue& pr, hipStream_t s);
hipError_t launch_copy_u32(const uint32_t* src, uint32_t* dst, int64_t n, hipStream_t s);
// n host floats -> dst on the device, carried in kernel arguments (no allocation)
hipError_t launch_write_floats(const float* host, size_t n, float* dst, hipStream_t s);
hipError_t launch_attn_int4(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, bool debug,
                            hipStream_t s);
hipError_t launch_attn_e2m3(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, bool debug,
                            hipStream_t s);
hipError_t launch_attn_e2m3_debug(const AttnArgs& a, int kv_block, bool k_per_token, bool sym7, hipStream_t s);
// (both launchers pick the key-bias variant when a.kbias is set and the
// quantized-normaliser variant when a.lq is set)
hipError_t launch_rope16(const RopeTables& t, const uint16_t* x, uint16_t* out, int BH, int N, int Npad,
                         int is_fp16, hipStream_t s);
hipError_t launch_v16_relayout(const uint16_t* v, uint16_t* out, int BH, int N, int Npad, hipStream_t s);
hipError_t launch_attn_fp16(const Fp16Args& a, int kv_block, hipStream_t s);

}  // namespace ra
