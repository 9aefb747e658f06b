// ra_host.cpp -- host side of librotate_attn.so: argument validation, RoPE
// table construction (host cache, copied into the caller's workspace on the
// caller's stream), workspace partitioning, kernel launches.  Every entry
// point validates before it touches the GPU; the library allocates no device
// memory and creates no streams.
#include <hip/hip_runtime.h>

#include <array>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/rotate_attn.h"
#include "ra_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define RA_CHECK_HIP(expr)                                                            \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) return fail(RA_ERR_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr int kD = 128;
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int64_t npad_of(int N) { return (static_cast<int64_t>(N) + 127) / 128 * 128; }

int validate(const ra_params* p) {
  if (!p) return fail(RA_ERR_INVALID, "params is NULL");
  if (p->D != kD) return fail(RA_ERR_UNSUPPORTED, "only D == 128 is supported");
  if (p->B < 1 || p->H < 1 || p->N < 1) return fail(RA_ERR_INVALID, "B, H, N must be >= 1");
  if (p->N > (1 << 21)) return fail(RA_ERR_UNSUPPORTED, "N above 2^21 tokens is not supported");
  if (static_cast<int64_t>(p->B) * p->H > (1 << 20)) return fail(RA_ERR_UNSUPPORTED, "B*H too large");
  for (int i = 0; i < 3; ++i)
    if (p->grid[i] < 1) return fail(RA_ERR_INVALID, "grid extents must be >= 1");
  if (static_cast<int64_t>(p->grid[0]) * p->grid[1] * p->grid[2] != p->N)
    return fail(RA_ERR_INVALID, "grid T*Hg*W must equal N");
  int sum = 0;
  for (int i = 0; i < 3; ++i) {
    if (p->rope_split[i] < 2 || (p->rope_split[i] & 1)) return fail(RA_ERR_INVALID, "rope_split entries must be even and >= 2");
    sum += p->rope_split[i];
  }
  if (sum != p->D) return fail(RA_ERR_INVALID, "rope_split must sum to D");
  if (!(p->rope_theta > 0.0f) || !std::isfinite(p->rope_theta)) return fail(RA_ERR_INVALID, "rope_theta must be > 0");
  if (p->rotation < RA_ROT_NONE || p->rotation > RA_ROT_HADAMARD) return fail(RA_ERR_INVALID, "unknown rotation");
  if (p->rot_blocks && (p->rotation == RA_ROT_INTERLEAVED || p->rotation == RA_ROT_HALF)) {
    // every block must be orthogonal (R R^T = I): a non-orthogonal R applied to
    // both Q and K would change Q K^T (Sec. 4.1 relies on R R^T = I)
    for (int b = 0; b < kD / 2; ++b) {
      const double* R = p->rot_blocks + 4 * b;
      for (int i = 0; i < 4; ++i)
        if (!std::isfinite(R[i])) return fail(RA_ERR_INVALID, "rot_blocks must be finite");
      const double e00 = R[0] * R[0] + R[1] * R[1] - 1.0, e11 = R[2] * R[2] + R[3] * R[3] - 1.0;
      const double e01 = R[0] * R[2] + R[1] * R[3];
      if (std::fabs(e00) > 1e-6 || std::fabs(e11) > 1e-6 || std::fabs(e01) > 1e-6)
        return fail(RA_ERR_INVALID, "rot_blocks[" + std::to_string(b) + "] is not orthogonal (R R^T != I)");
    }
  }
  if (p->p_quant != RA_PQ_RANGE15 && p->p_quant != RA_PQ_SYM7) return fail(RA_ERR_INVALID, "unknown p_quant");
  if (p->smooth < 0 || p->smooth > (RA_SMOOTH_K | RA_SMOOTH_V | RA_SMOOTH_Q))
    return fail(RA_ERR_INVALID, "unknown smooth flags");
  if (p->q_group < 1 || p->q_group > 128 || (128 % p->q_group) != 0)
    return fail(RA_ERR_UNSUPPORTED, "q_group must divide 128");
  if (p->k_group != 1 && p->k_group != 16 && p->k_group != 32 && p->k_group != 64 && p->k_group != 128)
    return fail(RA_ERR_UNSUPPORTED, "k_group must be 1, 16, 32, 64 or 128");
  if (p->kv_block != 64 && p->kv_block != 128) return fail(RA_ERR_UNSUPPORTED, "kv_block must be 64 or 128");
  if (p->v_group < 1) return fail(RA_ERR_INVALID, "v_group must be >= 1");
  if ((p->v_group % p->kv_block) != 0 && p->v_group < p->N)
    return fail(RA_ERR_UNSUPPORTED, "v_group must be a multiple of kv_block or >= N");
  if (!(p->sm_scale >= 0.0f) || !std::isfinite(p->sm_scale)) return fail(RA_ERR_INVALID, "sm_scale must be >= 0");
  if (p->in_dtype != RA_BF16 && p->in_dtype != RA_FP16) return fail(RA_ERR_INVALID, "in_dtype must be BF16 or FP16");
  if (p->code_format != RA_CODES_INT4 && p->code_format != RA_CODES_E2M3)
    return fail(RA_ERR_INVALID, "code_format must be RA_CODES_INT4 or RA_CODES_E2M3");
  if (p->out_dtype != RA_BF16 && p->out_dtype != RA_FP16 && p->out_dtype != RA_FP32)
    return fail(RA_ERR_INVALID, "out_dtype must be BF16, FP16 or FP32");
  if (p->v_rotation != RA_VROT_NONE && p->v_rotation != RA_VROT_HADAMARD)
    return fail(RA_ERR_INVALID, "unknown v_rotation");
  if (p->l_quant != 0 && p->l_quant != 1) return fail(RA_ERR_INVALID, "l_quant must be 0 or 1");
  return RA_OK;
}

// RoPE/rotation tables: for each axis a, grid[a] positions x rope_split[a]/2
// pairs of float4 blocks, then the 64 rotation blocks (float4 each).
size_t table_bytes(const ra_params* p) {
  size_t n = kD / 2;
  for (int a = 0; a < 3; ++a) n += static_cast<size_t>(p->grid[a]) * (p->rope_split[a] / 2);
  return n * 4 * sizeof(float);
}

struct Sizes {
  int64_t BH, Npad, ntiles, nvgroups;
  size_t codes, qscale, kscale, vscale, mu, partial, amax, kbias;
};

Sizes sizes_of(const ra_params* p) {
  Sizes s;
  s.BH = static_cast<int64_t>(p->B) * p->H;
  s.Npad = npad_of(p->N);
  s.ntiles = s.Npad / 128;
  s.nvgroups = (p->N + p->v_group - 1) / p->v_group;
  s.codes = static_cast<size_t>(s.BH * s.Npad * (p->code_format == RA_CODES_E2M3 ? 96 : 64));
  s.qscale = static_cast<size_t>(s.BH * (s.Npad / p->q_group));
  s.kscale = static_cast<size_t>(s.BH * (s.Npad / p->k_group));
  s.vscale = static_cast<size_t>(s.BH * s.nvgroups * kD);
  s.mu = static_cast<size_t>(s.BH * kD);
  s.partial = static_cast<size_t>(s.BH * kD);
  s.amax = s.vscale;
  s.kbias = static_cast<size_t>(s.BH * s.Npad);
  return s;
}

// Workspace partition of the INT4 path.  The quantize calls use only the head
// of it (partials, internal means, V maxima); fwd_int4 also keeps the codes.
struct Int4Ws {
  float* tables;
  double* ksum;
  double* vsum;
  double* qsum;
  float* mu_k;
  float* mu_v;
  float* mu_q;
  float* kbias;
  uint32_t* amax;
  uint8_t* qc;
  uint8_t* kc;
  uint8_t* vc;
  float* qs;
  float* ks;
  float* vs;
  size_t total;
};

Int4Ws carve_int4(const ra_params* p, void* base) {
  const Sizes s = sizes_of(p);
  Int4Ws w;
  size_t o = 0;
  char* b = static_cast<char*>(base);
  auto take = [&](size_t bytes) {
    char* r = b ? b + o : nullptr;
    o += align_up(bytes);
    return r;
  };
  w.tables = reinterpret_cast<float*>(take(table_bytes(p)));
  w.ksum = reinterpret_cast<double*>(take(s.partial * sizeof(double)));
  w.vsum = reinterpret_cast<double*>(take(s.partial * sizeof(double)));
  w.qsum = reinterpret_cast<double*>(take(s.partial * sizeof(double)));
  w.mu_k = reinterpret_cast<float*>(take(s.mu * sizeof(float)));
  w.mu_v = reinterpret_cast<float*>(take(s.mu * sizeof(float)));
  w.mu_q = reinterpret_cast<float*>(take(s.mu * sizeof(float)));
  w.kbias = reinterpret_cast<float*>(take((p->smooth & RA_SMOOTH_Q) ? s.kbias * sizeof(float) : 0));
  w.amax = reinterpret_cast<uint32_t*>(take(s.amax * sizeof(uint32_t)));
  w.qc = reinterpret_cast<uint8_t*>(take(s.codes));
  w.kc = reinterpret_cast<uint8_t*>(take(s.codes));
  w.vc = reinterpret_cast<uint8_t*>(take(s.codes));
  w.qs = reinterpret_cast<float*>(take(s.qscale * sizeof(float)));
  w.ks = reinterpret_cast<float*>(take(s.kscale * sizeof(float)));
  w.vs = reinterpret_cast<float*>(take(s.vscale * sizeof(float)));
  w.total = o;
  return w;
}

struct Fp16Ws {
  uint16_t* q;
  uint16_t* k;
  uint16_t* v;
  float* tables;
  size_t total;
};

Fp16Ws carve_fp16(const ra_params* p, void* base) {
  const Sizes s = sizes_of(p);
  Fp16Ws w;
  const size_t one = align_up(static_cast<size_t>(s.BH * s.Npad * kD * 2));
  char* b = static_cast<char*>(base);
  w.q = b ? reinterpret_cast<uint16_t*>(b) : nullptr;
  w.k = b ? reinterpret_cast<uint16_t*>(b + one) : nullptr;
  w.v = b ? reinterpret_cast<uint16_t*>(b + 2 * one) : nullptr;
  w.tables = b ? reinterpret_cast<float*>(b + 3 * one) : nullptr;
  w.total = 3 * one + align_up(table_bytes(p));
  return w;
}

int check_ws(void* ws, size_t have, size_t need) {
  if (!ws) return fail(RA_ERR_WORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(RA_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (have < need) return fail(RA_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) + " bytes");
  return RA_OK;
}

// ------------------------------------------------------------ RoPE tables --
// For axis a, position pos and pair k (global pair p): omega = theta^(-2k/D_a),
// phi = pos * omega, M = [[cos, sin], [-sin, cos]] (row-vector form), and for
// the merged interleaved rotation G = M R_p, all in binary64, rounded once to
// binary32.  R_p defaults to H_2 = (1/sqrt 2) [[1, 1], [1, -1]].
//
// The tables are built on the host once per (grid, split, theta, rotation,
// blocks) and kept in pinned host memory for the life of the process; every
// call that needs them copies them into its workspace on its own stream
// (asynchronous, stream-ordered), so no device memory is owned by the library.

struct HostTable {
  float* pinned = nullptr;  // hipHostMalloc'd, never freed
  const float* mapped = nullptr;  // the same memory as the device addresses it
  size_t bytes = 0;
  size_t off[4] = {0, 0, 0, 0};  // float offsets of the three axis tables and the rotation blocks
};

std::mutex g_mu;
std::map<std::string, HostTable> g_tables;

void rot_block(const ra_params* p, int pair, double R[4]) {
  if (p->rot_blocks) {
    std::memcpy(R, p->rot_blocks + 4 * pair, 4 * sizeof(double));
  } else {
    const double r = 1.0 / std::sqrt(2.0);
    R[0] = r;
    R[1] = r;
    R[2] = r;
    R[3] = -r;
  }
}

// The binary32 table of these parameters, in the order of table_bytes().
void build_table(const ra_params* p, std::vector<float>& host, size_t off[4]) {
  int first = 0;
  for (int a = 0; a < 3; ++a) {
    off[a] = host.size();
    const int np = p->rope_split[a] / 2;
    for (int pos = 0; pos < p->grid[a]; ++pos) {
      for (int k = 0; k < np; ++k) {
        const double omega = std::pow(static_cast<double>(p->rope_theta), -(2.0 * k) / static_cast<double>(p->rope_split[a]));
        const double phi = static_cast<double>(pos) * omega;
        const double cs = std::cos(phi), sn = std::sin(phi);
        const double M[4] = {cs, sn, -sn, cs};
        double G[4];
        if (p->rotation == RA_ROT_INTERLEAVED) {
          double R[4];
          rot_block(p, first + k, R);
          G[0] = M[0] * R[0] + M[1] * R[2];
          G[1] = M[0] * R[1] + M[1] * R[3];
          G[2] = M[2] * R[0] + M[3] * R[2];
          G[3] = M[2] * R[1] + M[3] * R[3];
        } else {
          std::memcpy(G, M, sizeof M);
        }
        for (int i = 0; i < 4; ++i) host.push_back(static_cast<float>(G[i]));
      }
    }
    first += np;
  }
  off[3] = host.size();
  for (int pr = 0; pr < kD / 2; ++pr) {
    double R[4];
    rot_block(p, pr, R);
    for (int i = 0; i < 4; ++i) host.push_back(static_cast<float>(R[i]));
  }
}

std::string table_key(const ra_params* p) {
  std::string key;
  auto put = [&](const void* d, size_t n) { key.append(static_cast<const char*>(d), n); };
  put(p->grid, sizeof p->grid);
  put(p->rope_split, sizeof p->rope_split);
  put(&p->rope_theta, sizeof p->rope_theta);
  put(&p->rotation, sizeof p->rotation);
  if ((p->rotation == RA_ROT_INTERLEAVED || p->rotation == RA_ROT_HALF) && p->rot_blocks)
    put(p->rot_blocks, 4 * (kD / 2) * sizeof(double));
  return key;
}

ra::RopeTables tables_at(const ra_params* p, const float* dev, const size_t off[4]) {
  ra::RopeTables t;
  const float4* base = reinterpret_cast<const float4*>(dev);
  for (int a = 0; a < 3; ++a) {
    t.axis[a] = base + off[a] / 4;
    t.split[a] = p->rope_split[a];
    t.grid[a] = p->grid[a];
  }
  t.rot = base + off[3] / 4;
  t.rotation = p->rotation;
  return t;
}

// The table copy a producer call still has to make (its prologue kernel does it).
struct TableCopy {
  const uint32_t* src = nullptr;
  uint32_t* dst = nullptr;
  int64_t nwords = 0;
};

// Describes the tables of p, placed at dev (table_bytes(p) bytes of the
// workspace), in *out, and copies them there on stream s -- or, with defer,
// leaves the copy to the caller's next kernel and describes it in *defer.
int put_tables(const ra_params* p, float* dev, hipStream_t s, ra::RopeTables* out, TableCopy* defer = nullptr) {
  const std::string key = table_key(p);
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_tables.find(key);
  if (it == g_tables.end()) {
    std::vector<float> host;
    HostTable ht;
    build_table(p, host, ht.off);
    ht.bytes = host.size() * sizeof(float);
    RA_CHECK_HIP(hipHostMalloc(reinterpret_cast<void**>(&ht.pinned), ht.bytes, hipHostMallocDefault));
    std::memcpy(ht.pinned, host.data(), ht.bytes);
    void* mapped = nullptr;
    RA_CHECK_HIP(hipHostGetDevicePointer(&mapped, ht.pinned, 0));
    ht.mapped = static_cast<const float*>(mapped);
    it = g_tables.emplace(key, ht).first;
  }
  const HostTable& ht = it->second;
  // a kernel on s reads the pinned table through its device mapping: the copy
  // stays on the kernel queue, with no hand-over to a copy engine and back
  if (defer) {
    defer->src = reinterpret_cast<const uint32_t*>(ht.mapped);
    defer->dst = reinterpret_cast<uint32_t*>(dev);
    defer->nwords = static_cast<int64_t>(ht.bytes / 4);
  } else {
    RA_CHECK_HIP(ra::launch_copy_u32(reinterpret_cast<const uint32_t*>(ht.mapped), reinterpret_cast<uint32_t*>(dev),
                                     static_cast<int64_t>(ht.bytes / 4), s));
  }
  *out = tables_at(p, dev, ht.off);
  return RA_OK;
}

float kc_of(const ra_params* p) {
  const double sigma = p->sm_scale > 0.0f ? static_cast<double>(p->sm_scale) : 1.0 / std::sqrt(static_cast<double>(p->D));
  return static_cast<float>(sigma * 1.4426950408889634074);
}

hipStream_t st(void* s) { return static_cast<hipStream_t>(s); }

// ------------------------------------------------------------- producers --

// Outputs of a producer call (device pointers; nullptr where not wanted).
struct ProdOut {
  uint8_t* qc = nullptr;
  float* qs = nullptr;
  uint8_t* kc = nullptr;
  float* ks = nullptr;
  uint8_t* vc = nullptr;
  float* vs = nullptr;
  float* mu_k = nullptr;
  float* mu_q = nullptr;
  float* mu_v = nullptr;
  float* kbias = nullptr;
};

// The Q/K producers (q and k given) and/or the V producer (v given) on the
// caller's stream: one prologue kernel (the table copy, the zero fills), then
// the passes.  Each pass is one launch holding every job whose inputs are
// ready, so independent work (the channel sums of K and V, the codes of an
// unsmoothed Q) shares one launch: pass 0 the sums and every code pass that
// needs none; pass 1 the codes that need sums (and the V group maxima when V
// groups straddle tiles); pass 2 the V codes after those maxima.
int produce(const ra_params* p, const ra::RopeTables& t, const TableCopy& tc, const void* q, const void* k,
            const void* v, const ProdOut& out, const Int4Ws& w, hipStream_t s) {
  const Sizes z = sizes_of(p);
  const bool do_qk = q != nullptr && k != nullptr, do_v = v != nullptr;
  const bool center_k = (p->smooth & RA_SMOOTH_K) != 0, center_q = (p->smooth & RA_SMOOTH_Q) != 0;
  const bool smooth_v = (p->smooth & RA_SMOOTH_V) != 0;
  // groups of 64 or 128 tokens never straddle a 128-token tile (they start at
  // multiples of the group size): the V code pass finds their maxima itself
  const bool local_amax = p->v_group == 64 || p->v_group == 128;

  ra::Prologue pr{};
  pr.src = tc.src;
  pr.dst = tc.dst;
  pr.ncopy = tc.nwords;
  int nz = 0;
  auto zero = [&](void* ptr, size_t words) {
    pr.zero[nz] = static_cast<uint32_t*>(ptr);
    pr.nzero[nz] = static_cast<int64_t>(words);
    ++nz;
  };
  if (do_qk) {
    // exact fixed-point channel sums are accumulated by atomics; an unsmoothed
    // tensor reports a zero mean
    if (center_k) zero(w.ksum, 2 * z.partial);
    else if (out.mu_k) zero(out.mu_k, z.mu);
    if (center_q) zero(w.qsum, 2 * z.partial);
    else if (out.mu_q) zero(out.mu_q, z.mu);
  }
  if (do_v) {
    if (smooth_v) zero(w.vsum, 2 * z.partial);
    else if (out.mu_v) zero(out.mu_v, z.mu);
    if (!local_amax) zero(w.amax, z.amax);
  }
  RA_CHECK_HIP(ra::launch_prologue(pr, s));

  ra::PassArgs pass[3];
  for (auto& ps : pass) {
    ps = ra::PassArgs{};
    ps.BH = static_cast<int>(z.BH);
    ps.Npad = static_cast<int>(z.Npad);
  }
  auto add = [&](int ph, int kind, const ra::QkArgs* a, const ra::VArgs* b) {
    ra::PassJob& j = pass[ph].job[pass[ph].njobs++];
    j.kind = kind;
    if (a) j.qk = *a;
    if (b) j.v = *b;
  };
  if (do_qk) {
    ra::QkArgs a{};
    a.N = p->N;
    a.Npad = static_cast<int>(z.Npad);
    a.is_fp16 = p->in_dtype == RA_FP16;
    a.e2m3 = p->code_format == RA_CODES_E2M3;
    ra::QkArgs qq = a;
    qq.x = static_cast<const uint16_t*>(q);
    qq.codes = out.qc;
    qq.scales = out.qs;
    qq.sums = w.qsum;
    qq.center = center_q;
    qq.mu_out = center_q ? (out.mu_q ? out.mu_q : w.mu_q) : nullptr;
    qq.group = p->q_group;
    // an unsmoothed Q's codes come first in the first pass, so that K and V,
    // read again by the code pass, are the most recently read inputs when it
    // starts (the memory-side cache still holds much of them; 0.168 -> 0.164
    // ms for the 32760-token layer's producers inside the INT4 step)
    if (!center_q) add(0, ra::kQkQuant, &qq, nullptr);
    if (center_k) {
      ra::QkArgs ak = a;
      ak.x = static_cast<const uint16_t*>(k);
      ak.sums = w.ksum;
      add(0, ra::kQkSums, &ak, nullptr);
    }
    if (center_q) {
      ra::QkArgs aq = a;
      aq.x = static_cast<const uint16_t*>(q);
      aq.sums = w.qsum;
      add(0, ra::kQkSums, &aq, nullptr);
      add(1, ra::kQkQuant, &qq, nullptr);
    }
    ra::QkArgs kq = a;
    kq.x = static_cast<const uint16_t*>(k);
    kq.codes = out.kc;
    kq.scales = out.ks;
    kq.sums = w.ksum;
    kq.center = center_k;
    kq.mu_out = center_k ? (out.mu_k ? out.mu_k : w.mu_k) : nullptr;
    kq.group = p->k_group;
    kq.qsums = center_q ? w.qsum : nullptr;
    kq.bias = center_q ? out.kbias : nullptr;
    add(center_k || center_q ? 1 : 0, ra::kQkQuant, &kq, nullptr);
  }
  if (do_v) {
    ra::VArgs a{};
    a.x = static_cast<const uint16_t*>(v);
    a.codes = out.vc;
    a.scales = out.vs;
    a.sums = w.vsum;
    a.amax = w.amax;
    a.N = p->N;
    a.Npad = static_cast<int>(z.Npad);
    a.group = p->v_group;
    a.ngroups = static_cast<int>(z.nvgroups);
    a.is_fp16 = p->in_dtype == RA_FP16;
    a.e2m3 = p->code_format == RA_CODES_E2M3;
    a.vhad = p->v_rotation == RA_VROT_HADAMARD;
    a.local_amax = local_amax;
    int ph = 0;
    if (smooth_v) {
      a.center = 0;
      add(0, ra::kVSums, nullptr, &a);
      a.center = 1;
      a.mu_out = out.mu_v ? out.mu_v : w.mu_v;
      ph = 1;
    }
    if (!local_amax) add(ph++, ra::kVAmax, nullptr, &a);
    add(ph, ra::kVQuant, nullptr, &a);
  }
  for (const auto& ps : pass)
    if (ps.njobs) RA_CHECK_HIP(ra::launch_pass(t, ps, s));
  return RA_OK;
}

int attn_impl(const ra_params* p, const uint8_t* qc, const float* qs, const uint8_t* kc, const float* ks,
              const uint8_t* vc, const float* vs, const float* mu_v, const float* kbias, void* o, bool debug, int bh,
              int row0, int rows, int32_t* s_out, uint8_t* u_out, float* m_out, hipStream_t s) {
  const Sizes z = sizes_of(p);
  ra::AttnArgs a{};
  a.qc = qc;
  a.qs = qs;
  a.kc = kc;
  a.ks = ks;
  a.vc = vc;
  a.vs = vs;
  a.mu_v = mu_v;
  a.kbias = (p->smooth & RA_SMOOTH_Q) ? kbias : nullptr;
  a.o = o;
  a.N = p->N;
  a.Npad = static_cast<int>(z.Npad);
  a.BH = static_cast<int>(z.BH);
  a.q_group = p->q_group;
  a.k_group = p->k_group;
  a.v_group = p->v_group;
  a.nvgroups = static_cast<int>(z.nvgroups);
  // v_group is a multiple of kv_block, or >= N (one group)
  a.v_bpg = z.nvgroups > 1 ? p->v_group / p->kv_block : INT32_MAX;
  a.Kc = kc_of(p);
  a.out_dtype = p->out_dtype;
  a.vhad = p->v_rotation == RA_VROT_HADAMARD;
  a.dbg_s = s_out;
  a.dbg_u = u_out;
  a.dbg_m = m_out;
  a.dbg_bh = bh;
  a.dbg_row0 = row0;
  a.dbg_rows = rows;
  a.lq = p->l_quant;
  if (p->code_format == RA_CODES_E2M3)
    RA_CHECK_HIP(ra::launch_attn_e2m3(a, p->kv_block, p->k_group < 32, p->p_quant == RA_PQ_SYM7, debug, s));
  else
    RA_CHECK_HIP(ra::launch_attn_int4(a, p->kv_block, p->k_group < 32, p->p_quant == RA_PQ_SYM7, debug, s));
  return RA_OK;
}

int fp16_prepare_impl(const ra_params* p, const void* q, const void* k, const void* v, const Fp16Ws& w, hipStream_t s) {
  const Sizes z = sizes_of(p);
  ra::RopeTables t;
  ra_params plain = *p;
  plain.rotation = RA_ROT_NONE;
  plain.rot_blocks = nullptr;
  int rc = put_tables(&plain, w.tables, s, &t);
  if (rc) return rc;
  const int is16 = p->in_dtype == RA_FP16;
  RA_CHECK_HIP(ra::launch_rope16(t, static_cast<const uint16_t*>(q), w.q, static_cast<int>(z.BH), p->N,
                                 static_cast<int>(z.Npad), is16, s));
  RA_CHECK_HIP(ra::launch_rope16(t, static_cast<const uint16_t*>(k), w.k, static_cast<int>(z.BH), p->N,
                                 static_cast<int>(z.Npad), is16, s));
  RA_CHECK_HIP(ra::launch_v16_relayout(static_cast<const uint16_t*>(v), w.v, static_cast<int>(z.BH), p->N,
                                       static_cast<int>(z.Npad), s));
  return RA_OK;
}

int fp16_attn_impl(const ra_params* p, const Fp16Ws& w, void* o, hipStream_t s) {
  const Sizes z = sizes_of(p);
  ra::Fp16Args a{};
  a.q = w.q;
  a.k = w.k;
  a.v = w.v;
  a.o = o;
  a.N = p->N;
  a.Npad = static_cast<int>(z.Npad);
  a.BH = static_cast<int>(z.BH);
  a.Kc = kc_of(p);
  a.is_fp16 = p->in_dtype == RA_FP16;
  a.out_dtype = p->out_dtype;
  RA_CHECK_HIP(ra::launch_attn_fp16(a, p->kv_block, s));
  return RA_OK;
}

// The whole INT4 forward on a carved workspace whose table region holds the
// tables t describes (or receives them through tc, in the producers'
// prologue): producers, then the attention (codes stay in w).
int int4_forward(const ra_params* p, const ra::RopeTables& t, const TableCopy& tc, const void* q, const void* k,
                 const void* v, void* o, const Int4Ws& w, hipStream_t s) {
  ProdOut out;
  out.qc = w.qc;
  out.qs = w.qs;
  out.kc = w.kc;
  out.ks = w.ks;
  out.vc = w.vc;
  out.vs = w.vs;
  out.kbias = w.kbias;
  int rc = produce(p, t, tc, q, k, v, out, w, s);
  if (rc) return rc;
  const float* mu = (p->smooth & RA_SMOOTH_V) ? w.mu_v : nullptr;
  return attn_impl(p, w.qc, w.qs, w.kc, w.ks, w.vc, w.vs, mu, w.kbias, o, false, 0, 0, 0, nullptr, nullptr, nullptr, s);
}

// ----------------------------------------------- allocation-free forward --
// rotate_attn_fwd_int4_noalloc keeps its INT4 workspace in this array: one
// copy per GPU, allocated with the code object and held until the process
// ends.  Host code never passes `scratch` itself (on the host it is only a
// stand-in symbol): the device address comes from hipGetSymbolAddress, taken
// once per device.

constexpr size_t kNoAllocBytes = RA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

struct NoAllocState {
  void* base = nullptr;       // device address of `scratch` on this device
  std::string resident;       // table key of the tables now in the scratch's table region
};

std::mutex g_na_mu;
std::map<int, NoAllocState> g_na;

int noalloc_state(NoAllocState** out) {
  int dev = 0;
  RA_CHECK_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lock(g_na_mu);
  auto it = g_na.find(dev);
  if (it == g_na.end()) {
    NoAllocState ns;
    RA_CHECK_HIP(hipGetSymbolAddress(&ns.base, HIP_SYMBOL(scratch)));
    if (!ns.base) return fail(RA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    it = g_na.emplace(dev, ns).first;
  }
  *out = &it->second;
  return RA_OK;
}

// Host tables of the allocation-free path (plain host vectors, built once per
// geometry and kept); written into the scratch through kernel arguments, and
// only when the scratch holds another geometry's tables.
std::map<std::string, std::pair<std::vector<float>, std::array<size_t, 4>>> g_na_tables;

int noalloc_tables(const ra_params* p, NoAllocState* ns, float* dev, hipStream_t s, ra::RopeTables* out) {
  const std::string key = table_key(p);
  std::lock_guard<std::mutex> lock(g_na_mu);
  auto it = g_na_tables.find(key);
  if (it == g_na_tables.end()) {
    std::vector<float> host;
    std::array<size_t, 4> off{};
    build_table(p, host, off.data());
    it = g_na_tables.emplace(key, std::make_pair(std::move(host), off)).first;
  }
  if (ns->resident != key) {
    RA_CHECK_HIP(ra::launch_write_floats(it->second.first.data(), it->second.first.size(), dev, s));
    ns->resident = key;
  }
  *out = tables_at(p, dev, it->second.second.data());
  return RA_OK;
}

}  // namespace

// Input tensors and code buffers are read and written in 16-byte pieces.
bool al16(const void* ptr) { return ptr == nullptr || reinterpret_cast<uintptr_t>(ptr) % 16 == 0; }

int check_align(std::initializer_list<const void*> ptrs) {
  for (const void* ptr : ptrs)
    if (!al16(ptr)) return fail(RA_ERR_INVALID, "tensor pointers must be 16-byte aligned");
  return RA_OK;
}

extern "C" {

int rotate_attn_layout(const ra_params* p, ra_layout* out) {
  int rc = validate(p);
  if (rc) return rc;
  if (!out) return fail(RA_ERR_INVALID, "out is NULL");
  const Sizes s = sizes_of(p);
  out->n_pad = s.Npad;
  out->qk_code_bytes = static_cast<int64_t>(s.codes);
  out->q_scale_count = static_cast<int64_t>(s.qscale);
  out->k_scale_count = static_cast<int64_t>(s.kscale);
  out->v_code_bytes = static_cast<int64_t>(s.codes);
  out->v_scale_count = static_cast<int64_t>(s.vscale);
  out->mu_count = static_cast<int64_t>(s.mu);
  out->k_bias_count = static_cast<int64_t>(s.kbias);
  return RA_OK;
}

int rotate_attn_workspace_size(const ra_params* p, int path, size_t* bytes) {
  int rc = validate(p);
  if (rc) return rc;
  if (!bytes) return fail(RA_ERR_INVALID, "bytes is NULL");
  if (path == RA_PATH_INT4) {
    *bytes = carve_int4(p, nullptr).total;
  } else if (path == RA_PATH_FP16) {
    *bytes = carve_fp16(p, nullptr).total;
  } else {
    return fail(RA_ERR_INVALID, "unknown path");
  }
  return RA_OK;
}

int rotate_attn_quantize_qk(const ra_params* p, const void* q, const void* k, uint8_t* q_codes, float* q_scale,
                            uint8_t* k_codes, float* k_scale, float* mu_k, float* mu_q, float* k_bias,
                            void* workspace, size_t workspace_bytes, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q || !k || !q_codes || !q_scale || !k_codes || !k_scale) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({q, k, q_codes, k_codes}))) return rc;
  if ((p->smooth & RA_SMOOTH_Q) && !k_bias) return fail(RA_ERR_INVALID, "RA_SMOOTH_Q needs k_bias");
  const Int4Ws need = carve_int4(p, nullptr);
  if ((rc = check_ws(workspace, workspace_bytes, need.total))) return rc;
  const Int4Ws w = carve_int4(p, workspace);
  ra::RopeTables t;
  TableCopy tc;
  if ((rc = put_tables(p, w.tables, st(stream), &t, &tc))) return rc;
  ProdOut out;
  out.qc = q_codes;
  out.qs = q_scale;
  out.kc = k_codes;
  out.ks = k_scale;
  out.mu_k = mu_k;
  out.mu_q = mu_q;
  out.kbias = k_bias;
  return produce(p, t, tc, q, k, nullptr, out, w, st(stream));
}

int rotate_attn_quantize_v(const ra_params* p, const void* v, uint8_t* v_codes, float* v_scale, float* mu_v,
                           void* workspace, size_t workspace_bytes, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!v || !v_codes || !v_scale) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({v, v_codes}))) return rc;
  const Int4Ws need = carve_int4(p, nullptr);
  if ((rc = check_ws(workspace, workspace_bytes, need.total))) return rc;
  ProdOut out;
  out.vc = v_codes;
  out.vs = v_scale;
  out.mu_v = mu_v;
  return produce(p, ra::RopeTables{}, TableCopy{}, nullptr, nullptr, v, out, carve_int4(p, workspace), st(stream));
}

int rotate_attn_quantize_qkv(const ra_params* p, const void* q, const void* k, const void* v, uint8_t* q_codes,
                             float* q_scale, uint8_t* k_codes, float* k_scale, uint8_t* v_codes, float* v_scale,
                             float* mu_k, float* mu_q, float* mu_v, float* k_bias, void* workspace,
                             size_t workspace_bytes, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q || !k || !v || !q_codes || !q_scale || !k_codes || !k_scale || !v_codes || !v_scale)
    return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({q, k, v, q_codes, k_codes, v_codes}))) return rc;
  if ((p->smooth & RA_SMOOTH_Q) && !k_bias) return fail(RA_ERR_INVALID, "RA_SMOOTH_Q needs k_bias");
  const Int4Ws need = carve_int4(p, nullptr);
  if ((rc = check_ws(workspace, workspace_bytes, need.total))) return rc;
  const Int4Ws w = carve_int4(p, workspace);
  ra::RopeTables t;
  TableCopy tc;
  if ((rc = put_tables(p, w.tables, st(stream), &t, &tc))) return rc;
  ProdOut out;
  out.qc = q_codes;
  out.qs = q_scale;
  out.kc = k_codes;
  out.ks = k_scale;
  out.vc = v_codes;
  out.vs = v_scale;
  out.mu_k = mu_k;
  out.mu_q = mu_q;
  out.mu_v = mu_v;
  out.kbias = k_bias;
  return produce(p, t, tc, q, k, v, out, w, st(stream));
}

int rotate_attn_attn_int4(const ra_params* p, const uint8_t* q_codes, const float* q_scale, const uint8_t* k_codes,
                          const float* k_scale, const uint8_t* v_codes, const float* v_scale, const float* mu_v,
                          const float* k_bias, void* o, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q_codes || !q_scale || !k_codes || !k_scale || !v_codes || !v_scale || !o)
    return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((p->smooth & RA_SMOOTH_Q) && !k_bias) return fail(RA_ERR_INVALID, "RA_SMOOTH_Q needs k_bias");
  return attn_impl(p, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, mu_v, k_bias, o, false, 0, 0, 0, nullptr,
                   nullptr, nullptr, st(stream));
}

int rotate_attn_attn_int4_debug(const ra_params* p, const uint8_t* q_codes, const float* q_scale,
                                const uint8_t* k_codes, const float* k_scale, const uint8_t* v_codes,
                                const float* v_scale, const float* mu_v, const float* k_bias, void* o, int32_t bh,
                                int32_t row0, int32_t rows, int32_t* s_out, uint8_t* u_out, float* m_out,
                                void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q_codes || !q_scale || !k_codes || !k_scale || !v_codes || !v_scale || !o)
    return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((p->smooth & RA_SMOOTH_Q) && !k_bias) return fail(RA_ERR_INVALID, "RA_SMOOTH_Q needs k_bias");
  if (bh < 0 || static_cast<int64_t>(bh) >= static_cast<int64_t>(p->B) * p->H) return fail(RA_ERR_INVALID, "bh out of range");
  if (row0 < 0 || rows < 0 || static_cast<int64_t>(row0) + rows > p->N) return fail(RA_ERR_INVALID, "rows out of range");
  return attn_impl(p, q_codes, q_scale, k_codes, k_scale, v_codes, v_scale, mu_v, k_bias, o, true, bh, row0, rows,
                   s_out, u_out, m_out, st(stream));
}

int rotate_attn_fwd_int4(const ra_params* p, const void* q, const void* k, const void* v, void* o, void* workspace,
                         size_t workspace_bytes, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q || !k || !v || !o) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({q, k, v}))) return rc;
  const Int4Ws need = carve_int4(p, nullptr);
  if ((rc = check_ws(workspace, workspace_bytes, need.total))) return rc;
  const Int4Ws w = carve_int4(p, workspace);
  ra::RopeTables t;
  TableCopy tc;
  if ((rc = put_tables(p, w.tables, st(stream), &t, &tc))) return rc;
  return int4_forward(p, t, tc, q, k, v, o, w, st(stream));
}

int rotate_attn_fwd_int4_noalloc(const ra_params* p, const void* q, const void* k, const void* v, void* o,
                                 void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q || !k || !v || !o) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({q, k, v}))) return rc;
  const size_t need = carve_int4(p, nullptr).total;
  if (need > kNoAllocBytes)
    return fail(RA_ERR_UNSUPPORTED, "problem needs " + std::to_string(need) + " bytes of scratch; the allocation-free "
                "entry point holds " + std::to_string(kNoAllocBytes));
  NoAllocState* ns = nullptr;
  if ((rc = noalloc_state(&ns))) return rc;
  const Int4Ws w = carve_int4(p, ns->base);
  ra::RopeTables t;
  if ((rc = noalloc_tables(p, ns, w.tables, st(stream), &t))) return rc;
  return int4_forward(p, t, TableCopy{}, q, k, v, o, w, st(stream));
}

int rotate_attn_prepare_fp16(const ra_params* p, const void* q, const void* k, const void* v, void* workspace,
                             size_t workspace_bytes, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q || !k || !v) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({q, k, v}))) return rc;
  const Fp16Ws need = carve_fp16(p, nullptr);
  if ((rc = check_ws(workspace, workspace_bytes, need.total))) return rc;
  return fp16_prepare_impl(p, q, k, v, carve_fp16(p, workspace), st(stream));
}

int rotate_attn_attn_fp16(const ra_params* p, const void* workspace, size_t workspace_bytes, void* o, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!o) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  const Fp16Ws need = carve_fp16(p, nullptr);
  if ((rc = check_ws(const_cast<void*>(workspace), workspace_bytes, need.total))) return rc;
  return fp16_attn_impl(p, carve_fp16(p, const_cast<void*>(workspace)), o, st(stream));
}

int rotate_attn_fwd_fp16(const ra_params* p, const void* q, const void* k, const void* v, void* o, void* workspace,
                         size_t workspace_bytes, void* stream) {
  int rc = validate(p);
  if (rc) return rc;
  if (!q || !k || !v || !o) return fail(RA_ERR_INVALID, "NULL tensor pointer");
  if ((rc = check_align({q, k, v}))) return rc;
  const Fp16Ws need = carve_fp16(p, nullptr);
  if ((rc = check_ws(workspace, workspace_bytes, need.total))) return rc;
  const Fp16Ws w = carve_fp16(p, workspace);
  if ((rc = fp16_prepare_impl(p, q, k, v, w, st(stream)))) return rc;
  return fp16_attn_impl(p, w, o, st(stream));
}

int rotate_attn_fwd(const ra_params* p, int fallback, const void* q, const void* k, const void* v, void* o,
                    void* workspace, size_t workspace_bytes, void* stream) {
  if (fallback) return rotate_attn_fwd_fp16(p, q, k, v, o, workspace, workspace_bytes, stream);
  return rotate_attn_fwd_int4(p, q, k, v, o, workspace, workspace_bytes, stream);
}

const char* rotate_attn_error_string(int status) {
  switch (status) {
    case RA_OK: return "ok";
    case RA_ERR_INVALID: return "invalid argument";
    case RA_ERR_UNSUPPORTED: return "unsupported configuration";
    case RA_ERR_WORKSPACE: return "workspace missing or too small";
    case RA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* rotate_attn_last_error(void) { return g_err.c_str(); }

}  // extern "C"
