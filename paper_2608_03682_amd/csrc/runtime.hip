// Host runtime behind the C ABI: validation, weight packing, working buffers,
// timestep tables, and capture/replay of the K-step loop as a HIP graph.
//
// The runner owns every mutable buffer of the loop and the graph buckets
// keyed by (batch, steps); the prefix state is a read-only per-call input
// whose validity is one chunk (Section "PhyAI Architecture", paragraphs
// "Overview" and "Graph replay").
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <functional>
#include <cstring>
#include <map>
#include <mutex>
#include <stdexcept>
#include <string>
#include <utility>
#include <vector>

#include "../../include/phyai.h"
#include "kernels.hpp"

using namespace phyai;

namespace {

thread_local std::string g_err;

struct Fail {
  int code;
  std::string msg;
};

[[noreturn]] void fail(int code, const std::string& msg) { throw Fail{code, msg}; }

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) fail(PHYAI_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}
#define HIPC(x) hip_check((x), #x)

uint16_t f2bf(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
float bf2f(uint16_t b) {
  const uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

struct DevMem {
  std::vector<void*> ptrs;
  void* alloc(size_t bytes) {
    if (bytes == 0) bytes = 16;
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) fail(PHYAI_ENOMEM, "hipMalloc(" + std::to_string(bytes) + ") failed: " + hipGetErrorString(e));
    ptrs.push_back(p);
    return p;
  }
  template <typename T> T* alloc_n(size_t n) { return static_cast<T*>(alloc(n * sizeof(T))); }
  ~DevMem() {
    for (void* p : ptrs) (void)hipFree(p);
  }
};

struct Lin {
  void* w = nullptr;
  float* scale = nullptr;
  uint8_t* mx = nullptr;    // fp4: E8M0 scale exponents
  int K = 0, NPT = 0, kind = W_BF16;
};

struct LayerW {
  Lin qkv, kv_cross, o, gu, down, attn_mod, mlp_mod, ada;
  float *attn_norm = nullptr, *mlp_norm = nullptr;
  float *attn_mod_b = nullptr, *mlp_mod_b = nullptr, *ada_b = nullptr, *mlp_b1 = nullptr, *mlp_b2 = nullptr;
  // vision tower: LayerNorm biases, the fused [q | k | v] bias and the O bias
  float *attn_norm_b = nullptr, *mlp_norm_b = nullptr, *qkv_b = nullptr, *o_b = nullptr;
};

struct Bucket {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

}  // namespace

struct phyai_expert {
  phyai_config c{};
  bool f32 = false;
  int L = 0, d = 0, D = 0, nq = 0, nkv = 0, H = 0, A = 0, F = 0, M = 0, off = 0, qd = 0, kd = 0;
  int Bmax = 0, Kmax = 0, P = 0, Wpre = 0, act_bytes = 2;
  DevMem mem;
  // parameters
  float *in_w = nullptr, *in_b = nullptr, *state_w = nullptr, *state_b = nullptr, *pos = nullptr;
  // pi0: the action embedding folded into the time MLP's first layer
  // (x -> W_in x + b_in -> W1a (.) is one affine map of x): [A][d] and [d]
  float *tin_w = nullptr, *tin_b = nullptr;
  float *out_w = nullptr, *out_b = nullptr, *final_norm = nullptr;
  float *time_b1 = nullptr, *time_b2 = nullptr, *cond_b1 = nullptr, *cond_b2 = nullptr, *final_b = nullptr;
  Lin time_w1t, time_w2, cond_w1, cond_w2, final_mod;
  // vision tower: patch embedding, final LayerNorm bias, projector
  Lin patch_lin, proj_lin;
  float *patch_b = nullptr, *final_norm_b = nullptr, *proj_b = nullptr;
  int n_img = 1;            // images per request (vision); 1 otherwise
  std::vector<LayerW> layers;
  float* inv_freq = nullptr;
  float2* rope_cs = nullptr;   // per-call RoPE table [max_batch * M][D/2]
  // working buffers
  float *x = nullptr, *h = nullptr, *e_state = nullptr, *part = nullptr;
  void *n = nullptr, *zbuf = nullptr, *q = nullptr;
  void *o = nullptr, *g = nullptr;
  // per-layer key ranges: K [L][Bmax][nkv][ldk][D], V transposed [L][Bmax][nkv][D][ldk]
  void *kall = nullptr, *vt = nullptr;
  float* pend = nullptr;    // split-K partial sums of the residual GEMMs (small batches)
  // norms folded into the GEMMs (pi0, small batches): per-32-column sums of
  // h^2 of the rows the next GEMM normalises, and the residual GEMMs' tile
  // counters (zero between launches)
  float* ss = nullptr;
  unsigned* fin_ctr = nullptr;
  // the partial buffers the next enqueue uses: part/pend, or the static
  // scratch for phyai_denoise_static
  float *part_cur = nullptr, *pend_cur = nullptr;
  float* static_scratch = nullptr;   // this device's copy of the static scratch array
  // persistent batch-1 loop (pi0, bf16; opt-in): its argument block in device
  // memory and own buffers, set up on first use
  bool persist_ok = false, persist_ready = false;
  PersistArgs pargs{};
  PersistArgs* pargs_dev = nullptr;
  int ldk = 0;
  int64_t kv_layer = 0;     // elements per layer
  // two-term activations (hi + lo bf16) for the GEMMs fed by a norm or by GeGLU
  bool split_act = false;
  void *n_lo = nullptr, *g_lo = nullptr;
  CallDesc* desc = nullptr;
  // timestep tables
  void *tau = nullptr, *c1 = nullptr, *cact = nullptr;
  float *T = nullptr, *modtab = nullptr, *adatab = nullptr, *fintab = nullptr, *dt = nullptr;
  std::vector<float> ts_cached;
  // pinned staging of the host-built tables (sinusoid, dt): a schedule change
  // enqueues its upload from here; stage_ev marks the last upload's end
  void* stage = nullptr;
  hipEvent_t stage_ev = nullptr;
  int last_batch = 0;       // batch of the last phyai_denoise (0: none yet)
  std::map<std::pair<int, int>, Bucket> buckets;
  hipStream_t cap = nullptr;

  ~phyai_expert() {
    for (auto& kv : buckets) {
      if (kv.second.exec) (void)hipGraphExecDestroy(kv.second.exec);
      if (kv.second.graph) (void)hipGraphDestroy(kv.second.graph);
    }
    if (cap) (void)hipStreamDestroy(cap);
    if (stage_ev) (void)hipEventDestroy(stage_ev);
    if (stage) (void)hipHostFree(stage);
  }
};

namespace {

// ---------------------------------------------------------------------------
// Static scratch of phyai_denoise_static: the split-K and attention key-split
// partials of one call, in a file-scope device array (32 MiB, one copy per
// device, held until the process ends).  Host code never uses the array's
// name as an address: its device address is looked up once per device with
// that device current and kept in g_scratch.
// ---------------------------------------------------------------------------
constexpr int64_t kStaticScratchFloats = int64_t(8) << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) float scratch[kStaticScratchFloats];
std::mutex g_scratch_mu;
float* g_scratch[kMaxDevices] = {};

float* static_scratch_ptr() {
  int dev = 0;
  HIPC(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) fail(PHYAI_EUNSUPPORTED, "device index beyond the static scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    HIPC(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) fail(PHYAI_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch[dev] = static_cast<float*>(p);
  }
  return g_scratch[dev];
}

// ---------------------------------------------------------------------------
// parameter lookup and packing
// ---------------------------------------------------------------------------
struct Params {
  std::map<std::string, const phyai_tensor*> by_name;
  const phyai_tensor* get(const std::string& n, int rows, int cols) const {
    auto it = by_name.find(n);
    if (it == by_name.end()) fail(PHYAI_EINVAL, "missing tensor '" + n + "'");
    const phyai_tensor* t = it->second;
    if (t->rows != rows || t->cols != cols)
      fail(PHYAI_EINVAL, "tensor '" + n + "' has shape [" + std::to_string(t->rows) + "][" +
                             std::to_string(t->cols) + "], expected [" + std::to_string(rows) + "][" +
                             std::to_string(cols) + "]");
    if (!t->data) fail(PHYAI_EINVAL, "tensor '" + n + "' has no data");
    return t;
  }
};

float elem_f32(const phyai_tensor* t, int64_t i) {
  if (t->dtype == PHYAI_DTYPE_F32) return static_cast<const float*>(t->data)[i];
  if (t->dtype == PHYAI_DTYPE_BF16) return bf2f(static_cast<const uint16_t*>(t->data)[i]);
  fail(PHYAI_EINVAL, std::string("tensor '") + t->name + "' must be F32 or BF16 here");
}

// Small parameters used by the row kernels are kept as fp32 (exact decode).
float* upload_f32(phyai_expert& e, const phyai_tensor* t, hipStream_t s) {
  const int64_t n = (int64_t)t->rows * t->cols;
  std::vector<float> v(n);
  for (int64_t i = 0; i < n; ++i) v[i] = elem_f32(t, i);
  float* p = e.mem.alloc_n<float>(n);
  HIPC(hipMemcpyAsync(p, v.data(), n * 4, hipMemcpyHostToDevice, s));
  HIPC(hipStreamSynchronize(s));
  return p;
}

// Vectors ([1][n] each) concatenated into one fp32 device array.
float* upload_concat_f32(phyai_expert& e, const std::vector<const phyai_tensor*>& srcs, hipStream_t s) {
  std::vector<float> v;
  for (auto* t : srcs)
    for (int64_t i = 0; i < (int64_t)t->rows * t->cols; ++i) v.push_back(elem_f32(t, i));
  float* p = e.mem.alloc_n<float>(v.size());
  HIPC(hipMemcpyAsync(p, v.data(), v.size() * 4, hipMemcpyHostToDevice, s));
  HIPC(hipStreamSynchronize(s));
  return p;
}

// Pack the column-concatenation of `srcs` ([K][sum cols]) into MFMA operand
// order.  perm(pc) gives the logical column of packed column pc (-1: zero).
template <class Perm>
Lin pack_linear(phyai_expert& e, const std::vector<const phyai_tensor*>& srcs, int Np, Perm perm, int kind,
                hipStream_t s) {
  const int K = srcs[0]->rows;
  std::vector<int> src_of, col_of;
  for (size_t i = 0; i < srcs.size(); ++i) {
    if (srcs[i]->rows != K) fail(PHYAI_EINVAL, "fused linear sources disagree in rows");
    const int want = kind == W_FP8   ? PHYAI_DTYPE_FP8E4M3
                     : kind == W_FP4 ? PHYAI_DTYPE_FP4E2M1
                     : kind == W_BF16 ? PHYAI_DTYPE_BF16 : PHYAI_DTYPE_F32;
    if (srcs[i]->dtype != want)
      fail(PHYAI_EINVAL, std::string("tensor '") + srcs[i]->name + "' has the wrong dtype for this path");
    if ((kind == W_FP8 || kind == W_FP4) && !srcs[i]->scale)
      fail(PHYAI_EINVAL, std::string("tensor '") + srcs[i]->name + "' needs scales");
    if (kind == W_FP4) {
      if (srcs[i]->cols % 2 || K % 32)
        fail(PHYAI_EINVAL, std::string("fp4 tensor '") + srcs[i]->name + "' needs even cols and rows % 32 == 0");
      // scales: finite powers of two in the normal range, 2^-126 .. 2^127
      const int64_t ns = (int64_t)(K / 32) * srcs[i]->cols;
      for (int64_t q = 0; q < ns; ++q) {
        uint32_t u;
        std::memcpy(&u, &srcs[i]->scale[q], 4);
        const uint32_t ex = (u >> 23) & 0xff;
        if ((u & 0x807fffffu) != 0 || ex == 0 || ex == 0xff)
          fail(PHYAI_EINVAL, std::string("fp4 tensor '") + srcs[i]->name + "' has a scale that is not a power of two");
      }
    }
    for (int c = 0; c < srcs[i]->cols; ++c) {
      src_of.push_back((int)i);
      col_of.push_back(c);
    }
  }
  if (Np % 32) fail(PHYAI_EINVAL, "packed width must be a multiple of 32");
  if (kind != W_F32 && K % 64) fail(PHYAI_EUNSUPPORTED, "MFMA linears need K % 64 == 0");
  Lin L;
  L.K = K;
  L.NPT = Np / 32;
  L.kind = kind;
  const int nkb = K / 64;
  if (kind == W_F32) {
    std::vector<float> buf((size_t)K * Np, 0.f);
    for (int pc = 0; pc < Np; ++pc) {
      const int lc = perm(pc);
      if (lc < 0) continue;
      const phyai_tensor* t = srcs[src_of[lc]];
      const int cc = col_of[lc];
      for (int k = 0; k < K; ++k) buf[(size_t)k * Np + pc] = static_cast<const float*>(t->data)[(int64_t)k * t->cols + cc];
    }
    L.w = e.mem.alloc(buf.size() * 4);
    HIPC(hipMemcpyAsync(L.w, buf.data(), buf.size() * 4, hipMemcpyHostToDevice, s));
    HIPC(hipStreamSynchronize(s));
    return L;
  }
  if (kind == W_FP4) {
    // codes: 8 bytes per (pair tile, k-block, half, lane): k-step 0 in bytes
    // 0-3, k-step 1 in bytes 4-7, value j of a step in byte j / 2 (low nibble
    // first); exponents: per (pair tile, k-block, half) [16 columns][2 steps]
    std::vector<uint8_t> buf((size_t)K * Np / 2, 0);
    std::vector<uint8_t> mx((size_t)(K / 32) * Np, 127);
    for (int pc = 0; pc < Np; ++pc) {
      const int lc = perm(pc);
      if (lc < 0) continue;
      const int p = pc / 32, hf = (pc % 32) / 16, c = pc % 16;
      const phyai_tensor* t = srcs[src_of[lc]];
      const int cc = col_of[lc];
      const uint8_t* codes = static_cast<const uint8_t*>(t->data);
      for (int k = 0; k < K; ++k) {
        const int kb = k / 64, st = (k % 64) / 32, kg = (k % 32) / 8, j = k % 8;
        const int lane = kg * 16 + c;
        const size_t frag = ((size_t)(p * nkb + kb) * 2 + hf) * 64 + lane;
        const uint8_t code = (codes[(int64_t)k * (t->cols / 2) + cc / 2] >> (4 * (cc & 1))) & 0xF;
        buf[frag * 8 + st * 4 + j / 2] |= code << (4 * (j & 1));
        if (k % 32 == 0) {
          uint32_t u;
          std::memcpy(&u, &t->scale[(int64_t)(k / 32) * t->cols + cc], 4);
          mx[((size_t)(p * nkb + kb) * 2 + hf) * 32 + 2 * c + st] = (u >> 23) & 0xff;
        }
      }
    }
    L.w = e.mem.alloc(buf.size());
    HIPC(hipMemcpyAsync(L.w, buf.data(), buf.size(), hipMemcpyHostToDevice, s));
    L.mx = static_cast<uint8_t*>(e.mem.alloc(mx.size()));
    HIPC(hipMemcpyAsync(L.mx, mx.data(), mx.size(), hipMemcpyHostToDevice, s));
    HIPC(hipStreamSynchronize(s));
    return L;
  }
  const size_t esz = kind == W_FP8 ? 1 : 2;
  std::vector<uint8_t> buf((size_t)K * Np * esz, 0);
  std::vector<float> sc(kind == W_FP8 ? Np : 0, 1.f);
  for (int pc = 0; pc < Np; ++pc) {
    const int lc = perm(pc);
    const int p = pc / 32, hf = (pc % 32) / 16, c = pc % 16;
    const phyai_tensor* t = lc >= 0 ? srcs[src_of[lc]] : nullptr;
    const int cc = lc >= 0 ? col_of[lc] : 0;
    if (kind == W_FP8 && t) sc[pc] = t->scale[cc];
    for (int k = 0; k < K; ++k) {
      const int kb = k / 64, st = (k % 64) / 32, kg = (k % 32) / 8, j = k % 8;
      const int lane = kg * 16 + c;
      const size_t frag = ((size_t)(p * nkb + kb) * 2 + hf) * 64 + lane;
      if (kind == W_FP8) {
        const uint8_t v = t ? static_cast<const uint8_t*>(t->data)[(int64_t)k * t->cols + cc] : 0;
        buf[frag * 16 + st * 8 + j] = v;
      } else {
        const uint16_t v = t ? static_cast<const uint16_t*>(t->data)[(int64_t)k * t->cols + cc] : 0;
        std::memcpy(&buf[(frag * 2 + st) * 16 + j * 2], &v, 2);
      }
    }
  }
  L.w = e.mem.alloc(buf.size());
  HIPC(hipMemcpyAsync(L.w, buf.data(), buf.size(), hipMemcpyHostToDevice, s));
  if (kind == W_FP8) {
    L.scale = e.mem.alloc_n<float>(Np);
    HIPC(hipMemcpyAsync(L.scale, sc.data(), Np * 4, hipMemcpyHostToDevice, s));
  }
  HIPC(hipStreamSynchronize(s));
  return L;
}

Lin pack_identity(phyai_expert& e, const std::vector<const phyai_tensor*>& srcs, int kind, hipStream_t s) {
  int N = 0;
  for (auto* t : srcs) N += t->cols;
  const int Np = (N + 31) / 32 * 32;
  return pack_linear(e, srcs, Np, [N](int pc) { return pc < N ? pc : -1; }, kind, s);
}

// Heads [q | k | v], each D wide: pair tile j of a head holds dims 16j+c and
// D/2 + 16j + c (the RoPE pair).
Lin pack_heads(phyai_expert& e, const std::vector<const phyai_tensor*>& srcs, int D, int kind, hipStream_t s) {
  int N = 0;
  for (auto* t : srcs) N += t->cols;
  return pack_linear(e, srcs, N, [D](int pc) {
    const int p = pc / 32, hf = (pc % 32) / 16, c = pc % 16;
    const int tiles = D / 32;
    const int head = p / tiles, j = p % tiles;
    return head * D + hf * (D / 2) + 16 * j + c;
  }, kind, s);
}

// [gate | up], F wide each: pair tile p holds gate col 16p+c and up col 16p+c.
Lin pack_geglu(phyai_expert& e, const phyai_tensor* gate, const phyai_tensor* up, int kind, hipStream_t s) {
  const int F = gate->cols;
  return pack_linear(e, {gate, up}, 2 * F, [F](int pc) {
    const int p = pc / 32, hf = (pc % 32) / 16, c = pc % 16;
    return hf * F + 16 * p + c;
  }, kind, s);
}

// ---------------------------------------------------------------------------
// launch helpers (overloads on the activation type)
// ---------------------------------------------------------------------------
void gemm_store(const GemmArgs& g, const EpiStore<bf16_t>& e, hipStream_t s) { gemm_store_bf16(g, e, s); }
void gemm_store(const GemmArgs& g, const EpiStore<float>& e, hipStream_t s) { gemm_store_f32(g, e, s); }
void gemm_geglu(const GemmArgs& g, const EpiGeglu<bf16_t>& e, hipStream_t s) { gemm_geglu_bf16(g, e, s); }
void gemm_geglu(const GemmArgs& g, const EpiGeglu<float>& e, hipStream_t s) { gemm_geglu_f32(g, e, s); }
void gemm_qkv(const GemmArgs& g, const EpiQkv<bf16_t>& e, hipStream_t s) { gemm_qkv_bf16(g, e, s); }
void gemm_qkv(const GemmArgs& g, const EpiQkv<float>& e, hipStream_t s) { gemm_qkv_f32(g, e, s); }
void gemm_kv(const GemmArgs& g, const EpiKV<bf16_t>& e, hipStream_t s) { gemm_kv_bf16(g, e, s); }
void gemm_kv(const GemmArgs& g, const EpiKV<float>& e, hipStream_t s) { gemm_kv_f32(g, e, s); }
void prefix_relayout(const RelayoutArgs& r, bf16_t*, hipStream_t s) { prefix_relayout_bf16(r, s); }
void prefix_relayout(const RelayoutArgs& r, float*, hipStream_t s) { prefix_relayout_f32(r, s); }
void norm_rows(float* h, bf16_t* n, bf16_t* n_lo, int R, int d, float eps, int mode, const float* mul,
               const float* sh, const PendingResid& p, hipStream_t s) {
  norm_rows_bf16(h, n, n_lo, R, d, eps, mode, mul, sh, p, s);
}
void norm_rows(float* h, float* n, float*, int R, int d, float eps, int mode, const float* mul, const float* sh,
               const PendingResid& p, hipStream_t s) {
  norm_rows_f32(h, n, R, d, eps, mode, mul, sh, p, s);
}

GemmArgs gargs(const Lin& w, const void* A, int lda, int R) {
  GemmArgs g{};
  g.A = A;
  g.lda = lda;
  g.R = R;
  g.K = w.K;
  g.NPT = w.NPT;
  g.W = w.w;
  g.scale = w.scale;
  g.mx = w.mx;
  g.kind = w.kind;
  return g;
}

template <typename T> EpiStore<T> store_epi(T* out, int ldo, const float* bias, const float* rowvec, int act) {
  EpiStore<T> e{};
  e.out = out;
  e.ldo = ldo;
  e.bias = bias;
  e.rowvec = rowvec;
  e.act = act;
  return e;
}

// split of the keys across blocks so that small batches still fill the chip
int attn_splits_for(int B, int rows, int nkv, int keys, int rpb) {
  const int base = ((rows + rpb - 1) / rpb) * B * nkv;   // blocks without a split
  int s = (256 + base - 1) / base;
  const int cap = (keys + 63) / 64;                     // at least one 64-key tile per split
  if (s > cap) s = cap;
  if (s > 16) s = 16;                                   // the merge kernel takes up to 16
  // a few key tiles over a grid that already covers a quarter of the chip:
  // the combine launch costs more than the split saves (vision tower, 256
  // keys, 96 blocks: 7.0 us unsplit against 12.8 with 3 splits + combine)
  if (cap <= 4 && base >= 64) s = 1;
  return s < 1 ? 1 : s;
}
int attn_splits(int B, int rows, int nkv, int keys) {
  return attn_splits_for(B, rows, nkv, keys, attention_rows_per_block(B, rows, nkv));
}
// the most splits either block height can ask for (buffers are sized with it,
// so that forcing the other height at a later call still fits)
int attn_splits_max(int B, int rows, int nkv, int keys) {
  return std::max(attn_splits_for(B, rows, nkv, keys, 64), attn_splits_for(B, rows, nkv, keys, 128));
}

// key splits of block l's attention at batch B (DiT: even blocks attend to
// the features, odd ones to the suffix)
int attn_split_of(const phyai_expert& e, int l, int B) {
  if (e.f32) return 1;
  const int rows = e.M * (e.nq / e.nkv);
  const int keys = e.c.variant != PHYAI_VARIANT_DIT ? e.P + e.M : (l % 2 == 0 ? e.P : e.M);
  return attn_splits(B, rows, e.nkv, keys);
}

// Whether block l's output projection merges the attention's key splits
// itself (small row counts; PHYAI_ATTN_MERGE=kernel keeps the separate merge
// kernel, read at enqueue time).  It then splits K into 256-wide slices.
bool oproj_merges(const phyai_expert& e, int l, int B) {
  if (e.f32 || B * e.M >= 256) return false;
  const char* f = getenv("PHYAI_ATTN_MERGE");
  if (f && strcmp(f, "kernel") == 0) return false;
  const int K = e.nq * e.D;
  return attn_split_of(e, l, B) > 1 && K % 256 == 0 && K / 256 <= 8 && 256 % e.D == 0;
}

// Split over K used for a residual GEMM of block l (which: 0 = O projection,
// 1 = down / MLP-out projection) at batch B; 1 means the epilogue adds into h
// directly.
int resid_split(const phyai_expert& e, int which, int l, int B) {
  if (e.f32) return 1;
  if (which == 0 && oproj_merges(e, l, B)) return e.nq * e.D / 256;
  const Lin& w = which == 0 ? e.layers[l].o : e.layers[l].down;
  return gemm_split_k(B * e.M, w.NPT, w.K);
}

// Counters of the residual GEMMs' split-K finishing: one per output tile.
constexpr int kFinCounters = 4096;

// Whether the RMSNorms of block l > 0 (before the QKV GEMM) and of every
// block's MLP fold into the GEMMs at batch B (the paper's fused residual-add
// + RMSNorm, paragraph "Kernel fusion"): pi0 on the bf16 path, every residual
// GEMM split over K (small batches), so that the block completing an output
// tile adds the split slices into h and leaves bf16(h (1 + w)) and the
// tile's sums of h^2 for the next GEMM, which scales its rows by 1/rms.
// Opt-in (PHYAI_NORM_FOLD=1, read at enqueue time): on MI355X the tile
// finishing (an atomic round trip, then the slices' device-scope loads) and
// the row scales cost the residual and consuming GEMMs more than the two norm
// launches per block they replace (pi0 batch 1: 8.86 against 8.29 ms).
bool fold_norms(const phyai_expert& e, int B) {
  if (e.c.variant != PHYAI_VARIANT_PI0 || e.f32 || !e.fin_ctr) return false;
  const char* f = getenv("PHYAI_NORM_FOLD");
  if (!f || f[0] != '1') return false;
  const int R = B * e.M;
  if ((int64_t)(e.d / 32) * ((R + 15) / 16) > kFinCounters) return false;
  for (int l = 0; l < e.L; ++l)
    if (resid_split(e, 0, l, B) <= 1 || resid_split(e, 1, l, B) <= 1) return false;
  return true;
}

// The residual contribution a split GEMM left pending, for its consumer.
PendingResid pending_of(const phyai_expert& e, int which, int l, int k, int B) {
  PendingResid p{};
  const int S = resid_split(e, which, l, B);
  if (S <= 1) return p;
  p.part = e.pend_cur;
  p.n = S;
  p.stride = (int64_t)B * e.M * e.d;
  if (e.c.variant == PHYAI_VARIANT_DIT) {
    const float* ada = e.adatab + ((int64_t)k * e.L + l) * 6 * e.d;
    p.gate = which == 0 ? ada + 2 * e.d : ada + 5 * e.d;
    p.bias = which == 0 ? nullptr : e.layers[l].mlp_b2;
  }
  if (e.c.variant == PHYAI_VARIANT_VISION) p.bias = which == 0 ? e.layers[l].o_b : e.layers[l].mlp_b2;
  return p;
}

// ---------------------------------------------------------------------------
// the K-step loop
// ---------------------------------------------------------------------------
// One stage of transformer block l at step k (the graph records them in
// order; phyai_profile_stage replays a single one).
enum Stage { ST_NORM1 = 0, ST_QKV, ST_ATTN, ST_OPROJ, ST_NORM2, ST_MLP_UP, ST_MLP_DOWN, kStages };

template <typename T>
void layer_stage(phyai_expert& e, int stage, int l, int k, int B, hipStream_t s) {
  const int d = e.d, M = e.M, L = e.L, D = e.D;
  const int R = B * M;
  T* n = static_cast<T*>(e.n);
  T* q = static_cast<T*>(e.q);
  // the vision tower needs a block's keys only inside that block: one range
  const int64_t kv_slot = e.c.variant == PHYAI_VARIANT_VISION ? 0 : l;
  T* kl = static_cast<T*>(e.kall) + kv_slot * e.kv_layer;
  T* vl = static_cast<T*>(e.vt) + kv_slot * e.kv_layer;
  T* o = static_cast<T*>(e.o);
  T* g = static_cast<T*>(e.g);
  T* n_lo = static_cast<T*>(e.n_lo);
  T* g_lo = static_cast<T*>(e.g_lo);
  auto with_lo = [](GemmArgs ga, const void* lo) { ga.A_lo = lo; return ga; };
  auto with_split = [&](GemmArgs ga, int which) {
    const int sk = resid_split(e, which, l, B);
    if (sk > 1) {
      ga.split_out = e.pend_cur;
      ga.split_stride = (int64_t)R * d;
      ga.split_k = sk;
    }
    return ga;
  };
  const int variant = e.c.variant;
  // a prefix LM's rows are the prefix tokens: keys at positions 0 .. M-1,
  // every valid token sees every valid token
  const bool plm = variant == PHYAI_VARIANT_PREFIX_LM;
  const int S = 2 * L + 1;   // pi0.5 norm sites
  const LayerW& w = e.layers[l];
  const float inv_sqrt_d = 1.0f / std::sqrt((float)D);
  AttnArgs at{};
  at.q = q; at.ldq = e.qd;
  at.K = kl; at.Vt = vl; at.ldk = e.ldk;
  at.out = o; at.ldo = e.qd;
  at.part = e.part_cur;
  at.desc = e.desc;
  at.B = B; at.M = M; at.nq = e.nq; at.nkv = e.nkv; at.D = D;
  at.scale = inv_sqrt_d;
  at.n_split = attn_split_of(e, l, B);
  const bool merge_in_o = oproj_merges(e, l, B);
  at.defer_merge = merge_in_o ? 1 : 0;
  // output projection: from the merged attention output, or from its key-split partials
  // folded norms: the residual GEMMs finish their tiles (next norm's gain
  // `gain`, null after the last block), the QKV and gate/up GEMMs scale rows
  const bool fold = fold_norms(e, B);
  auto with_fin = [&](GemmArgs ga, const float* gain) {
    if (fold) {
      ga.fin_h = e.h;
      ga.fin_a = static_cast<bf16_t*>(e.n);
      ga.fin_ss = e.ss;
      ga.fin_gain = gain;
      ga.fin_ctr = e.fin_ctr;
    }
    return ga;
  };
  auto with_rows = [&](GemmArgs ga) {
    ga.row_ss = e.ss;
    ga.row_nt = d / 32;
    ga.row_eps = e.c.rms_eps;
    return ga;
  };
  auto oproj = [&](const EpiResid& er) {
    const GemmArgs ga = with_fin(with_split(gargs(w.o, o, e.qd, R), 0), w.mlp_norm);
    if (merge_in_o) gemm_merge_resid(ga, attention_parts(at), er, s);
    else gemm_resid(ga, er, s);
  };

  if (variant == PHYAI_VARIANT_VISION) {
    // pre-norm ViT block over the patches of each image (the rows of one
    // image are one "request" of M = n_patches keys, all valid)
    switch (stage) {
      case ST_NORM1: {
        const PendingResid pd = l > 0 ? pending_of(e, 1, l - 1, k, B) : PendingResid{};
        norm_rows(e.h, n, n_lo, R, d, e.c.rms_eps, NORM_LN, w.attn_norm, w.attn_norm_b, pd, s);
        break;
      }
      case ST_QKV: {
        EpiQkv<T> eq{q, kl, vl, D, e.nq, e.nkv, 0, M, e.ldk, 0, nullptr, e.desc, w.qkv_b};
        gemm_qkv(gargs(w.qkv, n, d, R), eq, s);
        break;
      }
      case ST_ATTN: {
        at.keys_from_prefix = 1;
        at.n_suffix = 0;
        at.mask_mode = 0;
        if (e.f32) attention_f32(at, s); else attention_bf16(at, s);
        break;
      }
      case ST_OPROJ: oproj(EpiResid{e.h, d, w.o_b, nullptr}); break;
      case ST_NORM2:
        norm_rows(e.h, n, n_lo, R, d, e.c.rms_eps, NORM_LN, w.mlp_norm, w.mlp_norm_b, pending_of(e, 0, l, k, B), s);
        break;
      case ST_MLP_UP:
        gemm_store(gargs(w.gu, n, d, R), store_epi<T>(g, e.F, w.mlp_b1, nullptr, ACT_GELU), s);
        break;
      case ST_MLP_DOWN: gemm_resid(with_split(gargs(w.down, g, e.F, R), 1), EpiResid{e.h, d, w.mlp_b2, nullptr}, s); break;
    }
    return;
  }
  if (variant != PHYAI_VARIANT_DIT) {
    const float* mul1 = w.attn_norm;
    const float* sh1 = nullptr;
    const float* mul2 = w.mlp_norm;
    const float* sh2 = nullptr;
    if (variant == PHYAI_VARIANT_PI05) {
      mul1 = e.modtab + ((int64_t)k * S + 2 * l) * 2 * d;
      sh1 = mul1 + d;
      mul2 = e.modtab + ((int64_t)k * S + 2 * l + 1) * 2 * d;
      sh2 = mul2 + d;
    }
    switch (stage) {
      case ST_NORM1: {
        if (fold && l > 0) break;                 // done by the previous down projection
        const PendingResid pd = l > 0 ? pending_of(e, 1, l - 1, k, B) : PendingResid{};
        norm_rows(e.h, n, n_lo, R, d, e.c.rms_eps, NORM_RMS, mul1, sh1, pd, s);
        break;
      }
      case ST_QKV: {
        EpiQkv<T> eq{q, kl, vl, D, e.nq, e.nkv, e.c.rope, M, e.ldk, plm ? 0 : 1, e.rope_cs, e.desc};
        const GemmArgs ga = with_lo(gargs(w.qkv, n, d, R), n_lo);
        gemm_qkv(fold && l > 0 ? with_rows(ga) : ga, eq, s);
        break;
      }
      case ST_ATTN: {
        at.keys_from_prefix = 1;
        at.n_suffix = plm ? 0 : M;
        at.mask_mode = e.c.state_token ? 1 : 0;
        if (e.f32) attention_f32(at, s); else attention_bf16(at, s);
        break;
      }
      case ST_OPROJ: oproj(EpiResid{e.h, d, nullptr, nullptr}); break;
      case ST_NORM2:
        if (fold) break;                          // done by the output projection
        norm_rows(e.h, n, n_lo, R, d, e.c.rms_eps, NORM_RMS, mul2, sh2, pending_of(e, 0, l, k, B), s);
        break;
      case ST_MLP_UP: {
        const GemmArgs ga = with_lo(gargs(w.gu, n, d, R), n_lo);
        gemm_geglu(fold ? with_rows(ga) : ga, EpiGeglu<T>{g, e.F, g_lo}, s);
        break;
      }
      case ST_MLP_DOWN: {
        const float* next = l + 1 < L ? e.layers[l + 1].attn_norm : nullptr;
        gemm_resid(with_fin(with_split(with_lo(gargs(w.down, g, e.F, R), g_lo), 1), next),
                   EpiResid{e.h, d, nullptr, nullptr}, s);
        break;
      }
    }
    return;
  }
  // DiT block: adaLN-zero modulation from the per-step table
  const float* ada = e.adatab + ((int64_t)k * L + l) * 6 * d;
  const float *sh1 = ada, *sc1 = ada + d, *g1 = ada + 2 * d, *sh2 = ada + 3 * d, *sc2 = ada + 4 * d,
              *g2 = ada + 5 * d;
  const bool cross = (l % 2) == 0;
  switch (stage) {
    case ST_NORM1: {
      const PendingResid pd = l > 0 ? pending_of(e, 1, l - 1, k, B) : PendingResid{};
      norm_rows(e.h, n, n_lo, R, d, e.c.rms_eps, NORM_LN, sc1, sh1, pd, s);
      break;
    }
    case ST_QKV: {
      // cross blocks project only Q here (their K/V come from the features)
      EpiQkv<T> eq{q, kl, vl, D, e.nq, e.nkv, 0, M, e.ldk, 0, e.rope_cs, e.desc};
      gemm_qkv(with_lo(gargs(w.qkv, n, d, R), n_lo), eq, s);
      break;
    }
    case ST_ATTN: {
      at.keys_from_prefix = cross ? 1 : 0;
      at.n_suffix = cross ? 0 : M;
      at.mask_mode = 0;
      if (e.f32) attention_f32(at, s); else attention_bf16(at, s);
      break;
    }
    case ST_OPROJ: oproj(EpiResid{e.h, d, nullptr, g1}); break;
    case ST_NORM2: norm_rows(e.h, n, n_lo, R, d, e.c.rms_eps, NORM_LN, sc2, sh2, pending_of(e, 0, l, k, B), s); break;
    case ST_MLP_UP:
      gemm_store(with_lo(gargs(w.gu, n, d, R), n_lo), store_epi<T>(g, e.F, w.mlp_b1, nullptr, ACT_GELU), s);
      break;
    case ST_MLP_DOWN: gemm_resid(with_split(gargs(w.down, g, e.F, R), 1), EpiResid{e.h, d, w.mlp_b2, g2}, s); break;
  }
}

// Per-call work before the step loop: solver state from the noise, RoPE
// table of the call's positions, state-token embedding, the prefix K/V into
// the key ranges (DiT: the cross-attention K/V projection of the features).
template <typename T>
void enqueue_prologue(phyai_expert& e, int B, hipStream_t s) {
  const int d = e.d, M = e.M, H = e.H, L = e.L;
  const int variant = e.c.variant;
  copy_noise_to_state(e.desc, e.x, (int64_t)B * H * e.A, s);
  if (e.c.rope) rope_table(e.desc, e.inv_freq, e.rope_cs, B, M, e.D, 1, s);
  if (e.c.state_token) embed_state(e.desc, e.state_w, e.state_b, e.e_state, B, e.A, d, s);
  if (variant == PHYAI_VARIANT_DIT) {
    // request-local cross-attention K/V: project the VLM features once per call
    for (int l = 0; l < L; l += 2) {
      GemmArgs ga = gargs(e.layers[l].kv_cross, nullptr, e.c.d_feat, B * e.P);
      ga.A_ind = reinterpret_cast<const void* const*>(&e.desc->prefix);
      ga.a_off = 0;
      ga.rows_per_req = e.P;
      ga.desc = e.desc;
      EpiKV<T> ek{static_cast<T*>(e.kall) + (int64_t)l * e.kv_layer, static_cast<T*>(e.vt) + (int64_t)l * e.kv_layer,
                  e.D, e.nkv, e.P, e.ldk};
      gemm_kv(ga, ek, s);
    }
  } else if (e.P > 0) {
    RelayoutArgs ra{e.desc, e.kall, e.vt, e.kv_layer, e.ldk, L, B, e.P, e.nkv, e.D, M};
    prefix_relayout(ra, static_cast<T*>(nullptr), s);
  }
}

template <typename T>
void enqueue_loop(phyai_expert& e, int B, int K, hipStream_t s) {
  const int d = e.d, M = e.M, H = e.H, L = e.L;
  const int variant = e.c.variant;
  enqueue_prologue<T>(e, B, s);

  // the action-token embedding of step k (state rows of h reset too)
  auto embed_args = [&](int k) {
    EmbedArgs em{};
    em.x = e.x;
    em.in_w = e.in_w;
    em.in_b = e.in_b;
    em.pos = e.pos;
    em.e_state = e.e_state;
    em.h = e.h;
    em.act_is_bf16 = e.f32 ? 0 : 1;
    em.B = B; em.H = H; em.M = M; em.A = e.A; em.d = d; em.off = e.off;
    if (variant == PHYAI_VARIANT_PI0) {
      // z = swish(W1a (W_in x + b_in) + (W1t tau(t_k) + b1)), the embedding
      // folded into W1a (tin_w, tin_b)
      em.in_w = e.tin_w;
      em.in_b = e.tin_b;
      em.rowvec = e.T + (int64_t)k * d;
      em.act = ACT_SWISH;
      em.act_out = e.zbuf;
    }
    return em;
  };
  // the readout of step k also embeds the updated rows for step k + 1 where
  // its kernel can (one launch less per step)
  bool embedded = false;

  for (int k = 0; k < K; ++k) {
    // ---- action tokens -> h
    if (!embedded) embed_actions(embed_args(k), s);
    if (variant == PHYAI_VARIANT_PI0) {
      // u = W2 z + b2, written into the action rows of h
      EpiStore<float> ep = store_epi<float>(e.h, d, e.time_b2, nullptr, ACT_NONE);
      ep.grp = H; ep.grp_stride = M; ep.grp_off = e.off;
      gemm_store(gargs(e.time_w2, e.zbuf, d, B * H), ep, s);
    }

    for (int l = 0; l < L; ++l)
      for (int st = 0; st < kStages; ++st) layer_stage<T>(e, st, l, k, B, s);

    ReadoutArgs ro{};
    ro.h = e.h; ro.B = B; ro.H = H; ro.M = M; ro.off = e.off; ro.d = d; ro.A = e.A;
    ro.eps = e.c.rms_eps;
    ro.out_w = e.out_w; ro.out_b = e.out_b; ro.dt = e.dt + k; ro.x = e.x;
    ro.pend = fold_norms(e, B) ? PendingResid{} : pending_of(e, 1, L - 1, k, B);
    embedded = k + 1 < K && readout_fuses_embedding(e.A, d, B * H, ro.pend.n > 0);
    if (embedded) {
      ro.has_next = 1;
      ro.next = embed_args(k + 1);
    }
    if (variant == PHYAI_VARIANT_PI0) { ro.mode = NORM_RMS; ro.mul = e.final_norm; ro.shift = nullptr; }
    else if (variant == PHYAI_VARIANT_PI05) {
      ro.mode = NORM_RMS;
      ro.mul = e.modtab + ((int64_t)k * (2 * L + 1) + 2 * L) * 2 * d;
      ro.shift = ro.mul + d;
    } else {
      ro.mode = NORM_LN;
      ro.shift = e.fintab + (int64_t)k * 2 * d;
      ro.mul = ro.shift + d;
    }
    readout_euler(ro, s);
  }
  copy_state_to_out(e.desc, e.x, (int64_t)B * H * e.A, s);
}

// Tables that depend only on the schedule (paragraph "Graph replay"):
// sinusoid, dt, pi0 time-MLP input half, pi0.5 adaRMS scale/shift, DiT adaLN.
template <typename T>
void build_tables(phyai_expert& e, const float* ts, int K, hipStream_t s) {
  const int td = e.c.time_dim, d = e.d, L = e.L;
  std::vector<double> tau((size_t)K * td);
  const int half = td / 2;
  for (int k = 0; k < K; ++k)
    for (int i = 0; i < half; ++i) {
      const double frac = (double)i / (half - 1);
      const double period = (double)e.c.sin_min_period * std::pow((double)e.c.sin_max_period / e.c.sin_min_period, frac);
      const double ang = 2.0 * M_PI * (double)ts[k] / period;
      tau[(size_t)k * td + i] = std::sin(ang);
      tau[(size_t)k * td + half + i] = std::cos(ang);
    }
  // the staging buffer is rewritten only once the previous upload from it has
  // run (normally long done, so this does not wait)
  HIPC(hipEventSynchronize(e.stage_ev));
  float* dts = static_cast<float*>(e.stage);
  for (int k = 0; k < K; ++k) dts[k] = ts[k + 1] - ts[k];
  HIPC(hipMemcpyAsync(e.dt, dts, K * 4, hipMemcpyHostToDevice, s));
  void* tst = dts + e.Kmax;
  if (e.f32) {
    float* tf = static_cast<float*>(tst);
    for (size_t i = 0; i < tau.size(); ++i) tf[i] = (float)tau[i];
    HIPC(hipMemcpyAsync(e.tau, tf, tau.size() * 4, hipMemcpyHostToDevice, s));
  } else {
    uint16_t* tb = static_cast<uint16_t*>(tst);
    for (size_t i = 0; i < tau.size(); ++i) tb[i] = f2bf((float)tau[i]);
    HIPC(hipMemcpyAsync(e.tau, tb, tau.size() * 2, hipMemcpyHostToDevice, s));
  }
  HIPC(hipEventRecord(e.stage_ev, s));
  T* tau_d = static_cast<T*>(e.tau);
  if (e.c.variant == PHYAI_VARIANT_PI0) {
    gemm_store(gargs(e.time_w1t, tau_d, td, K), store_epi<float>(e.T, d, e.time_b1, nullptr, ACT_NONE), s);
  } else {
    T* c1 = static_cast<T*>(e.c1);
    T* ca = static_cast<T*>(e.cact);
    gemm_store(gargs(e.cond_w1, tau_d, td, K), store_epi<T>(c1, d, e.cond_b1, nullptr, ACT_SWISH), s);
    // pi0.5: c = swish(...); DiT: the adaLN maps read SiLU(c) -- both are swish of the second layer
    gemm_store(gargs(e.cond_w2, c1, d, K), store_epi<T>(ca, d, e.cond_b2, nullptr, ACT_SWISH), s);
    if (e.c.variant == PHYAI_VARIANT_PI05) {
      const int S = 2 * L + 1;
      for (int l = 0; l < L; ++l) {
        gemm_store(gargs(e.layers[l].attn_mod, ca, d, K),
                   store_epi<float>(e.modtab + (int64_t)(2 * l) * 2 * d, S * 2 * d, e.layers[l].attn_mod_b, nullptr, ACT_NONE), s);
        gemm_store(gargs(e.layers[l].mlp_mod, ca, d, K),
                   store_epi<float>(e.modtab + (int64_t)(2 * l + 1) * 2 * d, S * 2 * d, e.layers[l].mlp_mod_b, nullptr, ACT_NONE), s);
      }
      gemm_store(gargs(e.final_mod, ca, d, K),
                 store_epi<float>(e.modtab + (int64_t)(2 * L) * 2 * d, S * 2 * d, e.final_b, nullptr, ACT_NONE), s);
    } else {
      for (int l = 0; l < L; ++l)
        gemm_store(gargs(e.layers[l].ada, ca, d, K),
                   store_epi<float>(e.adatab + (int64_t)l * 6 * d, L * 6 * d, e.layers[l].ada_b, nullptr, ACT_NONE), s);
      gemm_store(gargs(e.final_mod, ca, d, K), store_epi<float>(e.fintab, 2 * d, e.final_b, nullptr, ACT_NONE), s);
    }
  }
  HIPC(hipGetLastError());
  e.ts_cached.assign(ts, ts + K + 1);
}

// Whether the persistent batch-1 loop takes this handle's shape (pi0, bf16
// weights, one KV head, at most 64 suffix tokens; decided at load).
bool persist_eligible(const phyai_expert& e) {
  const phyai_config& c = e.c;
  const int ntile_max = (e.P + e.M + 63) / 64;       // one attention block per key tile and head
  return c.variant == PHYAI_VARIANT_PI0 && c.weight_dtype == PHYAI_DTYPE_BF16 && e.nkv == 1 &&
         persist_supported(e.d, e.D, e.nq, e.F, e.M, e.A) && e.nq * ntile_max <= 256;
}

// Its buffers and argument block, on the first call that takes it.
void setup_persist(phyai_expert& e, hipStream_t s) {
  const phyai_config& c = e.c;
  const int ntile_max = (e.P + e.M + 63) / 64;
  const int d = e.d, L = e.L, D = e.D;
  PersistArgs& p = e.pargs;
  p = PersistArgs{};
  p.desc = e.desc;
  std::vector<PersistLayer> lt(L);
  for (int l = 0; l < L; ++l)
    lt[l] = PersistLayer{e.layers[l].qkv.w, e.layers[l].o.w, e.layers[l].gu.w, e.layers[l].down.w,
                         e.layers[l].attn_norm, e.layers[l].mlp_norm};
  PersistLayer* ltd = e.mem.alloc_n<PersistLayer>(L);
  HIPC(hipMemcpyAsync(ltd, lt.data(), L * sizeof(PersistLayer), hipMemcpyHostToDevice, s));
  p.layer = ltd;
  p.L = L; p.d = d; p.D = D; p.nq = e.nq; p.F = e.F; p.H = e.H; p.A = e.A; p.M = e.M; p.off = e.off;
  p.ldk = e.ldk;
  p.kv_layer = e.kv_layer;
  p.kall = static_cast<bf16_t*>(e.kall);
  p.vt = static_cast<bf16_t*>(e.vt);
  p.h = e.h;
  // per-step copies for up to R steps per launch, zeroed once (rows past M
  // are read as GEMM rows and never written)
  const size_t R = (size_t)std::min(e.Kmax, kPersistRing);
  auto zeroed = [&](size_t bytes) {
    void* q = e.mem.alloc(bytes);
    HIPC(hipMemsetAsync(q, 0, bytes, s));
    return q;
  };
  const size_t sites = R * (L + 1) * 2;
  p.a = static_cast<bf16_t*>(zeroed(sites * 64 * d * 2));
  p.ss = static_cast<float*>(zeroed(sites * 64 * (d / 32) * 4));
  p.z = static_cast<bf16_t*>(zeroed(R * 64 * d * 2));
  p.q = static_cast<bf16_t*>(zeroed(R * L * 64 * e.nq * D * 2));
  p.o = static_cast<bf16_t*>(zeroed(R * L * 64 * e.nq * D * 2));
  p.g = static_cast<bf16_t*>(zeroed(R * L * 64 * e.F * 2));
  p.apart = static_cast<bf16_t*>(e.mem.alloc((size_t)e.nq * ntile_max * 64 * D * 2));
  p.aml = static_cast<float2*>(e.mem.alloc((size_t)e.nq * ntile_max * 64 * sizeof(float2)));
  p.part = e.mem.alloc_n<float>((size_t)16 * 64 * d);
  p.x = e.x;
  p.e_state = c.state_token ? e.e_state : nullptr;
  p.tin_w = e.tin_w;
  p.tin_b = e.tin_b;
  p.T = e.T;
  p.time_w2 = e.time_w2.w;
  p.time_b2 = e.time_b2;
  p.out_w = e.out_w;
  p.out_b = e.out_b;
  p.final_norm = e.final_norm;
  p.dt = e.dt;
  p.rope_cs = c.rope ? e.rope_cs : nullptr;
  p.eps = c.rms_eps;
  p.scale = 1.0f / std::sqrt((float)D);
  p.ctr = static_cast<unsigned*>(e.mem.alloc(kPersistCounters * 4));
  e.pargs_dev = static_cast<PersistArgs*>(e.mem.alloc(sizeof(PersistArgs)));
  HIPC(hipMemcpyAsync(e.pargs_dev, &p, sizeof(PersistArgs), hipMemcpyHostToDevice, s));
}

// The persistent loop is opt-in (PHYAI_PERSIST=1): on MI355X it measures
// slower than the captured per-kernel graph at the pi0 shape.
bool use_persist() {
  const char* v = std::getenv("PHYAI_PERSIST");
  return v && v[0] == '1';
}

// The whole K-step loop of one request in one cooperative launch (after the
// per-call prologue kernels).
void enqueue_persist(phyai_expert& e, int K, hipStream_t s) {
  enqueue_prologue<bf16_t>(e, 1, s);
  for (int k0 = 0; k0 < K; k0 += kPersistRing) {
    HIPC(hipMemsetAsync(e.pargs.ctr, 0, kPersistCounters * 4, s));
    HIPC(persist_launch(e.pargs, e.pargs_dev, k0, std::min(K, k0 + kPersistRing), K, s));
  }
}

// The prefix LM over B requests: embeddings into the residual stream, the
// RoPE table of positions 0 .., then per layer the norm, the QKV projection
// (+ RoPE, K/V into the key range), the export of the layer's K/V into the
// caller's buffer, and (all but the last layer) attention, the output
// projection, the MLP norm and the MLP.  Eager launches: one pass per call,
// dominated by its GEMMs.
template <typename T>
void enqueue_prefill(phyai_expert& e, const float* embeds, void* kv_out, int B, hipStream_t s) {
  const int L = e.L;
  prefill_embed(e.desc, embeds, e.h, B, e.M, e.d, s);
  if (e.c.rope) rope_table(e.desc, e.inv_freq, e.rope_cs, B, e.M, e.D, 0, s);
  const int64_t half = (int64_t)B * e.M * e.kd;          // one of K, V of one layer, caller layout
  for (int l = 0; l < L; ++l) {
    layer_stage<T>(e, ST_NORM1, l, 0, B, s);
    layer_stage<T>(e, ST_QKV, l, 0, B, s);
    KvExportArgs ka{e.desc, static_cast<T*>(e.kall) + (int64_t)l * e.kv_layer,
                    static_cast<T*>(e.vt) + (int64_t)l * e.kv_layer,
                    static_cast<T*>(kv_out) + (int64_t)l * 2 * half, half, B, e.M, e.nkv, e.D, e.ldk};
    if (e.f32) kv_export_f32(ka, s); else kv_export_bf16(ka, s);
    if (l + 1 == L) break;
    for (int st : {ST_ATTN, ST_OPROJ, ST_NORM2, ST_MLP_UP, ST_MLP_DOWN}) layer_stage<T>(e, st, l, 0, B, s);
  }
}

// The vision tower over B requests (B * n_img images of M = n_patches rows):
// patches into the GEMM operand and position embeddings into the residual
// stream, the patch-embedding GEMM adding x W + b on top, the blocks, the
// final LayerNorm (folding the last block's pending residual), and the
// projector writing each request's tokens at rows 0 .. n_img*M-1 of its
// out_rows-row slab of the caller's buffer.  Eager launches, like the prefill.
template <typename T>
void enqueue_vision(phyai_expert& e, const float* patches, float* tokens_out, int out_rows, int B, hipStream_t s) {
  const int Bi = B * e.n_img, R = Bi * e.M, d = e.d, pd = e.c.patch_dim;
  T* a = static_cast<T*>(e.g);
  if constexpr (std::is_same<T, float>::value)
    vision_embed_f32(patches, a, e.h, e.pos, R, e.M, pd, d, s);
  else
    vision_embed_bf16(patches, a, e.h, e.pos, R, e.M, pd, d, s);
  gemm_resid(gargs(e.patch_lin, a, pd, R), EpiResid{e.h, d, e.patch_b, nullptr}, s);
  for (int l = 0; l < e.L; ++l)
    for (int st = 0; st < kStages; ++st) layer_stage<T>(e, st, l, 0, Bi, s);
  norm_rows(e.h, static_cast<T*>(e.n), static_cast<T*>(nullptr), R, d, e.c.rms_eps, NORM_LN, e.final_norm,
            e.final_norm_b, pending_of(e, 1, e.L - 1, 0, Bi), s);
  EpiStore<float> es = store_epi<float>(tokens_out, e.c.d_out, e.proj_b, nullptr, ACT_NONE);
  es.grp = e.n_img * e.M;
  es.grp_stride = out_rows;
  es.grp_off = 0;
  gemm_store(gargs(e.proj_lin, e.n, d, R), es, s);
}

void check_config(const phyai_config& c) {
  auto req = [](bool ok, const std::string& m) { if (!ok) fail(PHYAI_EINVAL, m); };
  req(c.variant >= 0 && c.variant <= 4, "variant out of range");
  req(c.n_layers >= 1 && c.d_model >= 64 && c.n_q_heads >= 1 && c.n_kv_heads >= 1, "non-positive size");
  req(c.n_q_heads % c.n_kv_heads == 0, "n_q_heads must be a multiple of n_kv_heads");
  req(c.head_dim == 64 || c.head_dim == 128 || c.head_dim == 256, "head_dim must be 64, 128 or 256");
  // the row kernels take whole 256-column groups per thread block
  req(c.d_model % 256 == 0 && c.d_model <= 2048, "d_model must be a multiple of 256, at most 2048");
  req(c.d_mlp >= 64 && c.d_mlp % 64 == 0, "d_mlp must be a positive multiple of 64");
  req(c.max_batch >= 1 && c.max_batch <= kMaxBatch, "max_batch out of range (1..512)");
  req(c.prefix_cap >= 0, "prefix_cap < 0");
  req(c.weight_dtype >= 0 && c.weight_dtype <= 3, "weight_dtype out of range");
  req(c.rms_eps > 0.f, "rms_eps must be positive");
  if (c.variant == PHYAI_VARIANT_VISION) {
    // the patches of every image are the model's rows; no actions, steps,
    // timestep tables or positions beyond the learned embedding
    req(c.n_images >= 1 && c.n_patches >= 1, "a vision tower needs n_images >= 1 and n_patches >= 1");
    req((int64_t)c.max_batch * c.n_images <= kMaxBatch, "max_batch * n_images must be at most 512");
    req(c.patch_dim >= 64 && c.patch_dim % 64 == 0, "patch_dim must be a positive multiple of 64");
    req(c.d_out >= 32 && c.d_out % 32 == 0, "d_out must be a positive multiple of 32");
    req(c.n_q_heads == c.n_kv_heads, "vision attention has one key/value head per query head");
    req(c.rope == 0 && c.state_token == 0 && c.d_feat == 0, "a vision tower has no RoPE, state token or features");
  } else if (c.variant == PHYAI_VARIANT_PREFIX_LM) {
    // the prefix tokens are the model's rows: no actions, steps or timestep
    // tables; keys and values per layer leave in the prefix layout
    req(c.prefix_cap >= 1, "a prefix LM needs prefix_cap >= 1 rows");
    req(c.state_token == 0 && c.d_feat == 0, "a prefix LM has no state token and no feature input");
  } else {
    req(c.horizon >= 1 && c.action_dim >= 1 && c.action_dim <= 64, "horizon >= 1 and 1 <= action_dim <= 64");
    req(c.max_steps >= 1 && c.max_steps <= 1024, "max_steps out of range");
    req(c.time_dim >= 4 && c.time_dim % 64 == 0, "time_dim must be a multiple of 64");
    req(c.sin_min_period > 0.f && c.sin_max_period > 0.f, "sinusoid periods must be positive");
  }
  const bool f32 = c.weight_dtype == PHYAI_DTYPE_F32;
  req(c.kv_dtype == (f32 ? PHYAI_DTYPE_F32 : PHYAI_DTYPE_BF16),
      "kv_dtype must be F32 on the fp32 path and BF16 on the bf16/fp8/fp4 path");
  if (c.variant == PHYAI_VARIANT_DIT) {
    req(c.d_feat >= 64 && c.d_feat % 64 == 0, "DiT needs d_feat, a multiple of 64");
    req(c.n_kv_heads == c.n_q_heads, "DiT attention has one key/value head per query head");
    req(c.prefix_cap >= 1, "DiT needs prefix_cap >= 1 feature rows");
    req(c.rope == 0, "DiT has no RoPE");
  }
  if (c.variant == PHYAI_VARIANT_PI05) req(c.state_token == 0, "pi0.5 has no state token");
  const int64_t qd = (int64_t)c.n_q_heads * c.head_dim;
  req(qd % 64 == 0, "n_q_heads * head_dim must be a multiple of 64");
}

// Layers whose output projection and MLP exist: a prefix LM's last layer
// only projects its keys and values.
int full_layers(const phyai_expert& e) {
  return e.c.variant == PHYAI_VARIANT_PREFIX_LM ? e.L - 1 : e.L;
}

// The prefix LM: the same blocks as the pi0 trunk over M = prefix_cap rows
// per request (the prefix tokens), keys written at positions 0.., no
// timestep tables.  Tensors: layers.l.{attn_norm, wq, wk, wv} for every
// layer, layers.l.{wo, mlp_norm, w_gate, w_up, w_down} for all but the last.
void load_prefix_lm(const phyai_tensor* tensors, int32_t n_tensors, hipStream_t s, phyai_expert* e) {
  const phyai_config& c = e->c;
  e->F = c.d_mlp;
  e->H = 0; e->A = 0; e->off = 0;
  e->M = c.prefix_cap;
  e->P = 0;                 // no prefix of its own: its keys are its rows
  e->qd = e->nq * e->D; e->kd = e->nkv * e->D;
  e->Bmax = c.max_batch; e->Kmax = 0;
  e->Wpre = e->kd;
  const int d = e->d, L = e->L, D = e->D, F = e->F;
  Params P;
  for (int i = 0; i < n_tensors; ++i) {
    if (!tensors[i].name) fail(PHYAI_EINVAL, "tensor with NULL name");
    P.by_name[tensors[i].name] = &tensors[i];
  }
  const int wk_trunk = e->f32                                   ? W_F32
                       : c.weight_dtype == PHYAI_DTYPE_FP8E4M3 ? W_FP8
                       : c.weight_dtype == PHYAI_DTYPE_FP4E2M1 ? W_FP4 : W_BF16;
  auto vec = [&](const std::string& n, int len) { return upload_f32(*e, P.get(n, 1, len), s); };
  e->layers.resize(L);
  for (int l = 0; l < L; ++l) {
    LayerW& w = e->layers[l];
    const std::string p = "layers." + std::to_string(l) + ".";
    w.attn_norm = vec(p + "attn_norm", d);
    w.qkv = pack_heads(*e, {P.get(p + "wq", d, e->qd), P.get(p + "wk", d, e->kd), P.get(p + "wv", d, e->kd)}, D,
                       wk_trunk, s);
    if (l + 1 == L) break;
    w.o = pack_identity(*e, {P.get(p + "wo", e->qd, d)}, wk_trunk, s);
    w.mlp_norm = vec(p + "mlp_norm", d);
    w.gu = pack_geglu(*e, P.get(p + "w_gate", d, F), P.get(p + "w_up", d, F), wk_trunk, s);
    w.down = pack_identity(*e, {P.get(p + "w_down", F, d)}, wk_trunk, s);
  }
  {
    std::vector<float> inv(D / 2);
    for (int i = 0; i < D / 2; ++i) inv[i] = (float)std::pow((double)c.rope_base, -2.0 * i / D);
    e->inv_freq = e->mem.alloc_n<float>(D / 2);
    HIPC(hipMemcpyAsync(e->inv_freq, inv.data(), inv.size() * 4, hipMemcpyHostToDevice, s));
    if (c.rope) e->rope_cs = static_cast<float2*>(e->mem.alloc((size_t)c.max_batch * e->M * (D / 2) * sizeof(float2)));
  }
  const int64_t Bm = e->Bmax, M = e->M, ab = e->act_bytes;
  e->h = e->mem.alloc_n<float>(Bm * M * d);
  e->n = e->mem.alloc(Bm * M * d * ab);
  e->q = e->mem.alloc(Bm * M * e->qd * ab);
  e->o = e->mem.alloc(Bm * M * e->qd * ab);
  e->g = e->mem.alloc(Bm * M * F * ab);
  // key ranges: keys 0 .. M-1 written by the QKV epilogue, the tail to the
  // next multiple of 64 stays zero (attention reads whole tiles)
  e->ldk = (M + 63) / 64 * 64;
  e->kv_layer = Bm * e->nkv * (int64_t)e->ldk * D;
  e->kall = e->mem.alloc(L * e->kv_layer * ab);
  e->vt = e->mem.alloc(L * e->kv_layer * ab);
  HIPC(hipMemsetAsync(e->kall, 0, L * e->kv_layer * ab, s));
  HIPC(hipMemsetAsync(e->vt, 0, L * e->kv_layer * ab, s));
  int64_t part = 0, pend = 4;
  if (!e->f32)
    for (int B = 1; B <= e->Bmax; ++B) {
      const int rows = e->M * (e->nq / e->nkv);
      part = std::max(part, attention_partial_floats(B, e->M, e->nq, e->nkv, D, attn_splits_max(B, rows, e->nkv, e->M)));
      const int R = B * e->M;
      for (int l = 0; l < full_layers(*e); ++l)
        for (int which = 0; which < 2; ++which) {
          const Lin& w = which == 0 ? e->layers[l].o : e->layers[l].down;
          const int sk = std::max(resid_split(*e, which, l, B), gemm_split_k(R, w.NPT, w.K));
          if (sk > 1) pend = std::max(pend, (int64_t)sk * R * d);
        }
    }
  e->part = e->mem.alloc_n<float>(part > 0 ? part : 4);
  e->pend = e->mem.alloc_n<float>(pend);
  e->part_cur = e->part;
  e->pend_cur = e->pend;
  e->desc = static_cast<CallDesc*>(e->mem.alloc(sizeof(CallDesc)));
  HIPC(hipStreamSynchronize(s));
}

// The vision tower: M = n_patches rows per image, B * n_images images per
// call; the key range of one block (reused by every block), no timestep
// tables.  Tensors as listed in the header.
void load_vision(const phyai_tensor* tensors, int32_t n_tensors, hipStream_t s, phyai_expert* e) {
  const phyai_config& c = e->c;
  e->F = c.d_mlp;
  e->H = 0; e->A = 0; e->off = 0;
  e->M = c.n_patches;
  e->n_img = c.n_images;
  e->P = 0;
  e->qd = e->nq * e->D; e->kd = e->nkv * e->D;
  e->Bmax = c.max_batch * c.n_images;    // image batch
  e->Kmax = 0;
  e->Wpre = e->kd;
  const int d = e->d, L = e->L, D = e->D, F = e->F;
  Params P;
  for (int i = 0; i < n_tensors; ++i) {
    if (!tensors[i].name) fail(PHYAI_EINVAL, "tensor with NULL name");
    P.by_name[tensors[i].name] = &tensors[i];
  }
  const int wk_plain = e->f32 ? W_F32 : W_BF16;
  const int wk_trunk = e->f32                                   ? W_F32
                       : c.weight_dtype == PHYAI_DTYPE_FP8E4M3 ? W_FP8
                       : c.weight_dtype == PHYAI_DTYPE_FP4E2M1 ? W_FP4 : W_BF16;
  auto vec = [&](const std::string& n, int len) { return upload_f32(*e, P.get(n, 1, len), s); };
  e->patch_lin = pack_identity(*e, {P.get("patch_w", c.patch_dim, d)}, wk_plain, s);
  e->patch_b = vec("patch_b", d);
  e->pos = upload_f32(*e, P.get("pos_emb", c.n_patches, d), s);
  e->layers.resize(L);
  for (int l = 0; l < L; ++l) {
    LayerW& w = e->layers[l];
    const std::string p = "layers." + std::to_string(l) + ".";
    w.attn_norm = vec(p + "ln1_w", d);
    w.attn_norm_b = vec(p + "ln1_b", d);
    w.qkv = pack_heads(*e, {P.get(p + "wq", d, e->qd), P.get(p + "wk", d, e->kd), P.get(p + "wv", d, e->kd)}, D,
                       wk_trunk, s);
    w.qkv_b = upload_concat_f32(*e, {P.get(p + "bq", 1, e->qd), P.get(p + "bk", 1, e->kd), P.get(p + "bv", 1, e->kd)},
                                s);
    w.o = pack_identity(*e, {P.get(p + "wo", e->qd, d)}, wk_trunk, s);
    w.o_b = vec(p + "bo", d);
    w.mlp_norm = vec(p + "ln2_w", d);
    w.mlp_norm_b = vec(p + "ln2_b", d);
    w.gu = pack_identity(*e, {P.get(p + "mlp_w1", d, F)}, wk_trunk, s);
    w.mlp_b1 = vec(p + "mlp_b1", F);
    w.down = pack_identity(*e, {P.get(p + "mlp_w2", F, d)}, wk_trunk, s);
    w.mlp_b2 = vec(p + "mlp_b2", d);
  }
  e->final_norm = vec("post_ln_w", d);
  e->final_norm_b = vec("post_ln_b", d);
  e->proj_lin = pack_identity(*e, {P.get("proj_w", d, c.d_out)}, wk_plain, s);
  e->proj_b = vec("proj_b", c.d_out);
  const int64_t Bm = e->Bmax, M = e->M, ab = e->act_bytes;
  e->h = e->mem.alloc_n<float>(Bm * M * d);
  e->n = e->mem.alloc(Bm * M * d * ab);
  e->q = e->mem.alloc(Bm * M * e->qd * ab);
  e->o = e->mem.alloc(Bm * M * e->qd * ab);
  // the MLP activations, and before the blocks the patch-embedding operand
  e->g = e->mem.alloc(Bm * M * std::max(F, c.patch_dim) * ab);
  // one key range: keys 0 .. M-1 written by the QKV epilogue, the tail to
  // the next multiple of 64 stays zero (attention reads whole tiles)
  e->ldk = (M + 63) / 64 * 64;
  e->kv_layer = Bm * e->nkv * (int64_t)e->ldk * D;
  e->kall = e->mem.alloc(e->kv_layer * ab);
  e->vt = e->mem.alloc(e->kv_layer * ab);
  HIPC(hipMemsetAsync(e->kall, 0, e->kv_layer * ab, s));
  HIPC(hipMemsetAsync(e->vt, 0, e->kv_layer * ab, s));
  int64_t part = 0, pend = 4;
  if (!e->f32)
    for (int B = 1; B <= e->Bmax; ++B) {
      const int rows = e->M * (e->nq / e->nkv);
      part = std::max(part, attention_partial_floats(B, e->M, e->nq, e->nkv, D, attn_splits_max(B, rows, e->nkv, e->M)));
      const int R = B * e->M;
      for (int l = 0; l < L; ++l)
        for (int which = 0; which < 2; ++which) {
          const Lin& w = which == 0 ? e->layers[l].o : e->layers[l].down;
          const int sk = std::max(resid_split(*e, which, l, B), gemm_split_k(R, w.NPT, w.K));
          if (sk > 1) pend = std::max(pend, (int64_t)sk * R * d);
        }
    }
  e->part = e->mem.alloc_n<float>(part > 0 ? part : 4);
  e->pend = e->mem.alloc_n<float>(pend);
  e->part_cur = e->part;
  e->pend_cur = e->pend;
  e->desc = static_cast<CallDesc*>(e->mem.alloc(sizeof(CallDesc)));
  HIPC(hipStreamSynchronize(s));
}

void load_impl(const phyai_config* cfg, const phyai_tensor* tensors, int32_t n_tensors, hipStream_t s,
               phyai_expert* e) {
  const phyai_config& c = *cfg;
  check_config(c);
  e->c = c;
  e->f32 = c.weight_dtype == PHYAI_DTYPE_F32;
  e->act_bytes = e->f32 ? 4 : 2;
  e->L = c.n_layers; e->d = c.d_model; e->D = c.head_dim; e->nq = c.n_q_heads; e->nkv = c.n_kv_heads;
  if (c.variant == PHYAI_VARIANT_PREFIX_LM) {
    load_prefix_lm(tensors, n_tensors, s, e);
    return;
  }
  if (c.variant == PHYAI_VARIANT_VISION) {
    load_vision(tensors, n_tensors, s, e);
    return;
  }
  e->H = c.horizon; e->A = c.action_dim; e->F = c.d_mlp;
  e->off = c.state_token ? 1 : 0;
  e->M = e->H + e->off;
  e->qd = e->nq * e->D; e->kd = e->nkv * e->D;
  e->Bmax = c.max_batch; e->Kmax = c.max_steps; e->P = c.prefix_cap;
  e->Wpre = c.variant == PHYAI_VARIANT_DIT ? c.d_feat : e->kd;
  const int d = e->d, L = e->L, D = e->D, F = e->F, A = e->A;

  Params P;
  for (int i = 0; i < n_tensors; ++i) {
    if (!tensors[i].name) fail(PHYAI_EINVAL, "tensor with NULL name");
    P.by_name[tensors[i].name] = &tensors[i];
  }
  const int wk_small = e->f32 ? W_F32 : W_BF16;
  const int wk_trunk = e->f32                                   ? W_F32
                       : c.weight_dtype == PHYAI_DTYPE_FP8E4M3 ? W_FP8
                       : c.weight_dtype == PHYAI_DTYPE_FP4E2M1 ? W_FP4 : W_BF16;
  auto vec = [&](const std::string& n, int len) { return upload_f32(*e, P.get(n, 1, len), s); };

  e->in_w = upload_f32(*e, P.get("in_w", A, d), s);
  e->in_b = vec("in_b", d);
  {
    // W_out is kept transposed, [A][d], so the readout streams rows along d
    const phyai_tensor* t = P.get("out_w", d, A);
    std::vector<float> wt((size_t)A * d);
    for (int k = 0; k < d; ++k)
      for (int a = 0; a < A; ++a) wt[(size_t)a * d + k] = elem_f32(t, (int64_t)k * A + a);
    e->out_w = e->mem.alloc_n<float>(wt.size());
    HIPC(hipMemcpyAsync(e->out_w, wt.data(), wt.size() * 4, hipMemcpyHostToDevice, s));
    HIPC(hipStreamSynchronize(s));
  }
  e->out_b = vec("out_b", A);
  if (c.state_token) {
    e->state_w = upload_f32(*e, P.get("state_w", A, d), s);
    e->state_b = vec("state_b", d);
  }
  if (c.variant == PHYAI_VARIANT_PI0) {
    const phyai_tensor* w1 = P.get("time_w1", d + c.time_dim, d);
    // split W1 into the rows acting on the action embedding and on tau(t)
    phyai_tensor ta = *w1, tt = *w1;
    const size_t esz = w1->dtype == PHYAI_DTYPE_F32 ? 4 : 2;
    ta.rows = d;
    tt.rows = c.time_dim;
    tt.data = static_cast<const char*>(w1->data) + (size_t)d * d * esz;
    {
      // tin_w = W_in W1a and tin_b = b_in W1a, in fp64 from the weights as
      // given, kept in fp32: the time MLP's first layer then reads x directly
      const phyai_tensor* wi = P.get("in_w", A, d);
      const phyai_tensor* bi = P.get("in_b", 1, d);
      std::vector<double> w1a((size_t)d * d), acc((size_t)(A + 1) * d, 0.0);
      for (int64_t i = 0; i < (int64_t)d * d; ++i) w1a[i] = elem_f32(&ta, i);
      for (int a = 0; a <= A; ++a) {
        double* row = &acc[(size_t)a * d];
        for (int k = 0; k < d; ++k) {
          const double xk = a < A ? elem_f32(wi, (int64_t)a * d + k) : elem_f32(bi, k);
          const double* wr = &w1a[(size_t)k * d];
          for (int c2 = 0; c2 < d; ++c2) row[c2] += xk * wr[c2];
        }
      }
      std::vector<float> f(acc.begin(), acc.end());
      e->tin_w = e->mem.alloc_n<float>((int64_t)A * d);
      e->tin_b = e->mem.alloc_n<float>(d);
      HIPC(hipMemcpyAsync(e->tin_w, f.data(), (size_t)A * d * 4, hipMemcpyHostToDevice, s));
      HIPC(hipMemcpyAsync(e->tin_b, f.data() + (size_t)A * d, (size_t)d * 4, hipMemcpyHostToDevice, s));
      HIPC(hipStreamSynchronize(s));
    }
    e->time_w1t = pack_identity(*e, {&tt}, wk_small, s);
    e->time_b1 = vec("time_b1", d);
    e->time_w2 = pack_identity(*e, {P.get("time_w2", d, d)}, wk_small, s);
    e->time_b2 = vec("time_b2", d);
    e->final_norm = vec("final_norm", d);
  } else {
    e->cond_w1 = pack_identity(*e, {P.get("cond_w1", c.time_dim, d)}, wk_small, s);
    e->cond_b1 = vec("cond_b1", d);
    e->cond_w2 = pack_identity(*e, {P.get("cond_w2", d, d)}, wk_small, s);
    e->cond_b2 = vec("cond_b2", d);
    if (c.variant == PHYAI_VARIANT_PI05) {
      e->final_mod = pack_identity(*e, {P.get("final_mod_w", d, 2 * d)}, wk_small, s);
      e->final_b = vec("final_mod_b", 2 * d);
    } else {
      e->final_mod = pack_identity(*e, {P.get("final_ada_w", d, 2 * d)}, wk_small, s);
      e->final_b = vec("final_ada_b", 2 * d);
      e->pos = upload_f32(*e, P.get("pos_emb", e->H, d), s);
    }
  }
  e->layers.resize(L);
  for (int l = 0; l < L; ++l) {
    LayerW& w = e->layers[l];
    const std::string p = "layers." + std::to_string(l) + ".";
    const bool cross = c.variant == PHYAI_VARIANT_DIT && (l % 2 == 0);
    const int kin = cross ? c.d_feat : d;
    const phyai_tensor* wq = P.get(p + "wq", d, e->qd);
    const phyai_tensor* wkt = P.get(p + "wk", kin, e->kd);
    const phyai_tensor* wvt = P.get(p + "wv", kin, e->kd);
    if (cross) {
      w.qkv = pack_heads(*e, {wq}, D, wk_trunk, s);
      w.kv_cross = pack_identity(*e, {wkt, wvt}, wk_trunk, s);
    } else {
      w.qkv = pack_heads(*e, {wq, wkt, wvt}, D, wk_trunk, s);
    }
    w.o = pack_identity(*e, {P.get(p + "wo", e->qd, d)}, wk_trunk, s);
    if (c.variant == PHYAI_VARIANT_DIT) {
      w.ada = pack_identity(*e, {P.get(p + "ada_w", d, 6 * d)}, wk_small, s);
      w.ada_b = vec(p + "ada_b", 6 * d);
      w.gu = pack_identity(*e, {P.get(p + "mlp_w1", d, F)}, wk_trunk, s);
      w.mlp_b1 = vec(p + "mlp_b1", F);
      w.down = pack_identity(*e, {P.get(p + "mlp_w2", F, d)}, wk_trunk, s);
      w.mlp_b2 = vec(p + "mlp_b2", d);
    } else {
      w.gu = pack_geglu(*e, P.get(p + "w_gate", d, F), P.get(p + "w_up", d, F), wk_trunk, s);
      w.down = pack_identity(*e, {P.get(p + "w_down", F, d)}, wk_trunk, s);
      if (c.variant == PHYAI_VARIANT_PI0) {
        w.attn_norm = vec(p + "attn_norm", d);
        w.mlp_norm = vec(p + "mlp_norm", d);
      } else {
        w.attn_mod = pack_identity(*e, {P.get(p + "attn_mod_w", d, 2 * d)}, wk_small, s);
        w.attn_mod_b = vec(p + "attn_mod_b", 2 * d);
        w.mlp_mod = pack_identity(*e, {P.get(p + "mlp_mod_w", d, 2 * d)}, wk_small, s);
        w.mlp_mod_b = vec(p + "mlp_mod_b", 2 * d);
      }
    }
  }
  // RoPE inverse frequencies
  {
    std::vector<float> inv(D / 2);
    for (int i = 0; i < D / 2; ++i) inv[i] = (float)std::pow((double)c.rope_base, -2.0 * i / D);
    e->inv_freq = e->mem.alloc_n<float>(D / 2);
    HIPC(hipMemcpyAsync(e->inv_freq, inv.data(), inv.size() * 4, hipMemcpyHostToDevice, s));
    if (c.rope) e->rope_cs = static_cast<float2*>(e->mem.alloc((size_t)c.max_batch * e->M * (D / 2) * sizeof(float2)));
  }
  // working buffers sized for max_batch
  const int64_t Bm = e->Bmax, M = e->M, ab = e->act_bytes;
  e->x = e->mem.alloc_n<float>(Bm * e->H * A);
  e->h = e->mem.alloc_n<float>(Bm * M * d);
  e->e_state = e->mem.alloc_n<float>(Bm * d);
  e->n = e->mem.alloc(Bm * M * d * ab);
  e->zbuf = e->mem.alloc(Bm * e->H * d * ab);
  e->q = e->mem.alloc(Bm * M * e->qd * ab);
  e->o = e->mem.alloc(Bm * M * e->qd * ab);
  {
    const int keys = c.variant == PHYAI_VARIANT_DIT ? std::max(e->P, e->M) : e->P + e->M;
    e->ldk = (keys + 63) / 64 * 64;
    e->kv_layer = Bm * e->nkv * (int64_t)e->ldk * D;
    e->kall = e->mem.alloc(L * e->kv_layer * ab);
    e->vt = e->mem.alloc(L * e->kv_layer * ab);
    HIPC(hipMemsetAsync(e->kall, 0, L * e->kv_layer * ab, s));
    HIPC(hipMemsetAsync(e->vt, 0, L * e->kv_layer * ab, s));
  }
  e->g = e->mem.alloc(Bm * M * F * ab);
  if (c.variant == PHYAI_VARIANT_PI0 && !e->f32) {
    e->ss = e->mem.alloc_n<float>(Bm * M * (d / 32));
    e->fin_ctr = static_cast<unsigned*>(e->mem.alloc(kFinCounters * sizeof(unsigned)));
    HIPC(hipMemsetAsync(e->fin_ctr, 0, kFinCounters * sizeof(unsigned), s));
  }
  // pi0.5's adaRMS path amplifies the bf16 rounding of the normalised
  // activations and of the GeGLU output; those GEMM operands carry a second
  // bf16 term there (weights are still read once).
  e->split_act = !e->f32 && c.variant == PHYAI_VARIANT_PI05;
  if (e->split_act) {
    e->n_lo = e->mem.alloc(Bm * M * d * ab);
    e->g_lo = e->mem.alloc(Bm * M * F * ab);
  }
  int64_t part = 0;
  if (!e->f32) {
    const int keys_main = c.variant == PHYAI_VARIANT_DIT ? e->M : e->P + e->M;
    for (int B = 1; B <= e->Bmax; ++B) {
      const int rows = e->M * (e->nq / e->nkv);
      const int s1 = attn_splits_max(B, rows, e->nkv, keys_main);
      const int s2 = attn_splits_max(B, rows, e->nkv, e->P);
      int64_t need = attention_partial_floats(B, e->M, e->nq, e->nkv, D, s1);
      if (c.variant == PHYAI_VARIANT_DIT)
        need = std::max(need, attention_partial_floats(B, e->M, e->nq, e->nkv, D, s2));
      part = std::max(part, need);
    }
  }
  e->part = e->mem.alloc_n<float>(part > 0 ? part : 4);
  {
    int64_t pend = 4;
    if (!e->f32)
      for (int B = 1; B <= e->Bmax; ++B) {
        const int R = B * e->M;
        for (int l = 0; l < L; ++l)
          for (int which = 0; which < 2; ++which) {
            // either O-projection form (the merge one may be switched off per call)
            const Lin& w = which == 0 ? e->layers[l].o : e->layers[l].down;
            const int sk = std::max(resid_split(*e, which, l, B), gemm_split_k(R, w.NPT, w.K));
            if (sk > 1) pend = std::max(pend, (int64_t)sk * R * d);
          }
      }
    e->pend = e->mem.alloc_n<float>(pend);
  }
  e->part_cur = e->part;
  e->pend_cur = e->pend;
  e->static_scratch = static_scratch_ptr();
  HIPC(hipStreamSynchronize(s));
  e->desc = static_cast<CallDesc*>(e->mem.alloc(sizeof(CallDesc)));
  // tables
  const int64_t Km = e->Kmax;
  e->tau = e->mem.alloc(Km * c.time_dim * ab);
  e->c1 = e->mem.alloc(Km * d * ab);
  e->cact = e->mem.alloc(Km * d * ab);
  e->dt = e->mem.alloc_n<float>(Km);
  if (c.variant == PHYAI_VARIANT_PI0) e->T = e->mem.alloc_n<float>(Km * d);
  if (c.variant == PHYAI_VARIANT_PI05) e->modtab = e->mem.alloc_n<float>(Km * (2 * L + 1) * 2 * d);
  if (c.variant == PHYAI_VARIANT_DIT) {
    e->adatab = e->mem.alloc_n<float>(Km * L * 6 * d);
    e->fintab = e->mem.alloc_n<float>(Km * 2 * d);
  }
  HIPC(hipStreamCreateWithFlags(&e->cap, hipStreamNonBlocking));
  HIPC(hipHostMalloc(&e->stage, (size_t)Km * 4 + (size_t)Km * c.time_dim * ab, hipHostMallocDefault));
  HIPC(hipEventCreateWithFlags(&e->stage_ev, hipEventDisableTiming));
  std::vector<float> ts(e->Kmax + 1);
  for (int k = 0; k <= e->Kmax; ++k) ts[k] = (float)(1.0 - (double)k / e->Kmax);
  if (e->f32) build_tables<float>(*e, ts.data(), e->Kmax, s);
  else build_tables<bf16_t>(*e, ts.data(), e->Kmax, s);
  e->persist_ok = persist_eligible(*e);
  HIPC(hipStreamSynchronize(s));
}

Bucket& get_bucket(phyai_expert& e, int B, int K) {
  auto key = std::make_pair(B, K);
  auto it = e.buckets.find(key);
  if (it != e.buckets.end()) return it->second;
  Bucket bk;
  HIPC(hipStreamBeginCapture(e.cap, hipStreamCaptureModeThreadLocal));
  try {
    if (e.f32) enqueue_loop<float>(e, B, K, e.cap);
    else enqueue_loop<bf16_t>(e, B, K, e.cap);
  } catch (...) {
    hipGraph_t junk = nullptr;
    (void)hipStreamEndCapture(e.cap, &junk);
    if (junk) (void)hipGraphDestroy(junk);
    throw;
  }
  HIPC(hipStreamEndCapture(e.cap, &bk.graph));
  hipError_t ie = hipGraphInstantiate(&bk.exec, bk.graph, nullptr, nullptr, 0);
  if (ie != hipSuccess) {
    (void)hipGraphDestroy(bk.graph);
    fail(PHYAI_EHIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(ie));
  }
  return e.buckets.emplace(key, bk).first->second;
}

bool use_graphs() {
  const char* v = std::getenv("PHYAI_NO_GRAPH");
  return !(v && v[0] == '1');
}

}  // namespace

namespace {

// Host validation shared by the denoising entry points (nothing enqueued yet).
void check_call(phyai_expert* e, const void* prefix, const int32_t* prefix_len, const float* noise,
                const float* timesteps, int n_steps, int batch, const float* state, const float* out_actions) {
  if (!e) fail(PHYAI_EINVAL, "NULL handle");
  if (e->c.variant == PHYAI_VARIANT_PREFIX_LM) fail(PHYAI_EINVAL, "a prefix-LM handle: call phyai_prefill");
  if (e->c.variant == PHYAI_VARIANT_VISION) fail(PHYAI_EINVAL, "a vision handle: call phyai_encode_images");
  if (batch < 1 || batch > e->Bmax) fail(PHYAI_EINVAL, "batch out of range 1..max_batch");
  if (n_steps < 1 || n_steps > e->Kmax) fail(PHYAI_EINVAL, "n_steps out of range 1..max_steps");
  if (!prefix_len || !noise || !timesteps || !out_actions) fail(PHYAI_EINVAL, "NULL argument");
  if (!prefix && e->P > 0) fail(PHYAI_EINVAL, "NULL prefix");
  if (e->c.state_token && !state) fail(PHYAI_EINVAL, "state is required when state_token = 1");
  for (int b = 0; b < batch; ++b) {
    if (prefix_len[b] < 0 || prefix_len[b] > e->P)
      fail(PHYAI_EINVAL, "prefix_len[" + std::to_string(b) + "] = " + std::to_string(prefix_len[b]) +
                             " outside 0..prefix_cap");
    if (e->c.variant == PHYAI_VARIANT_DIT && prefix_len[b] < 1)
      fail(PHYAI_EINVAL, "DiT requests need at least one feature row");
  }
  for (int k = 0; k <= n_steps; ++k)
    if (!std::isfinite(timesteps[k])) fail(PHYAI_EINVAL, "non-finite timestep");
  // the kernels move these buffers in 16-byte accesses
  auto aligned16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  if (!aligned16(prefix) || !aligned16(noise) || !aligned16(out_actions) || (e->c.state_token && !aligned16(state)))
    fail(PHYAI_EINVAL, "prefix, noise, state and out_actions must be 16-byte aligned");
}

// Rebuild the schedule-keyed tables when the timesteps differ from the last call's.
void refresh_tables(phyai_expert& e, const float* timesteps, int n_steps, hipStream_t s) {
  const bool same = (int)e.ts_cached.size() >= n_steps + 1 &&
                    std::memcmp(e.ts_cached.data(), timesteps, (n_steps + 1) * 4) == 0;
  if (same) return;
  if (e.f32) build_tables<float>(e, timesteps, n_steps, s);
  else build_tables<bf16_t>(e, timesteps, n_steps, s);
}

void write_call_desc(phyai_expert& e, const void* prefix, const int32_t* prefix_len, const float* noise, int batch,
                     const float* state, float* out_actions, hipStream_t s) {
  CallDesc hd;
  std::memset(&hd, 0, sizeof(hd));
  hd.prefix = prefix;
  hd.noise = noise;
  hd.state = state;
  hd.out = out_actions;
  for (int b = 0; b < batch; ++b) hd.prefix_len[b] = prefix_len[b];
  set_call_desc(hd, e.desc, s);
  HIPC(hipGetLastError());
  e.last_batch = batch;
}

int64_t round_up64(int64_t n) { return (n + 63) / 64 * 64; }

// Attention key-split partial floats one call at batch B uses (the larger of
// the two block heights, as the handle's own buffer is sized).
int64_t attn_part_floats(const phyai_expert& e, int B) {
  if (e.f32) return 0;
  const int rows = e.M * (e.nq / e.nkv);
  const int keys_main = e.c.variant == PHYAI_VARIANT_DIT ? e.M : e.P + e.M;
  int64_t need = attention_partial_floats(B, e.M, e.nq, e.nkv, e.D, attn_splits_max(B, rows, e.nkv, keys_main));
  if (e.c.variant == PHYAI_VARIANT_DIT)
    need = std::max(need, attention_partial_floats(B, e.M, e.nq, e.nkv, e.D, attn_splits_max(B, rows, e.nkv, e.P)));
  return need;
}

// Split-K partial floats of the residual GEMMs at batch B (either O-projection form).
int64_t pend_floats(const phyai_expert& e, int B) {
  if (e.f32) return 0;
  const int R = B * e.M;
  int64_t need = 0;
  for (int l = 0; l < full_layers(e); ++l)
    for (int which = 0; which < 2; ++which) {
      const Lin& w = which == 0 ? e.layers[l].o : e.layers[l].down;
      const int sk = std::max(resid_split(e, which, l, B), gemm_split_k(R, w.NPT, w.K));
      if (sk > 1) need = std::max(need, (int64_t)sk * R * e.d);
    }
  return need;
}

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
namespace {
int run_guarded(const std::function<void()>& f) {
  try {
    f();
    g_err.clear();
    return PHYAI_OK;
  } catch (const Fail& x) {
    g_err = x.msg;
    return x.code;
  } catch (const std::bad_alloc&) {
    g_err = "host allocation failed";
    return PHYAI_ENOMEM;
  } catch (const std::exception& x) {
    g_err = x.what();
    return PHYAI_EINVAL;
  }
}
}  // namespace

extern "C" {

int phyai_version(void) { return 100; }

const char* phyai_last_error(void) { return g_err.c_str(); }

int phyai_load_expert(const phyai_config* cfg, const phyai_tensor* tensors, int32_t n_tensors, void* stream,
                      phyai_expert** out) {
  if (out) *out = nullptr;
  return run_guarded([&] {
    if (!cfg || !out) fail(PHYAI_EINVAL, "cfg and out must not be NULL");
    if (n_tensors < 0 || (n_tensors > 0 && !tensors)) fail(PHYAI_EINVAL, "bad tensor list");
    phyai_expert* e = new phyai_expert();
    try {
      load_impl(cfg, tensors, n_tensors, static_cast<hipStream_t>(stream), e);
    } catch (...) {
      delete e;
      throw;
    }
    *out = e;
  });
}

int phyai_prepare(phyai_expert* e, int32_t batch, int32_t n_steps, void* stream) {
  (void)stream;
  return run_guarded([&] {
    if (!e) fail(PHYAI_EINVAL, "NULL handle");
    if (e->c.variant == PHYAI_VARIANT_PREFIX_LM) fail(PHYAI_EINVAL, "a prefix-LM handle has no denoising loop");
    if (e->c.variant == PHYAI_VARIANT_VISION) fail(PHYAI_EINVAL, "a vision handle has no denoising loop");
    if (batch < 1 || batch > e->Bmax) fail(PHYAI_EINVAL, "batch out of range");
    if (n_steps < 1 || n_steps > e->Kmax) fail(PHYAI_EINVAL, "n_steps out of range");
    if (use_graphs()) get_bucket(*e, batch, n_steps);
  });
}

int phyai_denoise(phyai_expert* e, const void* prefix, const int32_t* prefix_len, const float* noise,
                  const float* timesteps, int32_t n_steps, int32_t batch, const float* state, float* out_actions,
                  void* stream) {
  return run_guarded([&] {
    check_call(e, prefix, prefix_len, noise, timesteps, n_steps, batch, state, out_actions);
    hipStream_t s = static_cast<hipStream_t>(stream);
    refresh_tables(*e, timesteps, n_steps, s);
    if (e->persist_ok && batch == 1 && use_persist()) {
      if (!e->persist_ready) {
        setup_persist(*e, s);
        HIPC(hipStreamSynchronize(s));
        e->persist_ready = true;
      }
      write_call_desc(*e, prefix, prefix_len, noise, batch, state, out_actions, s);
      enqueue_persist(*e, n_steps, s);
      return;
    }
    Bucket* bk = use_graphs() ? &get_bucket(*e, batch, n_steps) : nullptr;
    write_call_desc(*e, prefix, prefix_len, noise, batch, state, out_actions, s);
    if (bk) {
      HIPC(hipGraphLaunch(bk->exec, s));
    } else {
      if (e->f32) enqueue_loop<float>(*e, batch, n_steps, s);
      else enqueue_loop<bf16_t>(*e, batch, n_steps, s);
      HIPC(hipGetLastError());
    }
  });
}

int phyai_denoise_static(phyai_expert* e, const void* prefix, const int32_t* prefix_len, const float* noise,
                         const float* timesteps, int32_t n_steps, int32_t batch, const float* state,
                         float* out_actions, void* stream) {
  return run_guarded([&] {
    check_call(e, prefix, prefix_len, noise, timesteps, n_steps, batch, state, out_actions);
    const int64_t part = round_up64(attn_part_floats(*e, batch));
    const int64_t need = part + pend_floats(*e, batch);
    if (need > kStaticScratchFloats)
      fail(PHYAI_EINVAL, "this batch needs " + std::to_string(need * 4) + " bytes of scratch; the static limit is " +
                             std::to_string(kStaticScratchFloats * 4));
    hipStream_t s = static_cast<hipStream_t>(stream);
    refresh_tables(*e, timesteps, n_steps, s);
    write_call_desc(*e, prefix, prefix_len, noise, batch, state, out_actions, s);
    // eager launches (no graph: instantiating one allocates), partials in the
    // device's static scratch; the handle's own buffers are restored after
    e->part_cur = e->static_scratch;
    e->pend_cur = e->static_scratch + part;
    try {
      if (e->f32) enqueue_loop<float>(*e, batch, n_steps, s);
      else enqueue_loop<bf16_t>(*e, batch, n_steps, s);
    } catch (...) {
      e->part_cur = e->part;
      e->pend_cur = e->pend;
      throw;
    }
    e->part_cur = e->part;
    e->pend_cur = e->pend;
    HIPC(hipGetLastError());
  });
}

int phyai_debug_hidden(phyai_expert* e, float* dst, int32_t batch, void* stream) {
  return run_guarded([&] {
    if (!e || !dst) fail(PHYAI_EINVAL, "NULL argument");
    if (batch < 1 || batch > e->Bmax) fail(PHYAI_EINVAL, "batch out of range");
    HIPC(hipMemcpyAsync(dst, e->h, (size_t)batch * e->M * e->d * 4, hipMemcpyDeviceToDevice,
                        static_cast<hipStream_t>(stream)));
  });
}

int phyai_fp8_to_bf16(const uint8_t* codes, uint16_t* out, int64_t n, void* stream) {
  return run_guarded([&] {
    if (n < 0) fail(PHYAI_EINVAL, "n < 0");
    if (n == 0) return;
    if (!codes || !out) fail(PHYAI_EINVAL, "NULL argument");
    fp8_to_bf16(codes, out, n, static_cast<hipStream_t>(stream));
    HIPC(hipGetLastError());
  });
}

int phyai_profile_stage(phyai_expert* e, int32_t stage, int32_t reps, void* stream) {
  return run_guarded([&] {
    if (!e) fail(PHYAI_EINVAL, "NULL handle");
    if (stage < 0 || stage >= kStages) fail(PHYAI_EINVAL, "stage out of range 0..6");
    if (reps < 1) fail(PHYAI_EINVAL, "reps < 1");
    if (e->last_batch < 1) fail(PHYAI_EINVAL, "call phyai_denoise first (the stage reads its inputs)");
    hipStream_t s = static_cast<hipStream_t>(stream);
    for (int r = 0; r < reps; ++r)
      for (int l = 0; l < full_layers(*e); ++l) {
        if (e->f32) layer_stage<float>(*e, stage, l, 0, e->last_batch, s);
        else layer_stage<bf16_t>(*e, stage, l, 0, e->last_batch, s);
      }
    HIPC(hipGetLastError());
  });
}

int phyai_prefill(phyai_expert* e, const float* embeds, const int32_t* prefix_len, void* kv_out, int32_t batch,
                  void* stream) {
  return run_guarded([&] {
    if (!e) fail(PHYAI_EINVAL, "NULL handle");
    if (e->c.variant != PHYAI_VARIANT_PREFIX_LM) fail(PHYAI_EINVAL, "not a prefix-LM handle");
    if (batch < 1 || batch > e->Bmax) fail(PHYAI_EINVAL, "batch out of range 1..max_batch");
    if (!embeds || !prefix_len || !kv_out) fail(PHYAI_EINVAL, "NULL argument");
    for (int b = 0; b < batch; ++b)
      if (prefix_len[b] < 0 || prefix_len[b] > e->M)
        fail(PHYAI_EINVAL, "prefix_len[" + std::to_string(b) + "] = " + std::to_string(prefix_len[b]) +
                               " outside 0..prefix_cap");
    auto aligned16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
    if (!aligned16(embeds) || !aligned16(kv_out)) fail(PHYAI_EINVAL, "embeds and kv_out must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    write_call_desc(*e, embeds, prefix_len, nullptr, batch, nullptr, nullptr, s);
    if (e->f32) enqueue_prefill<float>(*e, embeds, kv_out, batch, s);
    else enqueue_prefill<bf16_t>(*e, embeds, kv_out, batch, s);
    HIPC(hipGetLastError());
  });
}

int phyai_encode_images(phyai_expert* e, const float* patches, float* tokens_out, int32_t out_rows,
                        int32_t batch, void* stream) {
  return run_guarded([&] {
    if (!e) fail(PHYAI_EINVAL, "NULL handle");
    if (e->c.variant != PHYAI_VARIANT_VISION) fail(PHYAI_EINVAL, "not a vision handle");
    if (batch < 1 || batch > e->c.max_batch) fail(PHYAI_EINVAL, "batch out of range 1..max_batch");
    if (!patches || !tokens_out) fail(PHYAI_EINVAL, "NULL argument");
    if (out_rows < e->n_img * e->M) fail(PHYAI_EINVAL, "out_rows < n_images * n_patches");
    auto aligned16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
    if (!aligned16(patches) || !aligned16(tokens_out))
      fail(PHYAI_EINVAL, "patches and tokens_out must be 16-byte aligned");
    hipStream_t s = static_cast<hipStream_t>(stream);
    // every image is one attention "request" whose M patches are all valid keys
    const int Bi = batch * e->n_img;
    std::vector<int32_t> keys(Bi, e->M);
    write_call_desc(*e, nullptr, keys.data(), nullptr, Bi, nullptr, nullptr, s);
    if (e->f32) enqueue_vision<float>(*e, patches, tokens_out, out_rows, batch, s);
    else enqueue_vision<bf16_t>(*e, patches, tokens_out, out_rows, batch, s);
    HIPC(hipGetLastError());
  });
}

void phyai_free_expert(phyai_expert* e) { delete e; }

}  // extern "C"
