// Kernel interfaces of the denoising loop: argument blocks, GEMM epilogues
// and the host-side launchers the runtime composes into a HIP graph.
#pragma once

#include "common.hpp"

#include <type_traits>

namespace phyai {

constexpr int kMaxBatch = 512;

// Per-call arguments, written into device memory by a one-block kernel right
// before each graph replay (kernel arguments are copied at launch, so the
// host copy can go away immediately).  Kernels inside the graph read the
// caller's pointers and prefix lengths from here.
struct CallDesc {
  const void* prefix;
  const float* noise;
  const float* state;
  float* out;
  int32_t prefix_len[kMaxBatch];
};

// ---------------------------------------------------------------------------
// GEMM: C[R][N] = A[R][K] * W[K][N], W pre-packed in MFMA operand order.
// Columns are processed in "pair tiles" of 32: packed columns 32p .. 32p+15
// (half 0) and 32p+16 .. 32p+31 (half 1) reach the epilogue together, in the
// same thread, so that pairs (GeGLU gate/up, RoPE x1/x2) can be combined
// without a shuffle.  Which logical columns a pair tile holds is decided by
// the packing order chosen on the host.
// ---------------------------------------------------------------------------
enum WeightKind { W_F32 = 0, W_BF16 = 1, W_FP8 = 2, W_FP4 = 3 };

struct GemmArgs {
  const void* A;            // [R][lda], bf16 (MFMA path) or f32 (fp32 path)
  const void* A_lo;         // optional second bf16 term: A = A + A_lo (compensated operand)
  const void* const* A_ind; // if set: A = *A_ind + a_off (a per-call pointer in CallDesc)
  int64_t a_off;
  int lda;
  int R;
  int K;                    // multiple of 64 on the MFMA path
  int NPT;                  // pair tiles (N / 32)
  const void* W;            // packed weights
  const float* scale;       // fp8: one scale per packed column
  const uint8_t* mx;        // fp4: E8M0 scale exponents, per (pair tile, k-block, half) [16 columns][2 k-steps]
  int kind;                 // WeightKind
  // optional A-row validity: rows r with (r % rows_per_req) >= prefix_len[r / rows_per_req]
  // read as zero (used for feature rows beyond a request's length)
  int rows_per_req;
  const CallDesc* desc;
  // optional split over K (small row counts): raw partial sums go to
  // split_out + z * split_stride ([R][32*NPT] fp32 each) and the epilogue is
  // not run; the consumer adds the split_k slices in order
  float* split_out;
  int64_t split_stride;
  int split_k;
  // optional row scale of the output, the RMSNorm folded into this GEMM: A
  // holds bf16(h (1 + w)) and row r of the product is multiplied by
  // 1 / sqrt(sum_t row_ss[r][t] / (32 row_nt) + row_eps) (row_nt = d / 32
  // per-32-column sums of h^2 per row; small-row kernel only)
  const float* row_ss;
  int row_nt;
  float row_eps;
  // optional finishing of a split-K residual GEMM (with split_out; small-row
  // and merging kernels): the last block to arrive at an output tile adds
  // the split slices in order into fin_h (h += sum_s part[s]) and, with
  // fin_gain set, stores bf16(h (1 + fin_gain)) into fin_a and the tile's
  // per-row sums of h^2 into fin_ss [R][N / 32].  fin_ctr holds one counter
  // per output tile, zero at launch and left zero.
  float* fin_h;
  bf16_t* fin_a;
  float* fin_ss;
  const float* fin_gain;
  unsigned* fin_ctr;
};

// Split factor gemm launches use for a small-row GEMM (1 = no split).
int gemm_split_k(int R, int NPT, int K);

// Residual contribution left pending by split GEMMs, folded in by the next
// row kernel: h += gate * (sum_s part[s] + bias) (gate/bias optional).
struct PendingResid {
  const float* part;
  int n;
  int64_t stride;
  const float* gate;
  const float* bias;
};

// Epilogues take a pair-tile element (row r, pair tile p, column c, the two
// halves a0, a1).  Each has two phases so that a tile kernel can request the
// loads of all its elements before any store: colpre() loads what depends on
// the column only (once per pair tile), pre() what depends on the element,
// apply() computes and stores; operator() is all three in turn.
template <typename OutT>
struct EpiStore {
  static constexpr bool kWaveTile = false;
  OutT* out; int ldo;
  const float* bias;        // [N] or null
  const float* rowvec;      // [N] added to every row, or null
  int act;                  // Act
  int grp, grp_stride, grp_off;   // row remap: (r/grp)*grp_stride + grp_off + r%grp (grp=0: identity)
  struct ColPre { float b[2], rv[2]; };
  struct Pre {};
  __device__ __forceinline__ ColPre colpre(int p, int c) const {
    ColPre q;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int col = 32 * p + 16 * hf + c;
      q.b[hf] = bias ? bias[col] : 0.f;
      q.rv[hf] = rowvec ? rowvec[col] : 0.f;
    }
    return q;
  }
  __device__ __forceinline__ Pre pre(int, int, int) const { return Pre{}; }
  __device__ __forceinline__ void apply(int r, int p, int c, const ColPre& q, const Pre&, float a0, float a1) const {
    int orow = r;
    if (grp > 0) orow = (r / grp) * grp_stride + grp_off + (r % grp);
    float v[2] = {a0, a1};
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int col = 32 * p + 16 * hf + c;
      float t = v[hf];
      if (bias) t += q.b[hf];
      if (rowvec) t += q.rv[hf];
      ActIO<OutT>::store(out + (int64_t)orow * ldo + col, apply_act(act, t));
    }
  }
  __device__ __forceinline__ void operator()(int r, int p, int c, float a0, float a1) const {
    apply(r, p, c, colpre(p, c), pre(r, p, c), a0, a1);
  }
};

// h[r][col] += gate[col] * (acc + bias[col])
struct EpiResid {
  static constexpr bool kWaveTile = false;
  float* h; int ldh;
  const float* bias;
  const float* gate;
  struct ColPre { float b[2], g[2]; };
  struct Pre { float h[2]; };
  __device__ __forceinline__ ColPre colpre(int p, int c) const {
    ColPre q;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int col = 32 * p + 16 * hf + c;
      q.b[hf] = bias ? bias[col] : 0.f;
      q.g[hf] = gate ? gate[col] : 1.f;
    }
    return q;
  }
  __device__ __forceinline__ Pre pre(int r, int p, int c) const {
    Pre q;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) q.h[hf] = h[(int64_t)r * ldh + 32 * p + 16 * hf + c];
    return q;
  }
  __device__ __forceinline__ void apply(int r, int p, int c, const ColPre& cq, const Pre& q, float a0, float a1) const {
    float v[2] = {a0, a1};
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int col = 32 * p + 16 * hf + c;
      float t = v[hf];
      if (bias) t += cq.b[hf];
      if (gate) t *= cq.g[hf];
      h[(int64_t)r * ldh + col] = q.h[hf] + t;
    }
  }
  __device__ __forceinline__ void operator()(int r, int p, int c, float a0, float a1) const {
    apply(r, p, c, colpre(p, c), pre(r, p, c), a0, a1);
  }
};

// pair tile p holds gate column 16p+c (half 0) and up column 16p+c (half 1).
// With `lo` set (bf16 only) the rounding residue is stored there, so that
// out + lo carries about 16 significant bits into the next GEMM.
template <typename OutT>
struct EpiGeglu {
  static constexpr bool kWaveTile = false;
  OutT* out; int ldo;
  OutT* lo;
  struct ColPre {};
  struct Pre {};
  __device__ __forceinline__ ColPre colpre(int, int) const { return ColPre{}; }
  __device__ __forceinline__ Pre pre(int, int, int) const { return Pre{}; }
  __device__ __forceinline__ void apply(int r, int p, int c, const ColPre&, const Pre&, float a0, float a1) const {
    const float v = gelu_tanh_f(a0) * a1;
    const int64_t i = (int64_t)r * ldo + 16 * p + c;
    ActIO<OutT>::store(out + i, v);
    if (lo) ActIO<OutT>::store(lo + i, v - ActIO<OutT>::round(v));
  }
  __device__ __forceinline__ void operator()(int r, int p, int c, float a0, float a1) const {
    apply(r, p, c, ColPre{}, Pre{}, a0, a1);
  }
};

// Fused QKV.  Heads are ordered [n_q query | n_kv key | n_kv value], each
// head_dim wide; head h owns pair tiles h*D/32 .. (h+1)*D/32-1, and pair tile
// j of a head holds dimension i = 16j+c (half 0) and i + D/2 (half 1), the
// two halves that RoPE rotates together.  q goes to [R][nq*D]; k and v go
// into the layer's key range (K [b][kvh][key][D], V transposed
// [b][kvh][D][key]) at key = (prefix_len[b] if keys_after_prefix) + token.
// An optional bias [(nq + 2 nkv) * D], in the unpacked head order, is added
// before RoPE.
template <typename OutT>
struct EpiQkv {
  static constexpr bool kWaveTile = true;   // see wave_tile
  OutT* q; OutT* kall; OutT* vt;
  int D, nq, nkv;
  int rope;
  int M;                    // suffix tokens per request
  int ldk;                  // key capacity of a key range
  int keys_after_prefix;
  const float2* rope_cs;    // [rows][D/2]: (cos, sin) of position * base^(-2i/D)
  const CallDesc* desc;     // positions start at prefix_len[b]
  const float* bias;        // or null
  struct ColPre {};
  struct Pre { float2 cs; int plen; };
  __device__ __forceinline__ ColPre colpre(int, int) const { return ColPre{}; }
  __device__ __forceinline__ Pre pre(int r, int p, int c) const {
    const int tiles = D / 32;
    const int head = p / tiles;
    const int i = 16 * (p % tiles) + c;
    Pre q;
    q.cs = (rope && head < nq + nkv) ? rope_cs[(int64_t)r * (D / 2) + i] : make_float2(1.f, 0.f);
    q.plen = head >= nq ? desc->prefix_len[r / M] : 0;
    return q;
  }
  __device__ __forceinline__ void apply(int r, int p, int c, const ColPre&, const Pre& q, float a0, float a1) const {
    const int tiles = D / 32;
    const int head = p / tiles;
    const int i = 16 * (p % tiles) + c;
    const int b = r / M, tok = r % M;
    if (bias) {
      a0 += bias[head * D + i];
      a1 += bias[head * D + i + D / 2];
    }
    if (rope && head < nq + nkv) {
      const float x1 = a0, x2 = a1;
      a0 = x1 * q.cs.x - x2 * q.cs.y;
      a1 = x2 * q.cs.x + x1 * q.cs.y;
    }
    if (head < nq) {
      OutT* dst = this->q + (int64_t)r * nq * D + head * D + i;
      ActIO<OutT>::store(dst, a0);
      ActIO<OutT>::store(dst + D / 2, a1);
      return;
    }
    const int key = (keys_after_prefix ? q.plen : 0) + tok;
    if (head < nq + nkv) {
      OutT* dst = kall + (((int64_t)b * nkv + (head - nq)) * ldk + key) * D + i;
      ActIO<OutT>::store(dst, a0);
      ActIO<OutT>::store(dst + D / 2, a1);
    } else {
      OutT* dst = vt + (((int64_t)b * nkv + (head - nq - nkv)) * D + i) * ldk + key;
      ActIO<OutT>::store(dst, a0);
      ActIO<OutT>::store(dst + (int64_t)(D / 2) * ldk, a1);
    }
  }
  __device__ __forceinline__ void operator()(int r, int p, int c, float a0, float a1) const {
    apply(r, p, c, ColPre{}, pre(r, p, c), a0, a1);
  }

  // Epilogue of a wave's 64 x 64 tile of a many-row GEMM: rows r0 + 16mt +
  // 4lg + v, pair tiles p0 (even) and p0 + 1, which always belong to one
  // head, so whether the tile is Q, K or V (and whether it is rotated) is
  // known once per tile.  Per group of four rows every RoPE factor and
  // prefix length is requested before the group's stores; the per-element
  // form above would wait for each element's loads in turn.  Tiles that
  // reach past R take the per-element form.
  // V tiles through LDS: `st` (kVStage elements per wave, or null) receives the
  // wave's 64 x 64 tile as [column][row], and each store instruction then
  // writes 64 consecutive keys of one V^T row (128 contiguous bytes) instead of
  // 16 rows x 4 keys.
  static constexpr int kVRow = 66;                    // padded row: 64 tokens, no bank conflicts
  static constexpr int kVStage = 64 * kVRow;
  __device__ __forceinline__ void wave_tile(const GemmArgs& g, const f32x4 (&acc)[4][4], int r0, int p0, int lc,
                                            int lg, bf16_t* st = nullptr) const {
    const int tiles = D / 32;
    const int head = p0 / tiles;
    float sc[2][2];
#pragma unroll
    for (int pp = 0; pp < 2; ++pp) {
      sc[pp][0] = g.scale ? g.scale[32 * (p0 + pp) + lc] : 1.f;
      sc[pp][1] = g.scale ? g.scale[32 * (p0 + pp) + 16 + lc] : 1.f;
    }
    if (r0 + 64 > g.R) {      // bias added by the per-element form
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = r0 + 16 * mt + 4 * lg + v;
            if (row < g.R)
              (*this)(row, p0 + pp, lc, acc[mt][2 * pp][v] * sc[pp][0], acc[mt][2 * pp + 1][v] * sc[pp][1]);
          }
      return;
    }
    float bs[2][2] = {{0.f, 0.f}, {0.f, 0.f}};
    if (bias) {
#pragma unroll
      for (int pp = 0; pp < 2; ++pp) {
        const int i = 16 * ((p0 + pp) % tiles) + lc;
        bs[pp][0] = bias[head * D + i];
        bs[pp][1] = bias[head * D + i + D / 2];
      }
    }
    auto emit = [&](auto kind) {
      constexpr int KIND = decltype(kind)::value;     // 0: q, 1: k, 2: v
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        float2 cs[2][4];
        int key[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = r0 + 16 * mt + 4 * lg + v;
#pragma unroll
          for (int pp = 0; pp < 2; ++pp) {
            const int i = 16 * ((p0 + pp) % tiles) + lc;
            cs[pp][v] = (KIND < 2 && rope) ? rope_cs[(int64_t)row * (D / 2) + i] : make_float2(1.f, 0.f);
          }
          key[v] = KIND > 0 ? (keys_after_prefix ? desc->prefix_len[row / M] : 0) + row % M : 0;
        }
#pragma unroll
        for (int pp = 0; pp < 2; ++pp)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = r0 + 16 * mt + 4 * lg + v;
            const int i = 16 * ((p0 + pp) % tiles) + lc;
            const float x1 = acc[mt][2 * pp][v] * sc[pp][0] + bs[pp][0];
            const float x2 = acc[mt][2 * pp + 1][v] * sc[pp][1] + bs[pp][1];
            float a0 = x1, a1 = x2;
            if (KIND < 2 && rope) {
              a0 = x1 * cs[pp][v].x - x2 * cs[pp][v].y;
              a1 = x2 * cs[pp][v].x + x1 * cs[pp][v].y;
            }
            if (KIND == 0) {
              OutT* dst = q + (int64_t)row * nq * D + head * D + i;
              ActIO<OutT>::store(dst, a0);
              ActIO<OutT>::store(dst + D / 2, a1);
            } else if (KIND == 1) {
              OutT* dst = kall + (((int64_t)(row / M) * nkv + (head - nq)) * ldk + key[v]) * D + i;
              ActIO<OutT>::store(dst, a0);
              ActIO<OutT>::store(dst + D / 2, a1);
            } else {
              OutT* dst = vt + (((int64_t)(row / M) * nkv + (head - nq - nkv)) * D + i) * ldk + key[v];
              ActIO<OutT>::store(dst, a0);
              ActIO<OutT>::store(dst + (int64_t)(D / 2) * ldk, a1);
            }
          }
      }
    };
    if (head < nq) emit(std::integral_constant<int, 0>{});
    else if (head < nq + nkv) emit(std::integral_constant<int, 1>{});
    else {
      if constexpr (std::is_same<OutT, bf16_t>::value) {
        if (st != nullptr) {
          store_v_staged(acc, sc, bs, r0, p0, lc, lg, st);
          return;
        }
      }
      emit(std::integral_constant<int, 2>{});
    }
  }

  __device__ __forceinline__ void store_v_staged(const f32x4 (&acc)[4][4], const float (&sc)[2][2],
                                                 const float (&bs)[2][2], int r0, int p0, int lc, int lg,
                                                 bf16_t* st) const {
    const int tiles = D / 32;
    const int head = p0 / tiles;
    {
#pragma unroll
      for (int pp = 0; pp < 2; ++pp)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = 16 * mt + 4 * lg + v;
            st[(32 * pp + lc) * kVRow + row] = f32_to_bf16(acc[mt][2 * pp][v] * sc[pp][0] + bs[pp][0]);
            st[(32 * pp + 16 + lc) * kVRow + row] = f32_to_bf16(acc[mt][2 * pp + 1][v] * sc[pp][1] + bs[pp][1]);
          }
      const int lane = 16 * lg + lc;
      const int row = r0 + lane;
      const int key = (keys_after_prefix ? desc->prefix_len[row / M] : 0) + row % M;
      bf16_t* vrow = reinterpret_cast<bf16_t*>(vt) + ((int64_t)(row / M) * nkv + (head - nq - nkv)) * D * ldk + key;
      __builtin_amdgcn_s_waitcnt(0xC07F);             // the wave's LDS writes are done (lgkmcnt 0)
#pragma unroll 8
      for (int col = 0; col < 64; ++col) {
        const int i = 16 * ((p0 + col / 32) % tiles) + col % 16;
        const int d = i + ((col / 16) % 2) * (D / 2);
        vrow[(int64_t)d * ldk] = st[col * kVRow + lane];
      }
    }
  }
};

// K|V projection of feature rows r = b*P + key (identity packing): columns
// [0, nkv*D) are K heads, [nkv*D, 2*nkv*D) V heads, stored like EpiQkv's k/v.
template <typename OutT>
struct EpiKV {
  static constexpr bool kWaveTile = false;
  OutT* kall; OutT* vt;
  int D, nkv, P, ldk;
  struct ColPre {};
  struct Pre {};
  __device__ __forceinline__ ColPre colpre(int, int) const { return ColPre{}; }
  __device__ __forceinline__ Pre pre(int, int, int) const { return Pre{}; }
  __device__ __forceinline__ void apply(int r, int p, int c, const ColPre&, const Pre&, float a0, float a1) const {
    const int b = r / P, key = r % P;
    float v[2] = {a0, a1};
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int col = 32 * p + 16 * hf + c;
      const int kv = col / (nkv * D), rem = col % (nkv * D);
      const int h = rem / D, i = rem % D;
      if (kv == 0) ActIO<OutT>::store(kall + (((int64_t)b * nkv + h) * ldk + key) * D + i, v[hf]);
      else ActIO<OutT>::store(vt + (((int64_t)b * nkv + h) * D + i) * ldk + key, v[hf]);
    }
  }
  __device__ __forceinline__ void operator()(int r, int p, int c, float a0, float a1) const {
    apply(r, p, c, ColPre{}, Pre{}, a0, a1);
  }
};

void gemm_store_bf16(const GemmArgs&, const EpiStore<bf16_t>&, hipStream_t);
void gemm_store_f32(const GemmArgs&, const EpiStore<float>&, hipStream_t);
void gemm_resid(const GemmArgs&, const EpiResid&, hipStream_t);
void gemm_geglu_bf16(const GemmArgs&, const EpiGeglu<bf16_t>&, hipStream_t);
void gemm_geglu_f32(const GemmArgs&, const EpiGeglu<float>&, hipStream_t);
void gemm_qkv_bf16(const GemmArgs&, const EpiQkv<bf16_t>&, hipStream_t);
void gemm_qkv_f32(const GemmArgs&, const EpiQkv<float>&, hipStream_t);
void gemm_kv_bf16(const GemmArgs&, const EpiKV<bf16_t>&, hipStream_t);
void gemm_kv_f32(const GemmArgs&, const EpiKV<float>&, hipStream_t);

// ---------------------------------------------------------------------------
// Attention of suffix queries over one key range per (request, kv head):
// K [key][D] and V^T [D][key] at grp * ldk * D (grp = b * nkv + kvh).  The
// range holds n_keys(b) = (keys_from_prefix ? prefix_len[b] : 0) + n_suffix
// keys.  Query rows of (b, kv head h) are token*G + g for the G = nq/nkv
// query heads sharing kv head h.  mask_mode 1 is the pi0 block mask: the
// state token (suffix token 0, key prefix_len[b]) sees the prefix and
// itself only.
// ---------------------------------------------------------------------------
struct AttnArgs {
  const void* q; int ldq;
  const void* K; const void* Vt;
  int ldk;
  int keys_from_prefix, n_suffix;
  int mask_mode;
  void* out; int ldo;
  float* part;              // split partials (n_split > 1)
  int64_t part_ml_off;      // set by the launcher
  int rows_per_tile;        // query rows per block, set by the launcher
  int n_split;
  int defer_merge;          // n_split > 1: leave the partials for gemm_merge_resid
  const CallDesc* desc;
  int B, M, nq, nkv, D;
  float scale;              // 1/sqrt(D)
};

void attention_bf16(const AttnArgs&, hipStream_t);
void attention_f32(const AttnArgs&, hipStream_t);
int64_t attention_partial_floats(int B, int M, int nq, int nkv, int D, int n_split);
int attention_rows_per_block(int B, int rows, int nkv);

// Key-split partials of one bf16 attention launch: O rows [tile][split][rows_per_tile][D]
// (bf16, each split normalised by its own softmax sum) and (m, l) [tile][split][rows_per_tile]
// (float2).  Query row qr = token * G + (head % G) of group b * nkv + head / G sits in tile
// group * ntiles + qr / rows_per_tile.
struct AttnParts {
  const bf16_t* o;
  const float* ml;
  int n_split, ntiles, rows_per_tile;
  int M, G, nkv, D;
};
AttnParts attention_parts(const AttnArgs&);

// Output projection that takes its A operand (the attention output, [R][nq*D]) straight
// from the key-split partials, merging them on the way in (small row counts).  K runs in
// slices of 256 (blockIdx.z); with g.split_out set each slice goes there raw (g.split_k =
// K / 256 slices), otherwise the epilogue adds into h.  Needs K % 256 == 0, 256 % D == 0,
// 2 <= n_split <= 16 and bf16 or fp8 weights.
void gemm_merge_resid(const GemmArgs&, const AttnParts&, const EpiResid&, hipStream_t);

// Copy the caller's prefix K and transpose its V ([L][2][B][P][nkv*D]) into
// the per-layer key ranges (layer l at K/Vt + l * layer_stride).
struct RelayoutArgs {
  const CallDesc* desc;
  void* K; void* Vt;
  int64_t layer_stride;
  int ldk, L, B, P, nkv, D;
  int n_suffix;             // suffix keys that follow the prefix (zero-fill starts after them)
};
void prefix_relayout_bf16(const RelayoutArgs&, hipStream_t);
void prefix_relayout_f32(const RelayoutArgs&, hipStream_t);

// The prefix LM's keys and values of one layer, out of the library's key
// ranges (K [ldk][D], V transposed [D][ldk] per request and kv head) into the
// caller's prefix layout [2][B][P][nkv*D] (`out` points at the layer's
// block; the V half starts `half` elements later): the layout the denoising
// loop reads back as its frozen prefix.  Keys at or beyond prefix_len[b]
// are written as zeros.
struct KvExportArgs {
  const CallDesc* desc;
  const void* K; const void* Vt;
  void* out;
  int64_t half;
  int B, P, nkv, D, ldk;
};
void kv_export_bf16(const KvExportArgs&, hipStream_t);
void kv_export_f32(const KvExportArgs&, hipStream_t);

// ---------------------------------------------------------------------------
// Row kernels
// ---------------------------------------------------------------------------
enum NormMode { NORM_RMS = 0, NORM_LN = 1 };

// n = normalise(h) * (1 + mul) + shift ; RMS or mean-centred LayerNorm.
// With n_lo set, n_lo receives the bf16 rounding residue of n (two-term operand).
// With pend.n > 0 the pending residual is first added into h (written back):
// the fused residual-add + norm.
void norm_rows_bf16(float* h, bf16_t* n, bf16_t* n_lo, int R, int d, float eps, int mode,
                    const float* mul, const float* shift, const PendingResid& pend, hipStream_t);
void norm_rows_f32(float* h, float* n, int R, int d, float eps, int mode,
                   const float* mul, const float* shift, const PendingResid& pend, hipStream_t);

struct EmbedArgs {
  const float* x;           // solver state [B][H][A]
  const float* in_w;        // [A][d] fp32
  const float* in_b;        // [d]
  const float* rowvec;      // [d] also added to every action row, or null
  int act;                  // Act applied to action rows
  const float* pos;         // [H][d] or null
  const float* e_state;     // [B][d] or null (state rows of h)
  float* h;                 // [B*M][d]: destination of state rows, and of action rows if act_out == null
  void* act_out;            // [B*H][d] Act: destination of action rows (pi0 time MLP input)
  int act_is_bf16;
  int B, H, M, A, d, off;   // off = 1 if a state token leads each request
};
void embed_actions(const EmbedArgs&, hipStream_t);

// e[b][c] = state[b] . W[:, c] + bias[c]; state read from CallDesc.
void embed_state(const CallDesc* desc, const float* w, const float* b, float* e, int B, int A, int d,
                 hipStream_t);

struct ReadoutArgs {
  float* h; int B, H, M, off, d, A;
  PendingResid pend;        // residual still pending from the last block
  float eps; int mode;
  const float* mul; const float* shift;   // final norm: * (1 + mul) + shift
  const float* out_w;       // [A][d] fp32 (transposed W_out)
  const float* out_b;       // [A]
  const float* dt;          // t_{k+1} - t_k (device scalar)
  float* x;                 // [B][H][A], updated in place
  // With has_next, the next step's embedding of the updated rows (and the
  // state rows' reset) as embed_actions would do it with `next`; only where
  // readout_fuses_embedding says so.
  int has_next;
  EmbedArgs next;
};
void readout_euler(const ReadoutArgs&, hipStream_t);
// Whether readout_euler can take has_next for these sizes: only its one-row
// blocks (the four-row form needs too many registers with the embedding).
bool readout_fuses_embedding(int A, int d, int rows, bool pending);

void copy_noise_to_state(const CallDesc* desc, float* x, int64_t n, hipStream_t);
void copy_state_to_out(const CallDesc* desc, const float* x, int64_t n, hipStream_t);
void set_call_desc(const CallDesc& host_desc, CallDesc* dev, hipStream_t);
// RoPE table of one call: tab[b*M + t][i] = (cos, sin)((p0 + t) * inv_freq[i]),
// i < D/2, with p0 = prefix_len[b] when pos_after_prefix (the suffix tokens'
// positions follow their request's prefix) and 0 otherwise (the prefix
// tokens themselves).
void rope_table(const CallDesc* desc, const float* inv_freq, float2* tab, int B, int M, int D, int pos_after_prefix,
                hipStream_t);
// Residual stream of the prefix LM from the caller's embeddings:
// h[b*M + t] = embeds[b][t] for t < prefix_len[b], zero after (the caller's
// rows past the prefix are never read).  d a multiple of 4, embeds 16-byte
// aligned.
void prefill_embed(const CallDesc* desc, const float* embeds, float* h, int B, int M, int d, hipStream_t);
// Vision tower input: patches [R][patch_dim] float32 into the GEMM operand
// `a` (bf16 or float32, same layout) and the position embedding of each row's
// patch (row % n_patches) into the residual stream h [R][d].
void vision_embed_bf16(const float* patches, bf16_t* a, float* h, const float* pos, int R, int n_patches,
                       int patch_dim, int d, hipStream_t);
void vision_embed_f32(const float* patches, float* a, float* h, const float* pos, int R, int n_patches,
                      int patch_dim, int d, hipStream_t);
void fp8_to_bf16(const uint8_t* codes, bf16_t* out, int64_t n, hipStream_t);

// ---------------------------------------------------------------------------
// Persistent batch-1 loop: one cooperative launch runs all K Euler steps of
// one pi0 request (bf16 weights, one KV head, at most 64 suffix tokens).
// Blocks hand activations to each other through write-through device-scope
// stores and a grid barrier.  Data rewritten within a launch (the residual,
// partials, the suffix keys) is read back with device-scope loads; the GEMM
// operands get a fresh copy per step and site, written once per launch, so
// their readers use plain cached loads (a launch starts with the L2s
// invalidated).  Residual split-K partials are reduced by the last block to
// finish each column tile; every norm is folded into the GEMM that consumes
// it (the producer leaves bf16(h (1 + w)) and per-tile sums of squares, the
// consumer scales its rows by 1/rms).
// ---------------------------------------------------------------------------
struct PersistLayer {
  const void* qkv; const void* o; const void* gu; const void* down;   // packed bf16 weights
  const float* attn_norm; const float* mlp_norm;                      // RMSNorm gains w ((1 + w))
};

struct PersistArgs {
  const CallDesc* desc;
  const PersistLayer* layer;   // device array [L]
  int L, d, D, nq, F, H, A, M, off;
  int ldk;
  int64_t kv_layer;            // elements per layer of the key ranges
  bf16_t* kall; bf16_t* vt;    // key ranges: K [L][ldk][D], V^T [L][D][ldk] (prefix relaid before launch)
  float* h;                    // residual stream [64][d]
  // per-step copies, r = the step's place in the launch (< kPersistRing)
  bf16_t* a;                   // bf16(h (1 + w)) per norm site [R][L+1][2][64][d]
  float* ss;                   // sums of h^2 per 32-column tile [R][L+1][2][64][d/32]
  bf16_t* z;                   // time-MLP hidden [R][64][d]
  bf16_t* q;                   // queries [R][L][64][nq*D]
  bf16_t* o;                   // merged attention output [R][L][64][nq*D]
  bf16_t* g;                   // GeGLU output [R][L][64][F]
  bf16_t* apart;               // key-split attention partials [nq][ntile][64][D] (normalised)
  float2* aml;                 // (max, sum) of each partial row [nq][ntile][64] (log2 domain)
  float* part;                 // residual split-K partials [16][64][d]
  float* x;                    // solver state [H][A]
  const float* e_state;        // state-token embedding [d] (or null)
  const float* tin_w; const float* tin_b;   // action embedding folded into the time MLP [A][d], [d]
  const float* T;              // time-MLP tau half per step [K][d]
  const void* time_w2; const float* time_b2;
  const float* out_w;          // [A][d] (transposed)
  const float* out_b; const float* final_norm; const float* dt;
  const float2* rope_cs;       // [M][D/2] or null
  float eps, scale;
  unsigned* ctr;               // barrier and tile counters, zero at launch
};

// Whether the persistent loop takes this shape (see the launcher).
bool persist_supported(int d, int D, int nq, int F, int M, int A);
// Launch it for steps k0 .. k1 - 1 (k1 - k0 <= kPersistRing) of a K-step
// schedule, with the arguments at dev_args (device memory holding a copy of
// `a`, which the launcher reads for the shape).  The counters must be zero.
// Cooperative: fails with the HIP error if the grid cannot be co-resident.
hipError_t persist_launch(const PersistArgs& a, const PersistArgs* dev_args, int k0, int k1, int K, hipStream_t);
constexpr int kPersistCounters = 1024;
constexpr int kPersistRing = 16;   // steps per launch (per-step copies held)

}  // namespace phyai
