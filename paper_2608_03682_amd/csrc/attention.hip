// Suffix-query attention over the frozen prefix K/V and the suffix tokens'
// own K/V (the "50-token query against a longer prefix, head dimension 256"
// shape of Section "PhyAI Architecture", paragraph "Profiled operator
// selection"), with online softmax and an optional split over the keys.
//
// Key layout.  Per layer, request and kv head the library keeps one key
// range: K row-major [key][D] and V transposed [D][key].  Keys
// 0 .. prefix_len-1 are the frozen prefix (relaid once per call by
// prefix_relayout_kernel, which is the "retained prefix state" of the
// paragraph "Graph replay"); the suffix tokens' K/V of the current layer
// are written behind them by the QKV epilogue.  Attention then reads one
// contiguous range with 16-byte loads, and V arrives already in the
// key-contiguous order the P.V product needs.
//
// MFMA formulation: S^T = K Q^T and O^T = V^T P^T, so a query is always
// the MFMA column (lane % 16): its softmax statistics live in the four lanes
// l%16 == q (two cross-lane steps), and the probabilities leave the S^T
// accumulators already laid out as the B operand of the P.V product (the
// key order inside k is permuted identically on both operands).
//
// Block: 4 waves x 32 query rows (two 16-row groups per wave, so every K/V
// fragment read from LDS feeds two MFMAs); 64-key tiles double-buffered in
// LDS and filled by direct global->LDS loads, the next tile in flight while
// the current one is computed.
// With n_split > 1 the key range is split over blocks, whose partials a
// second kernel merges in a fixed order.
#include "kernels.hpp"

namespace phyai {

namespace {

constexpr int kKT = 64;          // keys per tile
constexpr int kRows = 128;       // query rows per block

typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from `src` into LDS at (wave-uniform) lds + 16 * lane.
// Issued as asm so that the compiler does not put a vmcnt(0) in front of
// every LDS read (it cannot tell the tile in flight from the one being
// read); completion is awaited explicitly with PHYAI_WAIT_VMCNT.  Vector
// loads retire in order, so the compiler's own vmcnt waits stay valid.
__device__ __forceinline__ void lds_dma16(const void* src, lds_void* lds) {
  const uint32_t m = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(m), "v"(src) : "memory", "m0");
}

// s_waitcnt with vmcnt = n (n < 64) and the other counters left open.
#define PHYAI_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x70 | 0xF00)
// Workgroup barrier without __syncthreads()'s memory fence (which would also
// wait for the prefetch in flight).  LDS reads of the caller are complete
// (lgkmcnt 0) before the barrier; LDS written by global->LDS loads is
// published by the explicit vmcnt wait that precedes the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt/expcnt left open
  __builtin_amdgcn_s_barrier();
}

// LDS tiles, 16-byte chunks XOR-swizzled so that the MFMA fragment reads of
// 16 lanes (16 rows, same column) fall in 16 different bank groups:
//   K  [64 keys][D]:   chunk c of key row r sits at position c ^ (r & 15)
//   Vt [D][64 keys]:   chunk c of row d sits at position c ^ ((d >> 1) & 7)
template <int D>
struct AttnTile {
  bf16_t K[kKT * D];
  bf16_t Vt[D * kKT];
};

template <int D>
__device__ __forceinline__ int kswz(int r) { return (D / 8 >= 16) ? (r & 15) : (r & (D / 8 - 1)); }
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 7; }

// One 64-key tile of the online-softmax attention for the wave's two query
// groups, reading K and V^T from the LDS tile T.
template <int D>
__device__ __forceinline__ void attn_tile(const AttnTile<D>& T, const bf16x8 (&qf)[2][D / 32],
                                          f32x4 (&o)[2][D / 16], float (&m_run)[2], float (&l_run)[2],
                                          int kt0, int kend, int plen, bool state0, bool state1, float sl2,
                                          int lc, int lg) {
  f32x4 st[2][4];
#pragma unroll
  for (int kt = 0; kt < 4; ++kt) {
    const int r = 16 * kt + lc;
    bf16x8 kf[D / 32];
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      kf[s] = *reinterpret_cast<const bf16x8*>(T.K + r * D + 8 * ((4 * s + lg) ^ kswz<D>(r)));
    st[0][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
    st[1][kt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      st[0][kt] = mfma16x16x32(kf[s], qf[0][s], st[0][kt]);
      st[1][kt] = mfma16x16x32(kf[s], qf[1][s], st[1][kt]);
    }
  }
  // Scores are masked only where a mask can bite: the tile holding the end
  // of the key range, and state-token queries (wave-uniform test).
  const bool need_mask = !(kt0 + kKT <= kend) || state0 || state1;
  bf16x8 pf[2][2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const bool state_q = c == 0 ? state0 : state1;
    float sc[16];
    float tmax = -INFINITY;
    if (__ballot(need_mask)) {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int key = kt0 + 16 * kt + 4 * lg + v;
          const bool ok = key < kend && (!state_q || key <= plen);
          const float s = ok ? st[c][kt][v] * sl2 : -INFINITY;
          sc[kt * 4 + v] = s;
          tmax = fmaxf(tmax, s);
        }
    } else {
#pragma unroll
      for (int kt = 0; kt < 4; ++kt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float s = st[c][kt][v] * sl2;
          sc[kt * 4 + v] = s;
          tmax = fmaxf(tmax, s);
        }
    }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    // Lazy rescaling: the running reference m only moves when the tile max
    // exceeds it by more than 8 (log2 units), so exp2(s - m) <= 256 and the
    // accumulators are rescaled only a few times per key range.
    if (__ballot(tmax > m_run[c] + 8.f)) {
      const float m_new = fmaxf(m_run[c], tmax);
      const float alpha = __builtin_amdgcn_exp2f(m_run[c] - m_new);
      m_run[c] = m_new;
      l_run[c] *= alpha;
#pragma unroll
      for (int i = 0; i < D / 16; ++i) o[c][i] *= alpha;
    }
    float p[16], psum = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      p[i] = __builtin_amdgcn_exp2f(sc[i] - m_run[c]);
      psum += p[i];
    }
    l_run[c] += psum;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint4 w;
      w.x = pack_bf16x2(p[8 * h + 0], p[8 * h + 1]);
      w.y = pack_bf16x2(p[8 * h + 2], p[8 * h + 3]);
      w.z = pack_bf16x2(p[8 * h + 4], p[8 * h + 5]);
      w.w = pack_bf16x2(p[8 * h + 6], p[8 * h + 7]);
      pf[c][h] = as_bf16x8(w);
    }
  }
  // V^T fragments, four d-tiles per batch
  const int vo = 4 * (lg & 1);
#pragma unroll
  for (int d0 = 0; d0 < D / 16; d0 += 4) {
    bf16x8 vf[4][2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int d = 16 * (d0 + j) + lc;
      const bf16_t* vrow = T.Vt + d * kKT + vo;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int c0 = 4 * h + (lg >> 1);
        const uint2 lo = *reinterpret_cast<const uint2*>(vrow + 8 * (c0 ^ vswz(d)));
        const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 8 * ((c0 + 2) ^ vswz(d)));
        vf[j][h] = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        o[0][d0 + j] = mfma16x16x32(vf[j][h], pf[0][h], o[0][d0 + j]);
        o[1][d0 + j] = mfma16x16x32(vf[j][h], pf[1][h], o[1][d0 + j]);
      }
  }
}

template <int D>
__global__ __launch_bounds__(256) void attn_mfma_kernel(AttnArgs a) {
  // two separate LDS objects so that loads into one and reads of the other
  // are visibly independent
  __shared__ __attribute__((aligned(1024))) AttnTile<D> smA;
  __shared__ __attribute__((aligned(1024))) AttnTile<D> smB;
  constexpr int CPR = D / 8;                  // 16-byte chunks per K row
  constexpr int NLD = kKT * D / 8 / 256;      // loads per thread per operand per tile
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int lg = lane / 16, lc = lane % 16;
  const int G = a.nq / a.nkv;
  const int rows = a.M * G;
  // 1-D grid, XCD-aware: blocks are dealt to the 8 XCDs round-robin, so the
  // row tiles of one (request, kv head, split) get ids that are equal mod 8
  // and share that XCD's L2 while they stream the same keys.
  const int ntiles = (rows + kRows - 1) / kRows;
  const int ngroups = a.B * a.nkv * a.n_split;
  const int xcd = blockIdx.x % 8, j = blockIdx.x / 8;
  const int rt = j % ntiles;
  const int gi = (j / ntiles) * 8 + xcd;
  if (gi >= ngroups) return;
  const int grp = gi / a.n_split, split = gi % a.n_split;
  const int b = grp / a.nkv, kvh = grp % a.nkv;

  const int plen = a.desc->prefix_len[b];
  const int n_keys = (a.keys_from_prefix ? plen : 0) + a.n_suffix;
  int chunk = (n_keys + a.n_split - 1) / a.n_split;
  chunk = (chunk + kKT - 1) / kKT * kKT;
  const int kbeg = split * chunk;
  const int kend = min(n_keys, kbeg + chunk);

  const bf16_t* Kb = static_cast<const bf16_t*>(a.K) + (int64_t)grp * a.ldk * D;
  const bf16_t* Vb = static_cast<const bf16_t*>(a.Vt) + (int64_t)grp * a.ldk * D;

  int qr[2], qtok[2];
  bool qv[2];
  bf16x8 qf[2][D / 32];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    qr[c] = rt * kRows + wave * 32 + c * 16 + lc;
    qv[c] = qr[c] < rows;
    qtok[c] = qv[c] ? qr[c] / G : 0;
    const int qhead = kvh * G + (qv[c] ? qr[c] % G : 0);
    const bf16_t* qp = static_cast<const bf16_t*>(a.q) + (int64_t)(b * a.M + qtok[c]) * a.ldq + qhead * D + 8 * lg;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qv[c]) v = *reinterpret_cast<const uint4*>(qp + 32 * s);
      qf[c][s] = as_bf16x8(v);
    }
  }
  // Direct global->LDS loads of one tile (the key range always holds whole,
  // finite 64-key tiles).  Wave w's i-th load fills 1 KiB block 4i + w; the
  // per-thread source offsets (elements) do not depend on the tile.
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  int koff[NLD], voff[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int pos = (4 * i + wave) * 64 + lane;
    const int r = pos / CPR, pc = pos % CPR;
    koff[i] = r * D + 8 * (pc ^ kswz<D>(r));
    const int d = pos / 8, vc = pos % 8;
    voff[i] = d * a.ldk + 8 * (vc ^ vswz(d));
  }
  auto issue = [&](AttnTile<D>& T, int kt0) {
    const bf16_t* kbase = Kb + (int64_t)kt0 * D;
    const bf16_t* vbase = Vb + kt0;
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      lds_dma16(kbase + koff[i], (lds_void*)(T.K + (4 * i + wv) * 512));
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      lds_dma16(vbase + voff[i], (lds_void*)(T.Vt + (4 * i + wv) * 512));
  };

  // first tile in flight while the Q fragments land (loads retire in order)
  if (kbeg < kend) {
    issue(smA, kbeg);
    PHYAI_WAIT_VMCNT(2 * NLD);
  } else {
    PHYAI_WAIT_VMCNT(0);
  }
  const bool wave_active = rt * kRows + wave * 32 < rows;
  const bool state0 = a.mask_mode == 1 && qtok[0] == 0;
  const bool state1 = a.mask_mode == 1 && qtok[1] == 0;

  f32x4 o[2][D / 16];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[c][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[2] = {-1e30f, -1e30f}, l_run[2] = {0.f, 0.f};
  const float sl2 = a.scale * 1.4426950408889634f;

  for (int kt0 = kbeg; kt0 < kend; kt0 += 2 * kKT) {
    // tile in A (next one into B)
    {
      const bool more = kt0 + kKT < kend;
      if (more) {
        issue(smB, kt0 + kKT);
        PHYAI_WAIT_VMCNT(2 * NLD);
      } else {
        PHYAI_WAIT_VMCNT(0);
      }
      lds_barrier();
      if (wave_active) attn_tile<D>(smA, qf, o, m_run, l_run, kt0, kend, plen, state0, state1, sl2, lc, lg);
      lds_barrier();
      if (!more) break;
    }
    // tile in B (next one into A)
    {
      const int kt1 = kt0 + kKT;
      const bool more = kt1 + kKT < kend;
      if (more) {
        issue(smA, kt1 + kKT);
        PHYAI_WAIT_VMCNT(2 * NLD);
      } else {
        PHYAI_WAIT_VMCNT(0);
      }
      lds_barrier();
      if (wave_active) attn_tile<D>(smB, qf, o, m_run, l_run, kt1, kend, plen, state0, state1, sl2, lc, lg);
      lds_barrier();
    }
  }

#pragma unroll
  for (int c = 0; c < 2; ++c) {
    l_run[c] += __shfl_xor(l_run[c], 16, kWave);
    l_run[c] += __shfl_xor(l_run[c], 32, kWave);
  }

  if (a.n_split == 1) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      if (!qv[c]) continue;
      const float inv = l_run[c] > 0.f ? 1.f / l_run[c] : 0.f;
      const int qhead = kvh * G + qr[c] % G;
      bf16_t* op = static_cast<bf16_t*>(a.out) + (int64_t)(b * a.M + qtok[c]) * a.ldo + qhead * D + 4 * lg;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        uint2 w;
        w.x = pack_bf16x2(o[c][dt][0] * inv, o[c][dt][1] * inv);
        w.y = pack_bf16x2(o[c][dt][2] * inv, o[c][dt][3] * inv);
        *reinterpret_cast<uint2*>(op + 16 * dt) = w;
      }
    }
    return;
  }

  // ---- split: write this block's partial (O normalised by its own l, as
  // bf16, plus m and l); attn_combine_kernel merges the splits
  const int64_t tile_id = (int64_t)grp * ntiles + rt;
  bf16_t* obase = reinterpret_cast<bf16_t*>(a.part) + tile_id * a.n_split * (int64_t)kRows * D;
  float* mlbase = a.part + (a.part_ml_off) + tile_id * a.n_split * (int64_t)kRows * 2;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int lrow = wave * 32 + c * 16 + lc;
    const float inv = l_run[c] > 0.f ? 1.f / l_run[c] : 0.f;
    bf16_t* op = obase + ((int64_t)split * kRows + lrow) * D + 4 * lg;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      uint2 w;
      w.x = pack_bf16x2(o[c][dt][0] * inv, o[c][dt][1] * inv);
      w.y = pack_bf16x2(o[c][dt][2] * inv, o[c][dt][3] * inv);
      *reinterpret_cast<uint2*>(op + 16 * dt) = w;
    }
    if (lg == 0) {
      mlbase[((int64_t)split * kRows + lrow) * 2] = m_run[c];
      mlbase[((int64_t)split * kRows + lrow) * 2 + 1] = l_run[c];
    }
  }
}

// Merge the key splits of one query row per wave: o = sum_s w_s o_s / sum_s w_s
// with w_s = l_s 2^(m_s - max m); every split's data is requested at once.
// Lane i merges elements 4i .. 4i+3 (lanes >= D/4 idle).
template <int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int G = a.nq / a.nkv;
  const int rows = a.M * G;
  const int ntiles = (rows + kRows - 1) / kRows;
  const int grp = blockIdx.y;
  const int r = blockIdx.x * 4 + wave;
  if (r >= rows || lane >= D / 4) return;
  const int b = grp / a.nkv, kvh = grp % a.nkv;
  const int rt = r / kRows, lrow = r % kRows;
  const int64_t tile_id = (int64_t)grp * ntiles + rt;
  const bf16_t* obase = reinterpret_cast<const bf16_t*>(a.part) + tile_id * a.n_split * (int64_t)kRows * D;
  const float* mlbase = a.part + a.part_ml_off + tile_id * a.n_split * (int64_t)kRows * 2;
  constexpr int SMAX = 16;
  float m[SMAX], l[SMAX];
  uint2 v[SMAX];
  float mmax = -1e30f;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    if (s < a.n_split) {
      const float* ml = mlbase + ((int64_t)s * kRows + lrow) * 2;
      m[s] = ml[0];
      l[s] = ml[1];
      v[s] = *reinterpret_cast<const uint2*>(obase + ((int64_t)s * kRows + lrow) * D + 4 * lane);
      mmax = fmaxf(mmax, m[s]);
    }
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  float lsum = 0.f;
#pragma unroll
  for (int s = 0; s < SMAX; ++s) {
    if (s < a.n_split) {
      const float w = l[s] * exp2f(m[s] - mmax);
      lsum += w;
      acc[0] += w * __uint_as_float(v[s].x << 16);
      acc[1] += w * __uint_as_float(v[s].x & 0xffff0000u);
      acc[2] += w * __uint_as_float(v[s].y << 16);
      acc[3] += w * __uint_as_float(v[s].y & 0xffff0000u);
    }
  }
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  const int tok = r / G, qhead = kvh * G + r % G;
  bf16_t* op = static_cast<bf16_t*>(a.out) + (int64_t)(b * a.M + tok) * a.ldo + qhead * D + 4 * lane;
  uint2 w;
  w.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  w.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  *reinterpret_cast<uint2*>(op) = w;
}

// fp32 path: one wave per (request, token, query head), keys one at a time.
template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  const int lane = threadIdx.x;
  const int row = blockIdx.x;                   // b*M + token
  const int h = blockIdx.y;
  const int b = row / a.M, tok = row % a.M;
  const int G = a.nq / a.nkv, kvh = h / G;
  const int plen = a.desc->prefix_len[b];
  const int n_keys = (a.keys_from_prefix ? plen : 0) + a.n_suffix;
  const float* q = static_cast<const float*>(a.q) + (int64_t)row * a.ldq + h * D;
  const float* Kb = static_cast<const float*>(a.K) + ((int64_t)b * a.nkv + kvh) * a.ldk * D;
  const float* Vb = static_cast<const float*>(a.Vt) + ((int64_t)b * a.nkv + kvh) * a.ldk * D;
  constexpr int PER = (D + 63) / 64;
  float qv[PER], acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = lane + 64 * i;
    qv[i] = d < D ? q[d] : 0.f;
    acc[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int kk = 0; kk < n_keys; ++kk) {
    if (a.mask_mode == 1 && !(kk <= plen || tok != 0)) continue;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int d = lane + 64 * i;
      if (d < D) s = fmaf(qv[i], Kb[(int64_t)kk * D + d], s);
    }
    s = wave_sum(s) * a.scale;
    const float mn = fmaxf(m, s);
    const float al = __expf(m - mn);
    const float p = __expf(s - mn);
    l = l * al + p;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int d = lane + 64 * i;
      acc[i] = acc[i] * al + (d < D ? p * Vb[(int64_t)d * a.ldk + kk] : 0.f);
    }
    m = mn;
  }
  float* op = static_cast<float*>(a.out) + (int64_t)row * a.ldo + h * D;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = lane + 64 * i;
    if (d < D) op[d] = l > 0.f ? acc[i] / l : 0.f;
  }
}

// Copy the caller's prefix K (row-major) and transpose its V into the
// library's key ranges, for every layer, request and kv head: keys
// 0 .. prefix_len[b]-1.  Block: 64 keys x D of one (layer, request, head).
template <typename T, int D>
__global__ __launch_bounds__(256) void prefix_relayout_kernel(RelayoutArgs r) {
  __shared__ T tile[64][D + 1];
  const int key0 = blockIdx.x * 64;
  const int grp = blockIdx.y;                  // b * nkv + kvh
  const int l = blockIdx.z;
  const int b = grp / r.nkv, kvh = grp % r.nkv;
  const int plen = r.desc->prefix_len[b];
  if (key0 >= plen && blockIdx.x != 0) return;
  const int W = r.nkv * D;
  const T* src = static_cast<const T*>(r.desc->prefix);
  const int64_t blk = (int64_t)r.B * r.P * W;
  const T* ks = src + ((int64_t)l * 2 + 0) * blk + (int64_t)b * r.P * W + kvh * D;
  const T* vs = src + ((int64_t)l * 2 + 1) * blk + (int64_t)b * r.P * W + kvh * D;
  T* kd = static_cast<T*>(r.K) + (int64_t)l * r.layer_stride + (int64_t)grp * r.ldk * D;
  T* vd = static_cast<T*>(r.Vt) + (int64_t)l * r.layer_stride + (int64_t)grp * r.ldk * D;
  if (blockIdx.x == 0) {
    // keys plen+n_suffix .. round-up to 64 are read as whole tiles: keep them zero
    const int t0 = plen + r.n_suffix, t1 = (t0 + 63) / 64 * 64;
    for (int i = threadIdx.x; i < (t1 - t0) * D; i += 256) {
      const int kr = t0 + i / D, c = i % D;
      kd[(int64_t)kr * D + c] = T(0);
      vd[(int64_t)c * r.ldk + kr] = T(0);
    }
  }
  const int nk = min(64, plen - key0);
  if (nk <= 0) return;
  for (int i = threadIdx.x; i < 64 * D; i += 256) {
    const int kr = i / D, c = i % D;
    if (kr < nk) {
      kd[(int64_t)(key0 + kr) * D + c] = ks[(int64_t)(key0 + kr) * W + c];
      tile[kr][c] = vs[(int64_t)(key0 + kr) * W + c];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 64 * D; i += 256) {
    const int c = i / 64, kr = i % 64;
    if (kr < nk) vd[(int64_t)c * r.ldk + key0 + kr] = tile[kr][c];
  }
}

}  // namespace

// Partials: bf16 O [tiles][split][kRows][D] followed (at part_ml_off floats)
// by float (m, l) [tiles][split][kRows][2].
int64_t attention_partial_ml_off(int B, int M, int nq, int nkv, int D, int n_split) {
  const int rows = M * (nq / nkv);
  const int64_t tiles = (int64_t)B * nkv * ((rows + kRows - 1) / kRows);
  return (tiles * n_split * kRows * D + 1) / 2;
}

int64_t attention_partial_floats(int B, int M, int nq, int nkv, int D, int n_split) {
  if (n_split <= 1) return 0;
  const int rows = M * (nq / nkv);
  const int64_t tiles = (int64_t)B * nkv * ((rows + kRows - 1) / kRows);
  return attention_partial_ml_off(B, M, nq, nkv, D, n_split) + tiles * n_split * kRows * 2;
}

int64_t attention_counters(int B, int M, int nq, int nkv) {
  const int rows = M * (nq / nkv);
  return (int64_t)B * nkv * ((rows + kRows - 1) / kRows);
}

void attention_bf16(const AttnArgs& a0, hipStream_t s) {
  AttnArgs a = a0;
  const int rows = a.M * (a.nq / a.nkv);
  const int ntiles = (rows + kRows - 1) / kRows;
  const int ngroups = a.B * a.nkv * a.n_split;
  a.part_ml_off = attention_partial_ml_off(a.B, a.M, a.nq, a.nkv, a.D, a.n_split);
  dim3 grid(8 * ntiles * ((ngroups + 7) / 8));
  if (a.D == 256) hipLaunchKernelGGL(attn_mfma_kernel<256>, grid, dim3(256), 0, s, a);
  else if (a.D == 128) hipLaunchKernelGGL(attn_mfma_kernel<128>, grid, dim3(256), 0, s, a);
  else if (a.D == 64) hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(256), 0, s, a);
  if (a.n_split > 1) {
    dim3 g2((rows + 3) / 4, a.B * a.nkv);
    if (a.D == 256) hipLaunchKernelGGL(attn_combine_kernel<256>, g2, dim3(256), 0, s, a);
    else if (a.D == 128) hipLaunchKernelGGL(attn_combine_kernel<128>, g2, dim3(256), 0, s, a);
    else if (a.D == 64) hipLaunchKernelGGL(attn_combine_kernel<64>, g2, dim3(256), 0, s, a);
  }
}

void attention_f32(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.B * a.M, a.nq);
  if (a.D == 64) hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
  else if (a.D == 128) hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
  else if (a.D == 256) hipLaunchKernelGGL(attn_f32_kernel<256>, grid, dim3(64), 0, s, a);
}

template <typename T>
static void relayout_t(const RelayoutArgs& r, hipStream_t s) {
  dim3 grid((r.P + 63) / 64, r.B * r.nkv, r.L);
  if (r.D == 256) hipLaunchKernelGGL((prefix_relayout_kernel<T, 256>), grid, dim3(256), 0, s, r);
  else if (r.D == 128) hipLaunchKernelGGL((prefix_relayout_kernel<T, 128>), grid, dim3(256), 0, s, r);
  else if (r.D == 64) hipLaunchKernelGGL((prefix_relayout_kernel<T, 64>), grid, dim3(256), 0, s, r);
}

void prefix_relayout_bf16(const RelayoutArgs& r, hipStream_t s) { relayout_t<bf16_t>(r, s); }
void prefix_relayout_f32(const RelayoutArgs& r, hipStream_t s) { relayout_t<float>(r, s); }

}  // namespace phyai
