// Suffix-query attention over the frozen prefix K/V and the suffix tokens'
// own K/V, with online softmax and an optional split over the keys.  The
// shape is the one the paper profiles for the action expert (section PhyAI
// Architecture, paragraph Profiled operator selection): some fifty suffix
// queries per head over a prefix of several hundred keys, head_dim 256.
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
// MFMA formulation: S^T = K Q^T and O^T = V^T P^T on 32x32x16 bf16 MFMAs,
// so a query is always the MFMA column (lane % 32): its softmax statistics
// live in lanes l and l^32 (one cross-lane step), and the probabilities
// leave the S^T accumulators already laid out as the B operand of the P.V
// product (the key order inside a tile is permuted identically on both
// operands).  The 32x32 shape issues half as many MFMA instructions per flop
// as 16x16, which is what a single wave per SIMD needs to keep the matrix
// core busy.
//
// Block: 4 waves x 32 query rows (2 waves for a batch-1-sized suffix, see
// attention_rows_per_block); 64-key tiles double-buffered in LDS and filled
// by direct global->LDS loads, the next tile in flight while the current one
// is computed.
// With n_split > 1 the key range is split over blocks, whose partials a
// second kernel merges in a fixed order.
#include "kernels.hpp"

#include <algorithm>
#include <cstdlib>
#include <type_traits>

namespace phyai {

namespace {

constexpr int kKT = 64;          // keys per tile

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

// MFMA formulation (32x32x16 bf16): S^T = K Q^T and O^T = V^T P^T.  A wave
// owns 32 query rows, one per MFMA column (lane % 32), so each lane keeps the
// softmax state of one query; lanes l and l^32 share it.
//
// Key order inside a tile.  The S^T MFMA of key block kb (0, 1: 32 keys
// each) reads its A-operand (K) row i = 8u + 4h + w (u < 4, h < 2, w < 4) from
// key 32kb + 16(u/2) + 8h + 4(u%2) + w.  Accumulator v = 8t + j of lane l
// (h = l/32) then holds key 32kb + 16t + 8h + j: the 8 consecutive keys that
// lane supplies as the k-slice of the P.V MFMA for key step 2kb + t.  So P
// needs no shuffle and each V^T fragment is one 16-byte LDS read.
__device__ __forceinline__ int perm_row(int i) {
  const int u = i >> 3, h = (i >> 2) & 1, w = i & 3;
  return 16 * (u >> 1) + 8 * h + 4 * (u & 1) + w;
}

// LDS tiles, 16-byte chunks XOR-swizzled so that the MFMA fragment reads of
// 16 lanes fall in 16 different bank groups (a 16-lane group reads 16
// consecutive keys (K) or 16 consecutive d (V^T) at one chunk):
//   K  [64 keys][D]:   chunk c of key row r sits at position c ^ kswz(r)
//   Vt [D][64 keys]:   chunk c of row d sits at position c ^ ((d >> 1) & 7)
//
// The two tile buffers are laid out [K0 | K1 | Vt0 | Vt1]: a fragment read of
// buffer 1 is then the same per-lane address as buffer 0's plus a constant
// that fits the LDS instruction's 16-bit offset, so one set of per-lane
// addresses serves both buffers (at D = 256 each array is 32 KiB).
template <int D>
struct AttnLds {
  bf16_t K[2][kKT * D];
  bf16_t Vt[2][D * kKT];
};

// D >= 128: a chunk's bank group is its position mod 16; D == 64: two rows
// share 256 bytes, the row's low bit separates them.
template <int D>
__device__ __forceinline__ int kswz(int r) { return D >= 128 ? (r & 15) : ((r >> 1) & 7); }
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 7; }

// max(a, b, c) as one v_max3_f32.  fmaxf makes the compiler quiet each input
// first (one extra instruction per operand); the scores reduced here are
// never NaN (masked keys are -inf, padding keys are zero), so that step is
// not needed.
__device__ __forceinline__ float max3_f32(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// The value of lane l ^ 32 combined with this lane's (gfx950 permlane32
// swap: the two results are this lane's and its partner's value).
__device__ __forceinline__ float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
  return max3_f32(a, b, b);
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS fragment reads issued this many MFMAs ahead of their use
constexpr int kReadAhead = 4;

// Instruction order of one MFMA loop of n products whose operands come from
// LDS: the first pd fragment reads, then each MFMA followed by the next read,
// so every read is issued pd MFMAs (32 cycles each) before its use.  With one
// wave per SIMD nothing else hides LDS latency, and left to itself the
// compiler keeps only two reads in flight.
template <int N, int PD>
__device__ __forceinline__ void lds_mfma_pipeline() {
#pragma unroll
  for (int i = 0; i < PD; ++i) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // DS read
#pragma unroll
  for (int i = 0; i < N - PD; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
#pragma unroll
  for (int i = 0; i < PD; ++i) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
}

// One 64-key tile of the online-softmax attention for the wave's 32 query
// rows, reading K and V^T from the LDS tile (TK, TVt).
template <int D>
__device__ __forceinline__ void attn_tile(const bf16_t* TK, const bf16_t* TVt, const bf16x8 (&qf)[D / 16], f32x16 (&o)[D / 32],
                                          float& m_run, float& l_run, int kt0, int kend, int plen, bool state_q,
                                          float sl2, int lr, int hl, bool first) {
  // S^T of the two 32-key blocks as two interleaved accumulator chains
  f32x16 st[2];
#pragma unroll
  for (int v = 0; v < 16; ++v) { st[0][v] = 0.f; st[1][v] = 0.f; }
  const int r0 = perm_row(lr), r1 = 32 + r0;
  bf16x8 kf[2][D / 16];
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    kf[0][s] = *reinterpret_cast<const bf16x8*>(TK + r0 * D + 8 * ((2 * s + hl) ^ kswz<D>(r0)));
    kf[1][s] = *reinterpret_cast<const bf16x8*>(TK + r1 * D + 8 * ((2 * s + hl) ^ kswz<D>(r1)));
  }
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    st[0] = mfma32x32x16(kf[0][s], qf[s], st[0]);
    st[1] = mfma32x32x16(kf[1][s], qf[s], st[1]);
  }
  lds_mfma_pipeline<D / 8, kReadAhead>();
  // Scores are masked only where a mask can bite: the tile holding the end
  // of the key range, and for state-token queries the tiles that reach past
  // the prefix (wave-uniform test; a state-token row shares its wave with
  // action rows, and the whole block waits for its slowest wave at every
  // tile).  The scale (> 0) is applied after the max, inside the exponent.
  const bool need_mask = !(kt0 + kKT <= kend) || (state_q && kt0 + kKT - 1 > plen);
  if (__ballot(need_mask)) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = kt0 + 32 * kb + 16 * (v >> 3) + 8 * hl + (v & 7);
        const bool ok = key < kend && (!state_q || key <= plen);
        st[kb][v] = ok ? st[kb][v] : -INFINITY;
      }
  }
  // tile max: four independent v_max3 chains over the 32 scores, then merged
  float mx[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const f32x16& a = st[c >> 1];
    const int o = 8 * (c & 1);
    float m = max3_f32(a[o], a[o + 1], a[o + 2]);
    m = max3_f32(m, a[o + 3], a[o + 4]);
    m = max3_f32(m, a[o + 5], a[o + 6]);
    mx[c] = max3_f32(m, a[o + 7], a[o + 7]);
  }
  const float tmax = pair_max(max3_f32(mx[0], mx[1], max3_f32(mx[2], mx[3], mx[3]))) * sl2;
  // Lazy rescaling: the running reference m only moves when the tile max
  // exceeds it by more than 8 (log2 units), so exp2(s - m) <= 256 and the
  // accumulators are rescaled only a few times per key range.
  // On the block's first tile nothing has been accumulated yet (o and l are
  // zero), so only the reference moves.
  if (__ballot(tmax > m_run + 8.f)) {
    const float m_new = fmaxf(m_run, tmax);
    if (!first) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < D / 32; ++i) o[i] *= alpha;
    }
    m_run = m_new;
  }
  // P^T fragment of key step t (0..3): keys 16t + 8h + j = accumulator
  // 8(t%2) + j of key block t/2
  bf16x8 pf[4];
  float ps[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float pv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) pv[j] = __builtin_amdgcn_exp2f(fmaf(st[t >> 1][8 * (t & 1) + j], sl2, -m_run));
    ps[t] = ((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7]));
    uint4 w;
    w.x = pack_bf16x2(pv[0], pv[1]);
    w.y = pack_bf16x2(pv[2], pv[3]);
    w.z = pack_bf16x2(pv[4], pv[5]);
    w.w = pack_bf16x2(pv[6], pv[7]);
    pf[t] = as_bf16x8(w);
  }
  l_run += (ps[0] + ps[1]) + (ps[2] + ps[3]);
  // O^T += V^T P^T: V^T fragment (d-block db, key step t) = row d = 32 db + lr,
  // keys 16t + 8h .. +7, one 16-byte read; consecutive MFMAs go to different
  // d-blocks
  bf16x8 vf[4][D / 32];
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int d = 32 * db + lr;
      vf[t][db] = *reinterpret_cast<const bf16x8*>(TVt + d * kKT + 8 * ((2 * t + hl) ^ vswz(d)));
    }
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int db = 0; db < D / 32; ++db) o[db] = mfma32x32x16(vf[t][db], pf[t], o[db]);
  lds_mfma_pipeline<D / 8, kReadAhead>();
}

template <int D, int NWB>
__global__ __launch_bounds__(64 * NWB) void attn_mfma_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) AttnLds<D> sm;
  constexpr int kRows = 32 * NWB;             // query rows per block
  constexpr int CPR = D / 8;                  // 16-byte chunks per K row
  constexpr int NLD = kKT * D / 8 / (64 * NWB);   // loads per thread per operand per tile
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int lr = lane % 32, hl = lane / 32;
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

  // this lane's query row: B operand of S^T, Q[row][16s + 8h .. +7]; requested
  // before the prefix length, whose load the key range and the tile loads wait on
  const int qr = rt * kRows + wave * 32 + lr;
  const bool qv = qr < rows;
  const int qtok = qv ? qr / G : 0;
  const int qhead = kvh * G + (qv ? qr % G : 0);
  bf16x8 qf[D / 16];
  {
    const bf16_t* qp = static_cast<const bf16_t*>(a.q) + (int64_t)(b * a.M + qtok) * a.ldq + qhead * D + 8 * hl;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qv) v = *reinterpret_cast<const uint4*>(qp + 16 * s);
      qf[s] = as_bf16x8(v);
    }
  }
  const int plen = a.desc->prefix_len[b];
  const int n_keys = (a.keys_from_prefix ? plen : 0) + a.n_suffix;
  int chunk = (n_keys + a.n_split - 1) / a.n_split;
  chunk = (chunk + kKT - 1) / kKT * kKT;
  const int kbeg = split * chunk;
  const int kend = min(n_keys, kbeg + chunk);

  const bf16_t* Kb = static_cast<const bf16_t*>(a.K) + (int64_t)grp * a.ldk * D;
  const bf16_t* Vb = static_cast<const bf16_t*>(a.Vt) + (int64_t)grp * a.ldk * D;

  // Direct global->LDS loads of one tile (the key range always holds whole,
  // finite 64-key tiles).  Wave w's i-th load fills 1 KiB block NWB i + w;
  // the per-thread source offsets (elements) do not depend on the tile.
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  int koff[NLD], voff[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int pos = (NWB * i + wave) * 64 + lane;
    const int r = pos / CPR, pc = pos % CPR;
    koff[i] = r * D + 8 * (pc ^ kswz<D>(r));
    const int d = pos / 8, vc = pos % 8;
    voff[i] = d * a.ldk + 8 * (vc ^ vswz(d));
  }
  auto issue = [&](int buf, int kt0) {
    const bf16_t* kbase = Kb + (int64_t)kt0 * D;
    const bf16_t* vbase = Vb + kt0;
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      lds_dma16(kbase + koff[i], (lds_void*)(sm.K[buf] + (NWB * i + wv) * 512));
#pragma unroll
    for (int i = 0; i < NLD; ++i)
      lds_dma16(vbase + voff[i], (lds_void*)(sm.Vt[buf] + (NWB * i + wv) * 512));
  };

  // first tile in flight while the Q fragments land.  The first tile's
  // compute needs both, and a full wait here is also what tells the compiler
  // that the Q fragments are complete: it cannot count the asm tile loads,
  // so after a partial wait it would put a full wait in front of the first
  // MFMA of every tile, stalling each tile on the prefetch of the next.
  if (kbeg < kend) issue(0, kbeg);
  PHYAI_WAIT_VMCNT(0);
  const bool wave_active = rt * kRows + wave * 32 < rows;
  const bool state_q = a.mask_mode == 1 && qtok == 0;

  f32x16 o[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[i][v] = 0.f;
  float m_run = -1e30f, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;

  for (int kt0 = kbeg; kt0 < kend; kt0 += 2 * kKT) {
    // tile in A (next one into B)
    {
      const bool more = kt0 + kKT < kend;
      if (more) {
        issue(1, kt0 + kKT);
        PHYAI_WAIT_VMCNT(2 * NLD);
      } else {
        PHYAI_WAIT_VMCNT(0);
      }
      lds_barrier();
      if (wave_active) attn_tile<D>(sm.K[0], sm.Vt[0], qf, o, m_run, l_run, kt0, kend, plen, state_q, sl2, lr, hl, kt0 == kbeg);
      lds_barrier();
      if (!more) break;
    }
    // tile in B (next one into A)
    {
      const int kt1 = kt0 + kKT;
      const bool more = kt1 + kKT < kend;
      if (more) {
        issue(0, kt1 + kKT);
        PHYAI_WAIT_VMCNT(2 * NLD);
      } else {
        PHYAI_WAIT_VMCNT(0);
      }
      lds_barrier();
      if (wave_active) attn_tile<D>(sm.K[1], sm.Vt[1], qf, o, m_run, l_run, kt1, kend, plen, state_q, sl2, lr, hl, false);
      lds_barrier();
    }
  }

  // lanes l and l^32 hold the same query over different keys
  l_run = pair_sum(l_run);

  // Output rows (final, or this split's partial normalised by its own l),
  // bf16.  Accumulator v of o[db] holds d = 32 db + 8(v/4) + 4h + v%4, so a
  // store straight from registers would write 16 bytes into each of 32 rows.
  // Each wave instead stages its 32 x D rows in LDS (the tiles are free once
  // the last barrier of the loop has passed; 16-byte chunk c of row r sits at
  // c ^ (r mod CPR)) and writes whole rows: every store instruction then
  // covers 64 / CPR complete rows.
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
  bf16_t* stage = reinterpret_cast<bf16_t*>(&sm) + wave * 32 * D;
  static_assert(sizeof(AttnLds<D>) >= NWB * 32 * D * sizeof(bf16_t), "staging needs NWB waves x 32 rows");
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint2 w;
      w.x = pack_bf16x2(o[db][4 * u + 0] * inv, o[db][4 * u + 1] * inv);
      w.y = pack_bf16x2(o[db][4 * u + 2] * inv, o[db][4 * u + 3] * inv);
      const int c = 4 * db + u;
      *reinterpret_cast<uint2*>(stage + lr * D + 8 * (c ^ (lr & (CPR - 1))) + 4 * hl) = w;
    }
  // the rows are read back by other lanes of the same wave; LDS operations of
  // one wave complete in order
  __builtin_amdgcn_s_waitcnt(0xC07F);
  constexpr int RPI = kWave / CPR;            // rows per store instruction
  const int sr = lane / CPR, sc = lane % CPR;
  const int64_t tile_id = (int64_t)grp * ntiles + rt;
  bf16_t* obase = reinterpret_cast<bf16_t*>(a.part) + (tile_id * a.n_split + split) * (int64_t)kRows * D;
#pragma unroll
  for (int i = 0; i < 32 / RPI; ++i) {
    const int r = RPI * i + sr;               // row within the wave
    const uint4 w = *reinterpret_cast<const uint4*>(stage + r * D + 8 * (sc ^ (r & (CPR - 1))));
    const int qrow = rt * kRows + wave * 32 + r;
    if (a.n_split == 1) {
      if (qrow < rows) {
        const int tok = qrow / G, head = kvh * G + qrow % G;
        *reinterpret_cast<uint4*>(static_cast<bf16_t*>(a.out) + (int64_t)(b * a.M + tok) * a.ldo + head * D +
                                  8 * sc) = w;
      }
    } else {
      // rows past the tile's queries are written too (never merged)
      *reinterpret_cast<uint4*>(obase + (int64_t)(wave * 32 + r) * D + 8 * sc) = w;
    }
  }
  if (a.n_split > 1 && hl == 0 && qv) {
    float* mlbase = a.part + a.part_ml_off + tile_id * a.n_split * (int64_t)kRows * 2;
    *reinterpret_cast<float2*>(mlbase + ((int64_t)split * kRows + wave * 32 + lr) * 2) = make_float2(m_run, l_run);
  }
}

// Merge the key splits of one query row per wave: o = sum_s w_s o_s / sum_s w_s
// with w_s = l_s 2^(m_s - max m).  Lane i merges elements 4i .. 4i+3 (lanes
// >= D/4 idle).  All NS slots are loaded unconditionally (slots past
// n_split re-read the last split and get weight 0), so every load is in
// flight at once instead of one round trip per split.
template <int D, int NS>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int G = a.nq / a.nkv;
  const int rows = a.M * G;
  const int kRows = a.rows_per_tile;
  const int ntiles = (rows + kRows - 1) / kRows;
  const int grp = blockIdx.y;
  const int r = blockIdx.x * 4 + wave;
  if (r >= rows || lane >= D / 4) return;
  const int b = grp / a.nkv, kvh = grp % a.nkv;
  const int rt = r / kRows, lrow = r % kRows;
  const int64_t tile_id = (int64_t)grp * ntiles + rt;
  const bf16_t* obase = reinterpret_cast<const bf16_t*>(a.part) + tile_id * a.n_split * (int64_t)kRows * D;
  const float* mlbase = a.part + a.part_ml_off + tile_id * a.n_split * (int64_t)kRows * 2;
  const int n = a.n_split;
  float2 ml[NS];
  uint2 v[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int se = s < n ? s : n - 1;
    ml[s] = *reinterpret_cast<const float2*>(mlbase + ((int64_t)se * kRows + lrow) * 2);
    v[s] = *reinterpret_cast<const uint2*>(obase + ((int64_t)se * kRows + lrow) * D + 4 * lane);
  }
  float mmax = -1e30f;
#pragma unroll
  for (int s = 0; s < NS; ++s) mmax = fmaxf(mmax, s < n ? ml[s].x : -1e30f);
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  float lsum = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float w = s < n ? ml[s].y * __builtin_amdgcn_exp2f(ml[s].x - mmax) : 0.f;
    lsum += w;
    acc[0] = fmaf(w, __uint_as_float(v[s].x << 16), acc[0]);
    acc[1] = fmaf(w, __uint_as_float(v[s].x & 0xffff0000u), acc[1]);
    acc[2] = fmaf(w, __uint_as_float(v[s].y << 16), acc[2]);
    acc[3] = fmaf(w, __uint_as_float(v[s].y & 0xffff0000u), acc[3]);
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
// Moves are 16 bytes wide (the caller's buffer permitting): K rows are copied
// directly; V rows go through an LDS tile (rows padded by 16 bytes, which
// keeps them aligned and spreads a column over the banks) and leave as runs
// of consecutive keys of one V^T row.
template <typename T, int D>
__global__ __launch_bounds__(256) void prefix_relayout_kernel(RelayoutArgs r) {
  constexpr int VE = 16 / sizeof(T);           // elements per 16-byte move
  __shared__ __attribute__((aligned(16))) T tile[64][D + VE];
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
  // the library's ranges are allocated aligned; the caller's rows are 16-byte
  // multiples apart, so its base decides
  const bool vec = (reinterpret_cast<uintptr_t>(src) & 15) == 0;
  constexpr int CPR = D / VE;                  // 16-byte chunks per key row
  for (int i = threadIdx.x; i < 64 * CPR; i += 256) {
    const int kr = i / CPR, c = (i % CPR) * VE;
    const int64_t so = (int64_t)(key0 + kr) * W + c;
    if (kr < nk) {
      if (vec) {
        *reinterpret_cast<uint4*>(kd + (int64_t)(key0 + kr) * D + c) = *reinterpret_cast<const uint4*>(ks + so);
        *reinterpret_cast<uint4*>(&tile[kr][c]) = *reinterpret_cast<const uint4*>(vs + so);
      } else {
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          kd[(int64_t)(key0 + kr) * D + c + e] = ks[so + e];
          tile[kr][c + e] = vs[so + e];
        }
      }
    }
  }
  __syncthreads();
  constexpr int KC = 64 / VE;                  // 16-byte runs per V^T row of the tile
  for (int i = threadIdx.x; i < D * KC; i += 256) {
    const int d = i / KC, k = (i % KC) * VE;
    T* dst = vd + (int64_t)d * r.ldk + key0 + k;
    if (k + VE <= nk) {
      __attribute__((aligned(16))) T run[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) run[e] = tile[k + e][d];
      *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(run);
    } else {
      for (int e = 0; k + e < nk; ++e) dst[e] = tile[k + e][d];
    }
  }
}

// The prefix LM's keys and values of one layer back into the caller's prefix
// layout, the inverse of prefix_relayout_kernel.  Block: 64 keys x D of one
// (request, kv head).  The V^T tile comes into LDS as 16-byte runs along the
// keys (the key range holds whole 64-key tiles) and leaves as rows; K rows
// are copied; keys at or beyond prefix_len[b] (up to P) leave as zeros.
template <typename T, int D>
__global__ __launch_bounds__(256) void kv_export_kernel(KvExportArgs r) {
  constexpr int VE = 16 / sizeof(T);           // elements per 16-byte move
  constexpr int KC = 64 / VE;                  // 16-byte runs per V^T row of the tile
  constexpr int CPR = D / VE;                  // 16-byte chunks per key row
  __shared__ __attribute__((aligned(16))) T tile[D][64 + VE];
  const int key0 = blockIdx.x * 64;
  const int grp = blockIdx.y;                  // b * nkv + kvh
  const int b = grp / r.nkv, kvh = grp % r.nkv;
  const int plen = r.desc->prefix_len[b];
  const int W = r.nkv * D;
  const T* ks = static_cast<const T*>(r.K) + (int64_t)grp * r.ldk * D;
  const T* vs = static_cast<const T*>(r.Vt) + (int64_t)grp * r.ldk * D;
  T* ko = static_cast<T*>(r.out) + (int64_t)b * r.P * W + kvh * D;
  T* vo = ko + r.half;
  for (int i = threadIdx.x; i < D * KC; i += 256) {
    const int d = i / KC, k = (i % KC) * VE;
    *reinterpret_cast<uint4*>(&tile[d][k]) = *reinterpret_cast<const uint4*>(vs + (int64_t)d * r.ldk + key0 + k);
  }
  __syncthreads();
  const int nk = min(64, r.P - key0);
  for (int i = threadIdx.x; i < 64 * CPR; i += 256) {
    const int kr = i / CPR, c = (i % CPR) * VE;
    if (kr >= nk) continue;
    const int key = key0 + kr;
    uint4 kw = make_uint4(0, 0, 0, 0), vw = make_uint4(0, 0, 0, 0);
    if (key < plen) {
      kw = *reinterpret_cast<const uint4*>(ks + (int64_t)key * D + c);
      __attribute__((aligned(16))) T run[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) run[e] = tile[c + e][kr];
      vw = *reinterpret_cast<const uint4*>(run);
    }
    *reinterpret_cast<uint4*>(ko + (int64_t)key * W + c) = kw;
    *reinterpret_cast<uint4*>(vo + (int64_t)key * W + c) = vw;
  }
}

}  // namespace

// Query rows per block: 128 (4 waves), or 64 (2 waves) when the 128-row
// blocks of all requests number fewer than 64 (batch 1) and a request has a
// suffix-sized query count, so that with the key splits the kernel spreads
// over more CUs and each block loads half the queries and stores half the
// partials.  A prefix LM's self-attention (thousands of query rows per
// request) keeps 128 rows: there four waves share each key tile (batch-1
// prefix of 816 tokens: 63 -> 34 us per launch).  PHYAI_ATTN_ROWS=64|128
// (tests, read at enqueue time) forces it.
int attention_rows_per_block(int B, int rows, int nkv) {
  const char* f = getenv("PHYAI_ATTN_ROWS");
  if (f) return atoi(f) == 64 ? 64 : 128;
  return rows <= 1024 && (int64_t)((rows + 127) / 128) * B * nkv < 64 ? 64 : 128;
}

// Partials: bf16 O [tiles][split][rows_per_block][D] followed (at part_ml_off
// floats) by float (m, l) [tiles][split][rows_per_block][2].  The buffer is
// sized for the larger of the 64- and 128-row layouts, so that forcing either
// fits.
int64_t attention_partial_ml_off(int B, int M, int nq, int nkv, int D, int n_split) {
  const int rows = M * (nq / nkv);
  const int rpt = attention_rows_per_block(B, rows, nkv);
  const int64_t tiles = (int64_t)B * nkv * ((rows + rpt - 1) / rpt);
  return (tiles * n_split * rpt * D + 1) / 2;
}

int64_t attention_partial_floats(int B, int M, int nq, int nkv, int D, int n_split) {
  if (n_split <= 1) return 0;
  const int rows = M * (nq / nkv);
  int64_t most = 0;
  for (int rpt = 64; rpt <= 128; rpt += 64) {
    const int64_t tiles = (int64_t)B * nkv * ((rows + rpt - 1) / rpt);
    most = std::max(most, (tiles * n_split * rpt * D + 1) / 2 + tiles * n_split * rpt * 2);
  }
  return most;
}

AttnParts attention_parts(const AttnArgs& a) {
  AttnParts p{};
  p.o = reinterpret_cast<const bf16_t*>(a.part);
  p.ml = a.part + attention_partial_ml_off(a.B, a.M, a.nq, a.nkv, a.D, a.n_split);
  p.n_split = a.n_split;
  p.G = a.nq / a.nkv;
  p.rows_per_tile = attention_rows_per_block(a.B, a.M * p.G, a.nkv);
  p.ntiles = (a.M * p.G + p.rows_per_tile - 1) / p.rows_per_tile;
  p.M = a.M;
  p.nkv = a.nkv;
  p.D = a.D;
  return p;
}

void attention_bf16(const AttnArgs& a0, hipStream_t s) {
  AttnArgs a = a0;
  const int rows = a.M * (a.nq / a.nkv);
  a.rows_per_tile = attention_rows_per_block(a.B, rows, a.nkv);
  const int ntiles = (rows + a.rows_per_tile - 1) / a.rows_per_tile;
  const int ngroups = a.B * a.nkv * a.n_split;
  a.part_ml_off = attention_partial_ml_off(a.B, a.M, a.nq, a.nkv, a.D, a.n_split);
  dim3 grid(8 * ntiles * ((ngroups + 7) / 8));
  auto go = [&](auto dtag) {
    constexpr int DD = decltype(dtag)::value;
    if (a.rows_per_tile == 64) hipLaunchKernelGGL((attn_mfma_kernel<DD, 2>), grid, dim3(128), 0, s, a);
    else hipLaunchKernelGGL((attn_mfma_kernel<DD, 4>), grid, dim3(256), 0, s, a);
  };
  if (a.D == 256) go(std::integral_constant<int, 256>{});
  else if (a.D == 128) go(std::integral_constant<int, 128>{});
  else if (a.D == 64) go(std::integral_constant<int, 64>{});
  if (a.n_split > 1 && !a.defer_merge) {
    dim3 g2((rows + 3) / 4, a.B * a.nkv);
    auto comb = [&](auto dtag) {
      constexpr int DD = decltype(dtag)::value;
      if (a.n_split <= 4) hipLaunchKernelGGL((attn_combine_kernel<DD, 4>), g2, dim3(256), 0, s, a);
      else if (a.n_split <= 8) hipLaunchKernelGGL((attn_combine_kernel<DD, 8>), g2, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((attn_combine_kernel<DD, 16>), g2, dim3(256), 0, s, a);
    };
    if (a.D == 256) comb(std::integral_constant<int, 256>{});
    else if (a.D == 128) comb(std::integral_constant<int, 128>{});
    else if (a.D == 64) comb(std::integral_constant<int, 64>{});
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

template <typename T>
static void kv_export_t(const KvExportArgs& r, hipStream_t s) {
  if (r.P <= 0 || r.B <= 0) return;
  dim3 grid((r.P + 63) / 64, r.B * r.nkv);
  if (r.D == 256) hipLaunchKernelGGL((kv_export_kernel<T, 256>), grid, dim3(256), 0, s, r);
  else if (r.D == 128) hipLaunchKernelGGL((kv_export_kernel<T, 128>), grid, dim3(256), 0, s, r);
  else if (r.D == 64) hipLaunchKernelGGL((kv_export_kernel<T, 64>), grid, dim3(256), 0, s, r);
}

void kv_export_bf16(const KvExportArgs& r, hipStream_t s) { kv_export_t<bf16_t>(r, s); }
void kv_export_f32(const KvExportArgs& r, hipStream_t s) { kv_export_t<float>(r, s); }

}  // namespace phyai
