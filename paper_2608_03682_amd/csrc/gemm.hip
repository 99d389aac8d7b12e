// Weight-streaming GEMMs with fused epilogues (bf16 / fp8-weight MFMA, and a
// plain fp32 path).
//
// Packed weight order (built on the host): for pair tile p, k-block kb of 64
// and half hf, 64 lanes each hold the operand fragment of two MFMA k-steps:
//   bf16: 32 bytes per lane, k = 64kb + 32s + 8(l/16) + j   (s = 0, 1; j < 8)
//   fp8 : 16 bytes per lane, same k order, one byte per value
// for packed column 32p + 16hf + l%16.  A wave streaming one pair tile along
// K therefore reads whole contiguous 2 KiB (bf16) / 1 KiB (fp8) blocks.
#include "kernels.hpp"

#include <cstdlib>
#include <cstring>
#include <type_traits>

namespace phyai {

namespace {

constexpr int kMT = 4;           // 16-row MFMA tiles per block (64 rows)

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef const __attribute__((address_space(1))) u32x4_t gu32x4_t;

// 16-, 8- and 2-byte loads through a global (not generic) pointer, which the
// compiler counts with vmcnt alone
__device__ __forceinline__ u32x4_t gload16(const void* p) { return *(gu32x4_t*)(p); }
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32x2_t gload8(const void* p) {
  return *(const __attribute__((address_space(1))) u32x2_t*)(p);
}
__device__ __forceinline__ uint32_t gload2(const void* p) {
  return *(const __attribute__((address_space(1))) uint16_t*)(p);
}

// The two 8-value k-steps of lane `lane`'s weight fragment (pair tile p,
// k-block kb, half hf) as bf16 MFMA operands, for the stored weight kinds:
//   bf16: 32 bytes per lane; fp8: 16 bytes per lane, decoded with a unit
//   scale (the column scale is applied to the result); fp4: 8 bytes per
//   lane (4 per k-step) plus one E8M0 exponent per (column, k-step), the
//   32-row group the step covers.
template <int WK>
__device__ __forceinline__ void load_wfrag(const GemmArgs& g, int p, int nkb, int kb, int hf, int lane, bf16x8 (&b)[2]) {
  const int64_t frag = ((int64_t)(p * nkb + kb) * 2 + hf) * kWave + lane;
  if constexpr (WK == W_FP8) {
    const u32x4_t v = gload16(static_cast<const uint4*>(g.W) + frag);
    b[0] = fp8x8_to_bf16x8(v.x, v.y);
    b[1] = fp8x8_to_bf16x8(v.z, v.w);
  } else if constexpr (WK == W_FP4) {
    const u32x2_t v = gload8(static_cast<const uint2*>(g.W) + frag);
    const uint32_t ex = gload2(g.mx + ((int64_t)(p * nkb + kb) * 2 + hf) * 32 + 2 * (lane % 16));
    b[0] = fp4x8_to_bf16x8(v.x, e8m0_to_f32(ex & 0xff));
    b[1] = fp4x8_to_bf16x8(v.y, e8m0_to_f32(ex >> 8));
  } else {
    const uint4* src = static_cast<const uint4*>(g.W) + frag * 2;
    b[0] = __builtin_bit_cast(bf16x8, gload16(src));
    b[1] = __builtin_bit_cast(bf16x8, gload16(src + 1));
  }
}

// One trip of the small-row GEMM: U k-blocks starting at kb, every operand
// load issued (as global loads, so that the compiler can count them) before
// the first MFMA; `hook` runs between the loads and the MFMAs.  Columns past
// N re-read the last pair tile.
template <int U, int WK, bool SPLIT, int NT, int MT, class Hook>
__device__ __forceinline__ void b1_trip(const GemmArgs& g, int pt0, int nkb, int lane, int kb,
                                        const bf16_t* const (&arp)[MT], const bf16_t* const (&alp)[MT],
                                        f32x4 (&acc)[MT][NT], const Hook& hook) {
  bf16x8 b[U][NT][2];
  bf16x8 a[U][MT][2], al[U][MT][2];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int kk = kb + u;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int p = min(pt0 + t / 2, g.NPT - 1), hf = t % 2;
      load_wfrag<WK>(g, p, nkb, kk, hf, lane, b[u][t]);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        a[u][mt][s] = __builtin_bit_cast(bf16x8, gload16(arp[mt] + kk * 64 + s * 32));
        if (SPLIT) al[u][mt][s] = __builtin_bit_cast(bf16x8, gload16(alp[mt] + kk * 64 + s * 32));
      }
  }
  hook();
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          acc[mt][t] = mfma16x16x32(a[u][mt][s], b[u][t][s], acc[mt][t]);
          if (SPLIT) acc[mt][t] = mfma16x16x32(al[u][mt][s], b[u][t][s], acc[mt][t]);
        }
}

// Finishing of a split-K residual tile: rows r0 .. r0 + nr - 1, columns c0 ..
// c0 + nc - 1 (nc a multiple of 32) of an output whose S blocks each stored
// one slice with device-scope stores.  Called by every thread of an
// NTHR-thread block after its own partial stores.  The block whose arrival
// completes the tile's count adds the slices (in slice order) into h, and
// with a gain stores the next norm's bf16(h (1 + gain)) and the per-row sums
// of h^2 over each 32 columns (fused residual-add + RMSNorm, the norm's
// row scale then applied by the consuming GEMM).  It also puts the counter
// back to zero for the next launch.
template <int NTHR>
__device__ __forceinline__ void finish_split_tile(const GemmArgs& g, int S, int tile, int r0, int nr, int c0, int nc,
                                                  int* flag) {
  __builtin_amdgcn_s_waitcnt(0);              // this thread's slice stores are complete
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned old = __hip_atomic_fetch_add(g.fin_ctr + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = old + 1 == static_cast<unsigned>(S);
    if (last) __hip_atomic_store(g.fin_ctr + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag = last;
  }
  __syncthreads();
  if (!*flag) return;
  const int N = 32 * g.NPT;
  const int q4 = nc / 4;                      // float4 columns per row; 8 consecutive ones per 32 columns
  const int items = nr * q4;
  for (int base = 0; base < items; base += NTHR) {
    const int it = base + static_cast<int>(threadIdx.x);
    const int row = r0 + (it < items ? it / q4 : 0);
    const int col = c0 + 4 * (it < items ? it % q4 : 0);
    const bool ok = it < items && row < g.R;
    const int lr = ok ? row : 0;
    // every load unconditional (slice index clamped, the extra slices not added)
    float4 hv = *reinterpret_cast<const float4*>(g.fin_h + (int64_t)lr * N + col);
    float4 ps[16];
#pragma unroll
    for (int sl = 0; sl < 16; ++sl)
      ps[sl] = ld_device_f32x4(g.split_out, min(sl, S - 1) * g.split_stride + (int64_t)lr * N + col);
#pragma unroll
    for (int sl = 0; sl < 16; ++sl)
      if (sl < S) {
        hv.x += ps[sl].x; hv.y += ps[sl].y; hv.z += ps[sl].z; hv.w += ps[sl].w;
      }
    float sq = 0.f;
    if (ok) {
      *reinterpret_cast<float4*>(g.fin_h + (int64_t)row * N + col) = hv;
      if (g.fin_gain) {
        const float4 gn = *reinterpret_cast<const float4*>(g.fin_gain + col);
        uint2 a;
        a.x = pack_bf16x2(hv.x * (1.f + gn.x), hv.y * (1.f + gn.y));
        a.y = pack_bf16x2(hv.z * (1.f + gn.z), hv.w * (1.f + gn.w));
        *reinterpret_cast<uint2*>(g.fin_a + (int64_t)row * N + col) = a;
        sq = (hv.x * hv.x + hv.y * hv.y) + (hv.z * hv.z + hv.w * hv.w);
      }
    }
    if (g.fin_gain) {
      // the 8 threads of one 32-column group are consecutive lanes
      sq += __shfl_xor(sq, 1, 64);
      sq += __shfl_xor(sq, 2, 64);
      sq += __shfl_xor(sq, 4, 64);
      if (ok && (col % 32) == 0) g.fin_ss[(int64_t)row * (N / 32) + col / 32] = sq;
    }
  }
}

// Small-row GEMM (batch-1 style): one block = 4 waves computing 16*MT rows x
// 32*NP columns; the block's K range is split between the 4 waves, whose
// partial sums are added through LDS.  Wave w finishes row tile w % MT, the
// MT of its accumulator rows starting at (w / MT) * MT: with fewer row tiles
// than waves, the waves share each tile's epilogue.
// Fewer row tiles per block mean fewer activation bytes per block; the row
// blocks of one column tile share its weights in their XCD's L2.  With g.split_out set, blockIdx.z
// selects a slice of K and the block writes its raw partial sums to
// split_out[z] (fp32 [R][32*NPT]) instead of running the epilogue; the
// consumer adds the slices in a fixed order.
template <class Epi, int WK, bool SPLIT, int NP, int MT>
__global__ __launch_bounds__(256) void gemm_mfma_kernel(GemmArgs g, Epi epi) {
  constexpr int NT = 2 * NP;
  static_assert(MT >= 1 && MT <= 4, "at most one row tile per wave");
  __shared__ float red[4][MT * NT * 4][kWave];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int pt0 = blockIdx.x * NP;
  const int m0 = blockIdx.y * 16 * MT;
  const bf16_t* A = g.A_ind ? static_cast<const bf16_t*>(*g.A_ind) + g.a_off
                            : static_cast<const bf16_t*>(g.A);
  const int nkb = g.K / 64;
  const int nz = gridDim.z, z = blockIdx.z;
  const int zb0 = z * nkb / nz, zb1 = (z + 1) * nkb / nz;
  const int kb0 = zb0 + wave * (zb1 - zb0) / 4, kb1 = zb0 + (wave + 1) * (zb1 - zb0) / 4;
  const int arow = lane % 16, akg = lane / 16;

  // rows this lane loads A for.  Every load below is unconditional: rows past
  // R read row 0, and columns past N re-read the last pair tile.  Row i of an
  // MFMA result depends on row i of A only, so such rows (and rows past a
  // request's prefix length, see the epilogue) are simply never used, which
  // keeps the loads free of branches the compiler could not count through.
  const bf16_t* arp[MT];
  const bf16_t* alp[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int row = m0 + 16 * mt + arow;
    const int lr = row < g.R ? row : 0;
    arp[mt] = A + (int64_t)lr * g.lda + akg * 8;
    alp[mt] = SPLIT ? static_cast<const bf16_t*>(g.A_lo) + (int64_t)lr * g.lda + akg * 8 : nullptr;
  }

  // Epilogue inputs of the rows this wave finishes: they do not depend on the
  // products, so the first trip requests them right behind its operands and
  // they land together.  Rows past R read row 0, columns past N the last pair
  // tile; neither is stored.
  const int c = lane % 16;
  const int emt = wave % MT, ev0 = (wave / MT) * MT;   // row tile, first accumulator row
  typename Epi::ColPre cq[NP];
  typename Epi::Pre pre[NP][MT];
  float sc[NP][2];
  float rs[MT];                               // folded norm: 1/rms of the rows this lane finishes
  auto epi_loads = [&]() {
    if (g.row_ss) {
      // lanes c % 4 = j share a row's sums: chunks j, j + 4, ... of its row_nt / 4
      const int nch = g.row_nt / 4;
#pragma unroll
      for (int vv = 0; vv < MT; ++vv) {
        const int row = m0 + 16 * emt + 4 * akg + ev0 + vv;
        const float* rp = g.row_ss + (int64_t)(row < g.R ? row : 0) * g.row_nt;
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int ch = (c % 4) + 4 * i;
          const float4 v = *reinterpret_cast<const float4*>(rp + 4 * min(ch, nch - 1));
          if (ch < nch) sum += (v.x + v.y) + (v.z + v.w);
        }
        sum += __shfl_xor(sum, 1, 64);
        sum += __shfl_xor(sum, 2, 64);
        rs[vv] = 1.0f / sqrtf(sum / (float)(32 * g.row_nt) + g.row_eps);
      }
    }
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) {
      const int p = min(pt0 + pp, g.NPT - 1);
      cq[pp] = epi.colpre(p, c);
      sc[pp][0] = g.scale ? g.scale[32 * p + c] : 1.f;
      sc[pp][1] = g.scale ? g.scale[32 * p + 16 + c] : 1.f;
#pragma unroll
      for (int vv = 0; vv < MT; ++vv) {
        const int row = m0 + 16 * emt + 4 * akg + ev0 + vv;
        pre[pp][vv] = epi.pre(row < g.R ? row : 0, p, c);
      }
    }
  };
  auto no_loads = []() {};

  f32x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[mt][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  // trips of 4, then 2, then 1 k-blocks, so no k-block is loaded twice; the
  // first trip carries the epilogue loads
  int kb = kb0;
  if (kb + 4 <= kb1) {
    b1_trip<4, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb, arp, alp, acc, epi_loads);
    for (kb += 4; kb + 4 <= kb1; kb += 4) b1_trip<4, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb, arp, alp, acc, no_loads);
    if (kb + 2 <= kb1) {
      b1_trip<2, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb, arp, alp, acc, no_loads);
      kb += 2;
    }
    if (kb < kb1) b1_trip<1, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb, arp, alp, acc, no_loads);
  } else if (kb + 2 <= kb1) {
    b1_trip<2, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb, arp, alp, acc, epi_loads);
    if (kb + 3 == kb1) b1_trip<1, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb + 2, arp, alp, acc, no_loads);
  } else if (kb < kb1) {
    b1_trip<1, WK, SPLIT, NT, MT>(g, pt0, nkb, lane, kb, arp, alp, acc, epi_loads);
  } else {
    epi_loads();
  }

#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[wave][(mt * NT + t) * 4 + v][lane] = acc[mt][t][v];
  __syncthreads();

  const int mt = emt;
  const int N = 32 * g.NPT;
  float* sp = g.split_out ? g.split_out + (int64_t)z * g.split_stride : nullptr;
  // rows of a request past its prefix length (rows_per_req > 0) count as zero
  bool rowok[MT];
#pragma unroll
  for (int vv = 0; vv < MT; ++vv) {
    const int row = m0 + 16 * mt + 4 * akg + ev0 + vv;
    rowok[vv] = true;
    if (g.rows_per_req > 0 && row < g.R) rowok[vv] = (row % g.rows_per_req) < g.desc->prefix_len[row / g.rows_per_req];
  }
#pragma unroll
  for (int pp = 0; pp < NP; ++pp) {
    const int p = pt0 + pp;
    if (p >= g.NPT) break;
    float s0[MT], s1[MT];
#pragma unroll
    for (int vv = 0; vv < MT; ++vv) {
      s0[vv] = s1[vv] = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s0[vv] += red[w][(mt * NT + 2 * pp) * 4 + ev0 + vv][lane];
        s1[vv] += red[w][(mt * NT + 2 * pp + 1) * 4 + ev0 + vv][lane];
      }
      if (!rowok[vv]) s0[vv] = s1[vv] = 0.f;   // what a zero A row gives
    }
    // the epilogue loads landed with the operands; saying so here keeps the
    // compiler from waiting again, stores included, in front of each row's
    // guarded stores
    __builtin_amdgcn_s_waitcnt(0xF70);        // vmcnt(0), other counters open
#pragma unroll
    for (int vv = 0; vv < MT; ++vv) {
      const int row = m0 + 16 * mt + 4 * akg + ev0 + vv;
      if (row < g.R) {
        if (sp) {
          if (g.fin_ctr) {
            st_device_f32(sp, (int64_t)row * N + 32 * p + c, s0[vv] * sc[pp][0]);
            st_device_f32(sp, (int64_t)row * N + 32 * p + 16 + c, s1[vv] * sc[pp][1]);
          } else {
            sp[(int64_t)row * N + 32 * p + c] = s0[vv] * sc[pp][0];
            sp[(int64_t)row * N + 32 * p + 16 + c] = s1[vv] * sc[pp][1];
          }
        } else {
          const float r = g.row_ss ? rs[vv] : 1.f;
          epi.apply(row, p, c, cq[pp], pre[pp][vv], s0[vv] * sc[pp][0] * r, s1[vv] * sc[pp][1] * r);
        }
      }
    }
  }
  if (sp && g.fin_ctr) {
    __shared__ int last;
    const int nc = 32 * min(NP, g.NPT - pt0);
    finish_split_tile<256>(g, nz, blockIdx.y * gridDim.x + blockIdx.x, m0, 16 * MT, 32 * pt0, nc, &last);
  }
}

// fp32 path: weights stored [K][N] (packed column order).  Block: 16 rows x
// one pair tile (32 columns); K is split over 16 slices (thread = slice kq,
// column c), each slice accumulating all 16 rows of its two columns with
// 16-byte loads of four consecutive k of a row, and the slices are summed
// through LDS in slice order.  K a multiple of 64 (every K of the configs).
template <class Epi>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g, Epi epi) {
  __shared__ float red[16][16][33];             // [slice][row][column], padded
  const int c = threadIdx.x % 16, kq = threadIdx.x / 16;
  const int p = blockIdx.x;
  const int r0 = blockIdx.y * 16;
  const float* A = g.A_ind ? static_cast<const float*>(*g.A_ind) + g.a_off
                           : static_cast<const float*>(g.A);
  const float* w = static_cast<const float*>(g.W) + 32 * p + c;
  const int N = 32 * g.NPT;
  const int kc = g.K / 16;                      // slice length, a multiple of 4
  const int k0 = kq * kc;
  float s0[16], s1[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) s0[r] = s1[r] = 0.f;
  for (int k = k0; k < k0 + kc; k += 4) {
    float w0[4], w1[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w0[j] = w[(int64_t)(k + j) * N];
      w1[j] = w[(int64_t)(k + j) * N + 16];
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      // rows past R read row R-1 (their sums are never used)
      const float4 a = *reinterpret_cast<const float4*>(A + (int64_t)min(r0 + r, g.R - 1) * g.lda + k);
      s0[r] = fmaf(a.x, w0[0], s0[r]);
      s0[r] = fmaf(a.y, w0[1], s0[r]);
      s0[r] = fmaf(a.z, w0[2], s0[r]);
      s0[r] = fmaf(a.w, w0[3], s0[r]);
      s1[r] = fmaf(a.x, w1[0], s1[r]);
      s1[r] = fmaf(a.y, w1[1], s1[r]);
      s1[r] = fmaf(a.z, w1[2], s1[r]);
      s1[r] = fmaf(a.w, w1[3], s1[r]);
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    red[kq][r][c] = s0[r];
    red[kq][r][16 + c] = s1[r];
  }
  __syncthreads();
  const int rr = threadIdx.x / 16;
  const int row = r0 + rr;
  if (row >= g.R) return;
  float t0 = 0.f, t1 = 0.f;
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    t0 += red[q][rr][c];
    t1 += red[q][rr][16 + c];
  }
  // rows of a request past its prefix length (rows_per_req > 0) count as zero
  if (g.rows_per_req > 0 && (row % g.rows_per_req) >= g.desc->prefix_len[row / g.rows_per_req]) t0 = t1 = 0.f;
  epi(row, p, c, t0, t1);
}

// ---------------------------------------------------------------------------
// Tiled GEMM for many rows (rollout batches): 128 x 128 output tiles, 4 waves
// in a 2 x 2 arrangement of 64 x 64.  Per k-block of 64 the activation tile
// (128 x 64 bf16, 16-byte chunks XOR-swizzled against bank conflicts) and
// the block's 8 packed weight fragments are copied into LDS by direct
// global->LDS loads, double-buffered; fp8 codes are expanded to bf16 after
// the LDS read.  A grid-stride loop walks the output tiles.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void dma16(const void* src, lds_void_t* lds) {
  const uint32_t m = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" :: "s"(m), "v"(src) : "memory", "m0");
}
#define GEMM_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x70 | 0xF00)
__device__ __forceinline__ void bare_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
}
__device__ __forceinline__ int aswz(int row) { return (row >> 1) & 7; }

// XCD-aware tile order of the many-row GEMMs.  Blocks are dealt to the 8 XCDs
// round-robin and each XCD has its own L2, so with a plain order every XCD
// streams all of A and all of W.  When W is the larger operand the 128 x 128
// tiles are put in bands of kBand column tiles, row by row within a band,
// and XCD x takes the x-th eighth of that order (block b runs position
// (b % 8) * per + b / 8, plus multiples of the grid's share per XCD): an XCD
// then streams about one band of W.  Otherwise (and for the QKV epilogue,
// whose cost differs a lot between bands because of the transposed V
// stores) the plain order is kept: row tile fastest over the block index.
// With one tile per CU (the four-stage ring) and the activations the larger
// operand, the tiles go row by row and XCD x takes the x-th eighth, so that
// each activation row tile is streamed by one XCD.  (For the grid-strided
// kernel that row split measured no better than the plain order.)
constexpr int kOrderPlain = 0, kOrderRows = 1, kOrderBands = 2;
constexpr int kBand = 8;
__host__ __device__ inline int gemm_tiles(const GemmArgs& g) { return ((g.R + 127) / 128) * (g.NPT / 4); }
__host__ __device__ inline int tile_order(const GemmArgs& g, bool plain, bool rows_ok = false) {
  if (plain) return kOrderPlain;
  const int wb = g.kind == W_FP8 ? 1 : 2;
  if ((int64_t)32 * g.NPT * wb >= (int64_t)2 * g.R) return kOrderBands;
  return rows_ok ? kOrderRows : kOrderPlain;
}
// Position t of the order -> (row tile, column tile).  In the plain order a
// partial last row tile (tail) comes after all the full ones: the positions
// past two blocks per CU, which share a CU with two others, are then cheap
// half-empty tiles instead of full ones.
__device__ __forceinline__ void tile_at(int t, int mtiles, int ntiles, int order, bool tail, int& mi, int& ni) {
  if (order == kOrderPlain) {
    const int full = tail ? mtiles - 1 : mtiles;
    if (t < full * ntiles) {
      mi = t % full;
      ni = t / full;
    } else {
      mi = mtiles - 1;
      ni = t - full * ntiles;
    }
  } else if (order == kOrderRows) {
    mi = t / ntiles;
    ni = t % ntiles;
  } else {
    const int band = t / (mtiles * kBand);
    const int rem = t - band * mtiles * kBand;
    const int bw = min(kBand, ntiles - band * kBand);
    mi = rem / bw;
    ni = band * kBand + rem % bw;
  }
}
// The j-th tile of block b (j = 0, 1, ...) under the XCD split, -1 past the end;
// the grid is a multiple of 8.
__device__ __forceinline__ int xcd_tile(int b, int j, int grid, int T, int order) {
  if (order == kOrderPlain) {
    const int t = b + j * grid;
    return t < T ? t : -1;
  }
  const int per = (T + 7) / 8;
  const int k = b / 8 + j * (grid / 8);
  const int t = (b % 8) * per + k;
  return (k < per && t < T) ? t : -1;
}
// Grid for T tiles with at most `cap` blocks: a multiple of 8.
inline int xcd_grid(int T, int cap) {
  const int g = 8 * ((T + 7) / 8);
  return g < cap ? g : cap;
}


// Epilogue of a wave's 64 x 64 tile (4 x 4 MFMA tiles, two pair tiles):
// every load the epilogue needs (residual rows, biases, RoPE factors) is
// requested for all 32 elements of the lane before the first store, so the
// tile costs one memory round trip instead of one per element.
// Epilogue of a 64x32 wave tile held as acc[mt][n16][v] (rows r0 + 16mt + 4lg
// + v, pair tiles p0 and p0 + 1).  The element loads of MG row groups are
// requested together before any of their stores; MG trades registers (and so
// occupancy) against memory round trips.  MG = 0 finishes each element before
// loading the next.
template <int MG, class Epi, int NT>
__device__ __forceinline__ void tile_epilogue(const GemmArgs& g, const Epi& epi, const f32x4 (&acc)[4][NT], int r0,
                                              int p0, int lc, int lg) {
  static_assert(MG == 0 || 4 % MG == 0, "row groups come in 4s");
  constexpr int NP = NT / 2;                  // pair tiles of the wave tile
  if constexpr (MG == 0) {
#pragma unroll
    for (int pp = 0; pp < NP; ++pp) {
      const int p = p0 + pp;
      const float s0c = g.scale ? g.scale[32 * p + lc] : 1.f;
      const float s1c = g.scale ? g.scale[32 * p + 16 + lc] : 1.f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = r0 + 16 * mt + 4 * lg + v;
          if (row < g.R) epi(row, p, lc, acc[mt][2 * pp][v] * s0c, acc[mt][2 * pp + 1][v] * s1c);
        }
    }
    return;
  }
  typename Epi::ColPre cpre[NP];
  float sc[NP][2];
#pragma unroll
  for (int pp = 0; pp < NP; ++pp) {
    cpre[pp] = epi.colpre(p0 + pp, lc);
    sc[pp][0] = g.scale ? g.scale[32 * (p0 + pp) + lc] : 1.f;
    sc[pp][1] = g.scale ? g.scale[32 * (p0 + pp) + 16 + lc] : 1.f;
  }
  constexpr int MS = MG > 0 ? MG : 4;
#pragma unroll
  for (int m0 = 0; m0 < 4; m0 += MS) {
    typename Epi::Pre pre[NP][MS][4];
#pragma unroll
    for (int pp = 0; pp < NP; ++pp)
#pragma unroll
      for (int mi = 0; mi < MS; ++mi)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = r0 + 16 * (m0 + mi) + 4 * lg + v;
          if (row < g.R) pre[pp][mi][v] = epi.pre(row, p0 + pp, lc);
        }
#pragma unroll
    for (int pp = 0; pp < NP; ++pp)
#pragma unroll
      for (int mi = 0; mi < MS; ++mi)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = r0 + 16 * (m0 + mi) + 4 * lg + v;
          if (row < g.R)
            epi.apply(row, p0 + pp, lc, cpre[pp], pre[pp][mi][v], acc[m0 + mi][2 * pp][v] * sc[pp][0],
                      acc[m0 + mi][2 * pp + 1][v] * sc[pp][1]);
        }
  }
}

// The generic epilogue with the row inputs and column scales requested
// before the k-loop (four-stage ring); rows past R were loaded from row R-1
// and are not stored.
template <class Epi, int NT>
__device__ __forceinline__ void tile_epilogue_early(const GemmArgs& g, const Epi& epi, const f32x4 (&acc)[4][NT],
                                                    int r0, int p0, int lc, int lg,
                                                    const typename Epi::Pre (&pre)[NT / 2][4][4],
                                                    const float (&sc)[NT / 2][2]) {
#pragma unroll
  for (int pp = 0; pp < NT / 2; ++pp) {
    const typename Epi::ColPre cq = epi.colpre(p0 + pp, lc);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int row = r0 + 16 * mt + 4 * lg + v;
        if (row < g.R)
          epi.apply(row, p0 + pp, lc, cq, pre[pp][mt][v], acc[mt][2 * pp][v] * sc[pp][0],
                    acc[mt][2 * pp + 1][v] * sc[pp][1]);
      }
  }
}

template <bool FP8>
struct TiledSmem {
  bf16_t A[128 * 64];
  uint8_t B[8 * (FP8 ? 1024 : 2048)];
};

template <class Epi, bool FP8>
__global__ __launch_bounds__(256, 2) void gemm_tiled_kernel(GemmArgs g, Epi epi) {
  __shared__ __attribute__((aligned(1024))) TiledSmem<FP8> s0;
  __shared__ __attribute__((aligned(1024))) TiledSmem<FP8> s1;
  constexpr int FB = FP8 ? 1024 : 2048;          // bytes per weight fragment
  constexpr int NB = 8 * FB / 1024 / 4;          // weight DMA blocks per wave per k-block
  constexpr int NOPS = 4 + NB;                   // DMA ops per thread per k-block
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int wm = wave >> 1, wn = wave & 1;
  const int lc = lane % 16, lg = lane / 16;
  const int nkb = g.K / 64;
  const int mtiles = (g.R + 127) / 128, ntiles = g.NPT / 4;
  const bf16_t* A = static_cast<const bf16_t*>(g.A);
  const uint8_t* W = static_cast<const uint8_t*>(g.W);

  // per-thread A source offsets (row within tile, swizzled chunk) for loads i = 0..3
  int arow[4], acol[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pos = (4 * i + wave) * 64 + lane;
    arow[i] = pos / 8;
    acol[i] = 8 * ((pos % 8) ^ aswz(pos / 8));
  }

  const int order = tile_order(g, Epi::kWaveTile);
  for (int j = 0;; ++j) {
    const int tile = xcd_tile(blockIdx.x, j, gridDim.x, mtiles * ntiles, order);
    if (tile < 0) break;
    int mi, ni;
    tile_at(tile, mtiles, ntiles, order, g.R % 128 != 0, mi, ni);
    const int mt0 = mi * 128;
    const int pt0 = ni * 4;
    int aoff[4];       // element offsets of this thread's A chunks (rows clamped into range)
#pragma unroll
    for (int i = 0; i < 4; ++i) aoff[i] = min(mt0 + arow[i], g.R - 1) * g.lda + acol[i];

    auto issue = [&](TiledSmem<FP8>& S, int kb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16(A + aoff[i] + kb * 64, (lds_void_t*)(S.A + (4 * i + wv) * 512));
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int blk = 4 * i + wv;                  // 1 KiB block of the k-block's weights
        const int f = blk / (FB / 1024), part = blk % (FB / 1024);
        const int p = pt0 + f / 2, hf = f % 2;
        const uint8_t* src = W + ((int64_t)(p * nkb + kb) * 2 + hf) * FB + part * 1024 + lane * 16;
        dma16(src, (lds_void_t*)(S.B + blk * 1024));
      }
    };

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](const TiledSmem<FP8>& S) {
      bf16x8 af[4][2];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = 64 * wm + 16 * mt + lc;
#pragma unroll
        for (int st = 0; st < 2; ++st)
          af[mt][st] = *reinterpret_cast<const bf16x8*>(S.A + row * 64 + 8 * ((4 * st + lg) ^ aswz(row)));
      }
      bf16x8 bfr[4][2];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int f = (2 * wn + nt / 2) * 2 + nt % 2;
        if (FP8) {
          const uint4 v = *reinterpret_cast<const uint4*>(S.B + f * FB + lane * 16);
          bfr[nt][0] = fp8x8_to_bf16x8(v.x, v.y);
          bfr[nt][1] = fp8x8_to_bf16x8(v.z, v.w);
        } else {
          const uint4* src = reinterpret_cast<const uint4*>(S.B + f * FB + lane * 32);
          bfr[nt][0] = as_bf16x8(src[0]);
          bfr[nt][1] = as_bf16x8(src[1]);
        }
      }
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) acc[mt][nt] = mfma16x16x32(af[mt][st], bfr[nt][st], acc[mt][nt]);
    };

    issue(s0, 0);
    for (int kb = 0; kb < nkb; kb += 2) {
      if (kb + 1 < nkb) { issue(s1, kb + 1); GEMM_WAIT_VMCNT(NOPS); } else { GEMM_WAIT_VMCNT(0); }
      bare_barrier();
      compute(s0);
      bare_barrier();
      if (kb + 1 >= nkb) break;
      if (kb + 2 < nkb) { issue(s0, kb + 2); GEMM_WAIT_VMCNT(NOPS); } else { GEMM_WAIT_VMCNT(0); }
      bare_barrier();
      compute(s1);
      bare_barrier();
    }

    // epilogue: wave (wm, wn) holds rows mt0+64wm.., pair tiles pt0+2wn, +1
    if constexpr (Epi::kWaveTile) epi.wave_tile(g, acc, mt0 + 64 * wm, pt0 + 2 * wn, lc, lg);
    else tile_epilogue<4>(g, epi, acc, mt0 + 64 * wm, pt0 + 2 * wn, lc, lg);
  }
}

// ---------------------------------------------------------------------------
// Ring-pipelined 128 x 128 GEMM for many rows.  Waves in a 2 x 2 (64 x 64
// wave tiles) or 2 x 4 (64 x 32) arrangement; per k-block of 64 the
// activation tile and the block's 8 packed weight fragments go through an
// LDS ring of 2 or 4 stages (48 / 96 KiB per block for fp8 weights); one
// barrier per k-block; every fragment of a k-block is requested before its
// first MFMA.  On the rollout-batch shapes (3264 rows, fp8 weights) the
// two-stage form beat the grid-strided kernel above for K = 1024 (QKV 28.5
// vs 39 us, GeGLU 65 vs 77 us), and the four-stage eight-wave form beats
// both wherever a GEMM has at most one tile per CU (O 23.5, down 38.7 us).
// ---------------------------------------------------------------------------
template <bool FP8, int NW = 4>
struct RingCfg {
  static constexpr int FB = FP8 ? 1024 : 2048;   // bytes per (pair, half) fragment per k-block
  static constexpr int A_KB = 16, B_KB = 8 * FB / 1024;
  static constexpr int STAGE = (A_KB + B_KB) * 1024;
  static constexpr int A_LD = A_KB / NW, B_LD = B_KB / NW;   // 1 KiB DMA blocks per wave
};

// NS = 2: two stages (48 KiB fp8 / 64 KiB bf16), so three (two) blocks share
// a CU and cover each other's load latency.  NS = 4: for GEMMs with at most
// one tile per CU, where no other block is there to do that: four stages
// (96 / 128 KiB), two k-blocks in flight while one is computed, and the
// register room of a lone block for the batched epilogue.  WN = waves along
// N: 2 (four 64 x 64 wave tiles) or 4 (eight 64 x 32 wave tiles, two waves
// per SIMD for a lone block, so that one wave's LDS reads and fp8
// conversions overlap the other's MFMAs).
template <class Epi, bool FP8, int NS = 2, int WN = 2>
__global__ __launch_bounds__(128 * WN) __attribute__((amdgpu_waves_per_eu(NS > 2 ? WN / 2 : (WN == 4 ? 4 : (FP8 ? 3 : 2))))) void
gemm_ring_kernel(GemmArgs g, Epi epi) {
  constexpr int NW = 2 * WN;                  // waves per block
  constexpr int NT = 8 / WN;                  // 16-column MFMA tiles per wave (NT / 2 pair tiles)
  typedef RingCfg<FP8, NW> C;
  static_assert(NS == 2 || NS == 4, "two or four stages");
  static_assert(WN == 2 || (WN == 4 && !Epi::kWaveTile), "eight waves only with the generic epilogue");
  __shared__ __attribute__((aligned(1024))) uint8_t ring[NS * C::STAGE];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int wm = wave / WN, wn = wave % WN;
  const int lc = lane % 16, lg = lane / 16;
  const int mtiles = (g.R + 127) / 128, ntiles = g.NPT / 4;
  const int order = tile_order(g, Epi::kWaveTile, NS == 4);
  const int t = xcd_tile(blockIdx.x, 0, gridDim.x, mtiles * ntiles, order);
  if (t < 0) return;
  int mi, ni;
  tile_at(t, mtiles, ntiles, order, g.R % 128 != 0, mi, ni);
  const int m0 = mi * 128, pt0 = ni * 4;
  const bf16_t* A = static_cast<const bf16_t*>(g.A);
  const uint8_t* W = static_cast<const uint8_t*>(g.W);
  // K slice blockIdx.y of gridDim.y (split-K: the slice's raw sums go to
  // split_out, the consumer adds the slices); the ring runs over its k-blocks
  const int nkb = g.K / 64 / gridDim.y, kb0 = blockIdx.y * nkb;
  float* const sp = g.split_out ? g.split_out + (int64_t)blockIdx.y * g.split_stride : nullptr;

  int aoff[C::A_LD];
#pragma unroll
  for (int i = 0; i < C::A_LD; ++i) {
    const int row = 8 * (NW * i + wave) + lane / 8;      // 1 KiB block NW i + wave = rows 8 blk ..
    aoff[i] = min(m0 + row, g.R - 1) * g.lda + 8 * ((lane % 8) ^ aswz(row));
  }
  const uint8_t* bsrc[C::B_LD];
#pragma unroll
  for (int i = 0; i < C::B_LD; ++i) {
    const int blk = NW * i + wave;
    const int f = blk / (C::FB / 1024), part = blk % (C::FB / 1024);
    bsrc[i] = W + ((int64_t)(pt0 + f / 2) * (g.K / 64) * 2 + f % 2) * C::FB + part * 1024 + lane * 16;
  }
  auto issue = [&](int slot, int kbl) {
    const int kb = kb0 + kbl;
    uint8_t* base = ring + slot * C::STAGE;
#pragma unroll
    for (int i = 0; i < C::A_LD; ++i) dma16(A + aoff[i] + kb * 64, (lds_void_t*)(base + (NW * i + wv) * 1024));
#pragma unroll
    for (int i = 0; i < C::B_LD; ++i)
      dma16(bsrc[i] + (int64_t)kb * 2 * C::FB, (lds_void_t*)(base + (C::A_KB + NW * i + wv) * 1024));
  };

  // With one tile per CU (four-stage ring) nothing hides the round trip of
  // the epilogue's row inputs (the residual rows) after the last k-block, so
  // they and the fp8 column scales are requested here, before the first
  // tile load: as the wave's oldest loads, every in-order wait of the loop
  // covers them.  Unconditional (rows past R read row R-1), so that no
  // branch makes the compiler wait for them early.
  constexpr bool kEarly = NS == 4 && !Epi::kWaveTile;
  typename Epi::Pre epre[NT / 2][4][4];
  float esc[NT / 2][2];
  if constexpr (kEarly) {
#pragma unroll
    for (int pp = 0; pp < NT / 2; ++pp) {
      const int p = pt0 + (NT / 2) * wn + pp;
      esc[pp][0] = FP8 ? g.scale[32 * p + lc] : 1.f;
      esc[pp][1] = FP8 ? g.scale[32 * p + 16 + lc] : 1.f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          epre[pp][mt][v] = epi.pre(min(m0 + 64 * wm + 16 * mt + 4 * lg + v, g.R - 1), p, lc);
    }
  }

  f32x4 acc[4][NT];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int slot) {
    const bf16_t* As = reinterpret_cast<const bf16_t*>(ring + slot * C::STAGE);
    const uint8_t* Bs = ring + slot * C::STAGE + C::A_KB * 1024;
    constexpr int BW = FP8 ? 1 : 2;
    uint4 braw[NT][BW];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int f = 2 * ((NT / 2) * wn + nt / 2) + nt % 2;
#pragma unroll
      for (int w = 0; w < BW; ++w) braw[nt][w] = *reinterpret_cast<const uint4*>(Bs + f * C::FB + lane * 16 * BW + 16 * w);
    }
    bf16x8 af[2][4];
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = 64 * wm + 16 * mt + lc;
        af[st][mt] = *reinterpret_cast<const bf16x8*>(As + row * 64 + 8 * ((4 * st + lg) ^ aswz(row)));
      }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      bf16x8 bfr[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (FP8) bfr[nt] = st == 0 ? fp8x8_to_bf16x8(braw[nt][0].x, braw[nt][0].y)
                                   : fp8x8_to_bf16x8(braw[nt][0].z, braw[nt][0].w);
        else bfr[nt] = as_bf16x8(braw[nt][BW - 1 < st ? 0 : st]);
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = mfma16x16x32(af[st][mt], bfr[nt], acc[mt][nt]);
    }
  };

  if constexpr (NS == 2) {
    issue(0, 0);
    for (int kb = 0; kb < nkb; ++kb) {
      GEMM_WAIT_VMCNT(0);                    // this wave's loads of k-block kb have landed
      bare_barrier();                        // ... everyone's, and k-block kb-1 is consumed
      if (kb + 1 < nkb) issue((kb + 1) & 1, kb + 1);
      compute(kb & 1);
    }
  } else {
    constexpr int LPK = C::A_LD + C::B_LD;   // loads per wave per k-block
    for (int q = 0; q < NS - 1 && q < nkb; ++q) issue(q, q);
    for (int kb = 0; kb < nkb; ++kb) {
      // k-block kb landed; the (up to NS - 2) later ones issued may still fly
      const int later = min(NS - 2, nkb - 1 - kb);
      if (later >= 2) GEMM_WAIT_VMCNT(2 * LPK);
      else if (later == 1) GEMM_WAIT_VMCNT(LPK);
      else GEMM_WAIT_VMCNT(0);
      bare_barrier();                        // everyone's landed, and k-block kb-1's slot is free
      if (kb + NS - 1 < nkb) issue((kb + NS - 1) % NS, kb + NS - 1);
      compute(kb % NS);
    }
  }

  if constexpr (Epi::kWaveTile) {
    // the ring is free once every wave is past its last k-block: each wave
    // stages its V tile there
    static_assert(NW * Epi::kVStage * 2 <= NS * C::STAGE, "V staging fits the ring");
    bare_barrier();
    epi.wave_tile(g, acc, m0 + 64 * wm, pt0 + 2 * wn, lc, lg, reinterpret_cast<bf16_t*>(ring) + wave * Epi::kVStage);
  } else if constexpr (kEarly) {
    if (sp) {
      const int N = 32 * g.NPT;
#pragma unroll
      for (int pp = 0; pp < NT / 2; ++pp) {
        const int p = pt0 + (NT / 2) * wn + pp;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int row = m0 + 64 * wm + 16 * mt + 4 * lg + v;
            if (row < g.R) {
              sp[(int64_t)row * N + 32 * p + lc] = acc[mt][2 * pp][v] * esc[pp][0];
              sp[(int64_t)row * N + 32 * p + 16 + lc] = acc[mt][2 * pp + 1][v] * esc[pp][1];
            }
          }
      }
    } else {
      tile_epilogue_early<Epi, NT>(g, epi, acc, m0 + 64 * wm, pt0 + (NT / 2) * wn, lc, lg, epre, esc);
    }
  } else {
    tile_epilogue<0>(g, epi, acc, m0 + 64 * wm, pt0 + (NT / 2) * wn, lc, lg);
  }
}

}  // namespace

// Split-K GEMMs run 16-row blocks; the split brings the grid to about 256
// blocks.  At batch 1 the down projection then takes 2 slices of 2048 (256
// blocks) instead of 8 slices of 512 over 64-row blocks: the next norm
// folds a quarter of the slices (8.39 -> 8.31 ms per chunk).
int gemm_split_k(int R, int NPT, int K) {
  if (R >= 256) {
    // many rows: the one-tile-per-CU ring splits K when its tiles fill at
    // most half the CUs (the prefix LM's O and down projections: 112 tiles)
    // and each slice keeps at least 16 k-blocks, or 4 when the tiles fill at
    // most a quarter of the CUs (the vision tower's O projection, 48 tiles
    // of K = 1024: 14.8 -> 8.8 us, the norm adding the slices 3 -> 5 us);
    // PHYAI_GEMM_TILE (tests) forces a kernel without the split
    if (getenv("PHYAI_GEMM_TILE") || NPT % 4 != 0) return 1;
    const int tiles = ((R + 127) / 128) * (NPT / 4);
    const int minkb = tiles <= 64 ? 4 : 16;
    int s = 1;
    while (s < 4 && tiles * s * 2 <= 256 && (K / 64) % (2 * s) == 0 && K / 64 / (2 * s) >= minkb) s *= 2;
    return s;
  }
  const int blocks = NPT * ((R + 15) / 16);
  int s = (256 + blocks - 1) / blocks;
  const int cap = (K / 64) / 4;               // keep >= one k-block per wave
  if (s > cap) s = cap;
  if (s > 8) s = 8;
  return s < 1 ? 1 : s;
}

namespace {

// Output projection fed by key-split attention partials (small row counts).
// Block = 16 token rows x 4 pair tiles (128 columns) x one 256-wide slice z of
// K, i.e. of the concatenated heads; 8 waves.  Each thread first merges 8
// consecutive elements of one row from all splits, o = sum_s w_s o_s /
// sum_s w_s with w_s = l_s 2^(m_s - max m) (the split-softmax merge), into a
// bf16 LDS panel.  Waves w and w + 4 then multiply the two halves of the
// panel's K by pair tile w and add through LDS.  The split loads, the weights
// and the epilogue inputs are all requested before the first wait, so the
// block makes one memory round trip.  Rows past R merge row R-1 and are never
// stored; splits past n_split re-read the last one and are skipped.  The 1-D
// grid deals consecutive tiles (slice-major) to one XCD, so each XCD's L2
// fetches the partials and weights of its own slices only.
template <class Epi, int WK, int NS>
__global__ __launch_bounds__(512) void merge_gemm_kernel(GemmArgs g, AttnParts ap, Epi epi) {
  constexpr int KZ = 256;                     // K per slice
  constexpr int KH = KZ / 128;                // k-blocks of 64 per wave half
  __shared__ __attribute__((aligned(16))) bf16_t panel[16 * KZ];
  __shared__ f32x4 red[4][2][kWave];
  const int nx = (g.NPT + 3) / 4, ny = (g.R + 15) / 16;
  const int T = nx * ny * (g.K / KZ);
  const int t = (blockIdx.x % 8) * (int)(gridDim.x / 8) + blockIdx.x / 8;
  if (t >= T) return;
  const int z = t / (nx * ny), bx = t % nx, m0 = (t / nx) % ny * 16;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int wq = wave % 4, kh = wave / 4;     // pair tile within the block, K half
  const int pw = bx * 4 + wq;
  const int p = min(pw, g.NPT - 1);
  const int nkb = g.K / 64;
  const int c = lane % 16, akg = lane / 16;

  // weights of pair tile p over this wave's half of the slice
  bf16x8 b[KH][2][2];
#pragma unroll
  for (int j = 0; j < KH; ++j)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) load_wfrag<WK>(g, p, nkb, z * (KZ / 64) + kh * KH + j, hf, lane, b[j][hf]);

  // split partials of row i, elements 8 cc .. 8 cc + 7 of the slice
  const int i = threadIdx.x / 32, cc = threadIdx.x % 32;
  const int r = min(m0 + i, g.R - 1);
  const int rb = r / ap.M, tok = r % ap.M;
  const int n = ap.n_split;
  const int k = z * KZ + 8 * cc;
  const int head = k / ap.D, dd = k % ap.D;
  const int qr = tok * ap.G + head % ap.G;
  const int64_t tile = (int64_t)(rb * ap.nkv + head / ap.G) * ap.ntiles + qr / ap.rows_per_tile;
  const int lrow = qr % ap.rows_per_tile;
  uint4 ov[NS];
  f32x2 ml[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int se = s < n ? s : n - 1;
    const int64_t prow = (tile * n + se) * ap.rows_per_tile + lrow;
    ov[s] = *reinterpret_cast<const uint4*>(ap.o + prow * ap.D + dd);
    ml[s] = *reinterpret_cast<const f32x2*>(ap.ml + prow * 2);
  }
  // epilogue inputs last: a wait the compiler puts behind their branch then
  // finds every load already issued
  float* sp = g.split_out ? g.split_out + (int64_t)z * g.split_stride : nullptr;
  const float sc0 = g.scale ? g.scale[32 * p + c] : 1.f;
  const float sc1 = g.scale ? g.scale[32 * p + 16 + c] : 1.f;
  typename Epi::ColPre cq{};
  typename Epi::Pre pre[4]{};
  if (!sp) {
    cq = epi.colpre(p, c);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + 4 * akg + v;
      pre[v] = epi.pre(row < g.R ? row : 0, p, c);
    }
  }
  float mmax = -1e30f;
#pragma unroll
  for (int s = 0; s < NS; ++s) mmax = fmaxf(mmax, s < n ? ml[s][0] : -1e30f);
  float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float lsum = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    if (s < n) {
      const float w = ml[s][1] * __builtin_amdgcn_exp2f(ml[s][0] - mmax);
      lsum += w;
      const uint32_t q[4] = {ov[s].x, ov[s].y, ov[s].z, ov[s].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc8[2 * e] = fmaf(w, __uint_as_float(q[e] << 16), acc8[2 * e]);
        acc8[2 * e + 1] = fmaf(w, __uint_as_float(q[e] & 0xffff0000u), acc8[2 * e + 1]);
      }
    }
  }
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  uint4 pk;
  pk.x = pack_bf16x2(acc8[0] * inv, acc8[1] * inv);
  pk.y = pack_bf16x2(acc8[2] * inv, acc8[3] * inv);
  pk.z = pack_bf16x2(acc8[4] * inv, acc8[5] * inv);
  pk.w = pack_bf16x2(acc8[6] * inv, acc8[7] * inv);
  // 16-byte chunk cc of row i sits at cc ^ i: the 16 rows one MFMA operand
  // read covers then hit 16 different bank groups
  *reinterpret_cast<uint4*>(panel + i * KZ + 8 * (cc ^ i)) = pk;
  __syncthreads();

  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
  for (int j = 0; j < KH; ++j)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int ch = 8 * (kh * KH + j) + 4 * s + akg;
      const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4*>(panel + c * KZ + 8 * (ch ^ c)));
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) acc[hf] = mfma16x16x32(a, b[j][hf][s], acc[hf]);
    }
  if (kh == 1) {
    red[wq][0][lane] = acc[0];
    red[wq][1][lane] = acc[1];
  }
  __syncthreads();
  const int N = 32 * g.NPT;
  if (!(kh == 1 || pw >= g.NPT)) {
    acc[0] += red[wq][0][lane];
    acc[1] += red[wq][1][lane];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + 4 * akg + v;
      if (row >= g.R) continue;
      if (sp) {
        if (g.fin_ctr) {
          st_device_f32(sp, (int64_t)row * N + 32 * p + c, acc[0][v] * sc0);
          st_device_f32(sp, (int64_t)row * N + 32 * p + 16 + c, acc[1][v] * sc1);
        } else {
          sp[(int64_t)row * N + 32 * p + c] = acc[0][v] * sc0;
          sp[(int64_t)row * N + 32 * p + 16 + c] = acc[1][v] * sc1;
        }
      } else {
        epi.apply(row, p, c, cq, pre[v], acc[0][v] * sc0, acc[1][v] * sc1);
      }
    }
  }
  if (sp && g.fin_ctr) {
    __shared__ int last;
    const int nc = 32 * min(4, g.NPT - bx * 4);
    finish_split_tile<512>(g, g.K / KZ, (m0 / 16) * nx + bx, m0, 16, 32 * bx * 4, nc, &last);
  }
}

// Row tiles per small-row block without a K split: the fewest that keep the
// grid within 384 blocks.  Fewer rows per block cut the activation bytes each
// block re-reads for its columns (batch 1: QKV 7.9 -> 6.0 us with 16-row
// blocks); past ~384 blocks the weight re-reads of the extra row blocks
// cost more than that saves (gate/up keeps 64 rows).  Split-K GEMMs always
// run 16-row blocks (gemm_split_k).  PHYAI_SMALL_MT (tests, read at enqueue
// time): a positive value forces the row tiles, a negative one sets the
// block limit.
int small_row_tiles(int R, int NPT) {
  const char* f = getenv("PHYAI_SMALL_MT");
  int lim = 384;
  if (f) {
    const int v = atoi(f);
    if (v > 0) return v;
    lim = -v;
  }
  for (int mt = 1; mt < kMT; mt *= 2)
    if (NPT * ((R + 16 * mt - 1) / (16 * mt)) <= lim) return mt;
  return kMT;
}

template <class Epi>
void launch(const GemmArgs& g, const Epi& epi, hipStream_t s) {
  if (g.kind == W_F32) {
    dim3 grid(g.NPT, (g.R + 15) / 16);
    hipLaunchKernelGGL(gemm_f32_kernel<Epi>, grid, dim3(256), 0, s, g, epi);
  } else if (g.R >= 256 && g.A_lo == nullptr && g.A_ind == nullptr && g.rows_per_req == 0 && g.NPT % 4 == 0 &&
             g.kind != W_FP4) {
    const int tiles = gemm_tiles(g);
    const char* force = getenv("PHYAI_GEMM_TILE");   // tests: "ring" / "deep" / "strided" (read at enqueue time)
    // at most one tile per CU: no second block covers the load latency, so
    // the four-stage ring with eight waves (two per SIMD); otherwise the
    // two-stage ring for short K and the strided kernel for long K
    const int nz = g.split_out ? g.split_k : 1;       // K slices (gemm_split_k), deep ring only
    const bool deep = !Epi::kWaveTile && (nz > 1 || (force ? strcmp(force, "deep") == 0 : tiles <= 256));
    const bool ring = force ? strcmp(force, "strided") != 0 : g.K <= 2048;
    if (deep) {
      const dim3 rgrid(xcd_grid(tiles, 1 << 30), nz);
      if constexpr (!Epi::kWaveTile) {
        if (g.kind == W_FP8) hipLaunchKernelGGL((gemm_ring_kernel<Epi, true, 4, 4>), rgrid, dim3(512), 0, s, g, epi);
        else hipLaunchKernelGGL((gemm_ring_kernel<Epi, false, 4, 4>), rgrid, dim3(512), 0, s, g, epi);
      }
    } else if (ring) {
      // eight waves per block too, except for the QKV epilogue, whose wave-tile
      // form is written for 64 x 64 wave tiles
      const dim3 rgrid(xcd_grid(tiles, 1 << 30));
      constexpr int WN = Epi::kWaveTile ? 2 : 4;
      if (g.kind == W_FP8) hipLaunchKernelGGL((gemm_ring_kernel<Epi, true, 2, WN>), rgrid, dim3(128 * WN), 0, s, g, epi);
      else hipLaunchKernelGGL((gemm_ring_kernel<Epi, false, 2, WN>), rgrid, dim3(128 * WN), 0, s, g, epi);
    } else {
      dim3 grid(xcd_grid(tiles, 512));
      if (g.kind == W_FP8) hipLaunchKernelGGL((gemm_tiled_kernel<Epi, true>), grid, dim3(256), 0, s, g, epi);
      else hipLaunchKernelGGL((gemm_tiled_kernel<Epi, false>), grid, dim3(256), 0, s, g, epi);
    }
  } else {
    // 32 columns and 16 * MT rows per block; K split over blockIdx.z only
    // when the caller provides a partial-sum buffer (linear epilogues)
    const int nz = g.split_out ? g.split_k : 1;
    const bool two = g.A_lo != nullptr;
    auto go = [&](auto mtag) {
      constexpr int MT = decltype(mtag)::value;
      const dim3 grid(g.NPT, (g.R + 16 * MT - 1) / (16 * MT), nz);
      auto kind = [&](auto wk) {
        constexpr int WK = decltype(wk)::value;
        if (two) hipLaunchKernelGGL((gemm_mfma_kernel<Epi, WK, true, 1, MT>), grid, dim3(256), 0, s, g, epi);
        else hipLaunchKernelGGL((gemm_mfma_kernel<Epi, WK, false, 1, MT>), grid, dim3(256), 0, s, g, epi);
      };
      if (g.kind == W_FP8) kind(std::integral_constant<int, W_FP8>{});
      else if (g.kind == W_FP4) kind(std::integral_constant<int, W_FP4>{});
      else kind(std::integral_constant<int, W_BF16>{});
    };
    const int mt = nz > 1 ? 1 : small_row_tiles(g.R, g.NPT);
    if (mt == 1) go(std::integral_constant<int, 1>{});
    else if (mt == 2) go(std::integral_constant<int, 2>{});
    else go(std::integral_constant<int, kMT>{});
  }
}

}  // namespace

void gemm_store_bf16(const GemmArgs& g, const EpiStore<bf16_t>& e, hipStream_t s) { launch(g, e, s); }
void gemm_store_f32(const GemmArgs& g, const EpiStore<float>& e, hipStream_t s) { launch(g, e, s); }
void gemm_resid(const GemmArgs& g, const EpiResid& e, hipStream_t s) { launch(g, e, s); }
void gemm_geglu_bf16(const GemmArgs& g, const EpiGeglu<bf16_t>& e, hipStream_t s) { launch(g, e, s); }
void gemm_geglu_f32(const GemmArgs& g, const EpiGeglu<float>& e, hipStream_t s) { launch(g, e, s); }
void gemm_qkv_bf16(const GemmArgs& g, const EpiQkv<bf16_t>& e, hipStream_t s) { launch(g, e, s); }
void gemm_qkv_f32(const GemmArgs& g, const EpiQkv<float>& e, hipStream_t s) { launch(g, e, s); }
void gemm_kv_bf16(const GemmArgs& g, const EpiKV<bf16_t>& e, hipStream_t s) { launch(g, e, s); }
void gemm_kv_f32(const GemmArgs& g, const EpiKV<float>& e, hipStream_t s) { launch(g, e, s); }

void gemm_merge_resid(const GemmArgs& g, const AttnParts& ap, const EpiResid& e, hipStream_t s) {
  const int tiles = ((g.NPT + 3) / 4) * ((g.R + 15) / 16) * (g.K / 256);
  const dim3 grid(8 * ((tiles + 7) / 8));
  auto go = [&](auto ns) {
    constexpr int NS = decltype(ns)::value;
    if (g.kind == W_FP8) hipLaunchKernelGGL((merge_gemm_kernel<EpiResid, W_FP8, NS>), grid, dim3(512), 0, s, g, ap, e);
    else if (g.kind == W_FP4) hipLaunchKernelGGL((merge_gemm_kernel<EpiResid, W_FP4, NS>), grid, dim3(512), 0, s, g, ap, e);
    else hipLaunchKernelGGL((merge_gemm_kernel<EpiResid, W_BF16, NS>), grid, dim3(512), 0, s, g, ap, e);
  };
  if (ap.n_split <= 4) go(std::integral_constant<int, 4>{});
  else if (ap.n_split <= 8) go(std::integral_constant<int, 8>{});
  else go(std::integral_constant<int, 16>{});
}

}  // namespace phyai
