// Persistent batch-1 denoising loop: one cooperative launch of 256 blocks (one
// per CU) runs up to 16 Euler steps of one pi0 request, as the single
// scheduled kernel for the repeated expert path that the paper lists as
// future work (Section "Future Work", subsection "Mega Kernels").  Opt-in:
// on MI355X it runs slower than the captured per-kernel graph at the pi0
// shape, and the graph path stays the default.
//
// Each step is a fixed sequence of phases separated by a grid barrier:
//   time-MLP second layer, then per block of the transformer
//   QKV (+ RoPE, suffix K/V into the key range), attention (one 64-key tile
//   per block and head), split merge, O projection (+ residual), gate/up
//   (+ GeGLU), down (+ residual), and finally readout + Euler update (+ the
//   next step's action embedding).
//
// Cross-XCD hand-off without cache-wide fences.  Every store another block
// reads is a write-through device-scope (sc1) store; a thread waits for its
// own stores (s_waitcnt) before its block arrives at the barrier, and a block
// reads only after the barrier's counter shows every block arrived.  Data
// rewritten within a launch (the residual h, split-K and attention partials,
// the suffix keys) is read back with device-scope loads, which bypass a
// possibly stale L2 line.  The GEMM operands (the normed activations, their
// sums of squares, q, o, the GeGLU output, the time-MLP hidden) get a fresh
// copy per step and site instead, written once per launch before any block
// reads it; since a launch starts with every L2 invalidated, no L2 can hold
// a stale line of such an address and their readers use plain cached loads.
// Weights, the prefix K/V and the per-call tables are written before the
// launch and read with plain loads.  The residual GEMMs' split-K reduction:
// the block whose atomic arrival completes a column tile's count adds that
// tile's partials (in a fixed order, so results do not depend on arrival
// order).
//
// Norms are folded into the GEMMs (the fused residual-add + RMSNorm ahead of
// the QKV and gate/up GEMMs of Section "PhyAI Architecture", subsection
// "Optimization Methods", paragraph "Kernel fusion"): the block that finishes
// a residual tile stores bf16(h (1 + w)) of the next norm site and that
// tile's sums of h^2; the consuming GEMM multiplies its accumulator rows by
// 1/rms, since n W = (1/rms) ((h (1 + w)) W).
//
// Wave roles.  In the full-K GEMMs (QKV, gate/up) waves 0-5 each load all of
// their A operand in one batch and waves 6-7 copy the next phase's weight or
// key tiles into LDS with direct global->LDS loads, started once the GEMM
// waves' loads are queued; the GEMM waves sum their partials through LDS with
// LDS counters instead of block barriers, so the copies never hold them up.
// Elsewhere waves 0-3 compute and 4-7 copy.  Every wait is bounded: a wait
// that times out sets an error flag, later barriers stop waiting, and the
// output is NaN.
#include "kernels.hpp"

#include <cmath>

namespace phyai {

namespace {

constexpr int kBlocks = 256;
constexpr int kThreads = 512;
constexpr int kSlot = 64 * 1024;          // weight / key tile slot
constexpr int kWork = 32 * 1024;          // reductions and staging
constexpr int kSC1 = 16;                  // buffer cache policy: device scope
constexpr int kSpinMax = 1 << 20;         // barrier give-up (about a second)
constexpr float kLog2e = 1.4426950408889634f;

// counter layout in PersistArgs::ctr
constexpr int kErr = 0, kGroup = 32, kTop = 32 + 32 * 8, kTileTime = 384, kTileO = 512, kTileDown = 640;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, 0x7fffffff, 0x00020000);
}
// A resource of `bytes` bytes: loads past the end return zero without a
// memory access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_n(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}
// device-scope loads and stores (byte offsets from base)
__device__ __forceinline__ u32x4 ld16(const void* base, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ u32x2 ld8(const void* base, int off) {
  return __builtin_amdgcn_raw_buffer_load_b64(rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ float ldf(const void* base, int off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(base), off, 0, kSC1));
}
__device__ __forceinline__ uint32_t ld4(const void* base, int off) {
  return __builtin_amdgcn_raw_buffer_load_b32(rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ unsigned short ld2(const void* base, int off) {
  return __builtin_amdgcn_raw_buffer_load_b16(rsrc(base), off, 0, kSC1);
}
// Plain (L2-cached) loads, for the per-step activation copies: each address
// of those is written once per launch (write-through, device scope) before
// any block reads it, and the launch starts with the L2s invalidated, so no
// L2 can hold a stale line of it.
__device__ __forceinline__ u32x4 ldn16(const void* base, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(rsrc(base), off, 0, 0);
}
__device__ __forceinline__ u32x2 ldn8(const void* base, int off) {
  return __builtin_amdgcn_raw_buffer_load_b64(rsrc(base), off, 0, 0);
}
__device__ __forceinline__ float ldnf(const void* base, int off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(base), off, 0, 0));
}
// Element access goes through HIP's float2 / uint2 types: extracting elements
// of the builtin's own vector result lost all but the first element.
__device__ __forceinline__ float2 ld8f(const void* base, int off) { return __builtin_bit_cast(float2, ld8(base, off)); }
__device__ __forceinline__ uint2 ld8u(const void* base, int off) { return __builtin_bit_cast(uint2, ld8(base, off)); }
__device__ __forceinline__ void st16(void* base, int off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ void st8(void* base, int off, u32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ void stf(void* base, int off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ void st4(void* base, int off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, rsrc(base), off, 0, kSC1);
}
__device__ __forceinline__ void st2(void* base, int off, bf16_t v) {
  __builtin_amdgcn_raw_buffer_store_b16(v, rsrc(base), off, 0, kSC1);
}

// The block's LDS: two 64 KiB slots (weight or key tiles) and 32 KiB of work
// space.  Declared at file scope so that the out-of-line phase functions
// address it as LDS (ds instructions) rather than through generic pointers.
__shared__ __attribute__((aligned(1024))) char g_lds[2 * kSlot + kWork];

// The argument block, read through the constant address space at a
// wave-uniform address, so that its fields (and the buffer descriptors built
// from them) live in scalar registers.  Phase functions are out of line and
// receive their arguments in vector registers; readfirstlane restores the
// uniformity the compiler cannot see.
typedef const __attribute__((address_space(4))) PersistArgs CP;
__device__ __forceinline__ CP& uargs(const PersistArgs* pa) {
  const uint64_t a = reinterpret_cast<uint64_t>(pa);
  // readfirstlane returns int: widen through uint32_t, never by sign extension
  const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a)));
  const uint64_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32)));
  return *reinterpret_cast<CP*>((hi << 32) | lo);
}
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Layer l's table entry through the constant address space (scalar loads; l
// must be wave-uniform).
typedef const __attribute__((address_space(4))) PersistLayer CL;
__device__ __forceinline__ CL& lay(CP& p, int l) {
  return reinterpret_cast<CL*>(reinterpret_cast<uintptr_t>(p.layer))[l];
}

// Per-step copies, indexed by the step's place r in this launch.  Norm site
// (r, l, 0) precedes block l's attention and (r, l, 1) its MLP; (r, L, 0) is
// the final norm.
__device__ __forceinline__ int site_of(CP& p, int k, int l, int s) { return (k * (p.L + 1) + l) * 2 + s; }
__device__ __forceinline__ bf16_t* a_of(CP& p, int site) { return p.a + (int64_t)site * 64 * p.d; }
__device__ __forceinline__ float* ss_of(CP& p, int site) { return p.ss + (int64_t)site * 64 * (p.d / 32); }
__device__ __forceinline__ bf16_t* q_of(CP& p, int k, int l) { return p.q + (int64_t)(k * p.L + l) * 64 * p.nq * p.D; }
__device__ __forceinline__ bf16_t* o_of(CP& p, int k, int l) { return p.o + (int64_t)(k * p.L + l) * 64 * p.nq * p.D; }
__device__ __forceinline__ bf16_t* g_of(CP& p, int k, int l) { return p.g + (int64_t)(k * p.L + l) * 64 * p.F; }
__device__ __forceinline__ bf16_t* z_of(CP& p, int k) { return p.z + (int64_t)k * 64 * p.d; }

__device__ __forceinline__ unsigned ld_ctr(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 16 bytes per lane from src into LDS at the wave-uniform address lds + 16 *
// lane, device scope (the source may have been written by another block).
__device__ __forceinline__ void dma16(const void* src, lds_void_t* lds) {
  const uint32_t m = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off sc1" :: "s"(m), "v"(src) : "memory", "m0");
}

// The same without sc1, for data written before the launch and never during it.
__device__ __forceinline__ void dma16p(const void* src, lds_void_t* lds) {
  const uint32_t m = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds)));
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" :: "s"(m), "v"(src) : "memory", "m0");
}

__device__ __forceinline__ void block_sync() { __syncthreads(); }

// Grid barrier: two-level arrival (a counter per group of 32 blocks -- the
// blocks of one XCD -- then a top counter), bounded polling of the top
// counter.  Every thread's own memory operations are complete before its
// block arrives.
__device__ __forceinline__ void grid_sync(unsigned* ctr, unsigned& gen) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  ++gen;
  if (threadIdx.x == 0) {
    unsigned* lc = reinterpret_cast<unsigned*>(g_lds + 2 * kSlot + 24 * 1024 + 16);
    lc[0] = 0u;
    lc[1] = 0u;
    lc[2] = 0u;
    const unsigned per = gridDim.x / 8;
    const unsigned old = __hip_atomic_fetch_add(ctr + kGroup + 32 * (blockIdx.x % 8), 1u, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == gen * per) __hip_atomic_fetch_add(ctr + kTop, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (!ld_ctr(ctr + kErr)) {
      int spins = 0;
      while (ld_ctr(ctr + kTop) < gen * 8) {
        __builtin_amdgcn_s_sleep(1);
        if (++spins > kSpinMax) {
          __hip_atomic_fetch_or(ctr + kErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        if ((spins & 255) == 0 && ld_ctr(ctr + kErr)) break;
      }
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Weight tiles into LDS by the copy waves cw0 .. 7.  The packed weight order
// puts pair tile p's k-blocks kb .. kb+n-1 in n * 4 KiB contiguous bytes; the
// slot receives them as they are.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void copy_weights(const void* W, int64_t byte_off, int bytes, char* slot, int cw0) {
  const int w = threadIdx.x / 64 - cw0, lane = threadIdx.x % 64;
  const char* src = static_cast<const char*>(W) + byte_off;
  for (int i = w; i < bytes / 1024; i += 8 - cw0)
    dma16p(src + i * 1024 + lane * 16, (lds_void_t*)(slot + i * 1024));
}

// ---------------------------------------------------------------------------
// Small-row GEMM of one wave: acc[mt][t] += A[16 mt + i][k] * Wtile[k][16 t + c]
// over k-blocks kb0 .. kb0 + nk - 1 (nk <= NK) of the block's slot (slot
// k-block index = kb - kslot0).  A: bf16 [R][lda] (global, device scope),
// rows >= R read row 0 (never stored).
// ---------------------------------------------------------------------------
template <int NB>
__device__ __forceinline__ void wave_gemm_batch(const bf16_t* A, int lda, int R, int kb0, int nk, const char* slot,
                                                int kslot0, f32x4 (&acc)[4][2]) {
  const int lane = threadIdx.x % 64;
  const int arow = lane % 16, akg = lane / 16;
  u32x4 av[NB][4][2];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int kb = kb0 + min(i, nk - 1);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int row = 16 * mt + arow < R ? 16 * mt + arow : 0;
#pragma unroll
      for (int s = 0; s < 2; ++s) av[i][mt][s] = ldn16(A, (row * lda + kb * 64 + 32 * s + 8 * akg) * 2);
    }
  }
  // all of the batch's loads in flight before the first use
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (i >= nk) break;
    const char* wk = slot + (kb0 + i - kslot0) * 4096 + lane * 32;
    bf16x8 b[2][2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int s = 0; s < 2; ++s) b[t][s] = *reinterpret_cast<const bf16x8*>(wk + t * 2048 + s * 16);
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[mt][t] = mfma16x16x32(__builtin_bit_cast(bf16x8, av[i][mt][s]), b[t][s], acc[mt][t]);
  }
}

// Small-row GEMM of one wave: acc[mt][t] += A[16 mt + i][k] * Wtile[k][16 t + c]
// over k-blocks kb0 .. kb0 + nk - 1 (nk <= NK) of the block's slot (slot
// k-block index = kb - kslot0), in batches of two k-blocks.  A: bf16 [R][lda]
// (global, device scope), rows >= R read row 0 (never stored).
template <int NK>
__device__ __forceinline__ void wave_gemm(const bf16_t* A, int lda, int R, int kb0, int nk, const char* slot,
                                          int kslot0, f32x4 (&acc)[4][2]) {
  if constexpr (NK == 1) {
    wave_gemm_batch<1>(A, lda, R, kb0, nk, slot, kslot0, acc);
  } else {
#pragma unroll
    for (int i = 0; i < NK; i += 2)
      if (i < nk) wave_gemm_batch<2>(A, lda, R, kb0 + i, min(2, nk - i), slot, kslot0, acc);
  }
}

// Full-K small-row GEMM of one of up to eight waves, all of its A loads in one
// batch: acc[mt][t] += A[16 mt + i][k] * Wtile[k][16 t + c] over k-blocks kb0
// .. kb0 + nk - 1 (nk <= NK) of the slot.  Rows >= R of A read as zero (past
// the end of the bounded resource, no memory access).  Counts itself in at
// `issued` once its loads are issued.
template <int NK>
__device__ __forceinline__ void wave_gemm_full(const bf16_t* A, int lda, int R, int kb0, int nk, const char* slot,
                                               f32x4 (&acc)[4][2], unsigned* issued) {
  const int lane = threadIdx.x % 64;
  const int arow = lane % 16, akg = lane / 16;
  const __amdgpu_buffer_rsrc_t ra = rsrc_n(A, R * lda * 2);
  u32x4 av[NK][4][2];
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    const int kb = kb0 + min(i, nk - 1);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int s = 0; s < 2; ++s)
        av[i][mt][s] = __builtin_amdgcn_raw_buffer_load_b128(ra, ((16 * mt + arow) * lda + kb * 64 + 32 * s + 8 * akg) * 2, 0, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
  // the copy waves start their weight copies once every GEMM wave's operand
  // requests are queued ahead of them
  if (lane == 0) __hip_atomic_fetch_add(issued, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int i = 0; i < NK; ++i) {
    if (i >= nk) break;
    const char* wk = slot + (kb0 + i) * 4096 + lane * 32;
    bf16x8 b[2][2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int s = 0; s < 2; ++s) b[t][s] = *reinterpret_cast<const bf16x8*>(wk + t * 2048 + s * 16);
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[mt][t] = mfma16x16x32(__builtin_bit_cast(bf16x8, av[i][mt][s]), b[t][s], acc[mt][t]);
  }
}

// K split of the full-K GEMMs over waves 0 .. nw - 1 (nw = min(6, nkb); waves 6
// and 7 copy): wave w takes k-blocks kb0 .. kb0 + nk - 1.
__device__ __forceinline__ int full_k_waves(int nkb) { return nkb < 6 ? nkb : 6; }
__device__ __forceinline__ void full_k_split(int nkb, int w, int& kb0, int& nk) {
  const int nw = full_k_waves(nkb), base = nkb / nw, extra = nkb % nw;
  kb0 = w * base + min(w, extra);
  nk = base + (w < extra ? 1 : 0);
}

// Sum the accumulators of the nw (4..6) GEMM waves through `scratch` (the
// phase's weight slot, free once every GEMM wave is past its MFMAs) without a
// block barrier, so that the copy waves never hold the GEMM waves up.  The
// GEMM waves count themselves in at cnt[1] when done with the slot and wait
// for each other; each then stores its partials and counts itself in at
// cnt[0]; waves 0..3 wait until cnt[0] reaches `target` (nw, plus any other
// wave that counts itself in after an LDS write the epilogue reads) and sum
// row tile w over the waves in order.  Every wait is bounded.
// fin[t][v] is row 16 w + 4 (lane / 16) + v, column 16 t + lane % 16.
// Returns false for the waves without output (and on a wait that gave up,
// after raising the error flag).
// Wait (bounded) until the LDS counter reaches `target`; on giving up raise
// the error flag and return false.
__device__ __forceinline__ bool lds_wait(unsigned* c, int target, unsigned* ctr) {
  int spins = 0;
  while (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) < (unsigned)target) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kSpinMax) {
      if (threadIdx.x % 64 == 0) __hip_atomic_fetch_or(ctr + kErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return false;
    }
  }
  return true;
}
__device__ __forceinline__ bool reduce_gemm_waves(const f32x4 (&acc)[4][2], f32x4 (&fin)[2], char* scratch, int target,
                                                  int nw, unsigned* cnt, unsigned* ctr) {
  f32x4* red = reinterpret_cast<f32x4*>(scratch);        // [nw waves][4 mt][2 t][64 lanes]
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  if (w >= nw) return false;
  // one count per wave (lane 0: an atomic by every lane would add 64)
  if (lane == 0) __hip_atomic_fetch_add(cnt + 1, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  if (!lds_wait(cnt + 1, nw, ctr)) return false;
#pragma unroll
  for (int mt = 0; mt < 4; ++mt)
#pragma unroll
    for (int t = 0; t < 2; ++t) red[((w * 4 + mt) * 2 + t) * 64 + lane] = acc[mt][t];
  if (lane == 0) __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  if (w >= 4) return false;
  if (!lds_wait(cnt, target, ctr)) return false;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    f32x4 sum = red[((0 * 4 + w) * 2 + t) * 64 + lane];
    for (int ww = 1; ww < nw; ++ww) {
      const f32x4 x = red[((ww * 4 + w) * 2 + t) * 64 + lane];
      sum[0] += x[0]; sum[1] += x[1]; sum[2] += x[2]; sum[3] += x[3];
    }
    fin[t] = sum;
  }
  return true;
}

// Sum the four compute waves' accumulators through LDS: wave w ends with row
// tile w (rows 16 w + 4 (lane / 16) + v, columns c = lane % 16 of each half).
// A wave sends only the three row tiles it does not finish (24 KiB).  Called
// by all threads of the block (two block barriers).
__device__ __forceinline__ int red_slot(int w, int mt) { return w * 3 + (mt > w ? mt - 1 : mt); }
// Wave W's own sum, with every register index static (a runtime index would
// put the accumulators in scratch memory).
template <int W>
__device__ __forceinline__ void reduce_own(const f32x4 (&acc)[4][2], f32x4 (&fin)[2], const f32x4* red, int lane) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    f32x4 sum = acc[W][t];
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) {
      if (ww == W) continue;
      const f32x4 x = red[(red_slot(ww, W) * 2 + t) * 64 + lane];
      sum[0] += x[0]; sum[1] += x[1]; sum[2] += x[2]; sum[3] += x[3];
    }
    fin[t] = sum;
  }
}
__device__ __forceinline__ void reduce_waves(const f32x4 (&acc)[4][2], f32x4 (&fin)[2], char* work) {
  f32x4* red = reinterpret_cast<f32x4*>(work);          // [4 waves][3 row tiles][2 t][64 lanes]
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  if (w < 4) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt == w) continue;
#pragma unroll
      for (int t = 0; t < 2; ++t) red[(red_slot(w, mt) * 2 + t) * 64 + lane] = acc[mt][t];
    }
  }
  block_sync();
  switch (w) {
    case 0: reduce_own<0>(acc, fin, red, lane); break;
    case 1: reduce_own<1>(acc, fin, red, lane); break;
    case 2: reduce_own<2>(acc, fin, red, lane); break;
    case 3: reduce_own<3>(acc, fin, red, lane); break;
    default: break;
  }
  block_sync();
}

// Small shared values live after the reduction area of the work region:
// +0 the last-arriver flag, +16, +20 and +24 the LDS arrival counters of the
// full-K GEMM waves (zeroed by every grid barrier), +256 the row scales.
constexpr int kWorkSmall = 24 * 1024;

// 1/rms of rows 0..63 into rr[] from the per-tile sums of squares, by wave rw.
__device__ __forceinline__ void row_scales(CP& p, const float* ss, float* rr, int rw) {
  const int t = threadIdx.x - 64 * rw;
  if (t >= 0 && t < 64) {
    const int nt = p.d / 32;                       // tiles per row, a multiple of 8
    const int nc = nt / 4;                         // 16-byte chunks per row, at most 8
    float4 c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = __builtin_bit_cast(float4, ldn16(ss, (t * nt + 4 * min(i, nc - 1)) * 4));
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i < nc) s += (c[i].x + c[i].y) + (c[i].z + c[i].w);
    rr[t] = 1.0f / sqrtf(s / (float)p.d + p.eps);
  }
}

// ---------------------------------------------------------------------------
// The block that completes a residual column tile p: h_new = (h or 0) + bias
// + sum over the S partial slices (in slice order); store h_new, bf16(h_new
// (1 + gain)) and the tile's sums of h_new^2.  Rows 0..R-1 of the GEMM map to
// rows row0 + r of h.  Compute threads only.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void finish_tile(CP& p, int pt, int S, int R, int row0, bool add,
                                            const float* bias, const float* gain, bf16_t* a_out, float* ss_out) {
  const int t = threadIdx.x;                       // all 512 threads: row t / 8, columns 4 (t % 8) ..
  const int r = t / 8, cg = t % 8;
  const int c0 = 32 * pt + 4 * cg;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  float sq = 0.f;
  if (r < R) {
    const int hrow = row0 + r;
    const int hoff = (hrow * p.d + c0) * 4;
    // every load unconditional (slice index clamped; the extra slices are not
    // added): with loads guarded by s < S the compiler kept only the first
    // component of each 16-byte load
    const f32x4 hx = __builtin_bit_cast(f32x4, ld16(p.h, hoff));
    f32x4 ps[16];
#pragma unroll
    for (int s = 0; s < 16; ++s) ps[s] = __builtin_bit_cast(f32x4, ld16(p.part, ((min(s, S - 1) * 64 + r) * p.d + c0) * 4));
    f32x4 acc = add ? hx : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < 16; ++s)
      if (s < S) acc += ps[s];
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = acc[e];
    if (bias)
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += bias[c0 + e];
    st16(p.h, hoff, u32x4{__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                          __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])});
    st8(a_out, (hrow * p.d + c0) * 2,
        u32x2{pack_bf16x2(v[0] * (1.f + gain[c0]), v[1] * (1.f + gain[c0 + 1])),
              pack_bf16x2(v[2] * (1.f + gain[c0 + 2]), v[3] * (1.f + gain[c0 + 3]))});
#pragma unroll
    for (int e = 0; e < 4; ++e) sq += v[e] * v[e];
  }
  sq += __shfl_xor(sq, 1, 64);
  sq += __shfl_xor(sq, 2, 64);
  sq += __shfl_xor(sq, 4, 64);
  if (r < R && cg == 0) stf(ss_out, ((row0 + r) * (p.d / 32) + pt) * 4, sq);
}

enum ResidKind { RK_TIME = 0, RK_OPROJ = 1, RK_DOWN = 2 };

// K slices of a residual GEMM: whole k-blocks per slice, at most 16 slices and
// at most 256 blocks in all.
__device__ __forceinline__ int resid_split(CP& p, int kind) {
  const int nkb = kind == RK_TIME ? p.d / 64 : kind == RK_OPROJ ? p.nq * p.D / 64 : p.F / 64;
  int s = 1;
  for (int c = 16; c >= 1; c >>= 1)
    if (nkb % c == 0 && c * (p.d / 32) <= kBlocks) { s = c; break; }
  return s;
}

// LDS copies a block starts one phase ahead (into the slot the coming phase
// reads), so that its weights are on chip when that phase begins.
enum PfKind { PF_NONE = 0, PF_TIME, PF_QKV, PF_OPROJ, PF_GATEUP, PF_DOWN };
__device__ __forceinline__ void issue_prefetch(CP& p, int kind, int l, int slot, int cw0 = 4) {
  if (threadIdx.x < 64 * cw0 || kind == PF_NONE) return;
  char* dst = g_lds + slot * kSlot;
  const int b = blockIdx.x;
  if (kind == PF_TIME || kind == PF_OPROJ || kind == PF_DOWN) {
    const int rk = kind == PF_TIME ? RK_TIME : kind == PF_OPROJ ? RK_OPROJ : RK_DOWN;
    const int S = resid_split(p, rk), NPT = p.d / 32;
    if (b >= NPT * S) return;
    const int K = rk == RK_TIME ? p.d : rk == RK_OPROJ ? p.nq * p.D : p.F;
    const void* W = rk == RK_TIME ? p.time_w2 : rk == RK_OPROJ ? lay(p, l).o : lay(p, l).down;
    const int nkb = K / 64, nks = nkb / S, pt = b % NPT, s = b / NPT;
    copy_weights(W, ((int64_t)pt * nkb + s * nks) * 4096, nks * 4096, dst, cw0);
  } else {
    const int npt = kind == PF_QKV ? (p.nq + 2) * p.D / 32 : 2 * p.F / 32;
    if (b >= npt) return;
    const int nkb = p.d / 64;
    copy_weights(kind == PF_QKV ? lay(p, l).qkv : lay(p, l).gu, (int64_t)b * nkb * 4096, nkb * 4096, dst, cw0);
  }
}

// ---------------------------------------------------------------------------
// Residual GEMM phase (O projection, down projection, time-MLP second layer):
// block b takes pair tile pt = b % NPT and K slice s = b / NPT of S slices;
// partial sums go to part[s]; the block completing tile pt finishes it.
// ---------------------------------------------------------------------------
template <int NK>
__device__ __attribute__((noinline)) void phase_resid(const PersistArgs* pa, int kind_, int r_, int l_, int rslot,
                                                      int pf_kind, int pf_l, int pslot) {
  CP& p = uargs(pa);
  const int kind = uni(kind_), r = uni(r_), l = uni(l_);
  const int S = resid_split(p, kind);
  issue_prefetch(p, uni(pf_kind), uni(pf_l), uni(pslot));
  const void* W;
  const bf16_t* A;
  int K, R, row0;
  bool add;
  const float *bias, *gain;
  unsigned* tile_ctr;
  int site;
  if (kind == RK_TIME) {
    W = p.time_w2; A = z_of(p, r); K = p.d; R = p.H; row0 = p.off; add = false; bias = p.time_b2;
    gain = lay(p, 0).attn_norm; tile_ctr = p.ctr + kTileTime; site = site_of(p, r, 0, 0);
  } else if (kind == RK_OPROJ) {
    W = lay(p, l).o; A = o_of(p, r, l); K = p.nq * p.D; R = p.M; row0 = 0; add = true; bias = nullptr;
    gain = lay(p, l).mlp_norm; tile_ctr = p.ctr + kTileO; site = site_of(p, r, l, 1);
  } else {
    W = lay(p, l).down; A = g_of(p, r, l); K = p.F; R = p.M; row0 = 0; add = true; bias = nullptr;
    gain = l + 1 < p.L ? lay(p, l + 1).attn_norm : p.final_norm; tile_ctr = p.ctr + kTileDown;
    site = site_of(p, r, l + 1, 0);
  }
  const int lda = K;
  const int NPT = p.d / 32;
  const int nkb = K / 64, nks = nkb / S;
  const int b = blockIdx.x;
  const bool active = b < NPT * S;
  const int pt = b % NPT, s = b / NPT;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const char* slot = g_lds + uni(rslot) * kSlot;
  char* work = g_lds + 2 * kSlot;
  f32x4 acc[4][2] = {};
  if (active && w < 4) {
    const int per = (nks + 3) / 4;
    const int kb0 = s * nks + w * per;
    const int nk = min(per, s * nks + nks - kb0);
    if (nk > 0) wave_gemm<NK>(A, lda, R, kb0, nk, slot, s * nks, acc);
  }
  f32x4 fin[2];
  reduce_waves(acc, fin, work);
  int& last = *reinterpret_cast<int*>(work + kWorkSmall);
  if (active && w < 4) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 16 * w + 4 * (lane / 16) + v;
      if (row < R) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
          stf(p.part, ((s * 64 + row) * p.d + 32 * pt + 16 * t + lane % 16) * 4, fin[t][v]);
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  block_sync();
  if (threadIdx.x == 0) {
    int l = 0;
    if (active) {
      const unsigned old = __hip_atomic_fetch_add(tile_ctr + pt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      l = ((old + 1) % S) == 0;
    }
    last = l;
  }
  block_sync();
  if (last) finish_tile(p, pt, S, R, row0, add, bias, gain, a_of(p, site), ss_of(p, site));
}

template <int D>
__device__ __forceinline__ int kswz(int key) {
  constexpr int CPR = D / 8;
  if constexpr (CPR >= 16) return key % 16;
  else return (key / (16 / CPR)) % CPR;
}

// The K and V^T tiles of this block's attention (key tile s = b / nq) into
// `dst`, copied by waves cw0 .. 7: K [64 keys][D] with chunk pos ^ kswz(key), V^T
// [D][64 keys] with chunk pos ^ ((d / 2) % 8).  mode 1: only a tile that lies
// wholly in the prefix (it can be copied before the layer's QKV); mode 2: only
// a tile that holds suffix keys (copied once the QKV has written them).
template <int D>
__device__ __forceinline__ void copy_key_tile(CP& p, int l, int P, int mode, char* dst, int cw0 = 4) {
  constexpr int CPR = D / 8;
  const int ntile = (P + p.M + 63) / 64;
  const int b = blockIdx.x;
  if (threadIdx.x < 64 * cw0 || b >= p.nq * ntile) return;
  const int s = b / p.nq;
  const bool prefix_only = 64 * s + 64 <= P;
  if (prefix_only != (mode == 1)) return;
  const int dw = threadIdx.x / 64 - cw0, lane = threadIdx.x % 64, ncw = 8 - cw0;
  const char* kl = reinterpret_cast<const char*>(p.kall + (int64_t)l * p.kv_layer + (int64_t)64 * s * D);
  const char* vl = reinterpret_cast<const char*>(p.vt + (int64_t)l * p.kv_layer + 64 * s);
  char* kt = dst;
  char* vtt = dst + 64 * D * 2;
  for (int n = dw; n < (64 * D * 2) / 1024; n += ncw) {
    const int ci = n * 64 + lane;
    const int key = ci / CPR, pos = ci % CPR;
    dma16(kl + (key * D + 8 * (pos ^ kswz<D>(key))) * 2, (lds_void_t*)(kt + n * 1024));
  }
  for (int n = dw; n < (D * 64 * 2) / 1024; n += ncw) {
    const int ci = n * 64 + lane;
    const int d = ci / 8, pos = ci % 8;
    dma16(vl + ((int64_t)d * p.ldk + 8 * (pos ^ ((d / 2) % 8))) * 2, (lds_void_t*)(vtt + n * 1024));
  }
}

// ---------------------------------------------------------------------------
// QKV phase (block = pair tile): n = a / rms, q|k|v = n W, RoPE on q and k at
// positions prefix_len + token; q to p.q, k and v into the layer's key range.
// ---------------------------------------------------------------------------
template <int D, int NK>
__device__ __attribute__((noinline)) void phase_qkv(const PersistArgs* pa, int r_, int l_, int P_, int rslot, int pslot) {
  CP& p = uargs(pa);
  const int r = uni(r_), l = uni(l_), P = uni(P_);
  const int site = site_of(p, r, l, 0);
  bf16_t* qo = q_of(p, r, l);
  const int npt = (p.nq * D + 2 * D) / 32;
  const int nkb = p.d / 64;
  const int nw = full_k_waves(nkb);
  const int b = blockIdx.x;
  const bool active = b < npt;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  char* slot = g_lds + uni(rslot) * kSlot;
  char* work = g_lds + 2 * kSlot;
  float* rr = reinterpret_cast<float*>(work + kWorkSmall + 256);
  const int tiles = D / 32;
  const int head = b / tiles, i = 16 * (b % tiles) + lane % 16;
  const bool rope = p.rope_cs && head <= p.nq;
  float2* csl = reinterpret_cast<float2*>(work);   // RoPE factors [64 rows][16 columns]
  unsigned* cnt = reinterpret_cast<unsigned*>(work + kWorkSmall + 16);
  // wave 7: the RoPE factors of the block's 16 column pairs into LDS, then
  // (waves 6 and 7) the attention's prefix-only key tiles for the next phase
  if (active && rope && w == 7) {
    float2 c[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int e = min(lane + 64 * j, p.M * 16 - 1);
      c[j] = __builtin_bit_cast(float2, ldn8(p.rope_cs, ((e / 16) * (D / 2) + 16 * (b % tiles) + e % 16) * 8));
    }
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (lane + 64 * j < p.M * 16) csl[lane + 64 * j] = c[j];
    if (lane == 0) __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  if (active && w >= 6) lds_wait(cnt + 2, nw, p.ctr);
  copy_key_tile<D>(p, l, P, 1, g_lds + uni(pslot) * kSlot, 6);
  if (!active) return;
  f32x4 acc[4][2] = {};
  if (w < nw) {
    int kb0, nk;
    full_k_split(nkb, w, kb0, nk);
    wave_gemm_full<NK>(a_of(p, site), p.d, p.M, kb0, nk, slot, acc, cnt + 2);
    row_scales(p, ss_of(p, site), rr, nw - 1);
  }
  f32x4 fin[2];
  if (!reduce_gemm_waves(acc, fin, slot, nw + (rope ? 1 : 0), nw, cnt, p.ctr)) return;
  bf16_t* kl = p.kall + (int64_t)l * p.kv_layer;
  bf16_t* vl = p.vt + (int64_t)l * p.kv_layer;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int tok = 16 * w + 4 * (lane / 16) + v;
    if (tok >= p.M) continue;
    float x1 = fin[0][v] * rr[tok], x2 = fin[1][v] * rr[tok];
    if (rope) {
      const float2 cs = csl[tok * 16 + lane % 16];
      const float y1 = x1 * cs.x - x2 * cs.y, y2 = x2 * cs.x + x1 * cs.y;
      x1 = y1;
      x2 = y2;
    }
    if (head < p.nq) {
      const int off = (tok * p.nq * D + head * D + i) * 2;
      st2(qo, off, f32_to_bf16(x1));
      st2(qo, off + D, f32_to_bf16(x2));
    } else if (head == p.nq) {
      const int off = ((P + tok) * D + i) * 2;
      st2(kl, off, f32_to_bf16(x1));
      st2(kl, off + D, f32_to_bf16(x2));
    } else {
      st2(vl, (i * p.ldk + P + tok) * 2, f32_to_bf16(x1));
      st2(vl, ((i + D / 2) * p.ldk + P + tok) * 2, f32_to_bf16(x2));
    }
  }
}

// ---------------------------------------------------------------------------
// Gate/up phase (block = pair tile of gate column 16p + c and up column 16p + c):
// g = gelu_tanh(n W_g) * (n W_u) with n = a / rms.
// ---------------------------------------------------------------------------
template <int NK>
__device__ __attribute__((noinline)) void phase_gateup(const PersistArgs* pa, int r_, int l_, int rslot, int pf_kind,
                                                       int pf_l, int pslot) {
  CP& p = uargs(pa);
  const int r = uni(r_), l = uni(l_);
  const int site = site_of(p, r, l, 1);
  bf16_t* go = g_of(p, r, l);
  const int npt = 2 * p.F / 32;
  const int nkb = p.d / 64;
  const int nw = full_k_waves(nkb);
  const int b = blockIdx.x;
  const bool active = b < npt;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  char* slot = g_lds + uni(rslot) * kSlot;
  char* work = g_lds + 2 * kSlot;
  float* rr = reinterpret_cast<float*>(work + kWorkSmall + 256);
  unsigned* cnt = reinterpret_cast<unsigned*>(work + kWorkSmall + 16);
  if (active && w >= 6) lds_wait(cnt + 2, nw, p.ctr);
  issue_prefetch(p, uni(pf_kind), uni(pf_l), uni(pslot), 6);
  if (!active) return;
  f32x4 acc[4][2] = {};
  if (w < nw) {
    int kb0, nk;
    full_k_split(nkb, w, kb0, nk);
    wave_gemm_full<NK>(a_of(p, site), p.d, p.M, kb0, nk, slot, acc, cnt + 2);
    row_scales(p, ss_of(p, site), rr, nw - 1);
  }
  f32x4 fin[2];
  if (!reduce_gemm_waves(acc, fin, slot, nw, nw, cnt, p.ctr)) return;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int tok = 16 * w + 4 * (lane / 16) + v;
    if (tok >= p.M) continue;
    const float gate = fin[0][v] * rr[tok], up = fin[1][v] * rr[tok];
    st2(go, (tok * p.F + 16 * b + lane % 16) * 2, f32_to_bf16(gelu_tanh_f(gate) * up));
  }
}

// ---------------------------------------------------------------------------
// Attention phase: block (key tile s, head h) computes the softmax partial of
// its 64 keys for the head's query rows (the suffix tokens, one per row; wave
// w takes tokens 16w .. 16w+15).  S = Q K^T and O = P V on 16x16x32 MFMAs;
// K [key][D] and V^T [D][key] tiles in LDS with XOR-swizzled 16-byte chunks;
// P staged in LDS to become the A operand.  Masks: keys at or beyond
// prefix_len + M; with a state token, the state row sees the prefix and itself.
// Output: O normalised by its own sum (bf16) and (max, sum) in the log2 domain.
// ---------------------------------------------------------------------------
template <int D>
__device__ __attribute__((noinline)) void phase_attn(const PersistArgs* pa, int r_, int l_, int P_, int ntile_,
                                                     int rslot) {
  CP& p = uargs(pa);
  const bf16_t* qi = q_of(p, uni(r_), uni(l_));
  char* lds = g_lds + uni(rslot) * kSlot;
  const int l = uni(l_), P = uni(P_), ntile = uni(ntile_);
  const bool state_mask = p.e_state != nullptr;
  constexpr int CPR = D / 8;                       // 16-byte chunks per K row
  const int nkeys = P + p.M;
  const int b = blockIdx.x;
  const bool active = b < p.nq * ntile;
  const int s = b / p.nq, h = b % p.nq;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const char* kt = lds;                            // [64][D] bf16
  const char* vtt = lds + 64 * D * 2;              // [D][64] bf16
  char* work = g_lds + 2 * kSlot;
  copy_key_tile<D>(p, l, P, 2, lds);             // tiles holding suffix keys (the rest came earlier)
  // unconditional loads (inactive and copying waves read token 0 of head 0 and never use it)
  u32x4 qf[D / 32];
  {
    const int qtok = 16 * (w % 4) + lane % 16;
    const int t = active && qtok < p.M ? qtok : 0;
    const int hq = active ? h : 0;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) qf[ks] = ldn16(qi, (t * p.nq * D + hq * D + 32 * ks + 8 * (lane / 16)) * 2);
  }
  __builtin_amdgcn_s_waitcnt(0);
  block_sync();
  if (!active || w >= 4) return;

  // S = Q K^T: sacc[kt][v] = score of row 4 (lane / 16) + v, key 16 kt + lane % 16
  f32x4 sacc[4] = {};
#pragma unroll
  for (int ktile = 0; ktile < 4; ++ktile) {
    const int key = 16 * ktile + lane % 16;
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const int chunk = 4 * ks + lane / 16;
      const bf16x8 kb = *reinterpret_cast<const bf16x8*>(kt + (key * CPR + (chunk ^ kswz<D>(key))) * 16);
      sacc[ktile] = mfma16x16x32(__builtin_bit_cast(bf16x8, qf[ks]), kb, sacc[ktile]);
    }
  }
  // masks, row max and sum (log2 domain); a row lives in one group of 16 lanes
  const float sl2 = p.scale * kLog2e;
  float m[4], sum[4];
  bool ok[4][4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int tok = 16 * w + 4 * (lane / 16) + v;
    float mx = -3.0e38f;
#pragma unroll
    for (int ktile = 0; ktile < 4; ++ktile) {
      const int key = 64 * s + 16 * ktile + lane % 16;
      bool allowed = key < nkeys;
      if (state_mask && tok == 0 && key > P) allowed = false;
      ok[ktile][v] = allowed;
      sacc[ktile][v] *= sl2;
      if (allowed) mx = fmaxf(mx, sacc[ktile][v]);
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    m[v] = mx;
    float sm = 0.f;
#pragma unroll
    for (int ktile = 0; ktile < 4; ++ktile) {
      const float e = ok[ktile][v] ? exp2f(sacc[ktile][v] - mx) : 0.f;
      sacc[ktile][v] = e;
      sm += e;
    }
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) sm += __shfl_xor(sm, o, 64);
    sum[v] = sm;
  }
  // P (bf16) into this wave's staging rows: [16 rows][64 keys], chunk pos ^ ((row / 2) % 8)
  char* pst = work + w * 8192;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = 4 * (lane / 16) + v;
#pragma unroll
    for (int ktile = 0; ktile < 4; ++ktile) {
      const int key = 16 * ktile + lane % 16;
      const int chunk = key / 8;
      *reinterpret_cast<bf16_t*>(pst + row * 128 + (chunk ^ ((row / 2) % 8)) * 16 + (key % 8) * 2) =
          f32_to_bf16(sacc[ktile][v]);
    }
  }
  bf16x8 pf[2];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int row = lane % 16, chunk = 4 * ks + lane / 16;
    pf[ks] = *reinterpret_cast<const bf16x8*>(pst + row * 128 + (chunk ^ ((row / 2) % 8)) * 16);
  }
  // O = P V
  f32x4 oacc[D / 16] = {};
#pragma unroll
  for (int nt = 0; nt < D / 16; ++nt) {
    const int d = 16 * nt + lane % 16;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int chunk = 4 * ks + lane / 16;
      const bf16x8 vb = *reinterpret_cast<const bf16x8*>(vtt + (d * 8 + (chunk ^ ((d / 2) % 8))) * 16);
      oacc[nt] = mfma16x16x32(pf[ks], vb, oacc[nt]);
    }
  }
  // normalise, stage rows in LDS (this wave's region, after its P reads), store 16-byte chunks
  char* ost = work + w * 8192;                     // [16 rows][D] bf16
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int row = 4 * (lane / 16) + v;
    const float inv = sum[v] > 0.f ? 1.f / sum[v] : 0.f;
#pragma unroll
    for (int nt = 0; nt < D / 16; ++nt)
      *reinterpret_cast<bf16_t*>(ost + (row * D + 16 * nt + lane % 16) * 2) = f32_to_bf16(oacc[nt][v] * inv);
  }
  const int base = (h * ntile + s) * 64 + 16 * w;      // partial row of token 16w
  constexpr int CH = 16 * D / 8;                       // 16-byte chunks of the wave's rows
#pragma unroll
  for (int c = lane; c < CH; c += 64) {
    const int row = c / (D / 8), col = c % (D / 8);
    if (16 * w + row < p.M) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(ost + (row * D + 8 * col) * 2);
      st16(p.apart, ((base + row) * D + 8 * col) * 2, x);
    }
  }
  if (lane % 16 == 0) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int tok = 16 * w + 4 * (lane / 16) + v;
      if (tok < p.M)
        st8(p.aml, (base + 4 * (lane / 16) + v) * 8,
            u32x2{__builtin_bit_cast(uint32_t, m[v]), __builtin_bit_cast(uint32_t, sum[v])});
    }
  }
}

// Merge the key-tile partials of (head h, tokens 4 g .. 4 g + 3) in tile
// order: o = sum_s w_s o_s / sum_s w_s, w_s = sum_s 2^(m_s - max m), taken in
// chunks of 8 tiles whose loads are all issued first (running maximum
// rescaled between chunks).
template <int D>
__device__ __attribute__((noinline)) void phase_merge(const PersistArgs* pa, int r_, int l_, int ntile_, int pf_kind,
                                                      int pf_l, int pslot) {
  CP& p = uargs(pa);
  bf16_t* oo = o_of(p, uni(r_), uni(l_));
  const int ntile = uni(ntile_);
  issue_prefetch(p, uni(pf_kind), uni(pf_l), uni(pslot));
  constexpr int E = D / 64;                        // elements per thread
  const int ng = (p.M + 3) / 4;
  const int b = blockIdx.x;
  if (b >= p.nq * ng || threadIdx.x >= 256) return;
  const int h = b % p.nq, grp = b / p.nq;
  const int tok = 4 * grp + threadIdx.x / 64;
  const int e0 = (threadIdx.x % 64) * E;
  if (tok >= p.M) return;
  float mx = -3.0e38f, den = 0.f;
  float acc[E] = {};
  for (int s0 = 0; s0 < ntile; s0 += 8) {
    float2 ml[8];
    float x[8][E];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = (h * ntile + min(s0 + i, ntile - 1)) * 64 + tok;
      ml[i] = ld8f(p.aml, row * 8);
      if constexpr (E == 4) {
        const uint2 v = ld8u(p.apart, (row * D + e0) * 2);
        x[i][0] = bf16_to_f32(v.x & 0xffff); x[i][1] = bf16_to_f32(v.x >> 16);
        x[i][2] = bf16_to_f32(v.y & 0xffff); x[i][3] = bf16_to_f32(v.y >> 16);
      } else if constexpr (E == 2) {
        const uint32_t v = ld4(p.apart, (row * D + e0) * 2);
        x[i][0] = bf16_to_f32(v & 0xffff); x[i][1] = bf16_to_f32(v >> 16);
      } else {
        x[i][0] = bf16_to_f32(ld2(p.apart, (row * D + e0) * 2));
      }
    }
    float cm = -3.0e38f;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (s0 + i < ntile && ml[i].y > 0.f) cm = fmaxf(cm, ml[i].x);
    const float nm = fmaxf(mx, cm);
    const float r = exp2f(mx - nm);
    den *= r;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= r;
    mx = nm;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (!(s0 + i < ntile && ml[i].y > 0.f)) continue;
      const float wgt = ml[i].y * exp2f(ml[i].x - mx);
      den += wgt;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] += wgt * x[i][e];
    }
  }
  const float inv = 1.f / den;
  const int off = (tok * p.nq * D + h * D + e0) * 2;
  if constexpr (E == 4) st8(oo, off, u32x2{pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)});
  else if constexpr (E == 2) st4(oo, off, pack_bf16x2(acc[0] * inv, acc[1] * inv));
  else st2(oo, off, f32_to_bf16(acc[0] * inv));
}

// The state row (token 0) at the start of a step: h = e_state, a = bf16(h (1 +
// w_attn of block 0)), per-tile sums of squares.  All 256 compute threads.
__device__ __forceinline__ void state_row(CP& p, int k) {
  bf16_t* a0 = a_of(p, site_of(p, k, 0, 0));
  float* ss0 = ss_of(p, site_of(p, k, 0, 0));
  const int t = threadIdx.x;
  const int cpt = p.d / 256;                       // columns per thread (1..4)
  const float* w0 = lay(p, 0).attn_norm;
  float sq = 0.f;
  for (int j = 0; j < cpt; ++j) {
    const int c = t * cpt + j;
    const float v = p.e_state[c];
    stf(p.h, c * 4, v);
    st2(a0, c * 2, f32_to_bf16(v * (1.f + w0[c])));
    sq += v * v;
  }
  // a 32-column tile spans 32 / cpt consecutive threads
  for (int o = 1; o < 32 / cpt; o <<= 1) sq += __shfl_xor(sq, o, 64);
  if ((t * cpt) % 32 == 0) stf(ss0, ((t * cpt) / 32) * 4, sq);
}

// Action embedding of row j for step k: z = swish(x W' + b' + T[k]) (the
// action projection folded into the time MLP's first layer).  xs in LDS.
__device__ __forceinline__ void embed_row(CP& p, int j, int k, int r, const float* xs) {
  for (int g = threadIdx.x; g < p.d / 4; g += 256) {
    const int c = 4 * g;
    const float4 tb = *reinterpret_cast<const float4*>(p.tin_b + c);
    const float4 tt = *reinterpret_cast<const float4*>(p.T + (int64_t)k * p.d + c);
    float y[4] = {tb.x + tt.x, tb.y + tt.y, tb.z + tt.z, tb.w + tt.w};
    for (int a0 = 0; a0 < p.A; a0 += 8) {
      float4 w[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) w[i] = *reinterpret_cast<const float4*>(p.tin_w + min(a0 + i, p.A - 1) * p.d + c);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        if (a0 + i < p.A) {
          const float xa = xs[a0 + i];
          y[0] = fmaf(xa, w[i].x, y[0]); y[1] = fmaf(xa, w[i].y, y[1]);
          y[2] = fmaf(xa, w[i].z, y[2]); y[3] = fmaf(xa, w[i].w, y[3]);
        }
    }
    st8(z_of(p, r), (j * p.d + c) * 2, u32x2{pack_bf16x2(swish_f(y[0]), swish_f(y[1])), pack_bf16x2(swish_f(y[2]), swish_f(y[3]))});
  }
}

// Embedding of the launch's first step k0: block j < H embeds action row j
// from x (the noise, or the previous launch's result); block H resets the
// state row.
__device__ __attribute__((noinline)) void phase_embed0(const PersistArgs* pa, int k0_, int pslot) {
  CP& p = uargs(pa);
  const int k0 = uni(k0_);
  char* lds = g_lds;
  issue_prefetch(p, PF_TIME, 0, uni(pslot));
  float* xs = reinterpret_cast<float*>(lds + 2 * kSlot);
  const int b = blockIdx.x;
  const bool cw = threadIdx.x < 256;
  if (b < p.H && threadIdx.x < p.A) xs[threadIdx.x] = ldf(p.x, (b * p.A + threadIdx.x) * 4);
  block_sync();
  if (b < p.H && cw) embed_row(p, b, k0, 0, xs);
  else if (b == p.H && p.e_state && cw) state_row(p, 0);
}

// Readout of step k, the launch's r-th (block j < H, action row j = h row
// off + j): final norm (fp32, from h), v = n W_out + b_out, x += dt v; then
// the next step's embedding of the row when this launch runs it (k + 1 < k1),
// and the output after the last step K - 1.  Block H resets the state row.
// Every thread reaches every block barrier.
__device__ __attribute__((noinline)) void phase_readout(const PersistArgs* pa, int k_, int r_, int k1_, int K_,
                                                        int pslot) {
  CP& p = uargs(pa);
  const int k = uni(k_), r = uni(r_), k1 = uni(k1_), K = uni(K_);
  if (k + 1 < k1) issue_prefetch(p, PF_TIME, 0, uni(pslot));
  char* work = g_lds + 2 * kSlot;
  float* nrm = reinterpret_cast<float*>(work);                   // [d]
  float* vel = nrm + 1024;                                       // [64]
  float* xs = vel + 64;                                          // [64]
  float* rsh = xs + 64;
  const int b = blockIdx.x;
  const bool row = b < p.H;
  const int hrow = p.off + b;
  const int w = threadIdx.x / 64, lane = threadIdx.x % 64;
  const int d = p.d, A = p.A;
  // the row (four columns per thread) and its 1/rms, requested together
  float4 hv = {0.f, 0.f, 0.f, 0.f}, fn = {0.f, 0.f, 0.f, 0.f};
  const int c0 = 4 * threadIdx.x;
  if (row && c0 < d) {
    hv = __builtin_bit_cast(float4, ld16(p.h, (hrow * d + c0) * 4));
    fn = *reinterpret_cast<const float4*>(p.final_norm + c0);
  }
  if (row && threadIdx.x < 64) {
    const int nt = d / 32;
    float s = threadIdx.x < nt ? ldnf(ss_of(p, site_of(p, r, p.L, 0)), (hrow * nt + threadIdx.x) * 4) : 0.f;
    s = wave_sum(s);
    if (threadIdx.x == 0) *rsh = 1.0f / sqrtf(s / (float)d + p.eps);
  }
  block_sync();
  if (row && c0 < d) {
    const float rs = *rsh;
    nrm[c0] = hv.x * rs * (1.f + fn.x);
    nrm[c0 + 1] = hv.y * rs * (1.f + fn.y);
    nrm[c0 + 2] = hv.z * rs * (1.f + fn.z);
    nrm[c0 + 3] = hv.w * rs * (1.f + fn.w);
  }
  block_sync();
  // v_a = n . W_out[a]: wave w takes outputs a = w, w + 4, ...; lane l the
  // columns 4 l + 256 i (d <= 1024), all of an output's loads at once
  if (row && w < 4) {
    for (int a = w; a < A; a += 4) {
      float4 wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = min(4 * lane + 256 * i, d - 4);
        wv[i] = *reinterpret_cast<const float4*>(p.out_w + a * d + c);
      }
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = 4 * lane + 256 * i;
        if (c < d) {
          acc = fmaf(nrm[c], wv[i].x, acc);
          acc = fmaf(nrm[c + 1], wv[i].y, acc);
          acc = fmaf(nrm[c + 2], wv[i].z, acc);
          acc = fmaf(nrm[c + 3], wv[i].w, acc);
        }
      }
      acc = wave_sum(acc);
      if (lane == 0) vel[a] = acc;
    }
  }
  block_sync();
  if (row && threadIdx.x < A) {
    const int xi = (b * A + threadIdx.x) * 4;
    const float xn = ldf(p.x, xi) + p.dt[k] * (vel[threadIdx.x] + p.out_b[threadIdx.x]);
    stf(p.x, xi, xn);
    xs[threadIdx.x] = xn;
    if (k + 1 == K) p.desc->out[b * A + threadIdx.x] = xn;
  }
  block_sync();
  if (row && w < 4 && k + 1 < k1) embed_row(p, b, k + 1, r + 1, xs);
  else if (b == p.H && p.e_state && w < 4 && k + 1 < k1) state_row(p, r + 1);
}

template <int D, int NKD>
__global__ __launch_bounds__(kThreads, 1) void persist_kernel(const PersistArgs* __restrict__ pa, int k0, int k1,
                                                               int K) {
  CP& p = uargs(pa);
  unsigned gen = 0;
  const int P = p.desc->prefix_len[0];
  const int ntile = (P + p.M + 63) / 64;
  auto resid = [&](int kind, int k, int l, int rslot, int pf_kind, int pf_l, int pslot) {
    const int K_ = kind == RK_TIME ? p.d : kind == RK_OPROJ ? p.nq * D : p.F;
    const int nks = K_ / 64 / resid_split(p, kind);
    if (nks <= 4) phase_resid<1>(pa, kind, k, l, rslot, pf_kind, pf_l, pslot);
    else if (nks <= 8) phase_resid<2>(pa, kind, k, l, rslot, pf_kind, pf_l, pslot);
    else phase_resid<4>(pa, kind, k, l, rslot, pf_kind, pf_l, pslot);
  };
  // LDS slots: every phase that reads weights (or key tiles) reads the slot
  // opposite the previous such phase; the phase just before it fills that slot.
  int cur = 0;
  phase_embed0(pa, k0, cur);
  grid_sync(p.ctr, gen);
  for (int k = k0; k < k1; ++k) {
    const int r = k - k0;
    resid(RK_TIME, r, 0, cur, PF_QKV, 0, cur ^ 1);      // u = z W2 + b2 into the action rows of h
    cur ^= 1;
    grid_sync(p.ctr, gen);
    for (int l = 0; l < p.L; ++l) {
      phase_qkv<D, NKD>(pa, r, l, P, cur, cur ^ 1);
      cur ^= 1;
      grid_sync(p.ctr, gen);
      phase_attn<D>(pa, r, l, P, ntile, cur);
      grid_sync(p.ctr, gen);
      phase_merge<D>(pa, r, l, ntile, PF_OPROJ, l, cur ^ 1);
      cur ^= 1;
      grid_sync(p.ctr, gen);
      resid(RK_OPROJ, r, l, cur, PF_GATEUP, l, cur ^ 1);
      cur ^= 1;
      grid_sync(p.ctr, gen);
      phase_gateup<NKD>(pa, r, l, cur, PF_DOWN, l, cur ^ 1);
      cur ^= 1;
      grid_sync(p.ctr, gen);
      resid(RK_DOWN, r, l, cur, l + 1 < p.L ? PF_QKV : PF_NONE, l + 1, cur ^ 1);
      cur ^= 1;
      grid_sync(p.ctr, gen);
    }
    phase_readout(pa, k, r, k1, K, cur);
    grid_sync(p.ctr, gen);
  }
  // a barrier that gave up: make the failure visible in the output
  if (blockIdx.x == 0 && ld_ctr(p.ctr + kErr))
    for (int i = threadIdx.x; i < p.H * p.A; i += kThreads) p.desc->out[i] = __builtin_nanf("");
}

}  // namespace

bool persist_supported(int d, int D, int nq, int F, int M, int A) {
  if (D != 64 && D != 128 && D != 256) return false;
  if (d % 256 != 0 || d > 1024 || F % 512 != 0 || F > 32 * kBlocks / 2) return false;
  if ((nq * D) % 256 != 0 || (nq + 2) * D / 32 > kBlocks) return false;
  if (M > 64 || A > 64 || M < 1) return false;
  return true;
}

hipError_t persist_launch(const PersistArgs& a, const PersistArgs* dev_args, int k0, int k1, int K, hipStream_t s) {
  void* args[] = {const_cast<PersistArgs**>(&dev_args), &k0, &k1, &K};
  const int nkb = a.d / 64;
  const int nw = nkb < 6 ? nkb : 6;
  const int nkd = (nkb + nw - 1) / nw;             // k-blocks per wave of the full-K GEMMs (1..3)
  void* fn = nullptr;
  auto pick = [&](auto dd) {
    constexpr int DD = decltype(dd)::value;
    if (nkd <= 1) fn = (void*)persist_kernel<DD, 1>;
    else if (nkd <= 2) fn = (void*)persist_kernel<DD, 2>;
    else fn = (void*)persist_kernel<DD, 3>;
  };
  if (a.D == 64) pick(std::integral_constant<int, 64>{});
  else if (a.D == 128) pick(std::integral_constant<int, 128>{});
  else pick(std::integral_constant<int, 256>{});
  return hipLaunchCooperativeKernel(fn, dim3(kBlocks), dim3(kThreads), args, 0, s);
}

}  // namespace phyai
