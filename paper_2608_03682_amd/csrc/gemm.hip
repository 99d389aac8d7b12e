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

namespace phyai {

namespace {

constexpr int kMT = 4;           // 16-row MFMA tiles per block (64 rows)
constexpr int kNP = 2;           // pair tiles per block (64 columns)
constexpr int kNT = 2 * kNP;     // 16-column MFMA tiles per block

// One block = 4 waves computing a 64 x 64 output tile; the K range is split
// between the 4 waves and their partial sums are added through LDS.
template <class Epi, bool FP8, bool SPLIT>
__global__ __launch_bounds__(256) void gemm_mfma_kernel(GemmArgs g, Epi epi) {
  __shared__ float red[4][kMT * kNT * 4][kWave];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int pt0 = blockIdx.x * kNP;
  const int m0 = blockIdx.y * 16 * kMT;
  const bf16_t* A = g.A_ind ? static_cast<const bf16_t*>(*g.A_ind) + g.a_off
                            : static_cast<const bf16_t*>(g.A);
  const int nkb = g.K / 64;
  const int kb0 = wave * nkb / 4, kb1 = (wave + 1) * nkb / 4;
  const int arow = lane % 16, akg = lane / 16;

  // rows this lane loads A for, with validity
  const bf16_t* arp[kMT];
  const bf16_t* alp[kMT];
  bool aval[kMT];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    const int row = m0 + 16 * mt + arow;
    bool ok = row < g.R;
    if (ok && g.rows_per_req > 0) {
      const int b = row / g.rows_per_req;
      ok = (row % g.rows_per_req) < g.desc->prefix_len[b];
    }
    aval[mt] = ok;
    arp[mt] = A + (int64_t)(ok ? row : 0) * g.lda + akg * 8;
    alp[mt] = SPLIT ? static_cast<const bf16_t*>(g.A_lo) + (int64_t)(ok ? row : 0) * g.lda + akg * 8 : nullptr;
  }

  f32x4 acc[kMT][kNT];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int t = 0; t < kNT; ++t) acc[mt][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kb = kb0; kb < kb1; ++kb) {
    bf16x8 b[kNT][2];
#pragma unroll
    for (int t = 0; t < kNT; ++t) {
      const int p = pt0 + t / 2, hf = t % 2;
      const int64_t frag = ((int64_t)(p * nkb + kb) * 2 + hf) * kWave + lane;
      if (p >= g.NPT) {
        b[t][0] = as_bf16x8(make_uint4(0, 0, 0, 0));
        b[t][1] = b[t][0];
      } else if (FP8) {
        const uint4 v = static_cast<const uint4*>(g.W)[frag];
        b[t][0] = fp8x8_to_bf16x8(v.x, v.y);
        b[t][1] = fp8x8_to_bf16x8(v.z, v.w);
      } else {
        const uint4* src = static_cast<const uint4*>(g.W) + frag * 2;
        b[t][0] = as_bf16x8(src[0]);
        b[t][1] = as_bf16x8(src[1]);
      }
    }
    bf16x8 a[kMT][2], al[kMT][2];
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        uint4 v = make_uint4(0, 0, 0, 0), w = make_uint4(0, 0, 0, 0);
        if (aval[mt]) {
          v = *reinterpret_cast<const uint4*>(arp[mt] + kb * 64 + s * 32);
          if (SPLIT) w = *reinterpret_cast<const uint4*>(alp[mt] + kb * 64 + s * 32);
        }
        a[mt][s] = as_bf16x8(v);
        al[mt][s] = as_bf16x8(w);
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
        for (int t = 0; t < kNT; ++t) {
          acc[mt][t] = mfma16x16x32(a[mt][s], b[t][s], acc[mt][t]);
          if (SPLIT) acc[mt][t] = mfma16x16x32(al[mt][s], b[t][s], acc[mt][t]);
        }
  }

#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int t = 0; t < kNT; ++t)
#pragma unroll
      for (int v = 0; v < 4; ++v) red[wave][(mt * kNT + t) * 4 + v][lane] = acc[mt][t][v];
  __syncthreads();

  // wave w finishes row tile w
  const int mt = wave;
  const int c = lane % 16;
#pragma unroll
  for (int pp = 0; pp < kNP; ++pp) {
    const int p = pt0 + pp;
    if (p >= g.NPT) break;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + 16 * mt + 4 * akg + v;
      float s0 = 0.f, s1 = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        s0 += red[w][(mt * kNT + 2 * pp) * 4 + v][lane];
        s1 += red[w][(mt * kNT + 2 * pp + 1) * 4 + v][lane];
      }
      if (g.scale) {
        s0 *= g.scale[32 * p + c];
        s1 *= g.scale[32 * p + 16 + c];
      }
      if (row < g.R) epi(row, p, c, s0, s1);
    }
  }
}

// fp32 path: weights stored [K][N] (packed column order), one thread per
// (row, column pair).
template <class Epi>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g, Epi epi) {
  const int c = threadIdx.x % 16, rr = threadIdx.x / 16;
  const int p = blockIdx.x;
  const int row = blockIdx.y * 16 + rr;
  if (row >= g.R) return;
  const float* A = g.A_ind ? static_cast<const float*>(*g.A_ind) + g.a_off
                           : static_cast<const float*>(g.A);
  bool ok = true;
  if (g.rows_per_req > 0) ok = (row % g.rows_per_req) < g.desc->prefix_len[row / g.rows_per_req];
  const float* a = A + (int64_t)row * g.lda;
  const float* w = static_cast<const float*>(g.W) + 32 * p + c;
  const int N = 32 * g.NPT;
  float s0 = 0.f, s1 = 0.f;
  if (ok) {
    for (int k = 0; k < g.K; ++k) {
      const float av = a[k];
      s0 = fmaf(av, w[(int64_t)k * N], s0);
      s1 = fmaf(av, w[(int64_t)k * N + 16], s1);
    }
  }
  epi(row, p, c, s0, s1);
}

template <class Epi>
void launch(const GemmArgs& g, const Epi& epi, hipStream_t s) {
  if (g.kind == W_F32) {
    dim3 grid(g.NPT, (g.R + 15) / 16);
    hipLaunchKernelGGL(gemm_f32_kernel<Epi>, grid, dim3(256), 0, s, g, epi);
  } else {
    dim3 grid((g.NPT + kNP - 1) / kNP, (g.R + 16 * kMT - 1) / (16 * kMT));
    const bool split = g.A_lo != nullptr;
    if (g.kind == W_FP8) {
      if (split) hipLaunchKernelGGL((gemm_mfma_kernel<Epi, true, true>), grid, dim3(256), 0, s, g, epi);
      else hipLaunchKernelGGL((gemm_mfma_kernel<Epi, true, false>), grid, dim3(256), 0, s, g, epi);
    } else {
      if (split) hipLaunchKernelGGL((gemm_mfma_kernel<Epi, false, true>), grid, dim3(256), 0, s, g, epi);
      else hipLaunchKernelGGL((gemm_mfma_kernel<Epi, false, false>), grid, dim3(256), 0, s, g, epi);
    }
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

}  // namespace phyai
