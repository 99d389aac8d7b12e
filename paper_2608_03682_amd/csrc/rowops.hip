// Row-wise kernels of the denoising loop: (ada)RMSNorm / adaLN normalisation,
// action and state embedding, the fused final-norm + output-projection +
// Euler update, and the per-call copies.
#include "kernels.hpp"

namespace phyai {

namespace {

constexpr int kMaxPer = 8;   // d <= 2048 with 256 threads

// n = normalise(h) * (1 + mul) + shift.  RMS: h / sqrt(mean(h^2) + eps);
// LN: (h - mean) / sqrt(var + eps).  Statistics in fp32.
// h row += gate * (sum of pending slices + bias), written back; returns the row in v.
// Every load is requested before any is used (slots past pd.n re-read the
// last slice and are dropped; element groups past d are skipped on a
// wave-uniform test), so the row costs one memory round trip, not one per
// slice.
__device__ __forceinline__ void load_row_with_pending(float* hr, int64_t row, int d, const PendingResid& pd,
                                                      float (&v)[kMaxPer]) {
  constexpr int kMaxSplit = 8;
  const int n = pd.n;
  float hv[kMaxPer], sl[kMaxPer][kMaxSplit], bs[kMaxPer], gt[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (256 * i >= d) break;
    const int c = threadIdx.x + 256 * i;
    const int cc = c < d ? c : d - 1;
    hv[i] = hr[cc];
    if (n > 0) {
#pragma unroll
      for (int s = 0; s < kMaxSplit; ++s) {
        const int ss = s < n ? s : n - 1;
        sl[i][s] = pd.part[ss * pd.stride + row * d + cc];
      }
      bs[i] = pd.bias ? pd.bias[cc] : 0.f;
      gt[i] = pd.gate ? pd.gate[cc] : 1.f;
    }
  }
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (256 * i >= d) {
      v[i] = 0.f;
      continue;
    }
    float x = hv[i];
    if (n > 0) {
      float t = 0.f;
#pragma unroll
      for (int s = 0; s < kMaxSplit; ++s) t += s < n ? sl[i][s] : 0.f;
      x += (t + bs[i]) * gt[i];
      if (c < d) hr[c] = x;
    }
    v[i] = c < d ? x : 0.f;
  }
}

template <typename OutT>
__global__ __launch_bounds__(256) void norm_rows_kernel(float* __restrict__ h, OutT* __restrict__ n,
                                                        OutT* __restrict__ n_lo, int d, float eps, int mode,
                                                        const float* __restrict__ mul,
                                                        const float* __restrict__ shift, PendingResid pend) {
  __shared__ float scratch[4];
  const int row = blockIdx.x;
  float* hr = h + (int64_t)row * d;
  // the norm's own factors first: they do not wait on the row, and landing
  // with it saves a round trip after the statistics
  float mv[kMaxPer], sv[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (256 * i >= d) break;
    const int c = threadIdx.x + 256 * i;
    const int cc = c < d ? c : d - 1;
    mv[i] = mul[cc];
    sv[i] = shift ? shift[cc] : 0.f;
  }
  float v[kMaxPer];
  load_row_with_pending(hr, row, d, pend, v);
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) s += v[i];
  float mu = 0.f;
  if (mode == NORM_LN) mu = block_sum<256>(s, scratch) / d;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int c = threadIdx.x + 256 * i;
    const float t = c < d ? v[i] - mu : 0.f;
    ss += t * t;
  }
  const float r = rsqrtf(block_sum<256>(ss, scratch) / d + eps);
  OutT* nr = n + (int64_t)row * d;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (c < d) {
      float t = (v[i] - mu) * r * (1.f + mv[i]);
      if (shift) t += sv[i];
      ActIO<OutT>::store(nr + c, t);
      if (n_lo) ActIO<OutT>::store(n_lo + (int64_t)row * d + c, t - ActIO<OutT>::round(t));
    }
  }
}

// The same normalisation for d = 1024 with one block of 256 threads per row,
// thread t holding the four consecutive columns 4t .. 4t+3: every load of the
// row (h, each pending slice, the factors) is one 16-byte request per thread
// and the normalised values leave in one store, where the scalar layout above
// needs four of each.
// Columns c .. c+3 of row `row` (c a multiple of 4) with the pending residual
// folded in and written back, as load_row_with_pending does for one column:
// every request (the row, each slice, bias, gate) is one 16-byte load.
__device__ __forceinline__ void load_row4_with_pending(float* hr, int64_t row, int d, int c, const PendingResid& pd,
                                                       float (&v)[4]) {
  constexpr int kMaxSplit = 8;
  const int np = pd.n;
  const float4 hv = *reinterpret_cast<const float4*>(hr + c);
  float4 sl[kMaxSplit], bs = make_float4(0.f, 0.f, 0.f, 0.f), gt = make_float4(1.f, 1.f, 1.f, 1.f);
  if (np > 0) {
#pragma unroll
    for (int sp = 0; sp < kMaxSplit; ++sp) {
      const int ss = sp < np ? sp : np - 1;
      sl[sp] = *reinterpret_cast<const float4*>(pd.part + ss * pd.stride + row * d + c);
    }
    if (pd.bias) bs = *reinterpret_cast<const float4*>(pd.bias + c);
    if (pd.gate) gt = *reinterpret_cast<const float4*>(pd.gate + c);
  }
  v[0] = hv.x; v[1] = hv.y; v[2] = hv.z; v[3] = hv.w;
  if (np > 0) {
    const float b4[4] = {bs.x, bs.y, bs.z, bs.w}, g4[4] = {gt.x, gt.y, gt.z, gt.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float t = 0.f;
#pragma unroll
      for (int sp = 0; sp < kMaxSplit; ++sp) {
        const float q = e == 0 ? sl[sp].x : e == 1 ? sl[sp].y : e == 2 ? sl[sp].z : sl[sp].w;
        t += sp < np ? q : 0.f;
      }
      v[e] += (t + b4[e]) * g4[e];
    }
    *reinterpret_cast<float4*>(hr + c) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <typename OutT>
__global__ __launch_bounds__(256) void norm_rows_v4_kernel(float* __restrict__ h, OutT* __restrict__ n,
                                                           OutT* __restrict__ n_lo, int d, float eps, int mode,
                                                           const float* __restrict__ mul,
                                                           const float* __restrict__ shift, PendingResid pend) {
  __shared__ float scratch[4];
  const int row = blockIdx.x;
  const int c = 4 * threadIdx.x;
  const float4 mv = *reinterpret_cast<const float4*>(mul + c);
  const float4 sv = shift ? *reinterpret_cast<const float4*>(shift + c) : make_float4(0.f, 0.f, 0.f, 0.f);
  float v[4];
  load_row4_with_pending(h + (int64_t)row * d, row, d, c, pend, v);
  float mu = 0.f;
  if (mode == NORM_LN) mu = block_sum<256>(v[0] + v[1] + v[2] + v[3], scratch) / d;
  float ss = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) ss += (v[e] - mu) * (v[e] - mu);
  const float r = rsqrtf(block_sum<256>(ss, scratch) / d + eps);
  const float m4[4] = {mv.x, mv.y, mv.z, mv.w}, s4[4] = {sv.x, sv.y, sv.z, sv.w};
  float t[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) t[e] = (v[e] - mu) * r * (1.f + m4[e]) + s4[e];
  ActIO<OutT>::store4(n + (int64_t)row * d + c, t);
  if (n_lo) {
    float lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) lo[e] = t[e] - ActIO<OutT>::round(t[e]);
    ActIO<OutT>::store4(n_lo + (int64_t)row * d + c, lo);
  }
}

// The same normalisation with one wave per row, for d a multiple of 256 and
// at most 1024: lane l holds the float4 groups l, l + 64, ... of the row
// (every load of the row and of the norm's factors, pending slices included,
// requested before any is used; groups past d re-read the last one and are
// dropped), the statistics
// are wave sums (no LDS, no barrier), and a block holds blockDim.x / 64 rows.
// The pending slices are added in the same order as above.
template <typename OutT>
__global__ __launch_bounds__(256) void norm_rows_wave_kernel(float* __restrict__ h, OutT* __restrict__ n,
                                                             OutT* __restrict__ n_lo, int R, int d, float eps,
                                                             int mode, const float* __restrict__ mul,
                                                             const float* __restrict__ shift, PendingResid pend) {
  constexpr int kMaxG = 4;                      // float4 groups per lane (d <= 1024)
  constexpr int kMaxSplit = 8;
  const int lane = threadIdx.x % kWave;
  const int row = blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
  if (row >= R) return;
  const int ng = d / (4 * kWave);
  const int np = pend.n;
  float* hr = h + (int64_t)row * d;
  float4 hv[kMaxG], sl[kMaxG][kMaxSplit], bs[kMaxG], gt[kMaxG], mv[kMaxG], sv[kMaxG];
#pragma unroll
  for (int j = 0; j < kMaxG; ++j) {
    const int c = 4 * (lane + kWave * (j < ng ? j : ng - 1));
    mv[j] = *reinterpret_cast<const float4*>(mul + c);
    sv[j] = shift ? *reinterpret_cast<const float4*>(shift + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    hv[j] = *reinterpret_cast<const float4*>(hr + c);
    if (np > 0) {
#pragma unroll
      for (int sp = 0; sp < kMaxSplit; ++sp) {
        const int ss = sp < np ? sp : np - 1;
        sl[j][sp] = *reinterpret_cast<const float4*>(pend.part + ss * pend.stride + (int64_t)row * d + c);
      }
      bs[j] = pend.bias ? *reinterpret_cast<const float4*>(pend.bias + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      gt[j] = pend.gate ? *reinterpret_cast<const float4*>(pend.gate + c) : make_float4(1.f, 1.f, 1.f, 1.f);
    }
  }
  float x[kMaxG][4];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxG; ++j) {
    float v[4] = {hv[j].x, hv[j].y, hv[j].z, hv[j].w};
    if (np > 0) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float t = 0.f;
#pragma unroll
        for (int sp = 0; sp < kMaxSplit; ++sp) {
          const float4& q = sl[j][sp];
          const float qe = e == 0 ? q.x : e == 1 ? q.y : e == 2 ? q.z : q.w;
          t += sp < np ? qe : 0.f;
        }
        const float be = e == 0 ? bs[j].x : e == 1 ? bs[j].y : e == 2 ? bs[j].z : bs[j].w;
        const float ge = e == 0 ? gt[j].x : e == 1 ? gt[j].y : e == 2 ? gt[j].z : gt[j].w;
        v[e] += (t + be) * ge;
      }
      if (j < ng) *reinterpret_cast<float4*>(hr + 4 * (lane + kWave * j)) = make_float4(v[0], v[1], v[2], v[3]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[j][e] = j < ng ? v[e] : 0.f;
      s += x[j][e];
    }
  }
  float mu = 0.f;
  if (mode == NORM_LN) mu = wave_sum(s) / d;
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kMaxG; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float t = j < ng ? x[j][e] - mu : 0.f;
      ss += t * t;
    }
  const float r = rsqrtf(wave_sum(ss) / d + eps);
  OutT* nr = n + (int64_t)row * d;
#pragma unroll
  for (int j = 0; j < kMaxG; ++j) {
    if (j >= ng) break;
    const int c = 4 * (lane + kWave * j);
    const float m4[4] = {mv[j].x, mv[j].y, mv[j].z, mv[j].w}, s4[4] = {sv[j].x, sv[j].y, sv[j].z, sv[j].w};
    float t[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      t[e] = (x[j][e] - mu) * r * (1.f + m4[e]);
      if (shift) t[e] += s4[e];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      ActIO<OutT>::store(nr + c + e, t[e]);
      if (n_lo) ActIO<OutT>::store(n_lo + (int64_t)row * d + c + e, t[e] - ActIO<OutT>::round(t[e]));
    }
  }
}

// One block per suffix token row (b, t).
__global__ __launch_bounds__(256) void embed_kernel(EmbedArgs e) {
  __shared__ float xs[64];
  const int row = blockIdx.x;
  const int b = row / e.M, t = row % e.M;
  if (e.off && t == 0) {
    for (int c = threadIdx.x; c < e.d; c += 256) e.h[(int64_t)row * e.d + c] = e.e_state[(int64_t)b * e.d + c];
    return;
  }
  const int j = t - e.off;
  if (threadIdx.x < e.A) xs[threadIdx.x] = e.x[((int64_t)b * e.H + j) * e.A + threadIdx.x];
  __syncthreads();
  for (int c = threadIdx.x; c < e.d; c += 256) {
    float y = e.in_b[c];
#pragma unroll 16
    for (int a = 0; a < e.A; ++a) y = fmaf(xs[a], e.in_w[(int64_t)a * e.d + c], y);
    if (e.rowvec) y += e.rowvec[c];
    if (e.pos) y += e.pos[(int64_t)j * e.d + c];
    y = apply_act(e.act, y);
    if (e.act_out) {
      const int64_t o = ((int64_t)b * e.H + j) * e.d + c;
      if (e.act_is_bf16) static_cast<bf16_t*>(e.act_out)[o] = f32_to_bf16(y);
      else static_cast<float*>(e.act_out)[o] = y;
    } else {
      e.h[(int64_t)row * e.d + c] = y;
    }
  }
}

// The same embedding for A <= 32 and d a multiple of 4, RB suffix rows per
// block.  Thread t owns columns 4t .. 4t+3 of each 1024; every load of a
// group of 1024 columns (the weight columns for all A inputs, bias, rowvec,
// pos and state rows, and for the first group the rows' x entries) is
// requested before the first store, and the weight loads are shared by the
// block's RB rows.  Action rows: y = bias + sum_a x_a W[a] (+ rowvec)
// (+ pos), then act.  The loops run over 32 inputs without tests: inputs
// past A re-read weight row A-1 and meet x = 0.
template <int RB>
__global__ __launch_bounds__(256) void embed_rows_kernel(EmbedArgs e) {
  static_assert(RB * 32 <= 256, "one x entry per thread");
  __shared__ __attribute__((aligned(16))) float xs[RB][32];
  const int R = e.B * e.M;
  const int r0 = blockIdx.x * RB;
  float xv = 0.f;
  {
    const int rr = threadIdx.x / 32, a = threadIdx.x % 32;
    if (rr < RB && a < e.A) {
      const int r = min(r0 + rr, R - 1);
      const int b = r / e.M, j = max(r % e.M - e.off, 0);
      xv = e.x[((int64_t)b * e.H + j) * e.A + a];
    }
  }
  for (int g0 = 0; g0 < e.d; g0 += 1024) {
    const int c = g0 + 4 * threadIdx.x;
    const bool cv = c < e.d;
    const int cc = cv ? c : 0;
    float4 w[32];
#pragma unroll
    for (int a = 0; a < 32; ++a) w[a] = *reinterpret_cast<const float4*>(e.in_w + (int64_t)min(a, e.A - 1) * e.d + cc);
    const float4 bias = *reinterpret_cast<const float4*>(e.in_b + cc);
    const float4 rv = e.rowvec ? *reinterpret_cast<const float4*>(e.rowvec + cc) : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 pv[RB], sv[RB];
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) {
      const int r = min(r0 + rr, R - 1);
      const int b = r / e.M, j = max(r % e.M - e.off, 0);
      pv[rr] = e.pos ? *reinterpret_cast<const float4*>(e.pos + (int64_t)j * e.d + cc) : make_float4(0.f, 0.f, 0.f, 0.f);
      sv[rr] = e.off ? *reinterpret_cast<const float4*>(e.e_state + (int64_t)b * e.d + cc) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (g0 == 0) {
      if (threadIdx.x < RB * 32) xs[threadIdx.x / 32][threadIdx.x % 32] = xv;
      __syncthreads();
    }
    if (!cv) continue;
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) {
      const int r = r0 + rr;
      if (r >= R) break;
      const int b = r / e.M, t = r % e.M;
      if (e.off && t == 0) {
        *reinterpret_cast<float4*>(e.h + (int64_t)r * e.d + c) = sv[rr];
        continue;
      }
      float y[4] = {bias.x, bias.y, bias.z, bias.w};
      float xr[32];
#pragma unroll
      for (int a4 = 0; a4 < 8; ++a4) {
        const float4 x4 = reinterpret_cast<const float4*>(xs[rr])[a4];
        xr[4 * a4] = x4.x; xr[4 * a4 + 1] = x4.y; xr[4 * a4 + 2] = x4.z; xr[4 * a4 + 3] = x4.w;
      }
#pragma unroll
      for (int a = 0; a < 32; ++a) {
        y[0] = fmaf(xr[a], w[a].x, y[0]);
        y[1] = fmaf(xr[a], w[a].y, y[1]);
        y[2] = fmaf(xr[a], w[a].z, y[2]);
        y[3] = fmaf(xr[a], w[a].w, y[3]);
      }
      const float r4[4] = {rv.x, rv.y, rv.z, rv.w}, p4[4] = {pv[rr].x, pv[rr].y, pv[rr].z, pv[rr].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (e.rowvec) y[q] += r4[q];
        if (e.pos) y[q] += p4[q];
        y[q] = apply_act(e.act, y[q]);
      }
      const int j = t - e.off;
      if (e.act_out) {
        const int64_t o = ((int64_t)b * e.H + j) * e.d + c;
        if (e.act_is_bf16) {
          uint2 u;
          u.x = pack_bf16x2(y[0], y[1]);
          u.y = pack_bf16x2(y[2], y[3]);
          *reinterpret_cast<uint2*>(static_cast<bf16_t*>(e.act_out) + o) = u;
        } else {
          *reinterpret_cast<float4*>(static_cast<float*>(e.act_out) + o) = make_float4(y[0], y[1], y[2], y[3]);
        }
      } else {
        *reinterpret_cast<float4*>(e.h + (int64_t)r * e.d + c) = make_float4(y[0], y[1], y[2], y[3]);
      }
    }
  }
}

__global__ __launch_bounds__(256) void state_embed_kernel(const CallDesc* desc, const float* w, const float* bias,
                                                          float* e, int A, int d) {
  __shared__ float xs[64];
  const int b = blockIdx.x;
  if (threadIdx.x < A) xs[threadIdx.x] = desc->state[(int64_t)b * A + threadIdx.x];
  __syncthreads();
  for (int c = threadIdx.x; c < d; c += 256) {
    float y = bias[c];
#pragma unroll 16
    for (int a = 0; a < A; ++a) y = fmaf(xs[a], w[(int64_t)a * d + c], y);
    e[(int64_t)b * d + c] = y;
  }
}

// One block per action row: final norm -> v = n W_out + b_out -> x += dt v.
__global__ __launch_bounds__(256) void readout_kernel(ReadoutArgs r) {
  __shared__ float nrm[2048];
  __shared__ float red[1][64];
  __shared__ float scratch[4];
  const int ar = blockIdx.x;                 // b*H + j
  const int b = ar / r.H, j = ar % r.H;
  const int64_t hrow = (int64_t)b * r.M + r.off + j;
  float* hr = r.h + hrow * r.d;
  float v[kMaxPer];
  load_row_with_pending(hr, hrow, r.d, r.pend, v);
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) s += v[i];
  float mu = 0.f;
  if (r.mode == NORM_LN) mu = block_sum<256>(s, scratch) / r.d;
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int c = threadIdx.x + 256 * i;
    const float t = c < r.d ? v[i] - mu : 0.f;
    ss += t * t;
  }
  const float rs = rsqrtf(block_sum<256>(ss, scratch) / r.d + r.eps);
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (c < r.d) {
      float t = (v[i] - mu) * rs * (1.f + r.mul[c]);
      if (r.shift) t += r.shift[c];
      nrm[c] = t;
    }
  }
  __syncthreads();
  // v = n W_out with W_out^T rows contiguous along d: wave w computes outputs
  // a = w, w+4, ...; lane l takes 4 consecutive elements per 256 of each row
  // (8 groups cover d <= 2048).  Outputs go in chunks of 4 per wave: all
  // W_out loads of a chunk are requested before its first product, and a
  // wave sum finishes each output.
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  constexpr int QA = 4;                      // outputs per chunk
  constexpr int QC = kMaxPer;                // float4 groups per lane per row
  for (int a0 = wave; a0 < r.A; a0 += 4 * QA) {
    float4 w4[QA][QC];
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int a = a0 + 4 * q;
      if (a >= r.A) break;
      const float* wr = r.out_w + (int64_t)a * r.d + 4 * lane;
#pragma unroll
      for (int i = 0; i < QC; ++i)
        if (256 * i < r.d) w4[q][i] = *reinterpret_cast<const float4*>(wr + 256 * i);
    }
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      const int a = a0 + 4 * q;
      if (a >= r.A) break;
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < QC; ++i) {
        if (256 * i >= r.d) break;
        const int c = 4 * lane + 256 * i;
        acc = fmaf(nrm[c], w4[q][i].x, acc);
        acc = fmaf(nrm[c + 1], w4[q][i].y, acc);
        acc = fmaf(nrm[c + 2], w4[q][i].z, acc);
        acc = fmaf(nrm[c + 3], w4[q][i].w, acc);
      }
      acc = wave_sum(acc);
      if (lane == 0) red[0][a] = acc;
    }
  }
  __syncthreads();
  if (threadIdx.x < r.A) {
    const float vel = red[0][threadIdx.x] + r.out_b[threadIdx.x];
    r.x[(int64_t)ar * r.A + threadIdx.x] += r.dt[0] * vel;
  }
}

// Sums over the block of K values at once; scratch holds K floats per wave.
template <int K>
__device__ __forceinline__ void block_sums(float (&v)[K], float (*scratch)[K]) {
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = wave_sum(v[k]);
  __syncthreads();
  if (l == 0)
#pragma unroll
    for (int k = 0; k < K; ++k) scratch[w][k] = v[k];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < K; ++k) {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < 256 / kWave; ++i) t += scratch[i][k];
    v[k] = t;
  }
}

// The readout for d = 256 NG (NG <= 4) and A <= 32, RB action rows per
// block.  Every load the block needs is requested before any is used -- its
// waves' W_out rows (wave w takes outputs w, w + 4, ..., rows past A re-read
// row A-1 and are not stored), the final norm's factors, b_out, dt and the x
// entries it updates, then the rows -- so the block makes one memory round
// trip.  RB = 1 adds the pending split partials of the last block; RB > 1
// (rows without them) shares each W_out load among RB rows.  Per output the
// products are summed in the order of readout_kernel.
template <int RB, int NG, bool FUSE>
__global__ __launch_bounds__(256) void readout_rows_kernel(ReadoutArgs r) {
  constexpr int QA = 8;                      // outputs per wave
  __shared__ float4 nrm4[RB][NG * kWave];
  __shared__ float red[RB][32];
  __shared__ float scratch[256 / kWave][RB];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int nrows = r.B * r.H;
  const int ar0 = blockIdx.x * RB;
  const int d = 256 * NG;

  float4 w4[QA][NG];
#pragma unroll
  for (int q = 0; q < QA; ++q) {
    const int a = min(wave + 4 * q, r.A - 1);
#pragma unroll
    for (int i = 0; i < NG; ++i)
      w4[q][i] = *reinterpret_cast<const float4*>(r.out_w + (int64_t)a * d + 4 * lane + 256 * i);
  }
  // one row of width 1024: thread t holds columns 4t .. 4t+3 (16-byte
  // requests for the row and each pending slice); otherwise columns
  // t + 256 i
  constexpr bool V4 = RB == 1 && NG == 4;
  float mv[NG], sv[NG];
  if constexpr (V4) {
    const float4 m = *reinterpret_cast<const float4*>(r.mul + 4 * threadIdx.x);
    const float4 q = r.shift ? *reinterpret_cast<const float4*>(r.shift + 4 * threadIdx.x)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
    mv[0] = m.x; mv[1] = m.y; mv[2] = m.z; mv[3] = m.w;
    sv[0] = q.x; sv[1] = q.y; sv[2] = q.z; sv[3] = q.w;
  } else {
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      mv[i] = r.mul[threadIdx.x + 256 * i];
      sv[i] = r.shift ? r.shift[threadIdx.x + 256 * i] : 0.f;
    }
  }
  const int ur = threadIdx.x / r.A, ua = threadIdx.x % r.A;
  const bool upd = threadIdx.x < RB * r.A && ar0 + ur < nrows;
  const int64_t xi = upd ? (int64_t)(ar0 + ur) * r.A + ua : 0;
  const float xv = r.x[xi], bv = r.out_b[upd ? ua : 0], dtv = r.dt[0];

  float v[RB][NG];
  if constexpr (V4) {
    const int b = ar0 / r.H, j = ar0 % r.H;
    const int64_t hrow = (int64_t)b * r.M + r.off + j;
    load_row4_with_pending(r.h + hrow * d, hrow, d, 4 * threadIdx.x, r.pend, v[0]);
  } else if constexpr (RB == 1) {
    const int b = ar0 / r.H, j = ar0 % r.H;
    const int64_t hrow = (int64_t)b * r.M + r.off + j;
    float vv[kMaxPer];
    load_row_with_pending(r.h + hrow * d, hrow, d, r.pend, vv);
#pragma unroll
    for (int i = 0; i < NG; ++i) v[0][i] = vv[i];
  } else {
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) {
      const int ar = min(ar0 + rr, nrows - 1);
      const int b = ar / r.H, j = ar % r.H;
      const float* hr = r.h + ((int64_t)b * r.M + r.off + j) * d;
#pragma unroll
      for (int i = 0; i < NG; ++i) v[rr][i] = hr[threadIdx.x + 256 * i];
    }
  }

  // Fused with the next step's embedding: its inputs that do not depend on
  // the update (the embedding weights for this thread's four columns, bias,
  // row vector, position and state rows) are requested with the rows.
  const EmbedArgs& e = r.next;
  const int ec = 4 * threadIdx.x;              // d <= 1024: one group of four columns
  const bool ecv = ec < d;
  const int ecc = ecv ? ec : 0;
  float4 ew[FUSE ? 32 : 1], ebias = make_float4(0.f, 0.f, 0.f, 0.f), erv = ebias;
  float4 epv[FUSE ? RB : 1], esv[FUSE ? RB : 1];
  if constexpr (FUSE) {
#pragma unroll
    for (int a = 0; a < 32; ++a)
      ew[a] = *reinterpret_cast<const float4*>(e.in_w + (int64_t)min(a, e.A - 1) * d + ecc);
    ebias = *reinterpret_cast<const float4*>(e.in_b + ecc);
    if (e.rowvec) erv = *reinterpret_cast<const float4*>(e.rowvec + ecc);
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) {
      const int ar = min(ar0 + rr, nrows - 1);
      const int b = ar / r.H, j = ar % r.H;
      epv[rr] = e.pos ? *reinterpret_cast<const float4*>(e.pos + (int64_t)j * d + ecc) : make_float4(0.f, 0.f, 0.f, 0.f);
      esv[rr] = e.off ? *reinterpret_cast<const float4*>(e.e_state + (int64_t)b * d + ecc)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }

  float mu[RB], st[RB];
#pragma unroll
  for (int rr = 0; rr < RB; ++rr) {
    mu[rr] = 0.f;
#pragma unroll
    for (int i = 0; i < NG; ++i) mu[rr] += v[rr][i];
  }
  if (r.mode == NORM_LN) {
    block_sums<RB>(mu, scratch);
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) mu[rr] /= d;
  } else {
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) mu[rr] = 0.f;
  }
#pragma unroll
  for (int rr = 0; rr < RB; ++rr) {
    st[rr] = 0.f;
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const float t = v[rr][i] - mu[rr];
      st[rr] += t * t;
    }
  }
  block_sums<RB>(st, scratch);
  float* nrm = reinterpret_cast<float*>(nrm4);
#pragma unroll
  for (int rr = 0; rr < RB; ++rr) {
    const float rs = rsqrtf(st[rr] / d + r.eps);
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      float t = (v[rr][i] - mu[rr]) * rs * (1.f + mv[i]);
      if (r.shift) t += sv[i];
      nrm[rr * d + (V4 ? 4 * threadIdx.x + i : threadIdx.x + 256 * i)] = t;
    }
  }
  __syncthreads();

  // v = n W_out: lane l takes elements 4l .. 4l+3 of each 256, a wave sum
  // finishes each (row, output)
#pragma unroll
  for (int rr = 0; rr < RB; ++rr) {
    float4 n4[NG];
#pragma unroll
    for (int i = 0; i < NG; ++i) n4[i] = nrm4[rr][lane + kWave * i];
#pragma unroll
    for (int q = 0; q < QA; ++q) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < NG; ++i) {
        acc = fmaf(n4[i].x, w4[q][i].x, acc);
        acc = fmaf(n4[i].y, w4[q][i].y, acc);
        acc = fmaf(n4[i].z, w4[q][i].z, acc);
        acc = fmaf(n4[i].w, w4[q][i].w, acc);
      }
      acc = wave_sum(acc);
      if (lane == 0 && wave + 4 * q < r.A) red[rr][wave + 4 * q] = acc;
    }
  }
  __syncthreads();
  const float xn = xv + dtv * (red[ur][ua] + bv);
  if (upd) r.x[xi] = xn;
  if constexpr (FUSE) {
    // y = act(x_new . in_w + in_b + rowvec + pos[j]) into the next step's
    // embedding destination (embed_rows_kernel's arithmetic), and the state
    // row of request b reset with the row of its first action
    __shared__ __attribute__((aligned(16))) float xs[RB][32];
    if (threadIdx.x < RB * 32 && threadIdx.x % 32 >= r.A) xs[threadIdx.x / 32][threadIdx.x % 32] = 0.f;
    if (upd) xs[ur][ua] = xn;
    __syncthreads();
    if (!ecv) return;
#pragma unroll
    for (int rr = 0; rr < RB; ++rr) {
      const int ar = ar0 + rr;
      if (ar >= nrows) break;
      const int b = ar / r.H, j = ar % r.H;
      float y[4] = {ebias.x, ebias.y, ebias.z, ebias.w};
      float xr[32];
#pragma unroll
      for (int a4 = 0; a4 < 8; ++a4) {
        const float4 x4 = reinterpret_cast<const float4*>(xs[rr])[a4];
        xr[4 * a4] = x4.x; xr[4 * a4 + 1] = x4.y; xr[4 * a4 + 2] = x4.z; xr[4 * a4 + 3] = x4.w;
      }
#pragma unroll
      for (int a = 0; a < 32; ++a) {
        y[0] = fmaf(xr[a], ew[a].x, y[0]);
        y[1] = fmaf(xr[a], ew[a].y, y[1]);
        y[2] = fmaf(xr[a], ew[a].z, y[2]);
        y[3] = fmaf(xr[a], ew[a].w, y[3]);
      }
      const float r4[4] = {erv.x, erv.y, erv.z, erv.w}, p4[4] = {epv[rr].x, epv[rr].y, epv[rr].z, epv[rr].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (e.rowvec) y[q] += r4[q];
        if (e.pos) y[q] += p4[q];
        y[q] = apply_act(e.act, y[q]);
      }
      if (e.act_out) {
        const int64_t o = ((int64_t)b * e.H + j) * d + ec;
        if (e.act_is_bf16) {
          uint2 u;
          u.x = pack_bf16x2(y[0], y[1]);
          u.y = pack_bf16x2(y[2], y[3]);
          *reinterpret_cast<uint2*>(static_cast<bf16_t*>(e.act_out) + o) = u;
        } else {
          *reinterpret_cast<float4*>(static_cast<float*>(e.act_out) + o) = make_float4(y[0], y[1], y[2], y[3]);
        }
      } else {
        *reinterpret_cast<float4*>(e.h + ((int64_t)b * e.M + e.off + j) * d + ec) = make_float4(y[0], y[1], y[2], y[3]);
      }
      if (e.off && j == 0) *reinterpret_cast<float4*>(e.h + (int64_t)b * e.M * d + ec) = esv[rr];
    }
  }
}

__global__ __launch_bounds__(128) void rope_table_kernel(const CallDesc* desc, const float* inv_freq, float2* tab,
                                                        int M, int half, int after_prefix) {
  const int row = blockIdx.x;                    // b*M + t
  const int b = row / M, t = row % M;
  const float pos = (float)((after_prefix ? desc->prefix_len[b] : 0) + t);
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    float sn, cs;
    sincosf(pos * inv_freq[i], &sn, &cs);
    tab[(int64_t)row * half + i] = make_float2(cs, sn);
  }
}

__global__ __launch_bounds__(256) void prefill_embed_kernel(const CallDesc* desc, const float* embeds, float* h,
                                                           int M, int d) {
  const int row = blockIdx.x;                    // b*M + t
  const bool valid = row % M < desc->prefix_len[row / M];
  const float4* src = reinterpret_cast<const float4*>(embeds + (int64_t)row * d);
  float4* dst = reinterpret_cast<float4*>(h + (int64_t)row * d);
  for (int i = threadIdx.x; i < d / 4; i += 256) dst[i] = valid ? src[i] : make_float4(0.f, 0.f, 0.f, 0.f);
}

// One block per patch row: the patch (patch_dim a multiple of 64) converted
// into the patch-embedding GEMM's operand, and the row's position embedding
// into the residual stream (the GEMM then adds x W + b on top).
template <typename T>
__global__ __launch_bounds__(256) void vision_embed_kernel(const float* __restrict__ patches, T* __restrict__ a,
                                                           float* __restrict__ h, const float* __restrict__ pos,
                                                           int n_patches, int patch_dim, int d) {
  const int row = blockIdx.x;
  const float4* src = reinterpret_cast<const float4*>(patches + (int64_t)row * patch_dim);
  T* dst = a + (int64_t)row * patch_dim;
  for (int i = threadIdx.x; i < patch_dim / 4; i += 256) {
    const float4 v = src[i];
    const float w[4] = {v.x, v.y, v.z, v.w};
    ActIO<T>::store4(dst + 4 * i, w);
  }
  const float4* ps = reinterpret_cast<const float4*>(pos + (int64_t)(row % n_patches) * d);
  float4* hd = reinterpret_cast<float4*>(h + (int64_t)row * d);
  for (int i = threadIdx.x; i < d / 4; i += 256) hd[i] = ps[i];
}

__global__ void copy_in_kernel(const CallDesc* desc, float* x, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = desc->noise[i];
}

__global__ void copy_out_kernel(const CallDesc* desc, const float* x, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) desc->out[i] = x[i];
}

__global__ void set_desc_kernel(CallDesc d, CallDesc* dst) {
  constexpr int W = sizeof(CallDesc) / 4;
  const int32_t* src = reinterpret_cast<const int32_t*>(&d);
  int32_t* out = reinterpret_cast<int32_t*>(dst);
  for (int i = threadIdx.x; i < W; i += blockDim.x) out[i] = src[i];
}

__global__ void fp8_decode_kernel(const uint8_t* codes, bf16_t* out, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  uint32_t w = 0;
  for (int k = 0; k < 4 && i + k < n; ++k) w |= static_cast<uint32_t>(codes[i + k]) << (8 * k);
  const uint32_t lo = fp8x2_to_bf16x2<false>(w), hi = fp8x2_to_bf16x2<true>(w);
  const bf16_t r[4] = {static_cast<bf16_t>(lo & 0xffff), static_cast<bf16_t>(lo >> 16),
                       static_cast<bf16_t>(hi & 0xffff), static_cast<bf16_t>(hi >> 16)};
  for (int k = 0; k < 4 && i + k < n; ++k) out[i + k] = r[k];
}

}  // namespace

void norm_rows_bf16(float* h, bf16_t* n, bf16_t* n_lo, int R, int d, float eps, int mode, const float* mul,
                    const float* shift, const PendingResid& pend, hipStream_t s) {
  // many rows: four rows per block, one per wave (fewer, fuller blocks); a
  // few rows (batch 1) keep 256 threads per row, which spreads a row's loads
  // over four waves and measured faster there; at width 1024 each of those
  // threads takes four consecutive columns (batch-1 norm 3.4 -> 2.3 us)
  if (R >= 256 && d % 256 == 0 && d <= 1024 && pend.n <= 8) {
    hipLaunchKernelGGL(norm_rows_wave_kernel<bf16_t>, dim3((R + 3) / 4), dim3(4 * kWave), 0, s, h, n, n_lo, R, d,
                       eps, mode, mul, shift, pend);
    return;
  }
  if (d == 1024 && pend.n <= 8) {
    hipLaunchKernelGGL(norm_rows_v4_kernel<bf16_t>, dim3(R), dim3(256), 0, s, h, n, n_lo, d, eps, mode, mul, shift,
                       pend);
    return;
  }
  hipLaunchKernelGGL(norm_rows_kernel<bf16_t>, dim3(R), dim3(256), 0, s, h, n, n_lo, d, eps, mode, mul, shift, pend);
}
void norm_rows_f32(float* h, float* n, int R, int d, float eps, int mode, const float* mul,
                   const float* shift, const PendingResid& pend, hipStream_t s) {
  hipLaunchKernelGGL(norm_rows_kernel<float>, dim3(R), dim3(256), 0, s, h, n, nullptr, d, eps, mode, mul, shift,
                     pend);
}
void embed_actions(const EmbedArgs& e, hipStream_t s) {
  const int R = e.B * e.M;
  if (e.A <= 32 && e.d % 4 == 0) {
    if (R >= 1024) hipLaunchKernelGGL(embed_rows_kernel<8>, dim3((R + 7) / 8), dim3(256), 0, s, e);
    else hipLaunchKernelGGL(embed_rows_kernel<1>, dim3(R), dim3(256), 0, s, e);
  } else {
    hipLaunchKernelGGL(embed_kernel, dim3(R), dim3(256), 0, s, e);
  }
}
void embed_state(const CallDesc* desc, const float* w, const float* b, float* e, int B, int A, int d,
                 hipStream_t s) {
  hipLaunchKernelGGL(state_embed_kernel, dim3(B), dim3(256), 0, s, desc, w, b, e, A, d);
}
// the readout rows kernel takes four rows per block for many rows without a
// pending residual, one otherwise
static bool readout_four_rows(int rows, bool pending) { return !pending && rows >= 1024; }

bool readout_fuses_embedding(int A, int d, int rows, bool pending) {
  return A <= 32 && (d == 1024 || d == 256) && !readout_four_rows(rows, pending);
}

void readout_euler(const ReadoutArgs& r, hipStream_t s) {
  const int rows = r.B * r.H;
  const bool four = readout_four_rows(rows, r.pend.n > 0);
  auto rows_kernel = [&](auto ng) {
    constexpr int NG = decltype(ng)::value;
    if (four)
      hipLaunchKernelGGL((readout_rows_kernel<4, NG, false>), dim3((rows + 3) / 4), dim3(256), 0, s, r);
    else if (r.has_next)
      hipLaunchKernelGGL((readout_rows_kernel<1, NG, true>), dim3(rows), dim3(256), 0, s, r);
    else
      hipLaunchKernelGGL((readout_rows_kernel<1, NG, false>), dim3(rows), dim3(256), 0, s, r);
  };
  if (r.A <= 32 && r.d == 1024) rows_kernel(std::integral_constant<int, 4>{});
  else if (r.A <= 32 && r.d == 256) rows_kernel(std::integral_constant<int, 1>{});
  else {
    hipLaunchKernelGGL(readout_kernel, dim3(rows), dim3(256), 0, s, r);
  }
}
void copy_noise_to_state(const CallDesc* desc, float* x, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(copy_in_kernel, dim3((n + 255) / 256), dim3(256), 0, s, desc, x, n);
}
void copy_state_to_out(const CallDesc* desc, const float* x, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(copy_out_kernel, dim3((n + 255) / 256), dim3(256), 0, s, desc, x, n);
}
void rope_table(const CallDesc* desc, const float* inv_freq, float2* tab, int B, int M, int D, int pos_after_prefix,
                hipStream_t s) {
  hipLaunchKernelGGL(rope_table_kernel, dim3(B * M), dim3(128), 0, s, desc, inv_freq, tab, M, D / 2,
                     pos_after_prefix);
}
void prefill_embed(const CallDesc* desc, const float* embeds, float* h, int B, int M, int d, hipStream_t s) {
  if (B * M > 0) hipLaunchKernelGGL(prefill_embed_kernel, dim3(B * M), dim3(256), 0, s, desc, embeds, h, M, d);
}
void vision_embed_bf16(const float* patches, bf16_t* a, float* h, const float* pos, int R, int n_patches,
                       int patch_dim, int d, hipStream_t s) {
  if (R > 0)
    hipLaunchKernelGGL(vision_embed_kernel<bf16_t>, dim3(R), dim3(256), 0, s, patches, a, h, pos, n_patches,
                       patch_dim, d);
}
void vision_embed_f32(const float* patches, float* a, float* h, const float* pos, int R, int n_patches,
                      int patch_dim, int d, hipStream_t s) {
  if (R > 0)
    hipLaunchKernelGGL(vision_embed_kernel<float>, dim3(R), dim3(256), 0, s, patches, a, h, pos, n_patches,
                       patch_dim, d);
}
void set_call_desc(const CallDesc& d, CallDesc* dev, hipStream_t s) {
  hipLaunchKernelGGL(set_desc_kernel, dim3(1), dim3(256), 0, s, d, dev);
}
void fp8_to_bf16(const uint8_t* codes, bf16_t* out, int64_t n, hipStream_t s) {
  const int64_t groups = (n + 3) / 4;
  hipLaunchKernelGGL(fp8_decode_kernel, dim3((groups + 255) / 256), dim3(256), 0, s, codes, out, n);
}

}  // namespace phyai
