// Suffix-query attention over the frozen prefix K/V and the suffix tokens'
// own K/V (the "50-token query against a longer prefix, head dimension 256"
// shape of Section "PhyAI Architecture", paragraph "Profiled operator
// selection"), with online softmax and optional split over the keys.
//
// MFMA formulation: every product is computed transposed, S^T = K Q^T and
// O^T = V^T P^T, so that a query is always the MFMA column (lane % 16).  The
// softmax statistics of a query then live in the four lanes l%16 == q and
// only need two cross-lane steps, and the probabilities come out of the
// S^T accumulators already laid out as the B operand of the P.V product
// (the key order inside the k dimension is permuted identically on both
// operands).  One wave owns 16 query rows; a block of 4 waves owns 64 rows
// of one (request, kv head) and stages 32-key tiles of K (row-major) and V
// (transposed) in LDS.
#include "kernels.hpp"

namespace phyai {

namespace {

constexpr int kKT = 32;       // keys per LDS tile

template <int D>
__global__ __launch_bounds__(256) void attn_mfma_kernel(AttnArgs a) {
  constexpr int KLD = D + 8;       // LDS row stride of the K tile (elements)
  constexpr int VLD = kKT + 8;     // LDS row stride of the transposed V tile
  __shared__ __attribute__((aligned(16))) bf16_t Ks[kKT * KLD];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[D * VLD];

  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int G = a.nq / a.nkv;
  const int rows = a.M * G;
  const int grp = blockIdx.y;
  const int b = grp / a.nkv, kvh = grp % a.nkv;
  const int split = blockIdx.z;
  const int qr = blockIdx.x * 64 + wave * 16 + (lane % 16);
  const bool qvalid = qr < rows;
  const int qtok = qvalid ? qr / G : 0;
  const int qhead = kvh * G + (qvalid ? qr % G : 0);
  const int lg = lane / 16;

  const int len1 = a.use_seg1 ? a.desc->prefix_len[b] : 0;
  const int N = len1 + a.len2;
  int chunk = (N + a.n_split - 1) / a.n_split;
  chunk = (chunk + kKT - 1) / kKT * kKT;
  const int kbeg = split * chunk;
  const int kend = min(N, kbeg + chunk);

  const bf16_t* s1k = nullptr;
  const bf16_t* s1v = nullptr;
  if (a.use_seg1) {
    const bf16_t* bk = a.seg1_ind ? static_cast<const bf16_t*>(*a.seg1_ind) : static_cast<const bf16_t*>(a.seg1_k);
    const bf16_t* bv = a.seg1_ind ? static_cast<const bf16_t*>(*a.seg1_ind) : static_cast<const bf16_t*>(a.seg1_v);
    s1k = bk + a.seg1_k_off + (int64_t)b * a.seg1_bstride + kvh * D;
    s1v = bv + a.seg1_v_off + (int64_t)b * a.seg1_bstride + kvh * D;
  }
  const bf16_t* s2k = static_cast<const bf16_t*>(a.sk) + (int64_t)b * a.M * a.ld2 + kvh * D;
  const bf16_t* s2v = static_cast<const bf16_t*>(a.sv) + (int64_t)b * a.M * a.ld2 + kvh * D;

  bf16x8 qf[D / 32];
  {
    const bf16_t* qp = static_cast<const bf16_t*>(a.q) + (int64_t)(b * a.M + qtok) * a.ldq + qhead * D + 8 * lg;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qvalid) v = *reinterpret_cast<const uint4*>(qp + 32 * s);
      qf[s] = as_bf16x8(v);
    }
  }

  f32x4 o[D / 16];
#pragma unroll
  for (int i = 0; i < D / 16; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -1e30f, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;

  for (int kt0 = kbeg; kt0 < kend; kt0 += kKT) {
    __syncthreads();
    constexpr int CPR = D / 8;                 // 16-byte chunks per key row
    for (int ci = threadIdx.x; ci < kKT * CPR; ci += 256) {
      const int kr = ci / CPR, dc = (ci % CPR) * 8;
      const int kk = kt0 + kr;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (kk < kend) {
        if (kk < len1) {
          kv = *reinterpret_cast<const uint4*>(s1k + (int64_t)kk * a.seg1_ld + dc);
          vv = *reinterpret_cast<const uint4*>(s1v + (int64_t)kk * a.seg1_ld + dc);
        } else {
          const int j = kk - len1;
          kv = *reinterpret_cast<const uint4*>(s2k + (int64_t)j * a.ld2 + dc);
          vv = *reinterpret_cast<const uint4*>(s2v + (int64_t)j * a.ld2 + dc);
        }
      }
      *reinterpret_cast<uint4*>(Ks + kr * KLD + dc) = kv;
      const bf16_t* ve = reinterpret_cast<const bf16_t*>(&vv);
#pragma unroll
      for (int i = 0; i < 8; ++i) Vt[(dc + i) * VLD + kr] = ve[i];
    }
    __syncthreads();

    f32x4 st[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      st[kt] = f32x4{0.f, 0.f, 0.f, 0.f};
      const bf16_t* kp = Ks + (16 * kt + lane % 16) * KLD + 8 * lg;
#pragma unroll
      for (int s = 0; s < D / 32; ++s)
        st[kt] = mfma16x16x32(*reinterpret_cast<const bf16x8*>(kp + 32 * s), qf[s], st[kt]);
    }

    float sc[8];
    float tmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int key = kt0 + 16 * kt + 4 * lg + v;
        bool ok = key < kend;
        if (ok && a.mask_mode == 1 && key >= len1) ok = (key == len1) || (qtok != 0);
        const float s = ok ? st[kt][v] * sl2 : -INFINITY;
        sc[kt * 4 + v] = s;
        tmax = fmaxf(tmax, s);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, kWave));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, kWave));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float p[8], psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = exp2f(sc[i] - m_new);
      psum += p[i];
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int i = 0; i < D / 16; ++i) o[i] *= alpha;

    uint4 pw;
    pw.x = pack_bf16x2(p[0], p[1]);
    pw.y = pack_bf16x2(p[2], p[3]);
    pw.z = pack_bf16x2(p[4], p[5]);
    pw.w = pack_bf16x2(p[6], p[7]);
    const bf16x8 pf = as_bf16x8(pw);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const bf16_t* vr = Vt + (16 * dt + lane % 16) * VLD + 4 * lg;
      const uint2 lo = *reinterpret_cast<const uint2*>(vr);
      const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
      o[dt] = mfma16x16x32(as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y)), pf, o[dt]);
    }
  }

  l_run += __shfl_xor(l_run, 16, kWave);
  l_run += __shfl_xor(l_run, 32, kWave);
  if (!qvalid) return;
  if (a.n_split == 1) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    bf16_t* op = static_cast<bf16_t*>(a.out) + (int64_t)(b * a.M + qtok) * a.ldo + qhead * D + 4 * lg;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      uint2 w;
      w.x = pack_bf16x2(o[dt][0] * inv, o[dt][1] * inv);
      w.y = pack_bf16x2(o[dt][2] * inv, o[dt][3] * inv);
      *reinterpret_cast<uint2*>(op + 16 * dt) = w;
    }
  } else {
    const int rows_cap = gridDim.x * 64;
    float* pp = a.part + ((int64_t)(grp * a.n_split + split) * rows_cap + qr) * (D + 4);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt)
      *reinterpret_cast<float4*>(pp + 16 * dt + 4 * lg) = make_float4(o[dt][0], o[dt][1], o[dt][2], o[dt][3]);
    if (lg == 0) {
      pp[D] = m_run;
      pp[D + 1] = l_run;
    }
  }
}

// Merge the split partials of one query row (one wave per row).
template <int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a, int rows_cap) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int qr = blockIdx.x * 4 + wave;
  const int grp = blockIdx.y;
  const int G = a.nq / a.nkv;
  if (qr >= a.M * G) return;
  const int b = grp / a.nkv, kvh = grp % a.nkv;
  const int qtok = qr / G, qhead = kvh * G + qr % G;
  float mmax = -1e30f;
  for (int s = 0; s < a.n_split; ++s)
    mmax = fmaxf(mmax, a.part[((int64_t)(grp * a.n_split + s) * rows_cap + qr) * (D + 4) + D]);
  float acc[D / 64];
#pragma unroll
  for (int i = 0; i < D / 64; ++i) acc[i] = 0.f;
  float lsum = 0.f;
  for (int s = 0; s < a.n_split; ++s) {
    const float* pp = a.part + ((int64_t)(grp * a.n_split + s) * rows_cap + qr) * (D + 4);
    const float w = exp2f(pp[D] - mmax);
    lsum += w * pp[D + 1];
#pragma unroll
    for (int i = 0; i < D / 64; ++i) acc[i] += w * pp[lane + 64 * i];
  }
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  bf16_t* op = static_cast<bf16_t*>(a.out) + (int64_t)(b * a.M + qtok) * a.ldo + qhead * D;
#pragma unroll
  for (int i = 0; i < D / 64; ++i) op[lane + 64 * i] = f32_to_bf16(acc[i] * inv);
}

// fp32 path: one wave per (request, token, query head), keys one at a time.
template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  const int lane = threadIdx.x;
  const int row = blockIdx.x;                   // b*M + token
  const int h = blockIdx.y;
  const int b = row / a.M, tok = row % a.M;
  const int G = a.nq / a.nkv, kvh = h / G;
  const int len1 = a.use_seg1 ? a.desc->prefix_len[b] : 0;
  const int N = len1 + a.len2;
  const float* q = static_cast<const float*>(a.q) + (int64_t)row * a.ldq + h * D;
  const float* s1k = nullptr;
  const float* s1v = nullptr;
  if (a.use_seg1) {
    const float* bk = a.seg1_ind ? static_cast<const float*>(*a.seg1_ind) : static_cast<const float*>(a.seg1_k);
    const float* bv = a.seg1_ind ? static_cast<const float*>(*a.seg1_ind) : static_cast<const float*>(a.seg1_v);
    s1k = bk + a.seg1_k_off + (int64_t)b * a.seg1_bstride + kvh * D;
    s1v = bv + a.seg1_v_off + (int64_t)b * a.seg1_bstride + kvh * D;
  }
  const float* s2k = static_cast<const float*>(a.sk) + (int64_t)b * a.M * a.ld2 + kvh * D;
  const float* s2v = static_cast<const float*>(a.sv) + (int64_t)b * a.M * a.ld2 + kvh * D;
  constexpr int PER = (D + 63) / 64;
  float qv[PER], acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int d = lane + 64 * i;
    qv[i] = d < D ? q[d] : 0.f;
    acc[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int kk = 0; kk < N; ++kk) {
    bool ok = true;
    if (kk >= len1 && a.mask_mode == 1) ok = (kk == len1) || (tok != 0);
    if (!ok) continue;
    const float* kr = kk < len1 ? s1k + (int64_t)kk * a.seg1_ld : s2k + (int64_t)(kk - len1) * a.ld2;
    const float* vr = kk < len1 ? s1v + (int64_t)kk * a.seg1_ld : s2v + (int64_t)(kk - len1) * a.ld2;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int d = lane + 64 * i;
      if (d < D) s = fmaf(qv[i], kr[d], s);
    }
    s = wave_sum(s) * a.scale;
    const float mn = fmaxf(m, s);
    const float al = __expf(m - mn);
    const float p = __expf(s - mn);
    l = l * al + p;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int d = lane + 64 * i;
      acc[i] = acc[i] * al + (d < D ? p * vr[d] : 0.f);
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

}  // namespace

int64_t attention_partial_floats(int B, int M, int nq, int nkv, int D, int n_split) {
  if (n_split <= 1) return 0;
  const int rows = M * (nq / nkv);
  const int64_t rows_cap = (int64_t)((rows + 63) / 64) * 64;
  return (int64_t)B * nkv * n_split * rows_cap * (D + 4);
}

void attention_bf16(const AttnArgs& a, hipStream_t s) {
  const int rows = a.M * (a.nq / a.nkv);
  dim3 grid((rows + 63) / 64, a.B * a.nkv, a.n_split);
  if (a.D == 256) hipLaunchKernelGGL(attn_mfma_kernel<256>, grid, dim3(256), 0, s, a);
  else if (a.D == 128) hipLaunchKernelGGL(attn_mfma_kernel<128>, grid, dim3(256), 0, s, a);
  else if (a.D == 64) hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(256), 0, s, a);
  if (a.n_split > 1) {
    const int rows_cap = grid.x * 64;
    dim3 g2((rows + 3) / 4, a.B * a.nkv);
    if (a.D == 256) hipLaunchKernelGGL(attn_combine_kernel<256>, g2, dim3(256), 0, s, a, rows_cap);
    else if (a.D == 128) hipLaunchKernelGGL(attn_combine_kernel<128>, g2, dim3(256), 0, s, a, rows_cap);
    else if (a.D == 64) hipLaunchKernelGGL(attn_combine_kernel<64>, g2, dim3(256), 0, s, a, rows_cap);
  }
}

void attention_f32(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.B * a.M, a.nq);
  if (a.D == 64) hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(64), 0, s, a);
  else if (a.D == 128) hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(64), 0, s, a);
  else if (a.D == 256) hipLaunchKernelGGL(attn_f32_kernel<256>, grid, dim3(64), 0, s, a);
}

}  // namespace phyai
