// Device helpers shared by the gfx950 kernels: bf16/fp8 conversion, MFMA
// operand types, wave/block reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace phyai {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

typedef uint16_t bf16_t;   // storage type of bfloat16 values

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// bf16 <-> f32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even (NaN stays NaN): gfx950's v_cvt_pk_bf16_f32.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// ---------------------------------------------------------------------------
// fp8 (OCP e4m3fn) -> bf16, exact.  gfx950's v_cvt_scalef32_pk_bf16_fp8
// decodes two codes (selected by word_sel) with a unit scale.
// ---------------------------------------------------------------------------
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t codes4) {
  bf16x2 r = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(codes4, 1.0f, HI);
  return __builtin_bit_cast(uint32_t, r);
}

// 8 fp8 codes (two dwords) -> 8 bf16 as an MFMA operand.
__device__ __forceinline__ bf16x8 fp8x8_to_bf16x8(uint32_t lo, uint32_t hi) {
  uint4 r;
  r.x = fp8x2_to_bf16x2<false>(lo);
  r.y = fp8x2_to_bf16x2<true>(lo);
  r.z = fp8x2_to_bf16x2<false>(hi);
  r.w = fp8x2_to_bf16x2<true>(hi);
  return __builtin_bit_cast(bf16x8, r);
}

// ---------------------------------------------------------------------------
// fp4 (OCP e2m1) -> bf16 with a power-of-two scale, exact.  gfx950's
// v_cvt_scalef32_pk_bf16_fp4 decodes the two codes of one byte (low nibble
// first) and multiplies by 2^(exponent of the scale operand): only the
// scale's exponent is used, which is why the weight format keeps
// power-of-two scales (E8M0 bytes, value 2^(e - 127)).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float e8m0_to_f32(uint32_t e) { return __uint_as_float(e << 23); }

// 8 fp4 codes (one dword, low nibble of byte 0 first) -> 8 bf16 as an MFMA operand.
__device__ __forceinline__ bf16x8 fp4x8_to_bf16x8(uint32_t codes, float scale) {
  uint4 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, scale, 0));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, scale, 1));
  r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, scale, 2));
  r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, scale, 3));
  return __builtin_bit_cast(bf16x8, r);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// ---------------------------------------------------------------------------
// Device-scope (sc1) stores and loads, for data another block reads within
// the same kernel: the store writes through the writer's L2, and the load
// bypasses a possibly stale line in the reader's (the XCDs' L2s are not
// coherent with each other).  `base` must be the same for the whole wave (the
// buffer resource lives in scalar registers; a per-lane base would make the
// compiler loop over the distinct values); `off` is the lane's element
// offset, below 2^29.
// ---------------------------------------------------------------------------
constexpr int kDeviceScope = 16;   // buffer instruction cache policy: sc1
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ void st_device_f32(float* base, int64_t off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), raw_rsrc(base), static_cast<int>(off * 4), 0,
                                        kDeviceScope);
}
__device__ __forceinline__ float4 ld_device_f32x4(const float* base, int64_t off) {
  typedef unsigned int u4 __attribute__((ext_vector_type(4)));
  const u4 v = __builtin_amdgcn_raw_buffer_load_b128(raw_rsrc(base), static_cast<int>(off * 4), 0, kDeviceScope);
  return __builtin_bit_cast(float4, v);
}

// D = A(16x32) * B(32x16) + C, bf16 operands, fp32 accumulate.
// Lane l holds A[l%16][k8(l/16) .. +7], B[k8(l/16) .. +7][l%16] and
// C[4*(l/16) + v][l%16] (v = 0..3).  The k order inside a lane only has to
// agree between A and B.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// D = A(32x16) * B(16x32) + C.  Lane l holds A[l%32][8(l/32) .. +7],
// B[8(l/32) .. +7][l%32] and C[8(v/4) + 4(l/32) + v%4][l%32] (v = 0..15).
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// reductions
// ---------------------------------------------------------------------------
// The value of another lane of the same row of 16 (DPP control CTRL).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the wave, in every lane, on the VALU: lane ^ 1 and lane ^ 2 by
// quad permutes, the other quad of each 8 and the other 8 of each 16 by
// the half-row and row mirrors, then the other 16 and the other 32 by
// gfx950's permlane swaps.  Each step adds a lane's value to a partner
// holding the same partial sum of a disjoint lane set, so all lanes end
// with the same total.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_f32<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_f32<0x141>(v);   // row_half_mirror
  v += dpp_f32<0x140>(v);   // row_mirror
  {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return v;
}

// Sum over the block; `scratch` holds one float per wave.  All threads get it.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* scratch) {
  constexpr int NW = NT / kWave;
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) scratch[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += scratch[i];
  return t;
}

// ---------------------------------------------------------------------------
// activations (fp32)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float swish_f(float z) { return z / (1.0f + __expf(-z)); }

__device__ __forceinline__ float gelu_tanh_f(float z) {
  const float k0 = 0.7978845608028654f;   // sqrt(2/pi)
  const float u = k0 * (z + 0.044715f * z * z * z);
  return 0.5f * z * (1.0f + tanhf(u));
}

enum Act { ACT_NONE = 0, ACT_SWISH = 1, ACT_GELU = 2 };

__device__ __forceinline__ float apply_act(int act, float v) {
  if (act == ACT_SWISH) return swish_f(v);
  if (act == ACT_GELU) return gelu_tanh_f(v);
  return v;
}

// Activation storage: bf16 on the MFMA path, f32 on the fp32 path.
template <typename T> struct ActIO;
// store4: four consecutive values in one store (p aligned to 4 elements)
template <> struct ActIO<float> {
  static __device__ __forceinline__ float round(float v) { return v; }
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
  static __device__ __forceinline__ void store4(float* p, const float (&v)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  }
};
template <> struct ActIO<bf16_t> {
  static __device__ __forceinline__ float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
  static __device__ __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(*p); }
  static __device__ __forceinline__ void store(bf16_t* p, float v) { *p = f32_to_bf16(v); }
  static __device__ __forceinline__ void store4(bf16_t* p, const float (&v)[4]) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
};

}  // namespace phyai
