// Device helpers shared by the gfx950 kernels: 16-bit storage types (bf16, fp16),
// vector types, wavefront (64-lane) reductions, XCD-aware block remapping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rp {

typedef uint16_t bf16_t;  // raw bfloat16 bits
typedef _Float16 f16_t;   // IEEE binary16
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;  // LDS operand of ds_read_b64_tr_b16

// Host-side dispatch on the storage type of a model: calls f(T()) with T = float,
// bf16_t or f16_t for RP_F32, RP_BF16 and RP_F16.
template <class F>
inline void with_storage(int dtype, F&& f) {
  if (dtype == 1)
    f(bf16_t());
  else if (dtype == 2)
    f(f16_t());
  else
    f(float());
}
// The same over the two 16-bit types only (MFMA kernels).
template <class F>
inline void with_half16(int dtype, F&& f) {
  if (dtype == 2)
    f(f16_t());
  else
    f(bf16_t());
}

constexpr int kWave = 64;
constexpr int kXcds = 8;  // MI355X: 8 XCDs, workgroups dispatched round-robin

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// float -> bf16 and fp16 by the gfx950 packed conversions (v_cvt_pk_bf16_f32,
// v_cvt_pk_f16_f32): round to nearest even, NaN stays NaN, overflow goes to inf.
// Two floats pack into one word, lo in bits 0..15.
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ bf16_t f2bf(float f) { return (bf16_t)(pack_bf2(f, 0.f) & 0xffffu); }

__device__ __forceinline__ uint32_t pack_h2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, f16x2_t));
}
__device__ __forceinline__ f16_t f2h(float f) { return (f16_t)f; }
__device__ __forceinline__ float h2f_bits(uint32_t bits16) {
  return (float)__builtin_bit_cast(f16_t, (uint16_t)bits16);
}

// Generic scalar load/store of a storage element as float.
__device__ __forceinline__ float ldf(const float* p) { return *p; }
__device__ __forceinline__ float ldf(const bf16_t* p) { return bf2f(*p); }
__device__ __forceinline__ float ldf(const f16_t* p) { return (float)*p; }
__device__ __forceinline__ void stf(float* p, float v) { *p = v; }
__device__ __forceinline__ void stf(bf16_t* p, float v) { *p = f2bf(v); }
__device__ __forceinline__ void stf(f16_t* p, float v) { *p = f2h(v); }

// The two 16-bit storage types of the MFMA paths: operand vector type, the 32x32x16
// MFMA with fp32 accumulation, and float -> storage packing.
template <typename T16> struct Half16;
template <> struct Half16<bf16_t> {
  typedef bf16x8_t V8;
  static __device__ __forceinline__ V8 as_v8(uint4 v) { return __builtin_bit_cast(V8, v); }
  static __device__ __forceinline__ f32x16_t mma(V8 a, V8 b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack2(float lo, float hi) { return pack_bf2(lo, hi); }
  static __device__ __forceinline__ float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
  static __device__ __forceinline__ float hi_f(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
};
template <> struct Half16<f16_t> {
  typedef f16x8_t V8;
  static __device__ __forceinline__ V8 as_v8(uint4 v) { return __builtin_bit_cast(V8, v); }
  static __device__ __forceinline__ f32x16_t mma(V8 a, V8 b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack2(float lo, float hi) { return pack_h2(lo, hi); }
  static __device__ __forceinline__ float lo_f(uint32_t w) { return h2f_bits(w & 0xffffu); }
  static __device__ __forceinline__ float hi_f(uint32_t w) { return h2f_bits(w >> 16); }
};

// A pointer the caller knows to be the same in every lane, moved to scalar registers.
template <typename T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t u = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u), hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (T*)(((uint64_t)hi << 32) | lo);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Sum over the 16 lanes of a DPP row (lanes 16r .. 16r+15), every lane gets the total;
// in-register lane moves (quad_perm for xor 1 and 2, row_ror 4 and 8), no LDS traffic.
__device__ __forceinline__ float row16_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false));  // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xf, 0xf, false));  // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xf, 0xf, false)); // row_ror 4
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xf, 0xf, false)); // row_ror 8
  return v;
}
// Sum over aligned groups of 8 lanes (row_ror 4 wraps within 16, so use a half-row mask).
__device__ __forceinline__ float oct8_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false));
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xf, 0xf, false));
  v += __shfl_xor(v, 4, 64);
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024). `red` holds >= 16 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

// Bijective remap of a 1-D block index so that each XCD's blocks (dispatched
// round-robin: block i runs on XCD i % 8) form one contiguous range of the
// returned index; neighbouring tiles then share that XCD's L2.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  const int q = n / kXcds, r = n % kXcds;
  const int x = id % kXcds, local = id / kXcds;
  const int base = x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q;
  return base + local;
}

// Row copy helpers: 8 elements per step (d % 8 == 0).
__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const f16_t* p, float* v) {
  uint4 u = *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = h2f_bits(w[i] & 0xffffu);
    v[2 * i + 1] = h2f_bits(w[i] >> 16);
  }
}
// Raw 8-element chunks (16-bit types: one 16-byte load; fp32: two), loaded first and
// widened later.
struct Raw8b { uint4 a; };
struct Raw8h { uint4 a; };
struct Raw8f { uint4 a, b; };
template <typename T> struct Raw8;
template <> struct Raw8<bf16_t> { typedef Raw8b type; };
template <> struct Raw8<f16_t> { typedef Raw8h type; };
template <> struct Raw8<float> { typedef Raw8f type; };
__device__ __forceinline__ Raw8b ld_raw8(const bf16_t* p) { return Raw8b{*reinterpret_cast<const uint4*>(p)}; }
__device__ __forceinline__ Raw8h ld_raw8(const f16_t* p) { return Raw8h{*reinterpret_cast<const uint4*>(p)}; }
__device__ __forceinline__ void unpack8(const Raw8h& c, float* v) {
  const uint32_t w[4] = {c.a.x, c.a.y, c.a.z, c.a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = h2f_bits(w[i] & 0xffffu);
    v[2 * i + 1] = h2f_bits(w[i] >> 16);
  }
}
__device__ __forceinline__ Raw8f ld_raw8(const float* p) {
  return Raw8f{*reinterpret_cast<const uint4*>(p), *reinterpret_cast<const uint4*>(p + 4)};
}
__device__ __forceinline__ void unpack8(const Raw8b& c, float* v) {
  const uint32_t w[4] = {c.a.x, c.a.y, c.a.z, c.a.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void unpack8(const Raw8f& c, float* v) {
  v[0] = __uint_as_float(c.a.x); v[1] = __uint_as_float(c.a.y);
  v[2] = __uint_as_float(c.a.z); v[3] = __uint_as_float(c.a.w);
  v[4] = __uint_as_float(c.b.x); v[5] = __uint_as_float(c.b.y);
  v[6] = __uint_as_float(c.b.z); v[7] = __uint_as_float(c.b.w);
}
__device__ __forceinline__ void load8(const float* p, float* v) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(bf16_t* p, const float* v) {
  uint4 u;
  u.x = pack_bf2(v[0], v[1]);
  u.y = pack_bf2(v[2], v[3]);
  u.z = pack_bf2(v[4], v[5]);
  u.w = pack_bf2(v[6], v[7]);
  *reinterpret_cast<uint4*>(p) = u;
}
__device__ __forceinline__ void store8(f16_t* p, const float* v) {
  uint4 u;
  u.x = pack_h2(v[0], v[1]);
  u.y = pack_h2(v[2], v[3]);
  u.z = pack_h2(v[4], v[5]);
  u.w = pack_h2(v[6], v[7]);
  *reinterpret_cast<uint4*>(p) = u;
}
__device__ __forceinline__ void store8(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
// Four consecutive elements (8-byte aligned for 16-bit types, 16-byte for fp32).
__device__ __forceinline__ void store4(bf16_t* p, const float* v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_bf2(v[0], v[1]), pack_bf2(v[2], v[3]));
}
__device__ __forceinline__ void store4(f16_t* p, const float* v) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack_h2(v[0], v[1]), pack_h2(v[2], v[3]));
}
__device__ __forceinline__ void store4(float* p, const float* v) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void load4(const float* p, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}


// Position-dependent RoPE cos/sin: angle = pos * inv_freq formed in float64,
// reduced to [-pi, pi] in float64, then evaluated in float32.
__device__ __forceinline__ void rope_cs(int pos, double inv_freq, float* c, float* s) {
  const double a = (double)pos * inv_freq;
  const double k = rint(a * 0.15915494309189535);  // 1 / (2 pi)
  const double r = fma(-k, 6.283185307179586, a);
  const float rf = (float)r;
  *s = sinf(rf);
  *c = cosf(rf);
}

// Rotate-half pair (x1, x2) = (x_i, x_{i+D/2}) by the angle whose cosine and sine are
// (c, s).  Written with explicit fused multiply-adds so that every kernel that rotates
// (the RoPE kernels and the fused q/k/v GEMM epilogue) rounds identically.
__device__ __forceinline__ void rope_rotate(float x1, float x2, float c, float s, float* y1, float* y2) {
  *y1 = fmaf(x1, c, -(x2 * s));
  *y2 = fmaf(x2, c, x1 * s);
}

}  // namespace rp
