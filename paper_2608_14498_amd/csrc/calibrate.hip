// Matrix-core throughput probe (measurement aid).  The published dense 16-bit peak assumes
// the full engine clock; under a sustained MFMA load on random operands the part runs at a
// power-limited clock, so the benchmark reports this probe's rate beside the published
// figure.  Every wave issues iters x 8 independent 32x32x16 MFMAs (8 accumulator chains)
// on register operands that alternate between two random bit patterns per lane, as a
// GEMM's operands switch; nothing touches memory until the store that keeps the sums live.
#include "device_common.h"
#include "rp_internal.h"

namespace rp {

__device__ __forceinline__ float probe_uniform(uint32_t h) {
  h ^= h >> 16;
  h *= 0x7feb352du;
  h ^= h >> 15;
  h *= 0x846ca68bu;
  h ^= h >> 16;
  return (float)(h & 0xffffff) * (2.0f / 16777216.0f) - 1.0f;  // [-1, 1)
}

template <typename T16>
__global__ __launch_bounds__(256) void k_mfma_probe(int iters, float* __restrict__ sink) {
  typedef Half16<T16> H;
  typedef typename H::V8 V8;
  const uint32_t gid = blockIdx.x * 256u + threadIdx.x;
  V8 a[2], b[2];
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    uint32_t wa[4], wb[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t base = (gid * 16u + s * 8u + k * 2u) * 2654435761u;
      wa[k] = H::pack2(probe_uniform(base), probe_uniform(base + 1u));
      wb[k] = H::pack2(probe_uniform(base + 0x9e3779b9u), probe_uniform(base + 0x9e3779bau));
    }
    a[s] = H::as_v8(make_uint4(wa[0], wa[1], wa[2], wa[3]));
    b[s] = H::as_v8(make_uint4(wb[0], wb[1], wb[2], wb[3]));
  }
  f32x16_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = H::mma(a[j & 1], b[(j >> 1) & 1], acc[j]);
  }
  float t = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) t += acc[j][e];
  sink[gid] = t;
}

hipError_t launch_mfma_probe(hipStream_t s, rp_dtype dt, int32_t blocks, int32_t iters, float* sink) {
  if (dt == RP_F16)
    k_mfma_probe<f16_t><<<blocks, 256, 0, s>>>(iters, sink);
  else
    k_mfma_probe<bf16_t><<<blocks, 256, 0, s>>>(iters, sink);
  return hipGetLastError();
}

// HBM read probe: a grid-stride stream of 16-byte non-temporal loads, four in flight per
// thread, folded with XOR into one word per thread (sink) so no load is dead.
typedef uint32_t probe_u4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256) void k_read_probe(const probe_u4* __restrict__ src, int64_t n16,
                                                    uint32_t* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0u;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    probe_u4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = __builtin_nontemporal_load(src + i + u * stride);
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const probe_u4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  sink[blockIdx.x * 256 + threadIdx.x] = acc;
}

hipError_t launch_read_probe(hipStream_t s, const void* src, int64_t bytes, int32_t blocks, uint32_t* sink) {
  k_read_probe<<<blocks, 256, 0, s>>>((const probe_u4*)src, bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace rp
