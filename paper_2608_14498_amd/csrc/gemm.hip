// GEMMs of the backbone: C[M,N] (epi)= A[M,K] . B[N,K]^T with fp32 accumulation.
// A is row-major activations, B is nn.Linear weights [out, in] given as up to three
// row segments (fused q/k/v or gate/up projections without a concatenated copy).
//
// bf16: 256x256x64 macro-tile, 4 waves (2x2), each wave owns 128x128 of C as 4x4
// blocks of v_mfma_f32_32x32x16_bf16.  A/B tiles are staged through LDS, double
// buffered (2 x 64 KiB), with a 16-byte-chunk XOR swizzle so that the 32 rows read
// by one MFMA operand fetch hit distinct banks.  Tiles are visited in groups of 8
// tile-rows and the block index is remapped so each XCD walks a contiguous range of
// tiles (its L2 then holds the shared A rows / B columns).
//
// fp32: a plain 64x64 SIMT tile (exact fp32 FMAs) for the fp32 model.
#include "device_common.h"
#include "rp_internal.h"

namespace rp {

struct GemmArgs {
  int M, N, K;
  const void* A;
  int lda;
  BSeg B;
  int ldb;
  void* C;
  int ldc;
  int tiles_m, tiles_n;
  int k_chunk;       // K range per split (multiple of BK)
  float* partials;   // split-K: [splitk][M][N] fp32
};

template <typename T>
__device__ __forceinline__ const T* brow(const BSeg& b, int n, int ldb) {
  if (n < b.n1) return (const T*)b.b0 + (int64_t)n * ldb;
  if (n < b.n2) return (const T*)b.b1 + (int64_t)(n - b.n1) * ldb;
  return (const T*)b.b2 + (int64_t)(n - b.n2) * ldb;
}

__device__ __forceinline__ void tile_coords(int t, int tiles_m, int tiles_n, int* tm, int* tn) {
  constexpr int G = 8;
  const int per_group = G * tiles_n;
  const int group = t / per_group;
  const int first_m = group * G;
  const int gsize = min(tiles_m - first_m, G);
  const int in = t - group * per_group;
  *tm = first_m + in % gsize;
  *tn = in / gsize;
}

// ------------------------------------------------------------------------------------
// bf16 MFMA GEMM
// ------------------------------------------------------------------------------------
constexpr int GB_M = 256, GB_N = 256, GB_K = 64, G_THREADS = 256;

template <int EPI>
__global__ __launch_bounds__(G_THREADS) void k_gemm_bf16(GemmArgs g) {
  __shared__ uint4 As[2][GB_M * 8];  // [row][8 chunks of 8 bf16], swizzled
  __shared__ uint4 Bs[2][GB_N * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  int tm, tn;
  tile_coords(xcd_remap(blockIdx.x, gridDim.x), g.tiles_m, g.tiles_n, &tm, &tn);
  const int m0 = tm * GB_M, n0 = tn * GB_N;
  const int kbeg = blockIdx.y * g.k_chunk;
  const int kend = min(g.K, kbeg + g.k_chunk);
  const int KT = (kend - kbeg) / GB_K;

  // global->LDS mapping: thread loads chunk (tid & 7) of rows (tid >> 3) + 32 i
  const int lc = tid & 7, lr = tid >> 3;
  const bf16_t* Ab = (const bf16_t*)g.A + kbeg + lc * 8;
  uint4 ra0, ra1, ra2, ra3, ra4, ra5, ra6, ra7, rb0, rb1, rb2, rb3, rb4, rb5, rb6, rb7;
#define RP_LD1(i_, kt_)                                                                   \
  ra##i_ = *reinterpret_cast<const uint4*>(                                               \
      Ab + (int64_t)min(m0 + lr + 32 * i_, g.M - 1) * g.lda + (kt_) * GB_K);              \
  rb##i_ = *reinterpret_cast<const uint4*>(                                               \
      brow<bf16_t>(g.B, min(n0 + lr + 32 * i_, g.N - 1), g.ldb) + kbeg + lc * 8 + (kt_) * GB_K);
#define RP_GLOAD(kt_)                                                                     \
  RP_LD1(0, kt_) RP_LD1(1, kt_) RP_LD1(2, kt_) RP_LD1(3, kt_) RP_LD1(4, kt_) RP_LD1(5, kt_) \
  RP_LD1(6, kt_) RP_LD1(7, kt_)
#define RP_ST1(i_, buf_)                                                                  \
  {                                                                                       \
    const int r_ = lr + 32 * i_;                                                          \
    As[(buf_)][r_ * 8 + (lc ^ (r_ & 7))] = ra##i_;                                        \
    Bs[(buf_)][r_ * 8 + (lc ^ (r_ & 7))] = rb##i_;                                        \
  }
#define RP_LSTORE(buf_)                                                                   \
  RP_ST1(0, buf_) RP_ST1(1, buf_) RP_ST1(2, buf_) RP_ST1(3, buf_) RP_ST1(4, buf_)          \
  RP_ST1(5, buf_) RP_ST1(6, buf_) RP_ST1(7, buf_)

  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  if (KT > 0) {
    RP_GLOAD(0);
    RP_LSTORE(0);
  }
  __syncthreads();

  const int fr = lane & 31, fk = lane >> 5;
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) { RP_GLOAD(kt + 1); }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int ch = ks * 2 + fk;
      bf16x8_t af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wm * 128 + i * 32 + fr;
        af[i] = as_bf16x8(As[buf][r * 8 + (ch ^ (r & 7))]);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = wn * 128 + j * 32 + fr;
        bfr[j] = as_bf16x8(Bs[buf][r * 8 + (ch ^ (r & 7))]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) { RP_LSTORE(buf ^ 1); }
    __syncthreads();
  }

#undef RP_LD1
#undef RP_GLOAD
#undef RP_ST1
#undef RP_LSTORE

  // epilogue: acc[i][j][e] -> row 8*(e/4) + 4*(lane/32) + e%4, col lane%32 of block (i, j)
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + wn * 128 + j * 32 + fr;
      if (n >= g.N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = m0 + wm * 128 + i * 32 + 8 * (e >> 2) + 4 * fk + (e & 3);
        if (m >= g.M) continue;
        const float v = acc[i][j][e];
        if (EPI == -1) {
          g.partials[((int64_t)blockIdx.y * g.M + m) * g.N + n] = v;
        } else if (EPI == EPI_STORE) {
          ((bf16_t*)g.C)[(int64_t)m * g.ldc + n] = f2bf(v);
        } else if (EPI == EPI_STORE_F32) {
          ((float*)g.C)[(int64_t)m * g.ldc + n] = v;
        } else {
          ((float*)g.C)[(int64_t)m * g.ldc + n] += v;
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// fp32 SIMT GEMM (exact fp32 products, fp32 accumulation)
// ------------------------------------------------------------------------------------
constexpr int GF_M = 64, GF_N = 64, GF_K = 16;

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmArgs g) {
  __shared__ float As[GF_K][GF_M + 1];
  __shared__ float Bs[GF_K][GF_N + 1];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  int tm, tn;
  tile_coords(blockIdx.x, g.tiles_m, g.tiles_n, &tm, &tn);
  const int m0 = tm * GF_M, n0 = tn * GF_N;
  const int kbeg = blockIdx.y * g.k_chunk;
  const int kend = min(g.K, kbeg + g.k_chunk);
  float acc[4][4] = {};
  const float* A = (const float*)g.A;
  for (int k0 = kbeg; k0 < kend; k0 += GF_K) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + 256 * i;
      const int r = idx >> 4, kk = idx & 15;
      const int m = m0 + r, n = n0 + r, k = k0 + kk;
      As[kk][r] = (m < g.M && k < kend) ? A[(int64_t)m * g.lda + k] : 0.f;
      Bs[kk][r] = (n < g.N && k < kend) ? brow<float>(g.B, n, g.ldb)[k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < GF_K; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty + 16 * i;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx + 16 * j;
      if (n >= g.N) continue;
      const float v = acc[i][j];
      if (EPI == -1) {
        g.partials[((int64_t)blockIdx.y * g.M + m) * g.N + n] = v;
      } else if (EPI == EPI_ADD_F32) {
        ((float*)g.C)[(int64_t)m * g.ldc + n] += v;
      } else {
        ((float*)g.C)[(int64_t)m * g.ldc + n] = v;
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// split-K reduction + epilogue (fixed summation order: deterministic)
// ------------------------------------------------------------------------------------
template <int EPI, typename T>
__global__ __launch_bounds__(256) void k_splitk_reduce(const float* __restrict__ part, int splitk, int M,
                                                       int N, void* C, int ldc) {
  const int64_t total = (int64_t)M * N;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int z = 0; z < splitk; ++z) v += part[z * total + i];
    const int64_t m = i / N, n = i - m * N;
    if (EPI == EPI_STORE) {
      stf((T*)C + m * ldc + n, v);
    } else if (EPI == EPI_STORE_F32) {
      ((float*)C)[m * ldc + n] = v;
    } else {
      ((float*)C)[m * ldc + n] += v;
    }
  }
}

size_t gemm_partial_floats(int32_t M, int32_t N, int32_t splitk) {
  return splitk > 1 ? (size_t)splitk * M * N : 0;
}

hipError_t launch_gemm(hipStream_t s, bool bf16, int32_t M, int32_t N, int32_t K, const void* A,
                       int32_t lda, const BSeg& B, int32_t ldb, void* C, int32_t ldc, Epi epi,
                       int32_t splitk, float* partials) {
  if (M <= 0 || N <= 0) return hipSuccess;
  GemmArgs g;
  g.M = M;
  g.N = N;
  g.K = K;
  g.A = A;
  g.lda = lda;
  g.B = B;
  g.ldb = ldb;
  g.C = C;
  g.ldc = ldc;
  g.partials = partials;
  if (splitk < 1) splitk = 1;
  const int bk = bf16 ? GB_K : GF_K;
  const int kblocks = (K + bk - 1) / bk;
  if (splitk > kblocks) splitk = kblocks;
  g.k_chunk = ((kblocks + splitk - 1) / splitk) * bk;
  splitk = (K + g.k_chunk - 1) / g.k_chunk;
  const bool split = splitk > 1;
  if (bf16) {
    g.tiles_m = (M + GB_M - 1) / GB_M;
    g.tiles_n = (N + GB_N - 1) / GB_N;
    dim3 grid(g.tiles_m * g.tiles_n, splitk);
    if (split)
      k_gemm_bf16<-1><<<grid, G_THREADS, 0, s>>>(g);
    else if (epi == EPI_STORE)
      k_gemm_bf16<EPI_STORE><<<grid, G_THREADS, 0, s>>>(g);
    else if (epi == EPI_STORE_F32)
      k_gemm_bf16<EPI_STORE_F32><<<grid, G_THREADS, 0, s>>>(g);
    else
      k_gemm_bf16<EPI_ADD_F32><<<grid, G_THREADS, 0, s>>>(g);
  } else {
    g.tiles_m = (M + GF_M - 1) / GF_M;
    g.tiles_n = (N + GF_N - 1) / GF_N;
    dim3 grid(g.tiles_m * g.tiles_n, splitk);
    if (split)
      k_gemm_f32<-1><<<grid, 256, 0, s>>>(g);
    else if (epi == EPI_ADD_F32)
      k_gemm_f32<EPI_ADD_F32><<<grid, 256, 0, s>>>(g);
    else
      k_gemm_f32<EPI_STORE_F32><<<grid, 256, 0, s>>>(g);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !split) return e;
  const int64_t total = (int64_t)M * N;
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 4096);
  if (epi == EPI_STORE && bf16)
    k_splitk_reduce<EPI_STORE, bf16_t><<<blocks, 256, 0, s>>>(partials, splitk, M, N, C, ldc);
  else if (epi == EPI_STORE || epi == EPI_STORE_F32)
    k_splitk_reduce<EPI_STORE_F32, float><<<blocks, 256, 0, s>>>(partials, splitk, M, N, C, ldc);
  else
    k_splitk_reduce<EPI_ADD_F32, float><<<blocks, 256, 0, s>>>(partials, splitk, M, N, C, ldc);
  return hipGetLastError();
}

}  // namespace rp
