// Bandwidth-bound kernels of the prefix/suffix path: embedding with visual
// splice, RMSNorm (+ boundary row assembly), RoPE + KV materialisation,
// SwiGLU, boundary-state gather, fused log-softmax + gather, argmax.
// One row per workgroup; 16-byte vector accesses where the row allows.
#include "device_common.h"
#include "rp_internal.h"

namespace rp {

// ------------------------------------------------------------------------------------
// Visual-slot numbering: vis_idx[t] = number of visual slots (id < 0) before t, or -1.
// One workgroup walks the ids 1024 at a time: each wave numbers its 64 slots with a
// ballot (a lane's slot index is the count of set bits below it), wave totals are
// combined through LDS, and a running base carries over to the next 1024 (whose ids are
// loaded during the current round).
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_visual_index(const int32_t* __restrict__ ids, int T,
                                                       int32_t* __restrict__ vis_idx) {
  __shared__ int wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, nw = blockDim.x >> 6;
  int base = 0;
  int id = tid < T ? ids[tid] : 0;
  for (int t0 = 0; t0 < T; t0 += blockDim.x) {
    const int t = t0 + tid, tn = t + blockDim.x;
    const int id_next = tn < T ? ids[tn] : 0;  // in flight during this round
    const bool vis = t < T && id < 0;
    id = id_next;
    const uint64_t m = __ballot(vis);
    const int below = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[w] = __popcll(m);
    __syncthreads();
    int off = base, tot = 0;
    for (int i = 0; i < nw; ++i) {
      off += i < w ? wsum[i] : 0;
      tot += wsum[i];
    }
    if (t < T) vis_idx[t] = vis ? off + below : -1;
    __syncthreads();  // wsum is rewritten by the next round
    base += tot;
  }
}

hipError_t launch_visual_index(hipStream_t s, const int32_t* ids, int32_t T, int32_t* vis_idx) {
  k_visual_index<<<1, 1024, 0, s>>>(ids, T, vis_idx);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// RMSNorm: out = x / sqrt(mean(x^2) + eps) * w, fp32 math, stored as T.
// ------------------------------------------------------------------------------------
// load(c, v) hands over the row's values c .. c+7.
template <typename T, typename Load>
__device__ __forceinline__ void rmsnorm_row_from(Load load, const T* __restrict__ w, float eps, int d,
                                                 T* __restrict__ out, float* red) {
  constexpr int kMaxChunks = 4;  // rows of up to 4 x 8 values per thread stay in registers
  const int step = blockDim.x * 8;
  if (d <= kMaxChunks * step) {
    // one read of the row; the same summation order as the two-pass loop below
    float v[kMaxChunks][8];
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxChunks; ++j) {
      const int c = threadIdx.x * 8 + j * step;
      if (c < d) {
        load(c, v[j]);
#pragma unroll
        for (int i = 0; i < 8; ++i) ss = fmaf(v[j][i], v[j][i], ss);
      }
    }
    const float tot = block_sum(ss, red);
    const float inv = 1.0f / sqrtf(tot / (float)d + eps);
#pragma unroll
    for (int j = 0; j < kMaxChunks; ++j) {
      const int c = threadIdx.x * 8 + j * step;
      if (c < d) {
        float g[8];
        load8(w + c, g);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[j][i] = v[j][i] * inv * g[i];
        store8(out + c, v[j]);
      }
    }
    return;
  }
  float ss = 0.f;
  for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) {
    float v[8];
    load(c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(v[i], v[i], ss);
  }
  const float tot = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) {
    float v[8], g[8];
    load(c, v);
    load8(w + c, g);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = v[i] * inv * g[i];
    store8(out + c, v);
  }
}

template <typename T>
__device__ __forceinline__ void rmsnorm_row(const float* __restrict__ x, const T* __restrict__ w,
                                            float eps, int d, T* __restrict__ out, float* red) {
  rmsnorm_row_from([&](int c, float(&v)[8]) { load8(x + c, v); }, w, eps, d, out, red);
}

// ------------------------------------------------------------------------------------
// Embedding + visual splice -> fp32 residual rows; with norm_w, also the first layer's
// RMSNorm of each row, from the same registers (one pass over the row).
// ------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_embed(const int32_t* __restrict__ ids,
                                               const int32_t* __restrict__ vis_idx,
                                               const T* __restrict__ visual, int64_t n_visual,
                                               const T* __restrict__ embed, int vocab, int d,
                                               float* __restrict__ X, const T* __restrict__ norm_w, float eps,
                                               T* __restrict__ norm_out) {
  __shared__ float red[16];
  const int t = blockIdx.x;
  const int id = ids[t];
  const T* src = nullptr;
  if (id < 0) {
    const int vi = vis_idx[t];
    if (vi >= 0 && vi < n_visual) src = visual + (int64_t)vi * d;
  } else {
    src = embed + (int64_t)min(id, vocab - 1) * d;
  }
  float* dst = X + (int64_t)t * d;
  auto load = [&](int c, float(&v)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
    if (src) load8(src + c, v);
    store8(dst + c, v);
  };
  if (norm_w) {  // the values the norm reads are those stored to X, exactly
    rmsnorm_row_from(load, norm_w, eps, d, norm_out + (int64_t)t * d, red);
    return;
  }
  for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) {
    float v[8];
    load(c, v);
  }
}

hipError_t launch_embed(hipStream_t s, rp_dtype dt, const int32_t* ids, const int32_t* vis_idx,
                        const void* visual, int64_t n_visual, const void* embed, int32_t vocab,
                        int32_t T, int32_t d, float* X, const void* norm_w, float eps, void* norm_out) {
  if (T <= 0) return hipSuccess;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_embed<E><<<T, 256, 0, s>>>(ids, vis_idx, (const E*)visual, n_visual,
                                      (const E*)embed, vocab, d, X, (const E*)norm_w, eps, (E*)norm_out);
  });
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_decode_embed(const int32_t* __restrict__ ids,
                                                      const T* __restrict__ embed, int vocab, int d,
                                                      float* __restrict__ X) {
  const int b = blockIdx.x;
  const T* src = embed + (int64_t)min(max(ids[b], 0), vocab - 1) * d;
  for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) {
    float v[8];
    load8(src + c, v);
    store8(X + (int64_t)b * d + c, v);
  }
}

hipError_t launch_decode_embed(hipStream_t s, rp_dtype dt, const int32_t* ids, const void* embed,
                               int32_t vocab, int32_t B, int32_t d, float* X) {
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_decode_embed<E><<<B, 256, 0, s>>>(ids, (const E*)embed, vocab, d, X);
  });
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ X, const T* __restrict__ w,
                                                 float eps, int d, T* __restrict__ out) {
  __shared__ float red[16];
  const int64_t r = blockIdx.x;
  rmsnorm_row(X + r * d, w, eps, d, out + r * d, red);
}

hipError_t launch_rmsnorm(hipStream_t s, rp_dtype dt, const float* X, const void* w, float eps, int32_t M,
                          int32_t d, void* out) {
  if (M <= 0) return hipSuccess;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_rmsnorm<E><<<M, 256, 0, s>>>(X, (const E*)w, eps, d, (E*)out);
  });
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_final_norm_rows(SeqTable st, const float* __restrict__ Y,
                                                         const float* __restrict__ h_last,
                                                         const T* __restrict__ w, float eps, int d,
                                                         T* __restrict__ out) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  const int b = seq_of_row(st, r);
  const float* src = (r == st.q_cu[b]) ? h_last + (int64_t)st.grp[b] * d : Y + (int64_t)(r - 1) * d;
  rmsnorm_row(src, w, eps, d, out + (int64_t)r * d, red);
}

hipError_t launch_final_norm_rows(hipStream_t s, rp_dtype dt, const SeqTable& st, const float* Y,
                                  const float* h_last, const void* w, float eps, int32_t R, int32_t d,
                                  void* out) {
  if (R <= 0) return hipSuccess;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_final_norm_rows<E><<<R, 256, 0, s>>>(st, Y, h_last, (const E*)w, eps, d, (E*)out);
  });
  return hipGetLastError();
}

// Prompt scoring rows: row i scores the prompt token at packed position t = pos[i] from
// the final hidden state at t-1.  Valid iff 0 <= t < T, t is not its sequence's first
// token and ids[t] >= 0 (a text token); then out[i] = RMSNorm(hidden[t-1]) and tid[i] =
// ids[t], else out[i] = 0 and tid[i] = -1 (the scoring kernels turn -1 into NaN).
template <typename T>
__global__ __launch_bounds__(256) void k_prompt_rows(SeqTable st, const int32_t* __restrict__ pos,
                                                     const int32_t* __restrict__ ids, int32_t Ttot,
                                                     const float* __restrict__ hidden,
                                                     const T* __restrict__ w, float eps, int d,
                                                     T* __restrict__ out, int32_t* __restrict__ tid) {
  __shared__ float red[16];
  const int i = blockIdx.x;
  const int t = pos[i];
  bool ok = t > 0 && t < Ttot;
  int id = -1;
  if (ok) {
    const int b = seq_of_row(st, t);
    id = ids[t];
    ok = t != st.q_cu[b] && id >= 0;
  }
  T* o = out + (int64_t)i * d;
  if (ok) {
    rmsnorm_row(hidden + (int64_t)(t - 1) * d, w, eps, d, o, red);
  } else {
    float z[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) store8(o + c, z);
  }
  if (threadIdx.x == 0) tid[i] = ok ? id : -1;
}

hipError_t launch_prompt_rows(hipStream_t s, rp_dtype dt, const SeqTable& st, const int32_t* pos, int32_t n,
                              const int32_t* ids, int32_t T, const float* hidden, const void* w, float eps,
                              int32_t d, void* out, int32_t* tid) {
  if (n <= 0) return hipSuccess;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_prompt_rows<E><<<n, 256, 0, s>>>(st, pos, ids, T, hidden, (const E*)w, eps, d, (E*)out, tid);
  });
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// RoPE (rotate-half pairs (i, i+D/2)) + optional q/k/v bias + Q/K/V materialisation.
// The projection row arrives in fp32 (the GEMM accumulator); bias, rotation and the
// single rounding to the storage type happen here.  q (rotated) goes to q_dst, k
// (rotated) and v to k_dst / v_dst.
// ------------------------------------------------------------------------------------
// Pair i rotates by position pos[0] for i < sec0, pos[1] for i < sec01, else pos[2]
// (all equal for 1-D RoPE).
template <typename T>
__device__ __forceinline__ void rope_row(const float* __restrict__ row, const int (&pos)[3], int sec0, int sec01,
                                         int Hq, int Hkv, int D, const T* __restrict__ bq,
                                         const T* __restrict__ bk, const T* __restrict__ bv, const RopeFreq& rf,
                                         T* __restrict__ q_dst, T* __restrict__ k_dst, T* __restrict__ v_dst,
                                         float* cs, bool do_q = true) {
  const int half = D >> 1;
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    float c, s;
    rope_cs(i < sec0 ? pos[0] : i < sec01 ? pos[1] : pos[2], rf.inv_freq[i], &c, &s);
    cs[i] = c;
    cs[64 + i] = s;
  }
  __syncthreads();
  // four consecutive rotary pairs (i .. i+3) per thread: 16-byte loads of x1 and x2 and
  // 4-wide stores (D/2 is a multiple of 4; rows start 16-byte aligned)
  const int quads = half >> 2;
  const int nq = do_q ? Hq * quads : 0, nk = Hkv * quads;
  for (int p = threadIdx.x; p < nq + nk; p += blockDim.x) {
    const bool isq = p < nq;
    const int pp = isq ? p : p - nq;
    const int h = pp / quads, i = (pp - h * quads) * 4;
    const int col = (isq ? 0 : Hq * D) + h * D + i;
    float x1[4], x2[4], y1[4], y2[4];
    load4(row + col, x1);
    load4(row + col + half, x2);
    const T* b = isq ? bq : bk;
    if (b) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        x1[u] += ldf(b + h * D + i + u);
        x2[u] += ldf(b + h * D + i + half + u);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) rope_rotate(x1[u], x2[u], cs[i + u], cs[64 + i + u], &y1[u], &y2[u]);
    T* dst = (isq ? q_dst : k_dst) + h * D + i;
    store4(dst, y1);
    store4(dst + half, y2);
  }
  const int vbase = (Hq + Hkv) * D;
  for (int e = threadIdx.x * 4; e < Hkv * D; e += blockDim.x * 4) {
    float v[4];
    load4(row + vbase + e, v);
    if (bv) {
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] += ldf(bv + e + u);
    }
    store4(v_dst + e, v);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_rope_kv(SeqTable st, const float* __restrict__ qkv, int Hq, int Hkv,
                                                 int D, const T* __restrict__ bq, const T* __restrict__ bk,
                                                 const T* __restrict__ bv, RopeFreq rf, int max_pos, MRope mr, int M,
                                                 int q_last_only, T* __restrict__ q_out, T* __restrict__ k_out,
                                                 T* __restrict__ v_out) {
  __shared__ float cs[128];
  const int r = blockIdx.x;
  bool do_q = true;
  if (q_last_only) {
    const int b = seq_of_row(st, r);
    do_q = r == st.q_cu[b + 1] - 1;
  }
  int pos[3];
  if (mr.pos) {
#pragma unroll
    for (int k = 0; k < 3; ++k) pos[k] = min(max(mr.pos[(int64_t)k * M + r], 0), max_pos - 1);
  } else {
    const int b = seq_of_row(st, r);
    pos[0] = pos[1] = pos[2] = min(max(st.rpos0(b) + (r - st.q_cu[b]), 0), max_pos - 1);
  }
  const int64_t ld = (int64_t)(Hq + 2 * Hkv) * D;
  rope_row<T>(qkv + r * ld, pos, mr.pos ? mr.sec0 : D, mr.pos ? mr.sec01 : D, Hq, Hkv, D, bq, bk, bv, rf,
              q_out + (int64_t)r * Hq * D, k_out + (int64_t)r * Hkv * D, v_out + (int64_t)r * Hkv * D, cs, do_q);
}

// Rotation table of the fused q/k/v epilogue: cs[r * D/2 + i] = (cos, sin) of rotary pair
// i at row r's position (1-D from the sequence table, or multimodal), exactly the values
// k_rope_kv forms for that row.
__global__ __launch_bounds__(64) void k_rope_table(SeqTable st, RopeFreq rf, int max_pos, MRope mr, int M, int half,
                                                   float2* __restrict__ cs) {
  const int r = blockIdx.x;
  int pos[3];
  if (mr.pos) {
#pragma unroll
    for (int k = 0; k < 3; ++k) pos[k] = min(max(mr.pos[(int64_t)k * M + r], 0), max_pos - 1);
  } else {
    const int b = seq_of_row(st, r);
    pos[0] = pos[1] = pos[2] = min(max(st.rpos0(b) + (r - st.q_cu[b]), 0), max_pos - 1);
  }
  const int sec0 = mr.pos ? mr.sec0 : half, sec01 = mr.pos ? mr.sec01 : half;
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    float c, s;
    rope_cs(i < sec0 ? pos[0] : i < sec01 ? pos[1] : pos[2], rf.inv_freq[i], &c, &s);
    cs[(int64_t)r * half + i] = make_float2(c, s);
  }
}

hipError_t launch_rope_table(hipStream_t s, const SeqTable& st, const RopeFreq& rf, int32_t max_pos, const MRope& mr,
                             int32_t M, int32_t D, float2* cs) {
  if (M <= 0) return hipSuccess;
  k_rope_table<<<M, 64, 0, s>>>(st, rf, max_pos, mr, M, D / 2, cs);
  return hipGetLastError();
}

hipError_t launch_rope_kv(hipStream_t s, rp_dtype dt, const SeqTable& st, const float* qkv, int32_t M,
                          int32_t Hq, int32_t Hkv, int32_t D, const void* bq, const void* bk,
                          const void* bv, const RopeFreq& rf, int32_t max_pos, void* q_out, void* k_out,
                          void* v_out, const MRope& mr, bool q_last_only) {
  if (M <= 0) return hipSuccess;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_rope_kv<E><<<M, 256, 0, s>>>(st, qkv, Hq, Hkv, D, (const E*)bq, (const E*)bk,
                                        (const E*)bv, rf, max_pos, mr, M, q_last_only ? 1 : 0, (E*)q_out,
                                        (E*)k_out, (E*)v_out);
  });
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_decode_rope_kv(const float* __restrict__ qkv, int Hq, int Hkv, int D,
                                                        const T* __restrict__ bq, const T* __restrict__ bk,
                                                        const T* __restrict__ bv, RopeFreq rf,
                                                        const int32_t* __restrict__ kv_len, int cap,
                                                        int max_pos, T* __restrict__ q_out,
                                                        T* __restrict__ ck, T* __restrict__ cv) {
  __shared__ float cs[128];
  const int b = blockIdx.x;
  const int slot = min(max(kv_len[b], 0), min(cap, max_pos) - 1);
  const int64_t ld = (int64_t)(Hq + 2 * Hkv) * D;
  const int64_t dst = ((int64_t)b * cap + slot) * Hkv * D;
  const int p3[3] = {slot, slot, slot};
  rope_row<T>(qkv + b * ld, p3, D, D, Hq, Hkv, D, bq, bk, bv, rf, q_out + (int64_t)b * Hq * D, ck + dst, cv + dst, cs);
}

hipError_t launch_decode_rope_kv(hipStream_t s, rp_dtype dt, const float* qkv, int32_t B, int32_t Hq, int32_t Hkv,
                                 int32_t D, const void* bq, const void* bk, const void* bv,
                                 const RopeFreq& rf, const int32_t* kv_len, int32_t cap, int32_t max_pos,
                                 void* q_out, void* cache_k, void* cache_v) {
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_decode_rope_kv<E><<<B, 256, 0, s>>>(qkv, Hq, Hkv, D, (const E*)bq, (const E*)bk,
                                               (const E*)bv, rf, kv_len, cap, max_pos, (E*)q_out,
                                               (E*)cache_k, (E*)cache_v);
  });
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// SwiGLU: act[m, j] = silu(gu[m, j]) * gu[m, F + j]
// ------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_swiglu(const T* __restrict__ gu, int64_t M, int F,
                                                T* __restrict__ act) {
  const int64_t per_row = F / 8;
  const int64_t n = M * per_row;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = i / per_row;
    const int j = (int)(i - m * per_row) * 8;
    float g[8], u[8], o[8];
    load8(gu + m * 2 * F + j, g);
    load8(gu + m * 2 * F + F + j, u);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = g[e] / (1.0f + expf(-g[e])) * u[e];
    store8(act + m * F + j, o);
  }
}

hipError_t launch_swiglu(hipStream_t s, rp_dtype dt, const void* gu, int32_t M, int32_t F, void* act) {
  if (M <= 0) return hipSuccess;
  const int64_t n = (int64_t)M * (F / 8);
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 256 * 64);
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_swiglu<E><<<blocks, 256, 0, s>>>((const E*)gu, M, F, (E*)act);
  });
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Boundary state: h_last[b] = X[q_cu[b+1]-1].
// ------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gather_rows(SeqTable st, const float* __restrict__ X, int d,
                                                     float* __restrict__ h_last) {
  const int b = blockIdx.x;
  const float* src = X + (int64_t)(st.q_cu[b + 1] - 1) * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) h_last[(int64_t)b * d + c] = src[c];
}

hipError_t launch_gather_rows(hipStream_t s, const SeqTable& st, const float* X, int32_t d, float* h_last) {
  k_gather_rows<<<st.n, 256, 0, s>>>(st, X, d, h_last);
  return hipGetLastError();
}

__device__ __forceinline__ void copy_row16(char* __restrict__ dst, const char* __restrict__ src, int bytes) {
  for (int c = threadIdx.x * 16; c < bytes; c += blockDim.x * 16)
    *reinterpret_cast<uint4*>(dst + c) = *reinterpret_cast<const uint4*>(src + c);
}

__global__ __launch_bounds__(256) void k_gather_last(SeqTable st, const char* __restrict__ q, int q_bytes,
                                                     const char* __restrict__ k, const char* __restrict__ v,
                                                     int kv_bytes, const float* __restrict__ X, int d,
                                                     char* __restrict__ qs, char* __restrict__ ks,
                                                     char* __restrict__ vs, float* __restrict__ h) {
  const int b = blockIdx.x;
  const int64_t r = st.q_cu[b + 1] - 1;
  copy_row16(qs + (int64_t)b * q_bytes, q + r * q_bytes, q_bytes);
  copy_row16(ks + (int64_t)b * kv_bytes, k + r * kv_bytes, kv_bytes);
  copy_row16(vs + (int64_t)b * kv_bytes, v + r * kv_bytes, kv_bytes);
  copy_row16((char*)(h + (int64_t)b * d), (const char*)(X + r * d), d * 4);
}

__global__ __launch_bounds__(256) void k_copy_last_rows(SeqTable st, const char* __restrict__ src, int64_t sld,
                                                        char* __restrict__ dst, int64_t dld, int bytes, int scatter) {
  const int b = blockIdx.x;
  const int64_t last = st.q_cu[b + 1] - 1;
  copy_row16(dst + (scatter ? last : b) * dld, src + (scatter ? b : last) * sld, bytes);
}

hipError_t launch_copy_last_rows(hipStream_t s, const SeqTable& st, const void* src, int64_t src_ld, void* dst,
                                 int64_t dst_ld, int32_t bytes, bool scatter) {
  if ((bytes | src_ld | dst_ld) & 15) return hipErrorInvalidValue;
  k_copy_last_rows<<<st.n, 256, 0, s>>>(st, (const char*)src, src_ld, (char*)dst, dst_ld, bytes, scatter ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_gather_last(hipStream_t s, const SeqTable& st, const void* q, int32_t q_bytes, const void* k,
                              const void* v, int32_t kv_bytes, const float* X, int32_t d, void* qs, void* ks,
                              void* vs, float* h) {
  if ((q_bytes | kv_bytes | (d * 4)) & 15) return hipErrorInvalidValue;
  k_gather_last<<<st.n, 256, 0, s>>>(st, (const char*)q, q_bytes, (const char*)k, (const char*)v, kv_bytes, X, d,
                                     (char*)qs, (char*)ks, (char*)vs, h);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Fused log-softmax + gather: lp[r] = l[r, id_r] - (m + log sum exp(l - m)), one pass
// over the row with a running (max, scaled sum) per thread, merged across the block.
// ------------------------------------------------------------------------------------
__device__ __forceinline__ void lse_merge(float& m, float& s, float mo, float so) {
  const float mn = fmaxf(m, mo);
  if (mn == -INFINITY) return;
  s = (m == -INFINITY ? 0.f : s * exp2f(m - mn)) + (mo == -INFINITY ? 0.f : so * exp2f(mo - mn));
  m = mn;
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int NT>
__global__ __launch_bounds__(NT) void k_logsoftmax_gather(const float* __restrict__ logits,
                                                          const int32_t* __restrict__ ids, int V,
                                                          int neg_nan, float* __restrict__ lp) {
  const int r = blockIdx.x;
  const float* row = logits + (int64_t)r * V;
  float m = -INFINITY, s = 0.f;  // in log2 units
  if ((V & 3) == 0) {
    const f32x4_t* row4 = reinterpret_cast<const f32x4_t*>(row);
    const int n4 = V >> 2;
    int i = threadIdx.x;
    for (; i + 3 * NT < n4; i += 4 * NT) {
      f32x4_t a[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] = __builtin_nontemporal_load(row4 + i + u * NT);
      float mx = m;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        mx = fmaxf(mx, fmaxf(fmaxf(a[u].x, a[u].y), fmaxf(a[u].z, a[u].w)) * kLog2e);
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        acc += exp2f(fmaf(a[u].x, kLog2e, -mx)) + exp2f(fmaf(a[u].y, kLog2e, -mx)) +
               exp2f(fmaf(a[u].z, kLog2e, -mx)) + exp2f(fmaf(a[u].w, kLog2e, -mx));
      }
      s = (m == -INFINITY ? 0.f : s * exp2f(m - mx)) + acc;
      m = mx;
    }
    for (; i < n4; i += NT) {
      const f32x4_t a = row4[i];
      const float mx = fmaxf(m, fmaxf(fmaxf(a.x, a.y), fmaxf(a.z, a.w)) * kLog2e);
      const float acc = exp2f(fmaf(a.x, kLog2e, -mx)) + exp2f(fmaf(a.y, kLog2e, -mx)) +
                        exp2f(fmaf(a.z, kLog2e, -mx)) + exp2f(fmaf(a.w, kLog2e, -mx));
      s = (m == -INFINITY ? 0.f : s * exp2f(m - mx)) + acc;
      m = mx;
    }
  } else {
    for (int i = threadIdx.x; i < V; i += NT) {
      const float x = row[i] * kLog2e;
      const float mx = fmaxf(m, x);
      s = (m == -INFINITY ? 0.f : s * exp2f(m - mx)) + exp2f(x - mx);
      m = mx;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float mo = __shfl_xor(m, o, kWave), so = __shfl_xor(s, o, kWave);
    lse_merge(m, s, mo, so);
  }
  __shared__ float sm[NT / 64], ss[NT / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    sm[w] = m;
    ss[w] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = sm[0], S = ss[0];
    for (int k = 1; k < NT / 64; ++k) lse_merge(M, S, sm[k], ss[k]);
    const int id = min(max(ids[r], 0), V - 1);
    lp[r] = (neg_nan && ids[r] < 0) ? __builtin_nanf("") : row[id] - (M + log2f(S)) * kLn2;
  }
}

hipError_t launch_logsoftmax_gather(hipStream_t s, const float* logits, const int32_t* ids, int32_t R,
                                    int32_t V, float* lp, bool neg_nan) {
  if (R <= 0) return hipSuccess;
  k_logsoftmax_gather<256><<<R, 256, 0, s>>>(logits, ids, V, neg_nan ? 1 : 0, lp);
  return hipGetLastError();
}

// Log-probs from the lm_head's online log-sum-exp partials (EPI_LSE): one wave per row
// merges the row's n_part (max, sum) pairs, lp = tgt - (M + log2 S) ln 2.
__global__ __launch_bounds__(64) void k_lse_combine(const float2* __restrict__ lse, const float* __restrict__ tgt,
                                                    int n_part, const int32_t* __restrict__ nan_ids,
                                                    float* __restrict__ lp) {
  const int r = blockIdx.x;
  const float2* p = lse + (int64_t)r * n_part;
  float m = -INFINITY, s = 0.f;
  for (int i = threadIdx.x; i < n_part; i += 64) {
    const float2 v = p[i];
    lse_merge(m, s, v.x, v.y);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float mo = __shfl_xor(m, o, kWave), so = __shfl_xor(s, o, kWave);
    lse_merge(m, s, mo, so);
  }
  if (threadIdx.x == 0)
    lp[r] = (nan_ids && nan_ids[r] < 0) ? __builtin_nanf("") : tgt[r] - (m + log2f(s)) * kLn2;
}

hipError_t launch_lse_combine(hipStream_t s, const float* lse, const float* tgt, int32_t R, int32_t n_part,
                              float* lp, const int32_t* nan_ids) {
  if (R <= 0) return hipSuccess;
  k_lse_combine<<<R, 64, 0, s>>>(reinterpret_cast<const float2*>(lse), tgt, n_part, nan_ids, lp);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Greedy argmax per row (lowest index on ties).
// ------------------------------------------------------------------------------------
__device__ __forceinline__ void argmax_merge(float& best, int& bi, float vb, int ib) {
  if (vb > best || (vb == best && ib < bi)) {
    best = vb;
    bi = ib;
  }
}

__global__ __launch_bounds__(1024) void k_argmax(const float* __restrict__ logits, int V,
                                                 int32_t* __restrict__ out) {
  const int b = blockIdx.x;
  const float* row = logits + (int64_t)b * V;
  float best = -INFINITY;
  int bi = 0x7fffffff;
  if ((V & 3) == 0) {
    const f32x4_t* row4 = reinterpret_cast<const f32x4_t*>(row);
    const int n4 = V / 4, bd = blockDim.x;
    int i = threadIdx.x;
    for (; i + 3 * bd < n4; i += 4 * bd) {  // four independent loads in flight per thread
      f32x4_t x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = row4[i + u * bd];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int c = 0; c < 4; ++c) argmax_merge(best, bi, x[u][c], 4 * (i + u * bd) + c);
    }
    for (; i < n4; i += bd) {
      const f32x4_t x = row4[i];
#pragma unroll
      for (int c = 0; c < 4; ++c) argmax_merge(best, bi, x[c], 4 * i + c);
    }
  } else {
    for (int i = threadIdx.x; i < V; i += blockDim.x) argmax_merge(best, bi, row[i], i);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float vb = __shfl_xor(best, o, kWave);
    const int ib = __shfl_xor(bi, o, kWave);
    argmax_merge(best, bi, vb, ib);
  }
  __shared__ float sv[16];
  __shared__ int si[16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    sv[w] = best;
    si[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < (int)(blockDim.x >> 6); ++k) argmax_merge(best, bi, sv[k], si[k]);
    out[b] = bi == 0x7fffffff ? -1 : bi;
  }
}

hipError_t launch_argmax(hipStream_t s, const float* logits, int32_t B, int32_t V, int32_t* out) {
  k_argmax<<<B, 1024, 0, s>>>(logits, V, out);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Decode-step kernels that fold a split-K reduction (partials [splitk][M][N] fp32, summed
// in split order as k_splitk_reduce does) into the next step, saving a launch and a
// round trip of the reduced rows.
// ------------------------------------------------------------------------------------
// Sum over z < splitk of part[z*zstride + 0..3], four splits in flight (the rows come from
// few workgroups, so each thread keeps several loads outstanding).
__device__ __forceinline__ void splitk_sum4(const float* __restrict__ part, int64_t zstride, int splitk, float* a) {
  float b[4][4] = {};
  int z = 0;
  for (; z + 4 <= splitk; z += 4) {
    float p[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) load4(part + (int64_t)(z + u) * zstride, p[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) b[u][e] += p[u][e];
  }
  for (; z < splitk; ++z) {
    float p[4];
    load4(part + (int64_t)z * zstride, p);
#pragma unroll
    for (int e = 0; e < 4; ++e) b[0][e] += p[e];
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) a[e] = (b[0][e] + b[1][e]) + (b[2][e] + b[3][e]);
}

// X[m] += sum_z part[z][m]; out[m] = RMSNorm(X[m]) * w (one block of 1024 per row).
template <typename T>
__global__ __launch_bounds__(1024) void k_splitk_add_rmsnorm(const float* __restrict__ part, int splitk, int M,
                                                            int d, float* __restrict__ X, const T* __restrict__ w,
                                                            float eps, T* __restrict__ out) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  float* x = X + (int64_t)m * d;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    float a[4], v[4];
    splitk_sum4(part + (int64_t)m * d + c, (int64_t)M * d, splitk, a);
    load4(x + c, v);
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] += a[u];
    store4(x + c, v);
  }
  __syncthreads();  // the row is re-read below with another thread mapping
  rmsnorm_row(x, w, eps, d, out + (int64_t)m * d, red);
}

hipError_t launch_splitk_add_rmsnorm(hipStream_t s, rp_dtype dt, const float* part, int32_t splitk, int32_t M,
                                     int32_t d, float* X, const void* w, float eps, void* out) {
  if (M <= 0) return hipSuccess;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_splitk_add_rmsnorm<E><<<M, 1024, 0, s>>>(part, splitk, M, d, X, (const E*)w, eps, (E*)out);
  });
  return hipGetLastError();
}

// act[m][f] = silu(g) * u with g, u the split-K sums of columns f and F + f of [M][2F].
template <typename T>
__global__ __launch_bounds__(256) void k_splitk_swiglu(const float* __restrict__ part, int splitk, int M, int F,
                                                       T* __restrict__ act) {
  const int64_t per_row = F / 4;
  const int64_t n = (int64_t)M * per_row;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = i / per_row;
    const int f = (int)(i - m * per_row) * 4;
    float g[4], u[4], o[4];
    const float* row = part + m * 2 * F;
    splitk_sum4(row + f, (int64_t)M * 2 * F, splitk, g);
    splitk_sum4(row + F + f, (int64_t)M * 2 * F, splitk, u);
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = g[e] / (1.0f + expf(-g[e])) * u[e];
    store4(act + m * F + f, o);
  }
}

hipError_t launch_splitk_swiglu(hipStream_t s, rp_dtype dt, const float* part, int32_t splitk, int32_t M, int32_t F,
                                void* act) {
  if (M <= 0) return hipSuccess;
  const int64_t n = (int64_t)M * (F / 4);
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 256 * 16);
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_splitk_swiglu<E><<<blocks, 256, 0, s>>>(part, splitk, M, F, (E*)act);
  });
  return hipGetLastError();
}

// RoPE + K/V store from the split-K partials of the q/k/v projection, for rows at 1-D
// positions (the suffix): the row is summed into LDS (dynamic, (Hq + 2 Hkv) D floats), then
// rotated at its sequence position as k_rope_kv does.
template <typename T>
__global__ __launch_bounds__(1024) void k_rope_kv_splitk(SeqTable st, const float* __restrict__ part, int splitk,
                                                        int M, int Hq, int Hkv, int D, const T* __restrict__ bq,
                                                        const T* __restrict__ bk, const T* __restrict__ bv,
                                                        RopeFreq rf, int max_pos, T* __restrict__ q_out,
                                                        T* __restrict__ k_out, T* __restrict__ v_out) {
  extern __shared__ float4 rowsh4[];
  float* row = reinterpret_cast<float*>(rowsh4);
  __shared__ float cs[128];
  const int r = blockIdx.x;
  const int ld = (Hq + 2 * Hkv) * D;
  for (int c = threadIdx.x * 4; c < ld; c += blockDim.x * 4) {
    float a[4];
    splitk_sum4(part + (int64_t)r * ld + c, (int64_t)M * ld, splitk, a);
    *reinterpret_cast<float4*>(row + c) = make_float4(a[0], a[1], a[2], a[3]);
  }
  __syncthreads();
  const int b = seq_of_row(st, r);
  const int p = min(max(st.rpos0(b) + (r - st.q_cu[b]), 0), max_pos - 1);
  const int p3[3] = {p, p, p};
  rope_row<T>(row, p3, D, D, Hq, Hkv, D, bq, bk, bv, rf, q_out + (int64_t)r * Hq * D, k_out + (int64_t)r * Hkv * D,
              v_out + (int64_t)r * Hkv * D, cs);
}

hipError_t launch_rope_kv_splitk(hipStream_t s, rp_dtype dt, const SeqTable& st, const float* part, int32_t splitk,
                                 int32_t M, int32_t Hq, int32_t Hkv, int32_t D, const void* bq, const void* bk,
                                 const void* bv, const RopeFreq& rf, int32_t max_pos, void* q_out, void* k_out,
                                 void* v_out) {
  if (M <= 0) return hipSuccess;
  const size_t lds = (size_t)(Hq + 2 * Hkv) * D * sizeof(float);
  if (lds > 65536 || ((Hq + 2 * Hkv) * D) % 4) return hipErrorInvalidValue;
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_rope_kv_splitk<E><<<M, 1024, lds, s>>>(st, part, splitk, M, Hq, Hkv, D, (const E*)bq, (const E*)bk,
                                             (const E*)bv, rf, max_pos, (E*)q_out, (E*)k_out, (E*)v_out);
  });
  return hipGetLastError();
}

// Decode RoPE + cache write from the split-K partials of the q/k/v projection: the row is
// summed into LDS (dynamic, qkv floats), then rotated as k_decode_rope_kv does.
template <typename T>
__global__ __launch_bounds__(1024) void k_decode_rope_kv_splitk(const float* __restrict__ part, int splitk, int Hq,
                                                               int Hkv, int D, const T* __restrict__ bq,
                                                               const T* __restrict__ bk, const T* __restrict__ bv,
                                                               RopeFreq rf, const int32_t* __restrict__ kv_len,
                                                               int cap, int max_pos, int B, T* __restrict__ q_out,
                                                               T* __restrict__ ck, T* __restrict__ cv) {
  extern __shared__ float4 rowsh4[];
  float* row = reinterpret_cast<float*>(rowsh4);
  __shared__ float cs[128];
  const int b = blockIdx.x;
  const int ld = (Hq + 2 * Hkv) * D;
  for (int c = threadIdx.x * 4; c < ld; c += blockDim.x * 4) {
    float a[4];
    splitk_sum4(part + (int64_t)b * ld + c, (int64_t)B * ld, splitk, a);
    *reinterpret_cast<float4*>(row + c) = make_float4(a[0], a[1], a[2], a[3]);
  }
  __syncthreads();
  const int slot = min(max(kv_len[b], 0), min(cap, max_pos) - 1);
  const int64_t dst = ((int64_t)b * cap + slot) * Hkv * D;
  const int p3[3] = {slot, slot, slot};
  rope_row<T>(row, p3, D, D, Hq, Hkv, D, bq, bk, bv, rf, q_out + (int64_t)b * Hq * D, ck + dst, cv + dst, cs);
}

hipError_t launch_decode_rope_kv_splitk(hipStream_t s, rp_dtype dt, const float* part, int32_t splitk, int32_t B,
                                        int32_t Hq, int32_t Hkv, int32_t D, const void* bq, const void* bk,
                                        const void* bv, const RopeFreq& rf, const int32_t* kv_len, int32_t cap,
                                        int32_t max_pos, void* q_out, void* cache_k, void* cache_v) {
  if (B <= 0) return hipSuccess;
  const size_t lds = (size_t)(Hq + 2 * Hkv) * D * sizeof(float);
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_decode_rope_kv_splitk<E><<<B, 1024, lds, s>>>(part, splitk, Hq, Hkv, D, (const E*)bq, (const E*)bk,
                                                   (const E*)bv, rf, kv_len, cap, max_pos, B, (E*)q_out,
                                                   (E*)cache_k, (E*)cache_v);
  });
  return hipGetLastError();
}

// Decode embedding + the first layer's RMSNorm (one block per sequence).
template <typename T>
__global__ __launch_bounds__(256) void k_decode_embed_norm(const int32_t* __restrict__ ids,
                                                           const T* __restrict__ embed, int vocab, int d,
                                                           float* __restrict__ X, const T* __restrict__ w,
                                                           float eps, T* __restrict__ out) {
  __shared__ float red[16];
  const int b = blockIdx.x;
  const T* src = embed + (int64_t)min(max(ids[b], 0), vocab - 1) * d;
  float* x = X + (int64_t)b * d;
  for (int c = threadIdx.x * 8; c < d; c += blockDim.x * 8) {
    float v[8];
    load8(src + c, v);
    store8(x + c, v);
  }
  __syncthreads();
  rmsnorm_row(x, w, eps, d, out + (int64_t)b * d, red);
}

hipError_t launch_decode_embed_norm(hipStream_t s, rp_dtype dt, const int32_t* ids, const void* embed, int32_t vocab,
                                    int32_t B, int32_t d, float* X, const void* w, float eps, void* out) {
  with_storage(dt, [&](auto tag_) {
    using E = decltype(tag_);
    k_decode_embed_norm<E><<<B, 256, 0, s>>>(ids, (const E*)embed, vocab, d, X, (const E*)w, eps, (E*)out);
  });
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Debug-mode checks (RP_DEBUG): guard bytes between workspace slices, id ranges.
// ------------------------------------------------------------------------------------
__device__ __forceinline__ uint8_t guard_byte(int g, int i) { return (uint8_t)(0xA5 ^ (g * 7) ^ (i * 13)); }

__global__ __launch_bounds__(64) void k_debug_reset(int* rec) {
  if (threadIdx.x < 4) rec[threadIdx.x] = 0;
}

__global__ __launch_bounds__(256) void k_guard_fill(uint8_t* __restrict__ ws, GuardTable t) {
  const int g = blockIdx.x;
  ws[t.off[g] + threadIdx.x] = guard_byte(g, threadIdx.x);
}

__global__ __launch_bounds__(256) void k_guard_check(const uint8_t* __restrict__ ws, GuardTable t, int* rec) {
  const int g = blockIdx.x;
  if (ws[t.off[g] + threadIdx.x] != guard_byte(g, threadIdx.x)) {
    if (atomicCAS(&rec[0], 0, (int)DBG_GUARD) == 0) rec[1] = g;
  }
}

__global__ void k_guard_corrupt(uint8_t* __restrict__ ws, uint64_t off) {
  if (threadIdx.x == 0) ws[off + 17] ^= 0xFF;
}

__global__ __launch_bounds__(256) void k_check_range(const int32_t* __restrict__ v, int n, int lo, int hi, int code,
                                                     int* rec) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const int x = v[i];
    if (x < lo || x >= hi) {
      if (atomicCAS(&rec[0], 0, code) == 0) {
        rec[1] = i;
        rec[2] = x;
      }
    }
  }
}

hipError_t launch_debug_reset(hipStream_t s, int* rec) {
  k_debug_reset<<<1, 64, 0, s>>>(rec);
  return hipGetLastError();
}

hipError_t launch_guard_fill(hipStream_t s, uint8_t* ws, const GuardTable& t) {
  if (t.n <= 0) return hipSuccess;
  k_guard_fill<<<t.n, kGuardBytes, 0, s>>>(ws, t);
  return hipGetLastError();
}

hipError_t launch_guard_check(hipStream_t s, const uint8_t* ws, const GuardTable& t, int* rec) {
  if (t.n <= 0) return hipSuccess;
  k_guard_check<<<t.n, kGuardBytes, 0, s>>>(ws, t, rec);
  return hipGetLastError();
}

hipError_t launch_guard_corrupt(hipStream_t s, uint8_t* ws, const GuardTable& t) {
  if (t.n <= 0) return hipSuccess;
  k_guard_corrupt<<<1, 64, 0, s>>>(ws, t.off[0]);
  return hipGetLastError();
}

hipError_t launch_check_range(hipStream_t s, const int32_t* v, int32_t n, int32_t lo, int32_t hi, int code, int* rec) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>(((int64_t)n + 255) / 256, 1024);
  k_check_range<<<blocks, 256, 0, s>>>(v, n, lo, hi, code, rec);
  return hipGetLastError();
}

}  // namespace rp
