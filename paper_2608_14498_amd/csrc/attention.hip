// Attention kernels.
//
// One kernel serves both passes.  For sequence b the key space is the
// concatenation of segment 0 (the prefix KV rows, positions 0..n0-1; empty in the
// prefix pass) and segment 1 (the rows of the queries themselves, positions
// n0..), so a key's index in that space IS its position and the causal rule is
// "key index <= query position" everywhere: the prefix pass is causal attention
// over the prompt, the suffix pass sees every prefix key plus the causal block of
// its own response.
//
// bf16 (MFMA): a workgroup owns 4 waves x QW x 32 queries of one q head.  Each
// 64-key tile is staged in LDS (K row-major, V transposed); the wave computes
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16 so that every lane holds the scores of
// ONE query (its softmax row statistics stay in-lane), then O^T += V^T P^T reusing
// the score registers, converted to bf16, directly as the B operand.  K/V tile loads
// for tile t+1 are in flight while tile t is computed (double-buffered LDS).
//
// fp32: one thread per query, K/V tiles in LDS, exact fp32 math.
//
// decode: split-KV over 256-key chunks, all q heads of a kv head per workgroup,
// then a merge over chunks.
#include "device_common.h"
#include "rp_internal.h"

namespace rp {

struct QBlock {
  int b, q_begin, q_end;  // query rows of this block (absolute rows)
};

// Linear q-block index -> (sequence, block); blocks of a sequence are visited
// last-first (the longest causal rows start first).
__device__ __forceinline__ QBlock find_qblock(const SeqTable& st, int qbl, int BQ) {
  for (int b = 0; b < st.n; ++b) {
    const int nq = st.q_cu[b + 1] - st.q_cu[b];
    const int nb = (nq + BQ - 1) / BQ;
    if (qbl < nb) {
      const int qb = nb - 1 - qbl;
      QBlock r;
      r.b = b;
      r.q_begin = st.q_cu[b] + qb * BQ;
      r.q_end = min(st.q_cu[b + 1], r.q_begin + BQ);
      return r;
    }
    qbl -= nb;
  }
  QBlock r;
  r.b = -1;
  r.q_begin = r.q_end = 0;
  return r;
}

// ------------------------------------------------------------------------------------
// bf16 MFMA flash attention
// ------------------------------------------------------------------------------------
constexpr int FA_KT = 64;        // keys per tile
constexpr float kMaskVal = -1e30f;

template <int D, int QW>
__global__ __launch_bounds__(256) void k_attn_bf16(SeqTable st, AttnArgs a) {
  constexpr int BQ = 4 * 32 * QW;
  constexpr int CH = D / 8;              // 16-byte chunks per K row
  constexpr int VT_LD = FA_KT + 4;       // V^T row stride (bf16): 136 bytes
  constexpr int KSTEPS = D / 16;         // MFMA k-steps of S^T
  constexpr int DB = D / 32;             // 32-row blocks of O^T
  constexpr int LOADS = (FA_KT * CH) / 256;
  __shared__ uint4 Ks[2][FA_KT * CH];
  __shared__ __align__(16) bf16_t Vt[2][D * VT_LD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.x % a.Hq;
  const QBlock qb = find_qblock(st, blockIdx.x / a.Hq, BQ);
  if (qb.b < 0) return;
  const int b = qb.b;
  const int G = a.Hq / a.Hkv, g = h / G;
  const int n0 = st.pos0(b);
  const int nq_seq = st.q_cu[b + 1] - st.q_cu[b];
  const int qpos_first = n0 + (qb.q_begin - st.q_cu[b]);
  const int qpos_last = n0 + (qb.q_end - 1 - st.q_cu[b]);
  const int nk = qpos_last + 1;                       // keys needed by this block
  const int ntiles = (nk + FA_KT - 1) / FA_KT;
  const int64_t kv_ld = (int64_t)a.Hkv * D;
  const bf16_t* k0 = (const bf16_t*)a.k0 + (int64_t)g * D;
  const bf16_t* v0 = (const bf16_t*)a.v0 + (int64_t)g * D;
  const bf16_t* k1 = (const bf16_t*)a.k1 + (int64_t)g * D;
  const bf16_t* v1 = (const bf16_t*)a.v1 + (int64_t)g * D;
  const int krow0 = st.k_cu[b], qrow0 = st.q_cu[b];
  (void)nq_seq;

  // ---- queries of this lane: column (lane & 31) of each 32-query block ----
  const int fr = lane & 31, fk = lane >> 5;
  bf16x8_t qf[QW][KSTEPS];
  int qpos[QW];
#pragma unroll
  for (int qi = 0; qi < QW; ++qi) {
    const int qrow_raw = qb.q_begin + (wave * QW + qi) * 32 + fr;
    const int qrow = min(qrow_raw, qb.q_end - 1);
    qpos[qi] = n0 + (qrow_raw - qrow0);
    const bf16_t* qp = (const bf16_t*)a.q + (int64_t)qrow * a.q_ld + h * D + fk * 8;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      qf[qi][ks] = as_bf16x8(*reinterpret_cast<const uint4*>(qp + ks * 16));
    }
  }

  // ---- tile loader: thread handles chunks (key = id / CH, c = id % CH) ----
  static_assert(LOADS == 2 || LOADS == 4, "tile loader covers D = 64 or 128");
  uint4 rk0, rk1, rk2, rk3, rv0, rv1, rv2, rv3;
#define RP_FA_LD1(i_, t_)                                                                  \
  if (i_ < LOADS) {                                                                        \
    const int id = i_ * 256 + tid, key = id / CH, c = id % CH;                             \
    const int kv = min((t_) * FA_KT + key, nk - 1);                                        \
    const int64_t roff = kv < n0 ? (int64_t)(krow0 + kv) * kv_ld : (int64_t)(qrow0 + kv - n0) * kv_ld; \
    rk##i_ = *reinterpret_cast<const uint4*>((kv < n0 ? k0 : k1) + roff + c * 8);          \
    rv##i_ = *reinterpret_cast<const uint4*>((kv < n0 ? v0 : v1) + roff + c * 8);          \
  }
#define RP_FA_GLOAD(t_) RP_FA_LD1(0, t_) RP_FA_LD1(1, t_) RP_FA_LD1(2, t_) RP_FA_LD1(3, t_)
#define RP_FA_ST1(i_, buf_)                                                                \
  if (i_ < LOADS) {                                                                        \
    const int id = i_ * 256 + tid, key = id / CH, c = id % CH;                             \
    Ks[(buf_)][key * CH + (c ^ (key & 7))] = rk##i_;                                       \
    bf16_t* vt_ = &Vt[(buf_)][(c * 8) * VT_LD + (key ^ ((c << 2) & (FA_KT - 1)))];         \
    vt_[0 * VT_LD] = (bf16_t)(rv##i_.x & 0xffffu);                                         \
    vt_[1 * VT_LD] = (bf16_t)(rv##i_.x >> 16);                                             \
    vt_[2 * VT_LD] = (bf16_t)(rv##i_.y & 0xffffu);                                         \
    vt_[3 * VT_LD] = (bf16_t)(rv##i_.y >> 16);                                             \
    vt_[4 * VT_LD] = (bf16_t)(rv##i_.z & 0xffffu);                                         \
    vt_[5 * VT_LD] = (bf16_t)(rv##i_.z >> 16);                                             \
    vt_[6 * VT_LD] = (bf16_t)(rv##i_.w & 0xffffu);                                         \
    vt_[7 * VT_LD] = (bf16_t)(rv##i_.w >> 16);                                             \
  }
#define RP_FA_LSTORE(buf_) RP_FA_ST1(0, buf_) RP_FA_ST1(1, buf_) RP_FA_ST1(2, buf_) RP_FA_ST1(3, buf_)

  f32x16_t o[QW][DB];
  float m_run[QW], l_run[QW];
#pragma unroll
  for (int qi = 0; qi < QW; ++qi) {
    m_run[qi] = kMaskVal;
    l_run[qi] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[qi][db][e] = 0.f;
  }
  const float c2 = a.scale * 1.4426950408889634f;  // scores in log2 units

  RP_FA_GLOAD(0);
  RP_FA_LSTORE(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) { RP_FA_GLOAD(t + 1); }

    // ---- S^T = K Q^T: s[qi][kb][e] = score(key t*64 + kb*32 + 8(e/4) + 4 fk + e%4, query fr) ----
    f32x16_t s[QW][2];
#pragma unroll
    for (int qi = 0; qi < QW; ++qi)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) s[qi][kb][e] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int key = kb * 32 + fr;
        const bf16x8_t kf = as_bf16x8(Ks[buf][key * CH + ((ks * 2 + fk) ^ (key & 7))]);
#pragma unroll
        for (int qi = 0; qi < QW; ++qi)
          s[qi][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qi][ks], s[qi][kb], 0, 0, 0);
      }
    }

    // ---- mask, online softmax (per lane = per query) ----
    const bool need_mask = (t * FA_KT + FA_KT - 1) > qpos_first;
#pragma unroll
    for (int qi = 0; qi < QW; ++qi) {
      float mx = kMaskVal;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = t * FA_KT + kb * 32 + 8 * (e >> 2) + 4 * fk + (e & 3);
          float v = s[qi][kb][e] * c2;
          if (need_mask && key > qpos[qi]) v = kMaskVal;
          s[qi][kb][e] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float m_new = fmaxf(m_run[qi], mx);
      const float alpha = exp2f(m_run[qi] - m_new);
      m_run[qi] = m_new;
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = exp2f(s[qi][kb][e] - m_new);
          s[qi][kb][e] = p;
          ls += p;
        }
      l_run[qi] = l_run[qi] * alpha + ls;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[qi][db][e] *= alpha;
    }

    // ---- O^T += V^T P^T over the 4 sixteen-key steps (kb, hh) ----
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8_t pf[QW];
#pragma unroll
        for (int qi = 0; qi < QW; ++qi) {
          const f32x16_t& sv = s[qi][kb];
          pf[qi] = as_bf16x8(make_uint4(pack_bf2(sv[hh * 8 + 0], sv[hh * 8 + 1]),
                                        pack_bf2(sv[hh * 8 + 2], sv[hh * 8 + 3]),
                                        pack_bf2(sv[hh * 8 + 4], sv[hh * 8 + 5]),
                                        pack_bf2(sv[hh * 8 + 6], sv[hh * 8 + 7])));
        }
        const int key_lo = kb * 32 + hh * 16 + 4 * fk;  // keys key_lo..+3 and key_lo+8..+11
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int dh = db * 32 + fr;
          const int sw = ((dh >> 3) << 2) & (FA_KT - 1);
          const bf16_t* row = &Vt[buf][dh * VT_LD];
          uint2 lo = *reinterpret_cast<const uint2*>(row + (key_lo ^ sw));
          uint2 hi = *reinterpret_cast<const uint2*>(row + ((key_lo + 8) ^ sw));
          const bf16x8_t vf = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
          for (int qi = 0; qi < QW; ++qi)
            o[qi][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qi], o[qi][db], 0, 0, 0);
        }
      }
    }

    if (t + 1 < ntiles) { RP_FA_LSTORE(buf ^ 1); }
    __syncthreads();
  }
#undef RP_FA_LD1
#undef RP_FA_GLOAD
#undef RP_FA_ST1
#undef RP_FA_LSTORE

  // ---- normalise and store: o[qi][db][e] = O^T(dh = db*32 + 8(e/4) + 4 fk + e%4, query fr) ----
#pragma unroll
  for (int qi = 0; qi < QW; ++qi) {
    const int qrow = qb.q_begin + (wave * QW + qi) * 32 + fr;
    const float l = l_run[qi] + __shfl_xor(l_run[qi], 32, kWave);
    if (qrow >= qb.q_end) continue;
    const float inv = 1.0f / l;
    bf16_t* op = (bf16_t*)a.o + (int64_t)qrow * a.Hq * D + h * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int dh = db * 32 + 8 * e4 + 4 * fk;
        uint2 w;
        w.x = pack_bf2(o[qi][db][4 * e4] * inv, o[qi][db][4 * e4 + 1] * inv);
        w.y = pack_bf2(o[qi][db][4 * e4 + 2] * inv, o[qi][db][4 * e4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + dh) = w;
      }
  }
}

// ------------------------------------------------------------------------------------
// fp32 attention: one thread per query, 64-key tiles in LDS, exact fp32 arithmetic.
// ------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(64) void k_attn_f32(SeqTable st, AttnArgs a) {
  constexpr int BQ = 64, KT = 64;
  __shared__ float Ksh[KT][D];
  __shared__ float Vsh[KT][D];
  const int h = blockIdx.x % a.Hq;
  const QBlock qb = find_qblock(st, blockIdx.x / a.Hq, BQ);
  if (qb.b < 0) return;
  const int b = qb.b;
  const int g = h / (a.Hq / a.Hkv);
  const int n0 = st.pos0(b);
  const int qrow0 = st.q_cu[b], krow0 = st.k_cu[b];
  const int qrow_raw = qb.q_begin + threadIdx.x;
  const int qrow = min(qrow_raw, qb.q_end - 1);
  const int qpos = n0 + (qrow_raw - qrow0);
  const int nk = n0 + (qb.q_end - 1 - qrow0) + 1;
  const int64_t kv_ld = (int64_t)a.Hkv * D;
  float q[D], o[D];
  const float* qp = (const float*)a.q + (int64_t)qrow * a.q_ld + h * D;
#pragma unroll
  for (int i = 0; i < D; ++i) {
    q[i] = qp[i];
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int t0 = 0; t0 < nk; t0 += KT) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < KT * D; idx += 64) {
      const int key = idx / D, c = idx % D;
      const int kv = min(t0 + key, nk - 1);
      const int64_t roff = kv < n0 ? (int64_t)(krow0 + kv) * kv_ld : (int64_t)(qrow0 + kv - n0) * kv_ld;
      Ksh[key][c] = ((const float*)(kv < n0 ? a.k0 : a.k1))[roff + g * D + c];
      Vsh[key][c] = ((const float*)(kv < n0 ? a.v0 : a.v1))[roff + g * D + c];
    }
    __syncthreads();
    const int kend = min(KT, nk - t0);
    for (int j = 0; j < kend; ++j) {
      if (t0 + j > qpos) break;
      float sdot = 0.f;
#pragma unroll
      for (int i = 0; i < D; ++i) sdot = fmaf(q[i], Ksh[j][i], sdot);
      const float sv = sdot * a.scale;
      const float mn = fmaxf(m, sv);
      const float alpha = expf(m - mn), p = expf(sv - mn);
      l = l * alpha + p;
#pragma unroll
      for (int i = 0; i < D; ++i) o[i] = fmaf(p, Vsh[j][i], o[i] * alpha);
      m = mn;
    }
  }
  if (qrow_raw < qb.q_end) {
    float* op = (float*)a.o + (int64_t)qrow * a.Hq * D + h * D;
    const float inv = 1.0f / l;
#pragma unroll
    for (int i = 0; i < D; ++i) op[i] = o[i] * inv;
  }
}

static int count_qblocks(const SeqTable& st, int BQ) {
  int n = 0;
  for (int b = 0; b < st.n; ++b) n += (st.q_cu[b + 1] - st.q_cu[b] + BQ - 1) / BQ;
  return n;
}

hipError_t launch_attention(hipStream_t s, bool bf16, const SeqTable& st, const AttnArgs& a, int32_t total_q) {
  if (total_q <= 0) return hipSuccess;
  if (bf16) {
    // D = 128 keeps one 32-query block per wave (two would spill the accumulators).
    if (a.D == 128) {
      k_attn_bf16<128, 1><<<count_qblocks(st, 128) * a.Hq, 256, 0, s>>>(st, a);
    } else {
      const int nqb2 = count_qblocks(st, 256);
      if ((int64_t)nqb2 * a.Hq >= 512)
        k_attn_bf16<64, 2><<<nqb2 * a.Hq, 256, 0, s>>>(st, a);
      else
        k_attn_bf16<64, 1><<<count_qblocks(st, 128) * a.Hq, 256, 0, s>>>(st, a);
    }
  } else {
    const int nqb = count_qblocks(st, 64);
    if (a.D == 128)
      k_attn_f32<128><<<nqb * a.Hq, 64, 0, s>>>(st, a);
    else
      k_attn_f32<64><<<nqb * a.Hq, 64, 0, s>>>(st, a);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------
// Decode attention: split-KV partials + merge.
// ------------------------------------------------------------------------------------
constexpr int DC_KEYS = 256;  // keys per chunk
constexpr int DC_MAXG = 16;

template <typename T, int D>
__global__ __launch_bounds__(256) void k_decode_attn_part(const T* __restrict__ q, int q_ld,
                                                          const T* __restrict__ ck, const T* __restrict__ cv,
                                                          const int32_t* __restrict__ kv_len, int cap,
                                                          int max_pos, int Hq, int Hkv, float scale,
                                                          int nchunks, float* __restrict__ part) {
  constexpr int NPARTS = 256 / D;  // threads per output column
  __shared__ float qs[DC_MAXG][D];
  __shared__ float ps[DC_MAXG][DC_KEYS];
  __shared__ float red[DC_MAXG][4];
  __shared__ float osum[NPARTS][DC_MAXG][D];
  const int c = blockIdx.x % nchunks;
  const int bg = blockIdx.x / nchunks;
  const int g = bg % Hkv, b = bg / Hkv;
  const int G = Hq / Hkv;
  const int n = min(max(kv_len[b], 0), min(cap, max_pos) - 1);  // new token slot; keys 0..n
  const int k_begin = c * DC_KEYS;
  const int nkeys = min(DC_KEYS, n + 1 - k_begin);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  float* out = part + ((int64_t)(b * Hq + g * G) * nchunks + c) * (D + 2);
  const int64_t head_stride = (int64_t)nchunks * (D + 2);
  if (nkeys <= 0) {
    if (tid < G) {
      out[tid * head_stride] = -INFINITY;
      out[tid * head_stride + 1] = 0.f;
    }
    return;
  }
  for (int i = tid; i < G * D; i += 256)
    qs[i / D][i % D] = ldf(q + (int64_t)b * q_ld + (g * G + i / D) * D + i % D);
  __syncthreads();
  const int64_t row_ld = (int64_t)Hkv * D;
  const T* kbase = ck + ((int64_t)b * cap) * row_ld + g * D;
  const T* vbase = cv + ((int64_t)b * cap) * row_ld + g * D;
  // scores: one thread per key
  if (tid < nkeys) {
    const T* kr = kbase + (int64_t)(k_begin + tid) * row_ld;
    float acc[DC_MAXG];
#pragma unroll
    for (int hg = 0; hg < DC_MAXG; ++hg) acc[hg] = 0.f;
    for (int i = 0; i < D; i += 8) {
      float kv8[8];
      load8(kr + i, kv8);
#pragma unroll
      for (int hg = 0; hg < DC_MAXG; ++hg)
        if (hg < G) {
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[hg] = fmaf(qs[hg][i + e], kv8[e], acc[hg]);
        }
    }
#pragma unroll
    for (int hg = 0; hg < DC_MAXG; ++hg)
      if (hg < G) ps[hg][tid] = acc[hg] * scale;
  }
  __syncthreads();
  for (int hg = 0; hg < G; ++hg) {
    const float mx = wave_max(tid < nkeys ? ps[hg][tid] : -INFINITY);
    if (lane == 0) red[hg][w] = mx;
  }
  __syncthreads();
  for (int hg = 0; hg < G; ++hg) {
    const float mx = fmaxf(fmaxf(red[hg][0], red[hg][1]), fmaxf(red[hg][2], red[hg][3]));
    if (tid < nkeys) ps[hg][tid] = expf(ps[hg][tid] - mx);
  }
  __syncthreads();
  // o[hg][d]: thread (d = tid % D, part = tid / D) sums keys k = part, part + NPARTS, ...
  const int d = tid % D, pi = tid / D;
  float acc[DC_MAXG];
#pragma unroll
  for (int hg = 0; hg < DC_MAXG; ++hg) acc[hg] = 0.f;
  for (int k = pi; k < nkeys; k += NPARTS) {
    const float vv = ldf(vbase + (int64_t)(k_begin + k) * row_ld + d);
#pragma unroll
    for (int hg = 0; hg < DC_MAXG; ++hg)
      if (hg < G) acc[hg] = fmaf(ps[hg][k], vv, acc[hg]);
  }
#pragma unroll
  for (int hg = 0; hg < DC_MAXG; ++hg)
    if (hg < G) osum[pi][hg][d] = acc[hg];
  __syncthreads();
  for (int hg = 0; hg < G; ++hg) {
    float* o = out + hg * head_stride;
    if (tid == 0) {
      o[0] = fmaxf(fmaxf(red[hg][0], red[hg][1]), fmaxf(red[hg][2], red[hg][3]));
      float l = 0.f;
      for (int k = 0; k < nkeys; ++k) l += ps[hg][k];
      o[1] = l;
    }
    if (tid < D) {
      float sum = 0.f;
#pragma unroll
      for (int p2 = 0; p2 < NPARTS; ++p2) sum += osum[p2][hg][tid];
      o[2 + tid] = sum;
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(D) void k_decode_attn_merge(const float* __restrict__ part, int nchunks,
                                                         int Hq, T* __restrict__ o) {
  const int bh = blockIdx.x;
  const float* p = part + (int64_t)bh * nchunks * (D + 2);
  float M = -INFINITY;
  for (int c = 0; c < nchunks; ++c) M = fmaxf(M, p[(int64_t)c * (D + 2)]);
  float L = 0.f, acc = 0.f;
  for (int c = 0; c < nchunks; ++c) {
    const float mc = p[(int64_t)c * (D + 2)];
    if (mc == -INFINITY) continue;
    const float wgt = expf(mc - M);
    L += p[(int64_t)c * (D + 2) + 1] * wgt;
    acc += p[(int64_t)c * (D + 2) + 2 + threadIdx.x] * wgt;
  }
  stf(o + (int64_t)bh * D + threadIdx.x, acc / L);
}

size_t decode_attn_partial_floats(int32_t B, int32_t Hq, int32_t D, int32_t cap) {
  const int nchunks = (cap + DC_KEYS - 1) / DC_KEYS;
  return (size_t)B * Hq * nchunks * (D + 2);
}

hipError_t launch_decode_attention(hipStream_t s, bool bf16, const void* q, int32_t q_ld,
                                   const void* cache_k, const void* cache_v, const int32_t* kv_len,
                                   int32_t cap, int32_t max_pos, int32_t B, int32_t Hq, int32_t Hkv,
                                   int32_t D, float scale, float* partials, void* o) {
  const int nchunks = (cap + DC_KEYS - 1) / DC_KEYS;
  const int grid = B * Hkv * nchunks;
#define RP_DEC(T, DD)                                                                            \
  k_decode_attn_part<T, DD><<<grid, 256, 0, s>>>((const T*)q, q_ld, (const T*)cache_k,         \
                                                 (const T*)cache_v, kv_len, cap, max_pos, Hq, Hkv, \
                                                 scale, nchunks, partials);                    \
  k_decode_attn_merge<T, DD><<<B * Hq, DD, 0, s>>>(partials, nchunks, Hq, (T*)o);
  if (bf16) {
    if (D == 128) { RP_DEC(bf16_t, 128) } else { RP_DEC(bf16_t, 64) }
  } else {
    if (D == 128) { RP_DEC(float, 128) } else { RP_DEC(float, 64) }
  }
#undef RP_DEC
  return hipGetLastError();
}

}  // namespace rp
