// Internal interface between the host runtime (api.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rollplex.h"

namespace rp {

// Per-call sequence table passed by value as a kernel argument, so that launch
// geometry and row->sequence lookups need no device copy of the host lengths.
// The position of sequence b's first query row equals the length of its first key
// segment (0 in the prefix pass, P_b in the suffix pass).
struct SeqTable {
  int32_t n;                       // sequences
  int32_t q_cu[RP_MAX_SEQS + 1];   // query rows of sequence b: q_cu[b] .. q_cu[b+1]-1
  int32_t k_cu[RP_MAX_SEQS + 1];   // prefix p's KV rows: k_cu[p] .. k_cu[p+1]-1
  int32_t rope0[RP_MAX_SEQS];      // rotary position of the first query row after prefix p
  uint8_t grp[RP_MAX_SEQS];        // prefix of sequence b (b itself unless prefixes are shared)
  int32_t k_drop;                  // rows left out at the end of every first key segment
  // first row and length of sequence b's first key segment; the length is also the
  // index of b's first query row in its key space (the causal rule)
  __host__ __device__ int32_t k_beg(int b) const { return k_cu[grp[b]]; }
  __host__ __device__ int32_t pos0(int b) const { return k_cu[grp[b] + 1] - k_cu[grp[b]] - k_drop; }
  // rotary position of b's first query row (pos0 unless the prefix used multimodal RoPE)
  __host__ __device__ int32_t rpos0(int b) const { return rope0[grp[b]]; }
};
static_assert(RP_MAX_SEQS <= 256, "grp is one byte");

// Row r of the packed queries -> sequence index (binary search over q_cu).
__host__ __device__ inline int seq_of_row(const SeqTable& t, int r) {
  int lo = 0, hi = t.n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (t.q_cu[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

struct RopeFreq {
  double inv_freq[64];  // theta^(-2i/Dh), i < Dh/2 (host float64)
};

enum Epi : int {
  EPI_STORE = 0,      // C[T] = acc
  EPI_STORE_F32 = 1,  // C[f32] = acc
  EPI_ADD_F32 = 2,    // C[f32] += acc  (residual stream)
  EPI_SWIGLU = 3,     // C[T][m, f] = silu(gate) * up; B = {gate rows, up rows}, N = ffn features
  EPI_LSE = 4,        // no C: per-row log-sum-exp partials and the target logit (LseOut)
  EPI_PARTIALS = 5,   // split-K partials [splitk][M][N] only (also for splitk 1); the caller reduces
  EPI_ROPE = 6,       // q/k/v projection: bias, RoPE and the Q/K/V stores fused (RopeOut); 16-bit only
};

// Outputs of the EPI_ROPE epilogue.  The GEMM computes the [M, (Hq + 2 Hkv) D] projection
// rows; column c (head-aligned: D divides 128) gets its bias, the rotate-half pair of a q
// or k column is rotated by cs[m * D/2 + pair] (launch_rope_table), and the row is
// stored in the 16-bit type to q [M, Hq D], k and v [M, Hkv D].  Needs the LDS-staged
// epilogue (8-wave tiles: 128 columns per wave).
struct RopeOut {
  void* q;
  void* k;
  void* v;
  const void* bq;
  const void* bk;
  const void* bv;
  const float2* cs;
  int32_t hq, hkv, D;  // Hq*D, Hkv*D, head_dim
};
// Number of K splits launch_gemm actually uses for a requested splitk.
int32_t gemm_effective_splitk(rp_dtype dt, int32_t K, int32_t splitk);
// Split-K factor suited to launch_gemm's skinny kernel (16-bit, M <= 64 rows, K % 64 == 0).
int32_t gemm_skinny_splitk(int32_t M, int32_t N, int32_t K);

// Outputs of the EPI_LSE epilogue (an lm_head GEMM whose logits are never stored):
// lse[m * n_part + p] = (max, sum of 2^(x log2 e - max)) over column block p of row m, in
// log2 units, n_part = lse_parts(N) blocks of 128 columns; tgt[m] = logit of column ids[m]
// (ids clamped to [0, N)).
struct LseOut {
  const int32_t* ids;
  float* lse;  // float2 [M][n_part]
  float* tgt;  // [M]
};
int32_t lse_parts(int32_t N);

// B operand of a GEMM given as up to three row segments of nn.Linear weights:
// logical row n < n1 -> b0 + n*ldb; n < n2 -> b1 + (n-n1)*ldb; else b2 + (n-n2)*ldb.
// trans: B is one matrix stored transposed, [K][N] with row stride ldb (element (n, k)
// at b0 + k*ldb + n): a row-parallel weight kept in the layout whose shards are
// contiguous (Section "Parallelism-Aware Weight Sharing", Case 2).  Needs N % 8 == 0 and ldb % 8 == 0 for
// 16-bit types, and the EPI_ADD_F32 or split-K epilogue.
struct BSeg {
  const void* b0;
  const void* b1;
  const void* b2;
  int32_t n1, n2;
  bool trans = false;
};

// ---- launchers (return hipGetLastError() of the launch) ----
hipError_t launch_visual_index(hipStream_t s, const int32_t* ids, int32_t T, int32_t* vis_idx);
// With norm_w, also norm_out = RMSNorm(X) * norm_w (the first layer's attention norm).
hipError_t launch_embed(hipStream_t s, rp_dtype dt, const int32_t* ids, const int32_t* vis_idx,
                        const void* visual, int64_t n_visual, const void* embed, int32_t vocab,
                        int32_t T, int32_t d, float* X, const void* norm_w = nullptr, float eps = 0.f,
                        void* norm_out = nullptr);
hipError_t launch_rmsnorm(hipStream_t s, rp_dtype dt, const float* X, const void* w, float eps, int32_t M,
                          int32_t d, void* out);
// Final norm of the suffix rows with boundary assembly: row r of sequence b reads
// h_last[grp[b]] (its prefix's boundary state) if it is the sequence's first response
// row, else Y[r-1].
hipError_t launch_final_norm_rows(hipStream_t s, rp_dtype dt, const SeqTable& st, const float* Y,
                                  const float* h_last, const void* w, float eps, int32_t R, int32_t d,
                                  void* out);
// qkv: fp32 projection rows [M, (Hq+2Hkv)*D]; q_out [M, Hq*D], k_out/v_out [M, Hkv*D] in T.
// Row r of sequence b rotates by position st.rpos0(b) + (r - q_cu[b]), or, when mpos is
// given (device int32 [3][M]), pair i by mpos[sec(i)][r] with sec(i) = 0 for i < sec0,
// 1 for i < sec01, else 2 (multimodal RoPE).  Positions are clamped to [0, max_pos).
struct MRope {
  const int32_t* pos;  // NULL: 1-D positions
  int32_t sec0, sec01;
};
// q_last_only: rotate and store the queries of each sequence's last row only (the other
// rows' query columns are not read).
hipError_t launch_rope_kv(hipStream_t s, rp_dtype dt, const SeqTable& st, const float* qkv, int32_t M,
                          int32_t Hq, int32_t Hkv, int32_t D, const void* bq, const void* bk,
                          const void* bv, const RopeFreq& rf, int32_t max_pos, void* q_out, void* k_out,
                          void* v_out, const MRope& mr, bool q_last_only = false);
hipError_t launch_swiglu(hipStream_t s, rp_dtype dt, const void* gu, int32_t M, int32_t F, void* act);
hipError_t launch_gather_rows(hipStream_t s, const SeqTable& st, const float* X, int32_t d, float* h_last);
// Row copies between the packed rows and one row per sequence b (last(b) = q_cu[b+1]-1):
// gather: dst row b = src row last(b); scatter: dst row last(b) = src row b.  Row strides
// in bytes; bytes per row, strides and pointers 16-byte aligned.
hipError_t launch_copy_last_rows(hipStream_t s, const SeqTable& st, const void* src, int64_t src_ld, void* dst,
                                 int64_t dst_ld, int32_t bytes, bool scatter);
// Last row r = q_cu[b+1]-1 of every sequence b: qs[b] = q[r] (q_bytes), ks[b] = k[r] and
// vs[b] = v[r] (kv_bytes each), h[b] = X[r] (d floats).  Byte counts are multiples of 16.
hipError_t launch_gather_last(hipStream_t s, const SeqTable& st, const void* q, int32_t q_bytes, const void* k,
                              const void* v, int32_t kv_bytes, const float* X, int32_t d, void* qs, void* ks,
                              void* vs, float* h);
// lp[r] = log softmax(logits[r])[ids[r]] (ids clamped to [0, V)); NaN where ids[r] < 0
// when neg_nan is set.
hipError_t launch_logsoftmax_gather(hipStream_t s, const float* logits, const int32_t* ids, int32_t R,
                                    int32_t V, float* lp, bool neg_nan = false);
// Prompt scoring rows (see rp_prompt_logprob): out[i] = final-norm(hidden[pos[i] - 1]) and
// tid[i] = ids[pos[i]] for a valid text position, else a zero row and tid[i] = -1.
hipError_t launch_prompt_rows(hipStream_t s, rp_dtype dt, const SeqTable& st, const int32_t* pos, int32_t n,
                              const int32_t* ids, int32_t T, const float* hidden, const void* w, float eps,
                              int32_t d, void* out, int32_t* tid);
hipError_t launch_argmax(hipStream_t s, const float* logits, int32_t B, int32_t V, int32_t* out);

// GEMM: C[M,N] (epi)= A[M,K] . B[N,K]^T, fp32 accumulation.  For EPI_SWIGLU, N is the
// number of output features f and B = {b0 = gate [N,K], b1 = up [N,K]} (n1 = N); the fused
// epilogue writes silu(A.gate_f) * (A.up_f).  splitk > 1 needs EPI != EPI_SWIGLU.
hipError_t launch_gemm(hipStream_t s, rp_dtype dt, int32_t M, int32_t N, int32_t K, const void* A,
                       int32_t lda, const BSeg& B, int32_t ldb, void* C, int32_t ldc, Epi epi,
                       int32_t splitk, float* partials, const LseOut* lse = nullptr,
                       const RopeOut* rope = nullptr);
// out[m] = argmax over n of (A . B^T)[m][n] (lowest n among equal maxima; NaN never wins; -1
// when a row has no candidate), C itself never stored.  16-bit, one B segment [N][K], M <= 64,
// one K split (gemm_argmax_supported).  parts: gemm_argmax_parts(M, N) ArgmaxPart entries.
struct ArgmaxPart {
  float v;
  int32_t i;
};
bool gemm_argmax_supported(rp_dtype dt, int32_t M, int32_t N, int32_t K, int32_t lda, int32_t ldb);
size_t gemm_argmax_parts(int32_t M, int32_t N);
hipError_t launch_gemm_argmax(hipStream_t s, rp_dtype dt, int32_t M, int32_t N, int32_t K, const void* A,
                              int32_t lda, const BSeg& B, int32_t ldb, ArgmaxPart* parts, int32_t* out);

// Rotation table of EPI_ROPE for M rows (float2 [M][D/2]); positions as launch_rope_kv.
hipError_t launch_rope_table(hipStream_t s, const SeqTable& st, const RopeFreq& rf, int32_t max_pos, const MRope& mr,
                             int32_t M, int32_t D, float2* cs);
// lp[r] = tgt[r] - log sum_v exp(logit_rv) from the EPI_LSE partials; NaN where
// nan_ids[r] < 0 (nan_ids nullable).
hipError_t launch_lse_combine(hipStream_t s, const float* lse, const float* tgt, int32_t R, int32_t n_part,
                              float* lp, const int32_t* nan_ids = nullptr);
// Required float count of `partials` for a split-K GEMM.
size_t gemm_partial_floats(int32_t M, int32_t N, int32_t splitk);

// Attention over packed sequences.  Queries: rows st.q_cu[b].. of q (row stride q_ld,
// head h at column h*D), positions st.pos0(b) + i.  Keys: segment 0 = rows st.k_beg(b)..
// (st.pos0(b) rows, positions 0..) of k0/v0, the KV of b's prefix; segment 1 = the query
// rows themselves of k1/v1 (positions st.pos0(b)+j).  Key visible iff key pos <= query pos.
// k/v rows are [Hkv][D] contiguous.  Output o rows [Hq*D].
struct AttnArgs {
  const void* q;
  int32_t q_ld;
  const void* k0;
  const void* v0;
  const void* k1;
  const void* v1;
  void* o;
  int32_t Hq, Hkv, D;
  float scale;
  // Split-KV (16-bit models): when set, a sequence whose first key segment holds n0 rows
  // splits its keys attn_splits(n0) ways; the splits write (max, sum, unnormalised o)
  // partials here and a merge kernel writes o.  attn_partial_floats() floats: one record
  // of attn_part_record(S, D) floats per (query row, head) for a launch of S split slots,
  // split sp's o at sp * D and its (max, sum) at S * D + 2 sp, so each split's o is whole
  // 128-byte lines written by one workgroup.
  float* part = nullptr;
};
__host__ __device__ inline int attn_part_record(int S, int D) { return S * D + 32; }
// Key splits of a sequence with n0 first-segment keys: a function of n0 alone, so a
// sequence's result does not depend on the sequences packed with it.
#ifndef RP_ATTN_SPLIT_KEYS
#define RP_ATTN_SPLIT_KEYS 4096
#endif
constexpr int kAttnMaxSplits = 8;
__host__ __device__ inline int attn_splits(int n0) {
  const int sp = n0 / RP_ATTN_SPLIT_KEYS;
  return sp < 1 ? 1 : (sp > kAttnMaxSplits ? kAttnMaxSplits : sp);
}
// Partial floats for R query rows whose sequences split at most max_splits ways.
size_t attn_partial_floats(int64_t R, int32_t Hq, int32_t D, int32_t max_splits);
hipError_t launch_attention(hipStream_t s, rp_dtype dt, const SeqTable& st, const AttnArgs& a,
                            int32_t total_q);

// Matrix-core probe: blocks x 256 threads, each wave iters x 8 MFMAs of 32x32x16;
// sink receives blocks * 256 floats.
hipError_t launch_mfma_probe(hipStream_t s, rp_dtype dt, int32_t blocks, int32_t iters, float* sink);
// HBM read probe over bytes (a multiple of 16) of src; sink receives blocks * 256 words.
hipError_t launch_read_probe(hipStream_t s, const void* src, int64_t bytes, int32_t blocks, uint32_t* sink);

// Debug-mode checks (RP_DEBUG): guard bytes after every workspace slice and range checks
// of device-side ids.  rec is a device int[4]: rec[0] = first error code (0 = none),
// rec[1], rec[2] = its details.
struct GuardTable {
  int32_t n;             // guards used (at most kMaxGuards)
  uint64_t off[64];      // byte offset of each 256-byte guard from the workspace base
};
constexpr int kMaxGuards = 64;
constexpr int kGuardBytes = 256;
enum DebugCode : int { DBG_OK = 0, DBG_ID_RANGE = 1, DBG_GUARD = 2, DBG_KV_LEN = 3 };
hipError_t launch_debug_reset(hipStream_t s, int* rec);
hipError_t launch_guard_fill(hipStream_t s, uint8_t* ws, const GuardTable& t);
hipError_t launch_guard_check(hipStream_t s, const uint8_t* ws, const GuardTable& t, int* rec);
// Writes one byte into guard 0 (the host-forced overflow of the debug mode's self-test).
hipError_t launch_guard_corrupt(hipStream_t s, uint8_t* ws, const GuardTable& t);
// Records v[i] outside [lo, hi) as code, i, v[i] (the first one to win the record).
hipError_t launch_check_range(hipStream_t s, const int32_t* v, int32_t n, int32_t lo, int32_t hi, int code, int* rec);

// Decode step pieces.
hipError_t launch_decode_embed(hipStream_t s, rp_dtype dt, const int32_t* ids, const void* embed,
                               int32_t vocab, int32_t B, int32_t d, float* X);
hipError_t launch_decode_rope_kv(hipStream_t s, rp_dtype dt, const float* qkv, int32_t B, int32_t Hq, int32_t Hkv,
                                 int32_t D, const void* bq, const void* bk, const void* bv,
                                 const RopeFreq& rf, const int32_t* kv_len, int32_t cap, int32_t max_pos,
                                 void* q_out, void* cache_k, void* cache_v);
size_t decode_attn_partial_floats(int32_t B, int32_t Hq, int32_t D, int32_t cap);
// Decode kernels that consume split-K partials part[splitk][M][N] (EPI_PARTIALS):
// X[m] += sum; out[m] = RMSNorm(X[m]) * w.
hipError_t launch_splitk_add_rmsnorm(hipStream_t s, rp_dtype dt, const float* part, int32_t splitk, int32_t M,
                                     int32_t d, float* X, const void* w, float eps, void* out);
// act[m][f] = silu(sum of column f) * (sum of column F + f), N = 2F.
hipError_t launch_splitk_swiglu(hipStream_t s, rp_dtype dt, const float* part, int32_t splitk, int32_t M, int32_t F,
                                void* act);
// launch_decode_rope_kv on the summed q/k/v projection rows.
hipError_t launch_decode_rope_kv_splitk(hipStream_t s, rp_dtype dt, const float* part, int32_t splitk, int32_t B,
                                        int32_t Hq, int32_t Hkv, int32_t D, const void* bq, const void* bk,
                                        const void* bv, const RopeFreq& rf, const int32_t* kv_len, int32_t cap,
                                        int32_t max_pos, void* q_out, void* cache_k, void* cache_v);
// launch_rope_kv (1-D positions from the table, all rows) on the q/k/v projection rows
// summed from their split-K partials [splitk][M][(Hq + 2 Hkv) D]; hipErrorInvalidValue when
// a row does not fit 64 KiB of LDS.
hipError_t launch_rope_kv_splitk(hipStream_t s, rp_dtype dt, const SeqTable& st, const float* part, int32_t splitk,
                                 int32_t M, int32_t Hq, int32_t Hkv, int32_t D, const void* bq, const void* bk,
                                 const void* bv, const RopeFreq& rf, int32_t max_pos, void* q_out, void* k_out,
                                 void* v_out);
// X[b] = E[ids[b]] (clamped); out[b] = RMSNorm(X[b]) * w.
hipError_t launch_decode_embed_norm(hipStream_t s, rp_dtype dt, const int32_t* ids, const void* embed, int32_t vocab,
                                    int32_t B, int32_t d, float* X, const void* w, float eps, void* out);
hipError_t launch_decode_attention(hipStream_t s, rp_dtype dt, const void* q, int32_t q_ld,
                                   const void* cache_k, const void* cache_v, const int32_t* kv_len,
                                   int32_t cap, int32_t max_pos, int32_t B, int32_t Hq, int32_t Hkv,
                                   int32_t D, float scale, float* partials, void* o);

}  // namespace rp
