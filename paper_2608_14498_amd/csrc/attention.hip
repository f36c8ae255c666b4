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
// bf16 / fp16 MFMA flash attention
//
// K and V tiles are staged row-major in LDS ([key][Dh], 16-byte chunks, per-operand XOR
// swizzle) by direct global->LDS loads (buffer_load ... lds): one load instruction fills
// 64 consecutive chunks, and the swizzle is applied by choosing which global chunk each
// lane fetches.  The two LDS buffers are separate arrays and the tile loop is unrolled
// by two, so every LDS access names its buffer at compile time and the compiler waits
// on exactly the loads that filled it.  Each key segment of the sequence is one buffer
// resource whose extent ends at the segment's last row: rows past the end read as
// zeros (keys that the causal mask removes, with zero values), so no index is clamped.
//
// S^T = K Q^T reads K fragments with ds_read_b128.  The V^T operand of O^T += V^T P^T
// is read with ds_read_b64_tr_b16: within a 16-lane group, lane i receives column i%4
// of the 8-byte chunks addressed by lanes i/4, i/4+4, i/4+8, i/4+12, so lane p
// addressing V[k0 + p/4][d0 + 4(p%4)] hands lane i the four keys k0..k0+3 of head
// dimension d0+i -- the MFMA operand, with no transposed copy of V.
// ------------------------------------------------------------------------------------
// Block -> (q block, q head), XCD-aware.  Workgroup i runs on XCD i % 8, which has its
// own L2, so the q heads that share a kv head (one GQA group, reading the same K/V
// tiles) are kept on one XCD: with Hkv dividing 8, each group gets 8/Hkv XCDs that take
// its (q block, head) items in turn; with Hkv a multiple of 8, XCD x gets the groups
// g = x mod 8.  Items run q-block-major, longest q blocks first.  Other head counts use
// the plain order.  Returns the grid size; blocks past the work map to q blocks
// beyond the last (find_qblock reports none).
struct FaMap {
  int mode, G, X;  // mode 0: plain, 1: 8/Hkv XCDs per group, 2: Hkv/8 groups per XCD
};
__host__ __device__ inline FaMap fa_map(int Hq, int Hkv) {
  FaMap m;
  m.G = Hq / Hkv;
  if (8 % Hkv == 0) {
    m.mode = 1;
    m.X = 8 / Hkv;
  } else if (Hkv % 8 == 0) {
    m.mode = 2;
    m.X = Hkv / 8;
  } else {
    m.mode = 0;
    m.X = 1;
  }
  return m;
}
inline int fa_grid(const FaMap& m, int nqb, int Hq) {
  if (m.mode == 1) return 8 * ((nqb * m.G + m.X - 1) / m.X);
  return nqb * Hq;
}
__device__ __forceinline__ void fa_block(const FaMap& m, int bid, int Hq, int* qbl, int* h) {
  const int x = bid & 7, r = bid >> 3;
  if (m.mode == 1) {
    const int i = r * m.X + x % m.X;
    *qbl = i / m.G;
    *h = (x / m.X) * m.G + i % m.G;
  } else if (m.mode == 2) {
    const int per = m.X * m.G;  // items of one q block on one XCD
    const int rem = r % per;
    *qbl = r / per;
    *h = ((rem / m.G) * 8 + x) * m.G + rem % m.G;
  } else {
    *qbl = bid / Hq;
    *h = bid % Hq;
  }
}

constexpr float kMaskVal = -1e30f;
constexpr float kLazy = 8.f;  // log2 headroom of the lazily updated softmax max
typedef __attribute__((address_space(3))) void lds_void_t;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// LDS chunk swizzles (16-byte chunks of a K or V row).  K rows are read 16 bytes per lane
// (row = key), so consecutive keys take distinct chunks.  V rows are read with
// ds_read_b64_tr_b16: in each 32-lane half, lane bits 0,1,4 pick the column within a
// 32-column block and bits 2,3 the key within a group of four; XOR-ing the key's low two
// bits into chunk bits 2,3 (D = 128: a row spans all 64 banks) or 1,2 (D = 64: two rows
// do, the key's bit 0 picking the half) makes the 32 lanes of a half hit 64 distinct
// banks.  (Chunk bits 1,2 at D = 128 left one bank bit fixed: half the banks, and the
// LDS bank-conflict counter at 14% of the prefix kernel's cycles.)
template <int D>
__device__ __forceinline__ int kswz(int key) { return D == 128 ? (key & 15) : (key & 7); }
template <int D>
__device__ __forceinline__ int vswz(int key) { return D == 128 ? (key & 3) << 2 : (key & 3) << 1; }

template <typename T16, int D, int QW, int KT, int NW = 4>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(QW == 1 ? 2 : 1, QW == 1 ? 2 : 1)))
void k_attn_bf16(SeqTable st, AttnArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)  // buffer resources exist only in the device pass
  typedef Half16<T16> H;
  typedef typename H::V8 V8;
  constexpr int BQ = NW * 32 * QW;
  constexpr int CH = D / 8;               // 16-byte chunks per K/V row
  constexpr int KSTEPS = D / 16;          // MFMA k-steps of S^T (over Dh)
  constexpr int DB = D / 32;              // 32-row blocks of O^T
  constexpr int KB = KT / 32;             // 32-key blocks per tile
  constexpr int LOADS = (KT * CH) / (NW * 64);  // load instructions per wave per matrix
  static_assert(LOADS >= 1 && (KT * CH) % (NW * 64) == 0 && 64 % CH == 0, "tile loader");
  __shared__ u32x4_t Ks0[KT * CH], Ks1[KT * CH], Vs0[KT * CH], Vs1[KT * CH];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int h, qbl;
  fa_block(fa_map(a.Hq, a.Hkv), blockIdx.x, a.Hq, &qbl, &h);
  QBlock qb = find_qblock(st, qbl, BQ);
  if (qb.b < 0) return;
  // Block-uniform values, moved to scalar registers (the sequence table is indexed
  // dynamically, which the compiler cannot prove uniform).
  const int b = __builtin_amdgcn_readfirstlane(qb.b);
  qb.q_begin = __builtin_amdgcn_readfirstlane(qb.q_begin);
  qb.q_end = __builtin_amdgcn_readfirstlane(qb.q_end);
  const int G = a.Hq / a.Hkv, g = h / G;
  const int krow0 = __builtin_amdgcn_readfirstlane(st.k_beg(b));
  const int n0 = __builtin_amdgcn_readfirstlane(st.pos0(b));
  const int qrow0 = __builtin_amdgcn_readfirstlane(st.q_cu[b]);
  const int nq = __builtin_amdgcn_readfirstlane(st.q_cu[b + 1]) - qrow0;
  const int qpos_first = n0 + (qb.q_begin - qrow0);
  const int qpos_last = n0 + (qb.q_end - 1 - qrow0);
  // Key tiles: the first P0 tiles hold the n0 first-segment keys (the last of them may be
  // partial: its rows past n0 read as zeros and are masked), the rest the segment-1 keys
  // n0 .. qpos_last this block needs, from position n0 on.  No tile mixes the segments,
  // so each tile's copies name one buffer resource.  Tile t's first key position is
  // kpos0(t).
  const int P0 = (n0 + KT - 1) / KT;
  auto kpos0 = [&](int t) { return t < P0 ? t * KT : n0 + (t - P0) * KT; };
  // Tiles t_begin .. t_end-1 of this block.  Split-KV: a sequence with n0 first-segment
  // keys has nsp = attn_splits(n0) splits; split sp takes its share of the P0 first-
  // segment tiles, and the last split also the segment-1 tiles (the causal keys), so it
  // is the longest and runs at blockIdx.y 0.  Every split holds at least one tile
  // (P0 / nsp >= RP_ATTN_SPLIT_KEYS / KT).
  int t_begin = 0, t_end = P0 + (qpos_last - n0 + KT) / KT, sp = 0;
  const int nsp = a.part ? attn_splits(n0) : 1;
  if ((int)blockIdx.y >= nsp) return;
  if (nsp > 1) {
    sp = nsp - 1 - (int)blockIdx.y;
    const int per = (P0 + nsp - 1) / nsp;
    t_begin = sp * per;
    if (sp < nsp - 1) t_end = t_begin + per;
  }

  // Key segments as buffer resources: segment 0 = the n0 prefix rows, segment 1 = the
  // nq rows of the queries; key kv of segment s is at byte (kv - start_s) * row_bytes.
  // The host guarantees those offsets, past-the-end tile rows included, fit 32 bits.
  const int64_t kv_ld = (int64_t)a.Hkv * D;
  const uint32_t row_bytes = (uint32_t)kv_ld * sizeof(T16);
  const uint32_t ext0 = n0 > 0 ? (uint32_t)(n0 - 1) * row_bytes + D * sizeof(T16) : 0u;
  const uint32_t ext1 = (uint32_t)(nq - 1) * row_bytes + D * sizeof(T16);
  const int64_t e0 = (int64_t)krow0 * kv_ld + (int64_t)g * D, e1 = (int64_t)qrow0 * kv_ld + (int64_t)g * D;
  // (64-bit products are formed in vector registers: uniform_ptr returns them to scalar
  // registers, where a buffer resource must live.)
  const __amdgpu_buffer_rsrc_t rsK0 =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr((void*)((const T16*)a.k0 + e0)), 0, (int)ext0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsV0 =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr((void*)((const T16*)a.v0 + e0)), 0, (int)ext0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsK1 =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr((void*)((const T16*)a.k1 + e1)), 0, (int)ext1, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsV1 =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr((void*)((const T16*)a.v1 + e1)), 0, (int)ext1, 0x00020000);

  // Load instruction j of this wave fills LDS chunks (wave*LOADS + j)*64 + lane, i.e.
  // tile key (wave*LOADS + j)*64/CH + lane/CH, physical chunk lane%CH, which holds
  // logical chunk (lane%CH) ^ swizzle(key).
  uint32_t koff[LOADS], voff[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int slot = (wave * LOADS + j) * 64 + lane, key = slot / CH, cp = slot % CH;
    koff[j] = (uint32_t)key * row_bytes + (uint32_t)((cp ^ kswz<D>(key)) * 16);
    voff[j] = (uint32_t)key * row_bytes + (uint32_t)((cp ^ vswz<D>(key)) * 16);
  }
#define FA_DMA(RS_, OFF_, DST_, j_) \
  __builtin_amdgcn_raw_ptr_buffer_load_lds(RS_, (lds_void_t*)((DST_) + (wave * LOADS + (j_)) * 64), 16, OFF_, 0, 0, 0)
#define FA_LOAD_SEG(RK_, RV_, KD_, VD_, so_)            \
  _Pragma("unroll") for (int j = 0; j < LOADS; ++j) {   \
    FA_DMA(RK_, koff[j] + (so_), KD_, j);               \
    FA_DMA(RV_, voff[j] + (so_), VD_, j);               \
  }
  // Each (uniform) branch names its buffer resources (a selected resource would be formed
  // in vector registers); all offsets go in the range-checked vector offset (the scalar
  // offset is not range-checked).  Both branches issue the same copies, so the compiler
  // counts the outstanding ones exactly.
#define FA_LOAD(KD_, VD_, t_)                                                         \
  {                                                                                   \
    const int tt_ = __builtin_amdgcn_readfirstlane(t_);  /* uniform: scalar branch */ \
    if (tt_ < P0) {                                                                   \
      FA_LOAD_SEG(rsK0, rsV0, KD_, VD_, (uint32_t)(tt_ * KT) * row_bytes);            \
    } else {                                                                          \
      FA_LOAD_SEG(rsK1, rsV1, KD_, VD_, (uint32_t)((tt_ - P0) * KT) * row_bytes);     \
    }                                                                                 \
  }

  // ---- queries of this lane: column (lane & 31) of each 32-query block ----
  const int fr = lane & 31, fk = lane >> 5;
  V8 qf[QW][KSTEPS];
  int qpos[QW];
#pragma unroll
  for (int qi = 0; qi < QW; ++qi) {
    const int qrow_raw = qb.q_begin + (wave * QW + qi) * 32 + fr;
    const int qrow = min(qrow_raw, qb.q_end - 1);
    qpos[qi] = n0 + (qrow_raw - qrow0);
    const T16* qp = (const T16*)a.q + (int64_t)qrow * a.q_ld + h * D + fk * 8;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) qf[qi][ks] = H::as_v8(*reinterpret_cast<const uint4*>(qp + ks * 16));
  }

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
  // V^T fragment addressing (see header): 16-lane group -> d0, lane p = lane % 16
  const int tr_p = lane & 15;
  const int tr_key = fk * 4 + (tr_p >> 2);                     // + kb*32 + hh*16 (+8 for the second read)
  const int tr_col = ((lane & 16) ? 16 : 0) + 4 * (tr_p & 3);  // + db*32

  // One key tile computed from (Kc, Vc).
  auto compute = [&](const u32x4_t* Kc, const u32x4_t* Vc, int t) __attribute__((always_inline)) {
    // ---- S^T = K Q^T: s[qi][kb][e] = score(key t*KT + kb*32 + 8(e/4) + 4 fk + e%4, query fr) ----
    f32x16_t s[QW][KB];
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int key = kb * 32 + fr;
        const V8 kf = __builtin_bit_cast(V8, Kc[key * CH + ((ks * 2 + fk) ^ kswz<D>(key))]);
#pragma unroll
        for (int qi = 0; qi < QW; ++qi)
          s[qi][kb] = H::mma(kf, qf[qi][ks], ks == 0 ? f32x16_t{} : s[qi][kb]);
      }
    }

    // ---- mask (diagonal tiles only), online softmax per lane = per query ----
    // Scores stay raw until the exponent: p = 2^(s*c2 - m) with m in log2 units.  The
    // running max m is raised only when some lane's tile max exceeds it by more than
    // kLazy (wave-uniform test), so p <= 2^kLazy and the O^T rescale is skipped on most
    // tiles; numerator and denominator share the same m, so the result is unchanged.
    // masked: first-segment keys past n0 (the last first-segment tile only) and causal
    // keys past the query (segment-1 tiles that reach past the block's first query)
    const bool seg0 = t < P0;
    const bool need_mask = seg0 ? (t * KT + KT > n0) : (kpos0(t) + KT - 1 > qpos_first);
#pragma unroll
    for (int qi = 0; qi < QW; ++qi) {
      if (need_mask) {
        const int lim = (seg0 ? n0 - 1 : qpos[qi]) - kpos0(t) - 4 * fk;  // last visible offset - 4 fk
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (kb * 32 + 8 * (e >> 2) + (e & 3) > lim) s[qi][kb][e] = kMaskVal;
      }
      float mx = kMaskVal;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[qi][kb][e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave)) * c2;
      if (__any(mx > m_run[qi] + kLazy)) {
        const float m_new = fmaxf(m_run[qi], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[qi] - m_new);
        m_run[qi] = m_new;
        l_run[qi] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[qi][db][e] *= alpha;
      }
      const float nm = -m_run[qi];
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[qi][kb][e], c2, nm));
          s[qi][kb][e] = p;
          ls += p;
        }
      l_run[qi] += ls;
    }

    // ---- O^T += V^T P^T over the sixteen-key steps (kb, hh) ----
    const T16* vbase = reinterpret_cast<const T16*>(Vc);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        V8 pf[QW];
#pragma unroll
        for (int qi = 0; qi < QW; ++qi) {
          const f32x16_t& sv = s[qi][kb];
          pf[qi] = H::as_v8(make_uint4(H::pack2(sv[hh * 8 + 0], sv[hh * 8 + 1]), H::pack2(sv[hh * 8 + 2], sv[hh * 8 + 3]),
                                       H::pack2(sv[hh * 8 + 4], sv[hh * 8 + 5]), H::pack2(sv[hh * 8 + 6], sv[hh * 8 + 7])));
        }
        const int ka = kb * 32 + hh * 16 + tr_key, kc = ka + 8;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int col = db * 32 + tr_col;
          const int ca = ((col >> 3) ^ vswz<D>(ka)) * 8 + (col & 7);
          const int cc = ((col >> 3) ^ vswz<D>(kc)) * 8 + (col & 7);
          const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(vbase + ka * D + ca));
          const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(vbase + kc * D + cc));
          const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
          const V8 vf = H::as_v8(make_uint4(l2.x, l2.y, h2.x, h2.y));
#pragma unroll
          for (int qi = 0; qi < QW; ++qi) o[qi][db] = H::mma(vf, pf[qi], o[qi][db]);
        }
      }
    }
  };

  // Loads of tile t+1 into (Kn, Vn) are issued first and land while tile t is computed
  // from (Kc, Vc); the closing barrier (which waits for this wave's loads) makes them
  // visible to every wave.  (A third buffer with two tiles in flight and explicit
  // per-tile waits measured slower: 5.47 against 4.96 ms per layer at 2 x 16384 keys.)
  auto tile = [&](const u32x4_t* Kc, const u32x4_t* Vc, u32x4_t* Kn, u32x4_t* Vn, int t) __attribute__((always_inline)) {
    if (t + 1 < t_end) FA_LOAD(Kn, Vn, t + 1);
    compute(Kc, Vc, t);
    __syncthreads();
  };
  FA_LOAD(Ks0, Vs0, t_begin);
  __syncthreads();
  int t = t_begin;
  for (; t + 2 <= t_end; t += 2) {
    tile(Ks0, Vs0, Ks1, Vs1, t);
    tile(Ks1, Vs1, Ks0, Vs0, t + 1);
  }
  if (t < t_end) tile(Ks0, Vs0, Ks1, Vs1, t);
#undef FA_DMA
#undef FA_LOAD_SEG
#undef FA_LOAD

  // ---- normalise and store: o[qi][db][e] = O^T(dh = db*32 + 8(e/4) + 4 fk + e%4, query fr) ----
  if (nsp > 1) {  // split partial: (max in log2 units, sum, unnormalised o)
#pragma unroll
    for (int qi = 0; qi < QW; ++qi) {
      const int qrow = qb.q_begin + (wave * QW + qi) * 32 + fr;
      const float l = l_run[qi] + __shfl_xor(l_run[qi], 32, kWave);
      if (qrow >= qb.q_end) continue;
      float* pp = a.part + ((int64_t)qrow * a.Hq + h) * attn_part_record(gridDim.y, D);
      if (fk == 0) *reinterpret_cast<float2*>(pp + gridDim.y * D + 2 * sp) = make_float2(m_run[qi], l);
      pp += sp * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4)
          *reinterpret_cast<float4*>(pp + db * 32 + 8 * e4 + 4 * fk) =
              make_float4(o[qi][db][4 * e4], o[qi][db][4 * e4 + 1], o[qi][db][4 * e4 + 2], o[qi][db][4 * e4 + 3]);
    }
    return;
  }
#pragma unroll
  for (int qi = 0; qi < QW; ++qi) {
    const int qrow = qb.q_begin + (wave * QW + qi) * 32 + fr;
    const float l = l_run[qi] + __shfl_xor(l_run[qi], 32, kWave);
    if (qrow >= qb.q_end) continue;
    const float inv = 1.0f / l;
    T16* op = (T16*)a.o + (int64_t)qrow * a.Hq * D + h * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int dh = db * 32 + 8 * e4 + 4 * fk;
        uint2 w;
        w.x = H::pack2(o[qi][db][4 * e4] * inv, o[qi][db][4 * e4 + 1] * inv);
        w.y = H::pack2(o[qi][db][4 * e4 + 2] * inv, o[qi][db][4 * e4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + dh) = w;
      }
  }
#endif
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
  const int qrow0 = st.q_cu[b], krow0 = st.k_beg(b);
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

// Merge of split-KV partials: one wave per (query row, q head), lane i holding head
// dimensions i*D/64 ..; rows of sequences that did not split were written by the
// attention kernel.  Partial s of (row, head) is at ((row*Hq + head)*S + s)*(D + 4):
// max (log2 units), sum, two pad floats, unnormalised o[D].
template <typename T16, int D>
__global__ __launch_bounds__(256) void k_attn_split_merge(SeqTable st, const float* __restrict__ part, int S, int Hq,
                                                          int64_t items, T16* __restrict__ o) {
  typedef Half16<T16> H;
  constexpr int PER = D / 64;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= items) return;
  const int lane = threadIdx.x & 63;
  const int nsp = attn_splits(st.pos0(seq_of_row(st, (int)(item / Hq))));
  if (nsp == 1) return;
  const float* p = part + item * attn_part_record(S, D);
  const float* ml = p + S * D;
  float M = -INFINITY;
  for (int sp = 0; sp < nsp; ++sp) M = fmaxf(M, ml[2 * sp]);
  float L = 0.f, acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int sp = 0; sp < nsp; ++sp) {
    const float w = __builtin_amdgcn_exp2f(ml[2 * sp] - M);
    L = fmaf(ml[2 * sp + 1], w, L);
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = fmaf(p[sp * D + lane * PER + e], w, acc[e]);
  }
  const float inv = 1.0f / L;
  T16* op = o + item * D + lane * PER;
  if constexpr (PER == 2)
    *reinterpret_cast<uint32_t*>(op) = H::pack2(acc[0] * inv, acc[1] * inv);
  else
    stf(op, acc[0] * inv);
}

size_t attn_partial_floats(int64_t R, int32_t Hq, int32_t D, int32_t max_splits) {
  return max_splits > 1 ? (size_t)R * Hq * attn_part_record(max_splits, D) : 0;
}

int count_qblocks(const SeqTable& st, int BQ) {
  int n = 0;
  for (int b = 0; b < st.n; ++b) n += (st.q_cu[b + 1] - st.q_cu[b] + BQ - 1) / BQ;
  return n;
}

// Timing-harness hook: forced tile shape (0: 32 queries/wave x 64-key tiles,
// 1: 64 queries/wave x 32-key tiles).
hipError_t launch_attention_variant(hipStream_t s, int variant, const SeqTable& st, const AttnArgs& a) {
  const FaMap m = fa_map(a.Hq, a.Hkv);
  if (variant == 0)
    k_attn_bf16<bf16_t, 128, 1, 64><<<fa_grid(m, count_qblocks(st, 128), a.Hq), 256, 0, s>>>(st, a);
  else
    k_attn_bf16<bf16_t, 128, 2, 32><<<fa_grid(m, count_qblocks(st, 256), a.Hq), 256, 0, s>>>(st, a);
  return hipGetLastError();
}

hipError_t launch_attention(hipStream_t s, rp_dtype dt, const SeqTable& st, const AttnArgs& a, int32_t total_q) {
  if (total_q <= 0) return hipSuccess;
  if (dt != RP_F32) {
    // The 16-bit kernel addresses a sequence's keys with 32-bit byte offsets.
    for (int b = 0; b < st.n; ++b) {
      const int64_t keys = (int64_t)st.pos0(b) + (st.q_cu[b + 1] - st.q_cu[b]);
      if ((keys + 64) * a.Hkv * a.D * 2 > (int64_t)UINT32_MAX) return hipErrorInvalidValue;
    }
    int S = 1;  // split-KV ways of the most split sequence (grid y)
    if (a.part)
      for (int b = 0; b < st.n; ++b) S = std::max(S, attn_splits(st.pos0(b)));
    AttnArgs as = a;
    if (S == 1) as.part = nullptr;
    hipError_t e = hipSuccess;
    with_half16(dt, [&](auto tag_) {
      using H = decltype(tag_);
      // Long sequences: 8 waves (256 queries) share each K/V tile, halving the tile loads
      // per query; shorter ones keep 4 waves, whose smaller blocks balance better (also
      // measured faster for split suffix passes).  Each query sees the same key tiles in
      // the same order either way (same results).
      int max_q = 0;
      for (int b = 0; b < st.n; ++b) max_q = std::max(max_q, st.q_cu[b + 1] - st.q_cu[b]);
      const FaMap fm = fa_map(a.Hq, a.Hkv);
      if (max_q >= 8192) {
        const dim3 grid(fa_grid(fm, count_qblocks(st, 256), a.Hq), S);
        if (a.D == 128)
          k_attn_bf16<H, 128, 1, 64, 8><<<grid, 512, 0, s>>>(st, as);
        else
          k_attn_bf16<H, 64, 1, 64, 8><<<grid, 512, 0, s>>>(st, as);
      } else {
        const dim3 grid(fa_grid(fm, count_qblocks(st, 128), a.Hq), S);
        if (a.D == 128)
          k_attn_bf16<H, 128, 1, 64><<<grid, 256, 0, s>>>(st, as);
        else
          k_attn_bf16<H, 64, 1, 64><<<grid, 256, 0, s>>>(st, as);
      }
      if (S > 1 && (e = hipGetLastError()) == hipSuccess) {
        const int64_t items = (int64_t)total_q * a.Hq;
        const int mgrid = (int)((items + 3) / 4);
        if (a.D == 128)
          k_attn_split_merge<H, 128><<<mgrid, 256, 0, s>>>(st, as.part, S, a.Hq, items, (H*)a.o);
        else
          k_attn_split_merge<H, 64><<<mgrid, 256, 0, s>>>(st, as.part, S, a.Hq, items, (H*)a.o);
      }
    });
    if (e != hipSuccess) return e;
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
//
// A decode step reads every cached key and value once and does ~7 flop per byte for a
// 7-head GQA group, so it is bound by HBM bandwidth.  Each wave owns one 512-key chunk
// of one (sequence, kv head) and streams it with no block barrier: LPK lanes hold one
// key row (8 head dims each, one 16-byte load), KPW keys per pass, and an R-deep ring of
// K/V loads stays in flight (16 KB per wave at 16-bit) while earlier passes are scored.
// All G q heads of the group read the same loaded row.  Each group of LPK lanes keeps an
// online softmax per head (log2 domain, running max raised only when a score exceeds it
// by more than 2^8, so the rescale branch is rarely taken); the groups are merged with
// lane shuffles and the wave writes (max, sum, o[D]) per head for the merge kernel.
// Partial layout (both kernels and the merge): o of (item = b * Hq + q head, chunk c) at
// part[(item * nchunks + c) * D], whole 128-byte lines written by one wave, then the
// (max, sum) pairs at part[B * Hq * nchunks * D + (item * nchunks + c) * 2].
// ------------------------------------------------------------------------------------
constexpr int DC_KEYS = 1024;  // keys per chunk (one wave)
constexpr int DC_MAXG = 8;    // q heads per kv head (validated on the host)

template <typename T, int D>
__global__ __launch_bounds__(256) void k_decode_attn_part(const T* __restrict__ q, int q_ld,
                                                          const T* __restrict__ ck, const T* __restrict__ cv,
                                                          const int32_t* __restrict__ kv_len, int cap,
                                                          int max_pos, int B, int Hq, int Hkv, float scale,
                                                          int nchunks, float* __restrict__ part) {
  constexpr int LPK = D / 8;                  // lanes per key row
  constexpr int KPW = kWave / LPK;            // keys per pass
  constexpr int NPASS = DC_KEYS / KPW;        // passes per chunk
  constexpr int R = sizeof(T) == 4 ? 4 : 8;   // passes in flight
  static_assert(NPASS % R == 0, "ring");
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int c = wid % nchunks, bg = wid / nchunks;
  if (bg >= B * Hkv) return;
  const int g = bg % Hkv, b = bg / Hkv;
  const int G = Hq / Hkv;
  const int n = min(max(kv_len[b], 0), min(cap, max_pos) - 1);  // new token slot; keys 0..n
  const int k_begin = c * DC_KEYS;
  const int nkeys = min(DC_KEYS, n + 1 - k_begin);
  const int64_t rec = (int64_t)(b * Hq + g * G) * nchunks + c;
  float* out = part + rec * D;                                  // o records
  float* oml = part + (int64_t)B * Hq * nchunks * D + rec * 2;  // (max, sum)
  const int64_t head_stride = (int64_t)nchunks * D, ml_stride = (int64_t)nchunks * 2;
  if (nkeys <= 0) {
    if (lane < G) {
      oml[lane * ml_stride] = -INFINITY;
      oml[lane * ml_stride + 1] = 0.f;
    }
    return;
  }
  const int sub = lane % LPK, kk = lane / LPK;
  const float c2 = scale * 1.4426950408889634f;  // scores in log2 units
  float qr[DC_MAXG][8];
#pragma unroll
  for (int h = 0; h < DC_MAXG; ++h) {
    if (h < G) {
      float t[8];
      const T* qp = q + (int64_t)b * q_ld + (g * G + h) * D + sub * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = ldf(qp + e);
#pragma unroll
      for (int e = 0; e < 8; ++e) qr[h][e] = t[e] * c2;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) qr[h][e] = 0.f;
    }
  }
  const int64_t row_ld = (int64_t)Hkv * D;
  const T* kb = ck + ((int64_t)b * cap + k_begin) * row_ld + g * D + sub * 8;
  const T* vb = cv + ((int64_t)b * cap + k_begin) * row_ld + g * D + sub * 8;
  // rows past the chunk's last key re-read that key (in bounds) and are masked
  auto row = [&](int p) -> int64_t { return (int64_t)min(p * KPW + kk, nkeys - 1) * row_ld; };
  typename Raw8<T>::type kr[R], vr[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    kr[r] = ld_raw8(kb + row(r));
    vr[r] = ld_raw8(vb + row(r));
  }
  float m[DC_MAXG], l[DC_MAXG], o[DC_MAXG][8];
#pragma unroll
  for (int h = 0; h < DC_MAXG; ++h) {
    m[h] = -1e30f;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
  }
  const int npass = (nkeys + KPW - 1) / KPW;
  for (int p0 = 0; p0 < npass; p0 += R) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int p = p0 + r;
      if (p < npass) {
        float kv[8];
        unpack8(kr[r], kv);
        if (p + R < NPASS) kr[r] = ld_raw8(kb + row(p + R));
        const bool valid = p * KPW + kk < nkeys;
        float sc[DC_MAXG];
        bool raise = false;
#pragma unroll
        for (int h = 0; h < DC_MAXG; ++h) {
          if (h < G) {
            float a = 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) a = fmaf(qr[h][e], kv[e], a);
            a = LPK == 16 ? row16_sum(a) : oct8_sum(a);
            sc[h] = valid ? a : -1e30f;
            raise |= sc[h] > m[h] + 8.f;
          }
        }
        if (__any(raise)) {
#pragma unroll
          for (int h = 0; h < DC_MAXG; ++h) {
            if (h < G) {
              const float mn = fmaxf(m[h], sc[h]);
              const float al = __builtin_amdgcn_exp2f(m[h] - mn);
              m[h] = mn;
              l[h] *= al;
#pragma unroll
              for (int e = 0; e < 8; ++e) o[h][e] *= al;
            }
          }
        }
        float vv[8];
        unpack8(vr[r], vv);
        if (p + R < NPASS) vr[r] = ld_raw8(vb + row(p + R));
#pragma unroll
        for (int h = 0; h < DC_MAXG; ++h) {
          if (h < G) {
            const float pk = __builtin_amdgcn_exp2f(sc[h] - m[h]);
            l[h] += pk;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[h][e] = fmaf(pk, vv[e], o[h][e]);
          }
        }
      }
    }
  }
  // merge the KPW key groups of the wave, then write (max in natural-log units, sum, o)
#pragma unroll
  for (int h = 0; h < DC_MAXG; ++h) {
    if (h < G) {
      float M = m[h];
#pragma unroll
      for (int off = LPK; off < kWave; off <<= 1) M = fmaxf(M, __shfl_xor(M, off, kWave));
      const float f = __builtin_amdgcn_exp2f(m[h] - M);
      float L = l[h] * f;
#pragma unroll
      for (int off = LPK; off < kWave; off <<= 1) L += __shfl_xor(L, off, kWave);
      float ov[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float a = o[h][e] * f;
#pragma unroll
        for (int off = LPK; off < kWave; off <<= 1) a += __shfl_xor(a, off, kWave);
        ov[e] = a;
      }
      float* oh = out + h * head_stride;
      if (lane == 0) {
        oml[h * ml_stride] = M * 0.6931471805599453f;
        oml[h * ml_stride + 1] = L;
      }
      if (kk == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) oh[sub * 8 + e] = ov[e];
      }
    }
  }
}

// 16-bit models: the same split-KV chunks on the matrix cores.  One wave owns one chunk
// of one (sequence, kv head); the G q heads of the group are the query columns of the
// prefix kernel's tile (S^T = K Q^T with v_mfma_f32_32x32x16, the scores reused as the
// B operand of O^T += V^T P^T, V^T read with ds_read_b64_tr_b16; columns >= G are
// zero and ignored).  32-key K and V tiles stream into a 3-stage per-wave LDS ring by
// direct global->LDS loads through a buffer resource whose extent ends at the
// sequence's last key, so rows past it read as zeros; the wave needs no barrier: the
// compiler waits on the loads that filled a stage before reading it, and a stage is
// refilled only after the MFMAs that consumed it.  A workgroup holds DC_WAVES waves, the
// consecutive chunks of one group; at the end they combine their (max, sum, o) through
// LDS and the group writes one partial record, so the partials written and merged are a
// DC_WAVES-th of one record per chunk.
constexpr int DC_WAVES = 3;
__host__ __device__ inline int decode_groups(int nchunks) { return (nchunks + DC_WAVES - 1) / DC_WAVES; }
template <typename T16, int D>
__global__ __launch_bounds__(64 * DC_WAVES) void k_decode_attn_mfma(const T16* __restrict__ q, int q_ld,
                                                                    const T16* __restrict__ ck, const T16* __restrict__ cv,
                                                                    const int32_t* __restrict__ kv_len, int cap,
                                                                    int max_pos, int B, int Hq, int Hkv, float scale,
                                                                    int nchunks, float* __restrict__ part) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef Half16<T16> H;
  typedef typename H::V8 V8;
  constexpr int KT = 32;                 // keys per tile
  constexpr int NT = DC_KEYS / KT;       // tiles per chunk
  constexpr int CH = D / 8;              // 16-byte chunks per row
  constexpr int KSTEPS = D / 16;
  constexpr int DB = D / 32;
  constexpr int LOADS = (KT * CH) / 64;  // load instructions per matrix per tile
  static_assert(NT % 3 == 0 || NT > 3, "ring");
  constexpr int PSL = KT * CH * 4 / 64;  // floats per lane in one K stage
  static_assert(DB * 16 <= 2 * PSL && PSL >= 2, "merge data fits the wave's K stages");
  __shared__ u32x4_t Ksa[DC_WAVES][KT * CH], Ksb[DC_WAVES][KT * CH], Ksc[DC_WAVES][KT * CH];
  __shared__ u32x4_t Vsa[DC_WAVES][KT * CH], Vsb[DC_WAVES][KT * CH], Vsc[DC_WAVES][KT * CH];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  u32x4_t *Ks0 = Ksa[wave], *Ks1 = Ksb[wave], *Ks2 = Ksc[wave];
  u32x4_t *Vs0 = Vsa[wave], *Vs1 = Vsb[wave], *Vs2 = Vsc[wave];
  // kv head fastest: the Hkv workgroups that read the same cache rows (each its own
  // 2*D-byte slice of a row) are dispatched together, so each row is fetched while open
  const int nrec = decode_groups(nchunks);
  const int g = blockIdx.x % Hkv, bgr = blockIdx.x / Hkv;
  const int grp = bgr % nrec, b = bgr / nrec;
  const int c = grp * DC_WAVES + wave;
  const int G = Hq / Hkv;
  // query columns: lane column fr is q head g*G + fr (zero beyond G); issued first, so they
  // are in flight while kv_len is read and are covered by the wait for the first tile
  const int fr = lane & 31, fk = lane >> 5;
  V8 qf[KSTEPS];
#pragma unroll
  for (int ks = 0; ks < KSTEPS; ++ks) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (fr < G) v = *reinterpret_cast<const uint4*>(q + (int64_t)b * q_ld + (g * G + fr) * D + ks * 16 + fk * 8);
    qf[ks] = H::as_v8(v);
  }
  const int n = min(max(kv_len[b], 0), min(cap, max_pos) - 1);  // keys 0..n
  const int k_begin = c * DC_KEYS;
  const int nkeys = c < nchunks ? min(DC_KEYS, n + 1 - k_begin) : 0;
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] = 0.f;
  float m_run = kMaskVal, l_run = 0.f;
  if (nkeys > 0) {  // (uniform) this wave's chunk holds keys
  const int ntiles = (nkeys + KT - 1) / KT;
  // keys of this chunk as a buffer resource: rows k_begin .. n of (b, g); byte offsets
  // key * row_bytes fit 32 bits (cap * Hkv * D * 2 bytes is checked on the host)
  const uint32_t row_bytes = (uint32_t)Hkv * D * sizeof(T16);
  const uint32_t ext = (uint32_t)(nkeys - 1) * row_bytes + D * sizeof(T16);
  const int64_t e0 = ((int64_t)b * cap + k_begin) * Hkv * D + (int64_t)g * D;
  const __amdgpu_buffer_rsrc_t rsK =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr((void*)(ck + e0)), 0, (int)ext, 0x00020000);
  const __amdgpu_buffer_rsrc_t rsV =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr((void*)(cv + e0)), 0, (int)ext, 0x00020000);
  uint32_t koff[LOADS], voff[LOADS];
#pragma unroll
  for (int j = 0; j < LOADS; ++j) {
    const int slot = j * 64 + lane, key = slot / CH, cp = slot % CH;
    koff[j] = (uint32_t)key * row_bytes + (uint32_t)((cp ^ kswz<D>(key)) * 16);
    voff[j] = (uint32_t)key * row_bytes + (uint32_t)((cp ^ vswz<D>(key)) * 16);
  }
#define DM_LOAD(KD_, VD_, t_)                                                                                \
  _Pragma("unroll") for (int j = 0; j < LOADS; ++j) {                                                       \
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsK, (lds_void_t*)((KD_) + j * 64), 16, koff[j] + (uint32_t)(t_) * KT * row_bytes, 0, 0, 0); \
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsV, (lds_void_t*)((VD_) + j * 64), 16, voff[j] + (uint32_t)(t_) * KT * row_bytes, 0, 0, 0); \
  }
  const float c2 = scale * 1.4426950408889634f;
  const int tr_p = lane & 15;
  const int tr_key = fk * 4 + (tr_p >> 2);
  const int tr_col = ((lane & 16) ? 16 : 0) + 4 * (tr_p & 3);

  auto tile = [&](const u32x4_t* Kc, const u32x4_t* Vc, int t) __attribute__((always_inline)) {
    f32x16_t sc;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const V8 kf = __builtin_bit_cast(V8, Kc[fr * CH + ((ks * 2 + fk) ^ kswz<D>(fr))]);
      sc = H::mma(kf, qf[ks], ks == 0 ? f32x16_t{} : sc);
    }
    // sc[e] = score(key t*KT + 8(e/4) + 4 fk + e%4, head fr)
    const int lim = nkeys - 1 - t * KT - 4 * fk;
    if (t * KT + KT > nkeys) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (8 * (e >> 2) + (e & 3) > lim) sc[e] = kMaskVal;
    }
    float mx = kMaskVal;
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sc[e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave)) * c2;
    if (__any(mx > m_run + kLazy)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[db][e] *= alpha;
    }
    const float nm = -m_run;
    float ls = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float pv = __builtin_amdgcn_exp2f(fmaf(sc[e], c2, nm));
      sc[e] = pv;
      ls += pv;
    }
    l_run += ls;
    const T16* vbase = reinterpret_cast<const T16*>(Vc);
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const V8 pf = H::as_v8(make_uint4(H::pack2(sc[hh * 8 + 0], sc[hh * 8 + 1]), H::pack2(sc[hh * 8 + 2], sc[hh * 8 + 3]),
                                        H::pack2(sc[hh * 8 + 4], sc[hh * 8 + 5]), H::pack2(sc[hh * 8 + 6], sc[hh * 8 + 7])));
      const int ka = hh * 16 + tr_key, kc = ka + 8;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int col = db * 32 + tr_col;
        const int ca = ((col >> 3) ^ vswz<D>(ka)) * 8 + (col & 7);
        const int cc = ((col >> 3) ^ vswz<D>(kc)) * 8 + (col & 7);
        const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(vbase + ka * D + ca));
        const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(vbase + kc * D + cc));
        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
        o[db] = H::mma(H::as_v8(make_uint4(l2.x, l2.y, h2.x, h2.y)), pf, o[db]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Tile t reads stage t % 3; after it, the stage is refilled with tile t + 3 (rows past
  // the chunk's last key read as zeros and are never used).  The prologue and the steady
  // loop issue every load unconditionally (a short chunk re-reads its last tile), so the
  // compiler counts exactly which loads a stage waits for and the later ones stay in
  // flight; only the last few tiles (no loop) take branches.
  // Tile 0 runs before the loop: its wait for stage 0 also covers the query loads issued
  // ahead of the copies, so no register load is pending when the loop starts (a loop
  // whose loads fill only LDS but which reads registers still loading from before it
  // makes the compiler drain every load, these copies included, ahead of the loop).
  DM_LOAD(Ks0, Vs0, 0);
  DM_LOAD(Ks1, Vs1, min(1, ntiles - 1));
  DM_LOAD(Ks2, Vs2, min(2, ntiles - 1));
  tile(Ks0, Vs0, 0);
  DM_LOAD(Ks0, Vs0, min(3, ntiles - 1));
  int t = 1;  // tiles t, t+1, t+2 in (or on their way to) stages 1, 2, 0
  for (; t + 6 <= ntiles; t += 3) {
    tile(Ks1, Vs1, t);
    DM_LOAD(Ks1, Vs1, t + 3);
    tile(Ks2, Vs2, t + 1);
    DM_LOAD(Ks2, Vs2, t + 4);
    tile(Ks0, Vs0, t + 2);
    DM_LOAD(Ks0, Vs0, t + 5);
  }
  const int r = ntiles - t;  // 0 .. 5 tiles left
  if (r > 0) tile(Ks1, Vs1, t);
  if (r > 3) { DM_LOAD(Ks1, Vs1, t + 3); }
  if (r > 1) tile(Ks2, Vs2, t + 1);
  if (r > 4) { DM_LOAD(Ks2, Vs2, t + 4); }
  if (r > 2) tile(Ks0, Vs0, t + 2);
  if (r > 3) tile(Ks1, Vs1, t + 3);
  if (r > 4) tile(Ks2, Vs2, t + 4);
#undef DM_LOAD
  __builtin_amdgcn_s_waitcnt(0);  // this wave's copies have landed: its stages are free
  }
  // ---- combine the group's chunks: waves 1.. leave o in their own first two K stages and
  // (max, sum) in the third (lane-major, conflict-free); wave 0 rescales them to the
  // common max and adds ----
  // o[db][e] = O^T(dim db*32 + 8(e/4) + 4 fk + e%4, head fr), unnormalised; m in log2 units
  if (wave > 0) {
    float* mine0 = reinterpret_cast<float*>(Ks0);
    float* mine1 = reinterpret_cast<float*>(Ks1);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = db * 16 + e;
        (i < PSL ? mine0 : mine1)[(i % PSL) * 64 + lane] = o[db][e];
      }
    reinterpret_cast<float*>(Ks2)[lane] = m_run;
    reinterpret_cast<float*>(Ks2)[64 + lane] = l_run;
  }
  __syncthreads();
  if (wave != 0) return;
  if (nkeys <= 0) {  // the group's first chunk is past the last key: so are the others
    if (lane < G) {
      const int64_t rec = (int64_t)(b * Hq + g * G + lane) * nrec + grp;
      *reinterpret_cast<float2*>(part + (int64_t)B * Hq * nrec * D + rec * 2) = make_float2(-INFINITY, 0.f);
    }
    return;
  }
  float mw[DC_WAVES], M = m_run;
  mw[0] = m_run;
#pragma unroll
  for (int w = 1; w < DC_WAVES; ++w) {
    mw[w] = reinterpret_cast<const float*>(Ksc[w])[lane];
    M = fmaxf(M, mw[w]);
  }
  const float f0 = __builtin_amdgcn_exp2f(m_run - M);
  float lsum = l_run * f0;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] *= f0;
#pragma unroll
  for (int w = 1; w < DC_WAVES; ++w) {
    const float* t0 = reinterpret_cast<const float*>(Ksa[w]);
    const float* t1 = reinterpret_cast<const float*>(Ksb[w]);
    const float fw = __builtin_amdgcn_exp2f(mw[w] - M);  // 0 for an empty chunk (max kMaskVal)
    lsum = fmaf(reinterpret_cast<const float*>(Ksc[w])[64 + lane], fw, lsum);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = db * 16 + e;
        o[db][e] = fmaf((i < PSL ? t0 : t1)[(i % PSL) * 64 + lane], fw, o[db][e]);
      }
  }
  const float l = lsum + __shfl_xor(lsum, 32, kWave);
  if (fr < G) {
    const int64_t rec = (int64_t)(b * Hq + g * G + fr) * nrec + grp;
    float* oh = part + rec * D;
    if (fk == 0)
      *reinterpret_cast<float2*>(part + (int64_t)B * Hq * nrec * D + rec * 2) =
          make_float2(M * 0.6931471805599453f, l);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int dh = db * 32 + 8 * e4 + 4 * fk;
        *reinterpret_cast<float4*>(oh + dh) =
            make_float4(o[db][4 * e4], o[db][4 * e4 + 1], o[db][4 * e4 + 2], o[db][4 * e4 + 3]);
      }
  }
#endif
}

// Merge of the decode chunks: one wave per (sequence, q head).  Lane c holds chunk c's
// (max, sum) (chunks with keys come first; the rest have max -inf and stale o, never
// read), the wave reduces them, and each lane then sums its D/64 head dimensions over the
// chunks with every chunk's weight taken from its lane, all loads independent.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_decode_attn_merge(const float* __restrict__ part, int nchunks, int items,
                                                           T* __restrict__ o) {
  constexpr int PER = D / 64;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (item >= items) return;
  const float* p = part + (int64_t)item * nchunks * D;                                    // o records
  const float* pml = part + (int64_t)items * nchunks * D + (int64_t)item * nchunks * 2;  // (max, sum)
  float M = -INFINITY;
  for (int c = lane; c < nchunks; c += 64) M = fmaxf(M, pml[2 * c]);
  M = wave_max(M);
  float L = 0.f, acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int c0 = 0; c0 < nchunks; c0 += 64) {
    const int c = c0 + lane;
    const float mc = c < nchunks ? pml[2 * c] : -INFINITY;
    const bool has = mc > -INFINITY;
    const float w = has ? expf(mc - M) : 0.f;
    L += has ? w * pml[2 * c + 1] : 0.f;
    const int nv = __popcll(__ballot(has));  // chunks with keys: a prefix of c0 ..
#pragma unroll 4
    for (int j = 0; j < nv; ++j) {
      const float wj = __shfl(w, j, kWave);
      const float* oc = p + (int64_t)(c0 + j) * D + lane * PER;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc[e] = fmaf(wj, oc[e], acc[e]);
    }
  }
  L = wave_sum(L);
  const float inv = 1.0f / L;
#pragma unroll
  for (int e = 0; e < PER; ++e) stf(o + (int64_t)item * D + lane * PER + e, acc[e] * inv);
}

size_t decode_attn_partial_floats(int32_t B, int32_t Hq, int32_t D, int32_t cap) {
  const int nchunks = (cap + DC_KEYS - 1) / DC_KEYS;
  return (size_t)B * Hq * nchunks * (D + 2);
}

hipError_t launch_decode_attention(hipStream_t s, rp_dtype dt, const void* q, int32_t q_ld,
                                   const void* cache_k, const void* cache_v, const int32_t* kv_len,
                                   int32_t cap, int32_t max_pos, int32_t B, int32_t Hq, int32_t Hkv,
                                   int32_t D, float scale, float* partials, void* o) {
  const int nchunks = (cap + DC_KEYS - 1) / DC_KEYS;
  if (dt == RP_F32) {
    const int grid = (B * Hkv * nchunks + 3) / 4;  // one wave per chunk, 4 waves per workgroup
    if (D == 128)
      k_decode_attn_part<float, 128><<<grid, 256, 0, s>>>((const float*)q, q_ld, (const float*)cache_k,
                                                          (const float*)cache_v, kv_len, cap, max_pos, B, Hq, Hkv,
                                                          scale, nchunks, partials);
    else
      k_decode_attn_part<float, 64><<<grid, 256, 0, s>>>((const float*)q, q_ld, (const float*)cache_k,
                                                         (const float*)cache_v, kv_len, cap, max_pos, B, Hq, Hkv,
                                                         scale, nchunks, partials);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (D == 128)
      k_decode_attn_merge<float, 128><<<(B * Hq + 3) / 4, 256, 0, s>>>(partials, nchunks, B * Hq, (float*)o);
    else
      k_decode_attn_merge<float, 64><<<(B * Hq + 3) / 4, 256, 0, s>>>(partials, nchunks, B * Hq, (float*)o);
    return hipGetLastError();
  }
  // the 16-bit kernel addresses a sequence's cache rows with 32-bit byte offsets
  if ((int64_t)cap * Hkv * D * 2 > (int64_t)INT32_MAX) return hipErrorInvalidValue;
  const int nrec = decode_groups(nchunks);
  const int grid = B * Hkv * nrec;  // one workgroup per group of DC_WAVES chunks
  with_half16(dt, [&](auto tag_) {
    using H = decltype(tag_);
    if (D == 128) {
      k_decode_attn_mfma<H, 128><<<grid, 64 * DC_WAVES, 0, s>>>((const H*)q, q_ld, (const H*)cache_k,
                                                               (const H*)cache_v, kv_len, cap, max_pos, B, Hq, Hkv,
                                                               scale, nchunks, partials);
      k_decode_attn_merge<H, 128><<<(B * Hq + 3) / 4, 256, 0, s>>>(partials, nrec, B * Hq, (H*)o);
    } else {
      k_decode_attn_mfma<H, 64><<<grid, 64 * DC_WAVES, 0, s>>>((const H*)q, q_ld, (const H*)cache_k,
                                                              (const H*)cache_v, kv_len, cap, max_pos, B, Hq, Hkv,
                                                              scale, nchunks, partials);
      k_decode_attn_merge<H, 64><<<(B * Hq + 3) / 4, 256, 0, s>>>(partials, nrec, B * Hq, (H*)o);
    }
  });
  return hipGetLastError();
}

}  // namespace rp
