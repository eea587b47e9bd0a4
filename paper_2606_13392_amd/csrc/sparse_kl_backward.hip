// Sparse KL loss of the Index Branch on gfx950: gradients and loss terms.
//
// Sec. 3.2 ("KL Loss"): for query row i and group r, over the causally
// visible tokens T of the selected blocks, the student is
// P_idx = softmax(s_idx q_idx . k_idx_j) and the teacher is the mean over the
// group's G heads of the Main Branch softmax distributions,
// P = (1/G) sum_h softmax(s q_h . k_j).  The teacher is detached and, by the
// gradient detach of Sec. 3.2, no gradient reaches Q or K; with
// Delta_j = P_idx_j - P_j (the derivative of the KL with respect to the
// student's logit j):
//   d q_idx_i = s_idx sum_j Delta_j k_idx_j,
//   d k_idx_j = s_idx sum_{i, r} Delta_ij q_idx_ir,
//   KL_ir     = sum_j P_j (ln P_j - ln P_idx_j).
// The teacher's per-head normalisers are the forward's LSE (Sec. 4.3, "LSE
// fusion"); the student's LSE_idx is reduced over the selected blocks from
// per-block log-sum-exps (Sec. 4.3) computed in a first key-block-outer
// sweep.  Both sweeps use the reverse index of kvo_index.h, per chunk of
// query rows:
//   kl_lse           per incidence: ln sum_j exp(s_idx S_idx_j) over the block's visible keys
//   kl_lse_combine   per (row, group): LSE_idx over the valid slots
//   kl_grad          per work item (<= 256 queries of one tile): P, P_idx and
//                    Delta on MFMA 16x16x32 per gathered (query, head) row,
//                    the teacher's head mean in registers; d k_idx of the
//                    block in registers (an fp32 partial per item), d q_idx
//                    and the KL term of every incidence as fp32 partials
//                    (kl_grad_wave: one wave per 32-row pass against all 64
//                    keys, no barrier between passes)
//   kl_tile_reduce   per key block: the items of every group's tile, in
//                    order, added to the fp32 d k_idx accumulator
//   kl_combine       per (row, group): d q_idx and KL over the valid slots, in
//                    slot order
// and at the end kl_convert (accumulator times grad_scale to bf16).  No
// atomics touch a result except the reverse index's handle order, which
// fixes the order in which a block's queries add into d k_idx.
#include "kvo_index.h"

namespace {

constexpr int kKlBK = 64;
constexpr int kKlThreads = 256;                       // 4 waves: key quarters
constexpr int kKlRows = 32;                           // gathered (query, head) rows per pass


__device__ __forceinline__ uint16_t raw_elem16(const u32x4& w, int j) {
  return static_cast<uint16_t>(w[j >> 1] >> (16 * (j & 1)));
}

// Stage the index-key block (row-major and transposed) of keys key0 .. key0+63.
template <int D, typename Smem>
__device__ __forceinline__ void stage_index_keys(Smem& sm, const uint16_t* __restrict__ ikb, int nkeys) {
  for (int c = threadIdx.x; c < (kKlBK / 4) * (D / 8); c += kKlThreads) {
    const int key4 = c / (D / 8), dg = c % (D / 8);
    u32x4 rows[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key = 4 * key4 + j;
      rows[j] = key < nkeys ? load_raw(ikb + static_cast<int64_t>(key) * D + 8 * dg) : u32x4{};
      *reinterpret_cast<u32x4*>(&sm.ki[key][8 * dg]) = rows[j];
    }
    if constexpr (sizeof(sm.kit) > 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        uint2 w;
        w.x = static_cast<uint32_t>(raw_elem16(rows[0], e)) | (static_cast<uint32_t>(raw_elem16(rows[1], e)) << 16);
        w.y = static_cast<uint32_t>(raw_elem16(rows[2], e)) | (static_cast<uint32_t>(raw_elem16(rows[3], e)) << 16);
        *reinterpret_cast<uint2*>(&sm.kit[8 * dg + e][4 * key4]) = w;
      }
    }
  }
}

// ---------------------------------------------------------------- LSE_idx
template <int D>
struct KlLseSmem {
  uint16_t ki[kKlBK][D + 8];
  int32_t s_row[kItemQueries];
  int32_t s_slot[kItemQueries];
};

// Per work item: each wave takes 16 queries at a time; S_idx (16 queries x 64
// keys) on MFMA 16x16x32, masked to the visible keys, reduced to the block's
// log-sum-exp per query.
template <int D>
__global__ __launch_bounds__(kKlThreads) void kl_lse_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, msa_seqs sq,
    const int64_t* __restrict__ blk_base, const int32_t* __restrict__ tile_off, const int32_t* __restrict__ item_off,
    const uint32_t* __restrict__ handles, int H_kv, int topk, int64_t nbcap, int64_t row0, float sidx_log2,
    float* __restrict__ lse_part, int32_t* __restrict__ next_item) {
  static_assert(kItemQueries <= kKlThreads, "every thread loads at most one handle of an item");
  __shared__ KlLseSmem<D> sm;
  __shared__ int32_t s_claim;
  constexpr int KS = D / 32;
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int c16 = lane & 15, qd = lane >> 4;
  const int64_t ntile = static_cast<int64_t>(H_kv) * nbcap;
  const int32_t total_items = item_off[ntile];
  int64_t staged = -1;
  for (int32_t item = blockIdx.x; item < total_items; item = claim_next_item(next_item, &s_claim)) {
    const int64_t tile = upper_index(item_off, ntile + 1, item);
    const int32_t h0 = tile_off[tile] + (item - item_off[tile]) * kItemQueries;
    const int32_t nq = min(tile_off[tile + 1] - h0, kItemQueries);
    const int r = static_cast<int>(tile / nbcap);
    const int64_t gb = tile % nbcap;
    const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
    const SeqGeom g = seq_geom(sq, s);
    const int key0 = static_cast<int>(gb - blk_base[s]) * kKlBK;
    const int pos_base = g.kv_len - g.q_rows + static_cast<int>(row0 - g.q_begin);
    __syncthreads();
    if (static_cast<int>(threadIdx.x) < nq) {
      const uint32_t hd = handles[h0 + threadIdx.x];
      sm.s_row[threadIdx.x] = static_cast<int32_t>(hd >> 6);
      sm.s_slot[threadIdx.x] = static_cast<int32_t>(hd & 63u);
    }
    if (tile != staged) {
      const uint16_t* ikb = index_k + (g.kv_start + key0) * static_cast<int64_t>(D);
      for (int c = threadIdx.x; c < kKlBK * (D / 8); c += kKlThreads) {
        const int key = c / (D / 8), dg = c % (D / 8);
        *reinterpret_cast<u32x4*>(&sm.ki[key][8 * dg]) =
            key0 + key < g.kv_len ? load_raw(ikb + static_cast<int64_t>(key) * D + 8 * dg) : u32x4{};
      }
      staged = tile;
    }
    __syncthreads();
    for (int c = 16 * wave; c < nq; c += 64) {
      const int qa = min(c + c16, nq - 1);            // A-operand query of this lane (clamped)
      const int64_t grow = row0 + sm.s_row[qa];
      u32x4 a[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) a[ks] = load_raw(index_q + (grow * H_kv + r) * D + 32 * ks + 8 * qd);
      f32x4 acc[4];
#pragma unroll
      for (int kt = 0; kt < 4; ++kt) {
        acc[kt] = f32x4{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          acc[kt] = mfma16x16x32(__builtin_bit_cast(bf16x8, a[ks]), ld_bf16x8(&sm.ki[16 * kt + c16][32 * ks + 8 * qd]),
                                 acc[kt]);
      }
      // lane (key 16kt + c16, queries c + 4qd + i)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int qi = c + 4 * qd + i;
        const int pos = qi < nq ? pos_base + sm.s_row[qi] : -1;
        float m = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) {
          const float z = key0 + 16 * kt + c16 <= pos ? acc[kt][i] * sidx_log2 : -INFINITY;
          acc[kt][i] = z;
          m = fmaxf(m, z);
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
        const float mm = m == -INFINITY ? 0.f : m;
        float l = 0.f;
#pragma unroll
        for (int kt = 0; kt < 4; ++kt) l += exp2f(acc[kt][i] - mm);
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) l += __shfl_xor(l, off);
        if (c16 == 0 && qi < nq) {
          const int64_t inc = (static_cast<int64_t>(sm.s_row[qi]) * H_kv + r) * topk + sm.s_slot[qi];
          lse_part[inc] = l > 0.f ? (mm + __log2f(l)) * kLn2 : -INFINITY;
        }
      }
    }
  }
}

// One thread per (row, group) of the chunk: LSE_idx = ln sum over the valid
// slots of exp(partial).
__global__ __launch_bounds__(256) void kl_lse_combine_kernel(const int32_t* __restrict__ block_ids, msa_seqs sq,
                                                             const int64_t* __restrict__ blk_base, int H_kv, int topk,
                                                             int64_t row0, int64_t nrows,
                                                             const float* __restrict__ lse_part,
                                                             float* __restrict__ lse_idx) {
  const int64_t pr = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (pr >= nrows * H_kv) return;
  const int64_t row = row0 + pr / H_kv;
  const int r = static_cast<int>(pr % H_kv);
  int s;
  const int p = row_position(sq, row, &s);
  const int32_t* ids = block_ids + (row * H_kv + r) * topk;
  const float* lp = lse_part + pr * topk;
  float m = -INFINITY;
  for (int j = 0; j < topk; ++j)
    if (incidence_ok(ids[j], p, kKlBK, blk_base, s)) m = fmaxf(m, lp[j]);
  float l = 0.f;
  if (m > -INFINITY)
    for (int j = 0; j < topk; ++j)
      if (incidence_ok(ids[j], p, kKlBK, blk_base, s)) l += __expf(lp[j] - m);
  lse_idx[pr] = m > -INFINITY ? m + __logf(l) : -INFINITY;
}

// ---------------------------------------------------------------- gradients
// Mean over the G = 2^lg heads of a query of per-row values laid out as the
// C rows 16t + 4qd + i of MFMA 16x16x32 (lane = c16 + 16 qd): a query's rows
// are consecutive, so they sit in one lane (G <= 4), in lanes qd, qd ^ 1
// (G = 8) or in all four qd (G = 16) of one row tile.
__device__ __forceinline__ void head_mean(f32x4 (&v)[2], int lg) {
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    if (lg == 1) {
      const float a = v[t][0] + v[t][1], b = v[t][2] + v[t][3];
      v[t][0] = v[t][1] = 0.5f * a;
      v[t][2] = v[t][3] = 0.5f * b;
    } else if (lg >= 2) {
      float a = (v[t][0] + v[t][1]) + (v[t][2] + v[t][3]);
      if (lg >= 3) a += __shfl_xor(a, 16);
      if (lg >= 4) a += __shfl_xor(a, 32);
      a *= 1.f / static_cast<float>(1 << lg);
      v[t][0] = v[t][1] = v[t][2] = v[t][3] = a;
    }
  }
}

// ---------------------------------------------------------------- gradients, one wave per pass
// A wave takes whole passes (32 rows against all 64 keys of the block), so
// passes need no CTA barrier and each wave is its own stream of gathers; the
// block's K, index keys and their transpose are shared by the CTA per item.
// d k_idx of all 64 keys stays in the wave's registers (64 VGPRs at d_idx
// 64, 128 at d_idx 128); at item end the four waves' partials are added in
// wave order.
template <int D>
struct KlwWave {
  uint16_t qit[D][kKlRows + 8];                       // index query of each pass row, transposed
  uint16_t dlc[kKlRows][kKlBK + 8];                   // Delta of each pass query (its head-0 row), [query][key]
  float lse2[kKlRows];                                // Main Branch LSE * log2(e) per row (+inf: no row)
  float lsei2[kKlRows];                               // LSE_idx * log2(e) per row
  int32_t rpos[kKlRows];                              // position per row (-1: no row)
  int64_t incq[kKlRows];                              // incidence of pass query j (the trash one past the item)
};
template <int D>
struct KlwSmem {
  union {
    struct {
      uint16_t k[kKlBK][kHeadDim + 8];                // K block (Main Branch head r), row-major
      uint16_t ki[kKlBK][D + 8];                      // index-key block, row-major
      uint16_t kit[D][kKlBK + 8];                     // index-key block transposed
      KlwWave<D> wv[kKlThreads / kWave];
    } m;
    float red[kKlThreads / kWave][kKlBK * D];         // item end: each wave's d k_idx partial
  } u;
  int32_t s_row[kItemQueries];
  int32_t s_slot[kItemQueries];
};
// d_idx 64: two CTAs per CU (245 VGPRs at G = 8); d_idx 128: d k_idx alone
// takes 128 VGPRs, so one CTA per CU with up to 512 registers per wave
static_assert(sizeof(KlwSmem<64>) <= 80 * 1024, "LDS of a one-wave-per-pass KL CTA (two per CU)");
static_assert(sizeof(KlwSmem<128>) <= 160 * 1024, "LDS of a one-wave-per-pass KL CTA (one per CU)");

template <int D, int LG>
__global__ __launch_bounds__(kKlThreads, D == 64 ? 2 : 1) void kl_grad_wave_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k, const float* __restrict__ lse, const float* __restrict__ lse_idx, msa_seqs sq,
    const int64_t* __restrict__ blk_base, const int32_t* __restrict__ tile_off, const int32_t* __restrict__ item_off,
    const uint32_t* __restrict__ handles, int H_q, int H_kv, int topk, int64_t nbcap, int64_t row0,
    float s_main_log2, float sidx, int64_t trash_inc, float* __restrict__ dqp, float* __restrict__ klp,
    float* __restrict__ part, int32_t* __restrict__ next_item) {
  static_assert(kItemQueries <= kKlThreads, "every thread loads at most one handle of an item");
  __shared__ KlwSmem<D> sm;
  __shared__ int32_t s_claim;
  constexpr int KSM = kHeadDim / 32;                  // k-steps of S over the head dimension
  constexpr int KSI = D / 32;                         // k-steps of S_idx over d_idx
  constexpr int NT = D / 16;                          // dim tiles of d k_idx / d q_idx
  constexpr int NW = kKlThreads / kWave;
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int c16 = lane & 15, qd = lane >> 4;
  constexpr int G = 1 << LG;                          // H_q / H_kv
  constexpr int lg = LG;
  constexpr int qpw = 32 >> LG;                       // queries per pass
  const float sidx_log2 = sidx * kLog2e;
  const int64_t ntile = static_cast<int64_t>(H_kv) * nbcap;
  const int32_t total_items = item_off[ntile];
  const int64_t kv_stride = static_cast<int64_t>(H_kv) * kHeadDim;
  KlwWave<D>& wv = sm.u.m.wv[w];

  for (int32_t item = blockIdx.x; item < total_items; item = claim_next_item(next_item, &s_claim)) {
    const int64_t tile = upper_index(item_off, ntile + 1, item);
    const int32_t h0 = tile_off[tile] + (item - item_off[tile]) * kItemQueries;
    const int32_t nq = min(tile_off[tile + 1] - h0, kItemQueries);
    const int r = static_cast<int>(tile / nbcap);
    const int64_t gb = tile % nbcap;
    const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
    const SeqGeom g = seq_geom(sq, s);
    const int key0 = static_cast<int>(gb - blk_base[s]) * kKlBK;
    const int pos_base = g.kv_len - g.q_rows + static_cast<int>(row0 - g.q_begin);

    __syncthreads();                                  // the previous item is done with LDS
    if (static_cast<int>(threadIdx.x) < nq) {
      const uint32_t hd = handles[h0 + threadIdx.x];
      sm.s_row[threadIdx.x] = static_cast<int32_t>(hd >> 6);
      sm.s_slot[threadIdx.x] = static_cast<int32_t>(hd & 63u);
    }
    {                                                 // staged every item: the item-end sum reuses this LDS
      const uint16_t* kb = k + (g.kv_start + key0) * kv_stride + static_cast<int64_t>(r) * kHeadDim;
      for (int c = threadIdx.x; c < kKlBK * (kHeadDim / 8); c += kKlThreads) {
        const int key = c / (kHeadDim / 8), dg = c % (kHeadDim / 8);
        *reinterpret_cast<u32x4*>(&sm.u.m.k[key][8 * dg]) =
            key0 + key < g.kv_len ? load_raw(kb + static_cast<int64_t>(key) * kv_stride + 8 * dg) : u32x4{};
      }
      stage_index_keys<D>(sm.u.m, index_k + (g.kv_start + key0) * static_cast<int64_t>(D), g.kv_len - key0);
    }
    __syncthreads();

    f32x4 acc_dk[4][NT];                              // [key tile][dim tile]: lane column = dim, rows = keys 4qd + i
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int n = 0; n < NT; ++n) acc_dk[kt][n] = f32x4{};

    // A operands of a pass (rows 16t + c16): Q of the row's head, the index
    // query of the row's query, and the two LSEs; the next pass's are
    // requested once S and S_idx have consumed the current ones
    u32x4 bq[2][KSM], bi[2][KSI];
    float lse_v[2], lsei_v[2];
    bool arow[2];
    int32_t qrow[2];
    auto load_pass = [&](int cc) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int qa = cc + ((16 * t + c16) >> lg);
        arow[t] = qa < nq;
        qrow[t] = min(qa, nq - 1);
        const int64_t rl = sm.s_row[qrow[t]];
        const int64_t grow = row0 + rl;
        const int64_t hrow = grow * H_q + static_cast<int64_t>(r) * G + ((16 * t + c16) & (G - 1));
#pragma unroll
        for (int st = 0; st < KSM; ++st) bq[t][st] = load_raw(q + hrow * kHeadDim + 32 * st + 8 * qd);
#pragma unroll
        for (int st = 0; st < KSI; ++st) bi[t][st] = load_raw(index_q + (grow * H_kv + r) * D + 32 * st + 8 * qd);
        lse_v[t] = lse[hrow];
        lsei_v[t] = lse_idx[rl * H_kv + r];
      }
    };
    const int npass = (nq + qpw - 1) / qpw;
    int ps = w;
    if (ps < npass) load_pass(ps * qpw);
    for (; ps < npass; ps += NW) {
      const int cq = ps * qpw;                        // the pass's first query in the item
      // row scalars and the transposed index queries of the pass (wave-private)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int col = 16 * t + c16;
#pragma unroll
        for (int st = 0; st < KSI; ++st)
#pragma unroll
          for (int j = 0; j < 8; ++j) wv.qit[32 * st + 8 * qd + j][col] = raw_elem16(bi[t][st], j);
        if (qd == 0) {
          const int32_t rl = sm.s_row[qrow[t]];
          wv.lse2[col] = arow[t] ? lse_v[t] * kLog2e : INFINITY;
          wv.lsei2[col] = arow[t] ? lsei_v[t] * kLog2e : INFINITY;
          wv.rpos[col] = arow[t] ? pos_base + rl : -1;
          if ((col & (G - 1)) == 0)
            wv.incq[col >> lg] = arow[t] ? (static_cast<int64_t>(rl) * H_kv + r) * topk + sm.s_slot[qrow[t]]
                                         : trash_inc;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

      // two halves of 32 keys keep the score registers small; key tile kt,
      // row tile t: the lane holds key 16kt + c16 and rows 16t + 4qd + i
      float klrow[2][4];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) klrow[t][i] = 0.f;
#pragma unroll
      for (int hk = 0; hk < 2; ++hk) {
        // S and S_idx
        f32x4 acc_s[2][2], acc_i[2][2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int kt = 2 * hk + u;
            acc_s[u][t] = f32x4{};
            acc_i[u][t] = f32x4{};
#pragma unroll
            for (int st = 0; st < KSM; ++st)
              acc_s[u][t] = mfma16x16x32(__builtin_bit_cast(bf16x8, bq[t][st]),
                                         ld_bf16x8(&sm.u.m.k[16 * kt + c16][32 * st + 8 * qd]), acc_s[u][t]);
#pragma unroll
            for (int st = 0; st < KSI; ++st)
              acc_i[u][t] = mfma16x16x32(__builtin_bit_cast(bf16x8, bi[t][st]),
                                         ld_bf16x8(&sm.u.m.ki[16 * kt + c16][32 * st + 8 * qd]), acc_i[u][t]);
            __builtin_amdgcn_sched_barrier(0);      // bound how far LDS operand reads are hoisted
          }
        __builtin_amdgcn_sched_barrier(0);
        if (hk == 1 && ps + NW < npass) load_pass((ps + NW) * qpw);

#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int kt = 2 * hk + u;
          const int key = key0 + 16 * kt + c16;
          // teacher: per-head P, then the mean over the query's heads (in place)
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int row = 16 * t + 4 * qd + i;
              acc_s[u][t][i] = key <= wv.rpos[row] ? exp2_hw(acc_s[u][t][i] * s_main_log2 - wv.lse2[row]) : 0.f;
            }
          head_mean(acc_s[u], lg);
          // student, Delta = P_idx - P on head-0 rows (in place of S_idx), KL terms
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int row = 16 * t + 4 * qd + i;
              const bool on = key <= wv.rpos[row];
              const bool head0 = (row & (G - 1)) == 0;
              const float lz = acc_i[u][t][i] * sidx_log2 - wv.lsei2[row];   // log2 P_idx
              const float pidx = on ? exp2_hw(lz) : 0.f;
              const float pbar = acc_s[u][t][i];
              klrow[t][i] += (head0 && on && pbar > 0.f) ? pbar * (__log2f(pbar) - lz) * kLn2 : 0.f;
              acc_i[u][t][i] = head0 ? pidx - pbar : 0.f;
            }
          // d k_idx += Delta^T q_idx over the pass's rows (one k-step): k
          // index 8qd + 4t + i = row 16t + 4qd + i
          uint4 dw;
          dw.x = pack_bf16x2(acc_i[u][0][0], acc_i[u][0][1]);
          dw.y = pack_bf16x2(acc_i[u][0][2], acc_i[u][0][3]);
          dw.z = pack_bf16x2(acc_i[u][1][0], acc_i[u][1][1]);
          dw.w = pack_bf16x2(acc_i[u][1][2], acc_i[u][1][3]);
          const bf16x8 da = __builtin_bit_cast(bf16x8, dw);
#pragma unroll
          for (int n = 0; n < NT; ++n) {
            const uint16_t* qr = &wv.qit[16 * n + c16][4 * qd];
            const uint2 lo = *reinterpret_cast<const uint2*>(qr), hi = *reinterpret_cast<const uint2*>(qr + 16);
            acc_dk[kt][n] = mfma16x16x32(da, __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y)),
                                         acc_dk[kt][n]);
            if (n & 1) __builtin_amdgcn_sched_barrier(0);
          }
          // the pass queries' Delta rows for d q_idx
#pragma unroll
          for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int row = 16 * t + 4 * qd + i;
              const uint32_t pr = t == 0 ? (i < 2 ? dw.x : dw.y) : (i < 2 ? dw.z : dw.w);
              if ((row & (G - 1)) == 0) wv.dlc[row >> lg][16 * kt + c16] = static_cast<uint16_t>(pr >> (16 * (i & 1)));
            }
        }
      }
      // KL per head-0 row: sum over the 64 keys (registers, then the 16 lanes)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = klrow[t][i];
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off);
          const int row = 16 * t + 4 * qd + i;
          if (c16 == 0 && (row & (G - 1)) == 0) klp[wv.incq[row >> lg]] = v;
        }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

      // d q_idx of the pass queries (rows j = 16tq + 4qd + i of Delta), dims
      // 16n + c16, over the 64 keys
#pragma unroll
      for (int tq = 0; tq < 2; ++tq) {
        if (16 * tq >= qpw) break;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
          f32x4 acc = f32x4{};
#pragma unroll
          for (int ks = 0; ks < kKlBK / 32; ++ks)
            acc = mfma16x16x32(ld_bf16x8(&wv.dlc[16 * tq + c16][32 * ks + 8 * qd]),
                               ld_bf16x8(&sm.u.m.kit[16 * n + c16][32 * ks + 8 * qd]), acc);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int j = 16 * tq + 4 * qd + i;
            if (j < qpw) dqp[wv.incq[j] * D + 16 * n + c16] = acc[i];
          }
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    // item end: the four waves' d k_idx, added in wave order, as the item's
    // partial, laid out [key quarter][reg][lane] as kl_tile_reduce_kernel reads it
    __syncthreads();                                  // every pass is done: K and pass LDS are free
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int n = 0; n < NT; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) sm.u.red[w][kt * (NT * 4 * 64) + (4 * n + i) * 64 + lane] = acc_dk[kt][n][i];
    __syncthreads();
    float* dst = part + static_cast<int64_t>(item) * (kKlBK * D);
    for (int idx = threadIdx.x; idx < kKlBK * D; idx += kKlThreads)
      dst[idx] = (sm.u.red[0][idx] + sm.u.red[1][idx]) + (sm.u.red[2][idx] + sm.u.red[3][idx]);
  }
}

// Per key block: the items of the block's tiles of every group, in group and
// item order, added to the fp32 accumulator of the block's keys.
// kKlReduceSplit CTAs per block, one float4 of the partial per thread.
template <int D>
constexpr int kKlReduceSplit = kKlBK * D / (4 * 256);
template <int D>
__global__ __launch_bounds__(256) void kl_tile_reduce_kernel(msa_seqs sq, const int64_t* __restrict__ blk_base,
                                                             const int32_t* __restrict__ item_off, int H_kv,
                                                             int64_t nbcap, const float* __restrict__ part,
                                                             float* __restrict__ dk_acc) {
  constexpr int NT = D / 16;
  constexpr int SPLIT = kKlReduceSplit<D>;
  const int64_t gb = blockIdx.x / SPLIT;
  const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
  const SeqGeom g = seq_geom(sq, s);
  const int key0 = static_cast<int>(gb - blk_base[s]) * kKlBK;
  bool any = false;
  for (int r = 0; r < H_kv; ++r) any |= item_off[r * nbcap + gb] != item_off[r * nbcap + gb + 1];
  if (!any) return;
  const int c4 = (blockIdx.x % SPLIT) * 256 + threadIdx.x;   // float4 of the partial
  const float4* p4 = reinterpret_cast<const float4*>(part) + c4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int r = 0; r < H_kv; ++r) {
    const int64_t tile = r * nbcap + gb;
#pragma unroll 4
    for (int32_t it = item_off[tile]; it < item_off[tile + 1]; ++it) {
      const float4 x = p4[static_cast<int64_t>(it) * (kKlBK * D / 4)];
      acc.x += x.x;
      acc.y += x.y;
      acc.z += x.z;
      acc.w += x.w;
    }
  }
  // partial layout [kq][reg][lane]: 4 consecutive lanes = 4 consecutive dims
  const int idx = 4 * c4;
  const int kq = idx / (NT * 4 * 64);
  const int reg = (idx / 64) % (NT * 4);
  const int ln = idx & 63;
  const int key = 16 * kq + 4 * (ln >> 4) + (reg & 3);
  const int dim = 16 * (reg >> 2) + (ln & 15);
  if (key0 + key >= g.kv_len) return;
  float4* dst = reinterpret_cast<float4*>(dk_acc + (g.kv_start + key0 + key) * static_cast<int64_t>(D) + dim);
  float4 y = *dst;
  y.x += acc.x;
  y.y += acc.y;
  y.z += acc.z;
  y.w += acc.w;
  *dst = y;
}

// One wave per (row, group) of the chunk: d q_idx = grad_scale x sum of the
// valid slots' partials and KL = sum of their terms, in slot order.
constexpr int kKlCombWaves = 4;

template <int D>
__global__ __launch_bounds__(64 * kKlCombWaves) void kl_combine_kernel(
    const int32_t* __restrict__ block_ids, msa_seqs sq, const int64_t* __restrict__ blk_base, int H_kv, int topk,
    int64_t row0, int64_t nrows, const float* __restrict__ dqp, const float* __restrict__ klp, float grad_scale,
    uint16_t* __restrict__ d_index_q, float* __restrict__ kl) {
  const int lane = lane_id();
  const int64_t pr = static_cast<int64_t>(blockIdx.x) * kKlCombWaves + threadIdx.x / kWave;
  if (pr >= nrows * H_kv) return;
  const int64_t row = row0 + pr / H_kv;
  const int r = static_cast<int>(pr % H_kv);
  int s;
  const int p = row_position(sq, row, &s);
  const int32_t* ids = block_ids + (row * H_kv + r) * topk;
  constexpr int PER = D / 64;                         // dims per lane
  // slot validity, one slot per lane; every slot has a partial row, so the
  // loads below are unconditional and in flight together (unwritten partials
  // of invalid slots are dropped by a select, never multiplied)
  const bool mine = lane < topk && incidence_ok(ids[lane], p, kKlBK, blk_base, s);
  const uint64_t valid = __ballot(mine);
  const float* src = dqp + pr * topk * static_cast<int64_t>(D) + PER * lane;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
#pragma unroll 8
  for (int j = 0; j < topk; ++j) {
    const bool ok = (valid >> j) & 1ull;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const float x = src[static_cast<int64_t>(j) * D + e];
      acc[e] += ok ? x : 0.f;
    }
  }
  float klsum = mine ? klp[pr * topk + lane] : 0.f;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) klsum += __shfl_xor(klsum, off);
  uint16_t* dst = d_index_q + (row * H_kv + r) * static_cast<int64_t>(D) + PER * lane;
  if constexpr (PER == 1) {
    dst[0] = f32_to_bf16_bits(acc[0] * grad_scale);
  } else {
    *reinterpret_cast<uint32_t*>(dst) = pack_bf16x2(acc[0] * grad_scale, acc[1] * grad_scale);
  }
  if (kl && lane == 0) kl[row * H_kv + r] = klsum;
}

__global__ __launch_bounds__(256) void kl_convert_kernel(const float* __restrict__ acc, int64_t n2, float scale,
                                                         uint16_t* __restrict__ out) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n2;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    reinterpret_cast<uint32_t*>(out)[i] = pack_bf16x2(acc[2 * i] * scale, acc[2 * i + 1] * scale);
}

// ---------------------------------------------------------------- host plan
struct KlPlan {
  int64_t nbcap, ntile, chunk_rows, max_items;
  int nscan;
  size_t off_blk_base, off_cnt, off_tile_off, off_item_off, off_blk_tot, off_dk, off_handles, off_tpos, off_lsep,
      off_lsei, off_dqp, off_klp, off_part, total;
};

constexpr size_t kDefaultKlBytes = size_t(16) << 30;

void kl_layout(KlPlan& pl, const msa_seqs* seqs, int H_kv, int D, int topk) {
  using msa_host::align_up;
  size_t o = 0;
  pl.off_blk_base = o; o = align_up(o + sizeof(int64_t) * (seqs->num_seqs + 1), 256);
  pl.off_cnt = o;      o = align_up(o + sizeof(int32_t) * (pl.ntile + kWorkCounters), 256);
  pl.off_tile_off = o; o = align_up(o + sizeof(int32_t) * (pl.ntile + 1), 256);
  pl.off_item_off = o; o = align_up(o + sizeof(int32_t) * (pl.ntile + 1), 256);
  pl.off_blk_tot = o;  o = align_up(o + sizeof(int32_t) * 2 * pl.nscan, 256);
  pl.off_dk = o;       o = align_up(o + sizeof(float) * static_cast<size_t>(seqs->total_kv_rows) * D, 256);
  const size_t inc = static_cast<size_t>(pl.chunk_rows) * H_kv * topk;
  pl.max_items = pl.ntile + static_cast<int64_t>((inc + kItemQueries - 1) / kItemQueries);
  pl.off_handles = o;  o = align_up(o + sizeof(uint32_t) * inc, 256);
  pl.off_tpos = o;     o = align_up(o + sizeof(int32_t) * inc, 256);
  pl.off_lsep = o;     o = align_up(o + sizeof(float) * inc, 256);
  pl.off_lsei = o;     o = align_up(o + sizeof(float) * static_cast<size_t>(pl.chunk_rows) * H_kv, 256);
  pl.off_dqp = o;      o = align_up(o + sizeof(float) * (inc + 1) * D, 256);    // + trash slot
  pl.off_klp = o;      o = align_up(o + sizeof(float) * (inc + 1), 256);
  pl.off_part = o;     o = align_up(o + sizeof(float) * static_cast<size_t>(pl.max_items) * kKlBK * D, 256);
  pl.total = o;
}

int make_kl_plan(const msa_seqs* seqs, int H_kv, int D, int topk, size_t budget, KlPlan* pl) {
  const int64_t nb = (seqs->max_kv_len + kKlBK - 1) / kKlBK;
  pl->nbcap = static_cast<int64_t>(seqs->num_seqs) * (nb > 0 ? nb : 1);
  pl->ntile = static_cast<int64_t>(H_kv) * pl->nbcap;
  if (pl->ntile >= (int64_t(1) << 31) - 1 || pl->nbcap >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  pl->nscan = static_cast<int>((pl->ntile + kScanPerBlock - 1) / kScanPerBlock);
  if (pl->nscan > 1024 * 64) return MSA_ERR_UNSUPPORTED;
  const int64_t max_rows =
      std::min(kMaxChunkRows, ((int64_t(1) << 31) - 1) / (static_cast<int64_t>(H_kv) * topk));
  const int64_t all = std::max<int64_t>(1, seqs->total_q_rows);
  pl->chunk_rows = std::min(all, max_rows);
  kl_layout(*pl, seqs, H_kv, D, topk);
  if (pl->total > budget) {
    pl->chunk_rows = 1;
    kl_layout(*pl, seqs, H_kv, D, topk);
    const size_t one = pl->total;
    if (one > budget) return MSA_ERR_WORKSPACE;
    pl->chunk_rows = 2;
    kl_layout(*pl, seqs, H_kv, D, topk);
    const size_t per_row = pl->total - one + 1024;
    pl->chunk_rows = std::min(std::min(all, max_rows), 1 + static_cast<int64_t>((budget - one) / per_row));
    kl_layout(*pl, seqs, H_kv, D, topk);
    while (pl->total > budget && pl->chunk_rows > 1) {
      pl->chunk_rows = std::max<int64_t>(1, pl->chunk_rows * 7 / 8);
      kl_layout(*pl, seqs, H_kv, D, topk);
    }
    if (pl->total > budget) return MSA_ERR_WORKSPACE;
  }
  return MSA_OK;
}

int validate_kl(const msa_seqs* seqs, int H_q, int H_kv, int d_idx, int head_dim, int BK, int topk) {
  int st = msa_host::validate_seqs(seqs);
  if (st != MSA_OK) return st;
  if (H_q < 1 || H_kv < 1 || d_idx < 1 || head_dim < 1 || BK < 1 || topk < 1) return MSA_ERR_INVALID;
  if (H_q % H_kv != 0) return MSA_ERR_INVALID;
  if (head_dim != kHeadDim || (BK != kKlBK && BK != 2 * kKlBK) || (d_idx != 64 && d_idx != 128))
    return MSA_ERR_UNSUPPORTED;
  if (BK == 2 * kKlBK && topk > 32) return MSA_ERR_UNSUPPORTED;   // its 64-key halves fill <= 64 slots
  if (topk > 64 || H_q / H_kv > 16 || !msa_host::is_pow2(H_q / H_kv) || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (seqs->total_q_rows * H_kv >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  if (seqs->block_table) return MSA_ERR_UNSUPPORTED;   // contiguous key side only
  return MSA_OK;
}

// kl_grad_wave_kernel instance for G = 2^lg (lg <= 4, checked by validate_kl).
template <int D, typename... Args>
void launch_kl_grad_wave(int lg, dim3 grid, hipStream_t stream, Args... args) {
  switch (lg) {
    case 0: msa_prof::launch("kl_grad_wave_kernel", kl_grad_wave_kernel<D, 0>, grid, dim3(kKlThreads), 0, stream, args...); break;
    case 1: msa_prof::launch("kl_grad_wave_kernel", kl_grad_wave_kernel<D, 1>, grid, dim3(kKlThreads), 0, stream, args...); break;
    case 2: msa_prof::launch("kl_grad_wave_kernel", kl_grad_wave_kernel<D, 2>, grid, dim3(kKlThreads), 0, stream, args...); break;
    case 3: msa_prof::launch("kl_grad_wave_kernel", kl_grad_wave_kernel<D, 3>, grid, dim3(kKlThreads), 0, stream, args...); break;
    default: msa_prof::launch("kl_grad_wave_kernel", kl_grad_wave_kernel<D, 4>, grid, dim3(kKlThreads), 0, stream, args...); break;
  }
}

template <int D>
int run_kl(const void* index_q, const void* index_k, const void* q, const void* k, const float* lse,
           const int32_t* block_ids, const msa_seqs* seqs, int H_q, int H_kv, int topk, float softmax_scale,
           float grad_scale, void* d_index_q, void* d_index_k, float* kl, const KlPlan& pl, char* ws,
           hipStream_t stream) {
  auto* blk_base = reinterpret_cast<int64_t*>(ws + pl.off_blk_base);
  auto* cnt = reinterpret_cast<int32_t*>(ws + pl.off_cnt);
  auto* tile_off = reinterpret_cast<int32_t*>(ws + pl.off_tile_off);
  auto* item_off = reinterpret_cast<int32_t*>(ws + pl.off_item_off);
  auto* blk_tot = reinterpret_cast<int32_t*>(ws + pl.off_blk_tot);
  auto* dk_acc = reinterpret_cast<float*>(ws + pl.off_dk);
  auto* handles = reinterpret_cast<uint32_t*>(ws + pl.off_handles);
  auto* tpos = reinterpret_cast<int32_t*>(ws + pl.off_tpos);
  auto* lsep = reinterpret_cast<float*>(ws + pl.off_lsep);
  auto* lsei = reinterpret_cast<float*>(ws + pl.off_lsei);
  auto* dqp = reinterpret_cast<float*>(ws + pl.off_dqp);
  auto* klp = reinterpret_cast<float*>(ws + pl.off_klp);
  auto* part = reinterpret_cast<float*>(ws + pl.off_part);
  const msa_seqs sq = *seqs;
  const int64_t kv_floats = seqs->total_kv_rows * static_cast<int64_t>(D);
  const unsigned zero_blocks = static_cast<unsigned>(std::min<int64_t>((kv_floats + 255) / 256, 8192));
  const float sidx = 1.f / std::sqrt(static_cast<float>(D));
  const auto* iq = static_cast<const uint16_t*>(index_q);
  const auto* ik = static_cast<const uint16_t*>(index_k);

  msa_prof::launch("kvo_block_base_kernel", kvo_block_base_kernel, dim3(1), dim3(256), 0, stream, sq, kKlBK,
                   blk_base);
  msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                   reinterpret_cast<int32_t*>(dk_acc), kv_floats, 0);
  static std::atomic<int> ctas_lse {0}, ctas_grad {0};
  const int n_lse = persistent_ctas(kl_lse_kernel<D>, kKlThreads, &ctas_lse);
  const int n_grad = persistent_ctas(kl_grad_wave_kernel<D, 3>, kKlThreads, &ctas_grad);
  const int lg_g = __builtin_ctz(static_cast<unsigned>(H_q / H_kv));
  const int64_t trash_inc = pl.chunk_rows * H_kv * static_cast<int64_t>(topk);
  for (int64_t r0 = 0; r0 < seqs->total_q_rows; r0 += pl.chunk_rows) {
    const int64_t nr = std::min<int64_t>(pl.chunk_rows, seqs->total_q_rows - r0);
    const int64_t pairs = nr * H_kv;
    build_reverse_index(block_ids, sq, blk_base, H_kv, kKlBK, topk, pl.nbcap, pl.ntile, pl.nscan, r0, nr, cnt,
                        tile_off, item_off, blk_tot, tpos, handles, stream, true);
    msa_prof::launch("kl_lse_kernel", kl_lse_kernel<D>, dim3(n_lse), dim3(kKlThreads), 0, stream, iq, ik, sq,
                     static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(tile_off),
                     static_cast<const int32_t*>(item_off), static_cast<const uint32_t*>(handles), H_kv, topk,
                     pl.nbcap, r0, sidx * kLog2e, lsep, cnt + pl.ntile);
    msa_prof::launch("kl_lse_combine_kernel", kl_lse_combine_kernel, dim3(static_cast<unsigned>((pairs + 255) / 256)),
                     dim3(256), 0, stream, block_ids, sq, static_cast<const int64_t*>(blk_base), H_kv, topk, r0, nr,
                     static_cast<const float*>(lsep), lsei);
    launch_kl_grad_wave<D>(lg_g, dim3(n_grad), stream, iq, ik, static_cast<const uint16_t*>(q),
                        static_cast<const uint16_t*>(k), lse, static_cast<const float*>(lsei), sq,
                        static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(tile_off),
                        static_cast<const int32_t*>(item_off), static_cast<const uint32_t*>(handles), H_q, H_kv,
                        topk, pl.nbcap, r0, softmax_scale * kLog2e, sidx, trash_inc, dqp, klp, part,
                        cnt + pl.ntile + 1);
    msa_prof::launch("kl_tile_reduce_kernel", kl_tile_reduce_kernel<D>,
                     dim3(static_cast<unsigned>(pl.nbcap * kKlReduceSplit<D>)),
                     dim3(256), 0, stream, sq, static_cast<const int64_t*>(blk_base),
                     static_cast<const int32_t*>(item_off), H_kv, pl.nbcap, static_cast<const float*>(part), dk_acc);
    msa_prof::launch("kl_combine_kernel", kl_combine_kernel<D>,
                     dim3(static_cast<unsigned>((pairs + kKlCombWaves - 1) / kKlCombWaves)), dim3(64 * kKlCombWaves),
                     0, stream, block_ids, sq, static_cast<const int64_t*>(blk_base), H_kv, topk, r0, nr,
                     static_cast<const float*>(dqp), static_cast<const float*>(klp), grad_scale * sidx,
                     static_cast<uint16_t*>(d_index_q), kl);
  }
  if (kv_floats > 0)
    msa_prof::launch("kl_convert_kernel", kl_convert_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                     static_cast<const float*>(dk_acc), kv_floats / 2, grad_scale * sidx,
                     static_cast<uint16_t*>(d_index_k));
  return msa_host::launch_status();
}

// Block size 128: each id is expanded to its two 64-key halves in front of
// the workspace and the 64-key path runs on 2 topk slots.
size_t kl_expanded_ids_bytes(const msa_seqs* seqs, int H_kv, int BK, int topk) {
  if (BK == kKlBK) return 0;
  return msa_host::align_up(sizeof(int32_t) * static_cast<size_t>(seqs->total_q_rows) * H_kv * topk * (BK / kKlBK),
                            256);
}

}  // namespace

extern "C" size_t msa_sparse_kl_backward_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                                       int d_idx, int head_dim, int block_size, int topk) {
  if (validate_kl(seqs, num_q_heads, num_kv_heads, d_idx, head_dim, block_size, topk) != MSA_OK) return 0;
  const int topk64 = topk * (block_size / kKlBK);
  KlPlan pl;
  if (make_kl_plan(seqs, num_kv_heads, d_idx, topk64, kDefaultKlBytes, &pl) != MSA_OK) {
    if (make_kl_plan(seqs, num_kv_heads, d_idx, topk64, ~size_t(0) >> 1, &pl) != MSA_OK) return 0;
    pl.chunk_rows = 1;
    kl_layout(pl, seqs, num_kv_heads, d_idx, topk64);
  }
  return kl_expanded_ids_bytes(seqs, num_kv_heads, block_size, topk) + pl.total;
}

extern "C" int msa_sparse_kl_backward(const void* index_q, const void* index_k, const void* q, const void* k,
                                      const float* lse, const int32_t* block_ids, const msa_seqs* seqs,
                                      int num_q_heads, int num_kv_heads, int d_idx, int head_dim, int block_size,
                                      int topk, float softmax_scale, float grad_scale, void* d_index_q,
                                      void* d_index_k, float* kl, void* workspace, size_t workspace_bytes,
                                      hipStream_t stream) {
  int st = validate_kl(seqs, num_q_heads, num_kv_heads, d_idx, head_dim, block_size, topk);
  if (st != MSA_OK) return st;
  if (!index_q || !index_k || !q || !k || !lse || !block_ids || !d_index_q || !d_index_k) return MSA_ERR_INVALID;
  if (seqs->total_q_rows == 0 && seqs->total_kv_rows == 0) return MSA_OK;
  const size_t xb = kl_expanded_ids_bytes(seqs, num_kv_heads, block_size, topk);
  if (!workspace || workspace_bytes < xb) return MSA_ERR_WORKSPACE;
  const int f = block_size / kKlBK;
  const int32_t* ids = block_ids;
  if (f > 1) {
    auto* ids64 = static_cast<int32_t*>(workspace);
    const int64_t pairs = seqs->total_q_rows * num_kv_heads;
    if (pairs > 0)
      msa_prof::launch("expand_block_ids_kernel", expand_block_ids_kernel,
                       dim3(static_cast<unsigned>((pairs + 255) / 256)), dim3(256), 0, stream, block_ids, pairs, topk,
                       f, ids64);
    ids = ids64;
  }
  const int topk64 = topk * f;
  KlPlan pl;
  st = make_kl_plan(seqs, num_kv_heads, d_idx, topk64, workspace_bytes - xb, &pl);
  if (st != MSA_OK) return st;
  if (workspace_bytes - xb < pl.total) return MSA_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace) + xb;
  if (d_idx == 64)
    return run_kl<64>(index_q, index_k, q, k, lse, ids, seqs, num_q_heads, num_kv_heads, topk64, softmax_scale,
                      grad_scale, d_index_q, d_index_k, kl, pl, ws, stream);
  return run_kl<128>(index_q, index_k, q, k, lse, ids, seqs, num_q_heads, num_kv_heads, topk64, softmax_scale,
                     grad_scale, d_index_q, d_index_k, kl, pl, ws, stream);
}
