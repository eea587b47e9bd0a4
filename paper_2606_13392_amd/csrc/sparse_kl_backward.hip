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
// sweep.  The sweeps use the reverse index of kvo_index.h on the call's own
// key blocks (B_k = 64 or 128), per chunk of query rows:
//   kl_lse           per incidence: ln sum_j exp(s_idx S_idx_j) over the block's visible keys
//   kl_lse_combine   per (row, group): LSE_idx over the valid slots
//   kl_grad          per work item (<= 256 queries of one tile), one wave per
//                    pass of 16 queries: the teacher on MFMA 16x16x32 over the
//                    pass's 16 G (query, head) rows in sub-passes of 32, its
//                    head mean into an LDS tile; the student on the 16 query
//                    rows only: P_idx, Delta, the KL terms, d q_idx
//                    (Delta k_idx) as fp32 partials per incidence, and Delta
//                    in bf16 per incidence for the next kernel
//   kl_dk            per work item: d k_idx of the block = Delta^T q_idx over
//                    the item's queries (MFMA, both operands read down
//                    columns with transposing LDS reads), an fp32 partial
//   kl_tile_reduce   per key block: the items of every group's tile, in
//                    order, added to the fp32 d k_idx accumulator
//   kl_combine       per (row, group): d q_idx and KL over the valid slots, in
//                    slot order
// and at the end kl_convert (accumulator times grad_scale to bf16).  No
// atomics touch a result except the reverse index's handle order, which the
// index sorts per tile, so every output is bit-reproducible.
#include "kvo_index.h"

namespace {

constexpr int kKlThreads = 256;                       // LSE sweep: 4 waves
constexpr int kK2Waves = 8;                           // gradient and d k_idx kernels: 8 waves
constexpr int kK2Threads = kK2Waves * kWave;
constexpr int kK2Q = 16;                              // student queries per pass


// ---------------------------------------------------------------- LSE_idx
template <int BK, int D>
struct KlLseSmem {
  uint16_t ki[BK][D + 8];
  int32_t s_row[kItemQueries];
  int32_t s_slot[kItemQueries];
};

// Per work item: each wave takes 16 queries at a time; S_idx (16 queries x BK
// keys) on MFMA 16x16x32, masked to the visible keys, reduced to the block's
// log-sum-exp per query.
template <int BK, int D>
__global__ __launch_bounds__(kKlThreads) void kl_lse_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, msa_seqs sq,
    const int64_t* __restrict__ blk_base, const int32_t* __restrict__ tile_off, const int32_t* __restrict__ item_off,
    const uint32_t* __restrict__ handles, int H_kv, int topk, int64_t nbcap, int64_t row0, float sidx_log2,
    float* __restrict__ lse_part, int32_t* __restrict__ next_item) {
  static_assert(kItemQueries <= kKlThreads, "every thread loads at most one handle of an item");
  __shared__ KlLseSmem<BK, D> sm;
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
    const int key0 = static_cast<int>(gb - blk_base[s]) * BK;
    const int pos_base = g.kv_len - g.q_rows + static_cast<int>(row0 - g.q_begin);
    __syncthreads();
    if (static_cast<int>(threadIdx.x) < nq) {
      const uint32_t hd = handles[h0 + threadIdx.x];
      sm.s_row[threadIdx.x] = static_cast<int32_t>(hd >> 6);
      sm.s_slot[threadIdx.x] = static_cast<int32_t>(hd & 63u);
    }
    if (tile != staged) {
      const uint16_t* ikb = index_k + key_blocks(sq, g, s, BK).row(key0 / BK) * static_cast<int64_t>(D);
      for (int c = threadIdx.x; c < BK * (D / 8); c += kKlThreads) {
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
      constexpr int KT = BK / 16;
      f32x4 acc[KT];
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
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
        for (int kt = 0; kt < KT; ++kt) {
          const float z = key0 + 16 * kt + c16 <= pos ? acc[kt][i] * sidx_log2 : -INFINITY;
          acc[kt][i] = z;
          m = fmaxf(m, z);
        }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) m = fmaxf(m, __shfl_xor(m, off));
        const float mm = m == -INFINITY ? 0.f : m;
        float l = 0.f;
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) l += exp2f(acc[kt][i] - mm);
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

// One wave per (row, group) of the chunk, slot j on lane j: LSE_idx = ln sum
// over the valid slots of exp(partial) (a fixed butterfly order).
constexpr int kLseCombWaves = 4;
__global__ __launch_bounds__(64 * kLseCombWaves) void kl_lse_combine_kernel(
    const int32_t* __restrict__ block_ids, msa_seqs sq, const int64_t* __restrict__ blk_base, int BK, int H_kv,
    int topk, int64_t row0, int64_t nrows, const float* __restrict__ lse_part, float* __restrict__ lse_idx) {
  const int lane = lane_id();
  const int64_t pr = static_cast<int64_t>(blockIdx.x) * kLseCombWaves + threadIdx.x / kWave;
  if (pr >= nrows * H_kv) return;
  const int64_t row = row0 + pr / H_kv;
  const int r = static_cast<int>(pr % H_kv);
  int s;
  const int p = row_position(sq, row, &s);
  const bool ok = lane < topk && incidence_ok(block_ids[(row * H_kv + r) * topk + lane], p, BK, blk_base, s);
  const float x = ok ? lse_part[pr * topk + lane] : -INFINITY;
  float m = x;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  float l = m > -INFINITY && ok ? __expf(x - m) : 0.f;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) l += __shfl_xor(l, off);
  if (lane == 0) lse_idx[pr] = m > -INFINITY ? m + __logf(l) : -INFINITY;
}

// ---------------------------------------------------------------- LDS staging
// Staged rows of W bf16 (W = 64 or 128) have their 16-byte segments permuted
// (an XOR with a row-dependent mask) so that both read patterns below are
// free of bank conflicts: 16 consecutive rows at one segment (16 bytes per
// lane) and, for the transposing reads, 4 consecutive rows x 2 adjacent
// segments per 16 lanes.  A 128-element row fills the 64 banks, two
// 64-element rows share them.
template <int W>
__device__ __forceinline__ int kl_seg(int r, int s) {
  if constexpr (W == 128) return s ^ (((r & 7) << 1) | ((r >> 3) & 1));
  else return s ^ ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
}
// element offset of (row, col) in a permuted block; col % 8 is 0 or 4
template <int W>
__device__ __forceinline__ int kl_off(int r, int col) {
  return r * W + 8 * kl_seg<W>(r, col >> 3) + (col & 7);
}
// global_load_lds: lane l's 16 bytes land at dst + 16 l (dst wave-uniform)
__device__ __forceinline__ void kl_dma16(const uint16_t* src, uint16_t* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}
// transposing LDS read: in each 16-lane group, lane j addresses row k0 + j/4,
// columns n0 + 4(j%4) .. +3 and receives rows k0 .. k0+3 of column n0 + j
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short kl_v4i16;
__device__ __forceinline__ uint2 kl_tr4(const uint16_t* p) {
  const kl_v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) kl_v4i16*)(kl_v4i16*)(const_cast<uint16_t*>(p)));
  return __builtin_bit_cast(uint2, x);
}
// B operand (8 consecutive rows k0 .. k0+7 of column n0 + lane % 16) of
// MFMA 16x16x32 from a permuted block, by two transposing reads
template <int W>
__device__ __forceinline__ bf16x8 kl_col8(const uint16_t* blk, int k0, int n0, int c16) {
  const int col = n0 + 4 * (c16 & 3);
  const uint2 a = kl_tr4(blk + kl_off<W>(k0 + (c16 >> 2), col));
  const uint2 b = kl_tr4(blk + kl_off<W>(k0 + 4 + (c16 >> 2), col));
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}
// Rows 0 .. rows-1 of a block of row width W into LDS by DMA, by all NT
// threads: wave instruction `piece` fills 1 KiB = 64 / (W / 8) rows; a lane's
// source row comes from row_src (rows past the data re-read a valid row).
template <int W, int NT, typename RowSrc>
__device__ __forceinline__ void kl_stage(int rows, RowSrc row_src, uint16_t* dst) {
  constexpr int SEGS = W / 8;
  constexpr int RPI = 64 / SEGS;
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  for (int piece = wave; piece * RPI < rows; piece += NT / kWave) {
    const int row = piece * RPI + lane / SEGS;
    kl_dma16(row_src(row) + 8 * kl_seg<W>(row, lane % SEGS), dst + piece * RPI * W);
  }
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

template <int BK, int D>
struct Kl2Wave {
  float pbar[kK2Q][BK + 4];                           // teacher head mean per (pass query, key); Delta in
                                                      // bf16 then overwrites each row's front half
  float lse2[32];                                     // teacher rows of a sub-pass: LSE * log2(e) (+inf: none)
  int32_t pos[kK2Q];                                  // position of each pass query (-1: none)
  float lsei2[kK2Q];                                  // LSE_idx * log2(e) of each pass query
  int64_t inc[kK2Q];                                  // incidence of each pass query (the trash one for none)
};
template <int BK, int D>
struct Kl2Smem {
  uint16_t k[BK * kHeadDim];                          // K block of head group r, permuted rows
  uint16_t ki[BK * D];                                // index-key block, permuted rows
  Kl2Wave<BK, D> wv[kK2Waves];
  int32_t s_row[kItemQueries];
  int32_t s_slot[kItemQueries];
};
static_assert(sizeof(Kl2Smem<128, 128>) <= 160 * 1024, "LDS of the KL gradient CTA");

// One CTA of 8 waves per work item; wave w takes passes w, w + 8, ... of 16
// queries.  Teacher: the pass's 16 G (query, head) rows in sub-passes of 32
// (16 for G = 1), Q gathered one sub-pass ahead; S = Q K^T on MFMA 16x16x32,
// P = exp2(s S log2 e - LSE log2 e) on the visible keys, the head mean over
// each query's G rows (registers and lane swaps), stored per (query, key).
// Student, on the 16 query rows: S_idx, P_idx = exp2(s_idx S_idx log2 e -
// LSE_idx log2 e), Delta = P_idx - P, the KL terms (summed per query over the
// block's keys), d q_idx = Delta k_idx over the block's keys.
template <int BK, int D, int LG>
__global__ __launch_bounds__(kK2Threads, 1) void kl_grad_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k, const float* __restrict__ lse, const float* __restrict__ lse_idx, msa_seqs sq,
    const int64_t* __restrict__ blk_base, const int32_t* __restrict__ tile_off, const int32_t* __restrict__ item_off,
    const uint32_t* __restrict__ handles, int H_q, int H_kv, int topk, int64_t nbcap, int64_t row0,
    float s_main_log2, float sidx_log2, int64_t trash_inc, float* __restrict__ dqp, float* __restrict__ klp,
    uint16_t* __restrict__ dlt, int32_t* __restrict__ next_item) {
  static_assert(kItemQueries <= kK2Threads, "every thread loads at most one handle of an item");
  __shared__ __align__(16) Kl2Smem<BK, D> sm;
  __shared__ int32_t s_claim;
  constexpr int G = 1 << LG;
  constexpr int R = G >= 2 ? 32 : 16;                 // teacher rows per sub-pass
  constexpr int NTT = R / 16;                         // teacher row tiles
  constexpr int NSP = kK2Q * G / R;                   // sub-passes per pass
  constexpr int KT = BK / 16;                         // key tiles
  constexpr int KSM = kHeadDim / 32;                  // k-steps over the head dimension
  constexpr int KSI = D / 32;                         // k-steps over d_idx
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int c16 = lane & 15, qd = lane >> 4;
  const int64_t ntile = static_cast<int64_t>(H_kv) * nbcap;
  const int32_t total_items = item_off[ntile];
  const int64_t kv_stride = static_cast<int64_t>(H_kv) * kHeadDim;
  Kl2Wave<BK, D>& wv = sm.wv[w];
  int64_t staged = -1;

  for (int32_t item = blockIdx.x; item < total_items; item = claim_next_item(next_item, &s_claim)) {
    const int64_t tile = upper_index(item_off, ntile + 1, item);
    const int32_t h0 = tile_off[tile] + (item - item_off[tile]) * kItemQueries;
    const int32_t nq = min(tile_off[tile + 1] - h0, kItemQueries);
    const int r = static_cast<int>(tile / nbcap);
    const int64_t gb = tile % nbcap;
    const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
    const SeqGeom g = seq_geom(sq, s);
    const int key0 = static_cast<int>(gb - blk_base[s]) * BK;
    const int nkey = g.kv_len - key0;                 // >= 1: a tile with queries has a visible key
    const int pos_base = g.kv_len - g.q_rows + static_cast<int>(row0 - g.q_begin);

    __syncthreads();                                  // the previous item is done with LDS
    if (static_cast<int>(threadIdx.x) < nq) {
      const uint32_t hd = handles[h0 + threadIdx.x];
      sm.s_row[threadIdx.x] = static_cast<int32_t>(hd >> 6);
      sm.s_slot[threadIdx.x] = static_cast<int32_t>(hd & 63u);
    }
    if (tile != staged) {
      const int64_t krow0 = key_blocks(sq, g, s, BK).row(key0 / BK);   // contiguous, or inside its page
      const uint16_t* kb = k + krow0 * kv_stride + static_cast<int64_t>(r) * kHeadDim;
      const uint16_t* ikb = index_k + krow0 * static_cast<int64_t>(D);
      kl_stage<kHeadDim, kK2Threads>(BK, [&](int row) { return kb + min(row, nkey - 1) * kv_stride; }, sm.k);
      kl_stage<D, kK2Threads>(BK, [&](int row) { return ikb + min(row, nkey - 1) * static_cast<int64_t>(D); }, sm.ki);
      staged = tile;
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    const int npass = (nq + kK2Q - 1) / kK2Q;
    // teacher sub-pass (pass, sp): A operands (Q rows 16t + c16) and their LSEs
    // (loads only: their values are first used a sub-pass later)
    u32x4 aq[NTT][KSM], an[NTT][KSM];                // this sub-pass's, the next one's
    float al[NTT], aln[NTT];                         // raw LSEs
    bool av[NTT], avn[NTT];                          // row has a query
    auto load_sub = [&](int ps, int sp, u32x4 (&a)[NTT][KSM], float (&l)[NTT], bool (&v)[NTT]) {
#pragma unroll
      for (int t = 0; t < NTT; ++t) {
        const int x = sp * R + 16 * t + c16;          // teacher row of the pass
        const int jq = ps * kK2Q + (x >> LG);         // its query in the item
        const int j = min(jq, nq - 1);
        const int64_t hrow = (row0 + sm.s_row[j]) * H_q + static_cast<int64_t>(r) * G + (x & (G - 1));
#pragma unroll
        for (int st = 0; st < KSM; ++st) a[t][st] = load_raw(q + hrow * kHeadDim + 32 * st + 8 * qd);
        l[t] = lse[hrow];
        v[t] = jq < nq;
      }
    };
    // one teacher sub-pass on operands (a, l, v); the next sub-pass's
    // gathers (the wave's last one reloads a valid row) go out first into
    // (na, nl, nv), unconditionally, so that no copy waits on them
    auto sub = [&](int ps, int sp, u32x4 (&a)[NTT][KSM], float (&l)[NTT], bool (&v)[NTT],
                   u32x4 (&na)[NTT][KSM], float (&nl)[NTT], bool (&nv)[NTT]) {
      int nps = ps, nsp = sp + 1;
      if (nsp == NSP) { nps = min(ps + kK2Waves, npass - 1); nsp = 0; }
      load_sub(nps, nsp, na, nl, nv);
      asm volatile("" ::: "memory");                  // the gathers stay ahead of this sub-pass's MFMAs
      __builtin_amdgcn_sched_barrier(0);
      if (qd == 0) {
#pragma unroll
        for (int t = 0; t < NTT; ++t) wv.lse2[16 * t + c16] = v[t] ? l[t] * kLog2e : INFINITY;
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // this lane's rows' LSE and query position, read once for all key tiles
      float l2r[NTT][4];
      int posr[NTT][4];
#pragma unroll
      for (int t = 0; t < NTT; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int row = 16 * t + 4 * qd + i;
          l2r[t][i] = wv.lse2[row];
          posr[t][i] = wv.pos[(sp * R + row) >> LG];
        }
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        f32x4 acc[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) acc[t] = f32x4{};
#pragma unroll
        for (int st = 0; st < KSM; ++st) {
          const bf16x8 kb8 = ld_bf16x8(sm.k + kl_off<kHeadDim>(16 * kt + c16, 32 * st + 8 * qd));
#pragma unroll
          for (int t = 0; t < NTT; ++t) acc[t] = mfma16x16x32(__builtin_bit_cast(bf16x8, a[t][st]), kb8, acc[t]);
        }
        const int key = key0 + 16 * kt + c16;
#pragma unroll
        for (int t = 0; t < NTT; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            acc[t][i] = key <= posr[t][i] ? exp2_hw(acc[t][i] * s_main_log2 - l2r[t][i]) : 0.f;
        if constexpr (LG > 0) head_mean(acc, LG);
#pragma unroll
        for (int t = 0; t < NTT; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int row = 16 * t + 4 * qd + i;
            if ((row & (G - 1)) == 0) wv.pbar[(sp * R + row) >> LG][16 * kt + c16] = acc[t][i];
          }
      }
    };
    int ps = w;
    if (ps < npass) load_sub(ps, 0, aq, al, av);
    for (; ps < npass; ps += kK2Waves) {
      const int cq = ps * kK2Q;
      if (lane < kK2Q) {
        const bool ok = cq + lane < nq;
        const int j = min(cq + lane, nq - 1);
        const int32_t rl = sm.s_row[j];
        wv.pos[lane] = ok ? pos_base + rl : -1;
        wv.lsei2[lane] = ok ? lse_idx[static_cast<int64_t>(rl) * H_kv + r] * kLog2e : INFINITY;
        wv.inc[lane] = ok ? (static_cast<int64_t>(rl) * H_kv + r) * topk + sm.s_slot[j] : trash_inc;
      }
      // the student's index-query rows (lane c16 supplies query c16), in
      // flight during the teacher
      u32x4 ai[KSI];
      {
        const int j = min(cq + c16, nq - 1);
        const int64_t grow = row0 + sm.s_row[j];
#pragma unroll
        for (int ks = 0; ks < KSI; ++ks) ai[ks] = load_raw(index_q + (grow * H_kv + r) * D + 32 * ks + 8 * qd);
      }
      // ---- teacher: sub-passes in pairs, the two operand sets trading roles
      if constexpr (NSP % 2 == 0) {
#pragma unroll 1
        for (int sp = 0; sp < NSP; sp += 2) {
          sub(ps, sp, aq, al, av, an, aln, avn);
          sub(ps, sp + 1, an, aln, avn, aq, al, av);
        }
      } else {
        sub(ps, 0, aq, al, av, an, aln, avn);
#pragma unroll
        for (int t = 0; t < NTT; ++t) {
          al[t] = aln[t];
          av[t] = avn[t];
#pragma unroll
          for (int st = 0; st < KSM; ++st) aq[t][st] = an[t][st];
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

      // ---- student: rows = the pass's 16 queries (lane c16 supplies query c16)
      float klq[4] = {0.f, 0.f, 0.f, 0.f};
      int qpos[4];
      float ql2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        qpos[i] = wv.pos[4 * qd + i];
        ql2[i] = wv.lsei2[4 * qd + i];
      }
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) {
        f32x4 acc = f32x4{};
#pragma unroll
        for (int ks = 0; ks < KSI; ++ks)
          acc = mfma16x16x32(__builtin_bit_cast(bf16x8, ai[ks]), ld_bf16x8(sm.ki + kl_off<D>(16 * kt + c16, 32 * ks + 8 * qd)),
                             acc);
        // lane (key 16kt + c16, queries 4qd + i)
        const int key = key0 + 16 * kt + c16;
        float pb[4], dl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) pb[i] = wv.pbar[4 * qd + i][16 * kt + c16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool on = key <= qpos[i];
          const float lz = acc[i] * sidx_log2 - ql2[i];            // log2 P_idx
          const float pidx = on ? exp2_hw(lz) : 0.f;
          klq[i] += (on && pb[i] > 0.f) ? pb[i] * (__log2f(pb[i]) - lz) * kLn2 : 0.f;
          dl[i] = on ? pidx - pb[i] : 0.f;
        }
        // Delta in bf16 over the front of the row: bytes [32kt, 32kt + 32)
        // hold P of keys 8kt .. 8kt+7, read at key tile kt/2 <= kt
#pragma unroll
        for (int i = 0; i < 4; ++i)
          reinterpret_cast<uint16_t*>(wv.pbar[4 * qd + i])[16 * kt + c16] = f32_to_bf16_bits(dl[i]);
      }
      // KL per query: the 16 key lanes
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v = klq[i];
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off);
        if (c16 == 0) klp[wv.inc[4 * qd + i]] = v;
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // Delta rows of the pass to the incidence-major buffer (d k_idx pass)
#pragma unroll
      for (int c = lane; c < kK2Q * (BK / 8); c += kWave) {
        const int row = c / (BK / 8), seg = c % (BK / 8);
        *reinterpret_cast<uint4*>(dlt + wv.inc[row] * BK + 8 * seg) =
            *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(wv.pbar[row]) + 8 * seg);
      }
      // d q_idx = Delta (16 queries x BK keys) k_idx (BK x D): A = Delta rows,
      // B = k_idx columns by transposing reads
      int64_t incq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) incq[i] = wv.inc[4 * qd + i] * D;
#pragma unroll
      for (int n = 0; n < D / 16; ++n) {
        f32x4 acc = f32x4{};
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks)
          acc = mfma16x16x32(ld_bf16x8(reinterpret_cast<const uint16_t*>(wv.pbar[c16]) + 32 * ks + 8 * qd),
                             kl_col8<D>(sm.ki, 32 * ks + 8 * qd, 16 * n, c16), acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) dqp[incq[i] + 16 * n + c16] = acc[i];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }
}

// ---------------------------------------------------------------- d k_idx
template <int BK, int D>
struct Kl2DkSmem {
  uint16_t dl[kItemQueries * BK];                     // Delta row of each item query (permuted rows)
  uint16_t qi[kItemQueries * D];                      // index query row of each item query (permuted rows)
};
static_assert(sizeof(Kl2DkSmem<128, 128>) <= 160 * 1024, "LDS of the d k_idx CTA");

// One CTA of 8 waves per work item: d k_idx (BK x D) = sum over the item's
// queries (handle order) of Delta_q^T q_idx_q on MFMA 16x16x32, both
// operands read down columns with transposing reads; the item's fp32
// partial, row-major.  Query slots past the item read the trash incidence's
// Delta row, which is zero.
template <int BK, int D>
__global__ __launch_bounds__(kK2Threads, 1) void kl_dk_kernel(
    const uint16_t* __restrict__ index_q, msa_seqs sq, const int64_t* __restrict__ blk_base,
    const int32_t* __restrict__ tile_off, const int32_t* __restrict__ item_off, const uint32_t* __restrict__ handles,
    int H_kv, int topk, int64_t nbcap, int64_t row0, int64_t trash_inc, const uint16_t* __restrict__ dlt,
    float* __restrict__ part, int32_t* __restrict__ next_item) {
  __shared__ __align__(16) Kl2DkSmem<BK, D> sm;
  __shared__ int32_t s_claim;
  __shared__ int64_t s_inc[kItemQueries];
  __shared__ int64_t s_qrow[kItemQueries];
  constexpr int NTO = (BK / 16) * (D / 16);           // output tiles
  constexpr int PER = (NTO + kK2Waves - 1) / kK2Waves;
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int c16 = lane & 15, qd = lane >> 4;
  const int64_t ntile = static_cast<int64_t>(H_kv) * nbcap;
  const int32_t total_items = item_off[ntile];
  (void)sq;
  (void)blk_base;
  for (int32_t item = blockIdx.x; item < total_items; item = claim_next_item(next_item, &s_claim)) {
    const int64_t tile = upper_index(item_off, ntile + 1, item);
    const int32_t h0 = tile_off[tile] + (item - item_off[tile]) * kItemQueries;
    const int32_t nq = min(tile_off[tile + 1] - h0, kItemQueries);
    const int r = static_cast<int>(tile / nbcap);
    const int nq32 = (nq + 31) & ~31;
    __syncthreads();                                  // the previous item is done with LDS
    if (static_cast<int>(threadIdx.x) < nq32) {
      const int j = threadIdx.x;
      if (j < nq) {
        const uint32_t hd = handles[h0 + j];
        const int64_t rl = static_cast<int64_t>(hd >> 6);
        s_inc[j] = (rl * H_kv + r) * topk + static_cast<int64_t>(hd & 63u);
        s_qrow[j] = (row0 + rl) * H_kv + r;
      } else {
        s_inc[j] = trash_inc;
        s_qrow[j] = -1;
      }
    }
    __syncthreads();
    if (static_cast<int>(threadIdx.x) < nq32 && s_qrow[threadIdx.x] < 0) s_qrow[threadIdx.x] = s_qrow[0];
    __syncthreads();
    kl_stage<BK, kK2Threads>(nq32, [&](int row) { return dlt + s_inc[row] * BK; }, sm.dl);
    kl_stage<D, kK2Threads>(nq32, [&](int row) { return index_q + s_qrow[row] * D; }, sm.qi);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    f32x4 acc[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) acc[u] = f32x4{};
    for (int kk = 0; kk < nq32 / 32; ++kk) {
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int ot = w + kK2Waves * u;
        if (ot < NTO) {
          const int kt = ot / (D / 16), n = ot % (D / 16);
          // A: Delta^T rows = keys 16kt + c16, k = queries; B: q_idx columns
          acc[u] = mfma16x16x32(kl_col8<BK>(sm.dl, 32 * kk + 8 * qd, 16 * kt, c16),
                                kl_col8<D>(sm.qi, 32 * kk + 8 * qd, 16 * n, c16), acc[u]);
        }
      }
    }
    // C: lane (dim 16n + c16, keys 16kt + 4qd + i)
    float* dst = part + static_cast<int64_t>(item) * (BK * D);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int ot = w + kK2Waves * u;
      if (ot < NTO) {
        const int kt = ot / (D / 16), n = ot % (D / 16);
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[(16 * kt + 4 * qd + i) * D + 16 * n + c16] = acc[u][i];
      }
    }
  }
}

// Per key block: the items of the block's tiles of every group, in group and
// item order, added to the fp32 accumulator of the block's keys.
// BK D / 1024 CTAs per block, one float4 of the row-major partial per thread.
template <int BK, int D>
constexpr int kKlReduceSplit = BK * D / (4 * 256);
template <int BK, int D>
__global__ __launch_bounds__(256) void kl_tile_reduce_kernel(msa_seqs sq, const int64_t* __restrict__ blk_base,
                                                             const int32_t* __restrict__ item_off, int H_kv,
                                                             int64_t nbcap, const float* __restrict__ part,
                                                             float* __restrict__ dk_acc) {
  constexpr int SPLIT = kKlReduceSplit<BK, D>;
  const int64_t gb = blockIdx.x / SPLIT;
  const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
  const SeqGeom g = seq_geom(sq, s);
  const int key0 = static_cast<int>(gb - blk_base[s]) * BK;
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
      const float4 x = p4[static_cast<int64_t>(it) * (BK * D / 4)];
      acc.x += x.x;
      acc.y += x.y;
      acc.z += x.z;
      acc.w += x.w;
    }
  }
  const int key = (4 * c4) / D, dim = (4 * c4) % D;
  if (key0 + key >= g.kv_len) return;
  float4* dst = reinterpret_cast<float4*>(dk_acc + (key_blocks(sq, g, s, BK).row(key0 / BK) + key) *
                                                       static_cast<int64_t>(D) + dim);
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
    const int32_t* __restrict__ block_ids, msa_seqs sq, const int64_t* __restrict__ blk_base, int BK, int H_kv,
    int topk, int64_t row0, int64_t nrows, const float* __restrict__ dqp, const float* __restrict__ klp, float grad_scale,
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
  const bool mine = lane < topk && incidence_ok(ids[lane], p, BK, blk_base, s);
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
      off_lsei, off_dqp, off_klp, off_dlt, off_part, total;
};

constexpr size_t kDefaultKlBytes = size_t(16) << 30;

void kl_layout(KlPlan& pl, const msa_seqs* seqs, int H_kv, int BK, int D, int topk) {
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
  pl.off_dqp = o;      o = align_up(o + sizeof(float) * (inc + 1) * D, 256);        // + trash incidence
  pl.off_klp = o;      o = align_up(o + sizeof(float) * (inc + 1), 256);
  pl.off_dlt = o;      o = align_up(o + sizeof(uint16_t) * (inc + 1) * BK, 256);
  pl.off_part = o;     o = align_up(o + sizeof(float) * static_cast<size_t>(pl.max_items) * BK * D, 256);
  pl.total = o;
}

int make_kl_plan(const msa_seqs* seqs, int H_kv, int BK, int D, int topk, size_t budget, KlPlan* pl) {
  const int64_t nb = (seqs->max_kv_len + BK - 1) / BK;
  pl->nbcap = static_cast<int64_t>(seqs->num_seqs) * (nb > 0 ? nb : 1);
  pl->ntile = static_cast<int64_t>(H_kv) * pl->nbcap;
  if (pl->ntile >= (int64_t(1) << 31) - 1 || pl->nbcap >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  pl->nscan = static_cast<int>((pl->ntile + kScanPerBlock - 1) / kScanPerBlock);
  if (pl->nscan > 1024 * 64) return MSA_ERR_UNSUPPORTED;
  const int64_t max_rows =
      std::min(kMaxChunkRows, ((int64_t(1) << 31) - 1) / (static_cast<int64_t>(H_kv) * topk));
  const int64_t all = std::max<int64_t>(1, seqs->total_q_rows);
  pl->chunk_rows = std::min(all, max_rows);
  kl_layout(*pl, seqs, H_kv, BK, D, topk);
  if (pl->total > budget) {
    pl->chunk_rows = 1;
    kl_layout(*pl, seqs, H_kv, BK, D, topk);
    const size_t one = pl->total;
    if (one > budget) return MSA_ERR_WORKSPACE;
    pl->chunk_rows = 2;
    kl_layout(*pl, seqs, H_kv, BK, D, topk);
    const size_t per_row = pl->total - one + 1024;
    pl->chunk_rows = std::min(std::min(all, max_rows), 1 + static_cast<int64_t>((budget - one) / per_row));
    kl_layout(*pl, seqs, H_kv, BK, D, topk);
    while (pl->total > budget && pl->chunk_rows > 1) {
      pl->chunk_rows = std::max<int64_t>(1, pl->chunk_rows * 7 / 8);
      kl_layout(*pl, seqs, H_kv, BK, D, topk);
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
  if (head_dim != kHeadDim || (BK != 64 && BK != 128) || (d_idx != 64 && d_idx != 128)) return MSA_ERR_UNSUPPORTED;
  if (topk > 64 || H_q / H_kv > 16 || !msa_host::is_pow2(H_q / H_kv) || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (seqs->total_q_rows * H_kv >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  return msa_host::check_paged(seqs, BK, true);
}

// kl_grad_kernel instance for G = 2^lg (lg <= 4, checked by validate_kl).
template <int BK, int D, typename... Args>
void launch_kl_grad(int lg, dim3 grid, hipStream_t stream, Args... args) {
  switch (lg) {
    case 0: msa_prof::launch("kl_grad_kernel", kl_grad_kernel<BK, D, 0>, grid, dim3(kK2Threads), 0, stream, args...); break;
    case 1: msa_prof::launch("kl_grad_kernel", kl_grad_kernel<BK, D, 1>, grid, dim3(kK2Threads), 0, stream, args...); break;
    case 2: msa_prof::launch("kl_grad_kernel", kl_grad_kernel<BK, D, 2>, grid, dim3(kK2Threads), 0, stream, args...); break;
    case 3: msa_prof::launch("kl_grad_kernel", kl_grad_kernel<BK, D, 3>, grid, dim3(kK2Threads), 0, stream, args...); break;
    default: msa_prof::launch("kl_grad_kernel", kl_grad_kernel<BK, D, 4>, grid, dim3(kK2Threads), 0, stream, args...); break;
  }
}

template <int BK, int D>
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
  auto* dlt = reinterpret_cast<uint16_t*>(ws + pl.off_dlt);
  auto* part = reinterpret_cast<float*>(ws + pl.off_part);
  const msa_seqs sq = *seqs;
  const int64_t kv_floats = seqs->total_kv_rows * static_cast<int64_t>(D);
  const unsigned zero_blocks = static_cast<unsigned>(std::min<int64_t>((kv_floats + 255) / 256, 8192));
  const float sidx = 1.f / std::sqrt(static_cast<float>(D));
  const auto* iq = static_cast<const uint16_t*>(index_q);
  const auto* ik = static_cast<const uint16_t*>(index_k);
  const int64_t trash_inc = pl.chunk_rows * H_kv * static_cast<int64_t>(topk);

  msa_prof::launch("kvo_block_base_kernel", kvo_block_base_kernel, dim3(1), dim3(256), 0, stream, sq, BK,
                   blk_base);
  msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                   reinterpret_cast<int32_t*>(dk_acc), kv_floats, 0);
  // the trash incidence's Delta row stands in for the query slots past an item: zero
  msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(1), dim3(256), 0, stream,
                   reinterpret_cast<int32_t*>(dlt + trash_inc * BK), static_cast<int64_t>(BK / 2), 0);
  static std::atomic<int> ctas_lse {0}, ctas_grad {0}, ctas_dk {0};
  const int n_lse = persistent_ctas(kl_lse_kernel<BK, D>, kKlThreads, &ctas_lse);
  const int n_grad = persistent_ctas(kl_grad_kernel<BK, D, 3>, kK2Threads, &ctas_grad);
  const int n_dk = persistent_ctas(kl_dk_kernel<BK, D>, kK2Threads, &ctas_dk);
  const int lg_g = __builtin_ctz(static_cast<unsigned>(H_q / H_kv));
  for (int64_t r0 = 0; r0 < seqs->total_q_rows; r0 += pl.chunk_rows) {
    const int64_t nr = std::min<int64_t>(pl.chunk_rows, seqs->total_q_rows - r0);
    const int64_t pairs = nr * H_kv;
    build_reverse_index(block_ids, sq, blk_base, H_kv, BK, topk, pl.nbcap, pl.ntile, pl.nscan, r0, nr, cnt,
                        tile_off, item_off, blk_tot, tpos, handles, stream, true);
    msa_prof::launch("kl_lse_kernel", kl_lse_kernel<BK, D>, dim3(n_lse), dim3(kKlThreads), 0, stream, iq, ik, sq,
                     static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(tile_off),
                     static_cast<const int32_t*>(item_off), static_cast<const uint32_t*>(handles), H_kv, topk,
                     pl.nbcap, r0, sidx * kLog2e, lsep, cnt + pl.ntile);
    msa_prof::launch("kl_lse_combine_kernel", kl_lse_combine_kernel,
                     dim3(static_cast<unsigned>((pairs + kLseCombWaves - 1) / kLseCombWaves)),
                     dim3(64 * kLseCombWaves), 0, stream, block_ids, sq, static_cast<const int64_t*>(blk_base), BK, H_kv, topk, r0,
                     nr, static_cast<const float*>(lsep), lsei);
    launch_kl_grad<BK, D>(lg_g, dim3(n_grad), stream, iq, ik, static_cast<const uint16_t*>(q),
                          static_cast<const uint16_t*>(k), lse, static_cast<const float*>(lsei), sq,
                          static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(tile_off),
                          static_cast<const int32_t*>(item_off), static_cast<const uint32_t*>(handles), H_q, H_kv,
                          topk, pl.nbcap, r0, softmax_scale * kLog2e, sidx * kLog2e, trash_inc, dqp, klp, dlt,
                          cnt + pl.ntile + 1);
    // d k_idx's persistent loop reuses the LSE sweep's work counter, reset
    msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(1), dim3(256), 0, stream, cnt + pl.ntile,
                     static_cast<int64_t>(1), 0);
    msa_prof::launch("kl_dk_kernel", kl_dk_kernel<BK, D>, dim3(n_dk), dim3(kK2Threads), 0, stream, iq, sq,
                     static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(tile_off),
                     static_cast<const int32_t*>(item_off), static_cast<const uint32_t*>(handles), H_kv, topk,
                     pl.nbcap, r0, trash_inc, static_cast<const uint16_t*>(dlt), part, cnt + pl.ntile);
    msa_prof::launch("kl_tile_reduce_kernel", kl_tile_reduce_kernel<BK, D>,
                     dim3(static_cast<unsigned>(pl.nbcap * kKlReduceSplit<BK, D>)), dim3(256), 0, stream, sq,
                     static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(item_off), H_kv, pl.nbcap,
                     static_cast<const float*>(part), dk_acc);
    msa_prof::launch("kl_combine_kernel", kl_combine_kernel<D>,
                     dim3(static_cast<unsigned>((pairs + kKlCombWaves - 1) / kKlCombWaves)), dim3(64 * kKlCombWaves),
                     0, stream, block_ids, sq, static_cast<const int64_t*>(blk_base), BK, H_kv, topk, r0, nr,
                     static_cast<const float*>(dqp), static_cast<const float*>(klp), grad_scale * sidx,
                     static_cast<uint16_t*>(d_index_q), kl);
  }
  if (kv_floats > 0)
    msa_prof::launch("kl_convert_kernel", kl_convert_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                     static_cast<const float*>(dk_acc), kv_floats / 2, grad_scale * sidx,
                     static_cast<uint16_t*>(d_index_k));
  return msa_host::launch_status();
}

}  // namespace

extern "C" size_t msa_sparse_kl_backward_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                                       int d_idx, int head_dim, int block_size, int topk) {
  if (validate_kl(seqs, num_q_heads, num_kv_heads, d_idx, head_dim, block_size, topk) != MSA_OK) return 0;
  KlPlan pl;
  if (make_kl_plan(seqs, num_kv_heads, block_size, d_idx, topk, kDefaultKlBytes, &pl) != MSA_OK) {
    if (make_kl_plan(seqs, num_kv_heads, block_size, d_idx, topk, ~size_t(0) >> 1, &pl) != MSA_OK) return 0;
    pl.chunk_rows = 1;
    kl_layout(pl, seqs, num_kv_heads, block_size, d_idx, topk);
  }
  return pl.total;
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
  if (!workspace) return MSA_ERR_WORKSPACE;
  KlPlan pl;
  st = make_kl_plan(seqs, num_kv_heads, block_size, d_idx, topk, workspace_bytes, &pl);
  if (st != MSA_OK) return st;
  if (workspace_bytes < pl.total) return MSA_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  if (block_size == 64) {
    if (d_idx == 64)
      return run_kl<64, 64>(index_q, index_k, q, k, lse, block_ids, seqs, num_q_heads, num_kv_heads, topk,
                            softmax_scale, grad_scale, d_index_q, d_index_k, kl, pl, ws, stream);
    return run_kl<64, 128>(index_q, index_k, q, k, lse, block_ids, seqs, num_q_heads, num_kv_heads, topk,
                           softmax_scale, grad_scale, d_index_q, d_index_k, kl, pl, ws, stream);
  }
  if (d_idx == 64)
    return run_kl<128, 64>(index_q, index_k, q, k, lse, block_ids, seqs, num_q_heads, num_kv_heads, topk,
                           softmax_scale, grad_scale, d_index_q, d_index_k, kl, pl, ws, stream);
  return run_kl<128, 128>(index_q, index_k, q, k, lse, block_ids, seqs, num_q_heads, num_kv_heads, topk,
                          softmax_scale, grad_scale, d_index_q, d_index_k, kl, pl, ws, stream);
}
