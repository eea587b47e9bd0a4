// Training backward of the MSA Main Branch on gfx950, key-block-outer.
//
// Alg. 1 trains through the sparse attention of Sec. 3.1: O_i = sum_j P_ij V_j
// with P_i = softmax(scale Q_i K_j^T) over the causally visible tokens of the
// blocks row i selected.  For an upstream gradient dO, with P recomputed from
// the forward's log-sum-exp and D_i = dO_i . O_i (the softmax Jacobian's
// row term),
//   dV_j += P_ij dO_i,   dP_ij = dO_i . V_j,   dS_ij = P_ij (dP_ij - D_i),
//   dQ_i += scale dS_ij K_j,   dK_j += scale dS_ij Q_i.
// Key blocks are iterated on the outside (the reverse index of kvo_index.h):
// dK and dV of a block stay in registers while the queries that selected it
// stream past, each incidence costs a gather of its Q and dO rows, and its dQ
// contribution goes as a bf16 partial into the incidence's slot.  No
// atomics touch a gradient: dQ sums its slot partials in slot order, and dK
// and dV sum a block's queries in the order of its handle list, which is
// sorted into ascending (row, slot) order after the reverse index is built,
// so every gradient is bit-reproducible.
//
//   bwd_delta        D per (row, head)
//   per chunk of query rows:
//     reverse index  (kvo_index.h)
//     bwd_kvo        persistent CTAs of B_k / 16 waves (two CTAs per CU at
//                    B_k 64, one at 128) over the work items (<= 256 queries
//                    of one tile).  K and V of the block sit in LDS row-major
//                    (K's 16-byte segments permuted per row).
//                    A pass takes 32 gathered (query, head) rows, whose Q and
//                    dO rows are copied from HBM straight into LDS (DMA) one
//                    pass ahead; wave kq owns keys 16kq .. 16kq+15: S = Q K^T
//                    and dP = dO V^T (MFMA 16x16x32, one key per lane column),
//                    then dV += P^T dO and dK += dS^T Q, their B operands read
//                    down the columns of the row-major Q / dO rows with
//                    transposing LDS reads, then dQ over the block's keys for
//                    the wave's dims from dS staged in LDS (K read the same
//                    way); dQ partials are stored one pass late.  At the end
//                    of an item each wave writes its keys' dK / dV as the
//                    item's partial.
//     bwd_tile_reduce  per tile: its items' partials, in order, added to fp32
//                    dK / dV accumulators
//     bwd_dq_combine per (row, group): the valid slots' partials in slot order,
//                    times scale, to bf16 dQ
//   bwd_kv_convert   accumulators (dK times scale) to bf16 dK, dV
#include "kvo_index.h"

namespace {

// Key blocks of 64 or 128 keys: one wave per 16 keys (4 or 8 waves per CTA).
template <int BK>
constexpr int bwd_waves() { return BK / 16; }
template <int BK>
constexpr int bwd_threads() { return 64 * bwd_waves<BK>(); }
constexpr int kBwdPassRows = 32;                      // gathered (query, head) rows per CTA pass
template <int BK>
constexpr int bwd_part_floats() { return 2 * BK * kHeadDim; }   // dK and dV of one work item

template <int BK>
struct BwdSmem {
  uint16_t k[BK][kHeadDim];                           // K block, 256-byte rows, segments swizzled (bwd_swz)
  uint16_t v[BK][kHeadDim + 8];                       // V block, row-major
  // Q and dO rows of a pass (double-buffered), row-major with 16-byte
  // segments XOR-swizzled by row (bwd_qrow_off); filled by DMA
  uint16_t qdo[2][2][kBwdPassRows][kHeadDim];
  uint16_t ds[32][BK + 8];                            // dS of the pass, [row][key]
  float lse[2][kBwdPassRows];                         // forward LSE per pass row (copied by DMA; a valid
                                                      // row's for rows without a query)
  float dlt[2][kBwdPassRows];                         // D per pass row (likewise)
  int32_t rpos[2][kBwdPassRows];                      // absolute position per pass row (-1: no row)
  int64_t dqoff[2][kBwdPassRows];                     // element offset of the row's dQ partial (the trash row: no row)
  int32_t s_row[kItemQueries];                        // query row inside the chunk
  int32_t s_slot[kItemQueries];                       // slot of this block in the row's id list
};
// B_k 64: two CTAs per CU; B_k 128: one CTA of 8 waves
static_assert(sizeof(BwdSmem<64>) <= 80 * 1024, "LDS of a B_k 64 backward CTA");
static_assert(sizeof(BwdSmem<128>) <= 160 * 1024, "LDS of a B_k 128 backward CTA");

// 256-byte rows (a pass buffer's Q / dO rows, the K block) keep their 16-byte
// segment s in slot s ^ bwd_swz(row).  The permutation moves segment pairs
// (2p, 2p + 1) as pairs, by (row & 7), and flips the low bit by bit 3 of the
// row, so that both read shapes are free of bank conflicts: 16-byte operand
// reads of 16 consecutive rows at one segment (16 distinct slots), and
// transposing reads of 4 consecutive rows x 16 columns (one segment pair per
// row, the four pairs distinct).
__device__ __forceinline__ int bwd_swz(int row) { return ((row & 7) << 1) | ((row >> 3) & 1); }
// Byte offset of element (row, col) in such a buffer.
__device__ __forceinline__ int bwd_qrow_off(int row, int col) {
  return row * (kHeadDim * 2) + 16 * ((col >> 3) ^ bwd_swz(row)) + 2 * (col & 7);
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
// Transposing LDS read (ds_read_b64_tr_b16): within each 16-lane group, lane
// j supplies the address of 4 consecutive bf16 elements, and lane 4a + b
// receives element b of the loads of lanes a, a + 4, a + 8, a + 12.  With lane
// j pointing at row k0 + j / 4, columns n0 + 4 (j % 4) .. + 3 of a row-major
// tile, lane n receives rows k0 .. k0 + 3 of column n0 + n: a 4-element slice
// of an MFMA B operand that runs down a column.
__device__ __forceinline__ uint2 lds_tr4(const void* p) {
  const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(v4i16*)(const_cast<void*>(p)));
  return __builtin_bit_cast(uint2, x);
}
// One 16-byte (or 4-byte) piece per lane from global memory into LDS
// (global_load_lds): lane l writes bytes [16 l, 16 l + 16) (or [4 l, 4 l + 4))
// after the wave-uniform LDS address dst.  Issued from inline assembly so
// that the compiler, which cannot tell the buffers apart, does not wait for
// these copies before every later LDS read: the pass loop waits for them
// itself (s_waitcnt before the barrier that publishes them).  M0 holds the
// LDS address; one wait state separates its write from the copy.
__device__ __forceinline__ uint32_t bwd_lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      static_cast<uint32_t>(reinterpret_cast<size_t>((__attribute__((address_space(3))) const void*)(p))));
}
__device__ __forceinline__ void bwd_dma16(const void* src, void* dst) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(bwd_lds_addr(dst)) : "m0");
}
__device__ __forceinline__ void bwd_dma4(const void* src, void* dst) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :: "v"(src), "s"(bwd_lds_addr(dst)) : "m0");
}

__device__ __forceinline__ uint16_t raw_elem(const u32x4& w, int j) {
  return static_cast<uint16_t>(w[j >> 1] >> (16 * (j & 1)));
}
__device__ __forceinline__ bf16x8 lds_pair_bf16x8(const uint16_t* lo, const uint16_t* hi) {
  const uint2 a = *reinterpret_cast<const uint2*>(lo), b = *reinterpret_cast<const uint2*>(hi);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// D[row, head] = sum_d dO . O; 16 lanes per (row, head), 8 dims each.
__global__ __launch_bounds__(256) void bwd_delta_kernel(const uint16_t* __restrict__ o, const uint16_t* __restrict__ d_o,
                                                        int64_t pairs, float* __restrict__ delta) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t pair = t >> 4;
  const int part = static_cast<int>(t & 15);
  float acc = 0.f;
  if (pair < pairs) {
    const u32x4 a = load_raw(o + pair * kHeadDim + 8 * part);
    const u32x4 b = load_raw(d_o + pair * kHeadDim + 8 * part);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc += __uint_as_float(a[j] << 16) * __uint_as_float(b[j] << 16);
      acc += __uint_as_float(a[j] & 0xFFFF0000u) * __uint_as_float(b[j] & 0xFFFF0000u);
    }
  }
#pragma unroll
  for (int off = 8; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (pair < pairs && part == 0) delta[pair] = acc;
}

// Wave kq owns keys 16kq .. 16kq+15 of the block.  MFMA 16x16x32: lane
// l = (c = l % 16, quarter qd = l / 16).  In S = Q K^T and dP = dO V^T the
// lane holds key 16kq + c and, of row tile t, rows 16t + 4qd + i (i = 0..3).
// Those 8 rows are the k-slice the lane supplies to dV += P^T dO and
// dK += dS^T Q (k index 8qd + 4t + i); the B operands read the same rows down
// each column of the row-major Q / dO pass buffers with transposing LDS
// reads, and dQ's B operand reads K the same way.  A pass's Q and dO rows are
// gathered straight into LDS (DMA) one pass ahead; its dQ partials are
// stored at the start of the next pass, so neither waits on memory.
template <int BK>
__global__ __launch_bounds__(bwd_threads<BK>(), BK == 64 ? 2 : 1) void bwd_kvo_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ d_o, const float* __restrict__ lse, const float* __restrict__ delta, msa_seqs sq,
    const int64_t* __restrict__ blk_base, const int32_t* __restrict__ tile_off, const int32_t* __restrict__ item_off,
    const uint32_t* __restrict__ handles, int H_q, int H_kv, int topk, int64_t nbcap, int64_t row0, float scale_log2,
    uint16_t* __restrict__ dq_buf, int64_t dq_trash, float* __restrict__ part, int32_t* __restrict__ next_item) {
  constexpr int NKW = bwd_waves<BK>();                // waves = 16-key slices of the block
  constexpr int kThreads = bwd_threads<BK>();
  static_assert(kItemQueries <= kThreads, "every thread loads at most one handle of an item");
  static_assert(2 * (kBwdPassRows / 4) % NKW == 0, "DMA pieces split evenly over the waves");
  __shared__ BwdSmem<BK> sm;
  __shared__ int32_t s_claim;
  constexpr int KS = kHeadDim / 32;                   // k-steps of S and dP over the head dimension
  constexpr int DQU = 8 / NKW;                        // 16-dim tiles of dQ per wave
  constexpr int kDma = 2 * (kBwdPassRows / 4) / NKW;  // 1 KiB DMA pieces per wave and pass
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int kq = wave;
  const int c16 = lane & 15, qd = lane >> 4;
  const int G = H_q / H_kv;
  const int qpw = 32 / G;                             // queries per pass
  const int rows_g = qpw * G;                         // used rows of a pass
  const int64_t ntile = static_cast<int64_t>(H_kv) * nbcap;
  const int32_t total_items = item_off[ntile];
  const int64_t kv_stride = static_cast<int64_t>(H_kv) * kHeadDim;
  int64_t staged = -1;
  const uint8_t* kbytes = reinterpret_cast<const uint8_t*>(&sm.k[0][0]);
  // pass-invariant splits of pass rows into (query, head): G need not be a
  // power of two, so the divisions are taken once here, not in every pass
  int dma_rq[kDma], dma_rh[kDma];
#pragma unroll
  for (int i = 0; i < kDma; ++i) {
    const int ra = 4 * ((kq * kDma + i) & 7) + (lane >> 4);
    dma_rq[i] = ra / G;
    dma_rh[i] = ra % G;
  }
  const int lane_rq = lane / G, lane_rh = lane % G;

  for (int32_t item = blockIdx.x; item < total_items; item = claim_next_item(next_item, &s_claim)) {
    const int64_t tile = upper_index(item_off, ntile + 1, item);
    const int32_t h0 = tile_off[tile] + (item - item_off[tile]) * kItemQueries;
    const int32_t nq = min(tile_off[tile + 1] - h0, kItemQueries);
    const int r = static_cast<int>(tile / nbcap);
    const int64_t gb = tile % nbcap;
    const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
    const SeqGeom g = seq_geom(sq, s);
    const int key0 = static_cast<int>(gb - blk_base[s]) * BK;

    __syncthreads();                                  // the previous item is done with LDS
    if (static_cast<int>(threadIdx.x) < nq) {
      const uint32_t hd = handles[h0 + threadIdx.x];
      sm.s_row[threadIdx.x] = static_cast<int32_t>(hd >> 6);
      sm.s_slot[threadIdx.x] = static_cast<int32_t>(hd & 63u);
    }
    const int pos_base = g.kv_len - g.q_rows + static_cast<int>(row0 - g.q_begin);   // + row in chunk
    if (tile != staged) {
      // the block's first key row (contiguous, or inside its page)
      const int64_t krow0 = key_blocks(sq, g, s, BK).row(key0 / BK);
      const uint16_t* kb = k + krow0 * kv_stride + static_cast<int64_t>(r) * kHeadDim;
      const uint16_t* vb = v + krow0 * kv_stride + static_cast<int64_t>(r) * kHeadDim;
      for (int c = threadIdx.x; c < BK * (kHeadDim / 8); c += kThreads) {
        const int key = c / (kHeadDim / 8), dg = c % (kHeadDim / 8);
        const bool in = key0 + key < g.kv_len;
        *reinterpret_cast<u32x4*>(&sm.k[key][8 * (dg ^ bwd_swz(key))]) =
            in ? load_raw(kb + static_cast<int64_t>(key) * kv_stride + 8 * dg) : u32x4{};
        *reinterpret_cast<u32x4*>(&sm.v[key][8 * dg]) =
            in ? load_raw(vb + static_cast<int64_t>(key) * kv_stride + 8 * dg) : u32x4{};
      }
      staged = tile;
    }
    __syncthreads();                                  // handles (and K / V) in LDS

    // pass row ra of the pass at item query cc: (query cc + ra / G, head ra % G);
    // rows past the pass's queries read a valid row (their P and dS are zero)
    // (rq, rh = ra / G, ra % G, precomputed)
    auto pass_row = [&](int cc, int ra, int rq, int rh, bool& ok) -> int64_t {
      const int qa = cc + rq;
      ok = ra < rows_g && qa < nq;
      const int64_t grow = row0 + sm.s_row[ok ? qa : min(cc, nq - 1)];
      return grow * H_q + static_cast<int64_t>(r) * G + (ok ? rh : 0);
    };
    // Q and dO rows of the pass at cc into buffer b: wave kq issues kDma 1 KiB
    // pieces (4 rows each); lane l of a piece writes slot l % 16 of row
    // 4 piece + l / 16, which holds the row's segment slot ^ bwd_swz(row)
    // (a row past the pass's queries reads head r G + ra % G of a valid query
    // row: any valid row serves, its P and dS are zero)
    const uint16_t* dma_base[kDma];
#pragma unroll
    for (int i = 0; i < kDma; ++i) {
      const int piece = kq * kDma + i;                // 0 .. 15: tensor piece / 8, rows 4 (piece % 8) ..
      const int ra = 4 * (piece & 7) + (lane >> 4);
      dma_base[i] = ((piece >> 3) == 0 ? q : d_o) + (static_cast<int64_t>(r) * G + dma_rh[i]) * kHeadDim +
                    8 * ((lane & 15) ^ bwd_swz(ra));
    }
    const int64_t row_elems = static_cast<int64_t>(H_q) * kHeadDim;
    auto issue_dma = [&](int cc, int b) {
#pragma unroll
      for (int i = 0; i < kDma; ++i) {
        const int piece = kq * kDma + i;
        const int qa = cc + dma_rq[i];
        const int64_t grow = row0 + sm.s_row[qa < nq ? qa : min(cc, nq - 1)];
        bwd_dma16(dma_base[i] + grow * row_elems, &sm.qdo[b][piece >> 3][4 * (piece & 7)][0]);
      }
    };
    // the pass's row scalars: lanes 0..31 of wave 0 copy LSE and D into
    // buffer b by DMA and work out the position and dQ offset ...
    int32_t npos = -1;
    int64_t noff = dq_trash;
    auto load_scalars = [&](int cc, int b) {
      if (kq == 0 && lane < kBwdPassRows) {
        bool ok;
        const int64_t hr = pass_row(cc, lane, lane_rq, lane_rh, ok);
        bwd_dma4(lse + hr, &sm.lse[b][0]);
        bwd_dma4(delta + hr, &sm.dlt[b][0]);
        const int qa = cc + lane_rq;
        npos = ok ? pos_base + sm.s_row[qa] : -1;
        noff = ok ? (((static_cast<int64_t>(sm.s_row[qa]) * H_kv + r) * topk + sm.s_slot[qa]) * G + lane_rh) *
                        kHeadDim
                  : dq_trash;
      }
    };
    // ... and store those two into the other buffer once every wave has
    // stored the previous pass's dQ (which reads that buffer's offsets)
    auto store_scalars = [&](int b) {
      if (kq == 0 && lane < kBwdPassRows) {
        sm.rpos[b][lane] = npos;
        sm.dqoff[b][lane] = noff;
      }
    };

    f32x4 acc_dv[8], acc_dk[8];                       // [dim tile]: lane column = dim, rows = keys 4qd + i
#pragma unroll
    for (int t = 0; t < 8; ++t) { acc_dv[t] = f32x4{}; acc_dk[t] = f32x4{}; }
    const int key = key0 + 16 * kq + c16;             // this lane's key in the C layout of S
    // dQ values of the previous pass, stored one pass late
    uint32_t dq_pend[2][4];
    int pend_buf = -1;
    auto store_dq = [&](int b) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool odd = c16 & 1;
          uint16_t* base = dq_buf + sm.dqoff[b][16 * t + 4 * qd + i] + (kHeadDim / NKW) * kq;
          if constexpr (DQU == 2) *reinterpret_cast<uint32_t*>(base + (odd ? 15 + c16 : c16)) = dq_pend[t][i];
          else if (!odd) *reinterpret_cast<uint32_t*>(base + c16) = dq_pend[t][i];
        }
    };

    issue_dma(0, 0);
    load_scalars(0, 0);
    store_scalars(0);
    int buf = 0;
    for (int c = 0; c < nq; c += qpw, buf ^= 1) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's copies for the pass have landed
      __syncthreads();                                // every wave's pieces, the pass's scalars; the
                                                      // previous pass is done with ds and the other buffer
      if (pend_buf >= 0) store_dq(pend_buf);
      const bool more = c + qpw < nq;
      if (more) {
        issue_dma(c + qpw, buf ^ 1);
        load_scalars(c + qpw, buf ^ 1);
      }
      const uint8_t* qb = reinterpret_cast<const uint8_t*>(&sm.qdo[buf][0][0][0]);
      const uint8_t* dob = reinterpret_cast<const uint8_t*>(&sm.qdo[buf][1][0][0]);

      // S = Q K^T, dP = dO V^T for this key slice
      f32x4 acc_s[2], acc_dp[2];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        acc_s[t] = f32x4{};
        acc_dp[t] = f32x4{};
        const int ra = 16 * t + c16;
#pragma unroll
        for (int st = 0; st < KS; ++st) {
          const int off = bwd_qrow_off(ra, 32 * st + 8 * qd);
          acc_s[t] = mfma16x16x32(*reinterpret_cast<const bf16x8*>(qb + off),
                                  *reinterpret_cast<const bf16x8*>(kbytes + bwd_qrow_off(16 * kq + c16, 32 * st + 8 * qd)),
                                  acc_s[t]);
          acc_dp[t] = mfma16x16x32(*reinterpret_cast<const bf16x8*>(dob + off),
                                   ld_bf16x8(&sm.v[16 * kq + c16][32 * st + 8 * qd]), acc_dp[t]);
        }
      }
      // P and dS in place: lane holds rows 16t + 4qd + i
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int prow = 16 * t + 4 * qd + i;
          const float l2 = sm.lse[buf][prow] * kLog2e;
          const bool vis = key <= sm.rpos[buf][prow] && l2 > -INFINITY;
          const float p = vis ? exp2_hw(acc_s[t][i] * scale_log2 - l2) : 0.f;
          acc_s[t][i] = p;
          acc_dp[t][i] = p * (acc_dp[t][i] - sm.dlt[buf][prow]);
        }
      // A operands of dV and dK: k index 8qd + 4t + i = row 16t + 4qd + i
      uint4 pw, sw;
      pw.x = pack_bf16x2(acc_s[0][0], acc_s[0][1]);
      pw.y = pack_bf16x2(acc_s[0][2], acc_s[0][3]);
      pw.z = pack_bf16x2(acc_s[1][0], acc_s[1][1]);
      pw.w = pack_bf16x2(acc_s[1][2], acc_s[1][3]);
      sw.x = pack_bf16x2(acc_dp[0][0], acc_dp[0][1]);
      sw.y = pack_bf16x2(acc_dp[0][2], acc_dp[0][3]);
      sw.z = pack_bf16x2(acc_dp[1][0], acc_dp[1][1]);
      sw.w = pack_bf16x2(acc_dp[1][2], acc_dp[1][3]);
      const bf16x8 pa = __builtin_bit_cast(bf16x8, pw);
      const bf16x8 sa = __builtin_bit_cast(bf16x8, sw);
      // dS to LDS as [row][key] for dQ
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          sm.ds[16 * t + 4 * qd + i][16 * kq + c16] = static_cast<uint16_t>(sw[2 * t + (i >> 1)] >> (16 * (i & 1)));
      __builtin_amdgcn_sched_barrier(0);
      // dV += P^T dO, dK += dS^T Q over the 32 rows (one k-step), 8 dim tiles;
      // B: rows 4qd .. 4qd + 3 and 16 + 4qd .. 16 + 4qd + 3 of dim 16t + c16
      // (lane j of a quarter points at row 4qd (+ 16) + j / 4, dims 16t + 4 (j % 4) ..)
      const int tr_row = 4 * qd + (c16 >> 2);
      const int tr_col = 4 * (c16 & 3);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int o0 = bwd_qrow_off(tr_row, 16 * t + tr_col), o1 = bwd_qrow_off(16 + tr_row, 16 * t + tr_col);
        const uint2 d0 = lds_tr4(dob + o0), d1 = lds_tr4(dob + o1);
        const uint2 q0 = lds_tr4(qb + o0), q1 = lds_tr4(qb + o1);
        acc_dv[t] = mfma16x16x32(pa, __builtin_bit_cast(bf16x8, make_uint4(d0.x, d0.y, d1.x, d1.y)), acc_dv[t]);
        acc_dk[t] = mfma16x16x32(sa, __builtin_bit_cast(bf16x8, make_uint4(q0.x, q0.y, q1.x, q1.y)), acc_dk[t]);
        if (t & 1) __builtin_amdgcn_sched_barrier(0);   // bound the operand reads in flight
      }
      __syncthreads();                                // dS of every key slice in LDS; every wave's
                                                      // store_dq of this pass has read the other buffer
      if (more) store_scalars(buf ^ 1);               // the next pass's positions and dQ offsets

      // dQ of the pass, dims (128 / NKW) kq + 16u + c16, over the block's keys;
      // B: keys 32ks + 8qd .. + 7 of that dim, read down K's column
      f32x4 acc_q[2][DQU];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < DQU; ++u) acc_q[t][u] = f32x4{};
#pragma unroll
      for (int u = 0; u < DQU; ++u) {
        const int n0 = (kHeadDim / NKW) * kq + 16 * u;
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
          const int krow = 32 * ks + 8 * qd + (c16 >> 2);
          const uint2 k0v = lds_tr4(kbytes + bwd_qrow_off(krow, n0 + tr_col));
          const uint2 k1v = lds_tr4(kbytes + bwd_qrow_off(krow + 4, n0 + tr_col));
          const bf16x8 kb8 = __builtin_bit_cast(bf16x8, make_uint4(k0v.x, k0v.y, k1v.x, k1v.y));
#pragma unroll
          for (int t = 0; t < 2; ++t)
            acc_q[t][u] = mfma16x16x32(ld_bf16x8(&sm.ds[16 * t + c16][32 * ks + 8 * qd]), kb8, acc_q[t][u]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      // bf16 partials of the pass's rows, stored at the start of the next pass
      // (rows without a query go to the trash row).  Two dQ tiles (4 waves):
      // lanes c16 and c16 ^ 1 swap values so that each stores one bf16 pair
      // (even lanes dims c16, c16 + 1 of tile 0; odd lanes dims c16 - 1, c16
      // of tile 1).  One tile (8 waves): even lanes store dims c16, c16 + 1.
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool odd = c16 & 1;
          if constexpr (DQU == 2) {
            const float v0 = acc_q[t][0][i], v1 = acc_q[t][1][i];
            const float mine = odd ? v1 : v0;
            const float other = __uint_as_float(xor_lane_u32<1>(__float_as_uint(odd ? v0 : v1)));
            dq_pend[t][i] = odd ? pack_bf16x2(other, mine) : pack_bf16x2(mine, other);
          } else {
            const float mine = acc_q[t][0][i];
            const float other = __uint_as_float(xor_lane_u32<1>(__float_as_uint(mine)));
            dq_pend[t][i] = pack_bf16x2(mine, other);
          }
        }
      pend_buf = buf;
    }
    // the last pass's dQ: its scalars stay valid until the next item's barrier
    if (pend_buf >= 0) store_dq(pend_buf);

    // item end: the item's dV / dK partial, [tensor][kq][reg][lane]
#pragma unroll
    for (int tensor = 0; tensor < 2; ++tensor) {
      const f32x4* acc = tensor == 0 ? acc_dv : acc_dk;
      float* dst = part + (static_cast<int64_t>(item) * 2 + tensor) * (NKW * 32 * 64) + kq * (32 * 64) + lane;
#pragma unroll
      for (int reg = 0; reg < 32; ++reg) dst[reg * 64] = acc[reg >> 2][reg & 3];
    }
  }
}

// Per tile: the sum of its item partials, in item order, added to the fp32
// accumulators of the block's keys.  bwd_reduce_split<BK>() CTAs per tile,
// one float4 of the partial per thread, so every tile streams its partials
// with independent loads.
template <int BK>
constexpr int bwd_reduce_split() { return bwd_part_floats<BK>() / (4 * 256); }
template <int BK>
__global__ __launch_bounds__(256) void bwd_tile_reduce_kernel(msa_seqs sq, const int64_t* __restrict__ blk_base,
                                                              const int32_t* __restrict__ item_off, int H_kv,
                                                              int64_t nbcap, const float* __restrict__ part,
                                                              float* __restrict__ dk_acc, float* __restrict__ dv_acc) {
  constexpr int NKW = bwd_waves<BK>();
  constexpr int kSplit = bwd_reduce_split<BK>();
  const int64_t tile = blockIdx.x / kSplit;
  const int32_t i0 = item_off[tile], i1 = item_off[tile + 1];
  if (i0 == i1) return;
  const int r = static_cast<int>(tile / nbcap);
  const int64_t gb = tile % nbcap;
  const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
  const SeqGeom g = seq_geom(sq, s);
  const int key0 = static_cast<int>(gb - blk_base[s]) * BK;
  const int c4 = (blockIdx.x % kSplit) * 256 + threadIdx.x;   // float4 of the partial
  const float4* p4 = reinterpret_cast<const float4*>(part) + c4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int32_t it = i0; it < i1; ++it) {
    const float4 x = p4[static_cast<int64_t>(it) * (bwd_part_floats<BK>() / 4)];
    acc.x += x.x;
    acc.y += x.y;
    acc.z += x.z;
    acc.w += x.w;
  }
  // partial layout [tensor][kq][reg][lane]: 4 consecutive lanes = 4 consecutive dims
  const int idx = 4 * c4;
  const int tensor = idx / (NKW * 32 * 64);
  const int kq = (idx / (32 * 64)) % NKW;
  const int reg = (idx / 64) & 31;
  const int ln = idx & 63;
  const int key = 16 * kq + 4 * (ln >> 4) + (reg & 3);
  const int dim = 16 * (reg >> 2) + (ln & 15);
  if (key0 + key >= g.kv_len) return;
  float4* dst = reinterpret_cast<float4*>((tensor == 0 ? dv_acc : dk_acc) +
                                          ((key_blocks(sq, g, s, BK).row(key0 / BK) + key) * H_kv + r) *
                                              static_cast<int64_t>(kHeadDim) + dim);
  float4 y = *dst;
  y.x += acc.x;
  y.y += acc.y;
  y.z += acc.z;
  y.w += acc.w;
  *dst = y;
}

// One wave per (row, group) of the chunk: dQ = scale x sum of the valid slots'
// partials, in slot order.
constexpr int kCombWaves = 4;

__global__ __launch_bounds__(64 * kCombWaves) void bwd_dq_combine_kernel(
    const int32_t* __restrict__ block_ids, msa_seqs sq, const int64_t* __restrict__ blk_base, int H_q, int H_kv,
    int BK, int topk, int64_t row0, int64_t nrows, const uint16_t* __restrict__ dq_buf, float scale,
    uint16_t* __restrict__ dq) {
  const int lane = lane_id();
  const int64_t pr = static_cast<int64_t>(blockIdx.x) * kCombWaves + threadIdx.x / kWave;
  if (pr >= nrows * H_kv) return;
  const int64_t rl = pr / H_kv;
  const int r = static_cast<int>(pr % H_kv);
  const int G = H_q / H_kv;
  const int64_t row = row0 + rl;
  int s;
  const int p = row_position(sq, row, &s);
  const int32_t* ids = block_ids + (row * H_kv + r) * topk;
  const int E = G * kHeadDim;                         // elements of one slot
  const uint16_t* src = dq_buf + pr * topk * static_cast<int64_t>(E);
  uint16_t* dst = dq + (row * H_q + static_cast<int64_t>(r) * G) * kHeadDim;
  // slot validity, one slot per lane; the valid slots' partials are then
  // read 8 at a time (in slot order) so their loads are in flight together
  const bool mine = lane < topk && incidence_ok(ids[lane], p, BK, blk_base, s);
  const uint64_t valid = __ballot(mine);
  for (int c8 = lane; c8 < E / 8; c8 += kWave) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    uint64_t vm = valid;
    // batches of 8 valid slots in slot order; batch n + 1's loads are issued
    // before batch n is accumulated (two in flight; the sum order is unchanged)
    constexpr int kBatch = 8;
    auto take = [&](int (&js)[kBatch]) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        js[u] = vm != 0ull ? __ffsll(static_cast<unsigned long long>(vm)) - 1 : -1;
        vm &= vm - 1;
      }
    };
    auto issue = [&](const int (&js)[kBatch], u32x4 (&w)[kBatch]) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
        w[u] = load_raw(src + static_cast<int64_t>(js[u] >= 0 ? js[u] : js[0]) * E + 8 * c8);
    };
    auto accumulate = [&](const int (&js)[kBatch], const u32x4 (&w)[kBatch]) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        if (js[u] < 0) break;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += __uint_as_float(w[u][e] << 16);
          acc[2 * e + 1] += __uint_as_float(w[u][e] & 0xFFFF0000u);
        }
      }
    };
    int ja[kBatch], jb[kBatch];
    u32x4 wa[kBatch], wb[kBatch];
    take(ja);
    if (ja[0] >= 0) issue(ja, wa);
    while (ja[0] >= 0) {
      take(jb);
      if (jb[0] >= 0) issue(jb, wb);
      accumulate(ja, wa);
      if (jb[0] < 0) break;
      take(ja);
      if (ja[0] >= 0) issue(ja, wa);
      accumulate(jb, wb);
    }
    uint4 o;
    o.x = pack_bf16x2(acc[0] * scale, acc[1] * scale);
    o.y = pack_bf16x2(acc[2] * scale, acc[3] * scale);
    o.z = pack_bf16x2(acc[4] * scale, acc[5] * scale);
    o.w = pack_bf16x2(acc[6] * scale, acc[7] * scale);
    *reinterpret_cast<uint4*>(dst + 8 * c8) = o;
  }
}

__global__ __launch_bounds__(256) void bwd_kv_convert_kernel(const float* __restrict__ dk_acc,
                                                             const float* __restrict__ dv_acc, int64_t n4, float scale,
                                                             uint16_t* __restrict__ dk, uint16_t* __restrict__ dv) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n4;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    const f32x4 a = reinterpret_cast<const f32x4*>(dk_acc)[i];
    const f32x4 b = reinterpret_cast<const f32x4*>(dv_acc)[i];
    uint2 wa, wb;
    wa.x = pack_bf16x2(a[0] * scale, a[1] * scale);
    wa.y = pack_bf16x2(a[2] * scale, a[3] * scale);
    wb.x = pack_bf16x2(b[0], b[1]);
    wb.y = pack_bf16x2(b[2], b[3]);
    reinterpret_cast<uint2*>(dk)[i] = wa;
    reinterpret_cast<uint2*>(dv)[i] = wb;
  }
}

// ---------------------------------------------------------------- host plan
struct BwdPlan {
  int BK;                                             // key block size (64 or 128)
  int64_t nbcap, ntile, chunk_rows, max_items;
  int nscan;
  size_t off_blk_base, off_cnt, off_tile_off, off_item_off, off_blk_tot, off_delta, off_dk, off_dv, off_handles,
      off_tpos, off_dq, off_part, total;
};

constexpr size_t kDefaultBwdBytes = size_t(64) << 30;

void bwd_layout(BwdPlan& pl, const msa_seqs* seqs, int H_q, int H_kv, int topk) {
  using msa_host::align_up;
  size_t o = 0;
  pl.off_blk_base = o; o = align_up(o + sizeof(int64_t) * (seqs->num_seqs + 1), 256);
  pl.off_cnt = o;      o = align_up(o + sizeof(int32_t) * (pl.ntile + kWorkCounters), 256);
  pl.off_tile_off = o; o = align_up(o + sizeof(int32_t) * (pl.ntile + 1), 256);
  pl.off_item_off = o; o = align_up(o + sizeof(int32_t) * (pl.ntile + 1), 256);
  pl.off_blk_tot = o;  o = align_up(o + sizeof(int32_t) * 2 * pl.nscan, 256);
  pl.off_delta = o;    o = align_up(o + sizeof(float) * static_cast<size_t>(seqs->total_q_rows) * H_q, 256);
  const size_t kv_floats = static_cast<size_t>(seqs->total_kv_rows) * H_kv * kHeadDim;
  pl.off_dk = o;       o = align_up(o + sizeof(float) * kv_floats, 256);
  pl.off_dv = o;       o = align_up(o + sizeof(float) * kv_floats, 256);
  const size_t inc = static_cast<size_t>(pl.chunk_rows) * H_kv * topk;
  pl.max_items = pl.ntile + static_cast<int64_t>((inc + kItemQueries - 1) / kItemQueries);
  pl.off_handles = o;  o = align_up(o + sizeof(uint32_t) * inc, 256);
  pl.off_tpos = o;     o = align_up(o + sizeof(int32_t) * inc, 256);
  pl.off_dq = o;       o = align_up(o + sizeof(uint16_t) * (inc * (H_q / H_kv) + 1) * kHeadDim, 256);   // + trash row
  pl.off_part = o;     o = align_up(o + sizeof(float) * static_cast<size_t>(pl.max_items) * 2 * pl.BK * kHeadDim, 256);
  pl.total = o;
}

int make_bwd_plan(const msa_seqs* seqs, int H_q, int H_kv, int BK, int topk, size_t budget, BwdPlan* pl) {
  pl->BK = BK;
  const int64_t nb = (seqs->max_kv_len + BK - 1) / BK;
  pl->nbcap = static_cast<int64_t>(seqs->num_seqs) * (nb > 0 ? nb : 1);
  pl->ntile = static_cast<int64_t>(H_kv) * pl->nbcap;
  if (pl->ntile >= (int64_t(1) << 31) - 1) return MSA_ERR_UNSUPPORTED;
  pl->nscan = static_cast<int>((pl->ntile + kScanPerBlock - 1) / kScanPerBlock);
  if (pl->nscan > 1024 * 64) return MSA_ERR_UNSUPPORTED;
  const int64_t max_rows =
      std::min(kMaxChunkRows, ((int64_t(1) << 31) - 1) / (static_cast<int64_t>(H_kv) * topk));
  int64_t rows = std::max<int64_t>(1, seqs->total_q_rows);
  rows = std::min(rows, max_rows);
  pl->chunk_rows = rows;
  bwd_layout(*pl, seqs, H_q, H_kv, topk);
  if (pl->total > budget) {
    // bytes per chunk row, from the layout at one row and at two rows
    pl->chunk_rows = 1;
    bwd_layout(*pl, seqs, H_q, H_kv, topk);
    const size_t one = pl->total;
    if (one > budget) return MSA_ERR_WORKSPACE;
    pl->chunk_rows = 2;
    bwd_layout(*pl, seqs, H_q, H_kv, topk);
    const size_t per_row = pl->total - one + 1024;
    rows = 1 + static_cast<int64_t>((budget - one) / per_row);
    pl->chunk_rows = std::min(rows, std::min<int64_t>(max_rows, std::max<int64_t>(1, seqs->total_q_rows)));
    bwd_layout(*pl, seqs, H_q, H_kv, topk);
    while (pl->total > budget && pl->chunk_rows > 1) {
      pl->chunk_rows = std::max<int64_t>(1, pl->chunk_rows * 7 / 8);
      bwd_layout(*pl, seqs, H_q, H_kv, topk);
    }
    if (pl->total > budget) return MSA_ERR_WORKSPACE;
  }
  return MSA_OK;
}

int validate_bwd(const msa_seqs* seqs, int H_q, int H_kv, int head_dim, int BK, int topk) {
  int st = msa_host::validate_seqs(seqs);
  if (st != MSA_OK) return st;
  if (H_q < 1 || H_kv < 1 || head_dim < 1 || BK < 1 || topk < 1) return MSA_ERR_INVALID;
  if (H_q % H_kv != 0) return MSA_ERR_INVALID;
  if (head_dim != kHeadDim || (BK != 64 && BK != 128)) return MSA_ERR_UNSUPPORTED;
  if (topk > 64 || H_q / H_kv > 16 || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (seqs->total_q_rows * H_kv >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  return msa_host::check_paged(seqs, BK, true);
}

template <int BK>
int run_backward(const void* q, const void* k, const void* v, const void* o, const float* lse, const void* d_o,
                 const int32_t* block_ids, const msa_seqs* seqs, int H_q, int H_kv, int topk, float softmax_scale,
                 void* d_q, void* d_k, void* d_v, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st;
  BwdPlan pl;
  st = make_bwd_plan(seqs, H_q, H_kv, BK, topk, workspace_bytes, &pl);
  if (st != MSA_OK) return st;
  if (!workspace || workspace_bytes < pl.total) return MSA_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  auto* blk_base = reinterpret_cast<int64_t*>(ws + pl.off_blk_base);
  auto* cnt = reinterpret_cast<int32_t*>(ws + pl.off_cnt);
  auto* tile_off = reinterpret_cast<int32_t*>(ws + pl.off_tile_off);
  auto* item_off = reinterpret_cast<int32_t*>(ws + pl.off_item_off);
  auto* blk_tot = reinterpret_cast<int32_t*>(ws + pl.off_blk_tot);
  auto* delta = reinterpret_cast<float*>(ws + pl.off_delta);
  auto* dk_acc = reinterpret_cast<float*>(ws + pl.off_dk);
  auto* dv_acc = reinterpret_cast<float*>(ws + pl.off_dv);
  auto* handles = reinterpret_cast<uint32_t*>(ws + pl.off_handles);
  auto* tpos = reinterpret_cast<int32_t*>(ws + pl.off_tpos);
  auto* dq_buf = reinterpret_cast<uint16_t*>(ws + pl.off_dq);
  auto* part = reinterpret_cast<float*>(ws + pl.off_part);
  const msa_seqs sq = *seqs;
  const int64_t kv_floats = seqs->total_kv_rows * H_kv * static_cast<int64_t>(kHeadDim);
  const unsigned zero_blocks = static_cast<unsigned>(std::min<int64_t>((kv_floats + 255) / 256, 8192));

  msa_prof::launch("kvo_block_base_kernel", kvo_block_base_kernel, dim3(1), dim3(256), 0, stream, sq, BK, blk_base);
  msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                   reinterpret_cast<int32_t*>(dk_acc), kv_floats, 0);
  msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                   reinterpret_cast<int32_t*>(dv_acc), kv_floats, 0);
  const int64_t pairs = seqs->total_q_rows * H_q;
  if (pairs > 0)
    msa_prof::launch("bwd_delta_kernel", bwd_delta_kernel, dim3(static_cast<unsigned>((pairs * 16 + 255) / 256)),
                     dim3(256), 0, stream, static_cast<const uint16_t*>(o), static_cast<const uint16_t*>(d_o), pairs,
                     delta);
  static std::atomic<int> ctas {0};
  const int nctas = persistent_ctas(bwd_kvo_kernel<BK>, bwd_threads<BK>(), &ctas);
  const float sl2 = softmax_scale * kLog2e;
  for (int64_t r0 = 0; r0 < seqs->total_q_rows; r0 += pl.chunk_rows) {
    const int64_t nr = std::min<int64_t>(pl.chunk_rows, seqs->total_q_rows - r0);
    build_reverse_index(block_ids, sq, blk_base, H_kv, BK, topk, pl.nbcap, pl.ntile, pl.nscan, r0, nr, cnt,
                        tile_off, item_off, blk_tot, tpos, handles, stream, true);
    msa_prof::launch("bwd_kvo_kernel", bwd_kvo_kernel<BK>, dim3(nctas), dim3(bwd_threads<BK>()), 0, stream,
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(v), static_cast<const uint16_t*>(d_o), lse,
                     static_cast<const float*>(delta), sq, static_cast<const int64_t*>(blk_base),
                     static_cast<const int32_t*>(tile_off), static_cast<const int32_t*>(item_off),
                     static_cast<const uint32_t*>(handles), H_q, H_kv, topk, pl.nbcap, r0, sl2, dq_buf,
                     static_cast<int64_t>(pl.chunk_rows) * H_kv * topk * (H_q / H_kv) * kHeadDim, part,
                     cnt + pl.ntile);
    msa_prof::launch("bwd_tile_reduce_kernel", bwd_tile_reduce_kernel<BK>,
                     dim3(static_cast<unsigned>(pl.ntile * bwd_reduce_split<BK>())), dim3(256), 0, stream, sq,
                     static_cast<const int64_t*>(blk_base), static_cast<const int32_t*>(item_off), H_kv, pl.nbcap,
                     static_cast<const float*>(part), dk_acc, dv_acc);
    msa_prof::launch("bwd_dq_combine_kernel", bwd_dq_combine_kernel,
                     dim3(static_cast<unsigned>((nr * H_kv + kCombWaves - 1) / kCombWaves)), dim3(64 * kCombWaves),
                     0, stream, block_ids, sq, static_cast<const int64_t*>(blk_base), H_q, H_kv, BK, topk, r0, nr,
                     static_cast<const uint16_t*>(dq_buf), softmax_scale, static_cast<uint16_t*>(d_q));
  }
  if (kv_floats > 0)
    msa_prof::launch("bwd_kv_convert_kernel", bwd_kv_convert_kernel, dim3(zero_blocks), dim3(256), 0, stream,
                     static_cast<const float*>(dk_acc), static_cast<const float*>(dv_acc), kv_floats / 4,
                     softmax_scale, static_cast<uint16_t*>(d_k), static_cast<uint16_t*>(d_v));
  return msa_host::launch_status();
}

}  // namespace

extern "C" size_t msa_sparse_attn_backward_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                                         int head_dim, int block_size, int topk) {
  if (validate_bwd(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk) != MSA_OK) return 0;
  BwdPlan pl;
  if (make_bwd_plan(seqs, num_q_heads, num_kv_heads, block_size, topk, kDefaultBwdBytes, &pl) != MSA_OK) {
    if (make_bwd_plan(seqs, num_q_heads, num_kv_heads, block_size, topk, ~size_t(0) >> 1, &pl) != MSA_OK) return 0;
    pl.chunk_rows = 1;
    bwd_layout(pl, seqs, num_q_heads, num_kv_heads, topk);
  }
  return pl.total;
}

extern "C" int msa_sparse_attn_backward(const void* q, const void* k, const void* v, const void* o, const float* lse,
                                        const void* d_o, const int32_t* block_ids, const msa_seqs* seqs,
                                        int num_q_heads, int num_kv_heads, int head_dim, int block_size, int topk,
                                        float softmax_scale, void* d_q, void* d_k, void* d_v, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  const int H_q = num_q_heads, H_kv = num_kv_heads;
  int st = validate_bwd(seqs, H_q, H_kv, head_dim, block_size, topk);
  if (st != MSA_OK) return st;
  if (!q || !k || !v || !o || !lse || !d_o || !block_ids || !d_q || !d_k || !d_v) return MSA_ERR_INVALID;
  if (seqs->total_q_rows == 0 && seqs->total_kv_rows == 0) return MSA_OK;
  if (block_size == 64)
    return run_backward<64>(q, k, v, o, lse, d_o, block_ids, seqs, H_q, H_kv, topk, softmax_scale, d_q, d_k, d_v,
                            workspace, workspace_bytes, stream);
  return run_backward<128>(q, k, v, o, lse, d_o, block_ids, seqs, H_q, H_kv, topk, softmax_scale, d_q, d_k, d_v,
                           workspace, workspace_bytes, stream);
}
