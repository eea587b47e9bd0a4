// Prefill Main Branch of MSA on gfx950, key-block-outer.
//
// The sparse-attention equation of Sec. 3.1 restricted to one selected block
// is an ordinary softmax attention over <= B_k keys.  Iterating queries on the
// outside would fetch a 2 x B_k x d_h K/V block per (query, group, block)
// incidence; iterating key blocks on the outside fetches every block once and
// gathers the queries that picked it, so each incidence costs a Q gather, a
// partial write and a partial read instead (Sec. 4.2, the Q-outer / KV-outer
// IO comparison).  The partial of each incidence is normalised locally and
// merged afterwards with the log-sum-exp rule of Sec. 4.2 ("Two-phase
// forward"), so no atomics touch O.
//
// Per chunk of query rows (the partial buffer is k x rows x H_q x d_h):
//   kvo_count, kvo_scan*, kvo_fill (kvo_index.h)
//                the reverse index: per tile (group r, key block) the
//                (row, slot) handles that selected it, cut into work items
//   kvo_attn     persistent CTAs; a work item is <= kItemQueries queries of one
//                tile.  K and V^T of the block are staged in LDS once per tile,
//                each wave gathers 32 (query, head) rows, computes S^T = K Q^T
//                and O^T = V^T P^T with MFMA 32x32x16 and writes the bf16
//                partial and its LSE into the incidence's slot.
//   kvo_combine  O and LSE per (row, head) from the valid slots.
#include <algorithm>

#include "kvo_index.h"

namespace {

using namespace msa;

// waves per attention CTA: 4 for B_k 64; B_k 128 stages 88 KB of K / Vt per
// CTA, so one CTA fills a CU and 8 waves keep 2 per SIMD
template <int BK>
constexpr int kvo_waves() { return BK == 128 ? 8 : 4; }

// ---------------------------------------------------------------- attention
template <int BK>
struct KvoSmem {
  uint16_t k[BK][kHeadDim + 8];     // K block, row-major (+16 B pad per row)
  uint16_t vt[kHeadDim][BK + 4];    // V block transposed (+8 B pad per row)
  uint16_t ost[kvo_waves<BK>()][32][64];   // per wave: one 64-dim half of 32 partial rows (bf16),
                                    // 16-byte units XOR-swizzled by row & 7
};

// T: element type of Q, K and V (uint16_t = bf16 bits, uint8_t = e4m3 bits);
// o_scale multiplies the partial O (the V dequantisation scale for e4m3).
template <int BK, typename T>
__global__ __launch_bounds__(64 * kvo_waves<BK>(), BK == 128 ? 1 : 2) void kvo_attn_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, msa_seqs sq,
    const int64_t* __restrict__ blk_base, const int32_t* __restrict__ tile_off,
    const int32_t* __restrict__ item_off, const uint32_t* __restrict__ handles, int H_q, int H_kv, int topk,
    int64_t nbcap, int64_t row0, float scale_log2, float o_scale, uint16_t* __restrict__ o_buf,
    float* __restrict__ lse_buf, int32_t* __restrict__ next_item) {
  static_assert(kItemQueries <= 64 * kvo_waves<BK>(), "every thread loads at most one handle of an item");
  __shared__ KvoSmem<BK> sm;
  __shared__ int32_t s_claim;
  __shared__ int32_t s_row[kItemQueries];     // query row inside the chunk
  __shared__ int32_t s_pos[kItemQueries];     // its absolute position
  __shared__ int32_t s_slot[kItemQueries];    // slot of this block in the row's id list
  constexpr int MT = BK / 32;                 // 32-key tiles of S^T
  constexpr int KS = kHeadDim / 16;           // k-steps of S^T = K Q^T
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int n = lane & 31, h = lane >> 5;
  const int G = H_q / H_kv;
  const int qpw = 32 / G;                     // queries per wave pass
  const int jq = n / G, hh = n % G;           // this lane's (query within pass, head)
  const bool lane_row = n < qpw * G;
  const int64_t ntile = static_cast<int64_t>(H_kv) * nbcap;
  const int32_t total_items = item_off[ntile];
  const int64_t kv_stride = static_cast<int64_t>(H_kv) * kHeadDim;
  int64_t staged = -1;
  constexpr int kThr = 64 * kvo_waves<BK>();
  constexpr int KI = BK * (kHeadDim / 8) / kThr;          // K pieces per thread per block
  static_assert(KI * kThr == BK * (kHeadDim / 8) && (BK / 4) * (kHeadDim / 8) == kThr, "staging map");
  // B_k 64: the next item is claimed one ahead and its tile's K / V rows are
  // loaded into registers while the current item is computed (B_k 128 has no
  // registers to spare and stages after the barrier)
  constexpr bool kPrefetch = BK == 64;
  Raw<T> pk[KI], pv[4];
  int64_t pf_tile = -1;
  // K / V rows of `tl` into registers; keys at or past the sequence end read as zero
  auto load_tile = [&](int64_t tl) {
    const int r_ = static_cast<int>(tl / nbcap);
    const int64_t gb_ = tl % nbcap;
    const int s_ = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb_));
    const SeqGeom g_ = seq_geom(sq, s_);
    const int key0_ = static_cast<int>(gb_ - blk_base[s_]) * BK;
    const int64_t brow = key_blocks(sq, g_, s_, BK).row(static_cast<int>(gb_ - blk_base[s_]));
    const T* kb = k + brow * kv_stride + static_cast<int64_t>(r_) * kHeadDim;
    const T* vb = v + brow * kv_stride + static_cast<int64_t>(r_) * kHeadDim;
#pragma unroll
    for (int i = 0; i < KI; ++i) {
      const int c = threadIdx.x + kThr * i;
      const int key = c / (kHeadDim / 8), dg = c % (kHeadDim / 8);
      pk[i] = key0_ + key < g_.kv_len ? load_raw(kb + static_cast<int64_t>(key) * kv_stride + 8 * dg) : Raw<T>{};
    }
    {
      const int key4 = threadIdx.x / (kHeadDim / 8), dg = threadIdx.x % (kHeadDim / 8);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = 4 * key4 + j;
        pv[j] = key0_ + key < g_.kv_len ? load_raw(vb + static_cast<int64_t>(key) * kv_stride + 8 * dg) : Raw<T>{};
      }
    }
  };
  // registers to LDS: K row-major, V transposed
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KI; ++i) {
      const int c = threadIdx.x + kThr * i;
      const int key = c / (kHeadDim / 8), dg = c % (kHeadDim / 8);
      *reinterpret_cast<uint4*>(&sm.k[key][8 * dg]) = __builtin_bit_cast(uint4, widen(pk[i]));
    }
    const int key4 = threadIdx.x / (kHeadDim / 8), dg = threadIdx.x % (kHeadDim / 8);
    uint4 rows[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) rows[j] = __builtin_bit_cast(uint4, widen(pv[j]));
    const uint16_t* e0 = reinterpret_cast<const uint16_t*>(&rows[0]);
    const uint16_t* e1 = reinterpret_cast<const uint16_t*>(&rows[1]);
    const uint16_t* e2 = reinterpret_cast<const uint16_t*>(&rows[2]);
    const uint16_t* e3 = reinterpret_cast<const uint16_t*>(&rows[3]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint2 w;
      w.x = static_cast<uint32_t>(e0[e]) | (static_cast<uint32_t>(e1[e]) << 16);
      w.y = static_cast<uint32_t>(e2[e]) | (static_cast<uint32_t>(e3[e]) << 16);
      *reinterpret_cast<uint2*>(&sm.vt[8 * dg + e][4 * key4]) = w;
    }
  };

  int32_t item = blockIdx.x;
  int32_t nxt = 0;
  if (kPrefetch && item < total_items) nxt = claim_next_item(next_item, &s_claim);
  while (item < total_items) {
    const int64_t tile = upper_index(item_off, ntile + 1, item);
    const int32_t h0 = tile_off[tile] + (item - item_off[tile]) * kItemQueries;
    const int32_t nq = min(tile_off[tile + 1] - h0, kItemQueries);
    const int r = static_cast<int>(tile / nbcap);
    const int64_t gb = tile % nbcap;
    const int s = static_cast<int>(upper_index(blk_base, sq.num_seqs + 1, gb));
    const SeqGeom g = seq_geom(sq, s);
    const int key0 = static_cast<int>(gb - blk_base[s]) * BK;

    __syncthreads();                          // the previous item is finished with LDS
    if (static_cast<int>(threadIdx.x) < nq) {
      const uint32_t hd = handles[h0 + threadIdx.x];
      const int32_t rl = static_cast<int32_t>(hd >> 6);
      s_row[threadIdx.x] = rl;
      s_slot[threadIdx.x] = static_cast<int32_t>(hd & 63u);
      // every query of the tile belongs to sequence s
      s_pos[threadIdx.x] = g.kv_len - g.q_rows + static_cast<int>(row0 + rl - g.q_begin);
    }
    if (tile != staged) {
      if (pf_tile != tile) load_tile(tile);
      store_tile();
      staged = tile;
    }
    pf_tile = -1;
    if constexpr (kPrefetch) {
      if (nxt < total_items) {
        const int64_t ntl = upper_index(item_off, ntile + 1, nxt);
        if (ntl != tile) {
          load_tile(ntl);
          pf_tile = ntl;
        }
      }
    }
    __syncthreads();

    // passes of qpw queries x G heads = 32 rows per wave; Q of the next pass is
    // requested before the current pass computes.
    const int stride = kvo_waves<BK>() * qpw;
    int c = wave * qpw;
    Raw<T> bq[KS];                            // raw Q elements, widened at the MFMA
    auto load_q = [&](int cc, Raw<T>* dst) {
      const int qi = cc + jq;
      const bool ok = lane_row && qi < nq;
      const int64_t row = row0 + (ok ? s_row[qi] : 0);
      // k-step st: lane half h supplies dims 16*st + 8h .. +8 (32 contiguous bytes per row per load)
      const T* qrow = q + (row * H_q + static_cast<int64_t>(r) * G + hh) * kHeadDim + 8 * h;
#pragma unroll
      for (int st = 0; st < KS; ++st) dst[st] = ok ? load_raw(qrow + 16 * st) : Raw<T>{};
    };
    if (c < nq) load_q(c, bq);
    for (; c < nq; c += stride) {
      // B_k 64: the next pass's Q is requested now (unconditional: no wait on it
      // below); B_k 128 leaves latency to the second wave on the SIMD
      Raw<T> bq_next[KS];
      if constexpr (BK == 64) load_q(c + stride < nq ? c + stride : c, bq_next);
      const int qi = c + jq;
      const bool valid = lane_row && qi < nq;
      const int p = valid ? s_pos[qi] : -1;

      // S^T = K Q^T: lane (n, h) holds keys 32i + 8(e/4) + 4h + e%4 of row n
      f32x16 acc_s[MT];
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        acc_s[i] = f32x16{};
        const uint16_t* kr = &sm.k[32 * i + n][8 * h];
#pragma unroll
        for (int st = 0; st < KS; ++st)
          acc_s[i] = mfma32x32x16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kr + 16 * st)),
                                  widen_bf16x8(bq[st]), acc_s[i]);
        __builtin_amdgcn_sched_barrier(0);    // bound how far LDS operand reads are hoisted
      }
      float m = -INFINITY;
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
          float z = acc_s[i][e] * scale_log2;
          z = key <= p ? z : -INFINITY;
          acc_s[i][e] = z;
          m = fmaxf(m, z);
        }
      m = fmaxf(m, __shfl_xor(m, 32));
      const float mm = m == -INFINITY ? 0.f : m;
      float l = 0.f;
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float pe = exp2_hw(acc_s[i][e] - mm);
          acc_s[i][e] = pe;
          l += pe;
        }
      l += __shfl_xor(l, 32);

      // P in bf16 as the B operand of O^T = V^T P^T: k-step u covers keys
      // 32(u/2) + 16(u%2) + {4h + e, 8 + 4h + e}; the lane's P values for it
      // are acc_s[u/2][8(u%2) .. 8(u%2)+7].
      bf16x8 bp[BK / 16];
#pragma unroll
      for (int u = 0; u < BK / 16; ++u) {
        uint4 pw;
        const int i = u >> 1, e0 = 8 * (u & 1);
        pw.x = pack_bf16x2(acc_s[i][e0 + 0], acc_s[i][e0 + 1]);
        pw.y = pack_bf16x2(acc_s[i][e0 + 2], acc_s[i][e0 + 3]);
        pw.z = pack_bf16x2(acc_s[i][e0 + 4], acc_s[i][e0 + 5]);
        pw.w = pack_bf16x2(acc_s[i][e0 + 6], acc_s[i][e0 + 7]);
        bp[u] = __builtin_bit_cast(bf16x8, pw);
      }
      const bool empty = !(l > 0.f);
      const float inv_l = empty ? 0.f : o_scale / l;
      // partial slot of this incidence: [row][group][slot][head][d]
      const int64_t prow = valid ? ((static_cast<int64_t>(s_row[qi]) * H_kv + r) * topk + s_slot[qi]) * G + hh : 0;
      // two halves of d (64 dims = 2 tiles each) keep 32 accumulators live
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        __builtin_amdgcn_sched_barrier(0);
        f32x16 acc_o[2];
        acc_o[0] = f32x16{};
        acc_o[1] = f32x16{};
#pragma unroll
        for (int u = 0; u < BK / 16; ++u) {
          const int kbase = 32 * (u >> 1) + 16 * (u & 1) + 4 * h;
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2) {
            const uint16_t* vr = &sm.vt[32 * (2 * half + t2) + n][kbase];
            const uint2 lo = *reinterpret_cast<const uint2*>(vr);
            const uint2 hi2 = *reinterpret_cast<const uint2*>(vr + 8);
            uint4 w;
            w.x = lo.x; w.y = lo.y; w.z = hi2.x; w.w = hi2.y;
            acc_o[t2] = mfma32x32x16(__builtin_bit_cast(bf16x8, w), bp[u], acc_o[t2]);
          }
        }
        // O^T tile t: lane (n, h) holds d = 32t + 8(e/4) + 4h + e%4 of row n.
        // Stage the half in LDS, then each store writes 8 rows x 128 B.
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
          for (int e4 = 0; e4 < 4; ++e4) {
            uint2 w;
            w.x = pack_bf16x2(acc_o[t2][4 * e4 + 0] * inv_l, acc_o[t2][4 * e4 + 1] * inv_l);
            w.y = pack_bf16x2(acc_o[t2][4 * e4 + 2] * inv_l, acc_o[t2][4 * e4 + 3] * inv_l);
            *reinterpret_cast<uint2*>(&sm.ost[wave][n][(32 * t2 + 8 * e4 + 4 * h) ^ ((n & 7) << 3)]) = w;
          }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int pass = 0; pass < 4; ++pass) {
          const int srow = 8 * pass + (lane >> 3);        // staged row = lane column n of its pass
          const int seg = lane & 7;                       // 16-byte segment of the 128-byte half row
          const int sq_i = c + srow / G;
          if (srow < qpw * G && sq_i < nq) {
            const int64_t prow_s =
                ((static_cast<int64_t>(s_row[sq_i]) * H_kv + r) * topk + s_slot[sq_i]) * G + (srow % G);
            // nontemporal: the combine reads the partials only after the
            // whole chunk, so caching them only evicts Q rows and K/V tiles
            __builtin_nontemporal_store(
                *reinterpret_cast<const u32x4*>(&sm.ost[wave][srow][(8 * seg) ^ ((srow & 7) << 3)]),
                reinterpret_cast<u32x4*>(o_buf + prow_s * kHeadDim + 64 * half + 8 * seg));
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      }
      if (valid && h == 0) __builtin_nontemporal_store(empty ? -INFINITY : (mm + __log2f(l)) * kLn2, lse_buf + prow);
      if constexpr (BK == 64) {
#pragma unroll
        for (int st = 0; st < KS; ++st) bq[st] = bq_next[st];
      } else if (c + stride < nq) {
        load_q(c + stride, bq);
      }
    }
    if constexpr (kPrefetch) {
      item = nxt;
      if (item < total_items) nxt = claim_next_item(next_item, &s_claim);
    } else {
      item = claim_next_item(next_item, &s_claim);
    }
  }
}

// ---------------------------------------------------------------- combine
// One wave per (row, group) of the chunk: lane j reads slot j's LSEs, the
// per-head weights go through LDS, and each lane accumulates 2G of the 128
// dims of one of the group's G heads over the valid slots.
constexpr int kCombineWaves = 4;

template <int PER>
__global__ __launch_bounds__(64 * kCombineWaves) void kvo_combine_kernel(
    const int32_t* __restrict__ block_ids, msa_seqs sq, const int64_t* __restrict__ blk_base, int H_q, int H_kv,
    int BK, int topk, int64_t row0, int64_t nrows, const uint16_t* __restrict__ o_buf,
    const float* __restrict__ lse_buf, uint16_t* __restrict__ o, float* __restrict__ lse) {
  __shared__ float s_w[kCombineWaves][64][17];        // weight of slot j for head hh (G <= 16)
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  int64_t pr = static_cast<int64_t>(blockIdx.x) * kCombineWaves + wave;   // (row, group) pair
  const bool active = pr < nrows * H_kv;
  if (!active) pr = 0;                               // computes a row it does not store
  const int64_t rl = pr / H_kv;
  const int r = static_cast<int>(pr % H_kv);
  const int G = H_q / H_kv;
  const int64_t row = row0 + rl;
  int s;
  const int p = row_position(sq, row, &s);
  const int32_t* ids = block_ids + (row * H_kv + r) * topk;
  const bool valid = lane < topk && incidence_ok(ids[lane], p, BK, blk_base, s);
  const float* lrow = lse_buf + (rl * H_kv + r) * static_cast<int64_t>(topk) * G;
  // per head: max and sum over the valid slots (lane j = slot j)
  float tot[16];
#pragma unroll
  for (int hh = 0; hh < 16; ++hh) {
    tot[hh] = -INFINITY;
    if (hh >= G) continue;
    const float x = valid ? lrow[lane * G + hh] : -INFINITY;
    float a = x;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) a = fmaxf(a, __shfl_xor(a, off));
    float e = (valid && a > -INFINITY && x > -INFINITY) ? exp2f((x - a) * kLog2e) : 0.f;
    float sum = e;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
    const float t = a > -INFINITY ? a + __logf(sum) : -INFINITY;
    tot[hh] = t;
    s_w[wave][lane][hh] = (valid && x > -INFINITY && t > -INFINITY) ? exp2f((x - t) * kLog2e) : 0.f;
  }
  __syncthreads();
  // PER dims per lane: 8 for G <= 4, 16 for G <= 8, 32 for G <= 16 (a
  // multiple of the 16-byte loads); lane covers head hh, dims [dd, dd + PER);
  // lanes past G * 128 / PER idle.
  constexpr int E8 = PER / 8;                        // 16-byte loads per slot
  constexpr int NB = PER == 32 ? 2 : 4;              // slots per batch
  const int lanes_per_head = kHeadDim / PER;
  const bool lane_on = lane < G * lanes_per_head;
  const int hh = lane_on ? lane / lanes_per_head : 0;
  const int dd = (lane % lanes_per_head) * PER;
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  const uint16_t* obase = o_buf + ((rl * H_kv + r) * static_cast<int64_t>(topk)) * G * kHeadDim +
                          static_cast<int64_t>(hh) * kHeadDim + dd;
  // valid slots in batches of NB, ascending; batch n + 1's partial loads are
  // issued before batch n is accumulated (two batches in flight)
  uint64_t vmask = __ballot(valid);
  auto take = [&](int (&js)[NB]) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      js[u] = vmask != 0ull ? __ffsll(static_cast<unsigned long long>(vmask)) - 1 : -1;
      vmask &= vmask - 1;
    }
  };
  auto issue = [&](const int (&js)[NB], u32x4 (&x)[NB][E8]) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const uint16_t* src = obase + static_cast<int64_t>(js[u] >= 0 ? js[u] : js[0]) * G * kHeadDim;
#pragma unroll
      for (int e8 = 0; e8 < E8; ++e8) x[u][e8] = *reinterpret_cast<const u32x4*>(src + 8 * e8);
    }
  };
  auto accumulate = [&](const int (&js)[NB], const u32x4 (&x)[NB][E8]) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const float w = js[u] >= 0 ? s_w[wave][js[u]][hh] : 0.f;
#pragma unroll
      for (int e8 = 0; e8 < E8; ++e8)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[8 * e8 + 2 * e] += w * __uint_as_float(x[u][e8][e] << 16);
          acc[8 * e8 + 2 * e + 1] += w * __uint_as_float(x[u][e8][e] & 0xFFFF0000u);
        }
    }
  };
  if (lane_on) {
    int ja[NB], jb[NB];
    u32x4 xa[NB][E8], xb[NB][E8];
    take(ja);
    if (ja[0] >= 0) issue(ja, xa);
    while (ja[0] >= 0) {
      take(jb);
      if (jb[0] >= 0) issue(jb, xb);
      accumulate(ja, xa);
      if (jb[0] < 0) break;
      take(ja);
      if (ja[0] >= 0) issue(ja, xa);
      accumulate(jb, xb);
    }
  }
  if (!active || !lane_on) return;
  const int head = r * G + hh;
  uint16_t* dst = o + (row * H_q + head) * kHeadDim + dd;
#pragma unroll
  for (int e8 = 0; e8 < E8; ++e8) {
    uint4 wv;
    wv.x = pack_bf16x2(acc[8 * e8 + 0], acc[8 * e8 + 1]);
    wv.y = pack_bf16x2(acc[8 * e8 + 2], acc[8 * e8 + 3]);
    wv.z = pack_bf16x2(acc[8 * e8 + 4], acc[8 * e8 + 5]);
    wv.w = pack_bf16x2(acc[8 * e8 + 6], acc[8 * e8 + 7]);
    *reinterpret_cast<uint4*>(dst + 8 * e8) = wv;
  }
  if (lane % lanes_per_head == 0) {
    float t = -INFINITY;
#pragma unroll
    for (int x = 0; x < 16; ++x)
      if (x == hh) t = tot[x];
    lse[row * H_q + head] = t;
  }
}

// ---------------------------------------------------------------- host plan
struct KvoPlan {
  int64_t nbcap;        // key blocks over all sequences (upper bound)
  int64_t ntile;        // H_kv * nbcap
  int64_t chunk_rows;   // query rows per chunk
  int nscan;            // scan blocks
  // workspace offsets
  size_t off_blk_base, off_cnt, off_tile_off, off_item_off, off_blk_tot, off_handles, off_tpos, off_obuf, off_lse,
      total;
};

size_t fixed_bytes(KvoPlan& pl, const msa_seqs* seqs) {
  using msa_host::align_up;
  size_t o = 0;
  pl.off_blk_base = o; o = align_up(o + sizeof(int64_t) * (seqs->num_seqs + 1), 256);
  pl.off_cnt = o;      o = align_up(o + sizeof(int32_t) * (pl.ntile + kWorkCounters), 256);
  pl.off_tile_off = o; o = align_up(o + sizeof(int32_t) * (pl.ntile + 1), 256);
  pl.off_item_off = o; o = align_up(o + sizeof(int32_t) * (pl.ntile + 1), 256);
  pl.off_blk_tot = o;  o = align_up(o + sizeof(int32_t) * 2 * pl.nscan, 256);
  return o;
}

size_t per_row_bytes(int H_q, int H_kv, int topk) {
  return 2 * sizeof(uint32_t) * H_kv * topk + static_cast<size_t>(topk) * H_q * (kHeadDim * 2 + sizeof(float));
}

void layout_rows(KvoPlan& pl, size_t fixed, int H_q, int H_kv, int topk) {
  using msa_host::align_up;
  size_t o = fixed;
  pl.off_handles = o; o = align_up(o + sizeof(uint32_t) * pl.chunk_rows * H_kv * topk, 256);
  pl.off_tpos = o;    o = align_up(o + sizeof(int32_t) * pl.chunk_rows * H_kv * topk, 256);
  pl.off_obuf = o;    o = align_up(o + sizeof(uint16_t) * static_cast<size_t>(topk) * pl.chunk_rows * H_q * kHeadDim, 256);
  pl.off_lse = o;     o = align_up(o + sizeof(float) * static_cast<size_t>(topk) * pl.chunk_rows * H_q, 256);
  pl.total = o;
}

constexpr size_t kDefaultPartialBytes = size_t(32) << 30;

int make_kvo_plan(const msa_seqs* seqs, int H_q, int H_kv, int BK, int topk, size_t budget, KvoPlan* pl) {
  const int64_t nb = (seqs->max_kv_len + BK - 1) / BK;
  pl->nbcap = static_cast<int64_t>(seqs->num_seqs) * (nb > 0 ? nb : 1);
  pl->ntile = static_cast<int64_t>(H_kv) * pl->nbcap;
  if (pl->ntile >= (int64_t(1) << 31) - 1) return MSA_ERR_UNSUPPORTED;
  pl->nscan = static_cast<int>((pl->ntile + kScanPerBlock - 1) / kScanPerBlock);
  if (pl->nscan > 1024 * 64) return MSA_ERR_UNSUPPORTED;
  const size_t fixed = fixed_bytes(*pl, seqs);
  const size_t prb = per_row_bytes(H_q, H_kv, topk);
  int64_t rows = seqs->total_q_rows > 0 ? seqs->total_q_rows : 1;
  pl->chunk_rows = rows;
  layout_rows(*pl, fixed, H_q, H_kv, topk);
  if (pl->total <= budget) {
    // everything in one chunk
  } else if (budget > fixed) {
    const int64_t fit = static_cast<int64_t>((budget - fixed - 4 * 256) / prb);
    if (fit < rows) rows = fit;
  } else {
    rows = 0;
  }
  // incidences of a chunk must fit the int32 offsets
  const int64_t max_rows =
      std::min(kMaxChunkRows, ((int64_t(1) << 31) - 1) / (static_cast<int64_t>(H_kv) * topk));
  if (rows > max_rows) rows = max_rows;
  if (rows < 1) return MSA_ERR_WORKSPACE;
  pl->chunk_rows = rows;
  layout_rows(*pl, fixed, H_q, H_kv, topk);
  return MSA_OK;
}

}  // namespace

// Used by the prefill entry points in sparse_attn.hip.
size_t msa_kvo_workspace_size(const msa_seqs* seqs, int H_q, int H_kv, int BK, int topk) {
  KvoPlan pl;
  if (make_kvo_plan(seqs, H_q, H_kv, BK, topk, kDefaultPartialBytes, &pl) != MSA_OK) {
    // the default budget is too small for one row: ask for exactly one row
    if (make_kvo_plan(seqs, H_q, H_kv, BK, topk, ~size_t(0) >> 1, &pl) != MSA_OK) return 0;
    pl.chunk_rows = 1;
    layout_rows(pl, fixed_bytes(pl, seqs), H_q, H_kv, topk);
  }
  return pl.total;
}

namespace {

template <int BK, typename T>
void launch_kvo_attn(const void* q, const void* k, const void* v, const msa_seqs& sq, const int64_t* blk_base,
                     const int32_t* tile_off, const int32_t* item_off, const uint32_t* handles, int H_q, int H_kv,
                     int topk, int64_t nbcap, int64_t r0, float sl2, float o_scale, uint16_t* o_buf, float* lse_buf,
                     int32_t* next_item, hipStream_t stream) {
  static std::atomic<int> ctas {0};
  constexpr int threads = 64 * kvo_waves<BK>();
  msa_prof::launch("kvo_attn_kernel", kvo_attn_kernel<BK, T>,
                   dim3(persistent_ctas(kvo_attn_kernel<BK, T>, threads, &ctas)), dim3(threads), 0, stream,
                   static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), sq, blk_base,
                   tile_off, item_off, handles, H_q, H_kv, topk, nbcap, r0, sl2, o_scale, o_buf, lse_buf, next_item);
}

}  // namespace

// fp8: Q, K and V are OCP e4m3 with per-tensor scales (logits use
// scale * q_scale * k_scale, O is multiplied by v_scale); else bf16 (scales 1).
int msa_kvo_prefill(const void* q, const void* k, const void* v, const int32_t* block_ids, const msa_seqs* seqs,
                    int H_q, int H_kv, int BK, int topk, float scale, void* o, float* lse, void* workspace,
                    size_t workspace_bytes, hipStream_t stream, bool fp8, float q_scale, float k_scale,
                    float v_scale) {
  KvoPlan pl;
  int st = make_kvo_plan(seqs, H_q, H_kv, BK, topk, workspace_bytes, &pl);
  if (st != MSA_OK) return st;
  if (!workspace || workspace_bytes < pl.total) return MSA_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  auto* blk_base = reinterpret_cast<int64_t*>(ws + pl.off_blk_base);
  auto* cnt = reinterpret_cast<int32_t*>(ws + pl.off_cnt);
  auto* tile_off = reinterpret_cast<int32_t*>(ws + pl.off_tile_off);
  auto* item_off = reinterpret_cast<int32_t*>(ws + pl.off_item_off);
  auto* blk_tot = reinterpret_cast<int32_t*>(ws + pl.off_blk_tot);
  auto* handles = reinterpret_cast<uint32_t*>(ws + pl.off_handles);
  auto* tpos = reinterpret_cast<int32_t*>(ws + pl.off_tpos);
  auto* o_buf = reinterpret_cast<uint16_t*>(ws + pl.off_obuf);
  auto* lse_buf = reinterpret_cast<float*>(ws + pl.off_lse);
  const msa_seqs sq = *seqs;
  auto* op = static_cast<uint16_t*>(o);
  const float sl2 = scale * q_scale * k_scale * kLog2e;

  msa_prof::launch("kvo_block_base_kernel", kvo_block_base_kernel, dim3(1), dim3(256), 0, stream, sq, BK, blk_base);
  for (int64_t r0 = 0; r0 < seqs->total_q_rows; r0 += pl.chunk_rows) {
    const int64_t nr = std::min<int64_t>(pl.chunk_rows, seqs->total_q_rows - r0);
    build_reverse_index(block_ids, sq, blk_base, H_kv, BK, topk, pl.nbcap, pl.ntile, pl.nscan, r0, nr, cnt, tile_off,
                        item_off, blk_tot, tpos, handles, stream);
    if (BK == 64 && !fp8)
      launch_kvo_attn<64, uint16_t>(q, k, v, sq, blk_base, tile_off, item_off, handles, H_q, H_kv, topk, pl.nbcap, r0,
                                    sl2, v_scale, o_buf, lse_buf, cnt + pl.ntile, stream);
    else if (BK == 64)
      launch_kvo_attn<64, uint8_t>(q, k, v, sq, blk_base, tile_off, item_off, handles, H_q, H_kv, topk, pl.nbcap, r0,
                                   sl2, v_scale, o_buf, lse_buf, cnt + pl.ntile, stream);
    else if (!fp8)
      launch_kvo_attn<128, uint16_t>(q, k, v, sq, blk_base, tile_off, item_off, handles, H_q, H_kv, topk, pl.nbcap,
                                     r0, sl2, v_scale, o_buf, lse_buf, cnt + pl.ntile, stream);
    else
      launch_kvo_attn<128, uint8_t>(q, k, v, sq, blk_base, tile_off, item_off, handles, H_q, H_kv, topk, pl.nbcap,
                                    r0, sl2, v_scale, o_buf, lse_buf, cnt + pl.ntile, stream);
    const int64_t pairs = nr * H_kv;
    const int G = H_q / H_kv;
    auto combine = G <= 4 ? kvo_combine_kernel<8> : (G <= 8 ? kvo_combine_kernel<16> : kvo_combine_kernel<32>);
    msa_prof::launch("kvo_combine_kernel", combine, dim3(static_cast<unsigned>((pairs + kCombineWaves - 1) / kCombineWaves)),
                     dim3(64 * kCombineWaves), 0, stream, block_ids, sq, blk_base, H_q, H_kv, BK, topk, r0, nr,
                     o_buf, lse_buf, op, lse);
  }
  return msa_host::launch_status();
}
