// Reverse index of a block selection for key-block-outer kernels.
//
// A block selection lists, per (query row, group), the key blocks the row
// attends (Sec. 3.1, top-k equation).  Kernels that iterate key blocks on the
// outside need the transpose: per tile (group r, key block) the list of
// (query row, slot) handles that selected it, cut into work items of at most
// kItemQueries queries (Sec. 4.2 on the KV-outer order; Sec. 4.3 on work
// partitioned along the gathered-query dimension).  Built per chunk of query
// rows:
//   kvo_count    incidences per tile and each incidence's position in its tile
//   kvo_scan*    exclusive offsets of handles and of work items per tile
//   kvo_fill     handle (row in chunk << 6 | slot) lists per tile
// Included by the forward and backward Main Branch sources; everything here
// has internal linkage.
#pragma once

#include <algorithm>
#include <atomic>

#include "msa_common.h"
#include "msa_profile.h"

namespace {

using namespace msa;

constexpr int kHeadDim = 128;
constexpr int kItemQueries = 256;      // queries of one tile per work item
// A handle packs (row in chunk << 6 | slot) into 32 bits, so a chunk holds at
// most 2^26 query rows; the plans cap their chunks there.
constexpr int64_t kMaxChunkRows = int64_t(1) << 26;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bool slot_valid(int b, int p, int BK) { return b >= 0 && p >= 0 && b <= p / BK; }
// An incidence takes part in the reverse index, the attention and the combine
// iff its slot is valid and the block exists in the sequence's block range
// (always true for consistent layouts; the second test keeps every index in
// bounds when kv_lens exceed max_kv_len).
__device__ __forceinline__ bool incidence_ok(int b, int p, int BK, const int64_t* __restrict__ blk_base, int s) {
  return slot_valid(b, p, BK) && static_cast<int64_t>(b) < blk_base[s + 1] - blk_base[s];
}

__device__ __forceinline__ int row_position(const msa_seqs& sq, int64_t row, int* seq_out) {
  const int s = find_seq(sq.q_offsets, sq.num_seqs, row);
  const SeqGeom g = seq_geom(sq, s);
  int p = g.kv_len - g.q_rows + static_cast<int>(row - g.q_begin);
  if (p >= g.kv_len) p = -1;
  *seq_out = s;
  return p;
}

// ---------------------------------------------------------------- setup
// blk_base[s] = key blocks of the sequences before s (kv_len clamped to max_kv_len).
__global__ __launch_bounds__(256) void kvo_block_base_kernel(msa_seqs sq, int BK, int64_t* __restrict__ blk_base) {
  __shared__ int64_t part[256];
  const int t = threadIdx.x;
  const int S = sq.num_seqs;
  const int per = (S + 255) / 256;
  const int s0 = t * per, s1 = min(S, s0 + per);
  auto nblk = [&](int s) -> int64_t {
    int64_t len = seq_geom(sq, s).kv_len;
    if (len > sq.max_kv_len) len = sq.max_kv_len;
    return (len + BK - 1) / BK;
  };
  int64_t acc = 0;
  for (int s = s0; s < s1; ++s) acc += nblk(s);
  part[t] = acc;
  __syncthreads();
  if (t == 0) {
    int64_t run = 0;
    for (int i = 0; i < 256; ++i) { int64_t x = part[i]; part[i] = run; run += x; }
    blk_base[S] = run;
  }
  __syncthreads();
  acc = part[t];
  for (int s = s0; s < s1; ++s) { blk_base[s] = acc; acc += nblk(s); }
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = v;
}

// ---------------------------------------------------------------- reverse index
// Positions of every incidence inside its tile's handle list, with few device
// atomics: a CTA takes kHistRows query rows of one group, histograms their
// incidences over the key blocks of its sequences in LDS, claims one segment
// of each touched tile with a single device atomic (the returned count is the
// segment's start) and hands out positions inside its segments with LDS
// atomics.  A CTA whose sequences span more than kHistBins key blocks falls
// back to one device atomic per incidence.  Positions are relative to the
// tile; kvo_fill adds the tile offsets once the scan has run.  1024 rows per
// CTA: a 32K-row chunk of 8 groups gives 256 CTAs (with 4096 rows, 64 CTAs
// left most CUs idle and the kernel took 3.5x as long).
constexpr int kHistRows = 1024;
constexpr int kHistBins = 16384;

__global__ __launch_bounds__(256) void kvo_count_kernel(const int32_t* __restrict__ block_ids, msa_seqs sq,
                                                        const int64_t* __restrict__ blk_base, int H_kv, int BK,
                                                        int topk, int64_t nbcap, int64_t row0, int64_t nrows,
                                                        int32_t* __restrict__ cnt, int32_t* __restrict__ tpos) {
  __shared__ int32_t hist[kHistBins];
  const int r = blockIdx.y;
  const int64_t rb0 = row0 + static_cast<int64_t>(blockIdx.x) * kHistRows;
  const int64_t rb1 = min(rb0 + kHistRows, row0 + nrows);
  const int s_first = find_seq_wave(sq.q_offsets, sq.num_seqs, rb0);
  const int s_last = find_seq_wave(sq.q_offsets, sq.num_seqs, rb1 - 1);
  const int64_t g_lo = blk_base[s_first];
  const int64_t g_hi = blk_base[s_last + 1];
  const bool in_lds = g_hi - g_lo <= kHistBins;           // uniform over the CTA
  const int64_t tile_base = static_cast<int64_t>(r) * nbcap;

  if (in_lds) {
    for (int i = threadIdx.x; i < kHistBins; i += 256) hist[i] = 0;
    __syncthreads();
  }
  // pass 1: histogram (or, without LDS room, claim each position directly);
  // one row per thread keeps 64 rows' id lookups in flight per wave (one row
  // per wave, slot on lane, took twice as long); a row's ids are read four per
  // 16-byte load when topk % 4 == 0 and the id array is 16-byte aligned
  const bool vec = topk % 4 == 0 && (reinterpret_cast<uintptr_t>(block_ids) & 15) == 0;
  for (int64_t row = rb0 + threadIdx.x; row < rb1; row += 256) {
    int s;
    const int p = row_position(sq, row, &s);
    const int32_t* ids = block_ids + (row * H_kv + r) * topk;
    int32_t* tp = tpos + ((row - row0) * H_kv + r) * topk;
    const int64_t gb0 = blk_base[s];
    if (vec && in_lds) {
      for (int j = 0; j < topk; j += 4) {
        const int4 b4 = *reinterpret_cast<const int4*>(ids + j);
        const int bb[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (incidence_ok(bb[e], p, BK, blk_base, s)) atomicAdd(&hist[gb0 + bb[e] - g_lo], 1);
      }
      continue;
    }
    for (int j = 0; j < topk; ++j) {
      const int b = ids[j];
      if (!incidence_ok(b, p, BK, blk_base, s)) continue;
      if (in_lds) atomicAdd(&hist[gb0 + b - g_lo], 1);
      else tp[j] = atomicAdd(&cnt[tile_base + gb0 + b], 1);
    }
  }
  if (!in_lds) return;
  __syncthreads();
  // claim one segment per touched tile; hist becomes the segment cursor
  const int nbin = static_cast<int>(g_hi - g_lo);
  for (int i = threadIdx.x; i < nbin; i += 256) {
    const int c = hist[i];
    if (c > 0) hist[i] = atomicAdd(&cnt[tile_base + g_lo + i], c);
  }
  __syncthreads();
  // pass 2: positions inside the claimed segments (16-byte loads and stores
  // of four slots on the same condition; slots that are no incidence get
  // position 0, which nothing reads)
  for (int64_t row = rb0 + threadIdx.x; row < rb1; row += 256) {
    int s;
    const int p = row_position(sq, row, &s);
    const int32_t* ids = block_ids + (row * H_kv + r) * topk;
    int32_t* tp = tpos + ((row - row0) * H_kv + r) * topk;
    const int64_t gb0 = blk_base[s];
    if (vec) {
      for (int j = 0; j < topk; j += 4) {
        const int4 b4 = *reinterpret_cast<const int4*>(ids + j);
        const int bb[4] = {b4.x, b4.y, b4.z, b4.w};
        int t4[4] = {0, 0, 0, 0};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (incidence_ok(bb[e], p, BK, blk_base, s)) t4[e] = atomicAdd(&hist[gb0 + bb[e] - g_lo], 1);
        *reinterpret_cast<int4*>(tp + j) = make_int4(t4[0], t4[1], t4[2], t4[3]);
      }
      continue;
    }
    for (int j = 0; j < topk; ++j) {
      const int b = ids[j];
      if (!incidence_ok(b, p, BK, blk_base, s)) continue;
      tp[j] = atomicAdd(&hist[gb0 + b - g_lo], 1);
    }
  }
}

// One wave per (row, group) of the chunk, slot j on lane j: handle =
// (row in chunk << 6 | slot).
__global__ __launch_bounds__(256) void kvo_fill_kernel(const int32_t* __restrict__ block_ids, msa_seqs sq,
                                                       const int64_t* __restrict__ blk_base, int H_kv, int BK,
                                                       int topk, int64_t nbcap, int64_t row0, int64_t nrows,
                                                       const int32_t* __restrict__ tile_off,
                                                       const int32_t* __restrict__ tpos,
                                                       uint32_t* __restrict__ handles) {
  const int lane = lane_id();
  const int64_t i = static_cast<int64_t>(blockIdx.x) * (256 / kWave) + threadIdx.x / kWave;
  if (i >= nrows * H_kv) return;
  const int64_t rl = i / H_kv;
  const int64_t row = row0 + rl;
  const int r = static_cast<int>(i % H_kv);
  int s;
  const int p = row_position(sq, row, &s);
  const int32_t* ids = block_ids + (row * H_kv + r) * topk;
  const int32_t* tp = tpos + i * topk;
  const int64_t base = static_cast<int64_t>(r) * nbcap + blk_base[s];
  if (lane < topk) {
    const int b = ids[lane];
    if (incidence_ok(b, p, BK, blk_base, s))
      handles[tile_off[base + b] + tp[lane]] = (static_cast<uint32_t>(rl) << 6) | static_cast<uint32_t>(lane);
  }
}

// Two-array exclusive scan (handles per tile, work items per tile) in three
// kernels: per-block scan, scan of block totals, add.
constexpr int kScanPerBlock = 2048;   // 256 threads x 8

__global__ __launch_bounds__(256) void kvo_scan_block_kernel(const int32_t* __restrict__ cnt, int64_t n,
                                                             int32_t* __restrict__ tile_off,
                                                             int32_t* __restrict__ item_off,
                                                             int32_t* __restrict__ blk_tot) {
  __shared__ int32_t sa[256], sb[256];
  const int t = threadIdx.x;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanPerBlock + t * 8;
  int32_t a[8], b[8];
  int32_t ta = 0, tb = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int32_t c = base + e < n ? cnt[base + e] : 0;
    a[e] = ta; b[e] = tb;
    ta += c;
    tb += (c + kItemQueries - 1) / kItemQueries;
  }
  sa[t] = ta; sb[t] = tb;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int32_t xa = t >= off ? sa[t - off] : 0;
    const int32_t xb = t >= off ? sb[t - off] : 0;
    __syncthreads();
    sa[t] += xa; sb[t] += xb;
    __syncthreads();
  }
  const int32_t pa = sa[t] - ta, pb = sb[t] - tb;
#pragma unroll
  for (int e = 0; e < 8; ++e)
    if (base + e < n) { tile_off[base + e] = a[e] + pa; item_off[base + e] = b[e] + pb; }
  if (t == 255) { blk_tot[2 * blockIdx.x] = sa[255]; blk_tot[2 * blockIdx.x + 1] = sb[255]; }
}

__global__ __launch_bounds__(1024) void kvo_scan_top_kernel(int32_t* __restrict__ blk_tot, int nblk,
                                                            int32_t* __restrict__ tile_off,
                                                            int32_t* __restrict__ item_off, int64_t n) {
  __shared__ int32_t sa[1024], sb[1024];
  const int t = threadIdx.x;
  const int per = (nblk + 1023) / 1024;
  const int b0 = t * per, b1 = min(nblk, b0 + per);
  int32_t ta = 0, tb = 0;
  for (int b = b0; b < b1; ++b) { ta += blk_tot[2 * b]; tb += blk_tot[2 * b + 1]; }
  sa[t] = ta; sb[t] = tb;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t xa = t >= off ? sa[t - off] : 0;
    const int32_t xb = t >= off ? sb[t - off] : 0;
    __syncthreads();
    sa[t] += xa; sb[t] += xb;
    __syncthreads();
  }
  int32_t ra = sa[t] - ta, rb = sb[t] - tb;
  for (int b = b0; b < b1; ++b) {
    const int32_t xa = blk_tot[2 * b], xb = blk_tot[2 * b + 1];
    blk_tot[2 * b] = ra; blk_tot[2 * b + 1] = rb;
    ra += xa; rb += xb;
  }
  if (t == 1023) { tile_off[n] = sa[1023]; item_off[n] = sb[1023]; }
}

__global__ __launch_bounds__(256) void kvo_scan_add_kernel(const int32_t* __restrict__ blk_tot, int64_t n,
                                                           int32_t* __restrict__ tile_off,
                                                           int32_t* __restrict__ item_off) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int64_t b = i / kScanPerBlock;
  tile_off[i] += blk_tot[2 * b];
  item_off[i] += blk_tot[2 * b + 1];
}

// Largest i with arr[i] <= x, for arr non-decreasing with arr[0] <= x.
template <typename T>
__device__ __forceinline__ int64_t upper_index(const T* __restrict__ arr, int64_t n, int64_t x) {
  int64_t lo = 0, hi = n - 1;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if (static_cast<int64_t>(arr[mid]) <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// CTAs of a persistent kernel: every CU filled to the kernel's occupancy.  The
// value is cached per kernel instance; concurrent first calls may both compute
// it, and the atomic makes their stores and loads well defined.
template <typename K>
int persistent_ctas(K kernel, int threads, std::atomic<int>* cache) {
  int n = cache->load(std::memory_order_relaxed);
  if (n == 0) {
    int dev = 0, cus = 256, per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess || per_cu < 1)
      per_cu = 1;
    n = cus * per_cu;
    cache->store(n, std::memory_order_relaxed);
  }
  return n;
}
// Block ids of B_k = 64 f from ids of blocks of 64 f keys: block b becomes its
// f sub-blocks f b .. f b + f - 1 (ascending order and -1 padding kept), so a
// 64-key kernel covers exactly the same tokens.  One thread per (row, group).
__global__ __launch_bounds__(256) void expand_block_ids_kernel(const int32_t* __restrict__ ids, int64_t pairs,
                                                               int topk, int f, int32_t* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= pairs) return;
  const int32_t* src = ids + i * topk;
  int32_t* dst = out + i * topk * f;
  for (int j = 0; j < topk; ++j) {
    const int32_t b = src[j];
    for (int e = 0; e < f; ++e) dst[j * f + e] = b >= 0 ? b * f + e : -1;
  }
}

// Persistent work loops: a CTA's first item is blockIdx.x, later ones are
// claimed from a global counter, so CTAs that drew cheap items take more
// (the dynamic load balancing of Sec. 4.3).  The counters sit after the
// ntile tile counts (cnt has ntile + kWorkCounters entries) and are zeroed
// with them when the reverse index is built; each persistent launch that
// follows uses its own one.
constexpr int kWorkCounters = 2;
__device__ __forceinline__ int32_t claim_next_item(int32_t* __restrict__ next_item, int32_t* s_claim) {
  __syncthreads();                                    // every thread has read the previous claim
  if (threadIdx.x == 0) *s_claim = static_cast<int32_t>(gridDim.x) + atomicAdd(next_item, 1);
  __syncthreads();
  return *s_claim;
}

// ---------------------------------------------------------------- canonical handle order
// The reverse index hands out positions inside a tile with atomics, so a
// tile's handle list comes out in a run-dependent order.  Kernels whose sums
// run over a tile's handles (the training backward's dK / dV and d k_idx)
// sort each list into ascending handle order -- row, then slot -- which makes
// their results bit-reproducible.  A row selects a block once, so a tile's
// handles have distinct rows and the order is the rows' order.  One CTA per
// tile, two launches:
//   sort_tile_handles_kernel   tiles of at most kSortRun handles: bitonic
//                              sort in LDS;
//   rank_tile_handles_kernel   longer tiles: the rows are marked in an LDS
//                              bitmap over the tile's row span, and each
//                              handle's place is the number of marked rows
//                              below its own (popcounts; a prefix per 32
//                              words); spans of more than kRankMapWords * 32
//                              rows (or a row listed twice) fall back to
//                              merging sorted runs pairwise through `tmp` (a
//                              handle's place in a merged run is its rank in
//                              its own run plus its rank among the other
//                              run's handles).
constexpr int kSortRun = 2048;
constexpr int kRankMapWords = 32768;                  // 1M rows of span, 128 KiB of LDS

__device__ __forceinline__ int32_t count_below(const uint32_t* __restrict__ a, int32_t n, uint32_t x) {
  int32_t lo = 0, hi = n;                      // first index with a[i] >= x
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Bitonic sort of a[0 .. m) (m <= kSortRun) through the LDS array sh.
__device__ __forceinline__ void sort_run_lds(uint32_t* __restrict__ a, int32_t m, uint32_t* sh) {
  const int tid = threadIdx.x;
  int32_t P = 1;
  while (P < m) P <<= 1;
  for (int32_t i = tid; i < P; i += 256) sh[i] = i < m ? a[i] : 0xFFFFFFFFu;
  __syncthreads();
  for (int32_t kk = 2; kk <= P; kk <<= 1)
    for (int32_t j = kk >> 1; j > 0; j >>= 1) {
      for (int32_t i = tid; i < P; i += 256) {
        const int32_t ixj = i ^ j;
        if (ixj > i) {
          const uint32_t x = sh[i], y = sh[ixj];
          const bool up = (i & kk) == 0;
          if ((x > y) == up) { sh[i] = y; sh[ixj] = x; }
        }
      }
      __syncthreads();
    }
  for (int32_t i = tid; i < m; i += 256) a[i] = sh[i];
  __syncthreads();
}

__global__ __launch_bounds__(256) void sort_tile_handles_kernel(uint32_t* __restrict__ handles,
                                                                const int32_t* __restrict__ tile_off) {
  __shared__ uint32_t sh[kSortRun];
  const int64_t t = blockIdx.x;
  const int32_t beg = tile_off[t];
  const int32_t n = tile_off[t + 1] - beg;
  if (n <= 1 || n > kSortRun) return;                // uniform over the CTA
  sort_run_lds(handles + beg, n, sh);
}

// a[0 .. n) sorted as runs of kSortRun (through sh), then merged pairwise
// through b; the result ends in a.
__device__ __forceinline__ void sort_by_merging(uint32_t* __restrict__ a, uint32_t* __restrict__ b, int32_t n,
                                                uint32_t* sh) {
  const int tid = threadIdx.x;
  for (int32_t r0 = 0; r0 < n; r0 += kSortRun) sort_run_lds(a + r0, min(kSortRun, n - r0), sh);
  uint32_t* src = a;
  uint32_t* dst = b;
  for (int32_t w = kSortRun; w < n; w <<= 1) {
    for (int32_t i = tid; i < n; i += 256) {
      const int32_t l0 = (i / (2 * w)) * (2 * w);     // the pair of runs holding i
      const int32_t mid = min(l0 + w, n), h1 = min(l0 + 2 * w, n);
      const uint32_t x = src[i];
      const int32_t pos = i < mid ? l0 + (i - l0) + count_below(src + mid, h1 - mid, x)
                                  : l0 + (i - mid) + count_below(src + l0, mid - l0, x);
      dst[pos] = x;
    }
    __syncthreads();
    uint32_t* sw = src; src = dst; dst = sw;
  }
  if (src != a)
    for (int32_t i = tid; i < n; i += 256) a[i] = src[i];
}

__global__ __launch_bounds__(256) void rank_tile_handles_kernel(uint32_t* __restrict__ handles,
                                                                uint32_t* __restrict__ tmp,
                                                                const int32_t* __restrict__ tile_off) {
  __shared__ uint32_t map[kRankMapWords];
  __shared__ int32_t grp[kRankMapWords / 32];         // marked rows before each 32-word group
  __shared__ uint32_t red[2][256 / kWave];
  __shared__ int32_t scan[256];
  const int64_t t = blockIdx.x;
  const int32_t beg = tile_off[t];
  const int32_t n = tile_off[t + 1] - beg;
  if (n <= kSortRun) return;                          // uniform over the CTA
  const int tid = threadIdx.x, lane = lane_id(), wave = tid / kWave;
  uint32_t* a = handles + beg;
  uint32_t* b = tmp + beg;
  // the tile's row span
  uint32_t lo = 0xFFFFFFFFu, hi = 0;
  for (int32_t i = tid; i < n; i += 256) {
    const uint32_t r = a[i] >> 6;
    lo = min(lo, r);
    hi = max(hi, r);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    lo = min(lo, static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), off)));
    hi = max(hi, static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), off)));
  }
  if (lane == 0) { red[0][wave] = lo; red[1][wave] = hi; }
  __syncthreads();
  lo = red[0][0];
  hi = red[1][0];
#pragma unroll
  for (int w = 1; w < 256 / kWave; ++w) { lo = min(lo, red[0][w]); hi = max(hi, red[1][w]); }
  const int64_t words = (static_cast<int64_t>(hi) - lo + 32) / 32;
  if (words > kRankMapWords) {                        // span too wide for the bitmap
    sort_by_merging(a, b, n, map);
    return;
  }
  const int nw = static_cast<int>(words);
  const int ng = (nw + 31) / 32;
  for (int i = tid; i < nw; i += 256) map[i] = 0;
  __syncthreads();
  for (int32_t i = tid; i < n; i += 256) {
    const uint32_t r = (a[i] >> 6) - lo;
    atomicOr(&map[r >> 5], 1u << (r & 31));
  }
  __syncthreads();
  // marked rows per 32-word group, exclusive prefix over the groups (each
  // thread owns up to 4 consecutive groups)
  int32_t cnt[4];
  int32_t own = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int g = 4 * tid + q;
    int32_t c = 0;
    if (g < ng)
      for (int w = 32 * g; w < min(32 * g + 32, nw); ++w) c += __popc(map[w]);
    cnt[q] = c;
    own += c;
  }
  scan[tid] = own;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int32_t v = tid >= off ? scan[tid - off] : 0;
    __syncthreads();
    scan[tid] += v;
    __syncthreads();
  }
  if (scan[255] != n) {                               // a row listed twice (not a valid selection):
    __syncthreads();                                  // order by (row, slot) all the same
    sort_by_merging(a, b, n, map);
    return;
  }
  int32_t run = scan[tid] - own;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int g = 4 * tid + q;
    if (g < ng) grp[g] = run;
    run += cnt[q];
  }
  __syncthreads();
  for (int32_t i = tid; i < n; i += 256) {
    const uint32_t h = a[i];
    const uint32_t r = (h >> 6) - lo;
    const int w = static_cast<int>(r >> 5);
    int32_t rank = grp[w >> 5] + __popc(map[w] & ((1u << (r & 31)) - 1u));
    for (int v = w & ~31; v < w; ++v) rank += __popc(map[v]);
    b[rank] = h;
  }
  __syncthreads();
  for (int32_t i = tid; i < n; i += 256) a[i] = b[i];
}

// Reverse index of query rows r0 .. r0 + nr - 1 (one chunk): counts, scans
// and handle lists for every tile of H_kv x nbcap; `canonical` sorts each list.
void build_reverse_index(const int32_t* block_ids, const msa_seqs& sq, const int64_t* blk_base, int H_kv, int BK,
                         int topk, int64_t nbcap, int64_t ntile, int nscan, int64_t r0, int64_t nr, int32_t* cnt,
                         int32_t* tile_off, int32_t* item_off, int32_t* blk_tot, int32_t* tpos, uint32_t* handles,
                         hipStream_t stream, bool canonical = false) {
  const unsigned fill_blocks = static_cast<unsigned>(std::min<int64_t>((ntile + kWorkCounters + 255) / 256, 4096));
  const unsigned gthreads = static_cast<unsigned>((nr * H_kv + 256 / kWave - 1) / (256 / kWave));   // a wave per pair
  msa_prof::launch("fill_i32_kernel", fill_i32_kernel, dim3(fill_blocks), dim3(256), 0, stream, cnt,
                   ntile + kWorkCounters, 0);
  const dim3 hgrid(static_cast<unsigned>((nr + kHistRows - 1) / kHistRows), static_cast<unsigned>(H_kv));
  msa_prof::launch("kvo_count_kernel", kvo_count_kernel, hgrid, dim3(256), 0, stream, block_ids, sq, blk_base, H_kv,
                   BK, topk, nbcap, r0, nr, cnt, tpos);
  msa_prof::launch("kvo_scan_block_kernel", kvo_scan_block_kernel, dim3(nscan), dim3(256), 0, stream, cnt, ntile,
                   tile_off, item_off, blk_tot);
  msa_prof::launch("kvo_scan_top_kernel", kvo_scan_top_kernel, dim3(1), dim3(1024), 0, stream, blk_tot, nscan,
                   tile_off, item_off, ntile);
  msa_prof::launch("kvo_scan_add_kernel", kvo_scan_add_kernel, dim3(static_cast<unsigned>((ntile + 255) / 256)),
                   dim3(256), 0, stream, blk_tot, ntile, tile_off, item_off);
  msa_prof::launch("kvo_fill_kernel", kvo_fill_kernel, dim3(gthreads), dim3(256), 0, stream, block_ids, sq, blk_base,
                   H_kv, BK, topk, nbcap, r0, nr, tile_off, tpos, handles);
  // positions are no longer needed: tpos is the long tiles' scatter buffer
  if (canonical) {
    msa_prof::launch("sort_tile_handles_kernel", sort_tile_handles_kernel, dim3(static_cast<unsigned>(ntile)),
                     dim3(256), 0, stream, handles, static_cast<const int32_t*>(tile_off));
    msa_prof::launch("rank_tile_handles_kernel", rank_tile_handles_kernel, dim3(static_cast<unsigned>(ntile)),
                     dim3(256), 0, stream, handles, reinterpret_cast<uint32_t*>(tpos),
                     static_cast<const int32_t*>(tile_off));
  }
}

}  // namespace
