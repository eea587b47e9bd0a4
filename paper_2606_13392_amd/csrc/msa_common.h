// Shared device and host helpers of libmsa (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "msa.h"

namespace msa {

// ---------------------------------------------------------------- vector types
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;   // 16-byte register piece

constexpr int kWave = 64;

__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
}
__device__ __forceinline__ bf16x8 zero_bf16x8() { return __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0)); }

// Eight consecutive elements of a bf16 tensor (T = uint16_t) or of an OCP
// 8-bit E4M3 ("e4m3fn") tensor (T = uint8_t).  Raw<T> holds them as loaded;
// widen() gives 8 bf16 values (exact for e4m3: every e4m3 value is a bf16
// value; gfx950's v_cvt_scalef32_pk_bf16_fp8 at scale 1 converts two per
// instruction).  Kernels load raw under their bounds conditions and widen at
// the point of use, so no conversion sits inside a branch and forces a wait
// on the load right after issuing it.
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;
template <typename T> struct RawOf;
template <> struct RawOf<uint16_t> { using type = u32x4; };
template <> struct RawOf<uint8_t> { using type = u32x2; };
template <typename T> using Raw = typename RawOf<T>::type;

__device__ __forceinline__ u32x4 load_raw(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ u32x2 load_raw(const uint8_t* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ __forceinline__ u32x4 widen(u32x4 r) { return r; }
__device__ __forceinline__ u32x4 widen(u32x2 r) {
  u32x4 o;
  o[0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r[0], 1.0f, false));
  o[1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r[0], 1.0f, true));
  o[2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r[1], 1.0f, false));
  o[3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(r[1], 1.0f, true));
  return o;
}
template <typename R>
__device__ __forceinline__ bf16x8 widen_bf16x8(R r) { return __builtin_bit_cast(bf16x8, widen(r)); }

// Raw hardware 2^x (v_exp_f32, half rate on gfx950): results below the fp32
// normal range come out as zero, which a softmax weight relative to its
// row's maximum (at most 1) cannot notice; exp2f adds a range reduction of
// five more instructions for those results.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// MFMA 32x32x16 bf16 -> f32.  Lane l supplies row (A) / column (B) l%32 and
// eight consecutive k of the half l/32; C lane l holds column l%32, rows
// 8*(r/4) + 4*(l/32) + r%4 for r = 0..15.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// MFMA 16x16x32 bf16 -> f32.  Lane l supplies row/column l%16 and eight k of
// the quarter l/16; C lane l holds column l%16, rows 4*(l/16) + r, r = 0..3.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// float -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
// Two floats -> packed bf16 pair (lo in the low half), round to nearest even:
// one v_cvt_pk_bf16_f32 on gfx950.
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// ---------------------------------------------------------------- ranking keys
// Order-preserving map of a float score to uint32 (-0 and +0 compare equal).
__device__ __forceinline__ uint32_t ordered_u32(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// 64-bit ranking key: larger score first, then the smaller block id.  Every
// real key is non-zero, so 0 serves as the empty slot.
__device__ __forceinline__ uint64_t rank_key(float score, uint32_t block) {
  return (static_cast<uint64_t>(ordered_u32(score)) << 32) | static_cast<uint64_t>(0xFFFFFFFFu - block);
}
__device__ __forceinline__ uint32_t key_block(uint64_t key) {
  return 0xFFFFFFFFu - static_cast<uint32_t>(key);
}

// ---------------------------------------------------------------- wave helpers
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  int lo = __shfl_xor(static_cast<int>(static_cast<uint32_t>(v)), mask);
  int hi = __shfl_xor(static_cast<int>(static_cast<uint32_t>(v >> 32)), mask);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  int lo = __shfl(static_cast<int>(static_cast<uint32_t>(v)), src);
  int hi = __shfl(static_cast<int>(static_cast<uint32_t>(v >> 32)), src);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v)), lane);
  uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v >> 32)), lane);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Value of lane (lane ^ J): DPP quad permutes for J = 1, 2, ds_swizzle
// (bit-mask mode, within 32 lanes) for J = 4, 8, 16, permlane32 swap for 32.
template <int J>
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t v) {
  if constexpr (J == 1) {
    return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), 0xB1, 0xF, 0xF, false));
  } else if constexpr (J == 2) {
    return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), 0x4E, 0xF, 0xF, false));
  } else if constexpr (J < 32) {
    return static_cast<uint32_t>(__builtin_amdgcn_ds_swizzle(static_cast<int>(v), 0x1F | (J << 10)));
  } else {
    auto sw = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __lane_id() < 32 ? sw[1] : sw[0];
  }
}
template <int J>
__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t v) {
  const uint32_t lo = xor_lane_u32<J>(static_cast<uint32_t>(v));
  const uint32_t hi = xor_lane_u32<J>(static_cast<uint32_t>(v >> 32));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
// Transposed store of 8 consecutive bf16 (w: elements 2k, 2k+1 in word k) of
// row `col` into dst[d0 + e][col]: lanes l and l ^ 1 (rows col and col ^ 1)
// trade two words so that each writes four 32-bit row pairs, the even lane
// elements 0..3 and the odd lane elements 4..7.  Every lane must take part.
template <int P>
__device__ __forceinline__ void store_transposed_pairs(uint16_t (*dst)[P], int d0, int col, const u32x4& w) {
  const bool odd = col & 1;
  const uint32_t r0 = xor_lane_u32<1>(odd ? w[0] : w[2]);   // the neighbour's words of my half
  const uint32_t r1 = xor_lane_u32<1>(odd ? w[1] : w[3]);
  const uint32_t m0 = odd ? w[2] : w[0], m1 = odd ? w[3] : w[1];
  const uint32_t ev0 = odd ? r0 : m0, od0 = odd ? m0 : r0;   // even row's / odd row's word
  const uint32_t ev1 = odd ? r1 : m1, od1 = odd ? m1 : r1;
  const int dd = d0 + (odd ? 4 : 0);
  const int c0 = col & ~1;
  *reinterpret_cast<uint32_t*>(&dst[dd + 0][c0]) = (ev0 & 0xFFFFu) | (od0 << 16);
  *reinterpret_cast<uint32_t*>(&dst[dd + 1][c0]) = (ev0 >> 16) | (od0 & 0xFFFF0000u);
  *reinterpret_cast<uint32_t*>(&dst[dd + 2][c0]) = (ev1 & 0xFFFFu) | (od1 << 16);
  *reinterpret_cast<uint32_t*>(&dst[dd + 3][c0]) = (ev1 >> 16) | (od1 & 0xFFFF0000u);
}

// Value of lane - 1 (lane 0 receives `fill`): DPP wave shift right by one.
__device__ __forceinline__ uint64_t lane_shr1_u64(uint64_t v, uint64_t fill) {
  const int lo = __builtin_amdgcn_update_dpp(static_cast<int>(static_cast<uint32_t>(fill)),
                                             static_cast<int>(static_cast<uint32_t>(v)), 0x138, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(static_cast<int>(static_cast<uint32_t>(fill >> 32)),
                                             static_cast<int>(static_cast<uint32_t>(v >> 32)), 0x138, 0xF, 0xF, false);
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

// One compare-exchange step of a bitonic network: lanes with (lane & J) == 0
// keep the max when `desc` else the min; their partners the other one.
template <int J>
__device__ __forceinline__ uint64_t bitonic_step_u64(uint64_t v, bool desc) {
  const uint64_t o = xor_lane_u64<J>(v);
  const bool lower = (__lane_id() & J) == 0;
  return (desc == lower) ? (v > o ? v : o) : (v < o ? v : o);
}
template <int K, int J>
__device__ __forceinline__ uint64_t bitonic_stage_desc_u64(uint64_t v) {
  if constexpr (J == 0) {
    return v;
  } else {
    v = bitonic_step_u64<J>(v, (__lane_id() & K) == 0);
    return bitonic_stage_desc_u64<K, J / 2>(v);
  }
}
template <int K>
__device__ __forceinline__ uint64_t bitonic_sort_desc_u64(uint64_t v) {
  if constexpr (K > kWave) {
    return v;
  } else {
    v = bitonic_stage_desc_u64<K, K / 2>(v);
    return bitonic_sort_desc_u64<K * 2>(v);
  }
}
// Bitonic sort of one 64-bit key per lane across the wave, descending
// (lane 0 receives the largest key).
__device__ __forceinline__ uint64_t wave_sort_desc_u64(uint64_t v) { return bitonic_sort_desc_u64<2>(v); }
// Sorts a bitonic sequence (one key per lane) descending.
__device__ __forceinline__ uint64_t wave_bitonic_merge_desc_u64(uint64_t v) {
  // K = 128 > every lane index: all lanes sort descending
  return bitonic_stage_desc_u64<128, kWave / 2>(v);
}
// Bitonic sort of one uint32 per lane, ascending.
__device__ __forceinline__ uint32_t wave_sort_asc_u32(uint32_t v) {
  const int lane = lane_id();
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), j));
      bool asc_block = (lane & k) == 0;
      bool lower = (lane & j) == 0;
      bool take_min = (asc_block == lower);
      v = take_min ? (v < o ? v : o) : (v > o ? v : o);
    }
  }
  return v;
}

// Sequence of a packed query row: largest s with q_offsets[s] <= row.
__device__ __forceinline__ int find_seq(const int32_t* __restrict__ q_offsets, int num_seqs, int64_t row) {
  int lo = 0, hi = num_seqs - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (static_cast<int64_t>(q_offsets[mid]) <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// The same search for a wave-uniform row: each level samples 64 evenly spaced
// offsets (one load per lane) and keeps the last one <= row, so one level
// covers 64 sequences and two cover 4096.  Every lane of the wave must call it
// with the same row; offsets[0] <= row is assumed (offsets start at zero).
__device__ __forceinline__ int find_seq_wave(const int32_t* __restrict__ offsets, int num_seqs, int64_t row) {
  int lo = 0, n = num_seqs;                  // the answer lies in [lo, lo + n)
  while (n > 1) {
    const int stride = (n + kWave - 1) / kWave;
    const int idx = lo + __lane_id() * stride;
    const bool ok = idx < lo + n && static_cast<int64_t>(offsets[idx]) <= row;
    const uint64_t mask = __ballot(ok);      // a prefix of the lanes: offsets are non-decreasing
    const int j = 63 - __clzll(static_cast<long long>(mask | 1ull));
    const int lo_new = lo + j * stride;
    n = min(stride, lo + n - lo_new);
    lo = lo_new;
  }
  return lo;
}

// Per-sequence geometry read from the device layout arrays, with the key
// range clamped to the key-side tensor so no access can leave it.
struct SeqGeom {
  int64_t kv_start;   // first key row of the sequence
  int32_t kv_len;     // keys visible to the sequence's last query row
  int32_t q_begin;    // first packed query row
  int32_t q_rows;     // query rows of the sequence
};
__device__ __forceinline__ SeqGeom seq_geom(const msa_seqs& sq, int s) {
  SeqGeom g;
  g.q_begin = sq.q_offsets[s];
  g.q_rows = sq.q_offsets[s + 1] - g.q_begin;
  int64_t len = sq.kv_lens[s];
  int64_t st = 0;
  if (sq.block_table) {
    // paged: the block table bounds the sequence
    const int64_t cap = static_cast<int64_t>(sq.block_table_stride) * sq.page_size;
    if (len > cap) len = cap;
  } else {
    st = sq.kv_starts[s];
    if (st < 0) st = 0;
    if (st > sq.total_kv_rows) st = sq.total_kv_rows;
    if (len > sq.total_kv_rows - st) len = sq.total_kv_rows - st;
  }
  if (len < 0) len = 0;
  g.kv_start = st;
  g.kv_len = static_cast<int32_t>(len);
  return g;
}

// First key row of key block b (blocks of BK keys) of sequence s: kv_start +
// b BK on a contiguous key side, else inside the page the block table lists
// for it (pages of 2^lg_bpp blocks; page ids clamped into the pool).
struct KeyBlocks {
  const int32_t* table;      // the sequence's block-table row, or null
  int64_t base;              // kv_start
  int64_t max_page;
  int BK;
  int lg_bpp;                // log2 of key blocks per page
  // first key row of block b, given the page id of its page
  __device__ __forceinline__ int64_t block_row(int64_t page, int b) const {
    page = page < 0 ? 0 : (page > max_page ? max_page : page);
    return (page << lg_bpp) * BK + static_cast<int64_t>(b & ((1 << lg_bpp) - 1)) * BK;
  }
  __device__ __forceinline__ int page_index(int b) const { return b >> lg_bpp; }
  // PAGED fixes the layout at compile time (hot loops); row() decides at run time
  template <bool PAGED>
  __device__ __forceinline__ int64_t row_as(int b) const {
    if constexpr (PAGED) {
      return block_row(table[page_index(b)], b);
    } else {
      return base + static_cast<int64_t>(b) * BK;
    }
  }
  __device__ __forceinline__ int64_t row(int b) const { return table ? row_as<true>(b) : row_as<false>(b); }
};
__device__ __forceinline__ KeyBlocks key_blocks(const msa_seqs& sq, const SeqGeom& g, int s, int BK) {
  KeyBlocks kb;
  kb.table = sq.block_table ? sq.block_table + static_cast<int64_t>(s) * sq.block_table_stride : nullptr;
  kb.base = g.kv_start;
  kb.BK = BK;
  kb.lg_bpp = 0;
  if (sq.block_table)
    while ((BK << kb.lg_bpp) < sq.page_size) ++kb.lg_bpp;
  kb.max_page = sq.block_table ? sq.total_kv_rows / sq.page_size - 1 : 0;
  return kb;
}

}  // namespace msa

// ---------------------------------------------------------------- host helpers
namespace msa_host {

inline bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

inline int validate_seqs(const msa_seqs* s) {
  if (!s) return MSA_ERR_INVALID;
  if (s->num_seqs < 1 || s->total_q_rows < 0 || s->total_kv_rows < 0 || s->max_q_rows < 0 ||
      s->max_kv_len < 0)
    return MSA_ERR_INVALID;
  if (!s->q_offsets || !s->kv_lens) return MSA_ERR_INVALID;
  if (s->block_table) {
    if (s->block_table_stride < 1 || s->page_size < 1) return MSA_ERR_INVALID;
    if (s->max_kv_len > static_cast<int64_t>(s->block_table_stride) * s->page_size) return MSA_ERR_INVALID;
    if (s->total_kv_rows < s->page_size) return MSA_ERR_INVALID;
  } else if (!s->kv_starts) {
    return MSA_ERR_INVALID;
  }
  if (s->max_q_rows > s->max_kv_len) return MSA_ERR_INVALID;
  if (s->total_q_rows > (int64_t)s->num_seqs * s->max_q_rows) return MSA_ERR_INVALID;
  if (s->total_q_rows >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  return MSA_OK;
}

// A paged key side is accepted by calls that address keys per block; a page
// holds 1, 2, 4, ... or 64 key blocks.
inline int check_paged(const msa_seqs* s, int block_size, bool supported) {
  if (!s->block_table) return MSA_OK;
  if (!supported) return MSA_ERR_UNSUPPORTED;
  // pages of 2^j key blocks, j <= 6
  for (int j = 0; j <= 6; ++j)
    if (s->page_size == (block_size << j)) return MSA_OK;
  return MSA_ERR_INVALID;
}

inline int launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? MSA_OK : MSA_ERR_HIP;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace msa_host
