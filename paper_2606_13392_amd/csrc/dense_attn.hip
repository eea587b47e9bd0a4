// Dense causal GQA attention on gfx950: the baseline the sparse path is
// measured against.  Every query attends to all causally visible keys of its
// sequence (the full-attention form that MSA's sparse-attention equation of
// Sec. 3.1 reduces to when k covers every causal block), with the layout
// conventions of the sparse calls.
//
// Prefill (dense_prefill_kernel), FlashAttention-2 order: a CTA owns one KV
// group and a tile of consecutive query rows whose G heads share the group's
// K and V; its 8 waves hold 32 (query row, head) rows each, one CTA per CU.
// Key blocks of 64 are copied into a double-buffered LDS ring by DMA
// (global_load_lds, one block ahead, rows stored with a bank-conflict-free
// segment permutation); per block each wave computes S^T = K Q^T and
// O^T += V^T P^T with MFMA 32x32x16, the V^T operand read down V's columns
// with transposing LDS reads.  The O MFMAs of block b are interleaved by
// hand with the online softmax of block b+1 (running max and sum per row in
// registers, raw hardware exp2, row sums by bf16 dot products over the same
// rounded weights that multiply V).
//
// Decode (at most four query rows per sequence) runs the row kernel of the
// sparse decode call over every key block (msa_rows_dense).
#include <algorithm>
#include <type_traits>

#include "msa_common.h"
#include "msa_profile.h"

// every key block of each row, split over waves and CTAs (sparse_attn.hip)
size_t msa_rows_dense_workspace_size(const msa_seqs* seqs, int H_q, int H_kv);
int msa_rows_dense(const void* q, const void* k, const void* v, const msa_seqs* seqs, int H_q, int H_kv,
                   float scale, void* o, float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream);

namespace {

using namespace msa;

constexpr int kHeadDim = 128;
constexpr int kBK = 64;                  // keys per streamed block
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kDecodeRows = 4;           // sequences with at most this many query rows take the row kernel
constexpr int kWaves = 8;                // waves per CTA (32 MFMA rows each), one CTA per CU
constexpr int kThreads = kWaves * kWave;
constexpr int kAhead = 3;                // LDS operand reads issued this many MFMA slots ahead

// Key blocks in LDS, row-major, 16-byte segments permuted per row (an XOR
// with a row-dependent mask) so that every read pattern is free of bank
// conflicts whether the LDS serves 16 or 32 lanes of a wave per cycle:
//   K (16 bytes per lane: 32 consecutive rows x the two segments of a k-step)
//     segment s of row r at s ^ (2 (r & 7) + ((r >> 3) & 1));
//   V (ds_read_tr16_b64: 4 consecutive rows x 4 adjacent segments per 32
//     lanes) segment s of row r at s ^ 4 (r & 3).
struct DenseRing {
  uint16_t k[2][kBK * kHeadDim];
  uint16_t v[2][kBK * kHeadDim];
};
__device__ __forceinline__ int k_seg(int r, int s) { return s ^ (((r & 7) << 1) | ((r >> 3) & 1)); }
__device__ __forceinline__ int v_seg(int r, int s) { return s ^ ((r & 3) << 2); }

// tile_off[s] = query tiles before sequence s (tiles of qt rows).
__global__ __launch_bounds__(256) void dense_tile_offsets_kernel(msa_seqs sq, int qt, int32_t* __restrict__ tile_off) {
  __shared__ int32_t part[256];
  const int t = threadIdx.x;
  const int S = sq.num_seqs;
  const int per = (S + 255) / 256;
  const int s0 = t * per, s1 = min(S, s0 + per);
  auto tiles = [&](int s) -> int32_t {
    const int rows = sq.q_offsets[s + 1] - sq.q_offsets[s];
    return rows > 0 ? (rows + qt - 1) / qt : 0;
  };
  int32_t acc = 0;
  for (int s = s0; s < s1; ++s) acc += tiles(s);
  part[t] = acc;
  __syncthreads();
  if (t == 0) {
    int32_t run = 0;
    for (int i = 0; i < 256; ++i) { const int32_t x = part[i]; part[i] = run; run += x; }
    tile_off[S] = run;
  }
  __syncthreads();
  acc = part[t];
  for (int s = s0; s < s1; ++s) { tile_off[s] = acc; acc += tiles(s); }
}

// lsum + lo + hi of a packed bf16 pair (v_dot2c_f32_bf16 against (1, 1)):
// the row sum is taken over the same rounded weights that multiply V.
__device__ __forceinline__ float add_bf16_pair(float lsum, uint32_t pair) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2v;
  const bf16x2v ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v, pair), ones, lsum, false);
}
__device__ __forceinline__ float xor32f(float x) {
  return __builtin_bit_cast(float, xor_lane_u32<32>(__builtin_bit_cast(uint32_t, x)));
}
__device__ __forceinline__ uint2 lds_tr4(const uint16_t* p) {
  typedef __attribute__((__vector_size__(4 * sizeof(short)))) short v4i16;
  const v4i16 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) v4i16*)(v4i16*)(const_cast<uint16_t*>(p)));
  return __builtin_bit_cast(uint2, x);
}
// global_load_lds: lane l's 16 bytes land at dst + 16 l (dst wave-uniform).
__device__ __forceinline__ void dma16(const uint16_t* src, uint16_t* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}

// Per-lane byte offsets of one key block's DMA (global side, relative to
// the block's first key row) and of the MFMA operand reads (LDS side,
// relative to a ring buffer), fixed for the whole kernel.
struct DenseLaneOffsets {
  uint32_t kg[kBK / 4 / kWaves], vg[kBK / 4 / kWaves];   // DMA sources: row * stride + 16-byte segment
  uint32_t ks[kHeadDim / 16];                            // K operand, k-step st (rows 32i add 8 KiB)
  uint32_t vs[kHeadDim / 32];                            // V^T operand, dim tile td (row offsets are immediates)
};

// grid: (tiles, H_kv); tiles are taken last-first so the longest causal
// ranges start first.  Per iteration b (one barrier): the DMA for K_{b+2}
// and V_{b+1} is issued, S^T_{b+1} = K_{b+1} Q^T and O^T += V_b^T P_b^T are
// issued on the MFMA pipe, and the softmax of S_{b+1} runs on the VALU while
// the O MFMAs drain.
__global__ __launch_bounds__(kThreads, 1) void dense_prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, msa_seqs sq,
    const int32_t* __restrict__ tile_off, int H_q, int H_kv, int ntile_grid, float scale_log2,
    uint16_t* __restrict__ o, float* __restrict__ lse) {
  __shared__ __align__(16) DenseRing ring;
  constexpr int MT = kBK / 32;             // 32-key tiles of S^T
  constexpr int KS = kHeadDim / 16;        // k-steps of S^T = K Q^T
  constexpr int NDMA = kBK / 4 / kWaves;   // DMA instructions per wave per block and tensor
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int n = lane & 31, h = lane >> 5;
  const int G = H_q / H_kv;
  const int qpw = 32 / G;                  // query rows per wave
  const int qt = kWaves * qpw;             // query rows per CTA
  const int jq = n / G, hh = n % G;
  const int r = blockIdx.y;
  const int tile = ntile_grid - 1 - static_cast<int>(blockIdx.x);
  if (tile >= tile_off[sq.num_seqs]) return;              // uniform over the CTA
  const int s = find_seq_wave(tile_off, sq.num_seqs, tile);
  const SeqGeom g = seq_geom(sq, s);
  const int t0 = (tile - tile_off[s]) * qt;
  const int t_end = min(t0 + qt, g.q_rows);
  const int p_last = g.kv_len - g.q_rows + t_end - 1;
  if (p_last < 0 || t0 >= g.q_rows) return;               // uniform
  const int nblk = p_last / kBK + 1;

  const int t = t0 + wave * qpw + jq;                     // this lane's query row in the sequence
  const bool valid = n < qpw * G && t < t_end;
  const int p = valid ? g.kv_len - g.q_rows + t : -1;
  // smallest position among the wave's rows (invalid lanes see every key masked anyway);
  // blocks below nfree are visible to every row of the wave and need no mask
  const int p_wave = g.kv_len - g.q_rows + min(t0 + wave * qpw, t_end - 1);
  const int nfree = (p_wave + 1) / kBK;
  const int64_t head_row = (static_cast<int64_t>(g.q_begin) + (valid ? t : t0)) * H_q + static_cast<int64_t>(r) * G + hh;

  const int64_t stride = static_cast<int64_t>(H_kv) * kHeadDim;
  const char* kb = reinterpret_cast<const char*>(k + g.kv_start * stride + static_cast<int64_t>(r) * kHeadDim);
  const char* vb = reinterpret_cast<const char*>(v + g.kv_start * stride + static_cast<int64_t>(r) * kHeadDim);
  const uint32_t stride_b = static_cast<uint32_t>(stride) * 2;

  DenseLaneOffsets lo;
  {
    const int gq = lane >> 4, jj = lane & 15;
#pragma unroll
    for (int c = 0; c < NDMA; ++c) {
      const int ra = 4 * (c * kWaves + wave) + gq;
      lo.kg[c] = ra * stride_b + 16 * k_seg(ra, jj);        // the permutations are involutions
      lo.vg[c] = ra * stride_b + 16 * v_seg(ra, jj);
    }
#pragma unroll
    for (int st = 0; st < KS; ++st) lo.ks[st] = 2 * (n * kHeadDim + 8 * k_seg(n, 2 * st + h));
    // V^T operand: in each 16-lane group, lane j addresses row k0 + j/4, dims
    // n0 + 4(j%4) .. +3 of V and receives rows k0 .. k0+3 of dim n0 + j
    // (ds_read_tr16_b64); row r_l = 4h + j/4 within each 16-key k-step (rows
    // 16u + r_l and + 8 share the permutation)
    const int rl = 4 * h + (jj >> 2);
#pragma unroll
    for (int td = 0; td < kHeadDim / 32; ++td) {
      const int col = 32 * td + 16 * (gq & 1) + 4 * (jj & 3);
      lo.vs[td] = 2 * (rl * kHeadDim + 8 * v_seg(rl, col >> 3) + (col & 7));
    }
  }
  // One key block (K and / or V) into LDS by DMA: each wave instruction fills
  // 4 rows (1 KiB); lane l takes row 4 piece + l / 16 and the logical segment
  // that the row's permutation stores at physical segment l % 16.  In a block
  // running past kv_len the missing rows re-read the last key (finite values
  // whose scores are masked).
  auto dma = [&](const char* base, const uint32_t (&go)[NDMA], bool is_v, int key0, uint16_t* dst) {
    const char* blk = base + static_cast<int64_t>(key0) * stride_b;
    if (key0 + kBK <= g.kv_len) {
#pragma unroll
      for (int c = 0; c < NDMA; ++c)
        dma16(reinterpret_cast<const uint16_t*>(blk + go[c]), dst + 4 * (c * kWaves + wave) * kHeadDim);
    } else {
#pragma unroll
      for (int c = 0; c < NDMA; ++c) {
        const int ra = 4 * (c * kWaves + wave) + (lane >> 4);
        const int rr = min(ra, g.kv_len - 1 - key0);
        const uint32_t off = rr * stride_b + 16 * (is_v ? v_seg(ra, lane & 15) : k_seg(ra, lane & 15));
        dma16(reinterpret_cast<const uint16_t*>(blk + off), dst + 4 * (c * kWaves + wave) * kHeadDim);
      }
    }
  };
  dma(kb, lo.kg, false, 0, ring.k[0]);
  dma(vb, lo.vg, true, 0, ring.v[0]);
  if (nblk > 1) dma(kb, lo.kg, false, kBK, ring.k[1]);

  bf16x8 bq[KS];
  {
    const uint16_t* qrow = q + head_row * kHeadDim + 8 * h;
#pragma unroll
    for (int st = 0; st < KS; ++st) bq[st] = valid ? ld_bf16x8(qrow + 16 * st) : zero_bf16x8();
  }

  // S^T = K Q^T on one key block: lane (n, h) gets keys 32i + 8(e/4) + 4h + e%4 of row n
  auto scores = [&](const uint16_t* kbuf, f32x16 (&acc_s)[MT]) {
    const char* kbb = reinterpret_cast<const char*>(kbuf);
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      acc_s[i] = f32x16{};
#pragma unroll
      for (int st = 0; st < KS; ++st)
        acc_s[i] = mfma32x32x16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(
                                    kbb + lo.ks[st] + 2 * 32 * i * kHeadDim)),
                                bq[st], acc_s[i]);
    }
  };

  f32x16 acc_o[kHeadDim / 32];
#pragma unroll
  for (int i = 0; i < kHeadDim / 32; ++i) acc_o[i] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;
  // P of the pending block in bf16, as the B operand of O^T = V^T P^T: k-step
  // u covers keys 32(u/2) + 16(u%2) + {4h + e, 8 + 4h + e}, e = 0..3
  bf16x8 bp[kBK / 16];

  // online softmax of one block's scores (raw units; scale_log2 > 0 keeps
  // the order): updates m_run / l_run, leaves P in bp, returns alpha
  auto softmax = [&](f32x16 (&acc_s)[MT], int key0, auto masked) -> float {
    if constexpr (decltype(masked)::value) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = key0 + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
          acc_s[i][e] = key <= p ? acc_s[i][e] : -INFINITY;
        }
    }
    float bmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) bmax = fmaxf(bmax, acc_s[i][e]);
    bmax = fmaxf(bmax, xor32f(bmax));
    const float m_new = fmaxf(m_run, bmax);
    const float mm = m_new == -INFINITY ? 0.f : m_new;     // rows with nothing visible yet
    const float alpha = exp2_hw((m_run - mm) * scale_log2);
    const float neg = -mm * scale_log2;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc_s[i][e] = exp2_hw(fmaf(acc_s[i][e], scale_log2, neg));
    float lsum = 0.f;
#pragma unroll
    for (int u = 0; u < kBK / 16; ++u) {
      uint4 pw;
      const int i = u >> 1, e0 = 8 * (u & 1);
      pw.x = pack_bf16x2(acc_s[i][e0 + 0], acc_s[i][e0 + 1]);
      pw.y = pack_bf16x2(acc_s[i][e0 + 2], acc_s[i][e0 + 3]);
      pw.z = pack_bf16x2(acc_s[i][e0 + 4], acc_s[i][e0 + 5]);
      pw.w = pack_bf16x2(acc_s[i][e0 + 6], acc_s[i][e0 + 7]);
      lsum = add_bf16_pair(add_bf16_pair(add_bf16_pair(add_bf16_pair(lsum, pw.x), pw.y), pw.z), pw.w);
      bp[u] = __builtin_bit_cast(bf16x8, pw);
    }
    lsum += xor32f(lsum);
    l_run = l_run * alpha + lsum;
    m_run = m_new;
    return alpha;
  };

  // O^T += V^T P^T from one value block (A operand read down V's columns)
  auto pv = [&](const uint16_t* vbuf) {
    const char* vbb = reinterpret_cast<const char*>(vbuf);
#pragma unroll
    for (int u = 0; u < kBK / 16; ++u) {
      const int row0 = 32 * (u >> 1) + 16 * (u & 1);
#pragma unroll
      for (int td = 0; td < kHeadDim / 32; ++td) {
        const char* a0 = vbb + lo.vs[td] + 2 * row0 * kHeadDim;
        const uint2 x0 = lds_tr4(reinterpret_cast<const uint16_t*>(a0));
        const uint2 x1 = lds_tr4(reinterpret_cast<const uint16_t*>(a0 + 2 * 8 * kHeadDim));  // rows +8: same permutation
        acc_o[td] = mfma32x32x16(__builtin_bit_cast(bf16x8, make_uint4(x0.x, x0.y, x1.x, x1.y)), bp[u], acc_o[td]);
      }
    }
  };

  // iteration b: K_{b+1} is in k[(b+1)&1], V_b in v[b&1]
  // Iteration b (K_{b+1} in k[(b+1)&1], V_b in v[b&1]), laid out by hand as
  // 32 MFMA slots, each fenced off from the next so that the compiler keeps
  // the order: O is first rescaled by block b's alpha (only when some row's
  // maximum moved); slots 0..15 issue S^T_{b+1} = K_{b+1} Q^T, slots 16..31
  // O^T += V_b^T P_b^T with one sixteenth of block b+1's softmax after each
  // MFMA, so the VALU works while the MFMA pipe drains; LDS operands are read
  // kAhead slots before their MFMA.
  float alpha_pend = 0.f;                 // alpha of the block whose P is in bp
  auto step = [&](int b, auto masked) {
    __builtin_amdgcn_s_waitcnt(0);        // this thread's copies of K_{b+1} and V_b have landed
    __syncthreads();                      // everyone's have, and block b-1's readers are done
    if (b + 2 < nblk) dma(kb, lo.kg, false, (b + 2) * kBK, ring.k[b & 1]);
    dma(vb, lo.vg, true, (b + 1) * kBK, ring.v[(b + 1) & 1]);
    const char* kbb = reinterpret_cast<const char*>(ring.k[(b + 1) & 1]);
    const char* vbb = reinterpret_cast<const char*>(ring.v[b & 1]);
    if (__ballot(alpha_pend != 1.f)) {    // some row's maximum moved with block b
#pragma unroll
      for (int i = 0; i < kHeadDim / 32; ++i) acc_o[i] *= alpha_pend;
    }
    __builtin_amdgcn_sched_barrier(0);

    constexpr int NS = MT * KS;           // S^T slots
    auto kread = [&](int j) -> bf16x8 {
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kbb + lo.ks[j % KS] + 2 * 32 * (j / KS) * kHeadDim));
    };
    f32x16 acc_s[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc_s[i] = f32x16{};
    bf16x8 kr[NS];
#pragma unroll
    for (int j = 0; j < kAhead; ++j) kr[j] = kread(j);
#pragma unroll
    for (int j = 0; j < NS; ++j) {
      if (j + kAhead < NS) kr[j + kAhead] = kread(j + kAhead);
      acc_s[j / KS] = mfma32x32x16(kr[j], bq[j % KS], acc_s[j / KS]);
      __builtin_amdgcn_sched_barrier(0);
    }

    constexpr int NO = (kBK / 16) * (kHeadDim / 32);   // O^T slots
    auto vread = [&](int j) -> bf16x8 {
      const int u = j / (kHeadDim / 32), td = j % (kHeadDim / 32);
      const char* a0 = vbb + lo.vs[td] + 2 * (32 * (u >> 1) + 16 * (u & 1)) * kHeadDim;
      const uint2 x0 = lds_tr4(reinterpret_cast<const uint16_t*>(a0));
      const uint2 x1 = lds_tr4(reinterpret_cast<const uint16_t*>(a0 + 2 * 8 * kHeadDim));
      return __builtin_bit_cast(bf16x8, make_uint4(x0.x, x0.y, x1.x, x1.y));
    };
    bf16x8 vr[NO];
    bf16x8 bp_next[kBK / 16];
#pragma unroll
    for (int j = 0; j < kAhead; ++j) vr[j] = vread(j);
    const int key0 = (b + 1) * kBK;
    float m0 = -INFINITY, m_new = 0.f, alpha = 0.f, neg = 0.f, lsum = 0.f;
#pragma unroll
    for (int j = 0; j < NO; ++j) {
      if (j + kAhead < NO) vr[j + kAhead] = vread(j + kAhead);
      acc_o[j % (kHeadDim / 32)] = mfma32x32x16(vr[j], bp[j / (kHeadDim / 32)], acc_o[j % (kHeadDim / 32)]);
      if (j == 0) {
        if constexpr (decltype(masked)::value) {
#pragma unroll
          for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int key = key0 + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
              acc_s[i][e] = key <= p ? acc_s[i][e] : -INFINITY;
            }
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) m0 = fmaxf(m0, acc_s[0][e]);
      } else if (j == 1) {
#pragma unroll
        for (int e = 0; e < 16; ++e) m0 = fmaxf(m0, acc_s[1][e]);
        m0 = fmaxf(m0, xor32f(m0));
        m_new = fmaxf(m_run, m0);
        const float mm = m_new == -INFINITY ? 0.f : m_new;   // rows with nothing visible yet
        alpha = exp2_hw((m_run - mm) * scale_log2);
        neg = -mm * scale_log2;
      } else if (j < 14) {
#pragma unroll
        for (int x = 0; x < 32; ++x) {
          if (2 + (3 * x) / 8 != j) continue;
          acc_s[x >> 4][x & 15] = exp2_hw(fmaf(acc_s[x >> 4][x & 15], scale_log2, neg));
        }
      } else {
#pragma unroll
        for (int u = 2 * (j - 14); u < 2 * (j - 14) + 2; ++u) {
          uint4 pw;
          const int i = u >> 1, e0 = 8 * (u & 1);
          pw.x = pack_bf16x2(acc_s[i][e0 + 0], acc_s[i][e0 + 1]);
          pw.y = pack_bf16x2(acc_s[i][e0 + 2], acc_s[i][e0 + 3]);
          pw.z = pack_bf16x2(acc_s[i][e0 + 4], acc_s[i][e0 + 5]);
          pw.w = pack_bf16x2(acc_s[i][e0 + 6], acc_s[i][e0 + 7]);
          lsum = add_bf16_pair(add_bf16_pair(add_bf16_pair(add_bf16_pair(lsum, pw.x), pw.y), pw.z), pw.w);
          bp_next[u] = __builtin_bit_cast(bf16x8, pw);
        }
        if (j == 15) {
          lsum += xor32f(lsum);
          l_run = l_run * alpha + lsum;
          m_run = m_new;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int u = 0; u < kBK / 16; ++u) bp[u] = bp_next[u];
    alpha_pend = alpha;
  };

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  {
    f32x16 acc_s[MT];
    scores(ring.k[0], acc_s);
    alpha_pend = nfree > 0 ? softmax(acc_s, 0, std::false_type{}) : softmax(acc_s, 0, std::true_type{});
  }
  int b = 0;
  for (; b + 1 < min(nfree, nblk); ++b) step(b, std::false_type{});
  for (; b + 1 < nblk; ++b) step(b, std::true_type{});
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (__ballot(alpha_pend != 1.f)) {
#pragma unroll
    for (int i = 0; i < kHeadDim / 32; ++i) acc_o[i] *= alpha_pend;
  }
  pv(ring.v[b & 1]);

  if (!valid) return;
  const bool empty = !(l_run > 0.f);
  const float inv_l = empty ? 0.f : 1.f / l_run;
  // O^T tile td: lane (n, h) holds d = 32td + 8(e/4) + 4h + e%4 of row n
  uint16_t* orow = o + head_row * kHeadDim + 4 * h;
#pragma unroll
  for (int td = 0; td < kHeadDim / 32; ++td)
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      uint2 w;
      w.x = pack_bf16x2(acc_o[td][4 * e4 + 0] * inv_l, acc_o[td][4 * e4 + 1] * inv_l);
      w.y = pack_bf16x2(acc_o[td][4 * e4 + 2] * inv_l, acc_o[td][4 * e4 + 3] * inv_l);
      *reinterpret_cast<uint2*>(orow + 32 * td + 8 * e4) = w;
    }
  if (h == 0) lse[head_row] = empty ? -INFINITY : (m_run * scale_log2 + __log2f(l_run)) * kLn2;
}

int validate_dense(const msa_seqs* seqs, int H_q, int H_kv, int head_dim) {
  int st = msa_host::validate_seqs(seqs);
  if (st != MSA_OK) return st;
  if (H_q < 1 || H_kv < 1 || head_dim < 1 || H_q % H_kv != 0) return MSA_ERR_INVALID;
  if (head_dim != kHeadDim) return MSA_ERR_UNSUPPORTED;
  if (H_q / H_kv > 16 || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (seqs->total_q_rows * H_kv >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  if (seqs->block_table) return MSA_ERR_UNSUPPORTED;   // contiguous key side only
  return MSA_OK;
}

bool decode_like(const msa_seqs* seqs) { return seqs->max_q_rows <= kDecodeRows; }

}  // namespace

extern "C" size_t msa_dense_attn_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                               int head_dim) {
  if (validate_dense(seqs, num_q_heads, num_kv_heads, head_dim) != MSA_OK) return 0;
  if (decode_like(seqs)) return msa_rows_dense_workspace_size(seqs, num_q_heads, num_kv_heads);
  return msa_host::align_up(sizeof(int32_t) * (seqs->num_seqs + 1), 256);
}

extern "C" int msa_dense_attn(const void* q, const void* k, const void* v, const msa_seqs* seqs, int num_q_heads,
                              int num_kv_heads, int head_dim, float softmax_scale, void* o, float* lse,
                              void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = validate_dense(seqs, num_q_heads, num_kv_heads, head_dim);
  if (st != MSA_OK) return st;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if (!q || !k || !v || !o || !lse) return MSA_ERR_INVALID;
  const float scale = softmax_scale * kLog2e;
  if (decode_like(seqs))
    return msa_rows_dense(q, k, v, seqs, num_q_heads, num_kv_heads, softmax_scale, o, lse, workspace,
                          workspace_bytes, stream);
  const size_t need = msa_host::align_up(sizeof(int32_t) * (seqs->num_seqs + 1), 256);
  if (!workspace || workspace_bytes < need) return MSA_ERR_WORKSPACE;
  const int G = num_q_heads / num_kv_heads;
  const int qt = kWaves * (32 / G);
  // every sequence contributes at most q_rows / qt + 1 tiles
  const int64_t ntile = seqs->total_q_rows / qt + seqs->num_seqs;
  if (ntile >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  auto* tile_off = static_cast<int32_t*>(workspace);
  const msa_seqs sq = *seqs;
  msa_prof::launch("dense_tile_offsets_kernel", dense_tile_offsets_kernel, dim3(1), dim3(256), 0, stream, sq, qt,
                   tile_off);
  msa_prof::launch("dense_prefill_kernel", dense_prefill_kernel, dim3(static_cast<unsigned>(ntile), num_kv_heads),
                   dim3(kThreads), 0, stream, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                   static_cast<const uint16_t*>(v), sq, static_cast<const int32_t*>(tile_off), num_q_heads,
                   num_kv_heads, static_cast<int>(ntile), scale, static_cast<uint16_t*>(o), lse);
  return msa_host::launch_status();
}
