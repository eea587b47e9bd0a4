// Main Branch of MSA on gfx950: exact softmax attention over the causally
// visible tokens of the selected key blocks (Sec. 3.1, sparse-attention
// equation), returning O and the natural-log LSE.
//
// attn_rows_kernel: one CTA of four waves per (query row, group, split); each
// wave takes its own share of the group's selected blocks.  The G query heads
// of the group share the group's block list (Sec. 2.3, group-shared index
// set), so one wave computes S^T = K Q^T for all of them with MFMA 16x16x32
// (keys as M, heads as N, head_dim as K), keeps an online softmax per head in
// registers (each lane owns one head's column) and accumulates O^T = V^T P^T
// with V staged transposed in its own LDS area.  The four waves then merge
// their states through LDS with the log-sum-exp rule of Sec. 4.2 ("Two-phase
// forward").  With several splits per row the CTA writes a locally normalised
// partial that combine_kernel merges by the same rule.
#include "msa_common.h"
#include "msa_profile.h"

namespace {

using namespace msa;

constexpr int kHeadDim = 128;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

constexpr int kAttnWaves = 4;                 // waves per CTA, each with its own block share
constexpr int kRedStride = kHeadDim + 4;      // fp32 row stride of the merge buffer

constexpr int kKRowPad = kHeadDim + 8;       // bf16 K rows staged with 16 bytes of padding

template <int BK>
struct AttnSmem {
  union {                                        // kr: 64-key bf16 blocks only
    // bf16 K of one block, row-major kr[key][d]: the rows arrive as whole
    // 256-byte rows (16 lanes per row) and are read back as MFMA operands
    uint16_t kr[BK == 64 ? BK : 1][kKRowPad];
    // E4M3 K of one 64-key block, row-major kr8[key][d] (+16 B pad per row)
    uint8_t kr8[BK == 64 ? BK : 1][kHeadDim + 16];
    // V of one block, transposed: vt[d][key]; +4 keys of padding per row.
    // After the block loop the same bytes hold the wave's scaled O (16 x
    // kRedStride fp32).
    uint16_t vt[kHeadDim][BK + 4];
  };
};
static_assert(sizeof(AttnSmem<64>) >= 16 * kRedStride * sizeof(float), "merge buffer does not fit");

// Orders a wave's own LDS accesses (a wave's LDS operations complete in issue
// order; this keeps the compiler from moving them across).
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// V[b*BK .. b*BK+BK) of group r: each lane loads 4 keys x 8 dims per
// (4-key group, 8-dim group) pair; keys past the sequence's end read as zero.
template <int BK, typename T>
__device__ __forceinline__ void load_v_raw(const T* __restrict__ vbase, int64_t row_stride, int key0,
                                           int kv_len, Raw<T> (&raw)[BK / 16][4]) {
  const int lane = lane_id();
#pragma unroll
  for (int it = 0; it < BK / 16; ++it) {
    const int q = lane + kWave * it;        // (4-key group, 8-dim group)
    const int key4 = q >> 4, dg = q & 15;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int key = key0 + 4 * key4 + j;
      raw[it][j] = key < kv_len ? load_raw(vbase + static_cast<int64_t>(key) * row_stride + 8 * dg) : Raw<T>{};
    }
  }
}
// ... and stores them (widened to bf16) transposed into LDS as vt[d][key].
template <int BK, typename R>
__device__ __forceinline__ void store_v_transposed(AttnSmem<BK>& sm, const R (&raw_in)[BK / 16][4]) {
  const int lane = lane_id();
#pragma unroll
  for (int it = 0; it < BK / 16; ++it) {
    const int q = lane + kWave * it;
    const int key4 = q >> 4, dg = q & 15;
    u32x4 raw[1][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) raw[0][j] = widen(raw_in[it][j]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int w = e >> 1, sh = (e & 1) * 16;
      uint2 x;
      x.x = ((raw[0][0][w] >> sh) & 0xFFFFu) | (((raw[0][1][w] >> sh) & 0xFFFFu) << 16);
      x.y = ((raw[0][2][w] >> sh) & 0xFFFFu) | (((raw[0][3][w] >> sh) & 0xFFFFu) << 16);
      *reinterpret_cast<uint2*>(&sm.vt[8 * dg + e][4 * key4]) = x;
    }
  }
}

// T: element type of Q, K and V (uint16_t = bf16 bits, uint8_t = e4m3 bits);
// o_scale multiplies O (the V dequantisation scale for e4m3).
template <int BK, typename T, bool PAGED>
// (64-key bf16 blocks on a contiguous cache fit 2 CTAs per CU in 256
// registers: 108 -> 106 us per 128K step against one wave per SIMD.)
__global__ __launch_bounds__(64 * kAttnWaves, (BK == 64 && sizeof(T) == 2 && !PAGED) ? 2 : 1) void attn_rows_kernel(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const int32_t* __restrict__ block_ids, msa_seqs sq, int H_q, int H_kv, int topk,
    int slots_per_wave, float scale_log2, float o_scale, uint16_t* __restrict__ o, float* __restrict__ lse,
    float* __restrict__ o_part, float* __restrict__ lse_part) {
  __shared__ __align__(16) AttnSmem<BK> smw[kAttnWaves];
  __shared__ float mls[kAttnWaves][2][16];
  const int lane = lane_id();
  const int wv = threadIdx.x / kWave;
  AttnSmem<BK>& sm = smw[wv];
  const int G = H_q / H_kv;
  const int64_t row = blockIdx.x / H_kv;
  const int r = blockIdx.x % H_kv;
  const int sp = blockIdx.y;
  const int nsplit = gridDim.y;
  if (row >= sq.total_q_rows) return;                // uniform over the CTA
  const int s = find_seq_wave(sq.q_offsets, sq.num_seqs, row);
  const SeqGeom g = seq_geom(sq, s);
  int p = g.kv_len - g.q_rows + static_cast<int>(row - g.q_begin);
  if (p >= g.kv_len) p = -1;                        // inconsistent layout: attend to nothing

  const int n = lane & 15, q4 = lane >> 4;
  // B operand of S^T = K Q^T: head n of the group, dims 32*ks + 8*q4 .. +8.
  bf16x8 bq[kHeadDim / 32];
  const T* qrow = q + (row * H_q + static_cast<int64_t>(r) * G + n) * kHeadDim + 8 * q4;
#pragma unroll
  for (int ks = 0; ks < kHeadDim / 32; ++ks) bq[ks] = widen_bf16x8(n < G ? load_raw(qrow + 32 * ks) : Raw<T>{});

  const int64_t kv_stride = static_cast<int64_t>(H_kv) * kHeadDim;
  const KeyBlocks kbk = key_blocks(sq, g, s, BK);
  const int64_t seq0 = PAGED ? 0 : g.kv_start;           // contiguous: keys from kv_start
  const T* kbase = k + seq0 * kv_stride + static_cast<int64_t>(r) * kHeadDim + 8 * q4;
  const T* krow_base = k + seq0 * kv_stride + static_cast<int64_t>(r) * kHeadDim;   // row starts
  const T* vbase = v + seq0 * kv_stride + static_cast<int64_t>(r) * kHeadDim;
  // without block ids (dense mode) slot b is key block b
  const int32_t* ids = block_ids ? block_ids + (row * H_kv + r) * topk : nullptr;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 acc[kHeadDim / 16];
#pragma unroll
  for (int t = 0; t < kHeadDim / 16; ++t) acc[t] = f32x4{};

  const int slot0 = min(topk, (sp * kAttnWaves + wv) * slots_per_wave);
  const int slot1 = min(topk, slot0 + slots_per_wave);
  // the wave's block ids, one per lane, fetched at once (slots_per_wave <= 64 with ids)
  const int my_b = ids && slot0 + lane < slot1 ? ids[slot0 + lane] : -1;
  // paged: each lane fetches the page of its slot's block up front (no table
  // read between a block's id and its loads)
  int32_t my_pg = 0;
  if constexpr (PAGED) {
    const int bb = ids ? my_b : slot0 + lane;
    if (p >= 0 && slot0 + lane < slot1 && bb >= 0 && bb <= p / BK) my_pg = kbk.table[kbk.page_index(bb)];
  }
  // 64-key blocks: each load instruction takes whole K rows (bf16: 4 rows of
  // 256 bytes, 16 lanes per row; E4M3: 8 rows of 128 bytes) -- the rows are
  // scattered at the cache's token stride, and whole rows per instruction are
  // served faster than 64- or 32-byte pieces of 16 rows -- and the block goes
  // through LDS into the MFMA operand layout (bf16: 111 -> 107 us per 128K
  // decode step).  128-key blocks (equal or slower staged) load the operands
  // directly.
  constexpr bool kStageK = BK == 64;
  Raw<T> ka[BK / 16][kHeadDim / 32];
  u32x4 kw[sizeof(T) == 1 && kStageK ? BK / 8 : 1];     // E4M3 whole rows before staging
  Raw<T> vraw[BK / 16][4];
  // K and raw V of slot j (a valid slot of the current window) are requested;
  // the next valid slot's loads go out as soon as these registers are free
  // (K after the S^T MFMAs, V after its LDS staging), so they fly under this
  // block's softmax and O^T MFMAs.
  auto block_of = [&](int slot) { return ids ? __builtin_amdgcn_readlane(my_b, slot - slot0) : slot; };
  auto row_of = [&](int slot, int b) -> int64_t {
    return PAGED ? kbk.block_row(__builtin_amdgcn_readlane(my_pg, slot - slot0), b) : 0;
  };
  auto load_k = [&](int slot) {
    const int b = block_of(slot);
    const int key0 = b * BK;
    const int64_t page_row = row_of(slot, b);
    if constexpr (kStageK && sizeof(T) == 1) {
#pragma unroll
      for (int i = 0; i < BK / 8; ++i) {
        const int kr = 8 * i + (lane >> 3);                 // key row of this lane: lanes 8 (lane / 8) .. + 7
        const int key = key0 + kr;
        const T* kp = (PAGED ? krow_base + (page_row + kr) * kv_stride : krow_base + static_cast<int64_t>(key) * kv_stride) + 16 * (lane & 7);
        kw[i] = key < g.kv_len ? *reinterpret_cast<const u32x4*>(kp) : u32x4{};
      }
    } else if constexpr (kStageK) {
#pragma unroll
      for (int i = 0; i < BK / 16; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int kr = 16 * i + 4 * j + q4;            // key row of this lane: lanes 16 q4 .. + 15
          const int key = key0 + kr;
          const T* kp = (PAGED ? krow_base + (page_row + kr) * kv_stride : krow_base + static_cast<int64_t>(key) * kv_stride) + 8 * n;
          ka[i][j] = key < g.kv_len ? load_raw(kp) : Raw<T>{};
        }
    } else {
#pragma unroll
      for (int i = 0; i < BK / 16; ++i) {
        const int key = key0 + 16 * i + n;
        const T* kp = PAGED ? kbase + (page_row + 16 * i + n) * kv_stride : kbase + static_cast<int64_t>(key) * kv_stride;
#pragma unroll
        for (int ks = 0; ks < kHeadDim / 32; ++ks) ka[i][ks] = key < g.kv_len ? load_raw(kp + 32 * ks) : Raw<T>{};
      }
    }
  };
  auto load_v = [&](int slot) {
    const int b = block_of(slot);
    if constexpr (PAGED)
      load_v_raw<BK, T>(vbase + row_of(slot, b) * kv_stride, kv_stride, 0, g.kv_len - b * BK, vraw);
    else
      load_v_raw<BK, T>(vbase, kv_stride, b * BK, g.kv_len, vraw);
  };
  // windows of 64 slots (one slot per lane in the validity ballot)
  for (int w0 = slot0; w0 < slot1 && p >= 0; w0 += kWave) {
    const int bl = ids ? my_b : w0 + lane;
    const bool vl = w0 + lane < slot1 && bl >= 0 && bl <= p / BK;
    uint64_t pend = __ballot(vl);
    int slot = pend != 0ull ? w0 + __ffsll(static_cast<unsigned long long>(pend)) - 1 : -1;
    if (slot >= 0) {
      load_k(slot);
      load_v(slot);
    }
    while (slot >= 0) {
      pend &= pend - 1;
      const int next = pend != 0ull ? w0 + __ffsll(static_cast<unsigned long long>(pend)) - 1 : -1;
      const int b = block_of(slot);
      const int key0 = b * BK;
      if constexpr (kStageK && sizeof(T) == 1) {
        wave_lds_order();                               // the previous block's V^T reads are done
  #pragma unroll
        for (int i = 0; i < BK / 8; ++i) *reinterpret_cast<u32x4*>(&sm.kr8[8 * i + (lane >> 3)][16 * (lane & 7)]) = kw[i];
        wave_lds_order();                               // K staged
  #pragma unroll
        for (int i = 0; i < BK / 16; ++i)
  #pragma unroll
          for (int ks = 0; ks < kHeadDim / 32; ++ks)
            ka[i][ks] = *reinterpret_cast<const Raw<T>*>(&sm.kr8[16 * i + n][32 * ks + 8 * q4]);
      }
      if constexpr (kStageK && sizeof(T) == 2) {
        wave_lds_order();                               // the previous block's V^T reads are done
  #pragma unroll
        for (int i = 0; i < BK / 16; ++i)
  #pragma unroll
          for (int j = 0; j < 4; ++j)
            *reinterpret_cast<Raw<T>*>(&sm.kr[16 * i + 4 * j + q4][8 * n]) = ka[i][j];
        wave_lds_order();                               // K staged
  #pragma unroll
        for (int i = 0; i < BK / 16; ++i)
  #pragma unroll
          for (int ks = 0; ks < kHeadDim / 32; ++ks)
            ka[i][ks] = *reinterpret_cast<const Raw<T>*>(&sm.kr[16 * i + n][32 * ks + 8 * q4]);
      }
      // S^T tiles: keys 16i..16i+15 (rows) x heads (columns)
      f32x4 st[BK / 16];
  #pragma unroll
      for (int i = 0; i < BK / 16; ++i) {
        st[i] = f32x4{};
  #pragma unroll
        for (int ks = 0; ks < kHeadDim / 32; ++ks) st[i] = mfma16x16x32(widen_bf16x8(ka[i][ks]), bq[ks], st[i]);
      }
      if (next >= 0) load_k(next);
      // lane (n, q4) holds keys 16i + 4*q4 + e of head n
      float bmax = -INFINITY;
  #pragma unroll
      for (int i = 0; i < BK / 16; ++i)
  #pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = key0 + 16 * i + 4 * q4 + e;
          float z = st[i][e] * scale_log2;
          z = key <= p ? z : -INFINITY;
          st[i][e] = z;
          bmax = fmaxf(bmax, z);
        }
      bmax = fmaxf(bmax, __shfl_xor(bmax, 16));
      bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
      const float m_new = fmaxf(m_run, bmax);
      const float alpha = exp2_hw(m_run - m_new);
      float lsum = 0.f;
  #pragma unroll
      for (int i = 0; i < BK / 16; ++i)
  #pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pe = exp2_hw(st[i][e] - m_new);
          st[i][e] = pe;
          lsum += pe;
        }
      lsum += __shfl_xor(lsum, 16);
      lsum += __shfl_xor(lsum, 32);
      l_run = l_run * alpha + lsum;
      m_run = m_new;
  #pragma unroll
      for (int t = 0; t < kHeadDim / 16; ++t) acc[t] *= alpha;

      wave_lds_order();                                 // the previous block's V^T reads are done
      store_v_transposed<BK>(sm, vraw);
      if (next >= 0) load_v(next);
      // P^T as the B operand: k-step u covers keys 32u..32u+31; lane (n, q4)
      // supplies logical k = 8*q4 + e <-> key 32u + 4*q4 + e (e < 4) and
      // 32u + 16 + 4*q4 + e - 4 (e >= 4), exactly the keys its S^T tiles hold.
      wave_lds_order();                                 // V staged
  #pragma unroll
      for (int u = 0; u < BK / 32; ++u) {
        bf16x8 bp;
        {
          uint4 w;
          w.x = pack_bf16x2(st[2 * u][0], st[2 * u][1]);
          w.y = pack_bf16x2(st[2 * u][2], st[2 * u][3]);
          w.z = pack_bf16x2(st[2 * u + 1][0], st[2 * u + 1][1]);
          w.w = pack_bf16x2(st[2 * u + 1][2], st[2 * u + 1][3]);
          bp = __builtin_bit_cast(bf16x8, w);
        }
  #pragma unroll
        for (int t = 0; t < kHeadDim / 16; ++t) {
          // A operand V^T: row d = 16t + n (lane's m), the same key mapping.
          const uint16_t* vr = &sm.vt[16 * t + n][32 * u + 4 * q4];
          uint4 w;
          const uint2 lo = *reinterpret_cast<const uint2*>(vr);
          const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
          w.x = lo.x; w.y = lo.y; w.z = hi.x; w.w = hi.y;
          acc[t] = mfma16x16x32(__builtin_bit_cast(bf16x8, w), bp, acc[t]);
        }
      }
      slot = next;
    }
  }

  // Merge the waves' states (Sec. 4.2): M = max_w m_w, L = sum_w l_w 2^(m_w - M),
  // O = sum_w 2^(m_w - M) acc_w / L.  O^T tiles: lane (n, q4) holds
  // d = 16t + 4*q4 + e of head n.
  __syncthreads();                                    // every wave is done with its V^T area
  if (q4 == 0) {
    mls[wv][0][n] = m_run;
    mls[wv][1][n] = l_run;
  }
  __syncthreads();
  auto merged = [&](int h, float& M, float& L) {
    M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, mls[w][0][h]);
    L = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      const float mw = mls[w][0][h];
      L += mw > -INFINITY ? mls[w][1][h] * exp2f(mw - M) : 0.f;
    }
  };
  {
    float M, L;
    merged(n, M, L);
    const float f = m_run > -INFINITY ? exp2f(m_run - M) : 0.f;
    float* red = reinterpret_cast<float*>(&sm.vt[0][0]) + n * kRedStride + 4 * q4;
#pragma unroll
    for (int t = 0; t < kHeadDim / 16; ++t) *reinterpret_cast<f32x4*>(red + 16 * t) = acc[t] * f;
  }
  __syncthreads();
  // thread (head hn, dims d0 .. d0+8) sums the waves' scaled rows
  const int hn = threadIdx.x / 16, d0 = 8 * (threadIdx.x % 16);
  if (hn >= G) return;
  float M, L;
  merged(hn, M, L);
  float out[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
  for (int w = 0; w < kAttnWaves; ++w) {
    const float* red = reinterpret_cast<const float*>(&smw[w].vt[0][0]) + hn * kRedStride + d0;
    const f32x4 x0 = *reinterpret_cast<const f32x4*>(red);
    const f32x4 x1 = *reinterpret_cast<const f32x4*>(red + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      out[e] += x0[e];
      out[4 + e] += x1[e];
    }
  }
  const int64_t head_row = row * H_q + static_cast<int64_t>(r) * G + hn;
  const bool empty = !(L > 0.f);
  const float inv_l = empty ? 0.f : o_scale / L;
  const float lse_v = empty ? -INFINITY : (M + __log2f(L)) * kLn2;
  if (nsplit == 1) {
    uint4 wq;
    wq.x = pack_bf16x2(out[0] * inv_l, out[1] * inv_l);
    wq.y = pack_bf16x2(out[2] * inv_l, out[3] * inv_l);
    wq.z = pack_bf16x2(out[4] * inv_l, out[5] * inv_l);
    wq.w = pack_bf16x2(out[6] * inv_l, out[7] * inv_l);
    *reinterpret_cast<uint4*>(o + head_row * kHeadDim + d0) = wq;
    if (d0 == 0) lse[head_row] = lse_v;
  } else {
    const int64_t part_row = static_cast<int64_t>(sp) * sq.total_q_rows * H_q + head_row;
    float4* dst = reinterpret_cast<float4*>(o_part + part_row * kHeadDim + d0);
    dst[0] = make_float4(out[0] * inv_l, out[1] * inv_l, out[2] * inv_l, out[3] * inv_l);
    dst[1] = make_float4(out[4] * inv_l, out[5] * inv_l, out[6] * inv_l, out[7] * inv_l);
    if (d0 == 0) lse_part[part_row] = lse_v;
  }
}

// Merge `nsplit` partials per (row, head): a = max LSE_s,
// LSE = a + log sum exp(LSE_s - a), O = sum exp(LSE_s - LSE) O_s (Sec. 4.2).
// One thread per (row, head, 8 dims).
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ o_part,
                                                      const float* __restrict__ lse_part, int nsplit,
                                                      int64_t head_rows, uint16_t* __restrict__ o,
                                                      float* __restrict__ lse) {
  const int64_t tid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t hr = tid >> 4;
  const int d0 = static_cast<int>(tid & 15) * 8;
  if (hr >= head_rows) return;
  float a = -INFINITY;
  for (int s = 0; s < nsplit; ++s) a = fmaxf(a, lse_part[s * head_rows + hr]);
  float out[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  float total = -INFINITY;
  if (a > -INFINITY) {
    float sum = 0.f;
    for (int s = 0; s < nsplit; ++s) sum += exp2f((lse_part[s * head_rows + hr] - a) * kLog2e);
    total = a + __logf(sum);
    for (int s = 0; s < nsplit; ++s) {
      const float ls = lse_part[s * head_rows + hr];
      if (!(ls > -INFINITY)) continue;
      const float w = exp2f((ls - total) * kLog2e);
      const float4* src = reinterpret_cast<const float4*>(o_part + (s * head_rows + hr) * kHeadDim + d0);
      const float4 x0 = src[0], x1 = src[1];
      out[0] += w * x0.x; out[1] += w * x0.y; out[2] += w * x0.z; out[3] += w * x0.w;
      out[4] += w * x1.x; out[5] += w * x1.y; out[6] += w * x1.z; out[7] += w * x1.w;
    }
  }
  uint4 wv;
  wv.x = pack_bf16x2(out[0], out[1]);
  wv.y = pack_bf16x2(out[2], out[3]);
  wv.z = pack_bf16x2(out[4], out[5]);
  wv.w = pack_bf16x2(out[6], out[7]);
  *reinterpret_cast<uint4*>(o + hr * kHeadDim + d0) = wv;
  if (d0 == 0) lse[hr] = total;
}

// ---------------------------------------------------------------- host side
}  // namespace

// key-block-outer prefill (sparse_attn_prefill.hip)
size_t msa_kvo_workspace_size(const msa_seqs* seqs, int H_q, int H_kv, int BK, int topk);
int msa_kvo_prefill(const void* q, const void* k, const void* v, const int32_t* block_ids, const msa_seqs* seqs,
                    int H_q, int H_kv, int BK, int topk, float scale, void* o, float* lse, void* workspace,
                    size_t workspace_bytes, hipStream_t stream, bool fp8, float q_scale, float k_scale,
                    float v_scale);

namespace {

int validate_attn(const msa_seqs* seqs, int H_q, int H_kv, int head_dim, int BK, int topk) {
  int st = msa_host::validate_seqs(seqs);
  if (st != MSA_OK) return st;
  if (H_q < 1 || H_kv < 1 || head_dim < 1 || BK < 1 || topk < 1) return MSA_ERR_INVALID;
  if (H_q % H_kv != 0) return MSA_ERR_INVALID;
  if (head_dim != kHeadDim) return MSA_ERR_UNSUPPORTED;
  if (BK != 64 && BK != 128) return MSA_ERR_UNSUPPORTED;
  if (topk > 64 || H_q / H_kv > 16 || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (seqs->total_q_rows * H_kv >= (int64_t(1) << 31)) return MSA_ERR_UNSUPPORTED;
  return msa_host::check_paged(seqs, BK, true);
}

struct SplitPlan {
  int nsplit;           // CTAs per (row, group); above one, partials go through combine_kernel
  int slots_per_wave;
};

// Spread the k slots of each (row, group) over kAttnWaves waves per CTA and
// over enough CTAs to give the chip about 2048 waves.
SplitPlan split_plan(const msa_seqs* seqs, int H_kv, int topk) {
  SplitPlan sp;
  const int64_t pairs = seqs->total_q_rows * H_kv;
  const int max_ctas = (topk + kAttnWaves - 1) / kAttnWaves;
  int64_t want = pairs > 0 ? (2048 + pairs * kAttnWaves - 1) / (pairs * kAttnWaves) : 1;
  if (want < 1) want = 1;
  if (want > max_ctas) want = max_ctas;
  const int waves = static_cast<int>(want) * kAttnWaves;
  sp.slots_per_wave = (topk + waves - 1) / waves;
  sp.nsplit = (topk + sp.slots_per_wave * kAttnWaves - 1) / (sp.slots_per_wave * kAttnWaves);
  return sp;
}

size_t split_workspace(const msa_seqs* seqs, int H_q, const SplitPlan& sp) {
  if (sp.nsplit <= 1) return 0;
  const size_t hr = static_cast<size_t>(seqs->total_q_rows) * H_q;
  return msa_host::align_up(sp.nsplit * hr * kHeadDim * sizeof(float), 256) + sp.nsplit * hr * sizeof(float);
}

// fp8: Q, K and V are OCP e4m3 with per-tensor scales (logits use
// scale * q_scale * k_scale, O is multiplied by v_scale); else bf16 (scales 1).
int run_rows(const void* q, const void* k, const void* v, const int32_t* block_ids, const msa_seqs* seqs,
             int H_q, int H_kv, int BK, int topk, float scale, void* o, float* lse, const SplitPlan& sp,
             void* workspace, hipStream_t stream, bool fp8 = false, float q_scale = 1.f, float k_scale = 1.f,
             float v_scale = 1.f) {
  const int64_t hr = seqs->total_q_rows * H_q;
  float* o_part = nullptr;
  float* lse_part = nullptr;
  if (sp.nsplit > 1) {
    o_part = static_cast<float*>(workspace);
    lse_part = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                        msa_host::align_up(sp.nsplit * static_cast<size_t>(hr) * kHeadDim * sizeof(float), 256));
  }
  const dim3 grid(static_cast<unsigned>(seqs->total_q_rows * H_kv), static_cast<unsigned>(sp.nsplit));
  const float sl2 = scale * q_scale * k_scale * kLog2e;
  const msa_seqs sq = *seqs;
  auto* op = static_cast<uint16_t*>(o);
  const dim3 block(64 * kAttnWaves);
  auto launch = [&](auto kernel, auto elem) {
    using T = decltype(elem);
    msa_prof::launch("attn_rows_kernel", kernel, grid, block, 0, stream, static_cast<const T*>(q),
                     static_cast<const T*>(k), static_cast<const T*>(v), block_ids, sq, H_q, H_kv, topk,
                     sp.slots_per_wave, sl2, v_scale, op, lse, o_part, lse_part);
  };
  if (sq.block_table) {
    if (BK == 64 && !fp8) launch(attn_rows_kernel<64, uint16_t, true>, uint16_t{});
    else if (BK == 64) launch(attn_rows_kernel<64, uint8_t, true>, uint8_t{});
    else if (!fp8) launch(attn_rows_kernel<128, uint16_t, true>, uint16_t{});
    else launch(attn_rows_kernel<128, uint8_t, true>, uint8_t{});
  } else {
    if (BK == 64 && !fp8) launch(attn_rows_kernel<64, uint16_t, false>, uint16_t{});
    else if (BK == 64) launch(attn_rows_kernel<64, uint8_t, false>, uint8_t{});
    else if (!fp8) launch(attn_rows_kernel<128, uint16_t, false>, uint16_t{});
    else launch(attn_rows_kernel<128, uint8_t, false>, uint8_t{});
  }
  if (sp.nsplit > 1) {
    const int64_t threads = hr * 16;
    msa_prof::launch("combine_kernel", combine_kernel, dim3(static_cast<unsigned>((threads + 255) / 256)), dim3(256), 0, stream,
                       o_part, lse_part, sp.nsplit, hr, op, lse);
  }
  return msa_host::launch_status();
}

// Dense mode: every key block of the longest sequence is a slot.
SplitPlan dense_plan(const msa_seqs* seqs, int H_kv) {
  SplitPlan sp;
  const int nblk = (seqs->max_kv_len + 63) / 64 > 0 ? (seqs->max_kv_len + 63) / 64 : 1;
  const int64_t pairs = seqs->total_q_rows * H_kv;
  const int max_ctas = (nblk + kAttnWaves - 1) / kAttnWaves;
  int64_t want = pairs > 0 ? (8192 + pairs * kAttnWaves - 1) / (pairs * kAttnWaves) : 1;
  if (want < 1) want = 1;
  if (want > max_ctas) want = max_ctas;
  const int waves = static_cast<int>(want) * kAttnWaves;
  sp.slots_per_wave = (nblk + waves - 1) / waves;
  sp.nsplit = (nblk + sp.slots_per_wave * kAttnWaves - 1) / (sp.slots_per_wave * kAttnWaves);
  return sp;
}

int check_ptrs(const void* q, const void* k, const void* v, const int32_t* ids, const void* o, const float* lse) {
  return (q && k && v && ids && o && lse) ? MSA_OK : MSA_ERR_INVALID;
}

}  // namespace

// Dense causal attention of few-row sequences (the baseline call in
// dense_attn.hip): the row kernel over every key block, B_k = 64.
size_t msa_rows_dense_workspace_size(const msa_seqs* seqs, int H_q, int H_kv) {
  return split_workspace(seqs, H_q, dense_plan(seqs, H_kv));
}

int msa_rows_dense(const void* q, const void* k, const void* v, const msa_seqs* seqs, int H_q, int H_kv,
                   float scale, void* o, float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  const SplitPlan sp = dense_plan(seqs, H_kv);
  const size_t need = split_workspace(seqs, H_q, sp);
  if (need > 0 && (!workspace || workspace_bytes < need)) return MSA_ERR_WORKSPACE;
  const int nblk = (seqs->max_kv_len + 63) / 64 > 0 ? (seqs->max_kv_len + 63) / 64 : 1;
  return run_rows(q, k, v, nullptr, seqs, H_q, H_kv, 64, nblk, scale, o, lse, sp, workspace, stream);
}

extern "C" size_t msa_sparse_attn_decode_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                                       int head_dim, int block_size, int topk) {
  if (validate_attn(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk) != MSA_OK) return 0;
  return split_workspace(seqs, num_q_heads, split_plan(seqs, num_kv_heads, topk));
}

extern "C" int msa_sparse_attn_decode(const void* q, const void* k, const void* v, const int32_t* block_ids,
                                      const msa_seqs* seqs, int num_q_heads, int num_kv_heads, int head_dim,
                                      int block_size, int topk, float softmax_scale, void* o, float* lse,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = validate_attn(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk);
  if (st != MSA_OK) return st;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if ((st = check_ptrs(q, k, v, block_ids, o, lse)) != MSA_OK) return st;
  const SplitPlan sp = split_plan(seqs, num_kv_heads, topk);
  const size_t need = split_workspace(seqs, num_q_heads, sp);
  if (need > 0 && (!workspace || workspace_bytes < need)) return MSA_ERR_WORKSPACE;
  return run_rows(q, k, v, block_ids, seqs, num_q_heads, num_kv_heads, block_size, topk, softmax_scale, o, lse,
                  sp, workspace, stream);
}

extern "C" size_t msa_sparse_attn_prefill_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                                        int head_dim, int block_size, int topk) {
  if (validate_attn(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk) != MSA_OK) return 0;
  return msa_kvo_workspace_size(seqs, num_q_heads, num_kv_heads, block_size, topk);
}

extern "C" int msa_sparse_attn_prefill(const void* q, const void* k, const void* v, const int32_t* block_ids,
                                       const msa_seqs* seqs, int num_q_heads, int num_kv_heads, int head_dim,
                                       int block_size, int topk, float softmax_scale, void* o, float* lse,
                                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = validate_attn(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk);
  if (st != MSA_OK) return st;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if ((st = check_ptrs(q, k, v, block_ids, o, lse)) != MSA_OK) return st;
  return msa_kvo_prefill(q, k, v, block_ids, seqs, num_q_heads, num_kv_heads, block_size, topk, softmax_scale, o,
                         lse, workspace, workspace_bytes, stream, false, 1.f, 1.f, 1.f);
}

namespace {
bool scale_ok(float x) { return x > 0.f && x < 3.0e38f; }   // finite and positive
}  // namespace

extern "C" int msa_sparse_attn_prefill_fp8(const void* q, const void* k, const void* v, float q_scale,
                                           float k_scale, float v_scale, const int32_t* block_ids,
                                           const msa_seqs* seqs, int num_q_heads, int num_kv_heads, int head_dim,
                                           int block_size, int topk, float softmax_scale, void* o, float* lse,
                                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = validate_attn(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk);
  if (st != MSA_OK) return st;
  if (!scale_ok(q_scale) || !scale_ok(k_scale) || !scale_ok(v_scale)) return MSA_ERR_INVALID;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if ((st = check_ptrs(q, k, v, block_ids, o, lse)) != MSA_OK) return st;
  return msa_kvo_prefill(q, k, v, block_ids, seqs, num_q_heads, num_kv_heads, block_size, topk, softmax_scale, o,
                         lse, workspace, workspace_bytes, stream, true, q_scale, k_scale, v_scale);
}

extern "C" int msa_sparse_attn_decode_fp8(const void* q, const void* k, const void* v, float q_scale,
                                          float k_scale, float v_scale, const int32_t* block_ids,
                                          const msa_seqs* seqs, int num_q_heads, int num_kv_heads, int head_dim,
                                          int block_size, int topk, float softmax_scale, void* o, float* lse,
                                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  int st = validate_attn(seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk);
  if (st != MSA_OK) return st;
  if (!scale_ok(q_scale) || !scale_ok(k_scale) || !scale_ok(v_scale)) return MSA_ERR_INVALID;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if ((st = check_ptrs(q, k, v, block_ids, o, lse)) != MSA_OK) return st;
  const SplitPlan sp = split_plan(seqs, num_kv_heads, topk);
  const size_t need = split_workspace(seqs, num_q_heads, sp);
  if (need > 0 && (!workspace || workspace_bytes < need)) return MSA_ERR_WORKSPACE;
  return run_rows(q, k, v, block_ids, seqs, num_q_heads, num_kv_heads, block_size, topk, softmax_scale, o, lse,
                  sp, workspace, stream, true, q_scale, k_scale, v_scale);
}

extern "C" const char* msa_strerror(int status) {
  switch (status) {
    case MSA_OK: return "ok";
    case MSA_ERR_INVALID: return "invalid argument";
    case MSA_ERR_UNSUPPORTED: return "unsupported shape or parameter";
    case MSA_ERR_WORKSPACE: return "workspace too small";
    case MSA_ERR_HIP: return "HIP launch failure";
    default: return "unknown status";
  }
}
