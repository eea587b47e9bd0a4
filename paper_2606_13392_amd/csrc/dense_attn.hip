// Dense causal GQA attention on gfx950: the baseline the sparse path is
// measured against.  Every query attends to all causally visible keys of its
// sequence (the full-attention form that MSA's sparse-attention equation of
// Sec. 3.1 reduces to when k covers every causal block), with the layout
// conventions of the sparse calls.
//
// Prefill (dense_prefill_kernel), FlashAttention-2 order: a CTA owns one KV
// group and a tile of consecutive query rows whose G heads share the group's
// K and V; its 4 waves hold 32 (query row, head) rows each.  Key blocks of 64
// are streamed through a double-buffered LDS ring (K row-major, V transposed)
// fed by register prefetch one block ahead; per block each wave computes
// S^T = K Q^T and O^T += V^T P^T with MFMA 32x32x16 and keeps the online
// softmax (running max and sum per row) in registers.
//
// Decode (at most four query rows per sequence) runs the row kernel of the
// sparse decode call over every key block (msa_rows_dense).
#include <algorithm>

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
constexpr int kThreads = 256;            // 4 waves
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kDecodeRows = 4;           // sequences with at most this many query rows take the row kernel

struct DenseSmem {
  uint16_t k[2][kBK][kHeadDim + 8];      // K blocks, row-major (+16 B pad per row)
  uint16_t vt[2][kHeadDim][kBK + 4];     // V blocks transposed (+8 B pad per row)
};

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

// V staging map: thread tid takes 4-key group tid & 15 and 8-dim group
// 4 (tid / 64) + {0, 2, 1, 3}[(tid / 16) & 3], so each 32-lane half of a wave
// writes dim groups d and d + 2 of Vt, whose rows start 32 banks apart: the
// 8-byte transposed stores hit 64 distinct banks.
__device__ __forceinline__ void dense_v_map(int tid, int& key4, int& dg) {
  key4 = tid & 15;
  const int q = (tid >> 4) & 3;
  dg = 4 * (tid >> 6) + ((q & 1) << 1) + (q >> 1);
}

// One key block of group r: thread tid loads 4 K pieces (key, 16-byte
// segment) and 4 V rows of one (4-key group, 8-dim group); keys at or past
// kv_len read as zero.
__device__ __forceinline__ void dense_load_block(const uint16_t* __restrict__ kb, const uint16_t* __restrict__ vb,
                                                 int64_t stride, int key0, int kv_len, int tid, u32x4 (&rk)[4],
                                                 u32x4 (&rv)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int idx = tid + kThreads * c;
    const int key = idx / (kHeadDim / 8), seg = idx % (kHeadDim / 8);
    rk[c] = key0 + key < kv_len ? *reinterpret_cast<const u32x4*>(kb + static_cast<int64_t>(key0 + key) * stride + 8 * seg)
                                : u32x4{0, 0, 0, 0};
  }
  int key4, dg;
  dense_v_map(tid, key4, dg);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int key = key0 + 4 * key4 + j;
    rv[j] = key < kv_len ? *reinterpret_cast<const u32x4*>(vb + static_cast<int64_t>(key) * stride + 8 * dg)
                         : u32x4{0, 0, 0, 0};
  }
}
__device__ __forceinline__ void dense_store_block(DenseSmem& sm, int buf, int tid, const u32x4 (&rk)[4],
                                                  const u32x4 (&rv)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int idx = tid + kThreads * c;
    const int key = idx / (kHeadDim / 8), seg = idx % (kHeadDim / 8);
    *reinterpret_cast<u32x4*>(&sm.k[buf][key][8 * seg]) = rk[c];
  }
  int key4, dg;
  dense_v_map(tid, key4, dg);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int w = e >> 1, sh = (e & 1) * 16;
    uint2 x;
    x.x = ((rv[0][w] >> sh) & 0xFFFFu) | (((rv[1][w] >> sh) & 0xFFFFu) << 16);
    x.y = ((rv[2][w] >> sh) & 0xFFFFu) | (((rv[3][w] >> sh) & 0xFFFFu) << 16);
    *reinterpret_cast<uint2*>(&sm.vt[buf][8 * dg + e][4 * key4]) = x;
  }
}

// grid: (tiles, H_kv); tiles are taken last-first so the longest causal
// ranges start first.
__global__ __launch_bounds__(kThreads, 2) void dense_prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v, msa_seqs sq,
    const int32_t* __restrict__ tile_off, int H_q, int H_kv, int ntile_grid, float scale_log2,
    uint16_t* __restrict__ o, float* __restrict__ lse) {
  __shared__ __align__(16) DenseSmem sm;
  constexpr int MT = kBK / 32;             // 32-key tiles of S^T
  constexpr int KS = kHeadDim / 16;        // k-steps of S^T = K Q^T
  const int lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int tid = threadIdx.x;
  const int n = lane & 31, h = lane >> 5;
  const int G = H_q / H_kv;
  const int qpw = 32 / G;                  // query rows per wave
  const int qt = 4 * qpw;                  // query rows per CTA
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
  // smallest position among the wave's rows (invalid lanes see every key masked anyway)
  const int p_wave = g.kv_len - g.q_rows + min(t0 + wave * qpw, t_end - 1);
  const int64_t head_row = (static_cast<int64_t>(g.q_begin) + (valid ? t : t0)) * H_q + static_cast<int64_t>(r) * G + hh;

  bf16x8 bq[KS];
  {
    const uint16_t* qrow = q + head_row * kHeadDim + 8 * h;
#pragma unroll
    for (int st = 0; st < KS; ++st) bq[st] = valid ? ld_bf16x8(qrow + 16 * st) : zero_bf16x8();
  }
  const int64_t stride = static_cast<int64_t>(H_kv) * kHeadDim;
  const uint16_t* kb = k + g.kv_start * stride + static_cast<int64_t>(r) * kHeadDim;
  const uint16_t* vb = v + g.kv_start * stride + static_cast<int64_t>(r) * kHeadDim;

  f32x16 acc_o[kHeadDim / 32];
#pragma unroll
  for (int i = 0; i < kHeadDim / 32; ++i) acc_o[i] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  u32x4 rk[4], rv[4];
  dense_load_block(kb, vb, stride, 0, g.kv_len, tid, rk, rv);
  dense_store_block(sm, 0, tid, rk, rv);
  dense_load_block(kb, vb, stride, min(1, nblk - 1) * kBK, g.kv_len, tid, rk, rv);
  __syncthreads();
  for (int b = 0; b < nblk; ++b) {
    const int buf = b & 1;
    // block b+1 goes to the other buffer (its readers passed the last barrier);
    // block b+2 is requested before block b is computed
    if (b + 1 < nblk) dense_store_block(sm, buf ^ 1, tid, rk, rv);
    dense_load_block(kb, vb, stride, min(b + 2, nblk - 1) * kBK, g.kv_len, tid, rk, rv);

    // S^T = K Q^T: lane (n, h) holds keys 32i + 8(e/4) + 4h + e%4 of row n
    f32x16 acc_s[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      acc_s[i] = f32x16{};
      const uint16_t* kr = &sm.k[buf][32 * i + n][8 * h];
#pragma unroll
      for (int st = 0; st < KS; ++st)
        acc_s[i] = mfma32x32x16(__builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kr + 16 * st)), bq[st],
                                acc_s[i]);
    }
    const int key0 = b * kBK;
    // running max in raw score units (scale_log2 > 0 keeps the order);
    // only blocks reaching past the wave's first row need the causal mask
    if (key0 + kBK - 1 > p_wave) {
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
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
    const float m_new = fmaxf(m_run, bmax);
    const float mm = m_new == -INFINITY ? 0.f : m_new;     // rows with nothing visible yet
    const float alpha = exp2f((m_run - mm) * scale_log2);
    const float neg = -mm * scale_log2;
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float pe = exp2f(fmaf(acc_s[i][e], scale_log2, neg));
        acc_s[i][e] = pe;
        lsum += pe;
      }
    lsum += __shfl_xor(lsum, 32);
    l_run = l_run * alpha + lsum;
    m_run = m_new;
    if (__ballot(alpha != 1.f)) {                        // some row's maximum moved
#pragma unroll
      for (int i = 0; i < kHeadDim / 32; ++i) acc_o[i] *= alpha;
    }

    // P in bf16 as the B operand of O^T = V^T P^T: k-step u covers keys
    // 32(u/2) + 16(u%2) + {4h + e, 8 + 4h + e}, the lane's acc_s[u/2][8(u%2) ..].
#pragma unroll
    for (int u = 0; u < kBK / 16; ++u) {
      uint4 pw;
      const int i = u >> 1, e0 = 8 * (u & 1);
      pw.x = pack_bf16x2(acc_s[i][e0 + 0], acc_s[i][e0 + 1]);
      pw.y = pack_bf16x2(acc_s[i][e0 + 2], acc_s[i][e0 + 3]);
      pw.z = pack_bf16x2(acc_s[i][e0 + 4], acc_s[i][e0 + 5]);
      pw.w = pack_bf16x2(acc_s[i][e0 + 6], acc_s[i][e0 + 7]);
      const bf16x8 bp = __builtin_bit_cast(bf16x8, pw);
      const int kbase = 32 * (u >> 1) + 16 * (u & 1) + 4 * h;
#pragma unroll
      for (int td = 0; td < kHeadDim / 32; ++td) {
        const uint16_t* vr = &sm.vt[buf][32 * td + n][kbase];
        const uint2 lo = *reinterpret_cast<const uint2*>(vr);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
        uint4 w;
        w.x = lo.x; w.y = lo.y; w.z = hi.x; w.w = hi.y;
        acc_o[td] = mfma32x32x16(__builtin_bit_cast(bf16x8, w), bp, acc_o[td]);
      }
    }
    __syncthreads();                                      // buffer buf is free again
  }

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
  const int qt = 4 * (32 / G);
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
