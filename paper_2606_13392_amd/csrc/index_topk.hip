// Index Branch of MSA on gfx950: causal block max-pooled index scores and
// Top-k block selection with the local block forced.
//
// Sec. 3.1 (index-score equation): S_ij = q_idx[i,r] . k_idx[j] / sqrt(d_idx),
// M_ib = max over the visible tokens of block b.  Sec. 3.1 (top-k equation) and
// Sec. 3.2 ("Local Block"): the local block lb = p / B_k always takes a slot, the
// other k-1 slots go to the highest-scoring causal blocks.  Every candidate block
// b < lb is entirely visible, so the causal mask never enters the scored range;
// the local block is forced and never scored.  Selection ranks raw fp32 dot
// products (Sec. 4.1 "Exp-free selection": monotone maps keep the order).
//
// Two kernels per chunk of query rows:
//   index_block_max  MFMA 32x32x16 (keys as M, index rows as N) over one key
//                    block at a time; the block max is reduced in registers and
//                    one permlane32 swap, then written as M[row][block] (fp32).
//   index_topk       one wave per index row streams M[row][0..lb) 64 blocks at a
//                    time, filters against the current k-1-th best key and keeps
//                    a sorted 64-entry list (one 64-bit key per lane).
#include "msa_common.h"

namespace {

using namespace msa;

constexpr int kWavesPerBlock = 4;
constexpr int kBlocksPerWave = 16;     // key blocks one wave scores per launch slice
constexpr int kSmallInsert = 6;        // survivors per 64-block step inserted one by one

// ---------------------------------------------------------------- setup
// group_off[s] = number of row groups before sequence s; a row group is `qr`
// consecutive query rows of one sequence (qr * H_kv = 64 index rows).
__global__ __launch_bounds__(256) void row_group_offsets_kernel(msa_seqs sq, int qr,
                                                                int32_t* __restrict__ group_off) {
  __shared__ int32_t part[256];
  const int t = threadIdx.x;
  const int S = sq.num_seqs;
  const int per = (S + 255) / 256;
  const int s0 = t * per, s1 = min(S, s0 + per);
  int32_t acc = 0;
  for (int s = s0; s < s1; ++s) {
    int rows = sq.q_offsets[s + 1] - sq.q_offsets[s];
    acc += rows > 0 ? (rows + qr - 1) / qr : 0;
  }
  part[t] = acc;
  __syncthreads();
  if (t == 0) {
    int32_t run = 0;
    for (int i = 0; i < 256; ++i) { int32_t x = part[i]; part[i] = run; run += x; }
    group_off[S] = run;
  }
  __syncthreads();
  acc = part[t];
  for (int s = s0; s < s1; ++s) {
    group_off[s] = acc;
    int rows = sq.q_offsets[s + 1] - sq.q_offsets[s];
    acc += rows > 0 ? (rows + qr - 1) / qr : 0;
  }
}

struct GroupRows {
  bool ok;
  int s;
  SeqGeom g;
  int t0;       // first query row (inside the sequence) of the group
  int nq;       // valid query rows in the group
};

__device__ __forceinline__ GroupRows locate_group(const msa_seqs& sq, const int32_t* __restrict__ group_off,
                                                  int64_t gidx, int qr) {
  GroupRows r;
  r.ok = false;
  if (gidx >= group_off[sq.num_seqs]) return r;
  r.s = find_seq(group_off, sq.num_seqs, gidx);
  r.g = seq_geom(sq, r.s);
  r.t0 = static_cast<int>(gidx - group_off[r.s]) * qr;
  r.nq = min(qr, r.g.q_rows - r.t0);
  // never touch query rows past the query-side tensors
  const int64_t left = sq.total_q_rows - (static_cast<int64_t>(r.g.q_begin) + r.t0);
  if (left < r.nq) r.nq = static_cast<int>(left > 0 ? left : 0);
  r.ok = r.nq > 0 && r.g.q_begin >= 0;
  return r;
}

// ---------------------------------------------------------------- scores
// One wave: 64 index rows (qr query rows x H_kv groups, contiguous in index_q)
// against key blocks [kb0, kb0 + kBlocksPerWave) of its sequence.
template <int D_IDX, int BK>
__global__ __launch_bounds__(256) void index_block_max_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, msa_seqs sq,
    const int32_t* __restrict__ group_off, int H_kv, int qr, int64_t g0, int64_t g1,
    float* __restrict__ M, int64_t ldm) {
  constexpr int KS = D_IDX / 16;        // k-steps of the MFMA
  constexpr int HALF = D_IDX / 2;       // dims a lane half supplies
  constexpr int MT = BK / 32;           // 32-key M tiles per block
  const int lane = lane_id();
  const int64_t gidx = g0 + static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
  if (gidx >= g1) return;
  GroupRows gr = locate_group(sq, group_off, gidx, qr);
  if (!gr.ok) return;
  const int p_last = gr.g.kv_len - gr.g.q_rows + gr.t0 + gr.nq - 1;
  if (p_last < 0) return;
  const int lb_max = p_last / BK;                    // candidates are blocks < lb
  const int kb0 = blockIdx.y * kBlocksPerWave;
  const int kb1 = min(min(kb0 + kBlocksPerWave, lb_max), static_cast<int>(ldm));
  if (kb0 >= kb1) return;

  const int n = lane & 31, h = lane >> 5;
  const int nvalid = gr.nq * H_kv;
  // B operand: the wave's 64 index rows (two 32-column N tiles), kept in registers.
  const uint16_t* qbase = index_q + (static_cast<int64_t>(gr.g.q_begin + gr.t0) * H_kv) * D_IDX;
  bf16x8 bq[2][KS];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 32 * j + n;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      bq[j][s] = row < nvalid ? ld_bf16x8(qbase + static_cast<int64_t>(row) * D_IDX + h * HALF + 8 * s)
                              : zero_bf16x8();
  }
  const uint16_t* kbase = index_k + gr.g.kv_start * D_IDX + h * HALF;
  float* mrow = M + ((gidx - g0) * kWave + lane) * ldm;
  const bool store = lane < nvalid;

  for (int kb = kb0; kb < kb1; ++kb) {
    f32x16 acc[MT][2];
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const uint16_t* kp = kbase + static_cast<int64_t>(kb * BK + 32 * i + n) * D_IDX;
      bf16x8 a[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s) a[s] = ld_bf16x8(kp + 8 * s);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        acc[i][j] = f32x16{};
#pragma unroll
        for (int s = 0; s < KS; ++s) acc[i][j] = mfma32x32x16(a[s], bq[j][s], acc[i][j]);
      }
    }
    // block max: each lane holds half of the block's keys for its column
    float pm[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float m = acc[0][j][0];
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) m = fmaxf(m, acc[i][j][r]);
      pm[j] = m;
    }
    // lanes 0-31 gather column tile 0 (rows 0-31), lanes 32-63 tile 1 (rows 32-63)
    auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(pm[0]), __float_as_uint(pm[1]), false, false);
    const float bm = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
    if (store) mrow[kb] = bm;
  }
}

// ---------------------------------------------------------------- top-k
__global__ __launch_bounds__(256) void index_topk_kernel(
    const float* __restrict__ M, int64_t ldm, msa_seqs sq, const int32_t* __restrict__ group_off,
    int H_kv, int qr, int64_t g0, int64_t g1, int BK, int topk, int32_t* __restrict__ block_ids) {
  const int lane = lane_id();
  const int64_t slot = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave;
  if (slot >= (g1 - g0) * kWave) return;
  const int64_t gidx = g0 + slot / kWave;
  const int L = static_cast<int>(slot % kWave);
  GroupRows gr = locate_group(sq, group_off, gidx, qr);
  if (!gr.ok || L >= gr.nq * H_kv) return;
  const int t = gr.t0 + L / H_kv;
  const int r = L % H_kv;
  int32_t* out = block_ids + (static_cast<int64_t>(gr.g.q_begin + t) * H_kv + r) * topk;
  const int p = gr.g.kv_len - gr.g.q_rows + t;
  if (p < 0) {
    if (lane < topk) out[lane] = -1;
    return;
  }
  const int lb = p / BK;
  const int nscan = min(lb, static_cast<int>(ldm));   // == lb whenever kv_lens respect max_kv_len
  const int K1 = topk - 1;
  const float* mrow = M + slot * ldm;

  uint64_t list = 0;   // sorted descending across lanes; 0 marks an empty slot
  uint64_t tau = 0;    // key of the K1-th best so far (0 while fewer are known)
  if (K1 > 0) {
    for (int c0 = 0; c0 < nscan; c0 += kWave) {
      const int b = c0 + lane;
      const uint64_t v = b < nscan ? rank_key(mrow[b], static_cast<uint32_t>(b)) : 0ull;
      uint64_t pass = __ballot(v > tau);
      if (pass == 0) continue;
      if (__popcll(pass) <= kSmallInsert) {
        while (pass) {
          const int src = __ffsll(static_cast<unsigned long long>(pass)) - 1;
          pass &= pass - 1;
          const uint64_t x = readlane_u64(v, src);
          const int rnk = __popcll(__ballot(list > x));
          const uint64_t prev = shfl_u64(list, lane - 1);
          list = lane < rnk ? list : (lane == rnk ? x : prev);
        }
      } else {
        const uint64_t vs = wave_sort_desc_u64(v);
        const uint64_t rev = shfl_u64(vs, kWave - 1 - lane);
        list = wave_bitonic_merge_desc_u64(list > rev ? list : rev);
      }
      tau = readlane_u64(list, K1 - 1);
    }
  }
  const int cnt = K1 > 0 ? __popcll(__ballot(lane < K1 && list != 0ull)) : 0;
  uint32_t id = 0xFFFFFFFFu;
  if (lane < cnt) id = key_block(list);
  else if (lane == cnt) id = static_cast<uint32_t>(lb);
  id = wave_sort_asc_u32(id);
  if (lane < topk) out[lane] = lane <= cnt ? static_cast<int32_t>(id) : -1;
}

// ---------------------------------------------------------------- host side
struct IndexPlan {
  int qr;
  int64_t max_groups;
  int bcap;
  size_t hdr_bytes;
  size_t group_bytes;
};

int make_plan(const msa_seqs* seqs, int H_kv, int d_idx, int BK, int topk, IndexPlan* pl) {
  int st = msa_host::validate_seqs(seqs);
  if (st != MSA_OK) return st;
  if (H_kv < 1 || d_idx < 1 || BK < 1 || topk < 1) return MSA_ERR_INVALID;
  if (!msa_host::is_pow2(H_kv) || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (d_idx != 64 && d_idx != 128) return MSA_ERR_UNSUPPORTED;
  if (BK != 64 && BK != 128) return MSA_ERR_UNSUPPORTED;
  if (topk > 64) return MSA_ERR_UNSUPPORTED;
  pl->qr = 64 / H_kv;
  pl->max_groups = seqs->total_q_rows / pl->qr + seqs->num_seqs;
  int nb = (seqs->max_kv_len + BK - 1) / BK;
  pl->bcap = static_cast<int>(msa_host::align_up(static_cast<size_t>(nb > 0 ? nb : 1), 4));
  pl->hdr_bytes = msa_host::align_up(sizeof(int32_t) * (seqs->num_seqs + 1), 256);
  pl->group_bytes = static_cast<size_t>(kWave) * pl->bcap * sizeof(float);
  return MSA_OK;
}

constexpr size_t kDefaultScoreBytes = size_t(4) << 30;   // block-score staging per call

}  // namespace

extern "C" size_t msa_index_topk_workspace_size(const msa_seqs* seqs, int num_kv_heads, int d_idx,
                                                int block_size, int topk) {
  IndexPlan pl;
  if (make_plan(seqs, num_kv_heads, d_idx, block_size, topk, &pl) != MSA_OK) return 0;
  int64_t groups = static_cast<int64_t>(kDefaultScoreBytes / pl.group_bytes);
  if (groups < 1) groups = 1;
  if (groups > pl.max_groups) groups = pl.max_groups;
  return pl.hdr_bytes + static_cast<size_t>(groups) * pl.group_bytes;
}

extern "C" int msa_index_topk(const void* index_q, const void* index_k, const msa_seqs* seqs,
                              int num_kv_heads, int d_idx, int block_size, int topk,
                              int32_t* block_ids, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  IndexPlan pl;
  int st = make_plan(seqs, num_kv_heads, d_idx, block_size, topk, &pl);
  if (st != MSA_OK) return st;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if (!index_q || !index_k || !block_ids || !workspace) return MSA_ERR_INVALID;
  if (workspace_bytes < pl.hdr_bytes + pl.group_bytes) return MSA_ERR_WORKSPACE;
  int64_t chunk = static_cast<int64_t>((workspace_bytes - pl.hdr_bytes) / pl.group_bytes);
  if (chunk > pl.max_groups) chunk = pl.max_groups;

  int32_t* group_off = static_cast<int32_t*>(workspace);
  float* M = reinterpret_cast<float*>(static_cast<char*>(workspace) + pl.hdr_bytes);
  const msa_seqs sq = *seqs;
  const uint16_t* iq = static_cast<const uint16_t*>(index_q);
  const uint16_t* ik = static_cast<const uint16_t*>(index_k);

  hipLaunchKernelGGL(row_group_offsets_kernel, dim3(1), dim3(256), 0, stream, sq, pl.qr, group_off);
  const unsigned ny = static_cast<unsigned>((pl.bcap + kBlocksPerWave - 1) / kBlocksPerWave);
  for (int64_t g0 = 0; g0 < pl.max_groups; g0 += chunk) {
    const int64_t g1 = g0 + chunk < pl.max_groups ? g0 + chunk : pl.max_groups;
    const unsigned nx = static_cast<unsigned>((g1 - g0 + kWavesPerBlock - 1) / kWavesPerBlock);
    if (d_idx == 64 && block_size == 64)
      hipLaunchKernelGGL((index_block_max_kernel<64, 64>), dim3(nx, ny), dim3(256), 0, stream, iq, ik, sq,
                         group_off, num_kv_heads, pl.qr, g0, g1, M, static_cast<int64_t>(pl.bcap));
    else if (d_idx == 64)
      hipLaunchKernelGGL((index_block_max_kernel<64, 128>), dim3(nx, ny), dim3(256), 0, stream, iq, ik, sq,
                         group_off, num_kv_heads, pl.qr, g0, g1, M, static_cast<int64_t>(pl.bcap));
    else if (block_size == 64)
      hipLaunchKernelGGL((index_block_max_kernel<128, 64>), dim3(nx, ny), dim3(256), 0, stream, iq, ik, sq,
                         group_off, num_kv_heads, pl.qr, g0, g1, M, static_cast<int64_t>(pl.bcap));
    else
      hipLaunchKernelGGL((index_block_max_kernel<128, 128>), dim3(nx, ny), dim3(256), 0, stream, iq, ik, sq,
                         group_off, num_kv_heads, pl.qr, g0, g1, M, static_cast<int64_t>(pl.bcap));
    const unsigned nt = static_cast<unsigned>((g1 - g0) * kWave / kWavesPerBlock);
    hipLaunchKernelGGL(index_topk_kernel, dim3(nt), dim3(256), 0, stream, M, static_cast<int64_t>(pl.bcap), sq,
                       group_off, num_kv_heads, pl.qr, g0, g1, block_size, topk, block_ids);
  }
  return msa_host::launch_status();
}
