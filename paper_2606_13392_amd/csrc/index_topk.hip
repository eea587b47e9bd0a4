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
// Work units: a row group is qr = 64 / H_kv consecutive query rows of one
// sequence (64 index rows: query row x group, contiguous in index_q); a unit is
// U consecutive row groups of one sequence.  Per chunk of units:
//   index_block_max_lds   (U = 4, prefill) one CTA = 4 waves = 256 index rows
//                         sharing each K_idx block through a double-buffered LDS
//                         ring fed by register prefetch two blocks ahead;
//   index_block_max_wave  (U = 1, few rows per sequence, e.g. decode) one wave
//                         per row group and slice of key blocks;
// both run MFMA 32x32x16 with keys as M and index rows as N, reduce the block
// max in registers plus one permlane32 swap and write M[row][block] (fp32);
//   index_topk            one wave per index row streams M[row][0..lb) 64
//                         blocks at a time, filters against the current k-1-th
//                         best key and keeps a sorted list (one key per lane).
#include <algorithm>
#include <atomic>
#include <mutex>

#include "msa_common.h"
#include "msa_profile.h"

namespace {

using namespace msa;

constexpr int kWaves = 4;
constexpr int kBlocksPerCta = 64;      // key blocks per CTA slice, LDS kernel
constexpr int kSmallInsert = 6;        // survivors per 64-block step inserted one by one

// ---------------------------------------------------------------- setup
// unit_off[s] = units before sequence s.
__global__ __launch_bounds__(256) void unit_offsets_kernel(msa_seqs sq, int qr, int U,
                                                           int32_t* __restrict__ unit_off) {
  __shared__ int32_t part[256];
  const int t = threadIdx.x;
  const int S = sq.num_seqs;
  const int per = (S + 255) / 256;
  const int s0 = t * per, s1 = min(S, s0 + per);
  auto units = [&](int s) -> int32_t {
    const int rows = sq.q_offsets[s + 1] - sq.q_offsets[s];
    const int groups = rows > 0 ? (rows + qr - 1) / qr : 0;
    return (groups + U - 1) / U;
  };
  int32_t acc = 0;
  for (int s = s0; s < s1; ++s) acc += units(s);
  part[t] = acc;
  __syncthreads();
  if (t == 0) {
    int32_t run = 0;
    for (int i = 0; i < 256; ++i) { int32_t x = part[i]; part[i] = run; run += x; }
    unit_off[S] = run;
  }
  __syncthreads();
  acc = part[t];
  for (int s = s0; s < s1; ++s) { unit_off[s] = acc; acc += units(s); }
}

struct UnitRows {
  bool ok;
  int s;
  SeqGeom g;
  int t0;       // first query row (inside the sequence) of the unit
  int nq;       // valid query rows in the unit
};

// Without a unit table (every sequence has at most one row group and U = 1)
// unit s is sequence s.
__device__ __forceinline__ UnitRows locate_unit(const msa_seqs& sq, const int32_t* __restrict__ unit_off,
                                                int64_t uidx, int qr, int U) {
  UnitRows r;
  r.ok = false;
  if (!unit_off) {
    if (uidx >= sq.num_seqs) return r;
    r.s = static_cast<int>(uidx);
    r.g = seq_geom(sq, r.s);
    r.t0 = 0;
  } else {
    if (uidx >= unit_off[sq.num_seqs]) return r;
    r.s = find_seq_wave(unit_off, sq.num_seqs, uidx);
    r.g = seq_geom(sq, r.s);
    r.t0 = static_cast<int>(uidx - unit_off[r.s]) * qr * U;
  }
  r.nq = min(qr * U, r.g.q_rows - r.t0);
  // never touch query rows past the query-side tensors
  const int64_t left = sq.total_q_rows - (static_cast<int64_t>(r.g.q_begin) + r.t0);
  if (left < r.nq) r.nq = static_cast<int>(left > 0 ? left : 0);
  r.ok = r.nq > 0 && r.g.q_begin >= 0;
  return r;
}

// B operand of S^T = K Q^T for the wave's 32 NJ index rows (NJ 32-column
// tiles); lane (n, h) supplies dims h*D/2 + 8*st .. +8 of row 32j + n.
template <int D_IDX, int NJ = 2>
__device__ __forceinline__ void load_index_rows(const uint16_t* __restrict__ qbase, int nvalid, int n, int h,
                                                bf16x8 (&bq)[NJ][D_IDX / 16]) {
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int row = 32 * j + n;
#pragma unroll
    for (int st = 0; st < D_IDX / 16; ++st)
      bq[j][st] = row < nvalid ? ld_bf16x8(qbase + static_cast<int64_t>(row) * D_IDX + h * (D_IDX / 2) + 8 * st)
                               : zero_bf16x8();
  }
}

// Block max of one key block for the wave's 64 rows from the S^T tiles: each
// lane holds half of the block's keys for its column; lanes 0-31 then own rows
// 0-31 and lanes 32-63 rows 32-63.
// (Column tiles j0, j0 + 1 of wider accumulators: rows 64 (j0 / 2) + lane.)
template <int MT, int NJ = 2>
__device__ __forceinline__ float block_max_rows(const f32x16 (&acc)[MT][NJ], int j0 = 0) {
  float pm[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    float m = acc[0][j0 + j][0];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, acc[i][j0 + j][e]);
    pm[j] = m;
  }
  auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(pm[0]), __float_as_uint(pm[1]), false, false);
  return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}

// ---------------------------------------------------------------- scores, LDS
constexpr int kStageBlocks = 16;      // block maxima staged per row before a 64-byte store
constexpr int kPieceBlocks = 16;      // blocks per piece maximum (the Top-k's finer skip test)
constexpr int kSurvivorCap = 1024;    // pieces per round of the Top-k's piece scan
constexpr int kSlicePieces = 4;       // pieces per 64-block CTA slice: PM[slice][row][4]

// One 16-byte piece per lane from global memory straight into LDS
// (global_load_lds_dwordx4): lane l writes bytes [16 l, 16 l + 16) after the
// wave-uniform LDS address dst.  Completion is counted by vmcnt.
__device__ __forceinline__ void lds_dma16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}

// A 64-key sub-block of K_idx in LDS, unpadded: key row r keeps its 16-byte
// segment s in slot s ^ kswz(r), so the A-operand reads of 8 and of 16
// consecutive lanes (16 consecutive rows, one segment) hit distinct banks.
template <int D_IDX>
__device__ __forceinline__ int kswz(int r) {
  if constexpr (D_IDX == 64) return (r & 7) ^ ((r >> 3) & 1);
  else return r & 15;
}
template <int D_IDX, int RW>
struct IdxSmem {
  uint4 k[2][64 * D_IDX / 8];                      // two sub-blocks, swizzled rows
  float stage[kWaves][RW][kStageBlocks + 1];       // per wave: RW rows x 16 block maxima
};

// Besides M, each CTA writes its 64-block slice's maximum per row (over the
// row's candidate blocks only) to CM[slice][row], the bound the Top-k kernel
// prunes with.  RW index rows per wave (64 or 128; a unit is 4 RW / 64 row
// groups): with 128 every K_idx operand read from LDS feeds four MFMAs.
// Keys are staged and scored 64 at a time whatever B_k is (a 128-key block is
// two sub-blocks whose maxima are merged) and go from HBM to LDS without a
// register copy, which lets the d_idx 128 / B_k 128 kernel run 3 CTAs per CU.
template <int D_IDX, int BK, int RW, bool PAGED>
__global__ __launch_bounds__(256, (RW == 64) ? 3 : 2) void index_block_max_lds_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, msa_seqs sq,
    const int32_t* __restrict__ unit_off, int H_kv, int qr, int64_t u0, int64_t u1, float* __restrict__ M,
    int64_t ldm, float* __restrict__ CM, int64_t cm_stride, float* __restrict__ PM) {
  static_assert(kBlocksPerCta == kWave, "a CTA slice is one Top-k chunk");
  static_assert(kStageBlocks == kPieceBlocks, "a piece ends where a store pass does");
  constexpr int KS = D_IDX / 16;                        // k-steps of the MFMA
  constexpr int SEGS = D_IDX / 8;                       // 16-byte segments per key row
  constexpr int SUB = BK / 64;                          // 64-key sub-blocks staged per block
  constexpr int CH = 64 * SEGS / 256;                   // 16-byte loads per thread per sub-block
  constexpr int NJ = RW / 32;                           // 32-row column tiles per wave
  constexpr int NP = RW / 64;                           // row groups per wave
  __shared__ IdxSmem<D_IDX, RW> sm;
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int64_t uidx = u0 + blockIdx.x;
  if (uidx >= u1) return;
  UnitRows ur = locate_unit(sq, unit_off, uidx, qr, kWaves * NP);
  if (!ur.ok) return;
  const int p_last = ur.g.kv_len - ur.g.q_rows + ur.t0 + ur.nq - 1;
  if (p_last < 0) return;
  const int kb0 = blockIdx.y * kBlocksPerCta;
  const int kb1 = min(min(kb0 + kBlocksPerCta, p_last / BK), static_cast<int>(ldm));
  if (kb0 >= kb1) return;                               // uniform over the CTA

  const int n = lane & 31, h = lane >> 5;
  const int wq0 = w * NP * qr;                          // this wave's first query row in the unit
  const int nvalid = max(0, min(NP * qr, ur.nq - wq0)) * H_kv;
  bf16x8 bq[NJ][KS];
  load_index_rows<D_IDX, NJ>(index_q + (static_cast<int64_t>(ur.g.q_begin + ur.t0 + wq0) * H_kv) * D_IDX, nvalid,
                             n, h, bq);
  // this wave's RW rows of M; the block maxima of a 16-block group are staged
  // in LDS and stored as 64-byte row segments (blocks past kb1 in the last
  // group hold stale values that no row reads: they are >= its local block)
  const int64_t slot0 = (uidx - u0) * (kWaves * RW) + w * RW;   // this wave's first row of M
  float* mrow0 = M + slot0 * ldm;
  // lane holds rows 64 s + lane; their candidate blocks end at their local blocks
  int lb_lane[NP];
  float cmax[NP], pmax[NP];
#pragma unroll
  for (int sp = 0; sp < NP; ++sp) {
    lb_lane[sp] = (ur.g.kv_len - ur.g.q_rows + ur.t0 + wq0 + (64 * sp + lane) / H_kv) / BK;
    cmax[sp] = -INFINITY;
    pmax[sp] = -INFINITY;
  }

  const KeyBlocks kbk = key_blocks(sq, ur.g, ur.s, 64);   // 64-key view of the blocks
  const uint16_t* kseq = index_k + (PAGED ? 0 : ur.g.kv_start) * D_IDX;
  const int tid = threadIdx.x;
  float bm_sub[NP];
  auto compute = [&](int buf, int sb) {
    if (nvalid == 0) return;
    const int kb = sb / SUB;
    float bm[NP];
#pragma unroll
    for (int sp = 0; sp < NP; ++sp) bm[sp] = -INFINITY;
    {
      f32x16 acc[2][NJ];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = 32 * i + n;
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = f32x16{};
#pragma unroll
        for (int st = 0; st < KS; ++st) {
          const bf16x8 a = __builtin_bit_cast(bf16x8, sm.k[buf][row * SEGS + ((h * (SEGS / 2) + st) ^ kswz<D_IDX>(row))]);
#pragma unroll
          for (int j = 0; j < NJ; ++j) acc[i][j] = mfma32x32x16(a, bq[j][st], acc[i][j]);
        }
      }
#pragma unroll
      for (int sp = 0; sp < NP; ++sp) bm[sp] = fmaxf(bm[sp], block_max_rows<2, NJ>(acc, 2 * sp));
    }
    if constexpr (SUB > 1) {
      if (sb % SUB != SUB - 1) {
#pragma unroll
        for (int sp = 0; sp < NP; ++sp) bm_sub[sp] = sb % SUB == 0 ? bm[sp] : fmaxf(bm_sub[sp], bm[sp]);
        return;
      }
#pragma unroll
      for (int sp = 0; sp < NP; ++sp) bm[sp] = fmaxf(bm[sp], bm_sub[sp]);
    }
#pragma unroll
    for (int sp = 0; sp < NP; ++sp) {
      if (kb < lb_lane[sp]) {
        cmax[sp] = fmaxf(cmax[sp], bm[sp]);
        pmax[sp] = fmaxf(pmax[sp], bm[sp]);
      }
      sm.stage[w][64 * sp + lane][kb & (kStageBlocks - 1)] = bm[sp];
    }
    if ((kb & (kStageBlocks - 1)) == kStageBlocks - 1 || kb + 1 == kb1) {
      // the piece's maximum over each row's candidate blocks: the 4 pieces of
      // the CTA's slice sit together per row, PM[slice][row][4], so that the
      // Top-k kernel reads a row's piece maxima four per 16-byte load
#pragma unroll
      for (int sp = 0; sp < NP; ++sp) {
        if (64 * sp + lane < nvalid)
          PM[(static_cast<int64_t>(blockIdx.y) * cm_stride + slot0 + 64 * sp + lane) * kSlicePieces +
             (kb / kPieceBlocks) % kSlicePieces] = pmax[sp];
        pmax[sp] = -INFINITY;
      }
      // the wave writes 16 rows x 64 B per store pass (4 lanes per row, 16 B each)
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      const int kbase = kb & ~(kStageBlocks - 1);
      const int qd = lane & 3;
#pragma unroll
      for (int pass = 0; pass < RW / 16; ++pass) {
        const int row = 16 * pass + (lane >> 2);
        const int b = kbase + 4 * qd;
        if (row < nvalid && b < ldm) {
          const float* src = &sm.stage[w][row][4 * qd];
          *reinterpret_cast<float4*>(mrow0 + static_cast<int64_t>(row) * ldm + b) =
              make_float4(src[0], src[1], src[2], src[3]);
        }
      }
    }
  };

  // Sub-blocks go from HBM straight into LDS (one 1 KiB piece per wave and
  // load); sub-block sb + 1 is in flight while sb is scored.
  const int sb0 = kb0 * SUB, sb1 = kb1 * SUB;
  auto dma = [&](int buf, int sb) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int piece = w * CH + c;
      const int q = piece * kWave + lane;
      const int r = q / SEGS, slot = q % SEGS;
      const int seg = slot ^ kswz<D_IDX>(r);
      const uint16_t* src;
      if constexpr (PAGED) src = kseq + (kbk.template row_as<true>(sb) + r) * D_IDX + 8 * seg;
      else src = kseq + static_cast<int64_t>(sb * 64 + r) * D_IDX + 8 * seg;
      lds_dma16(src, &sm.k[buf][piece * kWave]);
    }
  };
  // s_waitcnt 0 before each barrier: this wave's pieces of the next
  // sub-block have landed in LDS
  dma(0, sb0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int sb = sb0; sb < sb1; sb += 2) {
    if (sb + 1 < sb1) dma(1, sb + 1);
    compute(0, sb);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (sb + 1 >= sb1) break;
    if (sb + 2 < sb1) dma(0, sb + 2);
    compute(1, sb + 1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  // rows whose local block is at or below kb0 never read this entry
#pragma unroll
  for (int sp = 0; sp < NP; ++sp)
    if (64 * sp + lane < nvalid) CM[static_cast<int64_t>(blockIdx.y) * cm_stride + slot0 + 64 * sp + lane] = cmax[sp];
}

// ---------------------------------------------------------------- scores, per wave
// One wave: one row group (U = 1) against kSliceBlocks consecutive key blocks;
// the 4 waves of a CTA take 4 consecutive slices of one unit, so a CTA streams
// 4 x kSliceBlocks contiguous blocks.  Each row's block maxima are kept in
// registers and written as two 16-byte stores.
constexpr int kSliceBlocks = 8;

template <int D_IDX, int BK, bool PAGED>
__global__ __launch_bounds__(256) void index_block_max_wave_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, msa_seqs sq,
    const int32_t* __restrict__ unit_off, int H_kv, int qr, int64_t u0, int64_t u1, float* __restrict__ M,
    int64_t ldm) {
  constexpr int KS = D_IDX / 16;
  constexpr int MT = BK / 32;
  const int lane = lane_id();
  const int64_t uidx = u0 + blockIdx.y;
  const int slice = blockIdx.x * kWaves + threadIdx.x / kWave;
  if (uidx >= u1) return;
  UnitRows ur = locate_unit(sq, unit_off, uidx, qr, 1);
  if (!ur.ok) return;
  const int p_last = ur.g.kv_len - ur.g.q_rows + ur.t0 + ur.nq - 1;
  if (p_last < 0) return;
  const int kb1 = min(p_last / BK, static_cast<int>(ldm));
  const int kb0 = slice * kSliceBlocks;
  if (kb0 >= kb1) return;

  const int n = lane & 31, h = lane >> 5;
  const int nvalid = ur.nq * H_kv;
  bf16x8 bq[2][KS];
  load_index_rows<D_IDX>(index_q + (static_cast<int64_t>(ur.g.q_begin + ur.t0) * H_kv) * D_IDX, nvalid, n, h, bq);
  const KeyBlocks kbk = key_blocks(sq, ur.g, ur.s, BK);
  // Lane (n, h) takes key row 32 i + n, dims h d_idx / 2 + 8 st .. +8 at
  // k-step st.  d_idx 64 / B_k 64: a block (64 contiguous keys) is loaded as
  // whole rows, lane l taking 16-byte unit 64 c + l of load c (1 KiB per
  // load), and goes through the wave's LDS rows into the operand layout
  // (214 -> 204 us for 64 sequences x 4 rows at 128K); the wider variants
  // load the operands directly (staged, they spill or lose occupancy).
  constexpr bool kWhole = D_IDX == 64 && BK == 64;
  const uint16_t* kbase = index_k + (PAGED ? 0 : ur.g.kv_start) * D_IDX + h * (D_IDX / 2);
  auto load_a = [&](int kb, bf16x8 (&a)[MT][KS]) {
    if constexpr (kWhole) {
      const uint16_t* sb = index_k + (PAGED ? kbk.template row_as<true>(kb) : ur.g.kv_start + static_cast<int64_t>(kb) * BK) * D_IDX;
#pragma unroll
      for (int c = 0; c < MT * KS; ++c) a[c / KS][c % KS] = ld_bf16x8(sb + 8 * (kWave * c + lane));
    } else {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const uint16_t* kp = PAGED ? kbase + (kbk.template row_as<true>(kb) + 32 * i + n) * D_IDX
                                   : kbase + static_cast<int64_t>(kb * BK + 32 * i + n) * D_IDX;
#pragma unroll
        for (int st = 0; st < KS; ++st) a[i][st] = ld_bf16x8(kp + 8 * st);
      }
    }
  };
  // rows padded by 16 bytes: the operand reads (16 rows, one column) are
  // free of bank conflicts
  __shared__ __align__(16) uint16_t ks_lds[kWhole ? kWaves : 1][kWhole ? BK : 1][D_IDX + 8];
  auto to_operands = [&](bf16x8 (&a)[MT][KS]) {
    if constexpr (!kWhole) return;
    auto& rows = ks_lds[threadIdx.x / kWave];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");     // the previous block's reads are done
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < MT * KS; ++c) {
      const int u = kWave * c + lane;
      *reinterpret_cast<bf16x8*>(&rows[u / (D_IDX / 8)][8 * (u % (D_IDX / 8))]) = a[c / KS][c % KS];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int st = 0; st < KS; ++st)
        a[i][st] = *reinterpret_cast<const bf16x8*>(&rows[32 * i + n][h * (D_IDX / 2) + 8 * st]);
  };
  bf16x8 a[MT][KS], an[MT][KS];
  float mb[kSliceBlocks];
  load_a(kb0, a);
#pragma unroll
  for (int i = 0; i < kSliceBlocks; ++i) {
    const int kb = kb0 + i;
    mb[i] = 0.f;
    if (kb < kb1) {                                   // uniform
      // next block in flight during this one (clamped, unconditional load)
      load_a(kb + 1 < kb1 ? kb + 1 : kb, an);
      to_operands(a);
      f32x16 acc[MT][2];
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        acc[t][0] = f32x16{};
        acc[t][1] = f32x16{};
#pragma unroll
        for (int st = 0; st < KS; ++st) {
          acc[t][0] = mfma32x32x16(a[t][st], bq[0][st], acc[t][0]);
          acc[t][1] = mfma32x32x16(a[t][st], bq[1][st], acc[t][1]);
        }
      }
      mb[i] = block_max_rows<MT>(acc);
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int st = 0; st < KS; ++st) a[t][st] = an[t][st];
    }
  }
  // values past kb1 are never read (they are >= every row's local block) and
  // stay inside this slice; quads start below ldm (a multiple of 4)
  if (lane < nvalid) {
    float* mrow = M + ((uidx - u0) * kWave + lane) * ldm + kb0;
#pragma unroll
    for (int q4 = 0; q4 < kSliceBlocks / 4; ++q4)
      if (kb0 + 4 * q4 < ldm)
        *reinterpret_cast<float4*>(mrow + 4 * q4) = make_float4(mb[4 * q4], mb[4 * q4 + 1], mb[4 * q4 + 2], mb[4 * q4 + 3]);
  }
}

// Narrow variant for row groups of at most 16 index rows (decode: one query
// row x H_kv <= 16 groups): MFMA 16x16x32 with keys as M and the rows as N
// needs a quarter of the registers, so DEPTH sub-blocks stream through
// registers per wave (clamped, unconditional whole-row loads, turned into
// operands through the wave's LDS rows) and more waves share each CU.
// Lane (n, q4) supplies key 16i + n / row n and dims 32ks + 8q4 .. +8; C lane
// (n, q4) holds row n, keys 16i + 4q4 + e.
template <int D_IDX, int BK, int DEPTH, bool PAGED>
__global__ __launch_bounds__(256) void index_block_max_narrow_kernel(
    const uint16_t* __restrict__ index_q, const uint16_t* __restrict__ index_k, msa_seqs sq,
    const int32_t* __restrict__ unit_off, int H_kv, int qr, int64_t u0, int64_t u1, float* __restrict__ M,
    int64_t ldm) {
  constexpr int KS = D_IDX / 32;
  constexpr int HB = BK / 64;                         // 64-key sub-blocks per block
  constexpr int MT = 4;                               // 16-key tiles per sub-block
  const int lane = lane_id();
  const int64_t uidx = u0 + blockIdx.y;
  const int slice = blockIdx.x * kWaves + threadIdx.x / kWave;
  if (uidx >= u1) return;
  UnitRows ur = locate_unit(sq, unit_off, uidx, qr, 1);
  if (!ur.ok) return;
  const int p_last = ur.g.kv_len - ur.g.q_rows + ur.t0 + ur.nq - 1;
  if (p_last < 0) return;
  const int kb1 = min(p_last / BK, static_cast<int>(ldm));
  const int kb0 = slice * kSliceBlocks;
  if (kb0 >= kb1) return;

  const int n = lane & 15, q4 = lane >> 4;
  const int nvalid = min(ur.nq * H_kv, 16);
  bf16x8 bq[KS];
  const uint16_t* qrow = index_q + (static_cast<int64_t>(ur.g.q_begin + ur.t0) * H_kv + n) * D_IDX + 8 * q4;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) bq[ks] = n < nvalid ? ld_bf16x8(qrow + 32 * ks) : zero_bf16x8();
  const KeyBlocks kbk = key_blocks(sq, ur.g, ur.s, BK);

  // sub-block j = keys 64 (j % HB) .. +63 of block kb0 + j / HB.  Blocks kb0
  // .. kb1-1 are entirely before every row's local block, hence inside the
  // sequence; loads past kb1 re-read block kb1-1.  Paged: lane i holds the
  // page of the slice's block i, fetched once.
  const int64_t my_prow = PAGED ? kbk.template row_as<true>(min(kb0 + (lane % kSliceBlocks), kb1 - 1)) : 0;
  // A sub-block (64 contiguous keys of d_idx bf16) is loaded as whole rows,
  // lane l taking 16-byte unit 64 c + l of load c (1 KiB per load, instead
  // of 64-byte pieces of 16 rows: 192 -> 187 us per 128K decode step at
  // d_idx 64), and goes through the wave's LDS rows into the operand layout.
  auto load_a = [&](int j, bf16x8 (&a)[MT][KS]) {
    const int kb = min(kb0 + j / HB, kb1 - 1);
    const int k0 = 64 * (j % HB);
    const int64_t prow = PAGED ? static_cast<int64_t>(readlane_u64(static_cast<uint64_t>(my_prow), j / HB)) : 0;
    const uint16_t* sb = index_k + (PAGED ? prow + k0 : (ur.g.kv_start + static_cast<int64_t>(kb) * BK + k0)) * D_IDX;
#pragma unroll
    for (int c = 0; c < MT * KS; ++c) a[c / KS][c % KS] = ld_bf16x8(sb + 8 * (kWave * c + lane));
  };
  // rows padded by 16 bytes: the operand reads (16 rows, one column) are
  // free of bank conflicts
  __shared__ __align__(16) uint16_t ks_lds[kWaves][64][D_IDX + 8];
  auto to_operands = [&](bf16x8 (&a)[MT][KS]) {
    auto& rows = ks_lds[threadIdx.x / kWave];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");     // the previous sub-block's reads are done
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < MT * KS; ++c) {
      const int u = kWave * c + lane;
      *reinterpret_cast<bf16x8*>(&rows[u / (D_IDX / 8)][8 * (u % (D_IDX / 8))]) = a[c / KS][c % KS];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) a[i][ks] = *reinterpret_cast<const bf16x8*>(&rows[16 * i + n][32 * ks + 8 * q4]);
  };
  bf16x8 buf[DEPTH][MT][KS];
#pragma unroll
  for (int d = 0; d < DEPTH; ++d) load_a(d, buf[d]);
  float mb[kSliceBlocks];
#pragma unroll
  for (int j = 0; j < kSliceBlocks * HB; ++j) {
    bf16x8 (&a)[MT][KS] = buf[j % DEPTH];
    to_operands(a);
    f32x4 acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      acc[t] = f32x4{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc[t] = mfma16x16x32(a[t][ks], bq[ks], acc[t]);
    }
    float m = acc[0][0];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e) m = fmaxf(m, acc[t][e]);
    m = fmaxf(m, __uint_as_float(xor_lane_u32<16>(__float_as_uint(m))));
    m = fmaxf(m, __uint_as_float(xor_lane_u32<32>(__float_as_uint(m))));
    mb[j / HB] = j % HB == 0 ? m : fmaxf(mb[j / HB], m);
    if (j + DEPTH < kSliceBlocks * HB) load_a(j + DEPTH, a);
  }
  // values past kb1 are never read (they are >= every row's local block) and
  // stay inside this slice; quads start below ldm (a multiple of 4)
  if (lane < nvalid) {
    float* mrow = M + ((uidx - u0) * kWave + lane) * ldm + kb0;
#pragma unroll
    for (int q = 0; q < kSliceBlocks / 4; ++q)
      if (kb0 + 4 * q < ldm)
        *reinterpret_cast<float4*>(mrow + 4 * q) = make_float4(mb[4 * q], mb[4 * q + 1], mb[4 * q + 2], mb[4 * q + 3]);
  }
}

// ---------------------------------------------------------------- top-k
// Inserts the keys v (one per lane; 0 = none) that beat `thr` into `list`
// (sorted descending across lanes) and returns the new K1-th best key.
__device__ __forceinline__ uint64_t insert_keys(uint64_t v, uint64_t thr, int K1, uint64_t& list) {
  const int lane = lane_id();
  uint64_t pass = __ballot(v > thr);
  if (pass == 0) return readlane_u64(list, K1 - 1);
  if (__popcll(pass) <= kSmallInsert) {
    while (pass) {
      const int src = __ffsll(static_cast<unsigned long long>(pass)) - 1;
      pass &= pass - 1;
      const uint64_t xk = readlane_u64(v, src);
      const int rnk = __popcll(__ballot(list > xk));
      const uint64_t prev = lane_shr1_u64(list, list);
      list = lane < rnk ? list : (lane == rnk ? xk : prev);
    }
  } else {
    const uint64_t vs = wave_sort_desc_u64(v > thr ? v : 0ull);
    const uint64_t rev = shfl_u64(vs, kWave - 1 - lane);
    list = wave_bitonic_merge_desc_u64(list > rev ? list : rev);
  }
  return readlane_u64(list, K1 - 1);
}

// Keys that beat the running threshold are appended to a per-wave LDS
// buffer (128 entries) and merged into the sorted list 64 at a time: one
// bitonic sort + merge per 64 candidates instead of one insertion each.  The
// threshold only rises at a merge, so some extra keys are buffered; the list
// after flush() is still exactly the best K1 (and more) of all pushed keys.
struct KeyBatch {
  uint64_t* pend;    // this wave's 128-entry LDS buffer
  int cnt;           // buffered keys (wave-uniform, < 64 between calls)
  int K1;
  uint64_t list;     // sorted descending across the lanes; 0 marks an empty slot

  __device__ __forceinline__ void merge(uint64_t v) {
    const uint64_t vs = wave_sort_desc_u64(v);
    const uint64_t rev = shfl_u64(vs, kWave - 1 - lane_id());
    list = wave_bitonic_merge_desc_u64(list > rev ? list : rev);
  }
  // pushes the lanes' keys above thr; returns the new threshold (>= thr)
  __device__ __forceinline__ uint64_t push(uint64_t v, uint64_t thr) {
    const int lane = lane_id();
    const bool take = v > thr;
    const uint64_t pass = __ballot(take);
    if (pass == 0) return thr;
    const int pos = cnt + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(pass >> 32),
                                                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(pass), 0));
    if (take) pend[pos] = v;
    cnt += __popcll(pass);
    if (cnt < kWave) return thr;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const uint64_t x = pend[lane];
    const uint64_t y = pend[kWave + lane];
    merge(x);
    cnt -= kWave;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < cnt) pend[lane] = y;
    const uint64_t t = readlane_u64(list, K1 - 1);
    return t > thr ? t : thr;
  }
  __device__ __forceinline__ void flush() {
    if (cnt == 0) return;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int lane = lane_id();
    merge(lane < cnt ? pend[lane] : 0ull);
    cnt = 0;
  }
};

// Streams chunks c_begin, c_begin + c_step, ... (64 scores each) of one row,
// score b read as load(b), and hands each chunk's keys to ins(v, tau) (which
// returns the new threshold).
template <typename Load, typename Ins>
__device__ __forceinline__ void stream_chunks(Load load, int nscan, int c_begin, int c_step, Ins ins) {
  const int lane = lane_id();
  uint64_t tau = 0;    // key of the K1-th best so far (0 while fewer are known)
  // block scores of the next kAhead chunks are in flight while one is ranked
  constexpr int kAhead = 4;
  float pf[kAhead];
#pragma unroll
  for (int a = 0; a < kAhead; ++a) {
    const int b = (c_begin + a * c_step) * kWave + lane;
    pf[a] = b < nscan ? load(b) : 0.f;
  }
  for (int c = c_begin; c * kWave < nscan; c += c_step) {
    const int b = c * kWave + lane;
    const float x = pf[0];
#pragma unroll
    for (int a = 0; a + 1 < kAhead; ++a) pf[a] = pf[a + 1];
    {
      const int bn = (c + kAhead * c_step) * kWave + lane;
      pf[kAhead - 1] = bn < nscan ? load(bn) : 0.f;
    }
    const uint64_t v = b < nscan ? rank_key(x, static_cast<uint32_t>(b)) : 0ull;
    tau = ins(v, tau);
  }
}

// The row's best keys of chunks c_begin, c_begin + c_step, ..., sorted
// descending across the lanes (at least the best K1 are exact); keys are
// inserted one chunk at a time.
template <typename Load>
__device__ __forceinline__ uint64_t scan_row_chunks(Load load, int nscan, int K1, int c_begin, int c_step) {
  uint64_t list = 0;
  if (K1 <= 0) return list;
  stream_chunks(load, nscan, c_begin, c_step, [&](uint64_t v, uint64_t t) { return insert_keys(v, t, K1, list); });
  return list;
}

// The same selection through a KeyBatch.
template <typename Load>
__device__ __forceinline__ uint64_t scan_row_batched(Load load, int nscan, KeyBatch& kb) {
  kb.list = 0;
  kb.cnt = 0;
  if (kb.K1 <= 0) return 0;
  stream_chunks(load, nscan, 0, 1, [&](uint64_t v, uint64_t t) { return kb.push(v, t); });
  kb.flush();
  return kb.list;
}

// The same selection with chunk and piece maxima: chunk c of the row
// (scores 64c .. 64c+63) has maximum cm(c), piece q (scores 16q .. 16q+15)
// maximum pm(q), both over candidate blocks only.  The K1-th largest chunk
// maximum t0 is a lower bound of the row's K1-th best score (K1 distinct
// chunks each hold a score >= t0), so pieces with maximum below t0 are
// skipped and scores below t0 are never ranked.  Surviving pieces are read
// four per wave load (lanes 16 k .. 16 k + 15 take the k-th).
template <typename Load, typename LoadCm, typename LoadPm>
__device__ __forceinline__ uint64_t scan_row_pruned(Load load, LoadCm cm, LoadPm pm, int nscan, KeyBatch& kb,
                                                    int32_t* surv) {
  const int lane = lane_id();
  const int K1 = kb.K1;
  const int nchunk = (nscan + kWave - 1) / kWave;
  if (K1 <= 0 || nchunk <= K1) return scan_row_batched(load, nscan, kb);
  const uint64_t t0key = readlane_u64(scan_row_batched(cm, nchunk, kb), K1 - 1);
  const uint32_t o0 = static_cast<uint32_t>(t0key >> 32);     // ordered score of t0
  // keys above floor_key have scores >= t0 (o0 > 0 for every non-NaN score)
  const uint64_t floor_key = o0 > 0 ? (static_cast<uint64_t>(o0) << 32) - 1 : 0ull;

  const int npiece = (nscan + kPieceBlocks - 1) / kPieceBlocks;
  kb.list = 0;
  kb.cnt = 0;
  uint64_t tau = floor_key;
  // pieces in rounds of kSurvivorCap: the round's piece maxima are loaded
  // together, the indices of the pieces that reach t0 appended to the wave's
  // LDS list in piece order, then their scores read four pieces per wave load
  // (lanes 16 k .. 16 k + 15 take the k-th) with kAhead loads in flight
  constexpr int kGroups = kSurvivorCap / kWave;
  for (int r0 = 0; r0 < npiece; r0 += kSurvivorCap) {
    float pv[kGroups];
#pragma unroll
    for (int k = 0; k < kGroups; ++k) {
      const int c = r0 + kWave * k + lane;
      pv[k] = c < npiece ? pm(c) : 0.f;
    }
    int ns = 0;
#pragma unroll
    for (int k = 0; k < kGroups; ++k) {
      const int c = r0 + kWave * k + lane;
      const bool ok = c < npiece && ordered_u32(pv[k]) >= o0;
      const uint64_t m = __ballot(ok);
      if (ok)
        surv[ns + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                            __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0))] = c;
      ns += __popcll(m);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int nquad = (ns + 3) / 4;
    auto quad_piece = [&](int i) -> int {
      const int q = 4 * i + (lane >> 4);
      return i < nquad && q < ns ? surv[q] : -1;
    };
    constexpr int kAhead = 4;
    int lp[kAhead];
    float pf[kAhead];
#pragma unroll
    for (int a = 0; a < kAhead; ++a) {
      lp[a] = quad_piece(a);
      const int b = lp[a] * kPieceBlocks + (lane & 15);
      pf[a] = (lp[a] >= 0 && b < nscan) ? load(b) : 0.f;
    }
    for (int i = 0; i < nquad; ++i) {
      const int b = lp[0] * kPieceBlocks + (lane & 15);
      const bool ok = lp[0] >= 0 && b < nscan;
      const float x = pf[0];
#pragma unroll
      for (int a = 0; a + 1 < kAhead; ++a) {
        lp[a] = lp[a + 1];
        pf[a] = pf[a + 1];
      }
      lp[kAhead - 1] = quad_piece(i + kAhead);
      {
        const int bn = lp[kAhead - 1] * kPieceBlocks + (lane & 15);
        pf[kAhead - 1] = (lp[kAhead - 1] >= 0 && bn < nscan) ? load(bn) : 0.f;
      }
      const uint64_t v = ok ? rank_key(x, static_cast<uint32_t>(b)) : 0ull;
      tau = kb.push(v, tau);
    }
    // the next round rewrites the list
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  kb.flush();
  return kb.list;
}

// ---------------------------------------------------------------- radix selection
// The largest t such that at least K of the wave's values x[0 .. V) (all
// lanes; absent values are 0) are >= t: the K-th largest value when at least K
// are present.  Bit by bit from the top, one compare per value and bit; the
// counts are wave-uniform (ballot + popcount), so no value moves between lanes.
// With LOBIT > 0 only bits 31 .. LOBIT are decided (the lower ones stay 0):
// a lower bound of that value, within 2^LOBIT of it.
template <int V, int LOBIT = 0>
__device__ __forceinline__ uint32_t kth_largest_u32(const uint32_t* x, int K) {
  uint32_t t = 0;
  for (int bit = 31; bit >= LOBIT; --bit) {
    const uint32_t c = t | (1u << bit);
    int n = 0;
#pragma unroll
    for (int v = 0; v < V; ++v) n += __popcll(__ballot(x[v] >= c));
    if (n >= K) t = c;
  }
  return t;
}

// A lower bound of the K-th largest of up to 16 values per lane (nv used),
// exact in its top 16 bits (for an ordered float: sign, exponent and 7
// mantissa bits).
__device__ __forceinline__ uint32_t kth_largest_bound(const uint32_t* x, int nv, int K) {
  if (nv <= 2) return kth_largest_u32<2, 16>(x, K);
  if (nv <= 4) return kth_largest_u32<4, 16>(x, K);
  if (nv <= 8) return kth_largest_u32<8, 16>(x, K);
  return kth_largest_u32<16, 16>(x, K);
}

__device__ __forceinline__ int lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0));
}

// The K best of the cnt (<= 2 kWave) distinct non-zero keys in the wave's
// LDS buffer `buf`: the K-th largest key kk is found by a radix search on the
// score half, and on the id half among equal scores at the boundary; the keys
// >= kk (all of them when cnt <= K) are compacted to the front of `buf` and
// returned one per lane in lanes 0 .. min(cnt, K)-1 (in no order; other
// lanes 0).  With `kth` non-null, *kth receives kk (0 when cnt <= K).
__device__ __forceinline__ uint64_t best_keys(uint64_t* buf, int cnt, int K, uint64_t* kth) {
  const int lane = lane_id();
  const uint64_t c0 = lane < cnt ? buf[lane] : 0ull;
  const uint64_t c1 = kWave + lane < cnt ? buf[kWave + lane] : 0ull;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  uint64_t kk = 0;
  if (cnt > K) {
    uint32_t h[2] = {static_cast<uint32_t>(c0 >> 32), static_cast<uint32_t>(c1 >> 32)};
    const uint32_t tv = kth_largest_u32<2>(h, K);
    const int n_gt = __popcll(__ballot(h[0] > tv)) + __popcll(__ballot(h[1] > tv));
    const int n_eq = __popcll(__ballot(h[0] == tv && c0 != 0ull)) + __popcll(__ballot(h[1] == tv && c1 != 0ull));
    const int need = K - n_gt;                              // 1 <= need <= n_eq
    kk = static_cast<uint64_t>(tv) << 32;
    if (n_eq != need) {
      uint32_t l[2] = {h[0] == tv && c0 != 0ull ? static_cast<uint32_t>(c0) : 0u,
                       h[1] == tv && c1 != 0ull ? static_cast<uint32_t>(c1) : 0u};
      kk |= kth_largest_u32<2>(l, need);
    }
  }
  if (kth) *kth = kk;
  const bool s0 = c0 != 0ull && c0 >= kk, s1 = c1 != 0ull && c1 >= kk;
  const uint64_t m0 = __ballot(s0), m1 = __ballot(s1);
  if (s0) buf[lanes_below(m0)] = c0;
  if (s1) buf[__popcll(m0) + lanes_below(m1)] = c1;
  const int nsel = __popcll(m0) + __popcll(m1);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const uint64_t list = lane < nsel && lane < K ? buf[lane] : 0ull;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  return list;
}

// Exact selection of a row through radix searches instead of sorting
// networks.  A bound t1 <= the row's K1-th best score -- the K1-th largest
// piece maximum (K1 distinct pieces each hold a score >= it), or for rows of
// at most K1 pieces the K1-th largest score itself, either to 16 bits from
// below -- leaves few candidates: the scores >= t1 (of the pieces that reach
// t1) are appended as keys to `buf` (2 kWave entries) and the K1-th largest
// key among them is found by a radix search on the score half, and on the id
// half among equal scores at the boundary.  On return lanes 0 .. K1-1 of
// `list` hold the K1 best keys (in no order).  Returns false, deciding
// nothing, when the candidates overflow `buf` (rows with many equal scores)
// or the row has more than kSurvivorCap pieces; the caller then ranks the row
// by the pruned scan.  M rows are 16-byte aligned with a multiple of 4 floats.
template <typename LoadPm4>
__device__ __forceinline__ bool select_row_radix(const float* __restrict__ mrow, LoadPm4 pm4, int nscan, int K1,
                                                 uint64_t* buf, int32_t* surv, uint64_t& list) {
  const int lane = lane_id();
  if (K1 <= 0) return false;
  if (nscan <= K1) {                                      // every candidate block is selected
    list = lane < nscan ? rank_key(0.f, static_cast<uint32_t>(lane)) : 0ull;
    return true;
  }
  const int npiece = (nscan + kPieceBlocks - 1) / kPieceBlocks;
  if (npiece > kSurvivorCap) return false;
  const bool direct = npiece <= K1;                       // rank the scores themselves
  const int nval = direct ? nscan : npiece;               // <= kSurvivorCap either way
  constexpr int kGroups = kSurvivorCap / kWave;
  // value k of this lane: score 64 k + lane (direct), else piece
  // 4 (64 (k / 4) + lane) + k % 4 (the lane's slices, four pieces per load)
  const int nv = direct ? (nval + kWave - 1) / kWave : kSlicePieces * ((nval + kSlicePieces * kWave - 1) / (kSlicePieces * kWave));
  auto value_id = [&](int k) { return direct ? kWave * k + lane : kSlicePieces * (kWave * (k / kSlicePieces) + lane) + k % kSlicePieces; };
  uint32_t pv[kGroups];
  if (direct) {
#pragma unroll
    for (int k = 0; k < kGroups; ++k) {
      const int c = kWave * k + lane;
      pv[k] = k < nv && c < nval ? ordered_u32(mrow[c]) : 0u;
    }
  } else {
#pragma unroll
    for (int kk = 0; kk < kGroups / kSlicePieces; ++kk) {
      const int ch = kWave * kk + lane;
      const f32x4 x = kSlicePieces * kk < nv && kSlicePieces * ch < nval ? pm4(ch) : f32x4{};
#pragma unroll
      for (int e = 0; e < kSlicePieces; ++e)
        pv[kSlicePieces * kk + e] = kSlicePieces * ch + e < nval ? ordered_u32(x[e]) : 0u;
    }
  }
  const uint32_t t1 = kth_largest_bound(pv, nv, K1);
  if (t1 == 0) return false;
  // the float with ordered value t1 (scores compare against it directly)
  const float t1f = __uint_as_float((t1 & 0x80000000u) ? (t1 & 0x7FFFFFFFu) : ~t1);
  constexpr int kBuf = 2 * kWave;
  int cnt = 0;
  auto append = [&](bool take, float x, int b) {
    const uint64_t m = __ballot(take);
    const int pos = cnt + lanes_below(m);
    if (take && pos < kBuf) buf[pos] = rank_key(x, static_cast<uint32_t>(b));
    cnt += __popcll(m);
  };
  if (direct) {
#pragma unroll
    for (int k = 0; k < kGroups; ++k)
      if (k < nv) {
        const int c = kWave * k + lane;
        append(pv[k] >= t1, __uint_as_float((pv[k] & 0x80000000u) ? (pv[k] & 0x7FFFFFFFu) : ~pv[k]), c);
      }
  } else {
    int ns = 0;
#pragma unroll
    for (int k = 0; k < kGroups; ++k)
      if (k < nv) {
        const bool ok = pv[k] >= t1;
        const uint64_t m = __ballot(ok);
        if (ok) surv[ns + lanes_below(m)] = value_id(k);
        ns += __popcll(m);
      }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // scores of the surviving pieces, 16 pieces per wave load: lane l reads
    // blocks 4 (l & 3) .. + 3 of piece surv[16 i + (l >> 2)] as one float4;
    // rounds of 8 loads, all in flight together
    constexpr int kLoads = 8;
    for (int r0 = 0; r0 < ns; r0 += 16 * kLoads) {
      f32x4 x[kLoads];
      int bb[kLoads];
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        const int q = r0 + 16 * i + (lane >> 2);
        bb[i] = q < ns ? kPieceBlocks * surv[q] + 4 * (lane & 3) : nscan;
        x[i] = bb[i] < nscan ? *reinterpret_cast<const f32x4*>(mrow + bb[i]) : f32x4{};
      }
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        if (r0 + 16 * i >= ns) break;
#pragma unroll
        for (int e = 0; e < 4; ++e) append(bb[i] + e < nscan && x[i][e] >= t1f, x[i][e], bb[i] + e);
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (cnt > kBuf || cnt < K1) return false;
  list = best_keys(buf, cnt, K1, nullptr);
  return true;
}

// Local block + the K1 best keys of `list`, ids ascending, -1 padded.
__device__ __forceinline__ void finish_row(uint64_t list, int K1, int lb, int topk, int32_t* __restrict__ out) {
  const int lane = lane_id();
  const int cnt = K1 > 0 ? __popcll(__ballot(lane < K1 && list != 0ull)) : 0;
  uint32_t id = 0xFFFFFFFFu;
  if (lane < cnt) id = key_block(list);
  else if (lane == cnt) id = static_cast<uint32_t>(lb);
  id = wave_sort_asc_u32(id);
  if (lane < topk) out[lane] = lane <= cnt ? static_cast<int32_t>(id) : -1;
}

struct RowTask {
  bool ok;
  int lb, nscan;
  int32_t* out;
  const float* mrow;
  int64_t slot;         // the row's index in the chunk's score rows
  bool no_position;
};

// Task `task` of a chunk: index row L = task % rpu of unit u0 + task / rpu,
// where rpu (<= U * 64) bounds the index rows a unit can hold.
__device__ __forceinline__ RowTask locate_row(const float* __restrict__ M, int64_t ldm, const msa_seqs& sq,
                                              const int32_t* __restrict__ unit_off, int H_kv, int qr, int U,
                                              int rpu, int64_t u0, int64_t task, int BK, int topk,
                                              int32_t* __restrict__ block_ids) {
  RowTask t;
  t.ok = false;
  t.no_position = false;
  // task is wave-uniform and below 2^32 (the host checks), H_kv and BK are
  // powers of two: the arithmetic stays scalar and 32-bit
  const uint32_t tk = static_cast<uint32_t>(task);
  const uint32_t uq = tk / static_cast<uint32_t>(rpu);
  const int64_t uidx = u0 + uq;
  const int L = static_cast<int>(tk - uq * static_cast<uint32_t>(rpu));   // index row inside the unit
  const int64_t slot = (uidx - u0) * (static_cast<int64_t>(U) * kWave) + L;
  UnitRows ur = locate_unit(sq, unit_off, uidx, qr, U);
  if (!ur.ok || L >= ur.nq * H_kv) return t;
  const int row = ur.t0 + (L >> __builtin_ctz(H_kv));
  const int r = L & (H_kv - 1);
  t.out = block_ids + (static_cast<int64_t>(ur.g.q_begin + row) * H_kv + r) * topk;
  const int p = ur.g.kv_len - ur.g.q_rows + row;
  t.ok = true;
  if (p < 0) {
    t.no_position = true;
    return t;
  }
  t.lb = p >> __builtin_ctz(BK);
  t.nscan = min(t.lb, static_cast<int>(ldm));      // == lb whenever kv_lens respect max_kv_len
  t.mrow = M + slot * ldm;
  t.slot = slot;
  return t;
}

// One wave per index row.  With chunk maxima (CM[chunk][row], row stride
// cm_stride) the row is ranked by the pruned scan.
__global__ __launch_bounds__(256) void index_topk_kernel(
    const float* __restrict__ M, int64_t ldm, const float* __restrict__ CM, int64_t cm_stride,
    const float* __restrict__ PM, msa_seqs sq,
    const int32_t* __restrict__ unit_off, int H_kv, int qr, int U, int rpu, int64_t u0, int64_t u1, int BK,
    int topk, int32_t* __restrict__ block_ids) {
  __shared__ uint64_t s_pend[kWaves][2 * kWave];
  __shared__ int32_t s_surv[kWaves][kSurvivorCap];
  const int lane = lane_id();
  const int64_t task = static_cast<int64_t>(blockIdx.x) * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x) / kWave;
  if (task >= (u1 - u0) * rpu) return;
  const RowTask t = locate_row(M, ldm, sq, unit_off, H_kv, qr, U, rpu, u0, task, BK, topk, block_ids);
  if (!t.ok) return;
  if (t.no_position) {
    if (lane < topk) t.out[lane] = -1;
    return;
  }
  const float* mrow = t.mrow;
  auto load = [=](int b) { return mrow[b]; };
  KeyBatch kb;
  kb.pend = s_pend[threadIdx.x / kWave];
  kb.K1 = topk - 1;
  uint64_t list;
  if (CM) {
    const float* cmrow = CM + t.slot;
    auto cm = [=](int c) { return cmrow[static_cast<int64_t>(c) * cm_stride]; };
    const float* pmrow = PM + t.slot * kSlicePieces;
    auto pm = [=](int q) { return pmrow[static_cast<int64_t>(q / kSlicePieces) * cm_stride * kSlicePieces + q % kSlicePieces]; };
    auto pm4 = [=](int ch) { return *reinterpret_cast<const f32x4*>(pmrow + static_cast<int64_t>(ch) * cm_stride * kSlicePieces); };
    if (!select_row_radix(mrow, pm4, t.nscan, topk - 1, kb.pend, s_surv[threadIdx.x / kWave], list))
      list = scan_row_pruned(load, cm, pm, t.nscan, kb, s_surv[threadIdx.x / kWave]);
  } else {
    list = scan_row_batched(load, t.nscan, kb);
  }
  finish_row(list, topk - 1, t.lb, topk, t.out);
}

// kSplitWaves waves per index row (for few rows): wave w scans chunks w,
// w + kSplitWaves, ...; the partial lists are merged pairwise through LDS in
// log2(kSplitWaves) steps.
constexpr int kSplitWaves = 16;

__global__ __launch_bounds__(64 * kSplitWaves) void index_topk_split_kernel(
    const float* __restrict__ M, int64_t ldm, msa_seqs sq, const int32_t* __restrict__ unit_off, int H_kv,
    int qr, int U, int rpu, int64_t u0, int64_t u1, int BK, int topk, int32_t* __restrict__ block_ids) {
  __shared__ uint64_t lists[kSplitWaves][kWave];
  const int lane = lane_id();
  const int w = threadIdx.x / kWave;
  const int64_t task = blockIdx.x;
  if (task >= (u1 - u0) * rpu) return;              // uniform over the CTA
  const RowTask t = locate_row(M, ldm, sq, unit_off, H_kv, qr, U, rpu, u0, task, BK, topk, block_ids);
  if (!t.ok) return;                                 // uniform
  if (t.no_position) {
    if (w == 0 && lane < topk) t.out[lane] = -1;
    return;
  }
  const int K1 = topk - 1;
  const float* mrow = t.mrow;
  uint64_t list = scan_row_chunks([=](int b) { return mrow[b]; }, t.nscan, K1, w, kSplitWaves);
  lists[w][lane] = list;
  // step s: wave w (a multiple of 2s) merges in wave w + s's list, written at
  // the previous step; the barrier orders the steps
#pragma unroll
  for (int s = 1; s < kSplitWaves; s <<= 1) {
    __syncthreads();
    if ((w & (2 * s - 1)) == 0) {
      const uint64_t rev = lists[w + s][kWave - 1 - lane];   // ascending: bitonic with `list`
      list = wave_bitonic_merge_desc_u64(list > rev ? list : rev);
      lists[w][lane] = list;
    }
  }
  if (w == 0) finish_row(list, K1, t.lb, topk, t.out);
}

// ---------------------------------------------------------------- row Top-k
// The k best (score, column) keys of one row of n fp32 scores, for one wave
// (k <= 64): lanes 0 .. min(n, k)-1 of the result hold them, in no order.
// The row is read in rounds of RP values per lane (VEC: float4 loads; the
// row is 16-byte aligned and a load that starts below n stays inside its
// allocation).  A round's bound is the k-th largest of the lanes' maxima (k
// distinct lanes hold a score at least that large), raised to the running
// bound; the round's scores at or above it are appended as keys to the
// wave's LDS buffer `buf` (2 kWave entries).  A buffer more than half full
// is cut to its k best, whose k-th key raises the bound.  The k best keys of
// the buffer are the row's.  A row whose candidates still overflow the
// buffer (many equal scores) is streamed again through a key batch.
template <bool VEC, int RP>
__device__ __forceinline__ uint64_t row_best_keys(const float* __restrict__ srow, int n, int k, uint64_t* buf) {
  const int lane = lane_id();
  constexpr int kBuf = 2 * kWave;
  uint32_t t = 0;                  // ordered bound: the row's k-th best score is >= it
  int cnt = 0;
  bool fits = true;
  for (int c0 = 0; c0 < n; c0 += kWave * RP) {
    // column of value v of this lane: VEC c0 + 256 (v / 4) + 4 lane + v % 4, else c0 + 64 v + lane
    auto col_of = [&](int v) { return VEC ? c0 + 4 * kWave * (v / 4) + 4 * lane + v % 4 : c0 + kWave * v + lane; };
    float x[RP];
    if constexpr (VEC) {
#pragma unroll
      for (int i = 0; i < RP / 4; ++i) {
        const int c = col_of(4 * i);
        const f32x4 q = c < n ? *reinterpret_cast<const f32x4*>(srow + c) : f32x4{};
#pragma unroll
        for (int e = 0; e < 4; ++e) x[4 * i + e] = q[e];
      }
    } else {
#pragma unroll
      for (int v = 0; v < RP; ++v) x[v] = col_of(v) < n ? srow[col_of(v)] : 0.f;
    }
    uint32_t lm = 0;
#pragma unroll
    for (int v = 0; v < RP; ++v) {
      const uint32_t o = col_of(v) < n ? ordered_u32(x[v]) : 0u;
      lm = o > lm ? o : lm;
    }
    // the k-th largest lane maximum to its top 16 bits (a lower bound: half
    // the search steps; the cut below raises the bound exactly)
    const uint32_t tr = kth_largest_u32<1, 16>(&lm, k);
    t = tr > t ? tr : t;
#pragma unroll
    for (int v = 0; v < RP; ++v) {
      const int c = col_of(v);
      const bool take = c < n && ordered_u32(x[v]) >= t;
      const uint64_t m = __ballot(take);
      if (m == 0) continue;
      const int pos = cnt + lanes_below(m);
      if (take && pos < kBuf) buf[pos] = rank_key(x[v], static_cast<uint32_t>(c));
      cnt += __popcll(m);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (cnt > kBuf) {
      fits = false;
      break;
    }
    if (cnt > kBuf / 2 && cnt > k) {
      uint64_t kk;
      best_keys(buf, cnt, k, &kk);
      cnt = k;
      const uint32_t tk = static_cast<uint32_t>(kk >> 32);
      t = tk > t ? tk : t;
    }
  }
  if (fits) return best_keys(buf, cnt, k, nullptr);
  KeyBatch kb;
  kb.pend = buf;
  kb.K1 = k;
  kb.list = 0;
  kb.cnt = 0;
  stream_chunks([=](int b) { return srow[b]; }, n, 0, 1, [&](uint64_t v, uint64_t th) { return kb.push(v, th); });
  kb.flush();
  return kb.list;
}

// One wave per index row of a chunk without chunk or piece maxima (few rows,
// e.g. decode): the K1 best of the row's candidate blocks by row_best_keys,
// then the local block.
constexpr int kRowWaves = 4;

__global__ __launch_bounds__(kRowWaves * kWave) void index_topk_rows_kernel(
    const float* __restrict__ M, int64_t ldm, msa_seqs sq, const int32_t* __restrict__ unit_off, int H_kv, int qr,
    int U, int rpu, int64_t u0, int64_t u1, int BK, int topk, int32_t* __restrict__ block_ids) {
  __shared__ uint64_t s_buf[kRowWaves][2 * kWave];
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x) / kWave;
  const int64_t task = static_cast<int64_t>(blockIdx.x) * kRowWaves + w;
  if (task >= (u1 - u0) * rpu) return;
  const RowTask t = locate_row(M, ldm, sq, unit_off, H_kv, qr, U, rpu, u0, task, BK, topk, block_ids);
  if (!t.ok) return;
  if (t.no_position) {
    if (lane < topk) t.out[lane] = -1;
    return;
  }
  const int K1 = topk - 1;
  // M rows are 16-byte aligned and hold a multiple of 4 floats
  const uint64_t list = K1 > 0 ? row_best_keys<true, 32>(t.mrow, t.nscan, K1, s_buf[w]) : 0ull;
  finish_row(list, K1, t.lb, topk, t.out);
}

// The Top-k operator on its own (msa_block_topk): the k best columns of each
// row of an fp32 score matrix, one wave per row, by row_best_keys with
// rounds of 16 values per lane for rows of at most 1024 columns, else 32.
template <bool VEC, int RP>
__global__ __launch_bounds__(kRowWaves * kWave) void row_topk_kernel(const float* __restrict__ scores,
                                                                     int64_t n_rows, int n_cols, int64_t ld, int k,
                                                                     int32_t* __restrict__ ids) {
  __shared__ uint64_t s_buf[kRowWaves][2 * kWave];
  const int lane = lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x) / kWave;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kRowWaves + w;
  if (row >= n_rows) return;
  const uint64_t list = row_best_keys<VEC, RP>(scores + row * ld, n_cols, k, s_buf[w]);
  const int nsel = __popcll(__ballot(lane < k && list != 0ull));
  uint32_t id = lane < nsel ? key_block(list) : 0xFFFFFFFFu;
  id = wave_sort_asc_u32(id);
  if (lane < k) ids[row * k + lane] = lane < nsel ? static_cast<int32_t>(id) : -1;
}

// ---------------------------------------------------------------- host side
struct IndexPlan {
  int qr;
  int U;                // row groups per unit
  bool narrow;          // U = 1 with at most 16 index rows per row group
  bool seq_units;       // U = 1 and no sequence longer than one row group
  int64_t max_units;    // upper bound of the units over all sequences
  int bcap;             // M row length (key blocks, multiple of 4)
  int cmcap;            // chunk maxima per row (64-block Top-k chunks; U = 4 only, else 0)
  int pcap;             // piece maxima per row (16-block pieces; with chunk maxima only)
  size_t hdr_bytes;
  size_t unit_bytes;    // M and chunk-maximum bytes per unit
};

int make_plan(const msa_seqs* seqs, int H_kv, int d_idx, int BK, int topk, IndexPlan* pl) {
  int st = msa_host::validate_seqs(seqs);
  if (st != MSA_OK) return st;
  if (H_kv < 1 || d_idx < 1 || BK < 1 || topk < 1) return MSA_ERR_INVALID;
  if (!msa_host::is_pow2(H_kv) || H_kv > 64) return MSA_ERR_UNSUPPORTED;
  if (d_idx != 64 && d_idx != 128) return MSA_ERR_UNSUPPORTED;
  if (BK != 64 && BK != 128) return MSA_ERR_UNSUPPORTED;
  if (topk > 64) return MSA_ERR_UNSUPPORTED;
  if ((st = msa_host::check_paged(seqs, BK, true)) != MSA_OK) return st;
  pl->qr = 64 / H_kv;
  // sequences longer than two row groups take the LDS-shared kernel: units of
  // 4 row groups (one per wave), or 8 (two per wave) for d_idx 64 and
  // sequences longer than four row groups
  const int64_t mq = seqs->max_q_rows;
  pl->U = mq > 4 * pl->qr && d_idx == 64 && BK == 64 ? 2 * kWaves : (mq > 2 * pl->qr ? kWaves : 1);
  pl->narrow = pl->U == 1 && std::min(pl->qr, seqs->max_q_rows) * H_kv <= 16;
  // at most one row group per sequence: unit s is sequence s, no unit table
  pl->seq_units = pl->U == 1 && seqs->max_q_rows <= pl->qr;
  const int64_t max_groups = seqs->total_q_rows / pl->qr + seqs->num_seqs;
  pl->max_units = pl->seq_units ? seqs->num_seqs : max_groups / pl->U + seqs->num_seqs;
  int nb = (seqs->max_kv_len + BK - 1) / BK;
  pl->bcap = static_cast<int>(msa_host::align_up(static_cast<size_t>(nb > 0 ? nb : 1), 4));
  pl->hdr_bytes = msa_host::align_up(sizeof(int32_t) * (seqs->num_seqs + 1), 256);
  pl->cmcap = pl->U >= kWaves ? (pl->bcap + kWave - 1) / kWave : 0;
  pl->pcap = pl->cmcap * kSlicePieces;
  pl->unit_bytes = static_cast<size_t>(pl->U) * kWave * (pl->bcap + pl->cmcap + pl->pcap) * sizeof(float);
  return MSA_OK;
}

constexpr size_t kDefaultScoreBytes = size_t(4) << 30;   // block-score staging per call
constexpr int64_t kSplitTopkRows = 4096;                 // fewer index rows: no chunk / piece maxima
// Few rows go one wave per row (index_topk_rows_kernel) when the rows are
// short (at most 4 rounds of 2048 blocks), numerous enough to spread and the
// Top-k small enough for the lane-maximum bound to keep a round's candidates
// within the wave's buffer; otherwise 16 waves share each row
// (index_topk_split_kernel).
constexpr int kRowTopkMaxK = 33;
constexpr int64_t kRowTopkMinRows = 64;
constexpr int kRowTopkMaxBlocks = 4 * 2048;

// 64-key sub-blocks in flight per wave of the narrow kernel: about 128 VGPRs of K_idx.
template <int D, int B>
constexpr int kNarrowDepth = D == 64 ? 4 : 2;

template <int D, int B, bool PAGED>
void launch_scores_as(const IndexPlan& pl, dim3 grid, hipStream_t stream, const uint16_t* iq, const uint16_t* ik,
                      const msa_seqs& sq, const int32_t* unit_off, int H_kv, int64_t u0, int64_t u1, float* M,
                      float* CM, int64_t cm_stride, float* PM) {
  if constexpr (D == 64 && B == 64) {
    if (pl.U == 2 * kWaves) {
      msa_prof::launch("index_block_max_lds_kernel", (index_block_max_lds_kernel<D, B, 128, PAGED>), grid, dim3(256),
                       0, stream, iq, ik, sq, unit_off, H_kv, pl.qr, u0, u1, M, static_cast<int64_t>(pl.bcap), CM,
                       cm_stride, PM);
      return;
    }
  }
  if (pl.U == kWaves)
    msa_prof::launch("index_block_max_lds_kernel", (index_block_max_lds_kernel<D, B, 64, PAGED>), grid, dim3(256), 0,
                     stream, iq, ik, sq, unit_off, H_kv, pl.qr, u0, u1, M, static_cast<int64_t>(pl.bcap), CM,
                     cm_stride, PM);
  else if (pl.narrow)
    msa_prof::launch("index_block_max_narrow_kernel", (index_block_max_narrow_kernel<D, B, kNarrowDepth<D, B>, PAGED>),
                     grid, dim3(256), 0, stream, iq, ik, sq, unit_off, H_kv, pl.qr, u0, u1, M,
                     static_cast<int64_t>(pl.bcap));
  else
    msa_prof::launch("index_block_max_wave_kernel", (index_block_max_wave_kernel<D, B, PAGED>), grid, dim3(256), 0,
                     stream, iq, ik, sq, unit_off, H_kv, pl.qr, u0, u1, M, static_cast<int64_t>(pl.bcap));
}

// A paged key side runs the kernels instantiated for it.
template <int D, int B>
void launch_scores(const IndexPlan& pl, dim3 grid, hipStream_t stream, const uint16_t* iq, const uint16_t* ik,
                   const msa_seqs& sq, const int32_t* unit_off, int H_kv, int64_t u0, int64_t u1, float* M,
                   float* CM, int64_t cm_stride, float* PM) {
  if (sq.block_table)
    launch_scores_as<D, B, true>(pl, grid, stream, iq, ik, sq, unit_off, H_kv, u0, u1, M, CM, cm_stride, PM);
  else
    launch_scores_as<D, B, false>(pl, grid, stream, iq, ik, sq, unit_off, H_kv, u0, u1, M, CM, cm_stride, PM);
}

}  // namespace

extern "C" size_t msa_index_topk_workspace_size(const msa_seqs* seqs, int num_kv_heads, int d_idx,
                                                int block_size, int topk) {
  IndexPlan pl;
  if (make_plan(seqs, num_kv_heads, d_idx, block_size, topk, &pl) != MSA_OK) return 0;
  int64_t units = static_cast<int64_t>(kDefaultScoreBytes / pl.unit_bytes);
  if (units < 1) units = 1;
  if (units > pl.max_units) units = pl.max_units;
  return pl.hdr_bytes + static_cast<size_t>(units) * pl.unit_bytes;
}

namespace {

// The call on a validated plan: block scores and Top-k per chunk of units, the
// chunk sized to the workspace.
int index_topk_run(const IndexPlan& pl, const void* index_q, const void* index_k, const msa_seqs* seqs,
                   int num_kv_heads, int d_idx, int block_size, int topk, int32_t* block_ids, void* workspace,
                   size_t workspace_bytes, hipStream_t stream) {
  int64_t chunk = static_cast<int64_t>((workspace_bytes - pl.hdr_bytes) / pl.unit_bytes);
  if (chunk > pl.max_units) chunk = pl.max_units;

  int32_t* unit_off = pl.seq_units ? nullptr : static_cast<int32_t*>(workspace);
  float* M = reinterpret_cast<float*>(static_cast<char*>(workspace) + pl.hdr_bytes);
  // chunk maxima CM[chunk][row] follow the chunk's score rows
  const int64_t cm_stride = chunk * pl.U * kWave;
  float* CM = pl.cmcap > 0 ? M + cm_stride * pl.bcap : nullptr;
  // piece maxima PM[slice][row][4] follow the chunk maxima
  float* PM = pl.cmcap > 0 ? CM + cm_stride * pl.cmcap : nullptr;
  const msa_seqs sq = *seqs;
  const uint16_t* iq = static_cast<const uint16_t*>(index_q);
  const uint16_t* ik = static_cast<const uint16_t*>(index_k);

  if (unit_off)
    msa_prof::launch("unit_offsets_kernel", unit_offsets_kernel, dim3(1), dim3(256), 0, stream, sq, pl.qr, pl.U,
                     unit_off);
  // per-wave kernel: slices of kSliceBlocks consecutive blocks, 4 per CTA
  const int nslice = (pl.bcap + kSliceBlocks - 1) / kSliceBlocks;
  const unsigned ny = static_cast<unsigned>((pl.bcap + kBlocksPerCta - 1) / kBlocksPerCta);
  for (int64_t u0 = 0; u0 < pl.max_units; u0 += chunk) {
    const int64_t u1 = u0 + chunk < pl.max_units ? u0 + chunk : pl.max_units;
    const dim3 grid = pl.U >= kWaves ? dim3(static_cast<unsigned>(u1 - u0), ny)
                                     : dim3(static_cast<unsigned>((nslice + kWaves - 1) / kWaves),
                                            static_cast<unsigned>(u1 - u0));
    if (d_idx == 64 && block_size == 64)
      launch_scores<64, 64>(pl, grid, stream, iq, ik, sq, unit_off, num_kv_heads, u0, u1, M, CM, cm_stride, PM);
    else if (d_idx == 64)
      launch_scores<64, 128>(pl, grid, stream, iq, ik, sq, unit_off, num_kv_heads, u0, u1, M, CM, cm_stride, PM);
    else if (block_size == 64)
      launch_scores<128, 64>(pl, grid, stream, iq, ik, sq, unit_off, num_kv_heads, u0, u1, M, CM, cm_stride, PM);
    else
      launch_scores<128, 128>(pl, grid, stream, iq, ik, sq, unit_off, num_kv_heads, u0, u1, M, CM, cm_stride, PM);
    // index rows a unit can hold: its query rows (<= U * qr, <= max_q_rows) x H_kv
    const int rpu = static_cast<int>(std::min<int64_t>(static_cast<int64_t>(pl.U) * pl.qr, seqs->max_q_rows)) *
                    num_kv_heads;
    const int64_t rows = (u1 - u0) * rpu;
    if (rows >= (int64_t(1) << 32)) return MSA_ERR_UNSUPPORTED;      // tasks are 32-bit in the kernels
    if (rows <= kSplitTopkRows && topk <= kRowTopkMaxK && rows >= kRowTopkMinRows && pl.bcap <= kRowTopkMaxBlocks)
      msa_prof::launch("index_topk_rows_kernel", index_topk_rows_kernel,
                       dim3(static_cast<unsigned>((rows + kRowWaves - 1) / kRowWaves)), dim3(kRowWaves * kWave), 0,
                       stream, M, static_cast<int64_t>(pl.bcap), sq, unit_off, num_kv_heads, pl.qr, pl.U, rpu, u0, u1,
                       block_size, topk, block_ids);
    else if (rows <= kSplitTopkRows)
      msa_prof::launch("index_topk_split_kernel", index_topk_split_kernel, dim3(static_cast<unsigned>(rows)),
                       dim3(64 * kSplitWaves), 0, stream, M, static_cast<int64_t>(pl.bcap), sq, unit_off,
                       num_kv_heads, pl.qr, pl.U, rpu, u0, u1, block_size, topk, block_ids);
    else
      msa_prof::launch("index_topk_kernel", index_topk_kernel, dim3(static_cast<unsigned>((rows + kWaves - 1) / kWaves)),
                       dim3(256), 0, stream, M, static_cast<int64_t>(pl.bcap), static_cast<const float*>(CM), cm_stride,
                       static_cast<const float*>(PM),
                       sq, unit_off, num_kv_heads, pl.qr, pl.U, rpu, u0, u1, block_size, topk, block_ids);
  }
  return msa_host::launch_status();
}

}  // namespace

extern "C" int msa_index_topk(const void* index_q, const void* index_k, const msa_seqs* seqs,
                              int num_kv_heads, int d_idx, int block_size, int topk,
                              int32_t* block_ids, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  IndexPlan pl;
  int st = make_plan(seqs, num_kv_heads, d_idx, block_size, topk, &pl);
  if (st != MSA_OK) return st;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if (!index_q || !index_k || !block_ids || !workspace) return MSA_ERR_INVALID;
  if (workspace_bytes < pl.hdr_bytes + pl.unit_bytes) return MSA_ERR_WORKSPACE;
  return index_topk_run(pl, index_q, index_k, seqs, num_kv_heads, d_idx, block_size, topk, block_ids, workspace,
                        workspace_bytes, stream);
}

// ---------------------------------------------------------------- row Top-k (host)
extern "C" int msa_block_topk(const float* scores, int64_t n_rows, int n_cols, int64_t ld, int k, int32_t* ids,
                              hipStream_t stream) {
  if (n_rows < 0 || n_cols < 0 || ld < n_cols || k < 1) return MSA_ERR_INVALID;
  if (k > kWave || n_cols > (1 << 30)) return MSA_ERR_UNSUPPORTED;
  if (n_rows == 0) return MSA_OK;
  if (!ids || (n_cols > 0 && !scores)) return MSA_ERR_INVALID;
  const int64_t grid = (n_rows + kRowWaves - 1) / kRowWaves;
  if (grid > 0x7FFFFFFF) return MSA_ERR_UNSUPPORTED;
  const bool vec = reinterpret_cast<uintptr_t>(scores) % 16 == 0 && ld % 4 == 0;
  auto launch_row_topk = [&](auto k16, auto k32) {
    const dim3 g(static_cast<unsigned>(grid)), b(kRowWaves * kWave);
    if (n_cols <= 16 * kWave)
      msa_prof::launch("row_topk_kernel", k16, g, b, 0, stream, scores, n_rows, n_cols, ld, k, ids);
    else
      msa_prof::launch("row_topk_kernel", k32, g, b, 0, stream, scores, n_rows, n_cols, ld, k, ids);
  };
  if (vec)
    launch_row_topk(row_topk_kernel<true, 16>, row_topk_kernel<true, 32>);
  else
    launch_row_topk(row_topk_kernel<false, 16>, row_topk_kernel<false, 32>);
  return msa_host::launch_status();
}

// ---------------------------------------------------------------- no-allocation entry point
// msa_index_topk_noalloc runs the same kernels on a workspace that lives in a
// device array of this file (one copy per GPU, held until the process ends),
// so the call allocates nothing.  Host code never passes the array's name to
// a kernel: it is a host-side stand-in for the symbol.  The device address is
// looked up once per device with hipGetSymbolAddress and cached.
static __device__ __align__(256) unsigned char scratch[MSA_INDEX_TOPK_NOALLOC_MAX_BYTES];

namespace {

constexpr size_t kNoallocScratchBytes = MSA_INDEX_TOPK_NOALLOC_MAX_BYTES;
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on the current device.
int scratch_on_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return MSA_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return MSA_ERR_UNSUPPORTED;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
        (void)hipGetLastError();
        return MSA_ERR_HIP;
      }
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return MSA_OK;
}

}  // namespace

extern "C" int msa_index_topk_noalloc(const void* index_q, const void* index_k, const msa_seqs* seqs,
                                      int num_kv_heads, int d_idx, int block_size, int topk,
                                      int32_t* block_ids, hipStream_t stream) {
  IndexPlan pl;
  int st = make_plan(seqs, num_kv_heads, d_idx, block_size, topk, &pl);
  if (st != MSA_OK) return st;
  if (seqs->total_q_rows == 0) return MSA_OK;
  if (!index_q || !index_k || !block_ids) return MSA_ERR_INVALID;
  // the smallest workspace the call can run in (one unit of rows) must fit
  if (pl.hdr_bytes + pl.unit_bytes > kNoallocScratchBytes) return MSA_ERR_WORKSPACE;
  void* ws = nullptr;
  if ((st = scratch_on_current_device(&ws)) != MSA_OK) return st;
  return index_topk_run(pl, index_q, index_k, seqs, num_kv_heads, d_idx, block_size, topk, block_ids, ws,
                        kNoallocScratchBytes, stream);
}

