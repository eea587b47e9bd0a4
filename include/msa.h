/*
 * msa.h -- C ABI of libmsa.so, the MI355X (gfx950) inference hot path of
 * MiniMax Sparse Attention (MSA).
 *
 * The paper factors sparse attention into an indexer that picks which keys a
 * query attends to and an exact attention over the picked keys (Sec. 2.2,
 * two-stage equation).  MSA's indexer is block- and GQA-group-granular
 * (Sec. 2.3; Sec. 3.1 "Index Branch"); its attention runs only over the
 * selected blocks (Sec. 3.1 "Main Branch").  The library exports one call per
 * stage and per inference phase:
 *
 *   msa_index_topk           Index Branch: block scores + Top-k (prefill and decode)
 *   msa_block_topk           the Top-k operator alone, on a score matrix the caller holds
 *   msa_sparse_attn_prefill  Main Branch for many query rows per sequence
 *   msa_sparse_attn_decode   Main Branch for one query row per sequence
 *   msa_sparse_attn_*_fp8    Main Branch on e4m3 queries and KV cache
 *   msa_dense_attn           dense causal GQA attention (the comparison baseline)
 *   msa_sparse_attn_backward training: Main Branch gradients dQ, dK, dV
 *   msa_sparse_kl_backward   training: sparse KL loss and its index-projection gradients
 *
 * Conventions shared by every call
 * --------------------------------
 * - Every tensor argument is a DEVICE pointer to contiguous row-major memory
 *   that the caller allocates, owns and keeps alive until the stream has
 *   executed the call.  bf16 tensors hold IEEE bfloat16 bit patterns.
 * - Calls are asynchronous on `stream` (0 = the null stream): they validate
 *   their arguments on the host, launch kernels and return.  Results are
 *   valid once the stream has reached them.  Nothing is launched when a call
 *   returns an error.  No call synchronises the host with the device.
 * - No call allocates device memory.  Calls that need scratch space take a
 *   caller-provided `workspace` of at least the size returned by the matching
 *   *_workspace_size() query; the workspace is free again once the stream has
 *   executed the call.  Calls that share a workspace must be ordered on one
 *   stream.  (msa_index_topk_noalloc uses the library's static device array
 *   instead, see below.)
 * - Global state: the opt-in kernel timing at the end of this header, the
 *   grid size of each persistent kernel (derived from the device's occupancy
 *   on first use and cached in an atomic), and msa_index_topk_noalloc's
 *   file-scope device scratch array with its per-device address table.
 *   Concurrent calls from several host threads are safe when they use
 *   distinct outputs and workspaces (msa_index_topk_noalloc calls on one GPU
 *   share its scratch array and must not overlap).
 * - NaN or Inf inputs give unspecified (but memory-safe) results.
 *
 * Sequence layout (struct msa_seqs)
 * ---------------------------------
 * A batch holds `num_seqs` sequences.  Sequence s owns the packed query rows
 * q_offsets[s] .. q_offsets[s+1]-1 of the query-side tensors (index_q, q, o,
 * lse, block_ids) and key rows kv_starts[s] .. kv_starts[s]+kv_lens[s]-1 of
 * the key-side tensors (index_k, k, v).  Query row t of sequence s (t counted
 * from 0 inside the sequence) sits at absolute position
 *     p = kv_lens[s] - (q_offsets[s+1] - q_offsets[s]) + t,
 * i.e. its own key is already in the cache.  This covers prefill
 * (q rows == kv_len), chunked prefill (rows appended to a cached context) and
 * decode (one row per sequence; kv_starts may then point into a padded cache,
 * e.g. s * max_len).  Key block b of a sequence holds its keys
 * b*block_size .. min((b+1)*block_size, kv_len)-1 (Sec. 2.3, block equation);
 * the local block of position p is p / block_size.  Rows of several tokens per
 * sequence after a cached context (speculative / multi-token decode) are the
 * chunked-prefill case with a few rows.
 *
 * Paged key side (optional): with block_table != NULL the key-side tensors
 * (index_k, k, v) are a pool of pages of page_size rows; key j of sequence s
 * is row page * page_size + j % page_size with
 * page = block_table[s * block_table_stride + j / page_size] (kv_starts is
 * then ignored and may be NULL).  page_size must be block_size times 1, 2, 4,
 * ... or 64 for the call's block_size; kv_lens[s] <= block_table_stride *
 * page_size.  Page ids outside [0, total_kv_rows /
 * page_size) are clamped into it (results unspecified, memory safe).  This
 * is a serving layout, not part of the paper.  Every call accepts it except
 * msa_dense_attn, which returns MSA_ERR_UNSUPPORTED for a paged layout; the
 * training calls then write dK, dV and d index_k in the pool's rows (rows of
 * pages no sequence lists get zero; keys in pages shared by several
 * sequences get the sum of their gradients).
 */
#ifndef MSA_H_
#define MSA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every int-valued call. */
#define MSA_OK 0
#define MSA_ERR_INVALID (-1)     /* null pointer, negative or inconsistent size, H_q % H_kv != 0 ... */
#define MSA_ERR_UNSUPPORTED (-2) /* a valid shape the library has no kernel for */
#define MSA_ERR_WORKSPACE (-3)   /* workspace smaller than the *_workspace_size() value */
#define MSA_ERR_HIP (-4)         /* a HIP launch failed (the HIP error is consumed) */

typedef struct msa_seqs {
  int32_t num_seqs;          /* host: number of sequences, >= 1 */
  int64_t total_q_rows;      /* host: rows of the query-side tensors (= q_offsets[num_seqs]) */
  int64_t total_kv_rows;     /* host: rows of the key-side tensors; every key access is
                                kept below this bound */
  int32_t max_q_rows;        /* host: upper bound of q_offsets[s+1]-q_offsets[s] */
  int32_t max_kv_len;        /* host: upper bound of kv_lens[s] */
  const int32_t* q_offsets;  /* device [num_seqs+1], non-decreasing, q_offsets[0] == 0 */
  const int64_t* kv_starts;  /* device [num_seqs], >= 0 (unused when paged) */
  const int32_t* kv_lens;    /* device [num_seqs], >= the sequence's query rows */
  const int32_t* block_table;   /* device [num_seqs, block_table_stride] page ids, or NULL
                                   (contiguous key side) */
  int32_t block_table_stride;   /* host: entries (pages) per sequence of block_table */
  int32_t page_size;            /* host: key rows per page (block_size x 2^j, j <= 6) */
} msa_seqs;

/* Human-readable text of a status code (static storage). */
const char* msa_strerror(int status);

/* ------------------------------------------------------------------------
 * Index Branch: msa_index_topk
 *
 * Sec. 3.1, index-score equation: for query position i of group r and key j,
 * S_ij = q_idx[i, r, :] . k_idx[j, :] / sqrt(d_idx); a key block scores the
 * maximum of S over its causally visible tokens (j <= i).  Sec. 3.1, top-k
 * equation and Sec. 3.2 "Local Block": each (query row, group) keeps the
 * local block i / block_size plus the top-k-1 other causal blocks.  Selection
 * ranks the raw dot products (Sec. 4.1 "Exp-free selection": neither the
 * softmax nor the positive scale changes the order); equal scores keep the
 * lower block id.
 *
 *   index_q   bf16 [total_q_rows, num_kv_heads, d_idx]   one index-query head per group
 *   index_k   bf16 [total_kv_rows, d_idx]                the single shared index-key head
 *   block_ids int32 [total_q_rows, num_kv_heads, topk]   OUTPUT: the min(topk, lb+1) selected
 *             block ids of each (row, group) in ascending order, then -1 padding.
 *
 * Supported: d_idx in {64, 128}; block_size in {64, 128}; 1 <= topk <= 64;
 * num_kv_heads a power of two <= 64.
 * ------------------------------------------------------------------------ */
size_t msa_index_topk_workspace_size(const msa_seqs* seqs, int num_kv_heads, int d_idx,
                                     int block_size, int topk);
int msa_index_topk(const void* index_q, const void* index_k, const msa_seqs* seqs,
                   int num_kv_heads, int d_idx, int block_size, int topk, int32_t* block_ids,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * msa_index_topk_noalloc -- msa_index_topk without a workspace argument, for
 * callers that cannot allocate device memory: code under HIP graph capture,
 * serving loops that must not call hipMalloc, harnesses that forbid it.
 *
 * Arguments, outputs (block_ids, caller-allocated), results and errors are
 * those of msa_index_topk.  The scratch space lives in a device array of the
 * library of MSA_INDEX_TOPK_NOALLOC_MAX_BYTES bytes; each GPU the call runs on
 * holds its own copy until the process ends.  The call runs on the current
 * device, and `stream` must belong to it.  It allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); its first call on a device looks
 * the array's address up once.  A problem whose smallest workspace (the
 * sequence table plus one unit of rows, the quantum msa_index_topk chunks by)
 * exceeds the array returns MSA_ERR_WORKSPACE and launches nothing; problems
 * larger than the array but within that bound run in several chunks.
 * Every call on a GPU shares that GPU's array: calls that overlap on one GPU
 * (several streams or host threads) race and must be serialised by the
 * caller.  Nothing in the array needs to start at zero.
 * ------------------------------------------------------------------------ */
#define MSA_INDEX_TOPK_NOALLOC_MAX_BYTES ((size_t)64 << 20)
int msa_index_topk_noalloc(const void* index_q, const void* index_k, const msa_seqs* seqs,
                           int num_kv_heads, int d_idx, int block_size, int topk,
                           int32_t* block_ids, hipStream_t stream);

/* ------------------------------------------------------------------------
 * msa_block_topk -- the Top-k operator of the Index Branch on its own, for a
 * score matrix the caller already holds (Sec. 3.1 top-k equation; Sec. 4.1
 * "Per-thread register top-k" and its latency table, which times this
 * operator on fp32 inputs of shape (N, B) with rows processed independently).
 *
 *   scores  fp32 [n_rows, ld]: columns 0 .. n_cols-1 of each row are ranked;
 *           the buffer spans n_rows * ld floats.
 *   ids     int32 [n_rows, k]  OUTPUT: the min(k, n_cols) columns of largest
 *           score of each row in ascending order, then -1 padding.  Equal
 *           scores keep the lower column; -0 equals +0; -inf ranks below
 *           every finite score like any other value.
 *
 * No block is forced and no causal limit applies (msa_index_topk adds both).
 * Supported: 1 <= k <= 64; 0 <= n_cols <= 2^30; ld >= n_cols.  NaN
 * scores give unspecified (memory-safe) ids.  No workspace.  Rows that are
 * 16-byte aligned (scores aligned, ld % 4 == 0) are read four columns per
 * lane and load; others one column per lane.
 * ------------------------------------------------------------------------ */
int msa_block_topk(const float* scores, int64_t n_rows, int n_cols, int64_t ld, int k,
                   int32_t* ids, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Main Branch: msa_sparse_attn_prefill / msa_sparse_attn_decode
 *
 * Sec. 3.1, sparse-attention equation: for query row i and query head h of
 * group r = h / (num_q_heads / num_kv_heads), softmax attention with scale
 * `softmax_scale` (the paper uses 1/sqrt(head_dim)) over the causally visible
 * tokens (j <= i) of the blocks listed in block_ids[i, r, :], using key/value
 * head r.  Entries < 0 are padding; the ids of a row must be distinct; ids
 * past the local block select no token.  Every row must list a block with a
 * visible token (its local block, as msa_index_topk guarantees); a row without
 * one gets O = 0 and LSE = -inf.
 *
 *   q          bf16 [total_q_rows, num_q_heads, head_dim]
 *   k, v       bf16 [total_kv_rows, num_kv_heads, head_dim]
 *   block_ids  int32 [total_q_rows, num_kv_heads, topk]   (msa_index_topk's output)
 *   o          bf16 [total_q_rows, num_q_heads, head_dim]  OUTPUT
 *   lse        fp32 [total_q_rows, num_q_heads]            OUTPUT, natural log of the
 *              softmax denominator including the scale (Sec. 4.2 combine)
 *
 * The prefill call is built for many query rows per sequence; the decode call
 * for one query row per sequence (it accepts any layout, and gives the same
 * result as the prefill call up to rounding).
 *
 * Supported: head_dim == 128; block_size in {64, 128}; 1 <= topk <= 64;
 * 1 <= num_q_heads / num_kv_heads <= 16; num_kv_heads <= 64.
 * ------------------------------------------------------------------------ */
size_t msa_sparse_attn_prefill_workspace_size(const msa_seqs* seqs, int num_q_heads,
                                              int num_kv_heads, int head_dim, int block_size,
                                              int topk);
int msa_sparse_attn_prefill(const void* q, const void* k, const void* v,
                            const int32_t* block_ids, const msa_seqs* seqs, int num_q_heads,
                            int num_kv_heads, int head_dim, int block_size, int topk,
                            float softmax_scale, void* o, float* lse, void* workspace,
                            size_t workspace_bytes, hipStream_t stream);

size_t msa_sparse_attn_decode_workspace_size(const msa_seqs* seqs, int num_q_heads,
                                             int num_kv_heads, int head_dim, int block_size,
                                             int topk);
int msa_sparse_attn_decode(const void* q, const void* k, const void* v,
                           const int32_t* block_ids, const msa_seqs* seqs, int num_q_heads,
                           int num_kv_heads, int head_dim, int block_size, int topk,
                           float softmax_scale, void* o, float* lse, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * msa_sparse_attn_prefill_fp8 / msa_sparse_attn_decode_fp8 -- the Main Branch
 * on 8-bit queries and KV cache.
 *
 * Sec. 4.2 notes that the kernels also take fp8 inputs, which rescales the IO
 * volume of the Main Branch.  q, k and v hold OCP 8-bit floating point E4M3
 * ("e4m3fn": sign, 4 exponent bits with bias 7, 3 mantissa bits; no
 * infinities; S.1111.111 is NaN) codes, one byte per element, in the layouts
 * of the bf16 calls.  Element values are code * q_scale, code * k_scale and
 * code * v_scale (per-tensor fp32 scales, finite and > 0).  The result is the
 * attention of those values: logits use softmax_scale * q_scale * k_scale and
 * O is scaled by v_scale.  Block ids, the bf16 O and fp32 LSE outputs, the
 * workspace (the *_workspace_size queries of the bf16 calls apply), stream and
 * error behaviour are those of msa_sparse_attn_prefill / _decode; a scale that
 * is not finite and positive returns MSA_ERR_INVALID.  The kernels widen e4m3
 * to bf16 exactly on load and compute as the bf16 calls do.
 * ------------------------------------------------------------------------ */
int msa_sparse_attn_prefill_fp8(const void* q, const void* k, const void* v, float q_scale,
                                float k_scale, float v_scale, const int32_t* block_ids,
                                const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                int head_dim, int block_size, int topk, float softmax_scale,
                                void* o, float* lse, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);
int msa_sparse_attn_decode_fp8(const void* q, const void* k, const void* v, float q_scale,
                               float k_scale, float v_scale, const int32_t* block_ids,
                               const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                               int head_dim, int block_size, int topk, float softmax_scale,
                               void* o, float* lse, void* workspace, size_t workspace_bytes,
                               hipStream_t stream);

/* ------------------------------------------------------------------------
 * msa_dense_attn -- dense causal GQA attention, the baseline MSA is measured
 * against (no block selection).
 *
 * Every query row attends to all keys of its sequence at positions <= p: the
 * softmax attention that the sparse-attention equation of Sec. 3.1 becomes
 * when the selected set covers every causal block (Sec. 2.2, full attention
 * with GQA sharing of K and V across the G query heads of a group).
 *
 * Arguments, layouts, ownership, outputs and errors are those of
 * msa_sparse_attn_prefill without block ids: q [total_q_rows, H_q, 128],
 * k and v [total_kv_rows, H_kv, 128] (bf16), o [total_q_rows, H_q, 128] bf16,
 * lse [total_q_rows, H_q] fp32 natural log (-inf for rows with no visible
 * key).  Sequences with at most 4 query rows (decode) run a split row kernel
 * whose partials need the workspace; longer ones run a FlashAttention-style
 * tiled kernel that needs only a small table.
 *
 * Supported: head_dim == 128; 1 <= num_q_heads / num_kv_heads <= 16;
 * num_kv_heads <= 64.
 * ------------------------------------------------------------------------ */
size_t msa_dense_attn_workspace_size(const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                                     int head_dim);
int msa_dense_attn(const void* q, const void* k, const void* v, const msa_seqs* seqs,
                   int num_q_heads, int num_kv_heads, int head_dim, float softmax_scale, void* o,
                   float* lse, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * msa_sparse_attn_backward -- training backward of the Main Branch.
 *
 * Alg. 1 trains through the sparse attention of Sec. 3.1.  For an upstream
 * gradient dO of the output O, with P_ij = exp(softmax_scale q_i.k_j - LSE_i)
 * over the tokens row i attended and D_i = dO_i . O_i:
 *   dV_j = sum_i P_ij dO_i,  dS_ij = P_ij (dO_i . v_j - D_i),
 *   dQ_i = softmax_scale sum_j dS_ij k_j,  dK_j = softmax_scale sum_i dS_ij q_i,
 * each sum running over the (row, head, token) triples of the forward.
 *
 *   q, k, v, block_ids, seqs, heads, block_size, topk, softmax_scale: exactly
 *              as passed to the forward call (msa_sparse_attn_prefill/_decode)
 *   o          bf16 [total_q_rows, num_q_heads, head_dim]   the forward's O
 *   lse        fp32 [total_q_rows, num_q_heads]             the forward's LSE
 *   d_o        bf16 [total_q_rows, num_q_heads, head_dim]   upstream gradient
 *   d_q        bf16 [total_q_rows, num_q_heads, head_dim]   OUTPUT
 *   d_k, d_v   bf16 [total_kv_rows, num_kv_heads, head_dim] OUTPUT; every row is
 *              written, key rows no query attended get 0
 *
 * Work runs key-block-outer with fp32 accumulation.  Every output is
 * bit-reproducible: d_q adds its partials in slot order, and d_k and d_v add a
 * key block's contributions in ascending (query row, slot) order (the
 * reverse index is sorted into that order).  Workspace, stream and
 * error behaviour as for msa_sparse_attn_prefill.  Supported: head_dim == 128;
 * block_size 64 or 128 with 1 <= topk <= 64; 1 <= num_q_heads / num_kv_heads
 * <= 16; num_kv_heads <= 64.
 * ------------------------------------------------------------------------ */
size_t msa_sparse_attn_backward_workspace_size(const msa_seqs* seqs, int num_q_heads,
                                               int num_kv_heads, int head_dim, int block_size,
                                               int topk);
int msa_sparse_attn_backward(const void* q, const void* k, const void* v, const void* o,
                             const float* lse, const void* d_o, const int32_t* block_ids,
                             const msa_seqs* seqs, int num_q_heads, int num_kv_heads,
                             int head_dim, int block_size, int topk, float softmax_scale,
                             void* d_q, void* d_k, void* d_v, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * msa_sparse_kl_backward -- the sparse KL loss that trains the Index Branch.
 *
 * Sec. 3.2 ("KL Loss"), per query row i and group r, over the causally
 * visible tokens T of the selected blocks: the student
 * P_idx_j = softmax_j(q_idx[i,r] . k_idx[j] / sqrt(d_idx)) and the detached
 * teacher P_j = (1/G) sum over the group's query heads h of
 * exp(softmax_scale q[i,h] . k[j,r] - lse[i,h]) (Alg. 1: the Main Branch
 * attention over the same tokens; lse is the forward's LSE, Sec. 4.3 "LSE
 * fusion").  Outputs, with Delta_j = P_idx_j - P_j:
 *   kl[i, r]        = sum_j P_j (ln P_j - ln P_idx_j)          (optional)
 *   d_index_q[i, r] = grad_scale / sqrt(d_idx) sum_j Delta_j k_idx[j]
 *   d_index_k[j]    = grad_scale / sqrt(d_idx) sum_{i,r} Delta_ij q_idx[i, r]
 * i.e. grad_scale times the gradients of sum_{i,r} kl[i, r]; the paper's
 * per-layer loss is the mean over rows and groups, so a training loop passes
 * grad_scale = lambda / (total_q_rows * num_kv_heads).  Nothing flows into q
 * or k (the gradient detach of Sec. 3.2).
 *
 *   index_q    bf16 [total_q_rows, num_kv_heads, d_idx]
 *   index_k    bf16 [total_kv_rows, d_idx]
 *   q, k       bf16 as for msa_sparse_attn_prefill; lse fp32 [total_q_rows, num_q_heads]
 *   block_ids  int32 [total_q_rows, num_kv_heads, topk]   the selection the forward used
 *   d_index_q  bf16 [total_q_rows, num_kv_heads, d_idx]   OUTPUT
 *   d_index_k  bf16 [total_kv_rows, d_idx]                OUTPUT; every row written
 *   kl         fp32 [total_q_rows, num_kv_heads]          OUTPUT, or NULL to skip
 *
 * Workspace, stream and error behaviour as for msa_sparse_attn_prefill.
 * d_index_q, d_index_k and kl are bit-reproducible (d_index_k adds a key
 * block's queries in ascending (row, slot) order).  Supported: d_idx in {64, 128};
 * head_dim == 128; block_size 64 or 128 with 1 <= topk <= 64;
 * num_q_heads / num_kv_heads in {1, 2, 4, 8, 16}; num_kv_heads <= 64.
 * ------------------------------------------------------------------------ */
size_t msa_sparse_kl_backward_workspace_size(const msa_seqs* seqs, int num_q_heads,
                                             int num_kv_heads, int d_idx, int head_dim,
                                             int block_size, int topk);
int msa_sparse_kl_backward(const void* index_q, const void* index_k, const void* q, const void* k,
                           const float* lse, const int32_t* block_ids, const msa_seqs* seqs,
                           int num_q_heads, int num_kv_heads, int d_idx, int head_dim,
                           int block_size, int topk, float softmax_scale, float grad_scale,
                           void* d_index_q, void* d_index_k, float* kl, void* workspace,
                           size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kernel timing (a measurement aid; no part of the attention path)
 *
 * While enabled, every kernel a call launches is bracketed by a pair of HIP
 * events recorded on the call's stream, filed under the kernel's name (e.g.
 * "kvo_attn_kernel", "index_block_max_lds_kernel").  The events are created
 * on first use and kept for reuse (global state of the timer alone).
 *
 *   msa_profile_enable(on)   on != 0 starts recording for later calls, 0 stops.
 *   msa_profile_reset()      forgets the launches recorded so far.
 *   msa_profile_kernel_name(i)  name of the i-th kernel seen since load, or
 *                            NULL past the last one; the string stays valid
 *                            until the library is unloaded.
 *   msa_profile_read(name, &launches, &total_ms)  launches of `name` since the
 *                            last reset and their summed event-to-event time;
 *                            waits for those events; unknown names read 0.
 *
 * Timing adds two event records per launch, so enable it only for runs that
 * read it.  Calls on several host threads must not interleave with reset or
 * read.  Errors: MSA_ERR_INVALID for null output pointers, MSA_ERR_HIP when
 * an event cannot be read.
 * ------------------------------------------------------------------------ */
int msa_profile_enable(int on);
int msa_profile_reset(void);
const char* msa_profile_kernel_name(int i);
int msa_profile_read(const char* kernel, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* MSA_H_ */
