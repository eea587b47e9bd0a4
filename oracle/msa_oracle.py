"""CPU oracle of the MiniMax Sparse Attention (MSA) inference hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the package entry's ``smoke()``
check and the benchmark's CPU-baseline leg may import or run this module.  It
shares no code with the HIP path (no kernels, helpers, tables or constants)
and imports nothing from the library package; the inputs it receives are bf16
bit patterns (numpy ``uint16``) or 8-bit E4M3 codes (numpy ``uint8``, Main
Branch only) that it decodes itself.

What it computes, in the paper's order and notation:

* Index Branch (Sec. 3.1, index-projection / index-score / top-k equations):
  token index scores S = q_idx . k_idx / sqrt(d_idx) over the visible tokens
  j <= i, causal block max-pooling M_b = max_{j in B_b, j <= i} S_j (blocks
  with no visible token score -inf), and Top-k block selection with the local
  block always included (Sec. 3.1 last paragraph of "Index Branch"; Sec. 3.2
  "Local Block"; Appendix C.2 final recipe: only the incomplete self block is
  forced, no sink); and the Top-k operator alone on a given score matrix
  (Sec. 4.1 latency table).
* Main Branch (Sec. 3.1, sparse-attention equation): exact softmax attention of
  each query head of group r over the causally visible tokens of the selected
  blocks, using key/value head r; also the natural-log log-sum-exp.
* Split combine (Sec. 4.2 "Two-phase forward"): merge of locally normalised
  partials through their log-sum-exps.
* Dense causal attention (Sec. 2.1, softmax-attention equation) and the FLOP
  model of Sec. 3.3.
* Training backward (Sec. 3.2 "KL Loss" and "Gradient Detach"; Alg. 1):
  gradients of the Main Branch output with respect to Q, K and V for a given
  upstream dO, and the sparse KL loss KL(sg(P) || P_idx) per (query, group)
  with its gradients with respect to the index query and index key.

Precision: float64 everywhere, with one deliberate exception.  Block
selection is an integer decision taken from floating point; it is taken on
each index dot product rounded once to float32 (the precision in which the GPU
kernels take it), before the positive 1/sqrt(d_idx) scale, which cannot change
the order (Sec. 4.1 "Exp-free selection": order-preserving maps leave Top-k
unchanged).  Score gaps used by the tie rule are reported in float64 on the
scaled scores S.

Readings of passages the paper leaves open (all used below):

 R1  Local block + Top-k: the local block lb = floor(p / B_k) takes one of the k
     slots and the other k-1 slots go to the best other causal blocks
     (Sec. 3.2 "Local Block": one slot is reserved, the remaining slots are
     chosen by the Index Branch; Sec. 3.1: budget at most k*B_k tokens).
 R2  Fewer causal blocks than k: all of them are selected; the row's id list is
     padded with -1 (blocks without a visible token score -inf, Sec. 3.1).
 R3  Ties: higher score first, then the lower block id.  Ids are returned in
     ascending order (Sec. 4.1 reports unsorted outputs and identical index
     sets across implementations; the order of the output is a convention).
 R4  Score gap g of a row: scaled score of the last selected non-local block
     minus that of the best unselected candidate; +inf when every candidate
     is selected.
 R5  No sink block is forced (Appendix C.2).
 R6  Softmax scale 1/sqrt(d_h); log-sum-exp uses the natural log (Sec. 4.2
     combine uses log/exp).
 R7  A partial last block holds min(b*B_k, N) - (b-1)*B_k tokens (Sec. 2.3).
 R8  Position convention: query row t of a sequence with kv_len keys and
     q_rows query rows sits at absolute position kv_len - q_rows + t; its own
     key is already in the cache (decode: p = kv_len - 1; chunked prefill is
     right-aligned).  The paper does not discuss decode or chunked prefill.
 R9  Index scores take the projected q_idx / k_idx as given (no RoPE on the
     Index Branch is described).
 R10 KL loss: the teacher P averages the heads' softmax distributions over
     the same selected-token set the Main Branch attends (its normaliser is
     the forward's LSE); the loss is the mean over rows and groups of the
     per-(row, group) KL, so the gradients returned here are those of the sum
     and a caller scales them by lambda / (N H_kv).  Detach (Sec. 3.2): no
     gradient reaches Q, K or the teacher.
 R11 A key row that no query selects gets a zero gradient; so does a (row,
     group) without visible tokens.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# representation
# --------------------------------------------------------------------------
def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64 values (exact)."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def decode_fp8_e4m3(codes: np.ndarray) -> np.ndarray:
    """OCP 8-bit floating point E4M3 codes (uint8) -> float64 values (exact).

    Bit 7 is the sign, bits 6..3 the exponent E (bias 7), bits 2..0 the
    mantissa M: E > 0 gives (-1)^s 2^(E-7) (1 + M/8), E = 0 the subnormals
    (-1)^s 2^-6 (M/8); the format has no infinities and E = 15, M = 7 is NaN.
    (Sec. 4.2 notes that the kernels also take fp8 inputs.)"""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    v = np.where(e > 0, np.ldexp(1.0 + m / 8.0, e - 7), np.ldexp(m / 8.0, -6))
    v = np.where((e == 15) & ((c & 0x7) == 7), np.nan, v)
    return sign * v


def _decoder(fmt: str):
    if fmt == "bf16":
        return decode_bf16
    if fmt == "e4m3":
        return decode_fp8_e4m3
    raise ValueError(f"unknown input format {fmt}")


class Layout:
    """Sequence layout: query rows of sequence s are q_offsets[s]..q_offsets[s+1];
    its keys are rows kv_starts[s] .. kv_starts[s]+kv_lens[s] of the key side."""

    def __init__(self, q_rows: Sequence[int], kv_lens: Sequence[int], kv_starts: Sequence[int]):
        self.q_rows = [int(x) for x in q_rows]
        self.kv_lens = [int(x) for x in kv_lens]
        self.kv_starts = [int(x) for x in kv_starts]
        self.q_offsets = [0]
        for r in self.q_rows:
            self.q_offsets.append(self.q_offsets[-1] + r)

    @property
    def total_q_rows(self) -> int:
        return self.q_offsets[-1]

    def locate(self, row: int) -> Tuple[int, int]:
        """(sequence, absolute position) of packed query row ``row`` (R8)."""
        s = int(np.searchsorted(self.q_offsets, row, side="right")) - 1
        t = row - self.q_offsets[s]
        return s, self.kv_lens[s] - self.q_rows[s] + t


def layout_of(problem) -> Layout:
    return Layout(problem.q_rows, problem.kv_lens, problem.kv_starts)


# --------------------------------------------------------------------------
# Index Branch (Sec. 3.1)
# --------------------------------------------------------------------------
def block_maxima(dots_row: np.ndarray, pos: int, block_size: int) -> np.ndarray:
    """Causal block max-pool of one (row, group): M_b over blocks
    b = 0 .. ceil(n / B_k) - 1 of the visible prefix j <= pos; blocks whose
    tokens are all in the future are -inf (Sec. 3.1, index-score equation)."""
    n = dots_row.shape[0]
    nblk = (n + block_size - 1) // block_size
    out = np.full(nblk, -np.inf, dtype=dots_row.dtype)
    vis = dots_row[:pos + 1]
    full = (pos + 1) // block_size
    if full:
        out[:full] = vis[:full * block_size].reshape(full, block_size).max(axis=1)
    if (pos + 1) % block_size:
        out[full] = vis[full * block_size:].max()
    return out


def select_row(m_rank: np.ndarray, m_scaled: np.ndarray, pos: int, block_size: int,
               topk: int) -> Tuple[np.ndarray, float]:
    """Top-k with the local block forced (R1-R5) for one (row, group).

    m_rank: block maxima used for ranking (float32-rounded unscaled dots),
    m_scaled: the same maxima in float64 on the scaled score S (for the gap).
    Returns (ids ascending, padded with -1 to ``topk``; gap g)."""
    lb = pos // block_size
    others = topk - 1                          # one slot is the local block's (R1)
    ids = np.full(topk, -1, dtype=np.int32)
    gap = math.inf
    chosen = np.zeros(0, dtype=np.int64)
    if lb > 0 and others > 0:
        cand = np.arange(lb)                   # every other causal block is fully visible
        # rank: higher score first, then the lower block id (R3)
        order = np.lexsort((cand, -m_rank[:lb].astype(np.float64)))
        chosen = cand[order[:others]]
        if lb > others:
            gap = float(m_scaled[order[others - 1]] - m_scaled[order[others]])
    sel = np.sort(np.concatenate([chosen, [lb]]).astype(np.int64))
    ids[:sel.shape[0]] = sel
    return ids, gap


def select_blocks(index_q_bits: np.ndarray, index_k_bits: np.ndarray, layout: Layout,
                  block_size: int, topk: int, rows: Optional[Iterable[int]] = None,
                  batch_rows: int = 256) -> Tuple[np.ndarray, np.ndarray]:
    """Index Branch for the given packed query rows (all rows by default).

    index_q_bits: (Tq, H_kv, d_idx) uint16; index_k_bits: (Tk, d_idx) uint16.
    Returns block_ids (R, H_kv, topk) int32 and gaps (R, H_kv) float64."""
    Tq, H_kv, d_idx = index_q_bits.shape
    rows = list(range(Tq)) if rows is None else [int(r) for r in rows]
    inv_sqrt = 1.0 / math.sqrt(d_idx)
    ids = np.full((len(rows), H_kv, topk), -1, dtype=np.int32)
    gaps = np.full((len(rows), H_kv), math.inf)
    # group the requested rows by sequence so each batch shares its keys, in
    # order of position so a batch's rows need keys up to similar depths
    by_seq = {}
    for i, r in enumerate(rows):
        s, pos = layout.locate(r)
        by_seq.setdefault(s, []).append((i, r, pos))
    for s, items in by_seq.items():
        items.sort(key=lambda it: it[2])
        kv0, kvl = layout.kv_starts[s], layout.kv_lens[s]
        b0 = 0
        while b0 < len(items):
            # at most ~2 GiB of float64 dot products per batch
            n_keys = min(kvl, items[min(len(items), b0 + batch_rows) - 1][2] + 1)
            nb = max(1, min(batch_rows, (1 << 31) // max(1, 8 * H_kv * n_keys)))
            batch = items[b0:b0 + nb]
            b0 += nb
            pmax = max(pos for _, _, pos in batch)
            ik = decode_bf16(index_k_bits[kv0:kv0 + min(kvl, pmax + 1)])
            iq = decode_bf16(index_q_bits[[r for _, r, _ in batch]])      # (B, H_kv, d)
            # float64 dot products of every (row, group) with every key
            dots = (iq.reshape(-1, d_idx) @ ik.T).reshape(len(batch), H_kv, -1)
            dots32 = dots.astype(np.float32)
            for j, (i, r, pos) in enumerate(batch):
                for g in range(H_kv):
                    m_rank = block_maxima(dots32[j, g], pos, block_size)
                    m_scaled = block_maxima(dots[j, g], pos, block_size) * inv_sqrt
                    ids[i, g], gaps[i, g] = select_row(m_rank, m_scaled, pos, block_size, topk)
    return ids, gaps


def row_block_scores(index_q_bits, index_k_bits, layout: Layout, row: int, group: int,
                     block_size: int) -> np.ndarray:
    """Scaled float64 block maxima M_b (Sec. 3.1) of one (row, group); used by
    the tie rule to judge a selection that differs from the oracle's."""
    s, pos = layout.locate(row)
    kv0 = layout.kv_starts[s]
    ik = decode_bf16(index_k_bits[kv0:kv0 + pos + 1])
    iq = decode_bf16(index_q_bits[row, group])
    d = ik @ iq
    return block_maxima(d, pos, block_size) / math.sqrt(iq.shape[0])


def selection_is_valid(ids: np.ndarray, block_scores: np.ndarray, pos: int, block_size: int,
                       topk: int, tol: float) -> bool:
    """A selection other than the oracle's is acceptable when it keeps the
    local block, has min(k, lb+1) distinct causal blocks, and every selected
    non-local block scores within ``tol`` of every unselected candidate."""
    lb = pos // block_size
    sel = [int(b) for b in ids if b >= 0]
    if len(sel) != len(set(sel)) or len(sel) != min(topk, lb + 1) or lb not in sel:
        return False
    if any(b < 0 or b > lb for b in sel):
        return False
    if list(ids[:len(sel)]) != sorted(sel) or any(int(b) != -1 for b in ids[len(sel):]):
        return False
    nonlocal_sel = [b for b in sel if b != lb]
    unsel = [b for b in range(lb) if b not in set(sel)]
    if not nonlocal_sel or not unsel:
        return True
    return min(block_scores[b] for b in nonlocal_sel) >= max(block_scores[b] for b in unsel) - tol


def row_topk(scores: np.ndarray, k: int) -> np.ndarray:
    """The Top-k operator on its own: for each row of an (N, B) score matrix,
    the min(k, B) columns of largest score, equal scores keeping the lower
    column (R3), listed ascending and padded with -1 to ``k`` (Sec. 3.1 top-k
    equation without the forced local block; Sec. 4.1 latency table: fp32
    inputs of shape (N, B), rows processed independently).  -0 equals +0."""
    scores = np.asarray(scores)
    n, B = scores.shape
    out = np.full((n, k), -1, dtype=np.int32)
    cols = np.arange(B)
    for i in range(n):
        order = np.lexsort((cols, -scores[i].astype(np.float64)))
        sel = np.sort(cols[order[:k]])
        out[i, :sel.shape[0]] = sel
    return out


# --------------------------------------------------------------------------
# Main Branch (Sec. 3.1, sparse-attention equation)
# --------------------------------------------------------------------------
def attend(qh: np.ndarray, keys: np.ndarray, vals: np.ndarray, scale: float):
    """Softmax attention of query heads qh (G, d) over keys/vals (n, d);
    returns O (G, d) and the natural-log LSE (G,)."""
    z = (qh @ keys.T) * scale                    # (G, n)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    l = e.sum(axis=1, keepdims=True)
    o = (e @ vals) / l
    lse = (m + np.log(l))[:, 0]
    return o, lse


def selected_tokens(block_ids_row: Sequence[int], pos: int, block_size: int) -> np.ndarray:
    """Causally visible tokens of the selected blocks (ids < 0 are padding)."""
    parts = [np.arange(b * block_size, min((b + 1) * block_size, pos + 1))
             for b in block_ids_row if b >= 0 and b * block_size <= pos]
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


def sparse_attention(q_bits, k_bits, v_bits, block_ids: np.ndarray, layout: Layout,
                     block_size: int, scale: Optional[float] = None,
                     rows: Optional[Iterable[int]] = None,
                     block_ids_are_for_rows: bool = False, fmt: str = "bf16",
                     input_scales: Tuple[float, float, float] = (1.0, 1.0, 1.0)):
    """O (R, H_q, d_h) and LSE (R, H_q), float64, for the given packed rows.

    q_bits: (Tq, H_q, d_h); k_bits, v_bits: (Tk, H_kv, d_h): bf16 bit patterns
    (uint16), or E4M3 codes (uint8) with fmt="e4m3", whose values are the
    decoded codes times the per-tensor ``input_scales`` (q, k, v).
    block_ids: (Tq, H_kv, k) for all rows, or (R, H_kv, k) aligned with
    ``rows`` when ``block_ids_are_for_rows``.  Head h uses group h // G."""
    dec = _decoder(fmt)
    qs, ks, vs = (float(x) for x in input_scales)
    Tq, H_q, d_h = q_bits.shape
    H_kv = k_bits.shape[1]
    G = H_q // H_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d_h)
    rows = list(range(Tq)) if rows is None else [int(r) for r in rows]
    O = np.zeros((len(rows), H_q, d_h))
    L = np.zeros((len(rows), H_q))
    for i, r in enumerate(rows):
        s, pos = layout.locate(r)
        kv0 = layout.kv_starts[s]
        qf = dec(q_bits[r]) * qs
        ids_row = block_ids[i] if block_ids_are_for_rows else block_ids[r]
        for g in range(H_kv):
            toks = selected_tokens(ids_row[g], pos, block_size)
            keys = dec(k_bits[kv0 + toks, g]) * ks
            vals = dec(v_bits[kv0 + toks, g]) * vs
            O[i, g * G:(g + 1) * G], L[i, g * G:(g + 1) * G] = attend(
                qf[g * G:(g + 1) * G], keys, vals, scale)
    return O, L


def dense_causal_attention(q_bits, k_bits, v_bits, layout: Layout, scale: Optional[float] = None,
                           rows: Optional[Iterable[int]] = None):
    """Causal GQA softmax attention over all tokens j <= p (Sec. 2.1)."""
    Tq, H_q, d_h = q_bits.shape
    H_kv = k_bits.shape[1]
    G = H_q // H_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d_h)
    rows = list(range(Tq)) if rows is None else [int(r) for r in rows]
    O = np.zeros((len(rows), H_q, d_h))
    L = np.zeros((len(rows), H_q))
    for i, r in enumerate(rows):
        s, pos = layout.locate(r)
        kv0 = layout.kv_starts[s]
        qf = decode_bf16(q_bits[r])
        for g in range(H_kv):
            keys = decode_bf16(k_bits[kv0:kv0 + pos + 1, g])
            vals = decode_bf16(v_bits[kv0:kv0 + pos + 1, g])
            O[i, g * G:(g + 1) * G], L[i, g * G:(g + 1) * G] = attend(
                qf[g * G:(g + 1) * G], keys, vals, scale)
    return O, L


# --------------------------------------------------------------------------
# Split combine (Sec. 4.2, "Two-phase forward")
# --------------------------------------------------------------------------
def combine_partials(lse_parts: np.ndarray, o_parts: np.ndarray):
    """Merge S locally normalised partials: a = max_s LSE_s,
    LSE = a + log sum_s exp(LSE_s - a), w_s = exp(LSE_s - LSE), O = sum_s w_s O_s.

    lse_parts: (S,), o_parts: (S, d) -> (O (d,), LSE scalar)."""
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    a = lse_parts.max()
    lse = a + math.log(np.exp(lse_parts - a).sum())
    w = np.exp(lse_parts - lse)
    return (w[:, None] * np.asarray(o_parts, dtype=np.float64)).sum(axis=0), lse


# --------------------------------------------------------------------------
# FLOP model (Sec. 3.3) and effective work
# --------------------------------------------------------------------------
def flops_gqa(N: int, H_q: int, d_h: int) -> float:
    """Causal GQA attention FLOPs, F_GQA(N) = 2 H_q d_h N^2 (Sec. 3.3)."""
    return 2.0 * H_q * d_h * N * N


def flops_msa(N: int, H_q: int, H_kv: int, d_h: int, d_idx: int, block_size: int, k: int) -> float:
    """F_MSA(N) = H_kv d_idx N^2 (Index Branch) + 4 H_q d_h N k B_k (Main Branch)."""
    return float(H_kv) * d_idx * N * N + 4.0 * H_q * d_h * N * k * block_size


def effective_main_flops(block_ids: np.ndarray, positions: np.ndarray, H_q: int, d_h: int,
                         block_size: int) -> float:
    """4 d_h x (sum over rows and query heads of the number of attended
    tokens): QK^T and PV each cost 2 d_h FLOPs per (query head, token)."""
    H_kv = block_ids.shape[1]
    G = H_q // H_kv
    total = 0
    for i in range(block_ids.shape[0]):
        p = int(positions[i])
        for g in range(H_kv):
            for b in block_ids[i, g]:
                if b >= 0 and b * block_size <= p:
                    total += min((b + 1) * block_size, p + 1) - b * block_size
    return 4.0 * d_h * G * total


# --------------------------------------------------------------------------
# Training backward (Sec. 3.2 "KL Loss", "Gradient Detach"; Alg. 1; Sec. 4.3)
# --------------------------------------------------------------------------
def softmax_rows(z: np.ndarray) -> np.ndarray:
    """Row-wise softmax, float64."""
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attend_backward(qh: np.ndarray, keys: np.ndarray, vals: np.ndarray, d_o: np.ndarray, scale: float):
    """Gradients of sum(d_o * O) for O = softmax(scale qh keys^T) vals.

    qh, d_o: (G, d); keys, vals: (n, d).  Returns dq (G, d), dk (n, d), dv (n, d).
    The softmax Jacobian applied to dP = d_o vals^T gives, per row,
    dz_j = p_j (dP_j - sum_u p_u dP_u); z = scale q.k passes scale on."""
    p = softmax_rows((qh @ keys.T) * scale)      # (G, n)
    dv = p.T @ d_o
    dp = d_o @ vals.T                            # (G, n)
    dz = p * (dp - (p * dp).sum(axis=1, keepdims=True))
    dq = (dz @ keys) * scale
    dk = (dz.T @ qh) * scale
    return dq, dk, dv


def sparse_attention_backward(q_bits, k_bits, v_bits, d_o_bits, block_ids: np.ndarray, layout: Layout,
                              block_size: int, scale: Optional[float] = None):
    """dQ (Tq, H_q, d_h), dK and dV (Tk, H_kv, d_h), float64: gradients of
    sum(dO * O) for the Main Branch output O of every packed row (the
    sparse-attention equation of Sec. 3.1; Alg. 1 trains through it).

    All inputs are bf16 bit patterns; dO (Tq, H_q, d_h).  Key rows that no
    query attends receive zero gradient."""
    Tq, H_q, d_h = q_bits.shape
    H_kv = k_bits.shape[1]
    G = H_q // H_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d_h)
    dQ = np.zeros((Tq, H_q, d_h))
    dK = np.zeros((k_bits.shape[0], H_kv, d_h))
    dV = np.zeros_like(dK)
    for r in range(Tq):
        s, pos = layout.locate(r)
        kv0 = layout.kv_starts[s]
        qf = decode_bf16(q_bits[r])
        gf = decode_bf16(d_o_bits[r])
        for g in range(H_kv):
            toks = selected_tokens(block_ids[r, g], pos, block_size)
            if toks.shape[0] == 0:
                continue
            heads = slice(g * G, (g + 1) * G)
            dq, dk, dv = attend_backward(qf[heads], decode_bf16(k_bits[kv0 + toks, g]),
                                         decode_bf16(v_bits[kv0 + toks, g]), gf[heads], scale)
            dQ[r, heads] += dq
            dK[kv0 + toks, g] += dk
            dV[kv0 + toks, g] += dv
    return dQ, dK, dV


def kl_row(iq_r: np.ndarray, ik_toks: np.ndarray, q_heads: np.ndarray, k_toks: np.ndarray,
           scale_idx: float, scale_main: float):
    """KL(sg(P) || P_idx) of one (query, group) over its token set, and the
    gradients of that value with respect to S_idx, q_idx and the k_idx rows.

    P_idx = softmax(scale_idx q_idx . k_idx) over the tokens; the teacher P is
    the mean over the group's heads of the per-head Main Branch softmax
    distributions over the same tokens (the P / P_idx equation of Sec. 3.2).
    With P detached, d KL / d S_idx_j = P_idx_j - P_j."""
    s_idx = (ik_toks @ iq_r) * scale_idx                      # (n,)
    p_idx = softmax_rows(s_idx[None, :])[0]
    p = softmax_rows((q_heads @ k_toks.T) * scale_main).mean(axis=0)
    kl = float(np.sum(p * (np.log(p) - np.log(p_idx))))
    ds = p_idx - p
    d_iq = (ds @ ik_toks) * scale_idx
    d_ik = np.outer(ds, iq_r) * scale_idx
    return kl, d_iq, d_ik


def sparse_kl(index_q_bits, index_k_bits, q_bits, k_bits, block_ids: np.ndarray, layout: Layout,
              block_size: int, scale_idx: Optional[float] = None, scale_main: Optional[float] = None):
    """Sparse KL loss terms and their gradients for every packed row.

    Returns kl (Tq, H_kv): KL(sg(P^(r)_i) || P_idx^(r)_i) over the causally
    visible tokens of the selected blocks (Sec. 3.2, KL-loss equation; the
    loss is their mean over rows and groups), and the gradients of
    sum_{i,r} kl[i, r] with respect to index_q (Tq, H_kv, d_idx) and
    index_k (Tk, d_idx).  Under the gradient detach of Sec. 3.2 nothing flows
    into Q or K.  A (row, group) without visible tokens contributes 0."""
    Tq, H_kv, d_idx = index_q_bits.shape
    H_q, d_h = q_bits.shape[1], q_bits.shape[2]
    G = H_q // H_kv
    if scale_idx is None:
        scale_idx = 1.0 / math.sqrt(d_idx)
    if scale_main is None:
        scale_main = 1.0 / math.sqrt(d_h)
    kl = np.zeros((Tq, H_kv))
    d_iq = np.zeros((Tq, H_kv, d_idx))
    d_ik = np.zeros((index_k_bits.shape[0], d_idx))
    for r in range(Tq):
        s, pos = layout.locate(r)
        kv0 = layout.kv_starts[s]
        iq = decode_bf16(index_q_bits[r])
        qf = decode_bf16(q_bits[r])
        for g in range(H_kv):
            toks = selected_tokens(block_ids[r, g], pos, block_size)
            if toks.shape[0] == 0:
                continue
            kl[r, g], d_iq[r, g], dk = kl_row(iq[g], decode_bf16(index_k_bits[kv0 + toks]),
                                              qf[g * G:(g + 1) * G], decode_bf16(k_bits[kv0 + toks, g]),
                                              scale_idx, scale_main)
            d_ik[kv0 + toks] += dk
    return kl, d_iq, d_ik
