"""Seeded synthetic inputs for the MSA inference hot path.

This module draws the inputs that both the HIP path (tests, bench) and the CPU
oracle consume.  It holds none of the method's arithmetic: it draws N(0,1)
values, optionally plants "relevant" index-key blocks, rounds each tensor once
to bf16 (round to nearest even) and describes the sequence layout.

Layout conventions (shared by every entry point of the library):

* a batch is ``num_seqs`` sequences; sequence ``s`` owns query rows
  ``q_offsets[s] .. q_offsets[s+1]`` of the packed query-side tensors and key
  rows ``kv_starts[s] .. kv_starts[s] + kv_lens[s]`` of the key-side tensors;
* query row ``t`` (0-based inside its sequence) sits at absolute position
  ``kv_lens[s] - q_rows[s] + t``: its own key/value (and index key) are already
  in the cache.  Prefill has ``q_rows == kv_len``; decode has ``q_rows == 1``.

Two backends: ``numpy`` (row-addressable chunks, used by CPU tests and small
GPU cases) and ``torch`` (draws directly on a device, used for the large
workloads whose host-side generation would take minutes).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

CHUNK_ROWS = 65536

# tensor ids used to derive independent streams from one seed
TID_INDEX_Q, TID_INDEX_K, TID_Q, TID_K, TID_V, TID_PLANT, TID_LENS, TID_DO, TID_BLOCKS = range(9)


# --------------------------------------------------------------------------
# bf16 helpers (representation only)
# --------------------------------------------------------------------------
def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# problem description
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Problem:
    """Shapes, hyper-parameters and sequence layout of one workload."""

    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    d_idx: int
    block_size: int
    topk: int
    q_rows: List[int]
    kv_lens: List[int]
    kv_starts: List[int]
    total_kv_rows: int
    seed: int
    planted_blocks_per_group: int = 0
    plant_alpha: Optional[float] = None   # default 2*sqrt(d_idx)
    description: str = ""

    @property
    def num_seqs(self) -> int:
        return len(self.q_rows)

    @property
    def q_offsets(self) -> List[int]:
        out = [0]
        for r in self.q_rows:
            out.append(out[-1] + r)
        return out

    @property
    def total_q_rows(self) -> int:
        return sum(self.q_rows)

    @property
    def max_q_rows(self) -> int:
        return max(self.q_rows) if self.q_rows else 0

    @property
    def max_kv_len(self) -> int:
        return max(self.kv_lens) if self.kv_lens else 0

    @property
    def group_size(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def positions(self) -> np.ndarray:
        """Absolute position of every packed query row (int64)."""
        pos = np.empty(self.total_q_rows, dtype=np.int64)
        off = 0
        for s, qr in enumerate(self.q_rows):
            pos[off:off + qr] = self.kv_lens[s] - qr + np.arange(qr)
            off += qr
        return pos

    def seq_of_row(self) -> np.ndarray:
        out = np.empty(self.total_q_rows, dtype=np.int64)
        off = 0
        for s, qr in enumerate(self.q_rows):
            out[off:off + qr] = s
            off += qr
        return out


def packed_problem(name, q_rows, kv_lens, *, num_q_heads, num_kv_heads, head_dim=128,
                   d_idx=64, block_size=64, topk=8, seed=0, planted=0, description="",
                   kv_pad_to: Optional[int] = None) -> Problem:
    """Sequences packed back to back in the key-side tensors.

    ``kv_pad_to`` places sequence ``s`` at key row ``s * kv_pad_to`` instead
    (a padded cache, as decode uses)."""
    assert len(q_rows) == len(kv_lens)
    for qr, kl in zip(q_rows, kv_lens):
        assert 0 <= qr <= kl
    starts = []
    if kv_pad_to is None:
        acc = 0
        for kl in kv_lens:
            starts.append(acc)
            acc += kl
        total = acc
    else:
        assert all(kl <= kv_pad_to for kl in kv_lens)
        starts = [s * kv_pad_to for s in range(len(kv_lens))]
        total = kv_pad_to * len(kv_lens)
    return Problem(name=name, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                   head_dim=head_dim, d_idx=d_idx, block_size=block_size, topk=topk,
                   q_rows=list(q_rows), kv_lens=list(kv_lens), kv_starts=starts,
                   total_kv_rows=total, seed=seed, planted_blocks_per_group=planted,
                   description=description)


def chunked_contexts(seed: int, num_seqs: int, lo: int, hi: int) -> List[int]:
    """Cached context lengths drawn log-uniformly in [lo, hi]."""
    rng = np.random.default_rng([seed, TID_LENS])
    u = rng.uniform(math.log(lo), math.log(hi), size=num_seqs)
    return [int(math.floor(math.exp(x))) for x in u]


# The five workloads the library is measured on.
def workload(name: str) -> Problem:
    if name == "prefill_4k":
        return packed_problem(name, [4096], [4096], num_q_heads=8, num_kv_heads=2, topk=8,
                              seed=1001, description="prefill T=4096, 8q/2kv, k=8, i.i.d. N(0,1)")
    if name == "prefill_32k":
        return packed_problem(name, [32768], [32768], num_q_heads=64, num_kv_heads=8, topk=32,
                              seed=1002, planted=16,
                              description="prefill T=32768, 64q/8kv, k=32, 16 planted blocks/group")
    if name == "decode_128k":
        return packed_problem(name, [1] * 64, [131072] * 64, num_q_heads=64, num_kv_heads=8,
                              topk=32, seed=1003, kv_pad_to=131072,
                              description="decode 64 seqs x 1 token, context 131072, 64q/8kv, k=32")
    if name == "prefill_1m":
        return packed_problem(name, [1 << 20], [1 << 20], num_q_heads=64, num_kv_heads=8, topk=64,
                              seed=1004, planted=32,
                              description="prefill T=1048576, 64q/8kv, k=64, 32 planted blocks/group")
    if name == "prefill_1m_bk128":
        return packed_problem(name, [1 << 20], [1 << 20], num_q_heads=64, num_kv_heads=4, d_idx=128,
                              block_size=128, topk=16, seed=1006, planted=8,
                              description="prefill T=1048576, 64q/4kv, d_idx 128, B_k 128, k=16, "
                                          "8 planted blocks/group (the paper's deployed shape)")
    if name == "prefill_32k_bk128":
        return packed_problem(name, [32768], [32768], num_q_heads=64, num_kv_heads=4, d_idx=128,
                              block_size=128, topk=16, seed=1008, planted=8,
                              description="prefill T=32768, 64q/4kv, d_idx 128, B_k 128, k=16, "
                                          "8 planted blocks/group (the deployed shape at a training length)")
    if name == "decode_128k_bk128":
        return packed_problem(name, [1] * 64, [131072] * 64, num_q_heads=64, num_kv_heads=4, d_idx=128,
                              block_size=128, topk=16, seed=1007, kv_pad_to=131072,
                              description="decode 64 seqs x 1 token, context 131072, 64q/4kv, d_idx 128, "
                                          "B_k 128, k=16 (the paper's deployed shape)")
    if name == "chunked_8x8k":
        ctx = chunked_contexts(1005, 8, 16384, 524288)
        return packed_problem(name, [8192] * 8, [c + 8192 for c in ctx], num_q_heads=64,
                              num_kv_heads=8, topk=48, seed=1005,
                              description="chunked prefill, 8 seqs x 8192 new rows on 16K-512K contexts, k=48")
    raise KeyError(name)


WORKLOADS = ["prefill_4k", "prefill_32k", "decode_128k", "prefill_1m", "chunked_8x8k"]
# the paper's deployed shape (B_k 128, k 16, GQA 16, d_idx 128)
WORKLOADS_BK128 = ["prefill_1m_bk128", "decode_128k_bk128", "prefill_32k_bk128"]


def stratified_rows(p: Problem, n: int, seed: int) -> List[int]:
    """About ``n`` packed query rows spread over every depth, for checks and
    baselines that cannot afford every row: each sequence's rows are cut into
    equal bands (a count proportional to its rows) and one row is drawn per
    band; each sequence's first rows (its first two key blocks' worth) and its
    last row are always included.  Sorted, distinct."""
    rng = np.random.default_rng([seed, 99])
    T = p.total_q_rows
    out = set()
    for s in range(p.num_seqs):
        a, b = p.q_offsets[s], p.q_offsets[s + 1]
        if b <= a:
            continue
        m = b - a
        bands = max(1, min(m, round(n * m / max(T, 1))))
        edges = np.linspace(a, b, bands + 1).astype(np.int64)
        for lo, hi in zip(edges[:-1], edges[1:]):
            if hi > lo:
                out.add(int(rng.integers(lo, hi)))
        B = p.block_size
        for off in (0, 1, B - 1, B, B + 1, 2 * B - 1):
            if off < m:
                out.add(a + off)
        out.add(b - 1)
    return sorted(out)


# --------------------------------------------------------------------------
# numpy backend (row addressable)
# --------------------------------------------------------------------------
def _normal_rows(seed: int, tid: int, rows: int, row_width: int, row0: int = 0,
                 nrows: Optional[int] = None) -> np.ndarray:
    """N(0,1) float32 rows [row0, row0+nrows) of a (rows, row_width) tensor.

    Rows are drawn in chunks of CHUNK_ROWS from default_rng([seed, tid, chunk]),
    so any row range is reproducible without drawing the rows before it."""
    if nrows is None:
        nrows = rows - row0
    out = np.empty((nrows, row_width), dtype=np.float32)
    r = row0
    while r < row0 + nrows:
        c = r // CHUNK_ROWS
        c0 = c * CHUNK_ROWS
        c1 = min(c0 + CHUNK_ROWS, rows)
        rng = np.random.default_rng([seed, tid, c])
        chunk = rng.standard_normal((c1 - c0, row_width), dtype=np.float32)
        a = r - c0
        b = min(c1, row0 + nrows) - c0
        out[r - row0:r - row0 + (b - a)] = chunk[a:b]
        r = c0 + b
    return out


def plant_plan(p: Problem) -> Dict[int, List[int]]:
    """Per group r: the key blocks (block index inside sequence 0) that get
    shifted toward group r's random index query.  Blocks are disjoint across
    groups (the index key head is shared)."""
    if p.planted_blocks_per_group <= 0:
        return {}
    nblk = p.kv_lens[0] // p.block_size
    need = p.planted_blocks_per_group * p.num_kv_heads
    assert nblk > need
    rng = np.random.default_rng([p.seed, TID_PLANT])
    blocks = rng.choice(nblk - 1, size=need, replace=False)  # never the last block
    plan = {}
    for r in range(p.num_kv_heads):
        plan[r] = sorted(int(b) for b in blocks[r * p.planted_blocks_per_group:
                                                   (r + 1) * p.planted_blocks_per_group])
    return plan


def plant_anchor_rows(p: Problem) -> List[int]:
    rng = np.random.default_rng([p.seed, TID_PLANT, 1])
    return [int(x) for x in rng.integers(0, p.total_q_rows, size=p.num_kv_heads)]


def _plant_alpha(p: Problem) -> float:
    return p.plant_alpha if p.plant_alpha is not None else 2.0 * math.sqrt(p.d_idx)


def generate_numpy(p: Problem) -> Dict[str, np.ndarray]:
    """All five input tensors as uint16 bf16 bit patterns (numpy)."""
    Tq, Tk = p.total_q_rows, p.total_kv_rows
    out = {}
    iq = _normal_rows(p.seed, TID_INDEX_Q, Tq, p.num_kv_heads * p.d_idx)
    out["index_q"] = bf16_bits_from_f32(iq).reshape(Tq, p.num_kv_heads, p.d_idx)
    ik = _normal_rows(p.seed, TID_INDEX_K, Tk, p.d_idx)
    if p.planted_blocks_per_group:
        iqf = f32_from_bf16_bits(out["index_q"])
        anchors = plant_anchor_rows(p)
        alpha = _plant_alpha(p)
        base = p.kv_starts[0]
        for r, blocks in plant_plan(p).items():
            u = iqf[anchors[r], r].astype(np.float64)
            u = (u / np.linalg.norm(u)).astype(np.float32)
            for b in blocks:
                ik[base + b * p.block_size: base + (b + 1) * p.block_size] += alpha * u
    out["index_k"] = bf16_bits_from_f32(ik)
    out["q"] = bf16_bits_from_f32(_normal_rows(p.seed, TID_Q, Tq, p.num_q_heads * p.head_dim)
                                  ).reshape(Tq, p.num_q_heads, p.head_dim)
    out["k"] = bf16_bits_from_f32(_normal_rows(p.seed, TID_K, Tk, p.num_kv_heads * p.head_dim)
                                  ).reshape(Tk, p.num_kv_heads, p.head_dim)
    out["v"] = bf16_bits_from_f32(_normal_rows(p.seed, TID_V, Tk, p.num_kv_heads * p.head_dim)
                                  ).reshape(Tk, p.num_kv_heads, p.head_dim)
    return out


# --------------------------------------------------------------------------
# 8-bit E4M3 inputs for the Main Branch
# --------------------------------------------------------------------------
# Per-tensor scales of the e4m3 workloads: N(0,1) / 2^-4 keeps |code value| <=
# ~100, well inside e4m3's +-448 range.
FP8_SCALES = (2.0 ** -4, 2.0 ** -4, 2.0 ** -4)


def e4m3_codes(x, scale: float):
    """float32 values (numpy or torch) -> OCP E4M3 codes of x / scale, rounded
    to nearest even (torch's float8_e4m3fn cast), as uint8 of the same kind."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)) if isinstance(x, np.ndarray) else x
    codes = (t.float() / scale).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes.numpy() if isinstance(x, np.ndarray) else codes


def generate_fp8_numpy(p: Problem, scales=FP8_SCALES) -> Dict[str, np.ndarray]:
    """Index tensors as bf16 patterns (as generate_numpy) and q, k, v as E4M3
    codes (uint8) of the same N(0,1) draws divided by ``scales``."""
    Tq, Tk = p.total_q_rows, p.total_kv_rows
    out = {k: v for k, v in generate_numpy(p).items() if k in ("index_q", "index_k")}
    out["q"] = e4m3_codes(_normal_rows(p.seed, TID_Q, Tq, p.num_q_heads * p.head_dim), scales[0]
                          ).reshape(Tq, p.num_q_heads, p.head_dim)
    out["k"] = e4m3_codes(_normal_rows(p.seed, TID_K, Tk, p.num_kv_heads * p.head_dim), scales[1]
                          ).reshape(Tk, p.num_kv_heads, p.head_dim)
    out["v"] = e4m3_codes(_normal_rows(p.seed, TID_V, Tk, p.num_kv_heads * p.head_dim), scales[2]
                          ).reshape(Tk, p.num_kv_heads, p.head_dim)
    return out


# --------------------------------------------------------------------------
# torch backend (draws on the device; for the large workloads)
# --------------------------------------------------------------------------
def generate_torch(p: Problem, device, tensors=("index_q", "index_k", "q", "k", "v"), fp8_scales=None):
    """Same distributions and planting recipe, drawn with torch's generator on
    ``device``.  Returns bf16 torch tensors; with ``fp8_scales`` (q, k, v), q, k
    and v are E4M3 codes (uint8) of the draws divided by those scales.  (Values
    differ from the numpy backend; the oracle reads whatever rows it needs back
    from these inputs.)"""
    import torch

    def draw(tid, shape, fp8_scale=None):
        g = torch.Generator(device=device)
        g.manual_seed(int(p.seed) * 1000003 + tid)
        dtype = torch.bfloat16 if fp8_scale is None else torch.uint8
        out = torch.empty(shape, dtype=dtype, device=device)
        flat = out.view(shape[0], -1)
        step = max(1, (1 << 27) // max(1, flat.shape[1]))
        for r0 in range(0, shape[0], step):
            r1 = min(shape[0], r0 + step)
            x = torch.randn((r1 - r0, flat.shape[1]), generator=g, device=device, dtype=torch.float32)
            flat[r0:r1] = x.to(torch.bfloat16) if fp8_scale is None else e4m3_codes(x, fp8_scale)
        return out

    Tq, Tk = p.total_q_rows, p.total_kv_rows
    out = {}
    if "index_q" in tensors or p.planted_blocks_per_group:
        out["index_q"] = draw(TID_INDEX_Q, (Tq, p.num_kv_heads, p.d_idx))
    if "index_k" in tensors:
        g = torch.Generator(device=device)
        g.manual_seed(int(p.seed) * 1000003 + TID_INDEX_K)
        ik = torch.randn((Tk, p.d_idx), generator=g, device=device, dtype=torch.float32)
        if p.planted_blocks_per_group:
            anchors = plant_anchor_rows(p)
            alpha = _plant_alpha(p)
            base = p.kv_starts[0]
            for r, blocks in plant_plan(p).items():
                u = out["index_q"][anchors[r], r].float()
                u = u / torch.linalg.vector_norm(u.double()).float()
                for b in blocks:
                    ik[base + b * p.block_size: base + (b + 1) * p.block_size] += alpha * u
        out["index_k"] = ik.to(torch.bfloat16)
        del ik
    fs = (None, None, None) if fp8_scales is None else tuple(fp8_scales)
    if "q" in tensors:
        out["q"] = draw(TID_Q, (Tq, p.num_q_heads, p.head_dim), fs[0])
    if "k" in tensors:
        out["k"] = draw(TID_K, (Tk, p.num_kv_heads, p.head_dim), fs[1])
    if "v" in tensors:
        out["v"] = draw(TID_V, (Tk, p.num_kv_heads, p.head_dim), fs[2])
    if "d_o" in tensors:
        out["d_o"] = draw(TID_DO, (Tq, p.num_q_heads, p.head_dim))
    if "index_q" not in tensors:
        out.pop("index_q", None)
    return out


# --------------------------------------------------------------------------
# training-backward inputs
# --------------------------------------------------------------------------
def generate_grad_numpy(p: Problem) -> np.ndarray:
    """Upstream gradient dO of the Main Branch output: N(0,1) rounded to bf16,
    (Tq, H_q, d_h) uint16 bit patterns.  (Real upstream gradients are smaller;
    every bar on the backward is relative, and bf16 keeps its relative
    precision over the whole range used.)"""
    Tq = p.total_q_rows
    return bf16_bits_from_f32(_normal_rows(p.seed, TID_DO, Tq, p.num_q_heads * p.head_dim)
                              ).reshape(Tq, p.num_q_heads, p.head_dim)


def random_block_ids(p: Problem, pad_slots: int = 0) -> np.ndarray:
    """A seeded block selection with the structure of a Top-k output, drawn
    without looking at any score: per (row, group) the block holding the row's
    own position plus min(k - 1, lb) distinct earlier blocks chosen uniformly,
    ascending, padded with -1 to k (+ ``pad_slots`` extra -1 slots).  Rows
    at a position < 0 get only -1."""
    rng = np.random.default_rng([p.seed, TID_BLOCKS])
    k = p.topk
    ids = np.full((p.total_q_rows, p.num_kv_heads, k + pad_slots), -1, dtype=np.int32)
    pos = p.positions()
    for row in range(p.total_q_rows):
        if pos[row] < 0:
            continue
        lb = int(pos[row]) // p.block_size
        take = min(k - 1, lb)
        for g in range(p.num_kv_heads):
            others = rng.choice(lb, size=take, replace=False) if take else np.zeros(0, dtype=np.int64)
            sel = np.sort(np.concatenate([others, [lb]]))
            ids[row, g, :sel.shape[0]] = sel
    return ids


# --------------------------------------------------------------------------
# score matrices for the Top-k operator on its own
# --------------------------------------------------------------------------
# (N, B, k) of the paper's Top-k latency table (Sec. 4.1): N rows of B block
# scores each, k kept per row.  The paper does not state its score values;
# rows of i.i.d. N(0, 1) floats stand in (for i.i.d. continuous scores the
# rank pattern of a row, which is all a comparison-based Top-k sees, does not
# depend on the distribution).
TOPK_SHAPES = [(131072, 1024, 16), (131072, 2048, 32), (524288, 4096, 16), (524288, 8192, 32)]
TID_TOPK = 9


def topk_scores(n_rows: int, n_cols: int, seed: int, device, ld: Optional[int] = None,
                pool: Optional[List[float]] = None):
    """fp32 [n_rows, n_cols] score matrix: i.i.d. N(0, 1), or drawn uniformly
    from ``pool`` (to force ties, signed zeros, -inf).  With ``ld`` > n_cols
    it is a view of the first n_cols columns of an [n_rows, ld] matrix."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + TID_TOPK)
    width = n_cols if ld is None else int(ld)
    if pool is None:
        full = torch.randn((n_rows, width), generator=g, device=device, dtype=torch.float32)
    else:
        vals = torch.tensor(pool, dtype=torch.float32, device=device)
        full = vals[torch.randint(0, len(pool), (n_rows, width), generator=g, device=device)]
    return full[:, :n_cols]
