"""Training backward of the Main Branch (msa_sparse_attn_backward) against the
oracle's float64 gradients.

Block selections come from the seeded score-free generator (the structure of
a Top-k output), so these cases test the backward alone; O and LSE are the
library's own forward outputs, as in training.  Bar: check_grad (tests/util).
"""
from __future__ import annotations

import ctypes
import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle.msa_oracle as O
from paper_2606_13392_amd import msa, synth
from tests.util import check_grad, from_dev_bits, random_layouts, to_dev

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    msa.lib()
    yield
    torch.cuda.synchronize()


# name, q_rows, kv_lens, H_q, H_kv, topk, kv_pad_to[, block_size]
CASES = [
    ("bwd_T1000_g8", [1000], [1000], 16, 2, 8, None),
    ("bwd_ragged_T333_g4", [333], [333], 8, 2, 5, None),
    ("bwd_g16", [300], [300], 32, 2, 4, None),
    ("bwd_g1", [200], [200], 4, 4, 3, None),
    ("bwd_g3", [150], [150], 6, 2, 4, None),
    ("bwd_chunked_varlen", [130, 0, 64, 1, 257], [700, 300, 64, 900, 1500], 16, 4, 6, None),
    ("bwd_decode_padded", [1, 1, 1, 1, 1], [3000, 64, 65, 4097, 1], 16, 4, 6, 4160),
    ("bwd_many_items_k32", [2048], [2048], 16, 2, 32, None),
    ("bwd_bk128_g16", [900], [900], 32, 2, 5, None, 128),
    ("bwd_bk128_chunked_varlen", [200, 1, 129], [1000, 700, 1500], 16, 2, 4, None, 128),
    ("bwd_bk128_k48_g8", [3000], [3000], 32, 4, 24, None, 128),
    ("bwd_bk128_decode_padded", [1, 1, 1], [3000, 129, 4097], 16, 2, 6, 4224, 128),
]


def _setup(name, q_rows, kv_lens, H_q, H_kv, topk, pad, bk=64):
    p = synth.packed_problem(name, q_rows, kv_lens, num_q_heads=H_q, num_kv_heads=H_kv, topk=topk, block_size=bk,
                             seed=zlib.crc32(name.encode()) % 10000, kv_pad_to=pad)
    x = {k: v for k, v in synth.generate_numpy(p).items() if k in ("q", "k", "v")}
    x["d_o"] = synth.generate_grad_numpy(p)
    ids = synth.random_block_ids(p)
    return p, x, ids


def _run(p, x, ids, workspace_bytes=None):
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}
    ids_d = torch.from_numpy(ids).to(dev)
    fwd = msa.sparse_attn_decode if p.max_q_rows == 1 else msa.sparse_attn_prefill
    o, lse = fwd(d["q"], d["k"], d["v"], ids_d, seqs, p.block_size)
    if workspace_bytes is None:
        dq, dk, dv = msa.sparse_attn_backward(d["q"], d["k"], d["v"], o, lse, d["d_o"], ids_d, seqs, p.block_size)
    else:
        dq, dk, dv = (torch.empty_like(d[t]) for t in ("q", "k", "v"))
        ws = torch.empty(workspace_bytes, dtype=torch.uint8, device=dev)
        st = msa.lib().msa_sparse_attn_backward(
            d["q"].data_ptr(), d["k"].data_ptr(), d["v"].data_ptr(), o.data_ptr(), lse.data_ptr(),
            d["d_o"].data_ptr(), ids_d.data_ptr(), seqs.ref(), p.num_q_heads, p.num_kv_heads, p.head_dim,
            p.block_size, ids.shape[2], 1.0 / math.sqrt(p.head_dim), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
            ws.data_ptr(), workspace_bytes, msa._stream())
        assert st == 0, msa.lib().msa_strerror(st)
    torch.cuda.synchronize()
    return (t.float().cpu().numpy() for t in (dq, dk, dv))


def _check_all(name, got, ref):
    for t, g, r in zip(("dQ", "dK", "dV"), got, ref):
        stats = check_grad(g, r, f"{name} {t}")
        _say(f"  {t} max-err/max|ref| {stats[0]:.2e} rel-L2 {stats[1]:.2e}")


# seeded random batch layouts (sequence mix, head groups, block size, Top-k, key padding)
RANDOM = [(c["name"], c["q_rows"], c["kv_lens"], c["H_q"], c["H_kv"], c["topk"], c["pad"], c["bk"])
          for c in random_layouts(21, 8)]


@pytest.mark.parametrize("case", CASES + RANDOM, ids=[c[0] for c in CASES + RANDOM])
def test_backward_small(case):
    name = case[0]
    _say(f"[case] {name}")
    p, x, ids = _setup(*case)
    got = list(_run(p, x, ids))
    ref = O.sparse_attention_backward(x["q"], x["k"], x["v"], x["d_o"], ids, O.layout_of(p), p.block_size)
    _check_all(name, got, ref)
    # key rows outside every sequence (cache padding) and keys nobody attends are exactly zero
    lay = O.layout_of(p)
    used = np.zeros(got[1].shape[:2], dtype=bool)
    for r in range(p.total_q_rows):
        s, pos = lay.locate(r)
        for g in range(p.num_kv_heads):
            used[p.kv_starts[s] + O.selected_tokens(ids[r, g], pos, p.block_size), g] = True
    assert np.all(got[1][~used] == 0) and np.all(got[2][~used] == 0)


def test_backward_chunked_workspace_and_reproducibility():
    """A workspace below the one-chunk size runs several row chunks and meets
    the same bar.  dQ sums its slot partials in slot order, so it is equal bit
    for bit across runs and chunkings; dK and dV add a block's queries in the
    ascending (row, slot) order the reverse index is sorted into, so they are
    equal bit for bit across runs with the same chunking."""
    case = ("bwd_chunks", [700, 900], [700, 1200], 16, 2, 6, None)
    _say("[case] bwd_chunks")
    p, x, ids = _setup(*case)
    seqs_h = msa.Seqs.from_problem(p, torch.device("cuda"))
    full = msa.sparse_attn_backward_workspace_size(seqs_h, p.num_q_heads, p.num_kv_heads, p.head_dim,
                                                   p.block_size, p.topk)
    one = list(_run(p, x, ids))
    again = list(_run(p, x, ids))
    assert np.array_equal(one[0], again[0]), "dQ is not reproducible"
    assert np.array_equal(one[1], again[1]) and np.array_equal(one[2], again[2]), "dK / dV are not reproducible"
    small = list(_run(p, x, ids, workspace_bytes=int(full * 0.4)))
    ref = O.sparse_attention_backward(x["q"], x["k"], x["v"], x["d_o"], ids, O.layout_of(p), p.block_size)
    _check_all("bwd_chunks (one chunk)", one, ref)
    _check_all("bwd_chunks (small workspace)", small, ref)
    assert np.array_equal(one[0], small[0]), "chunked dQ differs from the one-chunk dQ"


def test_backward_reproducible_on_crowded_tiles():
    """Tiles of thousands of queries (every row of a 4096-row sequence picks
    the same hot blocks): the reverse index's atomics hand out positions in a
    different order on every run, and the sorted handle lists still give dK
    and dV equal bit for bit over three runs."""
    case = ("bwd_crowded", [4096], [4096], 16, 2, 8, None)
    _say("[case] bwd_crowded")
    p, x, ids = _setup(*case)
    ids[:, :, 0] = np.where(ids[:, :, 0] >= 0, 0, ids[:, :, 0])      # block 0 in every row that sees it
    for r in range(ids.shape[0]):
        for g in range(ids.shape[1]):
            sel = sorted(set(int(b) for b in ids[r, g] if b >= 0))
            ids[r, g, :] = -1
            ids[r, g, :len(sel)] = sel
    runs = [list(_run(p, x, ids)) for _ in range(3)]
    for t in range(3):
        assert all(np.array_equal(runs[0][t], rr[t]) for rr in runs[1:]), f"output {t} differs between runs"
    ref = O.sparse_attention_backward(x["q"], x["k"], x["v"], x["d_o"], ids, O.layout_of(p), p.block_size)
    _check_all("bwd_crowded", runs[0], ref)


def test_backward_block_128_limits():
    """Block size 128 runs its own kernel (8 waves of 16 keys) with up to 64
    slots, like block size 64; other block sizes are rejected."""
    p = synth.packed_problem("bwd_bk128", [10], [10], num_q_heads=8, num_kv_heads=2, topk=2, seed=1)
    seqs = msa.Seqs.from_problem(p, torch.device("cuda"))
    assert msa.sparse_attn_backward_workspace_size(seqs, 8, 2, 128, 128, 64) > 0
    assert msa.sparse_attn_backward_workspace_size(seqs, 8, 2, 128, 128, 65) == 0
    assert msa.sparse_attn_backward_workspace_size(seqs, 8, 2, 128, 256, 2) == 0


def test_backward_workload_sampled():
    """Full-size 32K prefill (64 query / 8 KV heads, k 32, B_k 64; block ids
    from msa_index_topk): dQ of sampled rows and dK / dV of the last two key
    blocks against the oracle (every row that selected those blocks is
    recomputed), and two identities over all keys: sum_j dV_j = sum_i dO_i per
    group (each row's P sums to 1) and sum_j dK_j = 0 (each row's dS sums to 0)."""
    p = synth.workload("prefill_32k")
    _say("[case] backward prefill_32k sampled")
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = synth.generate_torch(p, dev, tensors=("index_q", "index_k", "q", "k", "v", "d_o"))
    ids = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    del d["index_q"], d["index_k"]
    o, lse = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, p.block_size)
    dq, dk, dv = msa.sparse_attn_backward(d["q"], d["k"], d["v"], o, lse, d["d_o"], ids, seqs, p.block_size)
    torch.cuda.synchronize()
    lay = O.layout_of(p)
    G, H_kv, B = p.group_size, p.num_kv_heads, p.block_size
    scale = 1.0 / math.sqrt(p.head_dim)
    ids_h = ids.cpu().numpy()

    def row_grads(r, g):
        s, pos = lay.locate(r)
        toks = O.selected_tokens(ids_h[r, g], pos, B)
        tt = torch.from_numpy(p.kv_starts[s] + toks).to(dev)
        hs = slice(g * G, (g + 1) * G)
        qh = O.decode_bf16(from_dev_bits(d["q"][r, hs]))
        gh = O.decode_bf16(from_dev_bits(d["d_o"][r, hs]))
        kk = O.decode_bf16(from_dev_bits(d["k"][tt, g]))
        vv = O.decode_bf16(from_dev_bits(d["v"][tt, g]))
        return toks, O.attend_backward(qh, kk, vv, gh, scale)

    # dQ of sampled rows
    rng = np.random.default_rng(p.seed)
    rows = sorted(set(int(r) for r in rng.integers(0, p.total_q_rows, size=12)) | {0, p.total_q_rows - 1})
    dq_ref = np.zeros((len(rows), p.num_q_heads, p.head_dim))
    for i, r in enumerate(rows):
        for g in range(H_kv):
            dq_ref[i, g * G:(g + 1) * G] = row_grads(r, g)[1][0]
    rows_t = torch.tensor(rows, dtype=torch.int64, device=dev)
    stats = check_grad(dq[rows_t].float().cpu().numpy(), dq_ref, "dQ sampled rows")
    _say(f"  dQ ({len(rows)} rows) max-err/max|ref| {stats[0]:.2e} rel-L2 {stats[1]:.2e}")

    # dK / dV of the last two key blocks: every (row, group) that selected them
    nblk = p.kv_lens[0] // B
    for b in (nblk - 2, nblk - 1):
        k_ref = np.zeros((B, H_kv, p.head_dim))
        v_ref = np.zeros_like(k_ref)
        for g in range(H_kv):
            sel_rows = np.nonzero((ids_h[:, g, :] == b).any(axis=1))[0]
            for r in sel_rows:
                toks, (_, dkr, dvr) = row_grads(int(r), g)
                m = (toks >= b * B) & (toks < (b + 1) * B)
                k_ref[toks[m] - b * B, g] += dkr[m]
                v_ref[toks[m] - b * B, g] += dvr[m]
        sl = slice(b * B, (b + 1) * B)
        sk = check_grad(dk[sl].float().cpu().numpy(), k_ref, f"dK block {b}")
        sv = check_grad(dv[sl].float().cpu().numpy(), v_ref, f"dV block {b}")
        _say(f"  block {b}: dK {sk[0]:.2e}/{sk[1]:.2e} dV {sv[0]:.2e}/{sv[1]:.2e} (max-err/max|ref|, rel-L2)")

    # identities over every key
    sum_dv = dv.double().sum(dim=0)                                   # (H_kv, d)
    sum_do = d["d_o"].double().view(p.total_q_rows, H_kv, G, p.head_dim).sum(dim=(0, 2))
    rel = float((sum_dv - sum_do).norm() / sum_do.norm())
    _say(f"  sum dV vs sum dO rel {rel:.2e}")
    assert rel < 1e-2
    sum_dk = dk.double().sum(dim=0)
    ratio = float(sum_dk.norm() / dk.double().abs().sum(dim=0).norm())
    _say(f"  |sum dK| / |sum |dK|| {ratio:.2e}")
    assert ratio < 1e-2
    del d, o, lse, dq, dk, dv, ids
    torch.cuda.empty_cache()


def test_backward_tile_wider_than_the_rank_bitmap():
    """One tile whose handles span more rows than the ordering kernel's LDS
    row bitmap covers (2^20): every row of a 1.2M-row sequence (one head, one
    group, k 2) selects block 0 besides its local block, so block 0's tile
    holds 1.2M handles over rows 0 .. 1.2M-1 and is put in canonical order by
    the merge fallback.  dK / dV must be equal bit for bit over three runs,
    dQ of sampled rows must match the oracle, and over all keys
    sum_j dV_j = sum_i dO_i and sum_j dK_j = 0 (every handle counted once)."""
    T, B = 1_200_000, 64
    p = synth.packed_problem("bwd_wide_tile", [T], [T], num_q_heads=1, num_kv_heads=1, topk=2, seed=77)
    _say("[case] bwd_wide_tile (1.2M rows, tile of block 0 spans every row)")
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = synth.generate_torch(p, dev, tensors=("q", "k", "v", "d_o"))
    lb = torch.arange(T, device=dev, dtype=torch.int32) // B
    ids = torch.stack([torch.zeros_like(lb), torch.where(lb > 0, lb, torch.full_like(lb, -1))], dim=1)
    ids = ids.view(T, 1, 2).contiguous()
    o, lse = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, B)
    runs = []
    for _ in range(3):
        runs.append(msa.sparse_attn_backward(d["q"], d["k"], d["v"], o, lse, d["d_o"], ids, seqs, B))
        torch.cuda.synchronize()
    for t in range(3):
        a = runs[0][t].view(torch.int16)
        assert all(torch.equal(a, r[t].view(torch.int16)) for r in runs[1:]), f"output {t} differs between runs"
    dq, dk, dv = runs[0]
    # dQ of sampled rows against the oracle
    lay = O.layout_of(p)
    ids_h = ids.cpu().numpy()
    scale = 1.0 / math.sqrt(p.head_dim)
    rows = [0, 63, 64, 1000, 524288, 1048575, 1048576, T - 1]
    dq_ref = np.zeros((len(rows), 1, p.head_dim))
    for i, r in enumerate(rows):
        s, pos = lay.locate(r)
        toks = O.selected_tokens(ids_h[r, 0], pos, B)
        tt = torch.from_numpy(toks).to(dev)
        dq_ref[i] = O.attend_backward(O.decode_bf16(from_dev_bits(d["q"][r])), O.decode_bf16(from_dev_bits(d["k"][tt, 0])),
                                      O.decode_bf16(from_dev_bits(d["v"][tt, 0])),
                                      O.decode_bf16(from_dev_bits(d["d_o"][r])), scale)[0]
    rows_t = torch.tensor(rows, dtype=torch.int64, device=dev)
    stats = check_grad(dq[rows_t].float().cpu().numpy(), dq_ref, "dQ sampled rows")
    _say(f"  dQ ({len(rows)} rows) max-err/max|ref| {stats[0]:.2e} rel-L2 {stats[1]:.2e}")
    rel = float((dv.double().sum(dim=0) - d["d_o"].double().sum(dim=0)).norm() / d["d_o"].double().sum(dim=0).norm())
    ratio = float(dk.double().sum(dim=0).norm() / dk.double().abs().sum(dim=0).norm())
    _say(f"  sum dV vs sum dO rel {rel:.2e}; |sum dK| / |sum |dK|| {ratio:.2e}")
    assert rel < 1e-2 and ratio < 1e-2
