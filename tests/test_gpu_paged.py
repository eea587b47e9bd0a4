"""Paged key side (block table) and multi-token decode rows.

A paged layout stores every key-side tensor (index_k, k, v) as a pool of
pages of 1-8 key blocks in shuffled order, with spare pages in between; key
j of sequence s sits in page block_table[s][j // page_size].  Kernels address keys one
block at a time and compute in the same order, so every result must equal
the contiguous layout's bit for bit; the contiguous results are checked
against the oracle (here for multi-token "speculative" decode rows, whose
positions are the chunked-prefill convention) and elsewhere.
"""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest
import torch

import oracle.msa_oracle as O
from paper_2606_13392_amd import msa, synth
from tests.util import check_block_ids, check_outputs, to_dev

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


def _paged_copy(p, x, dev, spare=7, seed=0, blocks_per_page=1):
    """Page pool + block table for problem p's key-side tensors x (numpy bits);
    pages of blocks_per_page key blocks."""
    P = p.block_size * blocks_per_page
    npg = [(L + P - 1) // P for L in p.kv_lens]
    npages = sum(npg) + spare
    perm = np.random.default_rng(seed).permutation(npages)
    table = np.zeros((p.num_seqs, max(npg)), dtype=np.int32)
    pool = {}
    for name in ("index_k", "k", "v"):
        shape = (npages * P,) + x[name].shape[1:]
        pool[name] = np.zeros(shape, dtype=x[name].dtype)
    used = 0
    for s in range(p.num_seqs):
        for g in range(npg[s]):
            page = int(perm[used])
            used += 1
            table[s, g] = page
            r0 = p.kv_starts[s] + g * P
            r1 = min(p.kv_starts[s] + p.kv_lens[s], r0 + P)
            for name in pool:
                pool[name][page * P:page * P + (r1 - r0)] = x[name][r0:r1]
    seqs = msa.Seqs(p.q_rows, p.kv_lens, [0] * p.num_seqs, npages * P, dev,
                    block_table=torch.from_numpy(table).to(dev), page_size=P)
    return pool, seqs


# name, q_rows, kv_lens, H_q, H_kv, block, topk, d_idx, kv_pad_to, blocks per page
CASES = [
    ("paged_decode", [1] * 6, [3000, 64, 65, 4097, 1, 900], 16, 4, 64, 6, 64, 4160, 1),
    ("paged_decode_4blk_pages", [1] * 6, [3000, 64, 65, 4097, 1, 900], 16, 4, 64, 6, 64, 4160, 4),
    ("paged_speculative_4", [4, 4, 4, 4], [5000, 4, 700, 2049], 16, 2, 64, 8, 64, 5120, 1),
    ("paged_speculative_mixed_bk128", [2, 8, 1, 3], [3000, 1500, 129, 4100], 32, 2, 128, 5, 128, 4224, 2),
    ("paged_chunked_prefill", [300, 1, 130], [2300, 800, 1500], 16, 2, 64, 8, 64, None, 1),
    ("paged_chunked_prefill_8blk_pages", [300, 1, 130], [2300, 800, 1500], 16, 2, 64, 8, 64, None, 8),
    # 128-key blocks scored as two 64-key sub-blocks in the many-row score kernel
    ("paged_chunked_prefill_bk128", [300, 1, 130], [2300, 800, 1500], 32, 2, 128, 5, 128, None, 2),
    ("paged_chunked_prefill_bk128_didx64", [300, 1, 130], [2300, 800, 1500], 16, 2, 128, 6, 64, None, 1),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_paged_matches_contiguous(case):
    name, q_rows, kv_lens, H_q, H_kv, bk, topk, d_idx, pad, bpp = case
    _say(f"[case] {name}")
    p = synth.packed_problem(name, q_rows, kv_lens, num_q_heads=H_q, num_kv_heads=H_kv, block_size=bk, topk=topk,
                             d_idx=d_idx, seed=zlib.crc32(name.encode()) % 10000, kv_pad_to=pad)
    x = synth.generate_numpy(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {t: to_dev(v) for t, v in x.items()}
    pool, pseqs = _paged_copy(p, x, dev, blocks_per_page=bpp)
    pd = {t: to_dev(v) for t, v in pool.items()}
    decode = p.max_q_rows <= 8
    attn = msa.sparse_attn_decode if decode else msa.sparse_attn_prefill
    ids = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    pids = msa.index_topk(d["index_q"], pd["index_k"], pseqs, p.block_size, p.topk)
    o, lse = attn(d["q"], d["k"], d["v"], ids, seqs, p.block_size)
    po, plse = attn(d["q"], pd["k"], pd["v"], pids, pseqs, p.block_size)
    torch.cuda.synchronize()
    assert torch.equal(ids, pids), "paged block ids differ from contiguous"
    assert torch.equal(o.view(torch.int16), po.view(torch.int16)) and torch.equal(lse, plse), \
        "paged attention differs from contiguous"
    # the contiguous results against the oracle
    lay = O.layout_of(p)
    ids_h = ids.cpu().numpy()
    ora_ids, gaps = O.select_blocks(x["index_q"], x["index_k"], lay, p.block_size, p.topk)
    exact, ties = check_block_ids(ids_h, ora_ids, gaps, x, lay, p.block_size, p.topk)
    o_ref, l_ref = O.sparse_attention(x["q"], x["k"], x["v"], ids_h, lay, p.block_size)
    st = check_outputs(o.float().cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref, name)
    _say(f"  ids exact {exact} ties {ties}; O max-abs {st[0]:.2e} rel-L2 {st[1]:.2e}")


def test_paged_fp8_decode_matches_contiguous():
    name = "paged_fp8"
    p = synth.packed_problem(name, [1] * 4, [2000, 70, 4096, 513], num_q_heads=16, num_kv_heads=4, topk=6,
                             seed=31, kv_pad_to=4096)
    x = synth.generate_fp8_numpy(p, synth.FP8_SCALES)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    pool, pseqs = _paged_copy(p, x, dev, seed=3)
    iq, ik = to_dev(x["index_q"]), to_dev(x["index_k"])
    ids = msa.index_topk(iq, ik, seqs, p.block_size, p.topk)
    q8 = torch.from_numpy(x["q"]).to(dev)
    o, lse = msa.sparse_attn_decode_fp8(q8, torch.from_numpy(x["k"]).to(dev), torch.from_numpy(x["v"]).to(dev),
                                        synth.FP8_SCALES, ids, seqs, p.block_size)
    po, plse = msa.sparse_attn_decode_fp8(q8, torch.from_numpy(pool["k"]).to(dev), torch.from_numpy(pool["v"]).to(dev),
                                          synth.FP8_SCALES, ids, pseqs, p.block_size)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), po.view(torch.int16)) and torch.equal(lse, plse)


def test_paged_rejections():
    p = synth.packed_problem("paged_rej", [1, 1], [100, 200], num_q_heads=8, num_kv_heads=2, topk=2, seed=5)
    x = synth.generate_numpy(p)
    dev = torch.device("cuda")
    pool, pseqs = _paged_copy(p, x, dev)
    L = msa.lib()
    # the page size must be the call's block size times a power of two
    assert L.msa_index_topk_workspace_size(pseqs.ref(), 2, 64, 128, 2) == 0
    assert L.msa_index_topk_workspace_size(pseqs.ref(), 2, 64, 64, 2) > 0
    pool3, pseqs3 = _paged_copy(p, x, dev, blocks_per_page=3)
    assert L.msa_index_topk_workspace_size(pseqs3.ref(), 2, 64, 64, 2) == 0
    # the dense baseline addresses keys as contiguous ranges and rejects a paged layout
    assert L.msa_dense_attn_workspace_size(pseqs.ref(), 8, 2, 128) == 0
    assert L.msa_sparse_attn_backward_workspace_size(pseqs.ref(), 8, 2, 128, 64, 2) > 0
    assert L.msa_sparse_kl_backward_workspace_size(pseqs.ref(), 8, 2, 64, 128, 64, 2) > 0
    assert L.msa_sparse_kl_backward_workspace_size(pseqs3.ref(), 8, 2, 64, 128, 64, 2) == 0
    assert L.msa_sparse_attn_prefill_workspace_size(pseqs.ref(), 8, 2, 128, 64, 2) > 0


# name, q_rows, kv_lens, H_q, H_kv, block, topk, d_idx, blocks per page
TRAIN_CASES = [
    ("paged_train_chunked", [300, 1, 130], [2300, 800, 1500], 16, 2, 64, 8, 64, 1),
    ("paged_train_4blk_pages", [700, 200], [700, 1900], 16, 4, 64, 6, 64, 4),
    ("paged_train_bk128", [300, 129], [2300, 1500], 32, 2, 128, 5, 128, 2),
]


@pytest.mark.parametrize("case", TRAIN_CASES, ids=[c[0] for c in TRAIN_CASES])
def test_paged_training_matches_contiguous(case):
    """The training calls on a paged key side: dQ, d index_q and the KL equal
    the contiguous layout's bit for bit, dK, dV and d index_k equal it row for
    row through the block table, and pool rows no sequence uses stay zero."""
    name, q_rows, kv_lens, H_q, H_kv, bk, topk, d_idx, bpp = case
    _say(f"[case] {name}")
    p = synth.packed_problem(name, q_rows, kv_lens, num_q_heads=H_q, num_kv_heads=H_kv, block_size=bk, topk=topk,
                             d_idx=d_idx, seed=zlib.crc32(name.encode()) % 10000)
    x = synth.generate_numpy(p)
    x_do = synth.generate_grad_numpy(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {t: to_dev(v) for t, v in x.items()}
    d_o = to_dev(x_do)
    pool, pseqs = _paged_copy(p, x, dev, blocks_per_page=bpp, seed=11)
    pd = {t: to_dev(v) for t, v in pool.items()}
    ids = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    o, lse = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, p.block_size)
    dq, dk, dv = msa.sparse_attn_backward(d["q"], d["k"], d["v"], o, lse, d_o, ids, seqs, p.block_size)
    pdq, pdk, pdv = msa.sparse_attn_backward(d["q"], pd["k"], pd["v"], o, lse, d_o, ids, pseqs, p.block_size)
    diq, dik, kl = msa.sparse_kl_backward(d["index_q"], d["index_k"], d["q"], d["k"], lse, ids, seqs, p.block_size)
    pdiq, pdik, pkl = msa.sparse_kl_backward(d["index_q"], pd["index_k"], d["q"], pd["k"], lse, ids, pseqs,
                                             p.block_size)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int16) if t.dtype == torch.bfloat16 else t
    assert torch.equal(bits(dq), bits(pdq)), "paged dQ differs"
    assert torch.equal(bits(diq), bits(pdiq)) and torch.equal(kl, pkl), "paged d index_q / KL differ"
    # key-side gradients: contiguous row kv_start + j <-> pool row of key j
    P = p.block_size * bpp
    table = pseqs.block_table.cpu().numpy()
    used = np.zeros(pool["k"].shape[0], dtype=bool)
    for s in range(p.num_seqs):
        for j0 in range(0, p.kv_lens[s], P):
            n = min(P, p.kv_lens[s] - j0)
            prow = int(table[s, j0 // P]) * P
            crow = p.kv_starts[s] + j0
            used[prow:prow + n] = True
            for a, b in ((dk, pdk), (dv, pdv), (dik, pdik)):
                assert torch.equal(bits(a[crow:crow + n]), bits(b[prow:prow + n])), f"paged key gradient differs, seq {s}"
    unused = torch.from_numpy(~used).to(dev)
    if bool(unused.any()):
        for t in (pdk, pdv, pdik):
            assert float(t[unused].float().abs().max()) == 0.0, "an unused pool row has a gradient"
    _say(f"  equal bit for bit; {int((~used).sum())} unused pool rows zero")
