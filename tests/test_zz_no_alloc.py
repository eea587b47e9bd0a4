"""msa_index_topk_noalloc (the entry point for callers that cannot allocate)
against msa_index_topk on the same inputs, through the C ABI (needs an
MI355X).  Block ids are integers, so the two must agree bit for bit; two
calls in a row, the second on a smaller input, so the second call runs on
the scratch array the first one left filled.  The first input needs more
scratch than the array holds and runs in several chunks."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from paper_2606_13392_amd import msa, synth
from tests.util import to_dev

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


# name, q_rows, kv_lens, H_kv, d_idx, block, topk, kv_pad_to; in call order,
# each smaller than the one before
CASES = [
    ("prefill_64k_h8", [65536], [65536], 8, 64, 64, 16, None),
    ("chunked_varlen", [130, 64, 1, 257], [700, 64, 900, 1500], 4, 64, 64, 6, None),
    ("decode_padded", [1, 1, 1], [3000, 65, 4097], 2, 128, 128, 5, 4160),
]


def _inputs(name, q_rows, kv_lens, H_kv, d_idx, bk, topk, pad, dev):
    p = synth.packed_problem(name, q_rows, kv_lens, num_q_heads=H_kv, num_kv_heads=H_kv, d_idx=d_idx,
                             block_size=bk, topk=topk, seed=77 + len(q_rows), kv_pad_to=pad)
    if p.total_q_rows > 8192:
        x = synth.generate_torch(p, dev, tensors=("index_q", "index_k"))
        iq, ik = x["index_q"], x["index_k"]
    else:
        x = synth.generate_numpy(p)
        iq, ik = to_dev(x["index_q"], dev), to_dev(x["index_k"], dev)
    return p, iq, ik


def test_noalloc_matches_workspace_call():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    msa.lib()
    for name, q_rows, kv_lens, H_kv, d_idx, bk, topk, pad in CASES:
        _say(f"[noalloc] {name}: rows {sum(q_rows)} H_kv {H_kv} d_idx {d_idx} B_k {bk} k {topk}")
        p, iq, ik = _inputs(name, q_rows, kv_lens, H_kv, d_idx, bk, topk, pad, dev)
        seqs = msa.Seqs.from_problem(p, dev)
        want = msa.index_topk(iq, ik, seqs, bk, topk)
        ws_needed = msa.index_topk_workspace_size(seqs, H_kv, d_idx, bk, topk)
        # the output starts as garbage so a missing write shows
        got = torch.full_like(want, 0x7EADBEEF)
        msa.index_topk_noalloc(iq, ik, seqs, bk, topk, got)
        torch.cuda.synchronize()
        a, b = got.cpu().numpy(), want.cpu().numpy()
        bad = int((a != b).sum())
        _say(f"[noalloc] {name}: workspace call needs {ws_needed} B (array {msa.NOALLOC_MAX_BYTES} B), "
             f"{a.size} ids, {bad} differ")
        assert bad == 0
        assert (a >= -1).all()
