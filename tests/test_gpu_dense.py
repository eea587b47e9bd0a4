"""Dense causal GQA baseline (msa_dense_attn) vs the oracle's dense attention.

Same bar as the sparse outputs: within 1e-2 (+ bf16 output rounding) max-abs
and 5e-3 relative L2 of the float64 oracle; LSE within 1e-2.
"""
from __future__ import annotations

import math
import sys
import zlib

import numpy as np
import pytest
import torch

import oracle.msa_oracle as O
from paper_2606_13392_amd import msa, synth
from tests.util import check_outputs, from_dev_bits, to_dev

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


# name, q_rows, kv_lens, H_q, H_kv, kv_pad_to
CASES = [
    ("dense_T1000_g8", [1000], [1000], 16, 2, None),
    ("dense_ragged_T333_g4", [333], [333], 8, 2, None),
    ("dense_g16", [300], [300], 32, 2, None),
    ("dense_g1", [200], [200], 8, 8, None),
    ("dense_chunked_varlen", [130, 0, 64, 5, 257], [700, 90, 64, 900, 1500], 16, 4, None),
    ("dense_decode_padded", [1, 1, 1, 1, 1], [3000, 64, 65, 4097, 1], 16, 4, 4160),
    ("dense_three_rows", [3, 2, 3], [500, 129, 2000], 8, 2, None),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_dense_small(case):
    name, q_rows, kv_lens, H_q, H_kv, pad = case
    p = synth.packed_problem(name, q_rows, kv_lens, num_q_heads=H_q, num_kv_heads=H_kv, topk=1,
                             seed=zlib.crc32(name.encode()) % 10000, kv_pad_to=pad)
    _say(f"[case] {name}")
    x = {k: v for k, v in synth.generate_numpy(p).items() if k in ("q", "k", "v")}
    lay = O.layout_of(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}
    o, l = msa.dense_attn(d["q"], d["k"], d["v"], seqs)
    torch.cuda.synchronize()
    o_ref, l_ref = O.dense_causal_attention(x["q"], x["k"], x["v"], lay)
    stats = check_outputs(o.float().cpu().numpy(), l.cpu().numpy(), o_ref, l_ref, name)
    _say(f"  O max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e} lse {stats[2]:.2e}")


def _dense_rows_ref(p, d, rows):
    """Oracle dense attention of selected rows, reading the needed inputs back."""
    lay = O.layout_of(p)
    G = p.group_size
    o_ref = np.zeros((len(rows), p.num_q_heads, p.head_dim))
    l_ref = np.zeros((len(rows), p.num_q_heads))
    for i, r in enumerate(rows):
        s, pos = lay.locate(r)
        kv0 = p.kv_starts[s]
        qb = from_dev_bits(d["q"][r])
        for g in range(p.num_kv_heads):
            kb = from_dev_bits(d["k"][kv0:kv0 + pos + 1, g])
            vb = from_dev_bits(d["v"][kv0:kv0 + pos + 1, g])
            oo, ll = O.attend(O.decode_bf16(qb[g * G:(g + 1) * G]), O.decode_bf16(kb), O.decode_bf16(vb),
                              1.0 / math.sqrt(p.head_dim))
            o_ref[i, g * G:(g + 1) * G] = oo
            l_ref[i, g * G:(g + 1) * G] = ll
    return o_ref, l_ref


@pytest.mark.parametrize("name,n_rows", [("prefill_32k", 12), ("decode_128k", 8)])
def test_dense_workload_sampled(name, n_rows):
    p = synth.workload(name)
    _say(f"[case] dense {name}")
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = synth.generate_torch(p, dev, tensors=("q", "k", "v"))
    o, l = msa.dense_attn(d["q"], d["k"], d["v"], seqs)
    torch.cuda.synchronize()
    rng = np.random.default_rng(p.seed)
    rows = sorted(set(int(r) for r in rng.integers(0, p.total_q_rows, size=n_rows)) | {0, p.total_q_rows - 1})
    o_ref, l_ref = _dense_rows_ref(p, d, rows)
    stats = check_outputs(o.float().cpu().numpy()[rows], l.cpu().numpy()[rows], o_ref, l_ref, name)
    _say(f"  O max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e} lse {stats[2]:.2e} over {len(rows)} rows")
