"""The Top-k operator on its own (msa_block_topk) against the CPU oracle
through the C ABI (needs an MI355X).  Ids are integer results: bit-exact on
every row the oracle ranks; at the paper's full sizes every row is also
checked for a valid selection (ascending distinct ids, each selected score
>= every unselected one)."""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest
import torch

import oracle.msa_oracle as O
from paper_2606_13392_amd import msa, synth

pytestmark = pytest.mark.gpu

INF = float("inf")
POOL = [-INF, -3.0, -1.0, -0.0, 0.0, 0.25, 1.0, 2.0]


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


# name, rows, cols, k, row stride (None: cols), value pool (None: N(0, 1)), first column
SMALL = [
    ("k16_B1000", 37, 1000, 16, None, None, 0),
    ("k64_B64", 5, 64, 64, None, None, 0),
    ("k64_B63_fewer_cols_than_k", 9, 63, 64, None, None, 0),
    ("k1_B257", 100, 257, 1, None, None, 0),
    ("k32_B2048", 64, 2048, 32, None, None, 0),
    ("k48_B300_ragged_load", 40, 300, 48, None, None, 0),
    ("ties_k8_B300", 50, 300, 8, None, POOL, 0),
    ("ties_k64_B1000", 20, 1000, 64, None, POOL, 0),
    ("ties_k16_B5000", 8, 5000, 16, None, POOL, 0),
    ("stride_512_vector_loads", 33, 500, 16, 512, None, 0),
    ("stride_503_scalar_loads", 33, 500, 16, 503, None, 0),
    ("unaligned_start_scalar_loads", 17, 300, 12, 304, None, 1),
    ("one_row_B4097", 1, 4097, 20, None, None, 0),
    ("B3_k2", 6, 3, 2, None, POOL, 0),
    ("B0", 3, 0, 4, None, None, 0),
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: c[0])
def test_block_topk_small(case):
    name, n, B, k, ld, pool, off = case
    _say(f"[block_topk] {name}: rows {n} cols {B} k {k} stride {ld} first column {off}")
    dev = torch.device("cuda", torch.cuda.current_device())
    x = synth.topk_scores(n, off + B, seed=zlib.crc32(name.encode()), device=dev, ld=ld, pool=pool)[:, off:]
    got = msa.block_topk(x, k)
    torch.cuda.synchronize()
    want = O.row_topk(x.cpu().numpy(), k)
    assert np.array_equal(got.cpu().numpy(), want)


def test_block_topk_repeated_calls_agree():
    dev = torch.device("cuda", torch.cuda.current_device())
    x = synth.topk_scores(2000, 3000, seed=5, device=dev, pool=POOL)
    a = msa.block_topk(x, 32)
    b = msa.block_topk(x, 32)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("shape", synth.TOPK_SHAPES, ids=lambda s: f"N{s[0]}_B{s[1]}_k{s[2]}")
def test_block_topk_paper_shapes(shape):
    N, B, k = shape
    _say(f"[block_topk] paper shape N {N} B {B} k {k}")
    dev = torch.device("cuda", torch.cuda.current_device())
    x = synth.topk_scores(N, B, seed=N + B + k, device=dev)
    got = msa.block_topk(x, k)
    torch.cuda.synchronize()
    # the exact rule on ~1024 rows spread over the matrix, first and last included
    rng = np.random.default_rng(N + k)
    rows = np.unique(np.concatenate([[0, 1, N - 2, N - 1], rng.integers(0, N, size=1020)]))
    want = O.row_topk(x[torch.from_numpy(rows).to(dev)].cpu().numpy(), k)
    assert np.array_equal(got[torch.from_numpy(rows).to(dev)].cpu().numpy(), want)
    # every row: ascending distinct ids in range, selected scores dominate
    g = got.long()
    assert bool(((g >= 0) & (g < B)).all())
    assert bool((g[:, 1:] > g[:, :-1]).all())
    low = torch.gather(x, 1, g).amin(dim=1)
    x.scatter_(1, g, -INF)
    assert bool((low >= x.amax(dim=1)).all())
    _say(f"[block_topk] N {N}: {rows.size} rows exact, {N} rows valid")
