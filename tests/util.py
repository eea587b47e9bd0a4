"""Helpers shared by the GPU parity tests: upload of generated inputs and the
comparison rules (block ids: bit-exact where the oracle's score gap exceeds
the tolerance, otherwise a valid selection within that gap; outputs: max-abs
and relative-L2 bounds against the float64 oracle)."""
from __future__ import annotations

import numpy as np
import torch

import oracle.msa_oracle as O

GAP_TOL = 1e-3          # score gap below which several selections are correct
O_MAX_ABS = 1e-2        # outputs vs the fp64 oracle, on top of the output format's rounding
O_REL_L2 = 5e-3
# O is returned in bf16, which keeps 8 significant bits: rounding the exact
# result to the output format alone moves it by up to 2^-9 |O| (0.0078 at
# |O| = 4), so the element-wise bound is O_MAX_ABS + 2^-9 |O_ref|.
BF16_HALF_ULP_REL = 2.0 ** -9


def to_dev(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 bit patterns -> bf16 tensor on the device."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def from_dev_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def check_block_ids(gpu_ids, ora_ids, gaps, inputs, layout, block_size, topk, rows=None, tol=GAP_TOL):
    """Returns (exact rows, tie rows). Raises AssertionError on a violation."""
    rows = list(range(gpu_ids.shape[0])) if rows is None else list(rows)
    exact = ties = 0
    for i, r in enumerate(rows):
        for g in range(gpu_ids.shape[1]):
            a, b = gpu_ids[i, g], ora_ids[i, g]
            if np.array_equal(a, b):
                exact += 1
                continue
            assert gaps[i, g] <= tol, f"row {r} group {g}: ids differ with gap {gaps[i, g]}: {a} vs {b}"
            _, pos = layout.locate(r)
            sc = O.row_block_scores(inputs["index_q"], inputs["index_k"], layout, r, g, block_size)
            assert O.selection_is_valid(a, sc, pos, block_size, topk, tol), \
                f"row {r} group {g}: invalid tie selection {a} (oracle {b})"
            ties += 1
    return exact, ties


def check_outputs(o_gpu: np.ndarray, lse_gpu: np.ndarray, o_ref: np.ndarray, lse_ref: np.ndarray, what=""):
    o_gpu = o_gpu.astype(np.float64)
    err = np.abs(o_gpu - o_ref)
    rel = np.linalg.norm(o_gpu - o_ref) / max(np.linalg.norm(o_ref), 1e-30)
    lerr = np.abs(lse_gpu.astype(np.float64) - lse_ref)
    bound = O_MAX_ABS + BF16_HALF_ULP_REL * np.abs(o_ref)
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert (err <= bound).all(), \
        f"{what} O error {err[worst]:.3e} > bound {bound[worst]:.3e} at {worst} (max-abs {err.max():.3e})"
    assert rel <= O_REL_L2, f"{what} O rel-L2 {rel:.3e}"
    assert lerr.max() <= O_MAX_ABS, f"{what} LSE max-abs {lerr.max():.3e}"
    return float(err.max()), float(rel), float(lerr.max())


# Gradients of the training backward: each element is a sum of products in
# which one factor (P or dS) is rounded to bf16 for the MFMA (relative 2^-9),
# accumulated in fp32 and rounded once to bf16 on output (2^-9).  dQ and dK
# sum terms of both signs (the dS of a row sums to zero), so the error is
# bounded relative to the tensor's scale rather than to each element:
# |err| <= GRAD_MAX_ABS_REL * max|ref| + 2^-9 |ref| element-wise and
# relative L2 <= GRAD_REL_L2 per tensor.
GRAD_MAX_ABS_REL = 1e-2
GRAD_REL_L2 = 1e-2


def check_grad(got: np.ndarray, ref: np.ndarray, what=""):
    got = got.astype(np.float64)
    err = np.abs(got - ref)
    scale = max(float(np.abs(ref).max()), 1e-30)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    bound = GRAD_MAX_ABS_REL * scale + BF16_HALF_ULP_REL * np.abs(ref)
    worst = np.unravel_index(np.argmax(err - bound), err.shape)
    assert (err <= bound).all(), \
        f"{what} error {err[worst]:.3e} > bound {bound[worst]:.3e} at {worst} (max|ref| {scale:.3e})"
    assert rel <= GRAD_REL_L2, f"{what} rel-L2 {rel:.3e}"
    return float(err.max() / scale), float(rel)


def random_layouts(seed: int, n: int, *, max_seqs=4, max_kv=5000, max_q=300, pow2_groups=False, topk_range=(1, 33)):
    """``n`` seeded batch layouts for parity sweeps beyond the hand-picked cases.

    Each is a dict: per-sequence query rows and key lengths (queries are the
    last rows of their sequence, an empty sequence allowed), head counts, index
    dimension, block size, Top-k and, for about a third of them, a padded key
    stride. Sizes stay where the oracle finishes in seconds."""
    rng = np.random.default_rng(seed)
    groups = (1, 2, 4, 8, 16) if pow2_groups else (1, 2, 3, 4, 6, 8, 16)
    out = []
    for i in range(n):
        ns = int(rng.integers(1, max_seqs + 1))
        kv = [int(v) for v in rng.integers(1, max_kv + 1, ns)]
        q = [int(rng.integers(0, min(k, max_q) + 1)) for k in kv]
        if sum(q) == 0:
            q[0] = 1
        h_kv = int(rng.choice([1, 2, 4]))
        g = int(rng.choice(groups))
        bk = int(rng.choice([64, 128]))
        pad = None
        if rng.random() < 0.35:
            pad = ((max(kv) + 63) // 64 + int(rng.integers(0, 3))) * 64
        out.append(dict(name=f"rand{seed}_{i}", q_rows=q, kv_lens=kv, H_q=h_kv * g, H_kv=h_kv,
                        d_idx=int(rng.choice([64, 128])), bk=bk, topk=int(rng.integers(*topk_range)), pad=pad))
    return out
