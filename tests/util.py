"""Helpers shared by the GPU parity tests: upload of generated inputs and the
comparison rules (block ids: bit-exact where the oracle's score gap exceeds
the tolerance, otherwise a valid selection within that gap; outputs: max-abs
and relative-L2 bounds against the float64 oracle)."""
from __future__ import annotations

import numpy as np
import torch

import oracle.msa_oracle as O

GAP_TOL = 1e-3          # score gap below which several selections are correct
O_MAX_ABS = 1e-2        # outputs vs the fp64 oracle (the stated max-abs bar)
O_REL_L2 = 5e-3
BF16_HALF_ULP_REL = 2.0 ** -9

# Tally over a test session of output elements compared against the oracle
# and of those whose raw difference exceeds O_MAX_ABS (reported at the end of
# the session by tests/conftest.py).
OUTPUT_TALLY = {"elements": 0, "over": 0, "worst": 0.0, "calls": 0}


def bf16_rounding_interval(y: np.ndarray):
    """[lo, hi]: the real values that round (to nearest) to the bf16 values y
    (float32 arrays holding bf16 values exactly)."""
    y = np.ascontiguousarray(y, dtype=np.float32)
    b = (y.view(np.uint32) >> np.uint32(16)).astype(np.uint32)
    up = ((b + np.uint32(1)) << np.uint32(16)).view(np.float32).astype(np.float64)
    dn = ((b - np.uint32(1)) << np.uint32(16)).view(np.float32).astype(np.float64)
    yv = y.astype(np.float64)
    nb_lo, nb_hi = np.minimum(up, dn), np.maximum(up, dn)
    zero = (b & np.uint32(0x7FFF)) == 0
    lo = np.where(zero, 0.0, yv - (yv - nb_lo) / 2)
    hi = np.where(zero, 0.0, yv + (nb_hi - yv) / 2)
    return lo, hi


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
    """O within O_MAX_ABS of the oracle before the bf16 output rounding (the
    oracle's value lies within O_MAX_ABS of the set of reals that round to the
    kernel's bf16 output), relative L2 within O_REL_L2, LSE within O_MAX_ABS.
    The elements whose raw difference exceeds O_MAX_ABS (possible only where
    half a bf16 step adds to the arithmetic error) are counted and printed.
    Returns (max-abs, rel-L2, LSE max-abs, elements beyond
    O_MAX_ABS, their worst difference)."""
    o32 = np.asarray(o_gpu, dtype=np.float32)
    o64 = o32.astype(np.float64)
    err = np.abs(o64 - o_ref)
    rel = np.linalg.norm(o64 - o_ref) / max(np.linalg.norm(o_ref), 1e-30)
    lerr = np.abs(lse_gpu.astype(np.float64) - lse_ref)
    lo, hi = bf16_rounding_interval(o32)
    pre = np.maximum(np.maximum(lo - o_ref, o_ref - hi), 0.0)   # distance to the rounding interval
    worst = np.unravel_index(np.argmax(pre), pre.shape)
    assert (pre <= O_MAX_ABS).all(), \
        f"{what} O error before output rounding {pre[worst]:.3e} > {O_MAX_ABS} at {worst} " \
        f"(got {o64[worst]:.6f}, oracle {o_ref[worst]:.6f})"
    over = err > O_MAX_ABS
    n_over = int(over.sum())
    worst_over = float(err[over].max()) if n_over else 0.0
    if n_over:
        print(f"  {what}: {n_over} of {err.size} O elements beyond {O_MAX_ABS} (worst {worst_over:.4f}, "
              f"smallest |O| among them {float(np.abs(o_ref[over]).min()):.3f})", flush=True)
    assert rel <= O_REL_L2, f"{what} O rel-L2 {rel:.3e}"
    assert lerr.max() <= O_MAX_ABS, f"{what} LSE max-abs {lerr.max():.3e}"
    OUTPUT_TALLY["elements"] += int(err.size)
    OUTPUT_TALLY["over"] += n_over
    OUTPUT_TALLY["worst"] = max(OUTPUT_TALLY["worst"], worst_over)
    OUTPUT_TALLY["calls"] += 1
    return float(err.max()), float(rel), float(lerr.max()), n_over, worst_over


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
