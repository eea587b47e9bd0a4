#!/usr/bin/env python
"""Benchmark of the MSA hot path on one MI355X.

A step is one pass of the prefill hot path over the workload: msa_index_topk
(index scores, causal block max, Top-k with the local block) followed by
msa_sparse_attn_prefill (block-sparse attention, O and LSE).  The default
workload is prefill at T = 1,048,576 tokens (64 query / 8 KV heads, head dim
128, index dim 64, block 64, k = 64, planted blocks); ``value`` is its
throughput in tokens/s.  A decode phase (64 sequences x 1 token at context
131,072, k = 32: msa_index_topk + msa_sparse_attn_decode) is timed after it and
reported under "decode" (with the same step on a paged copy of the caches
under "decode.paged"), and a training step of the attention at T = 32,768
(forward, msa_sparse_attn_backward, msa_sparse_kl_backward) under "training".

Inputs are drawn on the device before timing (synthetic, seeded) and stay
resident in HBM.  Each library call is bracketed by HIP events on the stream
it runs on, and the library's kernel timing (msa_profile_*) brackets each of
its kernels with events on that same stream during the timed steps.
``roofline`` describes the kernel with the largest time per step: its
algorithmic bytes or FLOPs per launch (models below) over its average launch
duration.  ``calls`` gives both calls' times; the attention call's effective
FLOPs (selected tokens only) over its time is the MFMA utilisation of the
Main Branch.  ``cpu_baseline`` times the CPU oracle on a bounded sample of
query rows of the same workload.  ``dense_baseline`` times our dense causal
GQA kernel (msa_dense_attn) on the same inputs: the last rows of the prefill
(extrapolated to all rows at the measured rate) and the whole decode step.

  python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MSA prefill tok/s @1M + decode tok/s @128K; % of MFMA / HBM peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- work models
def attended_tokens(ids, positions, block_size):
    """Per (row, group) number of causally visible tokens of the selected blocks."""
    import torch
    pos = positions.view(-1, 1, 1)
    start = ids.to(torch.int64) * block_size
    n = torch.clamp(torch.minimum(start + block_size, pos + 1) - start, min=0)
    n = torch.where(ids >= 0, n, torch.zeros_like(n))
    return n.sum(dim=-1)                     # [rows, H_kv]


def index_scored_keys(positions, block_size):
    """Keys scored by the Index Branch per row: every candidate block < local block."""
    import torch
    return (torch.div(positions, block_size, rounding_mode="floor") * block_size).to(torch.int64)


# ---------------------------------------------------------------- timing
class CallTimer:
    def __init__(self):
        self.ms = []

    def time(self, fn):
        import torch
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        out = fn()
        b.record()
        self._pending = (a, b)
        self.ms.append((a, b))
        return out

    def mean_ms(self, skip=0):
        vals = [a.elapsed_time(b) for a, b in self.ms[skip:]]
        return sum(vals) / max(1, len(vals))


def run_prefill(args, dev):
    import torch
    from paper_2606_13392_amd import msa, synth
    p = synth.workload(args.workload)
    log(f"[bench] generating {p.name}: {p.description}")
    d = synth.generate_torch(p, dev)
    seqs = msa.Seqs.from_problem(p, dev)
    H_q, H_kv, dh = p.num_q_heads, p.num_kv_heads, p.head_dim
    ids = torch.empty((p.total_q_rows, H_kv, p.topk), dtype=torch.int32, device=dev)
    o = torch.empty((p.total_q_rows, H_q, dh), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((p.total_q_rows, H_q), dtype=torch.float32, device=dev)
    ws_i = torch.empty(msa.index_topk_workspace_size(seqs, H_kv, p.d_idx, p.block_size, p.topk),
                       dtype=torch.uint8, device=dev)
    ws_a_n = msa.sparse_attn_prefill_workspace_size(seqs, H_q, H_kv, dh, p.block_size, p.topk)
    ws_a = torch.empty(max(ws_a_n, 1), dtype=torch.uint8, device=dev)
    t_idx, t_att = CallTimer(), CallTimer()

    def step():
        t_idx.time(lambda: msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk,
                                          out=ids, workspace=ws_i))
        t_att.time(lambda: msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, p.block_size,
                                                   out=o, lse=lse, workspace=ws_a))

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    msa.profile_reset()
    msa.profile_enable(True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    msa.profile_enable(False)
    kernels = msa.profile_read()
    log(f"[bench] timed {args.steps} prefill steps in {t1 - t0:.3f} s")
    sec = (t1 - t0) / args.steps
    ms_idx = t_idx.mean_ms(skip=args.warmup)
    ms_att = t_att.mean_ms(skip=args.warmup)

    positions = torch.from_numpy(p.positions()).to(dev)
    toks = attended_tokens(ids, positions, p.block_size)
    pos3 = positions.view(-1, 1, 1)
    incidences = float(((ids >= 0) & (ids.to(torch.int64) * p.block_size <= pos3)).sum().item())
    scored_keys = float(index_scored_keys(positions, p.block_size).sum().item())
    topk_bytes = topk_read_bytes(positions, p)
    eff_flops = 4.0 * dh * (H_q // H_kv) * float(toks.sum().item())
    idx_flops = 2.0 * p.d_idx * H_kv * scored_keys
    paper_main = 4.0 * H_q * dh * p.total_q_rows * p.topk * p.block_size
    dense = dense_prefill_baseline(args, p, d, dev) if not args.no_dense else None
    fp8 = prefill_fp8(args, p, seqs, ids, dev) if args.fp8 else None
    res = {
        "fp8": fp8,
        "dense": dense,
        "workload": p,
        "sec": sec,
        "ms_idx": ms_idx,
        "ms_att": ms_att,
        "eff_flops": eff_flops,
        "idx_flops": idx_flops,
        "paper_main_flops": paper_main,
        "kernels": {k: {"launches_per_step": n / args.steps, "ms_per_step": ms / args.steps,
                        "ms_per_launch": ms / n} for k, (n, ms) in kernels.items()},
        "models": kernel_models(p, incidences, scored_keys, eff_flops, idx_flops, topk_bytes),
        "inputs": d,
        "ids": ids,
    }
    return res


def prefill_fp8(args, p, seqs, ids, dev):
    """msa_sparse_attn_prefill_fp8 on E4M3 codes of fresh N(0,1) draws (same
    shapes, same block ids): the attention call's time and kernels."""
    import torch
    from paper_2606_13392_amd import msa, synth
    x = synth.generate_torch(p, dev, tensors=("q", "k", "v"), fp8_scales=synth.FP8_SCALES)
    ws = torch.empty(max(1, msa.sparse_attn_prefill_workspace_size(seqs, p.num_q_heads, p.num_kv_heads, p.head_dim,
                                                                   p.block_size, p.topk)), dtype=torch.uint8, device=dev)
    o = torch.empty((p.total_q_rows, p.num_q_heads, p.head_dim), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((p.total_q_rows, p.num_q_heads), dtype=torch.float32, device=dev)
    call = lambda: msa.sparse_attn_prefill_fp8(x["q"], x["k"], x["v"], synth.FP8_SCALES, ids, seqs, p.block_size,
                                               out=o, lse=lse, workspace=ws)
    call()
    torch.cuda.synchronize()
    msa.profile_reset()
    msa.profile_enable(True)
    t = CallTimer()
    for _ in range(2):
        t.time(call)
    torch.cuda.synchronize()
    msa.profile_enable(False)
    kern = msa.profile_read()
    ms = t.mean_ms()
    del x, ws, o, lse
    torch.cuda.empty_cache()
    log(f"[bench] fp8 attention call {ms:.1f} ms")
    return {"ms_per_call": ms, "kernels_ms_per_call": {k: v[1] / 2 for k, v in kern.items()}}


def dense_prefill_baseline(args, p, d, dev):
    """Our dense causal GQA kernel (msa_dense_attn) on the same inputs.

    The full causal pass at T = 1M is ~1.8e16 FLOP, so by default only the last
    ``--dense-rows`` query rows are run (a chunked-prefill layout over the whole
    context: the most expensive rows) and the full time is extrapolated at the
    measured TFLOP/s; ``--dense-rows 0`` runs every row."""
    import torch
    from paper_2606_13392_amd import msa
    T = p.total_q_rows
    S = T if args.dense_rows <= 0 else min(args.dense_rows, T)
    seqs = msa.Seqs([S], [p.kv_lens[0]], [p.kv_starts[0]], p.total_kv_rows, dev) if p.num_seqs == 1 else None
    if seqs is None:
        return None
    q = d["q"][T - S:]
    o = torch.empty_like(q)
    lse = torch.empty((S, p.num_q_heads), dtype=torch.float32, device=dev)
    ws = torch.empty(max(1, msa.dense_attn_workspace_size(seqs, p.num_q_heads, p.num_kv_heads, p.head_dim)),
                     dtype=torch.uint8, device=dev)
    msa.dense_attn(q, d["k"], d["v"], seqs, out=o, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    msa.dense_attn(q, d["k"], d["v"], seqs, out=o, lse=lse, workspace=ws)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b)
    L = p.kv_lens[0]
    pos_sum = lambda lo, hi: (hi - lo) * (lo + hi + 1) / 2.0        # sum of (position + 1) over [lo, hi)
    slice_flops = 4.0 * p.num_q_heads * p.head_dim * pos_sum(L - S, L)
    full_flops = 4.0 * p.num_q_heads * p.head_dim * pos_sum(L - T, L)
    tflops = slice_flops / (ms * 1e-3) / 1e12
    del o, lse, ws
    log(f"[bench] dense baseline: {S} rows in {ms:.1f} ms ({tflops:.0f} TFLOP/s)")
    k0 = p.kv_starts[0]
    sdpa = torch_sdpa_reference(q, d["k"][k0:], d["v"][k0:], L, slice_flops)
    return {"rows_timed": S, "ms_timed": ms, "tflops": tflops, "frac_of_bf16_peak": tflops / PEAK_BF16_TFLOPS,
            "flops_full": full_flops, "ms_full": ms * full_flops / slice_flops,
            "full_is": "measured" if S == T else "extrapolated from the timed rows at the same TFLOP/s",
            "torch_sdpa_flash": sdpa}


def torch_sdpa_reference(q, k, v, L, flops):
    """torch's own flash attention (scaled_dot_product_attention restricted to
    its FLASH_ATTENTION backend, GQA) on the same dense rows, for context: the
    S query rows at the end of an L-key context as a non-causal pass over the
    keys before them plus a causal S x S square (the same FLOPs as the dense
    kernel's causal rows).  Timing only; None values and the error when the
    backend cannot run the shapes."""
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel
    S = q.shape[0]
    try:
        qh = q.permute(1, 0, 2).unsqueeze(0).contiguous()
        kh = k[:L].permute(1, 0, 2).unsqueeze(0).contiguous()
        vh = v[:L].permute(1, 0, 2).unsqueeze(0).contiguous()
        kp, vp, ks, vs = kh[:, :, :L - S], vh[:, :, :L - S], kh[:, :, L - S:], vh[:, :, L - S:]
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            def run():
                F.scaled_dot_product_attention(qh, kp, vp, enable_gqa=True)
                F.scaled_dot_product_attention(qh, ks, vs, is_causal=True, enable_gqa=True)
            run()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            run()
            b.record()
            torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        del qh, kh, vh, kp, vp, ks, vs
        torch.cuda.empty_cache()
        tflops = flops / (ms * 1e-3) / 1e12
        log(f"[bench] torch SDPA (flash backend) on the same rows: {ms:.1f} ms ({tflops:.0f} TFLOP/s)")
        return {"ms_timed": ms, "tflops": tflops, "frac_of_bf16_peak": tflops / PEAK_BF16_TFLOPS}
    except Exception as e:                      # a context figure only: never fails the bench
        torch.cuda.empty_cache()
        return {"ms_timed": None, "tflops": None, "error": f"{type(e).__name__}: {str(e)[:200]}"}


def topk_read_bytes(positions, p):
    """The least a pruned Top-k must move per step: per (row, group) the
    piece maxima (one per 16 candidate blocks), the scores of the k-1 pieces
    that at least reach the bound (all candidates when there are fewer), and
    the k ids written."""
    import torch
    lb = torch.clamp(torch.div(positions, p.block_size, rounding_mode="floor"), min=0).to(torch.int64)
    per_row = (lb + 15) // 16 + torch.clamp(lb, max=16 * (p.topk - 1))
    return float(4 * p.num_kv_heads * (per_row.sum().item() + p.topk * positions.numel()))


def kernel_models(p, incidences, scored_keys, eff_flops, idx_flops, topk_bytes):
    """Algorithmic work per step of the prefill kernels: (bound, amount, unit).

    An incidence is one valid (query row, group, selected block).  The
    key-block-outer attention reads each key block's K and V once per group and,
    per incidence, gathers the G query rows and writes a bf16 partial O plus its
    fp32 LSE (Sec. 4.2 IO analysis, KV-outer): its intensity, about 2/3 B_k
    FLOP/B, sits far below MI355X's bf16 ridge (2.5 PFLOP/s / 8 TB/s = 312), so
    it is HBM-bound.  The combine reads every partial and writes O and LSE.
    Index scoring is an MFMA contraction; Top-k reads the piece maxima and the
    pieces that reach its bound (topk_read_bytes)."""
    G = p.num_q_heads // p.num_kv_heads
    d, T, H_kv, H_q = p.head_dim, p.total_q_rows, p.num_kv_heads, p.num_q_heads
    kv_bytes = 4.0 * H_kv * float(sum(p.kv_lens)) * d
    attn_bytes = kv_bytes + incidences * (4.0 * G * d + 4.0 * G + 4.0)
    comb_bytes = incidences * (2.0 * G * d + 4.0 * G) + T * H_q * (2.0 * d + 4.0) + T * H_kv * p.topk * 4.0
    score_blocks = scored_keys / p.block_size * H_kv          # block scores written and read back
    return {
        "kvo_attn_kernel": ("hbm", attn_bytes, "bytes"),
        "kvo_combine_kernel": ("hbm", comb_bytes, "bytes"),
        "index_block_max_lds_kernel": ("mfma", idx_flops, "flops"),
        "index_block_max_wave_kernel": ("mfma", idx_flops, "flops"),
        "index_topk_kernel": ("hbm", topk_bytes, "bytes"),
        "index_topk_split_kernel": ("hbm", score_blocks * 4.0 + T * H_kv * p.topk * 4.0, "bytes"),
        "index_topk_rows_kernel": ("hbm", score_blocks * 4.0 + T * H_kv * p.topk * 4.0, "bytes"),
    }


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary
    (profiles/hbm_traffic_*.md), or None when there is none for this kernel and
    workload or the kernel's source has changed since the counters were taken."""
    import glob
    import hashlib
    for f in sorted(glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic_*.md"))):
        for line in open(f):
            if not line.startswith("<!-- traffic: "):
                continue
            rec = json.loads(line[len("<!-- traffic: "):].rsplit("-->", 1)[0])
            if rec.get("kernel") != kernel or rec.get("workload") != workload:
                continue
            h = hashlib.sha256()
            for rel in rec["sources"]:
                src = os.path.join(ROOT, rel)
                if not os.path.exists(src):
                    return None
                h.update(open(src, "rb").read())
            if h.hexdigest() != rec["sources_sha256"]:
                return None
            return float(rec["bytes_per_launch"])
    return None


def roofline_of(pre):
    """Roofline object of the kernel with the largest time per step."""
    kern = pre["kernels"]
    if not kern:
        return None
    return roofline_for(pre, max(kern, key=lambda k: kern[k]["ms_per_step"]))


def roofline_for(pre, name):
    """Roofline object of one prefill kernel: its algorithmic work per launch
    over its event-timed launch duration, against the bound's peak."""
    k = pre["kernels"][name]
    out = {"kernel": name, "ms_per_launch": k["ms_per_launch"], "launches_per_step": k["launches_per_step"],
           "traffic": measured_traffic(name, pre["workload"].name)}
    model = pre["models"].get(name)
    if model is None:
        out.update({"bound": None, "achieved": None, "peak": None, "unit": None, "frac": None})
        return out
    bound, amount, what = model
    per_launch = amount / k["launches_per_step"]
    if bound == "hbm":
        achieved = per_launch / (k["ms_per_launch"] * 1e-3) / 1e9
        out.update({"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": achieved / PEAK_HBM_GBS, "algorithmic_bytes_per_launch": per_launch})
    else:
        achieved = per_launch / (k["ms_per_launch"] * 1e-3) / 1e12
        out.update({"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / PEAK_BF16_TFLOPS, "algorithmic_flops_per_launch": per_launch})
    return out


def run_decode(args, dev):
    import torch
    from paper_2606_13392_amd import msa, synth
    p = synth.workload(args.decode_workload)
    log(f"[bench] generating {p.name}: {p.description}")
    d = synth.generate_torch(p, dev)
    seqs = msa.Seqs.from_problem(p, dev)
    H_q, H_kv, dh = p.num_q_heads, p.num_kv_heads, p.head_dim
    ids = torch.empty((p.total_q_rows, H_kv, p.topk), dtype=torch.int32, device=dev)
    o = torch.empty((p.total_q_rows, H_q, dh), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((p.total_q_rows, H_q), dtype=torch.float32, device=dev)
    ws_i = torch.empty(msa.index_topk_workspace_size(seqs, H_kv, p.d_idx, p.block_size, p.topk),
                       dtype=torch.uint8, device=dev)
    ws_a = torch.empty(max(1, msa.sparse_attn_decode_workspace_size(seqs, H_q, H_kv, dh, p.block_size, p.topk)),
                       dtype=torch.uint8, device=dev)
    t_idx, t_att = CallTimer(), CallTimer()

    def call_index():
        msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk, out=ids, workspace=ws_i)

    def call_attn():
        msa.sparse_attn_decode(d["q"], d["k"], d["v"], ids, seqs, p.block_size, out=o, lse=lse, workspace=ws_a)

    for _ in range(args.decode_warmup):
        call_index()
        call_attn()
    torch.cuda.synchronize()
    # step time: the two calls back to back, nothing else on the stream
    t0 = time.perf_counter()
    for _ in range(args.decode_steps):
        call_index()
        call_attn()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    sec = (t1 - t0) / args.decode_steps
    # per-call split, in a second pass with events around each call
    for _ in range(args.decode_steps):
        t_idx.time(call_index)
        t_att.time(call_attn)
    torch.cuda.synchronize()
    ref = (ids.clone(), o.clone(), lse.clone())      # the bf16 step's results (later legs reuse o / lse)
    fp8 = None
    if args.fp8:
        x8 = synth.generate_torch(p, dev, tensors=("q", "k", "v"), fp8_scales=synth.FP8_SCALES)

        def call_attn8():
            msa.sparse_attn_decode_fp8(x8["q"], x8["k"], x8["v"], synth.FP8_SCALES, ids, seqs, p.block_size,
                                       out=o, lse=lse, workspace=ws_a)

        for _ in range(args.decode_warmup):
            call_index()
            call_attn8()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.decode_steps):
            call_index()
            call_attn8()
        torch.cuda.synchronize()
        sec8 = (time.perf_counter() - t0) / args.decode_steps
        del x8
        torch.cuda.empty_cache()
        fp8 = {"ms_per_step": sec8 * 1e3, "value": p.total_q_rows / sec8, "unit": "tok/s"}
    dense = None
    if not args.no_dense:
        ws_d = torch.empty(max(1, msa.dense_attn_workspace_size(seqs, H_q, H_kv, dh)), dtype=torch.uint8, device=dev)
        msa.dense_attn(d["q"], d["k"], d["v"], seqs, out=o, lse=lse, workspace=ws_d)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.decode_steps):
            msa.dense_attn(d["q"], d["k"], d["v"], seqs, out=o, lse=lse, workspace=ws_d)
        torch.cuda.synchronize()
        dms = (time.perf_counter() - t0) / args.decode_steps * 1e3
        kv_bytes = 2.0 * float(sum(p.kv_lens)) * H_kv * dh * 2
        dense = {"ms_per_step": dms, "kv_bytes": kv_bytes, "hbm_gbs": kv_bytes / (dms * 1e-3) / 1e9,
                 "msa_speedup": dms / (sec * 1e3)}
        del ws_d
    paged = None
    if not args.no_paged:
        paged = run_decode_paged(p, d, seqs, *ref, args, dev)
        paged4 = run_decode_paged(p, d, seqs, *ref, args, dev, blocks_per_page=4)
    positions = torch.from_numpy(p.positions()).to(dev)
    toks = attended_tokens(ids, positions, p.block_size)
    scored = index_scored_keys(positions, p.block_size)
    rows = p.total_q_rows
    idx_bytes = float(scored.sum().item()) * p.d_idx * 2 + rows * H_kv * p.d_idx * 2 + rows * H_kv * p.topk * 4
    att_bytes = (float(toks.sum().item()) * dh * 2 * 2 + rows * H_q * dh * 2 * 2 + rows * H_q * 4
                 + rows * H_kv * p.topk * 4)
    out = {
        "workload": f"{p.name}: {p.description}",
        "value": rows / sec,
        "unit": "tok/s",
        "steps": args.decode_steps,
        "warmup": args.decode_warmup,
        "ms_per_step": sec * 1e3,
        "ms_index_topk": t_idx.mean_ms(),
        "ms_sparse_attn_decode": t_att.mean_ms(),
        "algorithmic_bytes_per_step": idx_bytes + att_bytes,
        "hbm_gbs": (idx_bytes + att_bytes) / sec / 1e9,
        "hbm_frac": (idx_bytes + att_bytes) / sec / 1e9 / PEAK_HBM_GBS,
        "index_gbs": idx_bytes / (t_idx.mean_ms() * 1e-3) / 1e9,
        "attn_gbs": att_bytes / (t_att.mean_ms() * 1e-3) / 1e9,
        "dense_baseline": dense,
        "paper_decode_speedup_h800": 7.6,
    }
    if paged is not None:
        for rec in (paged, paged4):
            rec["hbm_gbs"] = (idx_bytes + att_bytes) / (rec["ms_per_step"] * 1e-3) / 1e9
            rec["hbm_frac"] = rec["hbm_gbs"] / PEAK_HBM_GBS
        out["paged"] = paged
        out["paged_4_block_pages"] = paged4
    if fp8 is not None:
        # bytes of the step with 1-byte Q, K, V (index tensors stay bf16)
        att8 = (float(toks.sum().item()) * dh * 2 + rows * H_q * dh * (1 + 2) + rows * H_q * 4
                + rows * H_kv * p.topk * 4)
        fp8.update({"algorithmic_bytes_per_step": idx_bytes + att8,
                    "hbm_gbs": (idx_bytes + att8) / (fp8["ms_per_step"] * 1e-3) / 1e9})
        out["fp8"] = fp8
    del d
    return out


def run_training(args, dev):
    """One training step of an MSA layer's attention on the --train-workload
    shape: the forward (msa_index_topk + msa_sparse_attn_prefill, keeping O
    and LSE) and the backward (msa_sparse_attn_backward for an upstream dO,
    msa_sparse_kl_backward for the Index Branch's KL loss with
    grad_scale = 1 / (rows x H_kv))."""
    import torch
    from paper_2606_13392_amd import msa, synth
    p = synth.workload(args.train_workload)
    log(f"[bench] training step on {p.name}: {p.description}")
    d = synth.generate_torch(p, dev, tensors=("index_q", "index_k", "q", "k", "v", "d_o"))
    seqs = msa.Seqs.from_problem(p, dev)
    H_q, H_kv, dh = p.num_q_heads, p.num_kv_heads, p.head_dim
    rows = p.total_q_rows
    ids = torch.empty((rows, H_kv, p.topk), dtype=torch.int32, device=dev)
    o = torch.empty((rows, H_q, dh), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((rows, H_q), dtype=torch.float32, device=dev)
    dq, dk, dv = (torch.empty_like(d[t]) for t in ("q", "k", "v"))
    diq, dik = torch.empty_like(d["index_q"]), torch.empty_like(d["index_k"])
    kl = torch.empty((rows, H_kv), dtype=torch.float32, device=dev)
    ws = torch.empty(max(msa.index_topk_workspace_size(seqs, H_kv, p.d_idx, p.block_size, p.topk),
                         msa.sparse_attn_prefill_workspace_size(seqs, H_q, H_kv, dh, p.block_size, p.topk),
                         msa.sparse_attn_backward_workspace_size(seqs, H_q, H_kv, dh, p.block_size, p.topk),
                         msa.sparse_kl_backward_workspace_size(seqs, H_q, H_kv, p.d_idx, dh, p.block_size, p.topk)),
                     dtype=torch.uint8, device=dev)
    gscale = 1.0 / (rows * H_kv)
    timers = {n: CallTimer() for n in ("msa_index_topk", "msa_sparse_attn_prefill", "msa_sparse_attn_backward",
                                       "msa_sparse_kl_backward")}
    calls = {
        "msa_index_topk": lambda: msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk,
                                                 out=ids, workspace=ws),
        "msa_sparse_attn_prefill": lambda: msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, p.block_size,
                                                                   out=o, lse=lse, workspace=ws),
        "msa_sparse_attn_backward": lambda: msa.sparse_attn_backward(d["q"], d["k"], d["v"], o, lse, d["d_o"], ids,
                                                                     seqs, p.block_size, d_q=dq, d_k=dk, d_v=dv,
                                                                     workspace=ws),
        "msa_sparse_kl_backward": lambda: msa.sparse_kl_backward(d["index_q"], d["index_k"], d["q"], d["k"], lse, ids,
                                                                 seqs, p.block_size, grad_scale=gscale,
                                                                 d_index_q=diq, d_index_k=dik, kl=kl, workspace=ws),
    }
    for _ in range(args.warmup):
        for fn in calls.values():
            fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.train_steps):
        for fn in calls.values():
            fn()
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.train_steps
    msa.profile_reset()
    msa.profile_enable(True)
    for _ in range(args.train_steps):
        for n, fn in calls.items():
            timers[n].time(fn)
    torch.cuda.synchronize()
    prof = msa.profile_read()
    msa.profile_enable(False)
    loss = float(kl.double().mean())
    G, D = p.group_size, p.d_idx
    inc = int((ids >= 0).sum().item())
    # per-incidence algorithmic bytes of the two dominant backward kernels
    bwd_bytes = inc * (G * dh * 2 * 3 + G * 8)       # Q, dO gathers; bf16 dQ partial; LSE and D
    kl_bytes = inc * (G * (dh * 2 + 4) + D * 2 + D * 4 + 8)   # Q gather + LSE; index query; d q_idx partial; LSE_idx, KL
    kern = {n: {"launches_per_step": c / args.train_steps, "ms_per_step": ms / args.train_steps}
            for n, (c, ms) in prof.items()}
    out = {
        "workload": f"{p.name}: {p.description}",
        "value": rows / sec,
        "unit": "tok/s",
        "steps": args.train_steps,
        "ms_per_step": sec * 1e3,
        "calls": {n: {"ms_per_call": t.mean_ms()} for n, t in timers.items()},
        "kernels": kern,
        "incidences": inc,
        "kl_loss_mean": loss,
        "roofline": {},
    }
    for name, nbytes in (("bwd_kvo_kernel", bwd_bytes), ("kl_grad_kernel", kl_bytes)):
        if name in kern and kern[name]["ms_per_step"] > 0:
            gbs = nbytes / (kern[name]["ms_per_step"] * 1e-3) / 1e9
            out["roofline"][name] = {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                     "frac": gbs / PEAK_HBM_GBS, "algorithmic_bytes_per_launch": nbytes}
    del d, o, lse, dq, dk, dv, diq, dik, kl, ws, ids
    torch.cuda.empty_cache()
    return out


def run_decode_paged(p, d, seqs, ids_ref, o_ref, lse_ref, args, dev, blocks_per_page=1):
    """The decode step on a paged copy of the caches: every key-side tensor
    becomes a pool of pages (blocks_per_page key blocks each) in a seeded
    random order, read through a block table; checks the step reproduces the
    contiguous results bit for bit and times it the same way."""
    import torch
    from paper_2606_13392_amd import msa
    B = p.block_size * blocks_per_page                      # page rows
    nblk = [(L + B - 1) // B for L in p.kv_lens]
    npages = sum(nblk)
    g = torch.Generator(device="cpu")
    g.manual_seed(p.seed + 77)
    perm = torch.randperm(npages, generator=g).to(torch.int32)
    table = torch.zeros((p.num_seqs, max(nblk)), dtype=torch.int32)
    src_blocks = []
    used = 0
    for s_, n in enumerate(nblk):
        table[s_, :n] = perm[used:used + n]
        src_blocks.append(torch.arange(n, dtype=torch.int64) * B + p.kv_starts[s_])
        used += n
    src = torch.cat(src_blocks).to(dev)                      # first row of each source block
    dst = perm.to(torch.int64).to(dev)                       # its page
    pool = {}
    for name in ("index_k", "k", "v"):
        t = d[name]
        out = torch.empty((npages * B,) + tuple(t.shape[1:]), dtype=t.dtype, device=dev)
        rows = (src.view(-1, 1) + torch.arange(B, device=dev).view(1, -1)).clamp_max(t.shape[0] - 1)
        out.view(npages, B, -1)[dst] = t[rows.view(-1)].view(npages, B, -1)
        pool[name] = out
    pseqs = msa.Seqs(p.q_rows, p.kv_lens, [0] * p.num_seqs, npages * B, dev, block_table=table.to(dev),
                     page_size=B)
    B = p.block_size
    H_q, H_kv, dh = p.num_q_heads, p.num_kv_heads, p.head_dim
    ids = torch.empty_like(ids_ref)
    o = torch.empty_like(o_ref)
    lse = torch.empty_like(lse_ref)
    ws_i = torch.empty(msa.index_topk_workspace_size(pseqs, H_kv, p.d_idx, B, p.topk), dtype=torch.uint8,
                       device=dev)
    ws_a = torch.empty(max(1, msa.sparse_attn_decode_workspace_size(pseqs, H_q, H_kv, dh, B, p.topk)),
                       dtype=torch.uint8, device=dev)

    def step():
        msa.index_topk(d["index_q"], pool["index_k"], pseqs, B, p.topk, out=ids, workspace=ws_i)
        msa.sparse_attn_decode(d["q"], pool["k"], pool["v"], ids, pseqs, B, out=o, lse=lse, workspace=ws_a)

    for _ in range(args.decode_warmup):
        step()
    torch.cuda.synchronize()
    same = bool(torch.equal(ids, ids_ref) and torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
                and torch.equal(lse, lse_ref))
    t0 = time.perf_counter()
    for _ in range(args.decode_steps):
        step()
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t0) / args.decode_steps
    del pool, ws_i, ws_a
    torch.cuda.empty_cache()
    return {"ms_per_step": sec * 1e3, "value": p.total_q_rows / sec, "unit": "tok/s", "pages": npages,
            "page_rows": B * blocks_per_page, "bit_identical_to_contiguous": same}


# The paper's Top-k latency table (Sec. 4.1; H800, fp32 (N, B) inputs, unsorted
# outputs, median of 50 iterations): (N, B, k) -> torch.topk, TileLang, theirs, in us
PAPER_TOPK_US_H800 = {(131072, 1024, 16): (3970, 2864, 779), (131072, 2048, 32): (5378, 3630, 1991),
                      (524288, 4096, 16): (33810, 17779, 7880), (524288, 8192, 32): (57659, 26100, 21326)}


def run_topk_latency(args, dev):
    """msa_block_topk (the Top-k operator on its own) and torch.topk on the
    paper's table shapes, median of 50 individually event-timed calls after
    warm-up, as the paper measures."""
    import torch
    from paper_2606_13392_amd import msa, synth

    def median_us(fn, iters=50, warm=5):
        for _ in range(warm):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        t = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
        return t[len(t) // 2]

    rows = []
    for (N, B, k) in synth.TOPK_SHAPES:
        x = synth.topk_scores(N, B, seed=N + B + k, device=dev)
        out = torch.empty((N, k), dtype=torch.int32, device=dev)
        ours = median_us(lambda: msa.block_topk(x, k, out=out))
        ref = median_us(lambda: torch.topk(x, k, dim=1, sorted=False))
        p_torch, p_tl, p_ours = PAPER_TOPK_US_H800[(N, B, k)]
        rows.append({"N": N, "B": B, "k": k, "us": ours, "torch_topk_us": ref, "vs_torch_topk": ref / ours,
                     "score_read_gbs": N * B * 4 / (ours * 1e-6) / 1e9,
                     "hbm_frac": N * B * 4 / (ours * 1e-6) / 1e9 / PEAK_HBM_GBS,
                     "paper_h800_us": p_ours, "paper_h800_vs_torch": p_torch / p_ours,
                     "paper_h800_vs_tilelang": p_tl / p_ours})
        log(f"[bench] top-k N {N} B {B} k {k}: {ours:.1f} us (torch.topk {ref:.1f} us; paper H800 {p_ours} us)")
        del x, out
        torch.cuda.empty_cache()
    return {"inputs": "i.i.d. N(0,1) fp32 score rows (seeded, on the device)", "timing": "median of 50",
            "shapes": rows}


def cpu_baseline(pre, args):
    """The CPU oracle on a bounded sample of query rows spread evenly over
    depth (host cores); the full-problem time is extrapolated from it."""
    import numpy as np
    import torch
    import oracle.msa_oracle as O
    from paper_2606_13392_amd import synth
    p = pre["workload"]
    d = pre["inputs"]
    rows = synth.stratified_rows(p, args.cpu_sample_rows, seed=12345)
    to_np = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    # query-side rows the sample needs (np.zeros commits only the pages written)
    sel = torch.tensor(rows, device=d["q"].device)
    iq = np.zeros(tuple(d["index_q"].shape), dtype=np.uint16)
    iq[rows] = to_np(d["index_q"][sel])
    q = np.zeros(tuple(d["q"].shape), dtype=np.uint16)
    q[rows] = to_np(d["q"][sel])
    ik = to_np(d["index_k"])
    k = to_np(d["k"])
    v = to_np(d["v"])
    lay = O.layout_of(p)
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    cores = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    ids, _ = O.select_blocks(iq, ik, lay, p.block_size, p.topk, rows=rows, batch_rows=16)
    O.sparse_attention(q, k, v, ids, lay, p.block_size, rows=rows, block_ids_are_for_rows=True)
    dt = time.perf_counter() - t0
    full_s = dt * p.total_q_rows / len(rows)
    return {
        "value": len(rows) / dt,
        "unit": "tok/s",
        "cores": min(cores, blas_threads) if blas_threads > 1 else 1,
        "kind": "oracle",
        "sample": f"{len(rows)} query rows of {p.name} stratified over depth (one per equal band, plus the first "
                  f"two blocks' rows and the last row; all {p.num_kv_heads} groups, {p.num_q_heads} heads), "
                  f"index selection + sparse attention, fp64 numpy; {dt:.1f} s; host has {cores} cores, "
                  f"BLAS threads {blas_threads}",
        "extrapolated_full_s": full_s,
        "extrapolated_note": f"extrapolated: all {p.total_q_rows} rows at the sample's mean time per row",
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="prefill_1m")
    ap.add_argument("--decode-workload", default="decode_128k")
    ap.add_argument("--decode-steps", type=int, default=20)
    ap.add_argument("--decode-warmup", type=int, default=3)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-paged", action="store_true", help="skip the decode step on a paged KV cache")
    ap.add_argument("--train-workload", default="prefill_32k",
                    help="shape of the training step (forward + Main Branch backward + KL backward)")
    ap.add_argument("--train-steps", type=int, default=3)
    ap.add_argument("--no-train", action="store_true")
    ap.add_argument("--no-topk", action="store_true",
                    help="skip the Top-k operator on the paper's latency-table shapes")
    ap.add_argument("--cpu-sample-rows", type=int, default=300)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense causal GQA baseline")
    ap.add_argument("--no-fp8", dest="fp8", action="store_false",
                    help="skip the Main Branch on E4M3 Q/K/V (msa_sparse_attn_*_fp8), timed by default")
    ap.add_argument("--calib-copy-gib", type=float, default=0.0,
                    help="first run one in-place int32 add over this many GiB (reads and writes exactly "
                         "that much): the reference kernel for scaling HBM byte counters")
    ap.add_argument("--dense-rows", type=int, default=8192,
                    help="prefill rows the dense baseline runs (the last ones; 0 = all)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: the library runs the MSA hot path on one GPU; --gpus must be 1 "
              "(sharding across GPUs is not implemented)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_13392_amd import msa
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(2)
    msa.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.calib_copy_gib > 0:
        x = torch.zeros(int(args.calib_copy_gib * (1 << 30)) // 4, dtype=torch.int32, device=dev)
        x.add_(1)
        torch.cuda.synchronize()
        log(f"[bench] calibration: int32 add_ over {x.numel() * 4} bytes")
        del x
        torch.cuda.empty_cache()
    pre = run_prefill(args, dev)
    p = pre["workload"]
    sec = pre["sec"]
    att_tflops = pre["eff_flops"] / (pre["ms_att"] * 1e-3) / 1e12
    idx_tflops = pre["idx_flops"] / (pre["ms_idx"] * 1e-3) / 1e12
    line = {
        "metric": METRIC,
        "value": p.total_q_rows / sec,
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 inputs drawn on the device; planted index-key blocks)",
        "config": {"workload": p.name, "description": p.description, "T": p.total_q_rows,
                   "num_q_heads": p.num_q_heads, "num_kv_heads": p.num_kv_heads, "head_dim": p.head_dim,
                   "d_idx": p.d_idx, "block_size": p.block_size, "topk": p.topk},
        "roofline": roofline_of(pre),
        # the Main Branch call (msa_sparse_attn_prefill, incl. its reverse index and combine) on
        # selected-block FLOPs, against the dense bf16 MFMA peak
        "main_branch_frac_of_bf16_peak": att_tflops / PEAK_BF16_TFLOPS,
        "calls": {
            "msa_index_topk": {"ms_per_call": pre["ms_idx"], "algorithmic_flops": pre["idx_flops"],
                               "tflops": idx_tflops, "frac_of_bf16_peak": idx_tflops / PEAK_BF16_TFLOPS},
            "msa_sparse_attn_prefill": {"ms_per_call": pre["ms_att"], "effective_flops": pre["eff_flops"],
                                        "tflops": att_tflops, "frac_of_bf16_peak": att_tflops / PEAK_BF16_TFLOPS},
        },
        "kernels": pre["kernels"],
        "kernel_rooflines": {n: roofline_for(pre, n) for n in pre["kernels"] if n in pre["models"]},
        "fp8_attention": None if pre["fp8"] is None else dict(
            pre["fp8"], tflops=pre["eff_flops"] / (pre["fp8"]["ms_per_call"] * 1e-3) / 1e12,
            frac_of_bf16_peak=pre["eff_flops"] / (pre["fp8"]["ms_per_call"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS),
        "dense_baseline": None if pre["dense"] is None else dict(
            pre["dense"], msa_attention_speedup=pre["dense"]["ms_full"] / pre["ms_att"],
            msa_step_speedup=pre["dense"]["ms_full"] / (sec * 1e3), paper_prefill_speedup_h800=14.2),
        "main_branch_flops": {"effective": pre["eff_flops"], "paper_formula_4HqdhNkBk": pre["paper_main_flops"]},
    }
    ids = pre.pop("ids")
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(pre, args)
    del ids
    pre.pop("inputs")
    torch.cuda.empty_cache()
    if not args.no_decode:
        line["decode"] = run_decode(args, dev)
    if not args.no_train:
        line["training"] = run_training(args, dev)
    if not args.no_topk:
        line["topk_latency"] = run_topk_latency(args, dev)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
