"""HIP path vs the CPU oracle through the C ABI (needs an MI355X).

Block ids: bit-exact wherever the oracle's score gap exceeds 1e-3, otherwise
a valid selection within that gap.  O / LSE: within 1e-2 max-abs and 5e-3
relative L2 of the float64 oracle, computed on the same block ids.
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
from tests.util import check_block_ids, check_outputs, from_dev_bits, random_layouts, to_dev

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


# name, q_rows, kv_lens, H_q, H_kv, d_idx, block, topk, kv_pad_to, planted
SMALL = [
    ("ragged_T200_k3", [200], [200], 8, 2, 64, 64, 3, None, 0),
    ("prefill_T1000_k8", [1000], [1000], 16, 2, 64, 64, 8, None, 0),
    ("k1_local_only", [300], [300], 8, 2, 64, 64, 1, None, 0),
    ("k_covers_all", [700], [700], 8, 4, 64, 64, 64, None, 0),
    ("chunked_varlen", [130, 64, 1, 257], [700, 64, 900, 1500], 16, 4, 64, 64, 6, None, 0),
    ("empty_seq_in_batch", [50, 0, 70], [50, 300, 500], 8, 2, 64, 64, 4, None, 0),
    ("decode_padded", [1, 1, 1, 1, 1], [3000, 64, 65, 4097, 1], 16, 4, 64, 64, 6, 4160, 0),
    ("bk128_didx128_g16", [600], [600], 32, 2, 128, 128, 5, None, 0),
    ("bk64_didx128_g8", [900], [900], 32, 4, 128, 64, 7, None, 0),
    ("bk128_didx64_g1", [520], [520], 8, 8, 64, 128, 4, None, 0),
    ("many_blocks_k32", [5000], [5000], 16, 2, 64, 64, 32, None, 0),
    ("planted_k16", [4096], [4096], 16, 8, 64, 64, 16, None, 6),
    # one reverse-index CTA covers 3 x 6250 key blocks: more than its LDS histogram holds
    ("wide_block_range", [100, 100, 100], [400000, 400000, 400000], 4, 1, 64, 64, 8, None, 0),
    # rows with more 64-block chunks than k-1: Top-k skips chunks below the
    # (k-1)-th largest chunk maximum
    ("pruned_topk_long_ctx", [300, 200], [100000, 60000], 4, 2, 64, 64, 8, None, 0),
    ("pruned_topk_k2", [150], [40000], 4, 2, 64, 64, 2, None, 0),
    ("pruned_topk_planted", [300], [70000], 8, 2, 64, 64, 12, None, 4),
    # at most one row group per sequence: units are sequences (an empty one
    # included), 16-wave Top-k per row
    ("seq_units_empty_and_multirow", [1, 0, 1, 3, 2], [500, 300, 4097, 64, 9000], 16, 4, 64, 64, 6, None, 0),
    ("seq_units_k32_long", [1, 1, 2], [131072, 70000, 20000], 8, 8, 64, 64, 32, 131072, 0),
]


def _problem(case):
    name, q_rows, kv_lens, H_q, H_kv, d_idx, bk, topk, pad, planted = case
    p = synth.packed_problem(name, q_rows, kv_lens, num_q_heads=H_q, num_kv_heads=H_kv, d_idx=d_idx,
                             block_size=bk, topk=topk, seed=zlib.crc32(name.encode()) % 10000, planted=planted,
                             kv_pad_to=pad)
    return p


# seeded random batch layouts: sequence counts and lengths, head groups,
# index dimension, block size, Top-k and key padding drawn together
RANDOM = [(c["name"], c["q_rows"], c["kv_lens"], c["H_q"], c["H_kv"], c["d_idx"], c["bk"], c["topk"], c["pad"], 0)
          for c in random_layouts(11, 10) + random_layouts(41, 5, max_seqs=2, max_kv=60000, max_q=120,
                                                           topk_range=(33, 65))]


@pytest.mark.parametrize("case", SMALL + RANDOM, ids=[c[0] for c in SMALL + RANDOM])
def test_small_end_to_end(case):
    p = _problem(case)
    _say(f"[case] {p.name}")
    x = synth.generate_numpy(p)
    lay = O.layout_of(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}

    ids_gpu = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    torch.cuda.synchronize()
    ids_gpu = ids_gpu.cpu().numpy()
    ids_ora, gaps = O.select_blocks(x["index_q"], x["index_k"], lay, p.block_size, p.topk)
    exact, ties = check_block_ids(ids_gpu, ids_ora, gaps, x, lay, p.block_size, p.topk)
    _say(f"  ids exact={exact} ties={ties}")

    # Main branch on the oracle's ids (both entry points) and on the GPU's ids.
    o_ref, l_ref = O.sparse_attention(x["q"], x["k"], x["v"], ids_ora, lay, p.block_size)
    ids_dev = torch.from_numpy(ids_ora).to(dev)
    for fn in (msa.sparse_attn_prefill, msa.sparse_attn_decode):
        o, l = fn(d["q"], d["k"], d["v"], ids_dev, seqs, p.block_size)
        torch.cuda.synchronize()
        stats = check_outputs(o.float().cpu().numpy(), l.cpu().numpy(), o_ref, l_ref, f"{p.name}/{fn.__name__}")
        _say(f"  {fn.__name__}: max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e} lse {stats[2]:.2e}")
    if ties:
        o_ref2, l_ref2 = O.sparse_attention(x["q"], x["k"], x["v"], ids_gpu, lay, p.block_size)
        o, l = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], torch.from_numpy(ids_gpu).to(dev), seqs,
                                       p.block_size)
        check_outputs(o.float().cpu().numpy(), l.cpu().numpy(), o_ref2, l_ref2, p.name + "/gpu-ids")


def test_deterministic():
    p = _problem(SMALL[1])
    x = synth.generate_numpy(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}
    a = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    b = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    oa, la = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], a, seqs, p.block_size)
    ob, lb = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], b, seqs, p.block_size)
    od, ld = msa.sparse_attn_decode(d["q"], d["k"], d["v"], a, seqs, p.block_size)
    od2, ld2 = msa.sparse_attn_decode(d["q"], d["k"], d["v"], a, seqs, p.block_size)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert torch.equal(oa.view(torch.int16), ob.view(torch.int16)) and torch.equal(la, lb)
    assert torch.equal(od.view(torch.int16), od2.view(torch.int16)) and torch.equal(ld, ld2)


def test_kernel_timing_records_launches():
    p = _problem(SMALL[1])
    x = synth.generate_numpy(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}
    ids0 = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    o0, _ = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids0, seqs, p.block_size)
    torch.cuda.synchronize()
    msa.profile_reset()
    msa.profile_enable(True)
    try:
        ids = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
        o, _ = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, p.block_size)
        torch.cuda.synchronize()
    finally:
        msa.profile_enable(False)
    rec = msa.profile_read()
    assert rec.get("kvo_attn_kernel", (0, 0.0))[0] >= 1
    assert rec.get("kvo_combine_kernel", (0, 0.0))[0] >= 1
    assert any(k.startswith("index_block_max") for k in rec)
    assert all(n >= 1 and ms > 0.0 for n, ms in rec.values())
    # timing changes nothing in the results
    assert torch.equal(ids, ids0) and torch.equal(o.view(torch.int16), o0.view(torch.int16))
    msa.profile_reset()
    assert msa.profile_read() == {}


def test_workspace_rejected_when_small():
    p = _problem(SMALL[1])
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    x = synth.generate_numpy(p)
    d = {k: to_dev(v) for k, v in x.items()}
    small = torch.empty(16, dtype=torch.uint8, device=dev)
    out = torch.full((p.total_q_rows, p.num_kv_heads, p.topk), 7, dtype=torch.int32, device=dev)
    st = msa.lib().msa_index_topk(d["index_q"].data_ptr(), d["index_k"].data_ptr(), seqs.ref(), p.num_kv_heads,
                                  p.d_idx, p.block_size, p.topk, out.data_ptr(), small.data_ptr(), 16,
                                  msa._stream())
    assert st == msa.MSA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 7).all())          # nothing was launched


def test_forward_small_workspaces_run_several_chunks():
    """Workspaces far below the one-chunk size: the index call runs its rows in
    many unit chunks and the attention call in several row chunks (reverse
    index, partials and combine per chunk).  Results equal the one-chunk run
    bit for bit and the oracle within the bars."""
    p = _problem(("chunked_ws_small", [130, 64, 1, 257, 700], [700, 64, 900, 1500, 2000], 16, 4, 64, 64, 6,
                  None, 0))
    _say(f"[case] {p.name}")
    x = synth.generate_numpy(p)
    lay = O.layout_of(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}
    ids0 = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    o0, l0 = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids0, seqs, p.block_size)
    z = _plan_sizes(p)
    ws_i = z["hdr"] + 2 * z["unit_bytes"]
    ws_a = z["fixed"] + 4 * 256 + (p.total_q_rows // 5) * z["prb"]
    idx_starts, attn_starts = _launch_row_starts(p, ws_i, ws_a)
    wi = torch.empty(ws_i, dtype=torch.uint8, device=dev)
    wa = torch.empty(ws_a, dtype=torch.uint8, device=dev)
    msa.profile_reset()
    msa.profile_enable(True)
    try:
        ids1 = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk, workspace=wi)
        o1, l1 = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids1, seqs, p.block_size, workspace=wa)
        torch.cuda.synchronize()
    finally:
        msa.profile_enable(False)
    rec = msa.profile_read()
    msa.profile_reset()
    n_topk = sum(rec.get(kn, (0, 0))[0] for kn in ("index_topk_kernel", "index_topk_split_kernel", "index_topk_rows_kernel"))
    n_comb = rec.get("kvo_combine_kernel", (0, 0))[0]
    _say(f"  launches: index {n_topk} (plan {len(idx_starts)}), attention {n_comb} (plan {len(attn_starts)})")
    assert n_topk == len(idx_starts) >= 3 and n_comb == len(attn_starts) >= 3
    assert torch.equal(ids0, ids1)
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16)) and torch.equal(l0, l1)
    ids_ora, gaps = O.select_blocks(x["index_q"], x["index_k"], lay, p.block_size, p.topk)
    ids_h = ids1.cpu().numpy()
    exact, ties = check_block_ids(ids_h, ids_ora, gaps, x, lay, p.block_size, p.topk)
    o_ref, l_ref = O.sparse_attention(x["q"], x["k"], x["v"], ids_h, lay, p.block_size)
    stats = check_outputs(o1.float().cpu().numpy(), l1.cpu().numpy(), o_ref, l_ref, p.name)
    _say(f"  ids exact={exact} ties={ties}; O max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e}")


# ---------------------------------------------------------------- workloads
def _sample_rows(p, n, seed):
    rng = np.random.default_rng(seed)
    T = p.total_q_rows
    rows = set(int(r) for r in rng.integers(0, T, size=n))
    for s in range(p.num_seqs):
        a, b = p.q_offsets[s], p.q_offsets[s + 1]
        if b > a:
            rows |= {a, b - 1, min(b - 1, a + 63), min(b - 1, a + 64)}
    return sorted(rows)


def _align(x, a=256):
    return (x + a - 1) // a * a


def _plan_sizes(p):
    """Sizes behind the two prefill calls' chunk plans (mirrored from the
    library): index call: row-group size qr, rows per unit U, units, header and
    bytes per unit; attention call: fixed bytes and bytes per chunk row."""
    S, T, H_kv, H_q, k, B = p.num_seqs, p.total_q_rows, p.num_kv_heads, p.num_q_heads, p.topk, p.block_size
    qr = 64 // H_kv
    mq = p.max_q_rows
    U = 8 if (mq > 4 * qr and p.d_idx == 64 and B == 64) else (4 if mq > 2 * qr else 1)
    seq_units = U == 1 and mq <= qr
    max_units = S if seq_units else (T // qr + S) // U + S
    bcap = _align(-(-p.max_kv_len // B), 4)
    cmcap = -(-bcap // 64) if U >= 4 else 0
    pcap = 4 * cmcap                      # the four 16-block piece maxima of each 64-block chunk
    unit_bytes = U * 64 * (bcap + cmcap + pcap) * 4
    hdr = _align(4 * (S + 1))
    ntile = H_kv * S * max(1, -(-p.max_kv_len // B))
    nscan = -(-ntile // 2048)
    fixed = (_align(8 * (S + 1)) + _align(4 * (ntile + 2)) + 2 * _align(4 * (ntile + 1)) + _align(8 * nscan))
    prb = 8 * H_kv * k + k * H_q * (128 * 2 + 4)
    return dict(qr=qr, U=U, seq_units=seq_units, max_units=max_units, unit_bytes=unit_bytes, hdr=hdr,
                fixed=fixed, prb=prb)


def _launch_row_starts(p, ws_index, ws_attn):
    """First packed row of every launch of the two prefill calls, mirroring
    their chunk plans: the index call scores units of U row groups (a row group
    is 64 / H_kv rows of one sequence) in chunks sized to its workspace; the
    attention call builds its reverse index and partials for chunks of rows
    sized to its workspace.  Returns (index starts, attention starts); callers
    compare their number with the launches made."""
    S, T, H_kv, H_q, k = p.num_seqs, p.total_q_rows, p.num_kv_heads, p.num_q_heads, p.topk
    z = _plan_sizes(p)
    qr, U, seq_units, max_units = z["qr"], z["U"], z["seq_units"], z["max_units"]
    chunk = min((ws_index - z["hdr"]) // z["unit_bytes"], max_units)
    unit_off = [0]
    for s in range(S):
        rows = p.q_offsets[s + 1] - p.q_offsets[s]
        groups = -(-rows // qr)
        unit_off.append(unit_off[-1] + (1 if seq_units else -(-groups // U)))
    idx = []
    for u0 in range(0, max_units, chunk):
        for s in range(S):
            if unit_off[s] <= u0 < unit_off[s + 1]:
                idx.append(p.q_offsets[s] + (u0 - unit_off[s]) * (1 if seq_units else U * qr))
                break
    fixed, prb = z["fixed"], z["prb"]

    def total(c):
        return (fixed + 2 * _align(4 * c * H_kv * k) + _align(2 * k * c * H_q * 128) + _align(4 * k * c * H_q))

    cr = T if total(T) <= ws_attn else (ws_attn - fixed - 4 * 256) // prb
    cr = min(cr, ((1 << 31) - 1) // (H_kv * k), 1 << 26)
    return idx, list(range(0, T, cr))


def _stratified_with_launch_edges(p, n, idx_starts, attn_starts):
    rows = set(synth.stratified_rows(p, n, seed=p.seed))
    for r in list(idx_starts) + list(attn_starts):
        rows |= {r, max(0, r - 1)}            # first row of a launch, last row of the one before
    return sorted(x for x in rows if 0 <= x < p.total_q_rows)


def _sampled_workload(name, n_rows, gen="numpy", check_attn_rows=None, stratified=False):
    p = synth.workload(name)
    _say(f"[case] {p.name} rows={p.total_q_rows} kv_rows={p.total_kv_rows}")
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    if gen == "numpy":
        x = synth.generate_numpy(p)
        d = {k: to_dev(v) for k, v in x.items()}
    else:
        d = synth.generate_torch(p, dev)
        x = None
    lay = O.layout_of(p)
    decode = p.max_q_rows == 1
    fn = msa.sparse_attn_decode if decode else msa.sparse_attn_prefill
    msa.profile_reset()
    msa.profile_enable(True)
    try:
        ids = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
        o, l = fn(d["q"], d["k"], d["v"], ids, seqs, p.block_size)
        torch.cuda.synchronize()
    finally:
        msa.profile_enable(False)
    launches = msa.profile_read()
    msa.profile_reset()
    if decode:
        rows = list(range(p.total_q_rows))
    elif stratified:
        ws_i = msa.index_topk_workspace_size(seqs, p.num_kv_heads, p.d_idx, p.block_size, p.topk)
        ws_a = msa.sparse_attn_prefill_workspace_size(seqs, p.num_q_heads, p.num_kv_heads, p.head_dim,
                                                      p.block_size, p.topk)
        idx_starts, attn_starts = _launch_row_starts(p, ws_i, ws_a)
        n_topk = sum(launches.get(kn, (0, 0))[0] for kn in ("index_topk_kernel", "index_topk_split_kernel", "index_topk_rows_kernel"))
        n_comb = launches.get("kvo_combine_kernel", (0, 0))[0]
        _say(f"  launches: index {n_topk} (plan {len(idx_starts)}), attention {n_comb} (plan {len(attn_starts)})")
        assert n_topk == len(idx_starts) and n_comb == len(attn_starts), "chunk plan mirror out of date"
        rows = _stratified_with_launch_edges(p, n_rows, idx_starts, attn_starts)
    else:
        rows = _sample_rows(p, n_rows, seed=p.seed)
    # the oracle reads the input rows it needs back from the (generated) inputs;
    # only sampled rows of the query-side tensors and outputs leave the device
    rows_t = torch.tensor(rows, dtype=torch.int64, device=dev)
    if x is not None:
        iq_h, ik_h = x["index_q"], x["index_k"]
    else:
        iq_h = np.zeros(tuple(d["index_q"].shape), dtype=np.uint16)
        iq_h[rows] = from_dev_bits(d["index_q"][rows_t])
        ik_h = from_dev_bits(d["index_k"])
    ids_gpu = ids[rows_t].cpu().numpy()
    ids_ora, gaps = O.select_blocks(iq_h, ik_h, lay, p.block_size, p.topk, rows=rows)
    inputs = {"index_q": iq_h, "index_k": ik_h}
    exact, ties = check_block_ids(ids_gpu, ids_ora, gaps, inputs, lay, p.block_size, p.topk, rows=rows)
    _say(f"  ids exact={exact} ties={ties} over {len(rows)} rows")
    # Main branch on sampled rows, oracle fed with the GPU's (validated) ids
    if check_attn_rows is None:
        arows = rows
    else:
        step = max(1, len(rows) // check_attn_rows)
        arows = sorted(set(rows[::step]) | {rows[0], rows[-1]})
    arows_t = torch.tensor(arows, dtype=torch.int64, device=dev)
    o_h = o[arows_t].float().cpu().numpy()
    l_h = l[arows_t].cpu().numpy()
    ids_a = ids[arows_t].cpu().numpy()
    G = p.group_size
    o_ref = np.zeros((len(arows), p.num_q_heads, p.head_dim))
    l_ref = np.zeros((len(arows), p.num_q_heads))
    for i, r in enumerate(arows):
        s, pos = lay.locate(r)
        kv0 = p.kv_starts[s]
        qb = from_dev_bits(d["q"][r])
        for g in range(p.num_kv_heads):
            idr = ids_a[i, g]
            toks = O.selected_tokens(idr, pos, p.block_size)
            tt = torch.from_numpy(kv0 + toks).to(dev)
            kb = from_dev_bits(d["k"][tt, g])
            vb = from_dev_bits(d["v"][tt, g])
            oo, ll = O.attend(O.decode_bf16(qb[g * G:(g + 1) * G]), O.decode_bf16(kb), O.decode_bf16(vb),
                              1.0 / math.sqrt(p.head_dim))
            o_ref[i, g * G:(g + 1) * G] = oo
            l_ref[i, g * G:(g + 1) * G] = ll
    stats = check_outputs(o_h, l_h, o_ref, l_ref, p.name)
    _say(f"  O max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e} lse {stats[2]:.2e} over {len(arows)} rows")
    del d, o, l, ids
    torch.cuda.empty_cache()
    return len(rows), len(arows)


def test_workload_prefill_4k():
    p = synth.workload("prefill_4k")
    _say(f"[case] {p.name}")
    x = synth.generate_numpy(p)
    lay = O.layout_of(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    d = {k: to_dev(v) for k, v in x.items()}
    ids = msa.index_topk(d["index_q"], d["index_k"], seqs, p.block_size, p.topk)
    o, l = msa.sparse_attn_prefill(d["q"], d["k"], d["v"], ids, seqs, p.block_size)
    torch.cuda.synchronize()
    ids_gpu = ids.cpu().numpy()
    ids_ora, gaps = O.select_blocks(x["index_q"], x["index_k"], lay, p.block_size, p.topk)
    exact, ties = check_block_ids(ids_gpu, ids_ora, gaps, x, lay, p.block_size, p.topk)
    o_ref, l_ref = O.sparse_attention(x["q"], x["k"], x["v"], ids_gpu, lay, p.block_size)
    stats = check_outputs(o.float().cpu().numpy(), l.cpu().numpy(), o_ref, l_ref, p.name)
    _say(f"  ids exact={exact} ties={ties}; O max-abs {stats[0]:.2e} rel-L2 {stats[1]:.2e}")


def test_workload_prefill_32k_sampled():
    _sampled_workload("prefill_32k", 160, check_attn_rows=64)


def test_workload_decode_128k():
    _sampled_workload("decode_128k", 64, gen="torch")


def test_workload_chunked_8x8k_sampled():
    # every launch of both calls: its first row and the last row of the launch
    # before; plus rows stratified over every sequence's depth
    n, na = _sampled_workload("chunked_8x8k", 1024, gen="torch", check_attn_rows=256, stratified=True)
    assert n >= 1024 and na >= 256


def test_workload_prefill_1m_sampled():
    # the full 1M-token prefill in the launch configuration bench.py times;
    # ids on >= 1024 rows stratified over depth plus the first and last row of
    # every index and attention launch, outputs on >= 256 of them
    n, na = _sampled_workload("prefill_1m", 700, gen="torch", check_attn_rows=256, stratified=True)
    assert n >= 1024 and na >= 256


def test_workload_prefill_1m_bk128_sampled():
    _sampled_workload("prefill_1m_bk128", 40, gen="torch", check_attn_rows=20)


def test_workload_decode_128k_bk128():
    _sampled_workload("decode_128k_bk128", 64, gen="torch")


# Exact score ties: the key blocks of the index repeat a few patterns (each
# row sees every block maximum many times over), or the index queries are
# zero (every score ties).  Equal scores keep the lower block id on both
# sides, so the ids must equal the oracle's exactly.  The cases reach every
# selection path of the Top-k: rows with at most k-1 candidates, rows ranked
# on their scores directly, rows pruned by piece maxima with a tie at the
# boundary, and rows whose tied candidates overflow the radix buffer (ranked
# by the pruned scan instead).
TIE_CASES = [
    # name, T, H_kv, topk, repeat period of the key blocks (0: zero index queries)
    ("ties_period5_k8", 16384, 2, 8, 5),
    ("ties_period40_k16", 30000, 2, 16, 40),
    ("ties_period3_k64", 80000, 1, 64, 3),
    ("ties_all_equal_k16", 20000, 2, 16, 0),
]


@pytest.mark.parametrize("case", TIE_CASES, ids=[c[0] for c in TIE_CASES])
def test_index_exact_ties(case):
    name, T, H_kv, topk, period = case
    _say(f"[ties] {name}")
    p = synth.packed_problem(name, [T], [T], num_q_heads=2 * H_kv, num_kv_heads=H_kv, d_idx=64, block_size=64,
                             topk=topk, seed=zlib.crc32(name.encode()) % 10000)
    x = synth.generate_numpy(p)
    iq, ik = x["index_q"].copy(), x["index_k"].copy()
    B = p.block_size
    if period:
        for b in range(period, T // B):
            ik[b * B:(b + 1) * B] = ik[(b % period) * B:(b % period + 1) * B]
    else:
        iq[:] = 0
    lay = O.layout_of(p)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    ids = msa.index_topk(to_dev(iq), to_dev(ik), seqs, B, topk)
    torch.cuda.synchronize()
    rows = synth.stratified_rows(p, 160, seed=3)
    ids_ora, _ = O.select_blocks(iq, ik, lay, B, topk, rows=rows)
    got = ids.cpu().numpy()[rows]
    bad = [(r, g) for i, r in enumerate(rows) for g in range(H_kv) if not np.array_equal(got[i, g], ids_ora[i, g])]
    _say(f"  {len(rows)} rows x {H_kv} groups, {len(bad)} differ")
    assert not bad, f"first differing (row, group) {bad[0]}: {got[rows.index(bad[0][0]), bad[0][1]]} vs oracle"


# Decode-shaped batches (one query row per sequence) with exact score ties
# among key blocks: name, sequences, context, H_kv, topk, repeat period of
# each sequence's key blocks (0: zero index queries, every score equal; -1:
# no repeats, the boundary cases of the kernel choice).  One wave per index
# row takes a Top-k of at most 33 over at most 8192 blocks with >= 64 rows;
# the all-equal rows overflow that wave's candidate buffer and are ranked
# again through the key batch.  16 waves share each row otherwise (k 34 and
# 64, fewer rows, longer rows).
DECODE_TIE_CASES = [                           # ..., the Top-k kernel the call must launch
    ("dec_ties_period7_k16", 64, 8192, 1, 16, 7, "rows"),
    ("dec_ties_period5_k32", 32, 65536 - 100, 2, 32, 5, "rows"),
    ("dec_ties_all_equal_k32", 16, 135000, 4, 32, 0, "rows"),
    ("dec_ties_period3_k64", 16, 100000, 2, 64, 3, "split"),
    ("dec_rows_k33_64rows", 32, 30000, 2, 33, -1, "rows"),
    ("dec_split_k34_64rows", 32, 30000, 2, 34, -1, "split"),
    ("dec_split_k33_32rows", 16, 30000, 2, 33, -1, "split"),
    ("dec_rows_8192_blocks", 8, 8192 * 64, 8, 16, -1, "rows"),
]


@pytest.mark.parametrize("case", DECODE_TIE_CASES, ids=[c[0] for c in DECODE_TIE_CASES])
def test_decode_index_exact_ties(case):
    name, nseq, ctx, H_kv, topk, period, kernel = case
    _say(f"[decode ties] {name}: {nseq} x 1 row at {ctx}, H_kv {H_kv}, k {topk}")
    p = synth.packed_problem(name, [1] * nseq, [ctx] * nseq, num_q_heads=2 * H_kv, num_kv_heads=H_kv, d_idx=64,
                             block_size=64, topk=topk, seed=zlib.crc32(name.encode()) % 10000)
    B = p.block_size
    rng = np.random.default_rng(p.seed)
    iq = rng.standard_normal((nseq, H_kv, 64), dtype=np.float32)
    ik = rng.standard_normal((nseq * ctx, 64), dtype=np.float32)
    if period > 0:
        for s in range(nseq):
            seq = ik[s * ctx:(s + 1) * ctx]
            pat = seq[:period * B].copy()
            reps = -(-ctx // (period * B))
            seq[:] = np.tile(pat, (reps, 1))[:ctx]
    elif period == 0:
        iq[:] = 0
    iq, ik = synth.bf16_bits_from_f32(iq), synth.bf16_bits_from_f32(ik)
    dev = torch.device("cuda")
    seqs = msa.Seqs.from_problem(p, dev)
    msa.profile_reset()
    msa.profile_enable(True)
    try:
        ids = msa.index_topk(to_dev(iq), to_dev(ik), seqs, B, topk)
        torch.cuda.synchronize()
    finally:
        msa.profile_enable(False)
    launched = msa.profile_read()
    msa.profile_reset()
    assert f"index_topk_{kernel}_kernel" in launched, f"expected the {kernel} Top-k kernel, launched {sorted(launched)}"
    lay = O.layout_of(p)
    ids_ora, gaps = O.select_blocks(iq, ik, lay, B, topk, rows=list(range(nseq)))
    got = ids.cpu().numpy()
    if period < 0:                   # random scores: the oracle's gap rule decides near-ties
        check_block_ids(got, ids_ora, gaps, {"index_q": iq, "index_k": ik}, lay, B, topk, list(range(nseq)))
        _say(f"  {nseq} rows x {H_kv} groups checked")
        return
    bad = [(r, g) for r in range(nseq) for g in range(H_kv) if not np.array_equal(got[r, g], ids_ora[r, g])]
    _say(f"  {nseq} rows x {H_kv} groups, {len(bad)} differ")
    assert not bad, f"first differing (row, group) {bad[0]}: {got[bad[0][0], bad[0][1]]} vs oracle"
