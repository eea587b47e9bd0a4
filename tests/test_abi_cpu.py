"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host before launching."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2606_13392_amd import msa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "msa.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(msa_[a-z0-9_]+)\s*\(", src)))


def test_header_matches_binding():
    assert _declared() == sorted(msa.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = msa.lib()
    for name in _declared():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", msa.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (msa_\w+)", out))
    assert set(_declared()) <= exported


def test_strerror():
    L = msa.lib()
    assert L.msa_strerror(0) == b"ok"
    assert L.msa_strerror(msa.MSA_ERR_WORKSPACE) == b"workspace too small"


def _seqs(**kw):
    base = dict(num_seqs=1, total_q_rows=100, total_kv_rows=100, max_q_rows=100, max_kv_len=100,
                q_offsets=8, kv_starts=8, kv_lens=8)   # fake non-null pointers, never dereferenced
    base.update(kw)
    return msa.MsaSeqsC(**base)


def test_workspace_queries_are_host_only():
    L = msa.lib()
    s = _seqs()
    n = L.msa_index_topk_workspace_size(ctypes.byref(s), 2, 64, 64, 8)
    # row groups of 64 / H_kv = 32 query rows; sequences longer than two groups
    # take units of 4 groups.  Each unit holds 4 x 64 index rows of
    # ceil(100/64) = 2 block scores rounded up to 4, one 64-block chunk
    # maximum and the four 16-block piece maxima of that chunk, fp32; plus the
    # unit table.
    groups = 100 // 32 + 1
    units = groups // 4 + 1
    assert n == 256 + units * 4 * 64 * (4 + 1 + 4) * 4
    # at most one row group per sequence: one unit per sequence, no chunk maxima
    s1 = _seqs(num_seqs=4, total_q_rows=4, max_q_rows=1)
    n1 = L.msa_index_topk_workspace_size(ctypes.byref(s1), 2, 64, 64, 8)
    assert n1 == 256 + 4 * 64 * 4 * 4
    # two row groups per sequence: units of one group, bounded by the groups
    s2 = _seqs(num_seqs=2, total_q_rows=100, max_q_rows=50)
    n2 = L.msa_index_topk_workspace_size(ctypes.byref(s2), 2, 64, 64, 8)
    assert n2 == 256 + (100 // 32 + 2 + 2) * 64 * 4 * 4
    # partials (bf16 O + fp32 LSE per slot, row, head) and the (row, group, slot) handles
    n = L.msa_sparse_attn_prefill_workspace_size(ctypes.byref(s), 8, 2, 128, 64, 8)
    assert n >= 8 * 100 * 8 * (128 * 2 + 4) + 100 * 2 * 8 * 4
    assert n < 2 * (8 * 100 * 8 * (128 * 2 + 4) + 100 * 2 * 8 * 4) + (1 << 16)
    assert L.msa_index_topk_workspace_size(ctypes.byref(s), 3, 64, 64, 8) == 0      # H_kv not a power of 2


BAD_INDEX = [
    (dict(), dict(H_kv=3), msa.MSA_ERR_UNSUPPORTED),
    (dict(), dict(d_idx=96), msa.MSA_ERR_UNSUPPORTED),
    (dict(), dict(bk=32), msa.MSA_ERR_UNSUPPORTED),
    (dict(), dict(topk=65), msa.MSA_ERR_UNSUPPORTED),
    (dict(), dict(topk=0), msa.MSA_ERR_INVALID),
    (dict(num_seqs=0), dict(), msa.MSA_ERR_INVALID),
    (dict(max_q_rows=200), dict(), msa.MSA_ERR_INVALID),      # more query rows than keys
    (dict(q_offsets=0), dict(), msa.MSA_ERR_INVALID),
    (dict(), dict(null_out=True), msa.MSA_ERR_INVALID),
    (dict(), dict(ws_bytes=8), msa.MSA_ERR_WORKSPACE),
]


@pytest.mark.parametrize("seq_kw,arg_kw,want", BAD_INDEX)
def test_index_topk_rejects(seq_kw, arg_kw, want):
    L = msa.lib()
    s = _seqs(**seq_kw)
    a = dict(H_kv=2, d_idx=64, bk=64, topk=8, null_out=False, ws_bytes=1 << 20)
    a.update(arg_kw)
    st = L.msa_index_topk(8, 8, ctypes.byref(s), a["H_kv"], a["d_idx"], a["bk"], a["topk"],
                          None if a["null_out"] else 8, 8, a["ws_bytes"], None)
    assert st == want


BAD_ATTN = [
    (dict(H_q=6, H_kv=4), msa.MSA_ERR_INVALID),
    (dict(d_h=64), msa.MSA_ERR_UNSUPPORTED),
    (dict(H_q=64, H_kv=2), msa.MSA_ERR_UNSUPPORTED),           # group of 32 heads
    (dict(bk=256), msa.MSA_ERR_UNSUPPORTED),
    (dict(topk=0), msa.MSA_ERR_INVALID),
    (dict(null_q=True), msa.MSA_ERR_INVALID),
]


@pytest.mark.parametrize("kind", ["prefill", "decode"])
@pytest.mark.parametrize("arg_kw,want", BAD_ATTN)
def test_sparse_attn_rejects(kind, arg_kw, want):
    L = msa.lib()
    s = _seqs()
    a = dict(H_q=8, H_kv=2, d_h=128, bk=64, topk=8, null_q=False)
    a.update(arg_kw)
    fn = getattr(L, f"msa_sparse_attn_{kind}")
    st = fn(None if a["null_q"] else 8, 8, 8, 8, ctypes.byref(s), a["H_q"], a["H_kv"], a["d_h"], a["bk"],
            a["topk"], 0.1, 8, 8, 8, 1 << 30, None)
    assert st == want


def test_profile_api_without_launches():
    # enabling, resetting and reading touch no device while nothing was launched
    L = msa.lib()
    assert L.msa_profile_enable(1) == 0
    assert L.msa_profile_reset() == 0
    n = ctypes.c_int64(-1)
    ms = ctypes.c_double(-1.0)
    assert L.msa_profile_read(b"no_such_kernel", ctypes.byref(n), ctypes.byref(ms)) == 0
    assert n.value == 0 and ms.value == 0.0
    assert L.msa_profile_read(b"no_such_kernel", None, ctypes.byref(ms)) != 0
    assert L.msa_profile_enable(0) == 0
    assert msa.profile_read() == {} or all(v[0] > 0 for v in msa.profile_read().values())


def _all_queries(L, s):
    r = ctypes.byref(s)
    return (L.msa_index_topk_workspace_size(r, 2, 64, 64, 8),
            L.msa_index_topk_workspace_size(r, 4, 128, 128, 16),
            L.msa_sparse_attn_prefill_workspace_size(r, 8, 2, 128, 64, 8),
            L.msa_sparse_attn_decode_workspace_size(r, 8, 2, 128, 64, 8),
            L.msa_dense_attn_workspace_size(r, 8, 2, 128),
            L.msa_sparse_attn_backward_workspace_size(r, 8, 2, 128, 64, 8),
            L.msa_sparse_kl_backward_workspace_size(r, 8, 2, 64, 128, 64, 8))


def _all_rejections(L, s):
    r = ctypes.byref(s)
    return (L.msa_index_topk(8, 8, r, 3, 64, 64, 8, 8, 8, 1 << 20, None),
            L.msa_index_topk(8, 8, r, 2, 64, 64, 8, None, 8, 1 << 20, None),
            L.msa_index_topk(8, 8, r, 2, 64, 64, 8, 8, 8, 8, None),
            L.msa_sparse_attn_prefill(8, 8, 8, 8, r, 6, 4, 128, 64, 8, 0.1, 8, 8, 8, 1 << 30, None),
            L.msa_sparse_attn_decode(8, 8, 8, 8, r, 8, 2, 64, 64, 8, 0.1, 8, 8, 8, 1 << 30, None),
            L.msa_strerror(msa.MSA_ERR_HIP))


def test_host_calls_from_many_threads():
    """Workspace queries and host-side rejections give the same answers when
    8 host threads make them at once (ctypes drops the GIL around each call)."""
    import threading
    L = msa.lib()
    layouts = [_seqs(), _seqs(num_seqs=4, total_q_rows=4, max_q_rows=1),
               _seqs(total_q_rows=5000, total_kv_rows=5000, max_q_rows=5000, max_kv_len=5000)]
    want = [(_all_queries(L, s), _all_rejections(L, s)) for s in layouts]
    errors = []

    def work(t):
        try:
            for it in range(300):
                i = (t + it) % len(layouts)
                got = (_all_queries(L, layouts[i]), _all_rejections(L, layouts[i]))
                if got != want[i]:
                    errors.append((t, it, got, want[i]))
                    return
        except Exception as e:   # surfaced below
            errors.append((t, repr(e)))

    threads = [threading.Thread(target=work, args=(t,)) for t in range(8)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert not errors, errors[:2]


def test_chunks_stay_within_the_handle_row_field():
    """A reverse-index handle keeps the row inside its chunk in 26 bits, so a
    chunk never exceeds 2^26 rows even where the workspace would allow more
    (one KV head, Top-k 1: H_kv * topk < 32).  Twice the rows then need no
    more workspace, since both plans use chunks of 2^26 rows (the backward
    also keeps D = dO . O for every row: 4 bytes per row and head)."""
    L = msa.lib()
    big = 1 << 27
    a = _seqs(total_q_rows=1 << 26, total_kv_rows=big, max_q_rows=1 << 26, max_kv_len=big)
    b = _seqs(total_q_rows=big, total_kv_rows=big, max_q_rows=big, max_kv_len=big)
    for fn, args, per_row in ((L.msa_sparse_attn_prefill_workspace_size, (1, 1, 128, 64, 1), 0),
                              (L.msa_sparse_attn_backward_workspace_size, (1, 1, 128, 64, 1), 4),
                              (L.msa_sparse_kl_backward_workspace_size, (1, 1, 64, 128, 64, 1), 0)):
        na, nb = fn(ctypes.byref(a), *args), fn(ctypes.byref(b), *args)
        assert na > 0 and nb > 0
        assert nb - na == per_row * (big - (1 << 26)), (fn.__name__, na, nb)


def test_noalloc_rejects_problems_beyond_its_scratch():
    """msa_index_topk_noalloc checks the problem against its fixed scratch on
    the host: a sequence of 4M keys needs more than the 64 MiB array for one
    unit of rows, so the call returns MSA_ERR_WORKSPACE before any HIP call;
    invalid arguments are rejected as msa_index_topk rejects them."""
    L = msa.lib()
    n = 1 << 22
    s = _seqs(total_q_rows=n, total_kv_rows=n, max_q_rows=n, max_kv_len=n)
    assert L.msa_index_topk_noalloc(8, 8, ctypes.byref(s), 8, 64, 64, 16, 8, None) == msa.MSA_ERR_WORKSPACE
    s = _seqs()
    assert L.msa_index_topk_noalloc(8, 8, ctypes.byref(s), 3, 64, 64, 8, 8, None) == msa.MSA_ERR_UNSUPPORTED
    assert L.msa_index_topk_noalloc(8, 8, ctypes.byref(s), 2, 64, 64, 8, None, None) == msa.MSA_ERR_INVALID
    assert L.msa_index_topk_noalloc(8, 8, ctypes.byref(s), 2, 64, 64, 0, 8, None) == msa.MSA_ERR_INVALID


def test_block_topk_rejects_on_the_host():
    L = msa.lib()
    assert L.msa_block_topk(8, 0, 100, 100, 16, 8, None) == msa.MSA_OK          # no rows: nothing to do
    assert L.msa_block_topk(8, 4, 100, 100, 0, 8, None) == msa.MSA_ERR_INVALID  # k < 1
    assert L.msa_block_topk(8, 4, 100, 100, 65, 8, None) == msa.MSA_ERR_UNSUPPORTED
    assert L.msa_block_topk(8, 4, 100, 99, 16, 8, None) == msa.MSA_ERR_INVALID  # ld < n_cols
    assert L.msa_block_topk(8, -1, 100, 100, 16, 8, None) == msa.MSA_ERR_INVALID
    assert L.msa_block_topk(8, 4, -1, 100, 16, 8, None) == msa.MSA_ERR_INVALID
    assert L.msa_block_topk(8, 4, 100, 100, 16, None, None) == msa.MSA_ERR_INVALID
    assert L.msa_block_topk(None, 4, 100, 100, 16, 8, None) == msa.MSA_ERR_INVALID
    assert L.msa_block_topk(8, 4, (1 << 30) + 1, 1 << 31, 16, 8, None) == msa.MSA_ERR_UNSUPPORTED
