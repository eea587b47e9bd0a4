"""Host-side helpers that need no GPU: the seeded random batch layouts the
parity sweeps draw, and the committed HBM-traffic records bench.py reads."""
import glob
import hashlib
import json
import os
import sys

import pytest

from paper_2606_13392_amd import synth
from tests.util import random_layouts

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("kw", [dict(), dict(pow2_groups=True),
                                dict(max_seqs=2, max_kv=60000, max_q=120, topk_range=(33, 65))])
def test_random_layouts_are_valid_and_seeded(kw):
    for seed in range(5):
        a = random_layouts(seed, 12, **kw)
        assert a == random_layouts(seed, 12, **kw)          # same seed, same layouts
        for c in a:
            q, kv = c["q_rows"], c["kv_lens"]
            assert len(q) == len(kv) >= 1 and sum(q) >= 1
            assert all(0 <= r <= k for r, k in zip(q, kv))
            g = c["H_q"] // c["H_kv"]
            assert c["H_q"] % c["H_kv"] == 0 and g <= 16
            if kw.get("pow2_groups"):
                assert g & (g - 1) == 0
            assert c["bk"] in (64, 128) and c["d_idx"] in (64, 128)
            lo, hi = kw.get("topk_range", (1, 33))
            assert lo <= c["topk"] < hi
            if c["pad"] is not None:
                assert c["pad"] % 64 == 0 and c["pad"] >= max(kv)
            p = synth.packed_problem(c["name"], q, kv, num_q_heads=c["H_q"], num_kv_heads=c["H_kv"],
                                     d_idx=c["d_idx"], block_size=c["bk"], topk=c["topk"], kv_pad_to=c["pad"])
            assert p.total_q_rows == sum(q)


def _records():
    out = []
    for f in sorted(glob.glob(os.path.join(ROOT, "profiles", "hbm_traffic_*.md"))):
        for line in open(f):
            if line.startswith("<!-- traffic: "):
                out.append(json.loads(line[len("<!-- traffic: "):].rsplit("-->", 1)[0]))
    return out


def test_traffic_records_are_well_formed_and_read_by_bench():
    recs = _records()
    assert {r["kernel"] for r in recs} >= {"kvo_attn_kernel", "index_block_max_lds_kernel"}
    sys.path.insert(0, ROOT)
    import bench
    for r in recs:
        assert r["workload"] == "prefill_1m" and r["bytes_per_launch"] > 0
        assert len(r["sources_sha256"]) == 64
        h = hashlib.sha256()
        for rel in r["sources"]:
            h.update(open(os.path.join(ROOT, rel), "rb").read())
        got = bench.measured_traffic(r["kernel"], r["workload"])
        # current sources: the record's bytes; changed sources: no traffic figure
        assert got == (float(r["bytes_per_launch"]) if h.hexdigest() == r["sources_sha256"] else None)


def test_bench_refuses_more_than_one_gpu():
    """bench.py runs one GPU: --gpus N > 1 exits with status 2 and a message,
    before touching a GPU."""
    import subprocess
    import sys
    from pathlib import Path
    root = Path(__file__).resolve().parents[1]
    res = subprocess.run([sys.executable, str(root / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                         timeout=120)
    assert res.returncode == 2
    assert "--gpus must be 1" in res.stderr
    assert res.stdout == ""
