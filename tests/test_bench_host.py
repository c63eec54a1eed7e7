"""Host-side logic of the benchmark, on the CPU: the multi-GPU refusal, the input-copy rotation
that keeps each timed step's K/V out of the caches, launch statistics, the counter records and the
oracle baseline's worker pool (run on a small decode batch against the oracle's own output)."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import oracle  # noqa: E402
from paper_2609_35158_amd import workloads  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_replicas_cover_a_gibibyte_between_uses():
    case = workloads.qwen3_8b_decode("cpu", batch=4, lo=64, hi=128)
    reps = bench.make_replicas(torch, case)
    per = bench.input_bytes(case)
    assert len(reps) >= 2 and (len(reps) - 1) * per >= bench.REPLICA_MIN_OTHER_BYTES
    assert (len(reps) - 2) * per < bench.REPLICA_MIN_OTHER_BYTES      # no more copies than needed
    for r in reps[1:]:
        for name in ("k_pool", "v_pool", "q", "k_new", "v_new"):
            a, b = getattr(case, name), getattr(r, name)
            assert a.data_ptr() != b.data_ptr() and torch.equal(a.view(torch.int16), b.view(torch.int16))
        assert r.block_table is case.block_table and np.array_equal(r.ctx_lens, case.ctx_lens)


def test_launch_stats():
    st = bench.launch_stats([3.0, 1.0, 2.0, 10.0])
    assert st == {"kernel_ms_median": 2.5, "kernel_ms_min": 1.0}


def test_counter_records_are_tied_to_the_kernel_source():
    data = json.load(open(os.path.join(ROOT, "profiles", "kernel_counters.json")))
    for e in data["entries"]:
        assert e["sources"] and all(os.path.exists(os.path.join(ROOT, f)) for f in e["sources"])
        assert 0 < e["sclk_mhz"] < 3000 and 0 <= e["mfma_busy"] <= 1
    assert bench.kernel_counters("attn_kernel<128>", "no-such-workload") is None
    # a record is used only while its sources still hash to its sha256
    import hashlib
    e = dict(data["entries"][0])
    h = hashlib.sha256()
    for f in e["sources"]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    e["sources_sha256"] = h.hexdigest()
    assert bench._record_current(e)
    e["sources_sha256"] = "0" * 64
    assert not bench._record_current(e)


def test_oracle_pool_baseline_and_parity():
    pool = bench.OraclePool(2)
    try:
        case = workloads.qwen3_8b_decode("cpu", batch=3, lo=100, hi=300)
        bits = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)
        kr, vr = oracle.kv_append(bits(case.k_pool), bits(case.v_pool), bits(case.k_new), bits(case.v_new),
                                  case.block_table.numpy(), case.ctx_lens, None)
        case.k_pool = torch.from_numpy(kr.view(np.int16)).view(torch.bfloat16)
        case.v_pool = torch.from_numpy(vr.view(np.int16)).view(torch.bfloat16)
        o, _ = oracle.attention(bits(case.q), kr, vr, case.block_table.numpy(), case.ctx_lens, None, case.scale)
        out = torch.from_numpy(o.astype(np.float32)).to(torch.bfloat16)
        cb, parity = bench.cpu_baseline(torch, case, out, 0.5, pool)
    finally:
        pool.close()
    assert cb["kind"] == "oracle" and cb["cores"] == 2 and cb["value"] > 0
    assert parity["sequences"] == 3 and parity["max_abs"] <= 1e-2
