"""Host side of bench.py, no GPU: runs on more than one GPU are refused with a
message, the committed HBM traffic record was taken on the copy kernel as it
is now, and the CPU-baseline leg (the oracle on a bounded sample) runs."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_04749_amd.workloads import WORKLOADS  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_record_matches_the_kernel():
    """The committed traffic record covers every launch shape bench.py times
    (each mode of the 70B and 7B shares, and the 13B and 1.3B workloads),
    every entry carries the hash of the current copy-kernel sources, so
    bench.py reports it (a kernel change without new counters would make it
    null), and measured traffic is within 1 % of the algorithmic bytes."""
    with open(bench.TRAFFIC_FILE) as f:
        rec = json.load(f)
    kinds = {bench.launch_key("chunked", side, k) for side in ("pack", "unpack") for k in range(4)}
    need = {
        "llama-70b": {"direct/pack", "direct/unpack", "refer/refer", "refer/unpack", "coalesced/pack",
                      "coalesced/unpack", "failover/pack", "failover/unpack"} | kinds,
        "llama-7b": {"direct/pack", "direct/unpack", "refer/refer", "refer/unpack", "failover/pack",
                     "failover/unpack"} | kinds,
        "llama-13b": {"direct/pack", "direct/unpack", "refer/refer", "refer/pack"} | kinds,
        "gpt-1.3b": {"direct/pack", "direct/unpack"} | kinds,
    }
    for wl, keys in need.items():
        assert keys <= set(rec[wl]), (wl, keys - set(rec[wl]))
    for wl, launches in rec.items():
        for key, ent in launches.items():
            assert ent["kernel_hash"] == bench.kernel_hash(), (wl, key)
            assert bench.measured_traffic(wl, key) == ent["bytes_per_launch"]
            # within 1 % of the algorithmic bytes: nothing is fetched twice
            assert abs(ent["bytes_per_launch"] / ent["algorithmic_bytes"] - 1) < 0.01, (wl, key)


@pytest.mark.parametrize("pairing", ["identity", "sketch"])
def test_cpu_baseline_runs(pairing):
    out = bench.cpu_baseline(WORKLOADS["tiny-gpt"], pairing)
    assert out["kind"] == "oracle" and out["cores"] == min(16, bench.host_threads()) and out["unit"] == "GB/s"
    assert out["value"] > 0 and "layers 0-3" in out["sample"] and "on one thread" in out["sample"]
    assert "4-layer sample of the share, not the whole share" in out["sample"]


def test_oracle_threads_write_the_same_bytes():
    """cpu_baseline runs the oracle one tensor per thread: that must write
    exactly what one call over all tensors writes."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np
    import oracle
    from helpers import empty_arenas, host_arenas
    w = WORKLOADS["tiny-gpt"]
    m, a, b = w.model, w.src, w.dst
    hs = host_arenas(m, a, range(a.world), w.seed)
    outs = []
    for threaded in (False, True):
        hd = empty_arenas(m, b, range(b.world))
        hb = {s: np.zeros(oracle.send_layout(m, a, b, s)[3], np.uint8) for s in range(a.world)}
        if threaded:
            nt = len(oracle.tensors(m))
            with ThreadPoolExecutor(8) as ex:
                list(ex.map(lambda t: oracle.migrate(m, a, b, hs, hd, hb, t, t + 1), range(nt)))
        else:
            oracle.migrate(m, a, b, hs, hd, hb)
        outs.append((hd, hb))
    (d1, b1), (d2, b2) = outs
    for d in d1:
        for k in range(4):
            assert np.array_equal(d1[d][k], d2[d][k])
    for s in b1:
        assert np.array_equal(b1[s], b2[s])
