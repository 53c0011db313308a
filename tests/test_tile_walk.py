"""The copy tables on the host, no GPU: tests/tilewalk/tilewalk.cpp replays the
copy kernels' sub-chunk walk over every launch the planner builds (pack,
unpack, Refer; all kinds and one kind at a time) and checks bounds,
alignment and exact write coverage.  Plans: the five
workloads, micro models, data parallelism with failed ranks, coalesced and
random configurations, under the identity pairing, the sketch and direct
Refer.  This is the check run on the CPU before a plan shape first runs on
the GPU."""
import hashlib
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd.workloads import WORKLOADS, Parallel as P
from randcfg import cases, medium_cases

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_04749_amd", "csrc")
SRC = os.path.join(ROOT, "tests", "tilewalk", "tilewalk.cpp")
LIB_SOURCES = ("plan.hip", "tiles.hip", "sketch.hip")


def _binary():
    h = hashlib.sha256()
    for f in [SRC] + [os.path.join(CSRC, x) for x in os.listdir(CSRC)]:
        with open(f, "rb") as fh:
            h.update(fh.read())
    out_dir = os.path.join(ROOT, "_build", "tilewalk", h.hexdigest()[:16])
    exe = os.path.join(out_dir, "tilewalk")
    if not os.path.exists(exe):
        os.makedirs(out_dir, exist_ok=True)
        cmd = ["hipcc", "-x", "hip", "-O2", "-std=c++17", "--offload-arch=gfx950",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", os.path.join(ROOT, "include"), "-I", CSRC, SRC,
               *[os.path.join(CSRC, x) for x in LIB_SOURCES], "-o", exe + ".tmp"]
        subprocess.run(cmd, check=True, capture_output=True)
        os.replace(exe + ".tmp", exe)
    return exe


@pytest.fixture(scope="module")
def tilewalk():
    return _binary()


def _args(model, a, b, refer, pairing, failed=()):
    if not isinstance(pairing, str):
        pairing = ",".join(str(int(x)) for x in pairing)
    return [*map(str, model.astuple()), str(a.tp), str(a.pp), str(a.dp), str(b.tp), str(b.pp),
            str(b.dp), "1" if refer else "0", pairing, *map(str, failed)]


def _run_all(exe, jobs):
    def one(args):
        r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=600)
        return args, r
    bad = []
    with ThreadPoolExecutor(8) as ex:
        for args, r in ex.map(one, jobs):
            if r.returncode != 0 or r.stdout.strip() != "ok":
                bad.append((" ".join(args), r.stdout[-300:], r.stderr[-300:]))
    assert not bad, bad[:3]
    return len(jobs)


def _oracle_sketch(m, a, b, failed=None):
    C = oracle.matrices(m, a, b, failed=failed)["cost"]
    sk = oracle.sketch(C)[0]
    return [int(p) if p >= 0 and C[d, p] < oracle.COST_INF else -1 for d, p in enumerate(sk)]


def test_workloads(tilewalk):
    jobs = []
    for w in WORKLOADS.values():
        for refer in (False, True):
            for pairing in ("identity", "sketch"):
                jobs.append(_args(w.model, w.src, w.dst, refer, pairing))
        jobs.append(_args(w.model, w.dst, w.src, False, "sketch"))
    assert _run_all(tilewalk, jobs) == 25


def test_micro_models(tilewalk):
    jobs = []
    for m in MICRO_MODELS.values():
        for a, b in cfg_pairs(m)[::3]:
            for refer in (False, True):
                jobs.append(_args(m, a, b, refer, "identity"))
                jobs.append(_args(m, a, b, refer, _oracle_sketch(m, a, b)))
    assert _run_all(tilewalk, jobs) > 100


def test_data_parallel_and_failures(tilewalk):
    m = MICRO_MODELS["llama_gqa"]
    jobs = []
    for a, b, failed in ((P(2, 1, 2), P(1, 2, 3), ()), (P(2, 1, 3), P(1, 2, 2), (1, 2)),
                         (P(2, 2, 2), P(4, 1, 1), (0, 5)), (P(1, 2, 3), P(1, 2, 1), (2,))):
        for refer in (False, True):
            jobs.append(_args(m, a, b, refer, "identity", failed))
            jobs.append(_args(m, a, b, refer, _oracle_sketch(m, a, b, list(failed)), failed))
    _run_all(tilewalk, jobs)


def test_coalesced_pairings(tilewalk):
    m = MICRO_MODELS["gpt"]
    jobs = []
    for a, b in ((P(1, 4), P(1, 2)), (P(2, 4), P(4, 4)), (P(2, 2, 2), P(4, 2, 1))):
        sk = np.array(_oracle_sketch(m, a, b), np.int32)
        for mode in (oracle.DEFRAG_OCCUPANCY, oracle.DEFRAG_EFFICIENCY):
            pl, _ = oracle.defrag(a.world, b.world, sk, mode=mode)
            co = np.where(pl < a.world, pl, -1)
            for refer in (False, True):
                jobs.append(_args(m, a, b, refer, co))
    _run_all(tilewalk, jobs)


def test_random_configurations(tilewalk):
    jobs = []
    for m, a, b in cases(48):
        jobs.append(_args(m, a, b, False, "identity"))
        jobs.append(_args(m, a, b, True, _oracle_sketch(m, a, b)))
    _run_all(tilewalk, jobs)


def test_medium_random_configurations(tilewalk):
    """Boxes of several tiles with ragged tails and odd widths (randcfg's
    medium shapes), under the identity pairing and the oracle's sketch with
    direct Refer."""
    jobs = []
    for m, a, b in medium_cases(48):
        jobs.append(_args(m, a, b, False, "identity"))
        jobs.append(_args(m, a, b, True, _oracle_sketch(m, a, b)))
    _run_all(tilewalk, jobs)


def test_contiguous_run_beyond_2_32_elements(tilewalk):
    """GPT, hidden 17, vocab 2^28 + 1: the embedding is one contiguous run of
    4,563,402,769 elements, cut into 2^31-element rows and a ragged remainder
    (the pack pads 7 elements after it)."""
    from paper_2607_04749_amd.workloads import GPT, ModelShape
    m = ModelShape(GPT, 2, 17, 1, 1, 8, 2 ** 28 + 1, 0, 1)
    jobs = []
    for b in (P(1, 1), P(1, 2)):
        for refer in (False, True):
            jobs.append(_args(m, P(1, 1), b, refer, "identity"))
    _run_all(tilewalk, jobs)


PLANTS = {
    # one-kind windows rounded down: the last tiles of a launch get no workgroup
    "windows rounded down": ("return (ntiles + kXcds * kKindWindows - 1) / (kXcds * kKindWindows);",
                             "return ntiles / (kXcds * kKindWindows) + (ntiles < kXcds * kKindWindows);"),
    # a sub-chunk one item short: the last vector or element of each sub-chunk is never copied
    "sub-chunk one item short": ("*hi = a + per < n ? a + per : n;", "*hi = a + per - 1 < n ? a + per - 1 : n;"),
}


@pytest.mark.parametrize("plant", sorted(PLANTS))
def test_replay_catches_a_planted_geometry_mistake(tmp_path, plant):
    """The replay is built against a copy of the kernels' geometry header with
    one mistake planted; it must then fail on Tiny GPT under either pairing,
    with and without direct Refer."""
    old, new = PLANTS[plant]
    src = open(os.path.join(CSRC, "copy_geom.hpp")).read()
    assert src.count(old) == 1
    (tmp_path / "copy_geom.hpp").write_text(src.replace(old, new))
    exe = str(tmp_path / "tilewalk")
    subprocess.run(["hipcc", "-x", "hip", "-O2", "-std=c++17", "--offload-arch=gfx950",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-I", str(tmp_path), "-I", os.path.join(ROOT, "include"), "-I", CSRC, SRC,
                    *[os.path.join(CSRC, x) for x in LIB_SOURCES], "-o", exe],
                   check=True, capture_output=True)
    w = WORKLOADS["tiny-gpt"]
    for args in (_args(w.model, w.src, w.dst, False, "identity"), _args(w.model, w.src, w.dst, True, "sketch")):
        r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=600)
        assert r.returncode != 0 and r.stdout.strip() != "ok", (plant, " ".join(args))
