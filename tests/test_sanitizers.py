"""The host side of libetc under AddressSanitizer and UndefinedBehaviorSanitizer
(host code only; device code is built as usual): the C ABI exercised over
many host-only plans (tests/sanitize/capi_host.cpp), and the copy tables'
tile walk (tests/tilewalk/tilewalk.cpp) replayed for the workloads, micro
models and random configurations.  Any report fails the test."""
import hashlib
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

import test_tile_walk as tw
from micro import MICRO_MODELS, cfg_pairs
from paper_2607_04749_amd.workloads import WORKLOADS
from randcfg import cases

ROOT = tw.ROOT
CSRC = tw.CSRC
# each host sanitizer flag right after -Xarch_host: device code is not instrumented
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
BASE = ["-x", "hip", "-O1", "-g", "-std=c++17", "--offload-arch=gfx950",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", CSRC]
ALL_SOURCES = ("plan.hip", "tiles.hip", "sketch.hip", "defrag.hip", "copy.hip", "cost.hip", "capi.hip")


def _build(name, main_src, lib_sources):
    h = hashlib.sha256()
    for f in [main_src] + [os.path.join(CSRC, x) for x in sorted(os.listdir(CSRC))]:
        with open(f, "rb") as fh:
            h.update(fh.read())
    out = os.path.join(ROOT, "_build", "sanitize", h.hexdigest()[:16], name)
    if not os.path.exists(out):
        os.makedirs(os.path.dirname(out), exist_ok=True)
        cmd = ["hipcc", *BASE, *SAN, main_src, *[os.path.join(CSRC, x) for x in lib_sources], "-o", out + ".tmp"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        os.replace(out + ".tmp", out)
    return out


@pytest.fixture(scope="module")
def binaries():
    jobs = {"capi_host": (os.path.join(ROOT, "tests", "sanitize", "capi_host.cpp"), ALL_SOURCES),
            "tilewalk": (tw.SRC, tw.LIB_SOURCES)}
    with ThreadPoolExecutor(2) as ex:
        futs = {k: ex.submit(_build, k, *v) for k, v in jobs.items()}
        return {k: f.result() for k, f in futs.items()}


def _env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0"  # the HIP runtime keeps some allocations to exit
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    return env


def test_capi_host_paths(binaries):
    r = subprocess.run([binaries["capi_host"]], capture_output=True, text=True, timeout=900, env=_env())
    assert r.returncode == 0 and "ok" in r.stdout, (r.stdout[-2000:], r.stderr[-4000:])
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]


def test_tile_walk_under_sanitizers(binaries):
    jobs = []
    for w in WORKLOADS.values():
        if w.name in ("llama-70b", "llama-13b", "llama-7b"):
            continue  # the large shares are replayed without sanitizers; keep this test short
        for refer in (False, True):
            jobs.append(tw._args(w.model, w.src, w.dst, refer, "sketch"))
    for m in MICRO_MODELS.values():
        for a, b in cfg_pairs(m)[::7]:
            jobs.append(tw._args(m, a, b, True, "identity"))
    for m, a, b in cases(16, base=0x5A17):
        jobs.append(tw._args(m, a, b, True, "sketch"))

    def one(args):
        return args, subprocess.run([binaries["tilewalk"], *args], capture_output=True, text=True,
                                    timeout=900, env=_env())
    bad = []
    with ThreadPoolExecutor(8) as ex:
        for args, r in ex.map(one, jobs):
            if r.returncode != 0 or r.stdout.strip() != "ok" or "runtime error" in r.stderr:
                bad.append((" ".join(args), r.stdout[-300:], r.stderr[-1500:]))
    assert not bad, bad[:2]
