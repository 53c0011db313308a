"""The oracle and the HIP path share nothing, and the product never reaches
the oracle: no include, import or link in either direction, the shared
generator holds no resharding arithmetic, and importing the product loads
neither the oracle nor any CPU fallback."""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2607_04749_amd")
ORACLE = os.path.join(ROOT, "oracle")


def _files(d, exts):
    for base, _, names in os.walk(d):
        if "__pycache__" in base:
            continue
        for n in names:
            if n.endswith(exts):
                yield os.path.join(base, n)


def _needed(lib):
    out = subprocess.run(["readelf", "-d", lib], capture_output=True, text=True, check=True).stdout
    return re.findall(r"\(NEEDED\)\s+Shared library: \[([^\]]+)\]", out)


def test_oracle_sources_use_libc_only():
    for f in _files(ORACLE, (".c", ".h")):
        text = open(f).read()
        includes = re.findall(r'#\s*include\s*[<"]([^>"]+)[>"]', text)
        assert all(re.fullmatch(r"std\w+\.h|string\.h|math\.h|limits\.h", i) for i in includes), (f, includes)
        assert "etc.h" not in text and "csrc" not in text


def test_product_never_names_the_oracle():
    for f in _files(PKG, (".py", ".hip", ".hpp", ".h", ".cpp")):
        text = open(f).read()
        assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), f
        assert not re.search(r"liboracle|oracle\.c|orc_", text), f
    for f in _files(os.path.join(ROOT, "include"), (".h",)):
        assert "oracle" not in open(f).read().lower(), f


def test_synth_holds_no_resharding_arithmetic():
    """The generator shared by both sides only maps (seed, kind, tensor,
    index) to a value: it names no layout, route, message or plan."""
    for f in _files(os.path.join(ROOT, "synth"), (".py", ".hip", ".h")):
        text = open(f).read()
        assert not re.search(r"^\s*(import|from)\s+(oracle|paper_2607_04749_amd)\b", text, re.M), f
        assert not re.search(r"#\s*include\s*\"(etc|etc_internal|route|plan)\.h", text), f


def test_libraries_do_not_link_each_other():
    libs = {"etc": os.path.join(PKG, "libetc.so"), "oracle": os.path.join(ORACLE, "liboracle.so"),
            "synth": os.path.join(ROOT, "synth", "libsynth.so")}
    for name, lib in libs.items():
        if not os.path.exists(lib):
            pytest.skip(f"{name} library not built")
    assert not any("etc" in n or "synth" in n or "hip" in n for n in _needed(libs["oracle"]))
    assert not any("oracle" in n or "synth" in n for n in _needed(libs["etc"]))
    assert not any("oracle" in n or "libetc" in n for n in _needed(libs["synth"]))


def test_importing_the_product_loads_no_oracle():
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2607_04749_amd import etc\n"
            "bad = [m for m in sys.modules if m == 'oracle' or m.startswith('oracle.')]\n"
            "maps = open('/proc/self/maps').read()\n"
            "print('BAD' if bad or 'liboracle' in maps else 'OK', 'libetc' in maps)\n") % ROOT
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.split() == ["OK", "True"], r.stdout
