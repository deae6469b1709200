"""The lane16 generator's bit-sliced vote counts (CPU): counts of several term lists started
together with shared full adders (one adder for three terms several lists hold, possibly all
complemented in some of them) and finished per list, emitted as C++ and run on random words
against a direct count of each list's terms.  Lists are drawn like the write's: the channel's
old value, shared plus terms and complemented minus terms, threshold = #minus + 1 (paper
Sec. 2.1: a cell becomes 1 iff old + #plus - #minus >= 1), and also arbitrary thresholds."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "codegen")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.fixture(scope="module")
def emitter(tmp_path_factory):
    if not os.path.exists(HIPCC) or shutil.which("g++") is None:
        pytest.skip("hipcc or g++ missing")
    d = tmp_path_factory.mktemp("share")
    exe = str(d / "share_emit")
    subprocess.run([HIPCC, "-std=c++17", "-O1", "-I", os.path.join(ROOT, "paper_2407_04221_amd", "csrc"),
                    "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "share_emit.cpp"), "-o", exe],
                   check=True, capture_output=True)
    return d, exe


@pytest.mark.parametrize("seed", list(range(1, 13)))
def test_shared_counts_match_direct_counts(emitter, seed):
    d, exe = emitter
    inc = subprocess.run([exe, str(seed)], check=True, capture_output=True, text=True).stdout
    work = d / f"s{seed}"
    work.mkdir()
    (work / "counts.inc").write_text("#include <cstdint>\ntypedef uint32_t u32;\n" + inc)
    chk = str(work / "check")
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", str(work), os.path.join(HERE, "share_check.cpp"),
                    "-o", chk], check=True, capture_output=True)
    r = subprocess.run([chk], capture_output=True, text=True)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


def test_shared_adders_are_shared(emitter):
    """Lists with many common terms take fewer adders together than one by one."""
    d, exe = emitter
    saved = 0
    for seed in range(1, 13):
        out = subprocess.run([exe, str(seed), "ops"], check=True, capture_output=True, text=True).stdout
        shared, alone = (int(x) for x in out.split())
        assert shared <= alone, (seed, shared, alone)
        saved += alone - shared
    assert saved > 0
