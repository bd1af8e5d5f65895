"""The C header is plain C99: a C program (tests/c/abi_host.c) built with
-std=c99 -pedantic -Werror against include/rhymeflow.h and linked to
librhymeflow.so runs the host-only calls; its printed results are checked
against the oracle. Skipped when no C compiler is available."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2606_06309_amd")


@pytest.fixture(scope="module")
def output(tmp_path_factory):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    if not os.path.exists(os.path.join(LIBDIR, "librhymeflow.so")):
        pytest.skip("library not built")
    exe = str(tmp_path_factory.mktemp("cabi") / "abi_host")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_host.c"),
                    "-L", LIBDIR, "-lrhymeflow", f"-Wl,-rpath,{LIBDIR}", "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    return {line.split()[0]: line.split()[1:] for line in r.stdout.splitlines()}


def test_keyframe_sets(output):
    assert output["abi"] == ["2"]
    assert [int(x) for x in output["select"]] == oracle.select_keyframes([12, 4, 4, 20], 21).tolist()
    assert [int(x) for x in output["uniform"]] == oracle.uniform_keyframes(21, 6).tolist()


def test_adaptive_selection(output):
    sim = np.where(np.arange(16)[:, None] // 4 == np.arange(16)[None, :] // 4, 0.9, 0.1)
    exp = oracle.select_keyframes_adaptive(sim, 0.5, 8, 0.05, 1.0, 1.0)
    assert [int(x) for x in output["adaptive"]] == exp.tolist()


def test_schedule(output):
    plan = oracle.async_schedule(50, 8, 25, 2, 3)
    rp = [s["t"] for s in plan if s["phase"] == "rhythmic"]
    vals = [int(x) for x in output["schedule"]]
    assert vals[:2] == [len(rp), sum(s["phase"] == "skip" for s in plan)]
    assert vals[2:] == rp


def test_cache_bookkeeping(output):
    before2, after2, before4, after4 = (int(x) for x in output["cache"][:4])
    assert (before2, after2, before4, after4) == (2, 3, 4, 5)
    assert float(output["cache"][4]) == oracle.hidden_alpha(24.0, 21.0, 23.0)


def test_workspace_and_error(output):
    assert int(output["workspace"][0]) == 152 * 5 * 256 * (128 * 4 + 8)
    # 28,800 query rows = 113 tiles of 256 per head, 24 heads = 2,712 tiles = 10 rounds of 256 + 152;
    # 1,857 key tiles of 64 in 5 parts of 372
    assert [int(x) for x in output["plan"]] == [2712, 2560, 152, 5, 372, 152 * 5 * 256 * 520, 256]
    err = output["error"]
    assert err[0] == "RF_ERR_RANGE" and err[1] == "n=-7" and err[2].startswith("msg=rf_keyframes_uniform")
