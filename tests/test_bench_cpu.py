"""bench.py's host logic without a GPU: the one-GPU guard, the refusal to run
without a GPU, the code digest that keys the committed traffic counters, the
traffic lookup itself, and the guard that keeps a failing side measurement
from costing the JSON line."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _run(args, env=None):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args, capture_output=True, text=True,
                          env=e, timeout=300)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_world_size_above_one_is_refused():
    r = _run([], env={"WORLD_SIZE": "2"})
    assert r.returncode == 2


def _gpu_count():
    import torch   # counting devices does not initialise the GPU
    return torch.cuda.device_count()


@pytest.mark.skipif(_gpu_count() > 0, reason="a GPU is present")
def test_no_gpu_is_an_error():
    r = _run(["--steps", "1", "--warmup", "0"])
    assert r.returncode == 1
    assert "needs a GPU" in r.stderr


def test_source_digest_ignores_comments_and_whitespace(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    c = tmp_path / "c.hip"
    a.write_text("int f(int x) {\n  return x + 1;  // add one\n}\n")
    b.write_text("/* header */ int f(int x)\n{ return x + 1; }\n")
    c.write_text("int f(int x) { return x + 2; }\n")
    assert bench.source_digest(str(a)) == bench.source_digest(str(b))
    assert bench.source_digest(str(a)) != bench.source_digest(str(c))


def test_committed_traffic_is_reported_only_for_the_code_it_was_taken_on():
    """The bench reports the committed counter summary's traffic only while the
    attention code has the digest recorded there (then it exceeds the
    algorithmic bytes); after a change of the code it reports none."""
    path = os.path.join(ROOT, "profiles", "attn_bf16_long_traffic.txt")
    recorded = [l.split(":", 1)[1].strip() for l in open(path) if l.startswith("attention code sha256")]
    current = bench.source_digest(os.path.join(ROOT, "paper_2606_06309_amd", "csrc", "rf_attention.hip"))
    traffic = bench.profiled_traffic("long")
    if recorded == [current]:
        assert isinstance(traffic, int) and traffic > 1813708800
    else:
        assert traffic is None


def test_side_section_failure_is_reported(capsys):
    def broken():
        raise RuntimeError("no such device")
    out = bench._side("demo", broken)
    assert out["error"].startswith("RuntimeError")
    assert "demo failed" in capsys.readouterr().err
    assert bench._side("ok", lambda x: {"v": x}, 3) == {"v": 3}
