"""Host-side behaviour of bench.py that needs no GPU: a request for more than
one GPU, and the out-of-core modes that are switched off at full size, end
with a message and a non-zero status before any device work."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    env = dict(os.environ, HIP_VISIBLE_DEVICES="")
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=300, env=env, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = _bench("--gpus", "2")
    assert r.returncode != 0 and "--gpus 1" in r.stderr
    assert r.stdout.strip() == ""


def test_exact_modes_off_at_full_out_of_core_size():
    for mode in ("exact", "exact-early"):
        r = _bench("--workload", "rmat28b", "--batched-mode", mode)
        assert r.returncode != 0 and "switched off" in r.stderr
        assert r.stdout.strip() == ""
