"""bench.py's command-line contract on the CPU: refusals that happen before
any GPU work (several GPUs, a bad --batch), and the --batch workload names."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    return p.returncode, p.stdout.strip().splitlines()


@pytest.mark.parametrize("args, needle", [
    (("--gpus", "2"), "one MI355X"),
    (("--batch", "0"), "--batch must be >= 1"),
    (("--workload", "c4p", "--batch", "8"), "applies to the 8B decode workload"),
])
def test_bench_refuses_before_gpu_work(args, needle):
    rc, lines = run_bench(*args)
    assert rc == 2
    msg = json.loads(lines[-1])
    assert needle in msg["error"]


def test_batch_option_names_the_workload():
    sys.path.insert(0, ROOT)
    import bench
    wl, batch, layers = bench.build_workload("c2", 129)
    assert (wl.name, batch.n_rows, layers) == ("llama8b_decode_b129", 129, 1)
    wl64, batch64, _ = bench.build_workload("c2")
    assert (wl64.name, batch64.n_rows) == ("llama8b_decode_b64", 64)
