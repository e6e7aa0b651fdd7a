"""Host-side checks of bench.py that need no GPU: the CPU-only oracle timing
(the child process of the one-thread baseline) and the byte accounting the
roofline uses."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_cpu_only_prints_one_json_line():
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--cpu-only", "0.2"],
                       env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-500:]
    res = json.loads(r.stdout.strip().splitlines()[-1])
    assert res["kind"] == "oracle" and res["unit"] == "GB/s" and res["cores"] == 1
    assert res["value"] > 0 and res["ms_per_step"] > 0


def test_algorithmic_bytes_of_the_headline_launch():
    # 2 x 19 328 B per tile for 256 x 32 tiles, plus q, k, v, o, g, beta,
    # the slot ids and the permutation
    assert bench.algorithmic_bytes(19328, 256, 16, 32, 128, False, 2) == 322_999_296
    kda = bench.algorithmic_bytes(19328, 256, 32, 32, 128, True, 2)
    assert kda == 2 * 19328 * 256 * 32 + 2 * 256 * 32 * 128 * 2 + 256 * 32 * 128 * 4 \
        + 256 * 32 * 128 * 2 + 256 * 32 * 2 + 4 * 256 + 32 * 128
