"""bench.py's command-line contract, checked on the CPU: more than one GPU is
refused with a one-line JSON message and exit status 2 (the path runs on one
GPU; heads would shard with no communication), before anything touches a GPU
or builds inputs; and the producer byte count the bench line reports matches
the layouts of the header."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_producer_bytes_match_the_layouts():
    sys.path.insert(0, ROOT)
    import bench
    from paper_2607_02584_amd import datagen as dg
    w = dg.WORKLOADS["c2"]
    algo, moved = bench.producer_bytes(w, "e2m3")
    BH, N = w.B * w.H, w.N
    Npad = -(-N // 128) * 128
    inputs = 3 * BH * N * 128 * 2                       # bf16 Q, K, V read once
    codes = 3 * BH * Npad * 96                          # E2M3 records, 96 B per token
    scales = BH * (Npad // 128) * 4 * 2 + BH * (-(-N // 128)) * 128 * 4
    means = 2 * BH * 128 * 4
    assert algo == inputs + codes + scales + means
    assert moved == algo + 2 * BH * N * 128 * 2         # K and V read again for their means
    # the nibble container: 64 B per token
    algo4, _ = bench.producer_bytes(w, "int4")
    assert algo - algo4 == 3 * BH * Npad * 32
