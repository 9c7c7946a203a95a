"""The benchmark's metric is the paper's "network update frame rate": update
frequency times batch size (Section 4.2). Pinned against every Spreeze row of
Tables 2 and 3 (tests/golden/update_frame_rates.txt), whose printed frame rates
have two significant digits."""
import math
import os

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "update_frame_rates.txt")


def rows():
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if line:
            label, b, f, r = line.split()
            yield label, int(b), float(f), float(r)


def two_digits(x):
    e = math.floor(math.log10(x))
    return round(x / 10 ** (e - 1)) * 10 ** (e - 1)


def test_frame_rate_is_frequency_times_batch():
    seen = 0
    for label, batch, freq, printed in rows():
        # freq steps in one second of update time
        value = bench.frames_per_second(batch, steps=1, seconds=1.0 / freq)
        assert two_digits(value) == printed, (label, value, printed)
        seen += 1
    assert seen == 8


def test_throughput_scales_with_steps_and_time():
    assert bench.frames_per_second(131072, 500, 2.0) == 131072 * 250.0


def test_bench_refuses_more_than_one_gpu():
    """The benchmark runs on one GPU: --gpus above 1 (or a multi-rank launch) exits with
    status 2 and says so, before touching a GPU."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr, (r.returncode, r.stderr)
    env = dict(os.environ, WORLD_SIZE="2")
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py")], capture_output=True, text=True,
                       timeout=120, env=env)
    assert r.returncode == 2 and "single process" in r.stderr, (r.returncode, r.stderr)
