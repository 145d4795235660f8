"""bench.py on the host: it refuses more than one GPU before touching one, and
the committed HBM counter summary of the frontier kernel still matches the
kernel's sources (else the bench line would report its traffic as null)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def run_bench(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args,
                          capture_output=True, text=True, env=env, cwd=ROOT, timeout=120)


def test_more_than_one_gpu_is_refused():
    p = run_bench(["--gpus", "2"])
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout == ""


def test_several_ranks_are_refused():
    p = run_bench([], {"WORLD_SIZE": "4"})
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_counter_summary_matches_the_frontier_sources():
    import bench
    traffic = bench.measured_traffic(bench.DEFAULT_WORKLOAD)
    assert traffic is not None, "re-take the frontier's FETCH_SIZE/WRITE_SIZE summary"
    alg = 15_730_080_000  # 10 000 steps x (8 S R read + 12 S written), S = 12, R = 16384
    assert abs(traffic - alg) / alg < 0.01
