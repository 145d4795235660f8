"""The C ABI from a plain C99 host program (tests/c_client/sf_c_client.c,
built with gcc by build()): it allocates with the HIP runtime, runs
sf_frontier on a stream of its own and sf_window_summary on the NULL stream,
and its outputs must equal the oracle's bit for bit.  Its host-side argument
checks (no device work) must return the documented statuses."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
CLIENT = os.path.join(HERE, "c_client", "sf_c_client")
SF_OK, SF_EINVAL = 0, 1


def run_client(tmp_path, d: np.ndarray, window: int):
    if not os.path.exists(CLIENT):
        pytest.fail("the C client is not built: run __graft_entry__.build()")
    T, S, R = d.shape
    src, dst = tmp_path / "in.bin", tmp_path / "out.bin"
    np.ascontiguousarray(d, dtype="<i8").tofile(src)
    print("case T=%d R=%d S=%d window=%d" % (T, R, S, window), flush=True)
    proc = subprocess.run([CLIENT, str(src), str(dst), str(T), str(R), str(S), str(window)],
                          capture_output=True, text=True, timeout=120)
    assert proc.returncode == 0, proc.stdout + proc.stderr
    assert proc.stdout.strip().splitlines()[-1] == "done"
    W = oracle.num_windows(T, window)
    raw = dst.read_bytes()
    sizes = [T * S * 8, T * S * 4, W * S * 8, W * S * R * 4, W * 16]
    assert len(raw) == sum(sizes)
    parts, off = [], 0
    for n in sizes:
        parts.append(raw[off:off + n])
        off += n
    out = {
        "inc": np.frombuffer(parts[0], "<i8").reshape(T, S),
        "lead": np.frombuffer(parts[1], "<i4").reshape(T, S),
        "exposed": np.frombuffer(parts[2], "<i8").reshape(W, S),
        "counts": np.frombuffer(parts[3], "<i4").reshape(W, S, R),
        "top2": np.frombuffer(parts[4], "<i4").reshape(W, 2, 2),
    }
    lines = dict(line.split(" ", 1) for line in proc.stdout.strip().splitlines() if " " in line)
    return out, lines


@pytest.mark.parametrize("case", ["r8_s6_t1k", "ragged", "multi_tile", "one_rank"])
def test_c_client_matches_oracle(tmp_path, case):
    if case == "r8_s6_t1k":
        wl = synth.WORKLOADS[case]
        d, window = synth.generate(wl), wl.window
    else:
        T, S, R, window = {"ragged": (40, 5, 300, 7), "multi_tile": (6, 3, 5000, 4),
                           "one_rank": (3, 1, 1, 2)}[case]
        rng = np.random.Generator(np.random.PCG64(len(case)))
        d = rng.integers(0, 5, size=(T, S, R), dtype=np.int64)   # ties everywhere
    out, lines = run_client(tmp_path, d, window)
    oi, ol = oracle.frontier(d)
    oe, oc, ot = oracle.window_summary(oi, ol, d.shape[2], window)
    np.testing.assert_array_equal(out["inc"], oi)
    np.testing.assert_array_equal(out["lead"], ol)
    np.testing.assert_array_equal(out["exposed"], oe)
    np.testing.assert_array_equal(out["counts"], oc)
    np.testing.assert_array_equal(out["top2"], ot)


def test_c_client_argument_checks(tmp_path):
    d = np.arange(2 * 3 * 4, dtype=np.int64).reshape(2, 3, 4)
    _, lines = run_client(tmp_path, d, 1)
    assert lines["version"].startswith("libstagefrontier")
    assert int(lines["frontier_r0"]) == SF_EINVAL
    assert int(lines["frontier_null"]) == SF_EINVAL
    assert int(lines["frontier_r_too_big"]) == SF_EINVAL
    assert int(lines["summary_window0"]) == SF_EINVAL
    assert int(lines["frontier_t0"]) == SF_OK
    assert int(lines["num_windows"]) == 2
    assert lines["strerror_einval"] == "invalid argument"
