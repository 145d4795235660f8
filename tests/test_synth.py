"""The seeded input generator (CPU only): reproducibility, chunking and the
shape of each workload recipe."""
import numpy as np
import pytest

import synth

MS = synth.MS


def test_splitmix64_reference_outputs():
    # first outputs of SplitMix64 seeded with 0, as published with the
    # algorithm's reference implementation
    expect = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F,
              0xF88BB8A8724C81EC, 0x1B39896A51A8749B]
    assert [synth.splitmix64_at(0, i) for i in range(5)] == expect


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_chunks_concatenate_and_threads_agree(name):
    wl = synth.WORKLOADS[name]
    n = {8: 300, 128: 300, 1024: 40, 4096: 12, 16384: 4}[wl.R]
    t0 = {8: 0, 128: 5000, 1024: 100, 4096: 777, 16384: 9998}[wl.R]
    full = synth.generate(wl, t0, t0 + n, threads=4)
    k = n // 3
    a = synth.generate(wl, t0, t0 + k, threads=1)
    b = synth.generate(wl, t0 + k, t0 + n, threads=3)
    assert np.array_equal(np.concatenate([a, b]), full)
    assert (full > 0).all()
    assert full.shape == (n, wl.S, wl.R)


def test_lognormal_medians():
    wl = synth.WORKLOADS["r1024_s8_t50k"]
    x = synth.generate(wl, 0, 200)
    med = np.median(x, axis=(0, 2)) / MS
    assert np.allclose(med, wl.base_ms, rtol=0.02)
    # sigma of log durations (tail and straggler excluded by a robust estimate)
    lx = np.log(x[:, 0, :].astype(np.float64))
    iqr = np.subtract(*np.percentile(lx, [75, 25]))
    assert abs(iqr / 1.349 - wl.sigma) < 0.01


def test_stall_recipe():
    wl = synth.WORKLOADS["r8_s6_t1k"]
    inj = synth.injections(wl)
    assert len(inj) == 50 and len({t for t, _, _ in inj}) == 50
    rank = inj[0][2][0]
    assert all(k == "stall" and a[0] == rank for _, k, a in inj)
    x = synth.generate(wl)
    clean = synth.generate(wl)
    t = inj[0][0]
    # the stalled rank is late in data; the others wait in backward
    assert x[t, 0, rank] > 30 * MS + 5 * MS
    others = [r for r in range(wl.R) if r != rank]
    assert (x[t, 2, others] > 120 * MS).all()
    assert np.array_equal(x, clean)


def test_fault_recipe():
    wl = synth.WORKLOADS["r128_s6_t100k"]
    inj = synth.injections(wl)
    assert len(inj) == 1000
    assert all(10 * MS <= a[2] <= 50 * MS for _, _, a in inj)
    wl5 = synth.WORKLOADS["r16384_s12_t20k"]
    inj5 = synth.injections(wl5)
    assert len(inj5) == 100
    assert all(5 * MS <= a[2] <= 100 * MS for _, _, a in inj5)


def test_tie_recipe_makes_equal_prefixes():
    wl = synth.WORKLOADS["r4096_s12_t20k"]
    inj = synth.injections(wl)
    assert len(inj) == round(0.01 * wl.T * wl.S)
    # check the ties that land in the first 300 steps
    x = synth.generate(wl, 0, 300)
    P = np.cumsum(x, axis=1)
    seen = 0
    last = {}
    for t, kind, (s, r1, r2, _) in inj:
        if t < 300:
            last[t] = (s, r1, r2)
    for t, (s, r1, r2) in last.items():
        assert P[t, s, r1] == P[t, s, r2]
        seen += 1
    assert seen > 0


def test_straggler_recipe():
    wl = synth.WORKLOADS["r1024_s8_t50k"]
    r = synth.straggler_rank(wl)
    assert 0 <= r < wl.R
    x = synth.generate(wl, 0, 400).astype(np.float64)
    ratio = np.median(x[:, :, r]) / np.median(np.delete(x, r, axis=2))
    assert 1.0 < ratio < 1.07


def test_values_far_inside_prefix_bound():
    for name in synth.WORKLOAD_ORDER:
        wl = synth.WORKLOADS[name]
        x = synth.generate(wl, 0, 3)
        assert x.sum(axis=1).max() < (1 << 40)
