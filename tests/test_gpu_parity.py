"""GPU path against the CPU oracle, element by element (bit-exact: every
output is integer ns or an index).  Shapes sweep every launch variant of the
frontier kernel (tile widths, 8- and 16-byte loads, several tiles per rank
row, ragged rank and step counts), the window kernels (ragged last window,
several rank chunks, leaders outside [0, R)), and the degenerate cases."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def sf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_06751_amd import stagefrontier
    return stagefrontier


DEV = "cuda:0"


def gpu_frontier(sf, d: np.ndarray):
    dd = torch.from_numpy(np.ascontiguousarray(d)).to(DEV)
    inc, lead = sf.sf_frontier(dd)
    torch.cuda.synchronize()
    return inc.cpu().numpy(), lead.cpu().numpy()


def gpu_summary(sf, inc: np.ndarray, lead: np.ndarray, R: int, window: int):
    ti = torch.from_numpy(np.ascontiguousarray(inc)).to(DEV)
    tl = torch.from_numpy(np.ascontiguousarray(lead)).to(DEV)
    ex, cnt, top2 = sf.sf_window_summary(ti, tl, R, window)
    torch.cuda.synchronize()
    return ex.cpu().numpy(), cnt.cpu().numpy(), top2.cpu().numpy()


def assert_frontier_equal(sf, d):
    gi, gl = gpu_frontier(sf, d)
    oi, ol = oracle.frontier(d)
    np.testing.assert_array_equal(gi, oi)
    np.testing.assert_array_equal(gl, ol)
    return oi, ol


def assert_summary_equal(sf, inc, lead, R, window):
    ge, gc, gt = gpu_summary(sf, inc, lead, R, window)
    oe, oc, ot = oracle.window_summary(inc, lead, R, window)
    np.testing.assert_array_equal(ge, oe)
    np.testing.assert_array_equal(gc, oc)
    np.testing.assert_array_equal(gt, ot)


# rank counts at and around every tile boundary of the launch table, odd
# counts (8-byte loads), several tiles per row (R > 4096) and the maximum
RANKS = [1, 2, 3, 7, 8, 9, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 257,
         511, 512, 513, 1000, 1023, 1024, 1025, 2047, 2048, 2049, 4095, 4096, 4097,
         8192, 12289, 16384]


@pytest.mark.parametrize("R", RANKS)
def test_frontier_rank_sweep(sf, R):
    T = max(3, min(70, 200000 // (R * 6)))
    for S, hi in [(6, 10**9), (5, 3)]:          # tie-free-ish and tie-heavy
        d = synth.random_durations(T, S, R, seed=R * 31 + S, hi=hi)
        print("case R=%d S=%d T=%d hi=%d" % (R, S, T, hi), flush=True)
        assert_frontier_equal(sf, d)


@pytest.mark.parametrize("S", [1, 2, 3, 12, 13, 64, 200, 512])
def test_frontier_stage_sweep(sf, S):
    for R in (8, 128, 1024, 5000):
        T = max(2, min(40, 400000 // (R * S)))
        d = synth.random_durations(T, S, R, seed=S * 7 + R, hi=10**6)
        print("case R=%d S=%d T=%d" % (R, S, T), flush=True)
        assert_frontier_equal(sf, d)


@pytest.mark.parametrize("S", [513, 768, 4096])
@pytest.mark.parametrize("R", [8, 1024, 16384])
def test_frontier_large_stage_counts(sf, S, R):
    """Stage counts past what LDS holds (Sec. 3 expands accumulation
    micro-steps into stages before the frontier): the partial maxima go
    through the out_increment rows.  Ragged step counts against the steps a
    workgroup holds, tie-heavy and wide values, and the checked pass."""
    T = max(2, min(37, (1 << 27) // (R * S)))
    for hi in (3, 10**7):
        d = synth.random_durations(T, S, R, seed=S * 3 + R + hi, hi=hi)
        print("case R=%d S=%d T=%d hi=%d" % (R, S, T, hi), flush=True)
        oi, ol = assert_frontier_equal(sf, d)
        inc, lead, st = checked(sf, d)
        np.testing.assert_array_equal(inc, oi)
        np.testing.assert_array_equal(lead, ol)
        assert st == 0
    e = d.copy()
    e[T - 1, S - 1, R - 1] = -1
    assert checked(sf, e)[2] == oracle.range_status(e) == sf.SF_ERANGE


@pytest.mark.parametrize("S", [513, 2048, 2049, 4100])
def test_window_rows_large_stage_counts(sf, S):
    """The window summary, exposed time led, leader switches and the
    routing set at stage counts past 512 (and past the LDS staging of the
    stage totals at 2048 and of route's at 4096)."""
    R, T, window = 37, 90, 16
    d = synth.random_durations(T, S, R, seed=S, hi=4)
    oi, ol = oracle.frontier(d)
    assert_summary_equal(sf, oi, ol, R, window)
    ti = torch.from_numpy(oi).to(DEV)
    tl = torch.from_numpy(ol).to(DEV)
    le, letop = sf.sf_window_lead_exposed(ti, tl, R, window)
    torch.cuda.synchronize()
    ole, olt = oracle.window_lead_exposed(oi, ol, R, window)
    np.testing.assert_array_equal(le.cpu().numpy(), ole)
    np.testing.assert_array_equal(letop.cpu().numpy(), olt)
    ev = oracle.frontier_evidence(d)
    sw, el = sf.sf_window_leader_switches(tl, torch.from_numpy(ev["gap"]).to(DEV),
                                          torch.from_numpy(ev["ties"]).to(DEV), window, 1)
    torch.cuda.synchronize()
    osw, oel = oracle.window_leader_switches(ev["lead"], ev["gap"], ev["ties"], window, 1)
    np.testing.assert_array_equal(sw.cpu().numpy(), osw)
    np.testing.assert_array_equal(el.cpu().numpy(), oel)
    oe, _, _ = oracle.window_summary(oi, ol, R, window)
    oe[0, S // 3] = 1 << 50                     # one dominant stage
    oe[1] = 5                                   # every stage tied
    for num, den in ((4, 5), (1, 1), (0, 1)):
        go, gs = sf.sf_route(torch.from_numpy(oe).to(DEV), num, den)
        torch.cuda.synchronize()
        oo, os_ = oracle.route(oe, num, den)
        np.testing.assert_array_equal(go.cpu().numpy(), oo)
        np.testing.assert_array_equal(gs.cpu().numpy(), os_)


def test_selections_large_stage_counts(sf):
    """The lag, the raw spread and the window median at 600 stages."""
    d = synth.random_durations(12, 600, 300, seed=600, hi=10**6)
    lag, inc = sf.sf_frontier_lag(torch.from_numpy(d).to(DEV))
    sp, wsp = sf.sf_rank_spread(torch.from_numpy(d).to(DEV), 5)
    med = sf.sf_window_median(torch.from_numpy(d).to(DEV), 5)
    torch.cuda.synchronize()
    ol, oinc = oracle.frontier_lag(d)
    np.testing.assert_array_equal(lag.cpu().numpy(), ol)
    np.testing.assert_array_equal(inc.cpu().numpy(), oinc)
    osp, owsp = oracle.rank_spread(d, 5)
    np.testing.assert_array_equal(sp.cpu().numpy(), osp)
    np.testing.assert_array_equal(wsp.cpu().numpy(), owsp)
    np.testing.assert_array_equal(med.cpu().numpy(), oracle.window_median(d, 5))


@pytest.mark.parametrize("T", [1, 2, 3, 5, 15, 16, 17, 63, 65, 257])
def test_frontier_ragged_steps(sf, T):
    for R in (8, 24, 128, 300):
        d = synth.random_durations(T, 6, R, seed=T * 13 + R, hi=50)
        assert_frontier_equal(sf, d)


def test_frontier_max_ranks(sf):
    R = sf.SF_MAX_R
    d = synth.random_durations(3, 4, R, seed=11, hi=2)   # heavy ties over 65536 ranks
    d[1, :, R - 1] = 5                                   # last rank leads step 1
    oi, ol = assert_frontier_equal(sf, d)
    assert (ol[1] == R - 1).all()


def test_frontier_all_zero_and_single_rank(sf):
    d = np.zeros((9, 4, 300), dtype=np.int64)
    gi, gl = gpu_frontier(sf, d)
    assert (gi == 0).all() and (gl == 0).all()
    d1 = synth.random_durations(50, 7, 1, seed=3)
    gi, gl = gpu_frontier(sf, d1)
    np.testing.assert_array_equal(gi, d1[:, :, 0])
    assert (gl == 0).all()


def test_frontier_large_values(sf):
    """Prefixes close to the documented bound stay exact."""
    big = sf.SF_MAX_PREFIX_NS - 1
    d = np.zeros((2, 3, 130), dtype=np.int64)
    d[0, 0, 77] = big - 5
    d[0, 2, 77] = 5
    d[1, 1, 129] = big
    d[1, 0, 3] = big - 1
    assert_frontier_equal(sf, d)


def test_frontier_golden_examples(sf):
    import pins
    for name in pins.GOLDEN_FILES:
        g = pins.load_golden(name)
        gi, gl = gpu_frontier(sf, g["d"])
        assert gi[0].tolist() == g["inc"] and gl[0].tolist() == g["lead"]
    gi, gl = gpu_frontier(sf, pins.stall_case())
    assert gl[0].tolist() == [2, 2, 0, 0, 0, 0]


def test_frontier_misaligned_base_uses_narrow_loads(sf):
    """A base that is 8- but not 16-byte aligned takes the 8-byte-load path."""
    T, S, R = 20, 6, 256
    d = synth.random_durations(T, S, R, seed=5, hi=1000)
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    view = flat[1:].view(T, S, R)
    assert view.data_ptr() % 16 == 8
    inc, lead = sf.sf_frontier(view)
    torch.cuda.synchronize()
    oi, ol = oracle.frontier(d)
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(lead.cpu().numpy(), ol)


def test_frontier_chunks_compose(sf):
    """Step-axis chunks written into one output equal a single call."""
    T, S, R = 101, 12, 640
    d = synth.random_durations(T, S, R, seed=17, hi=10**5)
    dd = torch.from_numpy(d).to(DEV)
    inc = torch.full((T, S), -7, dtype=torch.int64, device=DEV)
    lead = torch.full((T, S), -7, dtype=torch.int32, device=DEV)
    for t0, t1 in [(0, 37), (37, 38), (38, 101)]:
        sf.sf_frontier(dd[t0:t1], inc[t0:t1], lead[t0:t1])
    torch.cuda.synchronize()
    oi, ol = oracle.frontier(d)
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(lead.cpu().numpy(), ol)


def test_frontier_empty(sf):
    dd = torch.empty((0, 6, 8), dtype=torch.int64, device=DEV)
    inc, lead = sf.sf_frontier(dd)
    assert inc.shape == (0, 6)


def test_frontier_repeatable(sf):
    """Integer outputs of repeated runs are identical (no lane races)."""
    d = synth.random_durations(64, 12, 4096, seed=23, hi=4)
    dd = torch.from_numpy(d).to(DEV)
    first = [x.clone() for x in sf.sf_frontier(dd)]
    for _ in range(5):
        again = sf.sf_frontier(dd)
        assert all(torch.equal(a, b) for a, b in zip(first, again))


@pytest.mark.parametrize("R,S,T,window", [
    (8, 6, 1000, 100), (8, 6, 1001, 100), (3, 1, 17, 4), (128, 6, 3000, 1000),
    (1024, 8, 1200, 500), (5, 13, 40, 1), (4096, 12, 600, 250), (16384, 12, 80, 7),
    (20000, 3, 50, 50), (40000, 2, 30, 16), (65536, 2, 10, 3)])
def test_summary_from_oracle_steps(sf, R, S, T, window):
    """Window summary of seeded per-step arrays (hot leaders, ties)."""
    rng = np.random.Generator(np.random.PCG64(R + S + T))
    inc = rng.integers(0, 10**9, size=(T, S), dtype=np.int64)
    # leaders concentrated on a few ranks so that counts and ties matter
    hot = rng.integers(0, R, size=4)
    lead = np.where(rng.random((T, S)) < 0.7, hot[rng.integers(0, 4, size=(T, S))],
                    rng.integers(0, R, size=(T, S))).astype(np.int32)
    print("case R=%d S=%d T=%d window=%d" % (R, S, T, window), flush=True)
    assert_summary_equal(sf, inc, lead, R, window)


def test_summary_ties_and_out_of_range_leaders(sf):
    T, S, R = 60, 5, 9
    inc = np.zeros((T, S), dtype=np.int64)
    inc[:, 1] = 5
    inc[:, 3] = 5                       # stages 1 and 3 tie on exposed
    lead = np.tile(np.array([0, 4, 2, 7, 1], dtype=np.int32), (T, 1))
    lead[::2, 1] = 6                    # ranks 4 and 6 tie on counts
    lead[::3, 0] = -1                   # not counted
    lead[::5, 2] = 9                    # == R: not counted
    lead[1::7, 4] = np.iinfo(np.int32).min
    for window in (1, 6, 7, 60, 61):
        assert_summary_equal(sf, inc, lead, R, window)


def assert_lead_exposed_equal(sf, inc, lead, R, window):
    ti = torch.from_numpy(np.ascontiguousarray(inc)).to(DEV)
    tl = torch.from_numpy(np.ascontiguousarray(lead)).to(DEV)
    le, top2 = sf.sf_window_lead_exposed(ti, tl, R, window)
    torch.cuda.synchronize()
    ole, ot = oracle.window_lead_exposed(inc, lead, R, window)
    np.testing.assert_array_equal(le.cpu().numpy(), ole)
    np.testing.assert_array_equal(top2.cpu().numpy(), ot)



@pytest.mark.parametrize("R", [1, 2, 7, 8, 9, 16, 17, 33, 64, 65, 128, 129, 200, 256, 257])
def test_frontier_summary_fused(sf, R):
    """sf_frontier_summary against the oracle's frontier and window summary,
    on both sides of every limit of its one-launch path (ranks, stages,
    window length, total samples) and on ragged windows."""
    cases = [(37, 5, 10, 3), (250, 6, 100, 10**6), (33, 64, 7, 2), (20, 65, 6, 5)]
    if R <= 32:
        cases += [(1030, 2, 1030, 10**4), (2100, 2, 1025, 4)]
    cases.append(((1 << 20) // (4 * R) + 3, 4, 64, 10**5))  # just past 2^20 samples
    for T, S, window, hi in cases:
        d = synth.random_durations(T, S, R, seed=R * 7 + S + window, hi=hi)
        print("case R=%d S=%d T=%d window=%d" % (R, S, T, window), flush=True)
        out = sf.sf_frontier_summary(torch.from_numpy(d).to(DEV), window)
        torch.cuda.synchronize()
        oi, ol = oracle.frontier(d)
        oe, oc, ot = oracle.window_summary(oi, ol, R, window)
        for got, want in zip(out, (oi, ol, oe, oc, ot)):
            np.testing.assert_array_equal(got.cpu().numpy(), want)


def test_frontier_summary_small_workload_and_stall(sf):
    """The 8-rank workload and the hand-built data stall through the fused
    call, against the oracle and the separate calls."""
    wl = synth.WORKLOADS["r8_s6_t1k"]
    d = synth.generate(wl)
    dd = torch.from_numpy(d).to(DEV)
    out = sf.sf_frontier_summary(dd, wl.window)
    inc, lead = sf.sf_frontier(dd)
    sep = (inc, lead) + sf.sf_window_summary(inc, lead, wl.R, wl.window)
    torch.cuda.synchronize()
    oi, ol = oracle.frontier(d)
    want = (oi, ol) + oracle.window_summary(oi, ol, wl.R, wl.window)
    for got, s_, w in zip(out, sep, want):
        np.testing.assert_array_equal(got.cpu().numpy(), w)
        np.testing.assert_array_equal(s_.cpu().numpy(), w)
    ms = 1_000_000
    st = np.ascontiguousarray(np.array([[20, 60, 120, 2, 15, 3]] * 4, dtype=np.int64).T[None] * ms)
    st[0, 0, 2] += 30 * ms
    st[0, 2, [0, 1, 3]] += 30 * ms
    out = sf.sf_frontier_summary(torch.from_numpy(st).to(DEV), 1)
    torch.cuda.synchronize()
    assert out[0].cpu().numpy().tolist() == [[50 * ms, 60 * ms, 120 * ms, 2 * ms, 15 * ms, 3 * ms]]
    assert out[1].cpu().numpy().tolist() == [[2, 2, 0, 0, 0, 0]]
    assert int(out[3].cpu()[0, 0, 2]) == 1


@pytest.mark.parametrize("R,S,T,window", [
    (8, 6, 1000, 100), (8, 6, 1001, 100), (3, 1, 17, 4), (128, 6, 3000, 1000),
    (1024, 8, 1200, 500), (5, 13, 40, 1), (4096, 12, 600, 250), (8192, 4, 90, 30),
    (8193, 4, 90, 31), (16384, 12, 80, 7), (20000, 3, 50, 50), (65536, 2, 10, 3),
    (7, 512, 70, 9)])
def test_lead_exposed_from_oracle_steps(sf, R, S, T, window):
    """Exposed time led and its top-2 on seeded per-step arrays: leaders
    concentrated on a few ranks, every rank-chunk boundary of the weighted
    histogram (8192 ranks), the largest stage count."""
    rng = np.random.Generator(np.random.PCG64(R * 7 + S + T))
    inc = rng.integers(0, 10**9, size=(T, S), dtype=np.int64)
    hot = rng.integers(0, R, size=4)
    lead = np.where(rng.random((T, S)) < 0.7, hot[rng.integers(0, 4, size=(T, S))],
                    rng.integers(0, R, size=(T, S))).astype(np.int32)
    print("case R=%d S=%d T=%d window=%d" % (R, S, T, window), flush=True)
    assert_lead_exposed_equal(sf, inc, lead, R, window)


def test_lead_exposed_ties_signs_and_out_of_range_leaders(sf):
    """Stage-total ties, rank ties on exposed time, zero rows (rank -1),
    negative advances (never a suspect) and leaders outside [0, R)."""
    T, S, R = 60, 6, 9
    inc = np.zeros((T, S), dtype=np.int64)
    inc[:, 1] = 5
    inc[:, 3] = 5                       # stages 1 and 3 tie on the total
    inc[:, 5] = -3                      # negative advances
    lead = np.tile(np.array([0, 4, 2, 7, 1, 3], dtype=np.int32), (T, 1))
    lead[::2, 1] = 6                    # ranks 4 and 6 tie on exposed time
    lead[::3, 0] = -1                   # not counted
    lead[::5, 2] = 9                    # == R: not counted
    lead[1::7, 4] = np.iinfo(np.int32).min
    for window in (1, 6, 7, 60, 61):
        assert_lead_exposed_equal(sf, inc, lead, R, window)
    # every advance negative or zero: no rank is a suspect
    assert_lead_exposed_equal(sf, -np.abs(inc), lead, R, 10)
    # large magnitudes of both signs (exact two's-complement sums)
    rng = np.random.Generator(np.random.PCG64(5))
    big = rng.integers(-(1 << 52), 1 << 52, size=(64, 3), dtype=np.int64)
    lead = rng.integers(0, 2, size=(64, 3), dtype=np.int32)
    assert_lead_exposed_equal(sf, big, lead, 2, 16)


def test_lead_exposed_after_frontier(sf):
    """sf_frontier then sf_window_lead_exposed on the 8-rank workload and
    on the stall pattern; the rows add up to the summary's stage totals."""
    wl = synth.WORKLOADS["r8_s6_t1k"]
    d = synth.generate(wl)
    oi, ol = oracle.frontier(d)
    dd = torch.from_numpy(d).to(DEV)
    inc, lead = sf.sf_frontier(dd)
    le, top2 = sf.sf_window_lead_exposed(inc, lead, wl.R, wl.window)
    ex, _, _ = sf.sf_window_summary(inc, lead, wl.R, wl.window)
    torch.cuda.synchronize()
    ole, ot = oracle.window_lead_exposed(oi, ol, wl.R, wl.window)
    np.testing.assert_array_equal(le.cpu().numpy(), ole)
    np.testing.assert_array_equal(top2.cpu().numpy(), ot)
    np.testing.assert_array_equal(le.sum(dim=2).cpu().numpy(), ex.cpu().numpy())


def assert_switches_equal(sf, lead, gap, ties, window, min_gap):
    tl, tg, tt = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in (lead, gap, ties))
    sw, el = sf.sf_window_leader_switches(tl, tg, tt, window, min_gap)
    torch.cuda.synchronize()
    osw, oel = oracle.window_leader_switches(lead, gap, ties, window, min_gap)
    np.testing.assert_array_equal(sw.cpu().numpy(), osw)
    np.testing.assert_array_equal(el.cpu().numpy(), oel)


@pytest.mark.parametrize("T,S", [(1, 1), (63, 3), (64, 2), (65, 6), (1000, 12), (3001, 5),
                                 (40, 512)])
def test_switches_from_random_evidence(sf, T, S):
    """Leader switches on seeded evidence arrays: 64-step chunk edges of the
    wave walk, ragged windows, thresholds at and around the gaps, no
    runner-up (gap -1), ties, leaders of any int32 value."""
    rng = np.random.Generator(np.random.PCG64(T * 31 + S))
    lead = rng.integers(0, 5, size=(T, S), dtype=np.int32)
    lead[::17] = rng.integers(np.iinfo(np.int32).min, np.iinfo(np.int32).max, size=lead[::17].shape,
                              dtype=np.int32)
    ties = rng.choice(np.array([1, 1, 1, 2, 7], dtype=np.int32), size=(T, S))
    gap = np.where(ties == 1, rng.integers(-1, 1000, size=(T, S)), 0).astype(np.int64)
    print("case T=%d S=%d" % (T, S), flush=True)
    for window in sorted({1, 5, 63, 64, 65, 128, 1000, T, T + 3}):
        for min_gap in (0, 500, 1000, -5):
            assert_switches_equal(sf, lead, gap, ties, window, min_gap)


def test_switches_after_evidence(sf):
    """sf_frontier_evidence then sf_window_leader_switches: the 8-rank
    workload (stalls on 5% of its steps) and the stall moving between two
    ranks, against the oracle's own evidence."""
    wl = synth.WORKLOADS["r8_s6_t1k"]
    d = synth.generate(wl)
    ev = sf.sf_frontier_evidence(torch.from_numpy(d).to(DEV))
    oev = oracle.frontier_evidence(d)
    for min_gap in (0, 10**6, 25 * 10**6):
        sw, el = sf.sf_window_leader_switches(ev["leader"], ev["gap"], ev["ties"], wl.window, min_gap)
        torch.cuda.synchronize()
        osw, oel = oracle.window_leader_switches(oev["lead"], oev["gap"], oev["ties"], wl.window,
                                                 min_gap)
        np.testing.assert_array_equal(sw.cpu().numpy(), osw)
        np.testing.assert_array_equal(el.cpu().numpy(), oel)
    # R = 1: every boundary qualifies (no runner-up), no switch
    d1 = synth.random_durations(70, 4, 1, seed=3, hi=10**6)
    ev = sf.sf_frontier_evidence(torch.from_numpy(d1).to(DEV))
    sw, el = sf.sf_window_leader_switches(ev["leader"], ev["gap"], ev["ties"], 32, 10**9)
    torch.cuda.synchronize()
    assert el.cpu().numpy().tolist() == [[32] * 4, [32] * 4, [6] * 4]
    assert (sw.cpu().numpy() == 0).all()


def test_end_to_end_small_workload(sf):
    """sf_frontier then sf_window_summary, as the benchmark chains them."""
    wl = synth.WORKLOADS["r8_s6_t1k"]
    d = synth.generate(wl)
    oi, ol = assert_frontier_equal(sf, d)
    dd = torch.from_numpy(d).to(DEV)
    inc, lead = sf.sf_frontier(dd)
    ex, cnt, top2 = sf.sf_window_summary(inc, lead, wl.R, wl.window)
    torch.cuda.synchronize()
    oe, oc, ot = oracle.window_summary(oi, ol, wl.R, wl.window)
    np.testing.assert_array_equal(ex.cpu().numpy(), oe)
    np.testing.assert_array_equal(cnt.cpu().numpy(), oc)
    np.testing.assert_array_equal(top2.cpu().numpy(), ot)


def test_bad_arguments_raise(sf):
    d = torch.zeros((4, 3, 8), dtype=torch.int32, device=DEV)
    with pytest.raises(TypeError):
        sf.sf_frontier(d)
    with pytest.raises(ValueError):
        sf.sf_frontier(torch.zeros((4, 3, 8), dtype=torch.int64))   # host tensor
    dd = torch.zeros((4, 3, 8), dtype=torch.int64, device=DEV)
    inc = torch.zeros((4, 3), dtype=torch.int64, device=DEV)
    with pytest.raises(sf.StageFrontierError):
        sf.sf_frontier(dd, inc, inc.view(torch.int32).view(-1)[:12].view(4, 3))  # overlap


# ----------------------------------------------------------------------------
# localization evidence and per-stage baselines (sf_frontier_evidence)

EV_KEYS = {"increment": "inc", "leader": "lead", "gap": "gap", "ties": "ties",
           "stage_max": "stage_max", "stage_sum": "stage_sum"}


def gpu_evidence(sf, d):
    out = sf.sf_frontier_evidence(torch.from_numpy(np.ascontiguousarray(d)).to(DEV))
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def assert_evidence_equal(sf, d):
    g = gpu_evidence(sf, d)
    o = oracle.frontier_evidence(d)
    for gk, ok in EV_KEYS.items():
        np.testing.assert_array_equal(g[gk], o[ok], err_msg=gk)
    # the frontier part equals sf_frontier's
    gi, gl = gpu_frontier(sf, d)
    np.testing.assert_array_equal(g["increment"], gi)
    np.testing.assert_array_equal(g["leader"], gl)


EV_RANKS = [1, 2, 3, 8, 63, 64, 65, 127, 128, 129, 300, 512, 513, 1000, 1024, 1025, 2048,
            2049, 4096, 5000, 16384]


@pytest.mark.parametrize("R", EV_RANKS)
def test_evidence_rank_sweep(sf, R):
    T = max(3, min(60, 200000 // (R * 6)))
    for S, hi in [(6, 10**9), (5, 2)]:
        d = synth.random_durations(T, S, R, seed=R * 17 + S, hi=hi)
        print("case R=%d S=%d T=%d hi=%d" % (R, S, T, hi), flush=True)
        assert_evidence_equal(sf, d)


@pytest.mark.parametrize("S", [1, 2, 13, 100, 512])
def test_evidence_stage_sweep(sf, S):
    for R in (8, 130, 3000):
        T = max(2, min(30, 300000 // (R * S)))
        d = synth.random_durations(T, S, R, seed=S * 5 + R, hi=10**5)
        print("case R=%d S=%d T=%d" % (R, S, T), flush=True)
        assert_evidence_equal(sf, d)


@pytest.mark.parametrize("S", [513, 819, 820, 1500, 4096])
@pytest.mark.parametrize("R", [8, 301, 1000, 1025, 16384])
def test_evidence_large_stage_counts(sf, S, R):
    """Stage counts past what LDS holds (the accumulation expansion of
    Sec. 3): from 820 stages the partial results of a step go through its
    own output rows.  Odd rank counts (8-byte loads), rank tiles with a
    ragged last one, step counts ragged against the steps a workgroup holds,
    tie-heavy and wide values."""
    T = max(2, min(37, (1 << 25) // (R * S)))
    T += 1 - T % 2  # odd
    for hi in (2, (1 << 47) // S - 1):  # every prefix stays below 2^47
        d = synth.random_durations(T, S, R, seed=S * 11 + R + (hi & 0xFF), hi=hi)
        print("case R=%d S=%d T=%d hi=%d" % (R, S, T, hi), flush=True)
        assert_evidence_equal(sf, d)


def test_evidence_max_ranks_and_odd_base(sf):
    d = synth.random_durations(2, 3, sf.SF_MAX_R, seed=19, hi=1)
    assert_evidence_equal(sf, d)
    # 8- but not 16-byte aligned base: narrow loads
    T, S, R = 9, 4, 1030
    d = synth.random_durations(T, S, R, seed=21, hi=3)
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    out = sf.sf_frontier_evidence(flat[1:].view(T, S, R))
    torch.cuda.synchronize()
    o = oracle.frontier_evidence(d)
    for gk, ok in EV_KEYS.items():
        np.testing.assert_array_equal(out[gk].cpu().numpy(), o[ok], err_msg=gk)


def test_evidence_golden_and_stall(sf):
    import pins
    g = pins.load_golden("motivating_example.txt")
    out = gpu_evidence(sf, g["d"])
    assert out["stage_max"][0].tolist() == g["stage_max"]
    out = gpu_evidence(sf, pins.stall_case())
    assert out["ties"][0].tolist() == [1, 1, 4, 4, 4, 4]
    assert out["gap"][0].tolist() == [30 * pins.MS, 30 * pins.MS, 0, 0, 0, 0]


# ----------------------------------------------------------------------------
# ingest (Appendix A closure) and routing candidate set (Sec. 4)

def _ingest_inputs(R, T, K, seed, slack=10**5):
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.integers(0, 10**6, size=(R, T, K), dtype=np.int64)
    w = x.sum(axis=2) + rng.integers(-slack, slack + 1, size=(R, T), dtype=np.int64)
    return x, w


@pytest.mark.parametrize("R,T,K", [(1, 1, 0), (1, 9, 5), (8, 100, 5), (7, 33, 1), (64, 64, 5),
                                   (65, 17, 11), (130, 50, 7), (1000, 12, 63), (3, 5, 64),
                                   (40, 3, 127), (17, 2, 255), (9, 2, 511), (65536, 2, 3),
                                   (4099, 19, 11), (5, 3, 512), (300, 7, 600), (257, 2, 4095),
                                   (1, 4, 1000)])
def test_ingest_matches_oracle(sf, R, T, K):
    x, w = _ingest_inputs(R, T, K, seed=R * 7 + T + K)
    print("case R=%d T=%d K=%d" % (R, T, K), flush=True)
    gd, go = sf.sf_ingest(torch.from_numpy(x).to(DEV), torch.from_numpy(w).to(DEV))
    torch.cuda.synchronize()
    od, oo = oracle.ingest(x, w)
    np.testing.assert_array_equal(gd.cpu().numpy(), od)
    np.testing.assert_array_equal(go.cpu().numpy(), oo)


def test_ingest_feeds_the_frontier(sf):
    """Ingested buffers give the same frontier as the matrix they came from."""
    wl = synth.WORKLOADS["r128_s6_t100k"]
    d0 = synth.generate(wl, 0, 500)
    x = d0[:, :-1, :].transpose(2, 0, 1).copy()
    w = d0.sum(axis=1).T.copy()
    gd, go = sf.sf_ingest(torch.from_numpy(x).to(DEV), torch.from_numpy(w).to(DEV))
    inc, lead = sf.sf_frontier(gd)
    torch.cuda.synchronize()
    assert np.array_equal(gd.cpu().numpy(), d0) and int(go.abs().sum()) == 0
    oi, ol = oracle.frontier(d0)
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(lead.cpu().numpy(), ol)


@pytest.mark.parametrize("S", [1, 2, 3, 6, 12, 64, 100, 511, 512])
def test_route_matches_oracle(sf, S):
    rng = np.random.Generator(np.random.PCG64(S))
    W = 37
    ex = rng.integers(0, 6, size=(W, S), dtype=np.int64) * rng.integers(1, 10**9)
    ex[0] = 0                                   # empty window total
    ex[1, :] = 7                                # all tied
    if S > 3:
        ex[2, 3] = 1 << 61                      # one dominant stage, large values
    te = torch.from_numpy(ex).to(DEV)
    for num, den in ((4, 5), (7, 10), (9, 10), (0, 1), (1, 1), (1, 3), (2147483646, 2147483647)):
        go, gs = sf.sf_route(te, num, den)
        torch.cuda.synchronize()
        oo, os_ = oracle.route(ex, num, den)
        np.testing.assert_array_equal(go.cpu().numpy(), oo)
        np.testing.assert_array_equal(gs.cpu().numpy(), os_)


def test_route_after_window_summary(sf):
    """Chained on the GPU: the first two routed stages are the top-2 stages."""
    wl = synth.WORKLOADS["r8_s6_t1k"]
    d = synth.generate(wl)
    inc, lead = sf.sf_frontier(torch.from_numpy(d).to(DEV))
    ex, cnt, top2 = sf.sf_window_summary(inc, lead, wl.R, wl.window)
    order, size = sf.sf_route(ex)
    torch.cuda.synchronize()
    oi, ol = oracle.frontier(d)
    oe, _, _ = oracle.window_summary(oi, ol, wl.R, wl.window)
    oo, os_ = oracle.route(oe)
    np.testing.assert_array_equal(order.cpu().numpy(), oo)
    np.testing.assert_array_equal(size.cpu().numpy(), os_)
    assert np.array_equal(order.cpu().numpy()[:, :2], top2.cpu().numpy()[:, :, 0])


# ----------------------------------------------------------------------------
# direct-exposure gain, Eq. (4)

GAIN_KEYS = ("gain", "makespan", "window_gain", "window_makespan")


def assert_gain_equal(sf, d, bt, window):
    out = sf.sf_exposure_gain(torch.from_numpy(np.ascontiguousarray(d)).to(DEV),
                              torch.from_numpy(np.ascontiguousarray(bt)).to(DEV), window)
    torch.cuda.synchronize()
    o = oracle.exposure_gain(d, bt, window)
    for k in GAIN_KEYS:
        np.testing.assert_array_equal(out[k].cpu().numpy(), o[k], err_msg=k)


@pytest.mark.parametrize("R", [1, 2, 3, 15, 16, 17, 31, 64, 65, 127, 128, 129, 255, 256, 257,
                               1000, 1024, 1025, 4096, 5000, 16384])
def test_gain_rank_sweep(sf, R):
    rng = np.random.Generator(np.random.PCG64(R))
    for S, window in [(6, 4), (12, 5)]:
        T = max(2, min(24, 60000 // (R * S)))
        d = rng.integers(0, 10**6, size=(T, S, R), dtype=np.int64)
        W = -(-T // window)
        bt = rng.integers(0, 10**6, size=(W, S, R), dtype=np.int64)
        print("case R=%d S=%d T=%d" % (R, S, T), flush=True)
        assert_gain_equal(sf, d, bt, window)


@pytest.mark.parametrize("S", [1, 2, 4, 5, 6, 7, 8, 9, 12, 13, 16, 17, 24, 25, 32, 33, 64, 65, 128,
                               200])
def test_gain_stage_sweep(sf, S):
    rng = np.random.Generator(np.random.PCG64(S + 100))
    for R in (8, 200, 1030):
        T = max(2, min(12, 40000 // (R * S)))
        d = rng.integers(0, 4, size=(T, S, R), dtype=np.int64)        # heavy ties
        bt = rng.integers(0, 4, size=(-(-T // 3), S, R), dtype=np.int64)
        print("case R=%d S=%d T=%d" % (R, S, T), flush=True)
        assert_gain_equal(sf, d, bt, 3)


def test_gain_many_stages_wide_values(sf):
    """Past 64 stages (the two-pass kernel): several rank tiles with a
    ragged last one, odd ranks (8-byte loads), wide values, a window
    boundary inside a workgroup's steps."""
    rng = np.random.Generator(np.random.PCG64(128))
    for T, S, R, window, hi in ((9, 128, 16384, 4, 10**9), (13, 100, 301, 5, 1 << 40),
                                (6, 65, 129, 2, 3)):
        d = rng.integers(0, hi, size=(T, S, R), dtype=np.int64)
        bt = rng.integers(0, hi, size=(-(-T // window), S, R), dtype=np.int64)
        print("case T=%d S=%d R=%d window=%d" % (T, S, R, window), flush=True)
        assert_gain_equal(sf, d, bt, window)


@pytest.mark.parametrize("S,R,T,window,hi", [
    (1, 2048, 40, 7, 10**6), (3, 2050, 30, 8, 10**6), (4, 4096, 700, 1000, 10**6),
    (5, 2560, 20, 3, 1 << 40), (8, 16384, 150, 100, 10**9), (9, 3000, 16, 5, 4),
    (13, 2048, 12, 4, 10**6), (16, 2048, 12, 5, 1 << 40),
    (1, 4098, 40, 7, 10**6), (3, 8192, 30, 8, 10**6), (5, 6000, 20, 3, 1 << 40),
    (13, 16384, 12, 4, 10**6), (16, 10000, 12, 5, 10**6), (9, 5002, 16, 5, 4),
    (12, 8192, 10, 5, 1 << 28), (7, 12288, 25, 6, 10**8)])
def test_gain_rank_tiles(sf, S, R, T, window, hi):
    """From 2048 ranks and up to 16 stages (even R, aligned): several
    512-rank tiles per step with a ragged last one, T below the window, a
    ragged last window, heavy ties, and values past 2^32; past 4096 ranks
    the near-frontier pass, full and ragged workgroups, steps with totals
    past 2^32 next to steps below it in one launch."""
    rng = np.random.Generator(np.random.PCG64(S * 7919 + R))
    d = rng.integers(0, hi, size=(T, S, R), dtype=np.int64)
    bt = rng.integers(0, hi, size=(-(-T // window), S, R), dtype=np.int64)
    print("case S=%d R=%d T=%d window=%d" % (S, R, T, window), flush=True)
    assert_gain_equal(sf, d, bt, window)


def test_gain_large_gain_column(sf):
    """Stage 2 carries more than 2^32 on every rank, so replacing it puts
    every candidate more than 2^32 below F (a gain past 4.3 s)."""
    rng = np.random.Generator(np.random.PCG64(4242))
    T, S, R, window = 10, 6, 4096, 3
    d = rng.integers(0, 1000, size=(T, S, R), dtype=np.int64)
    d[:, 2, :] += (1 << 34) + rng.integers(0, 1 << 20, size=(T, R))
    bt = rng.integers(0, 10, size=(-(-T // window), S, R), dtype=np.int64)
    assert_gain_equal(sf, d, bt, window)


def test_gain_stalled_near_frontier(sf):
    """Forty ranks stalled in one stage hold the frontier; replacing that
    stage drops all of them below ranks far from F, so the largest
    replaced-stage total comes from a rank outside the ranks near F (values
    below 2^32)."""
    rng = np.random.Generator(np.random.PCG64(515))
    for R, S in ((4096, 6), (16384, 12), (6000, 4)):
        T, window = 8, 3
        d = rng.integers(0, 1000, size=(T, S, R), dtype=np.int64)
        d[:, 1, :40] += 10**6 + rng.integers(0, 1000, size=(T, 40))
        bt = rng.integers(0, 10, size=(-(-T // window), S, R), dtype=np.int64)
        print("case R=%d S=%d" % (R, S), flush=True)
        assert_gain_equal(sf, d, bt, window)


def test_gain_wide_steps_among_narrow(sf):
    """Past 4096 ranks: the odd steps hold a duration past 2^32 (their
    totals span more than 2^32: the bound's radix passes run in 64 bits),
    the even ones stay below (32-bit passes), in one launch."""
    rng = np.random.Generator(np.random.PCG64(717))
    T, S, R, window = 9, 12, 8192, 4
    d = rng.integers(0, 1 << 28, size=(T, S, R), dtype=np.int64)
    d[1::2, 3, 77] += 1 << 32
    bt = rng.integers(0, 1 << 28, size=(-(-T // window), S, R), dtype=np.int64)
    assert_gain_equal(sf, d, bt, window)


def test_gain_near_frontier_random_shapes(sf):
    """Random shapes past 4096 ranks with stalls of random size on random
    ranks (large gains force the second pass over all ranks, small ones
    stay in the near set) and a baseline from the window median or random."""
    rng = np.random.Generator(np.random.PCG64(8086))
    for case in range(24):
        R = 2 * int(rng.integers(2049, 8193))
        S = int(rng.integers(1, 17))
        T = int(rng.integers(1, 9))
        window = int(rng.integers(1, 6))
        scale = int(rng.choice([10, 10**4, 10**6, 1 << 26]))
        d = rng.integers(0, scale, size=(T, S, R), dtype=np.int64)
        for _ in range(int(rng.integers(0, 4))):
            r0 = int(rng.integers(0, R))
            nr = int(rng.integers(1, 64))
            d[:, int(rng.integers(0, S)), r0:r0 + nr] += int(rng.integers(1, 100)) * scale
        W = -(-T // window)
        if case % 2:
            bt = oracle.window_median(d, window)
        else:
            bt = rng.integers(0, scale, size=(W, S, R), dtype=np.int64)
        print("case %d R=%d S=%d T=%d window=%d scale=%d" % (case, R, S, T, window, scale), flush=True)
        assert_gain_equal(sf, d, bt, window)


def test_gain_many_ranks_tied_at_frontier(sf):
    """600 ranks share the largest total (more than the near-frontier set
    holds) and the rest trail: the step is resolved from all ranks; then
    every total equal."""
    rng = np.random.Generator(np.random.PCG64(616))
    T, S, R, window = 6, 5, 8192, 4
    d = rng.integers(0, 1000, size=(T, S, R), dtype=np.int64)
    d[:, :, :600] = 5000
    bt = rng.integers(0, 3000, size=(-(-T // window), S, R), dtype=np.int64)
    assert_gain_equal(sf, d, bt, window)
    d[:, :, :] = 777
    assert_gain_equal(sf, d, bt, window)


def test_gain_golden_cases(sf):
    import pins
    pins.pin_gain_sync_wait(lambda d, b, w: {k: v.cpu().numpy() for k, v in sf.sf_exposure_gain(
        torch.from_numpy(d).to(DEV), torch.from_numpy(np.ascontiguousarray(b)).to(DEV), w).items()})
    pins.pin_gain_direct(lambda d, b, w: {k: v.cpu().numpy() for k, v in sf.sf_exposure_gain(
        torch.from_numpy(d).to(DEV), torch.from_numpy(np.ascontiguousarray(b)).to(DEV), w).items()})


def test_gain_odd_rank_count_and_misaligned(sf):
    rng = np.random.Generator(np.random.PCG64(7))
    T, S, R = 10, 6, 301
    d = rng.integers(0, 10**6, size=(T, S, R), dtype=np.int64)
    bt = rng.integers(0, 10**6, size=(2, S, R), dtype=np.int64)
    assert_gain_equal(sf, d, bt, 5)
    R = 300
    d = rng.integers(0, 10**6, size=(T, S, R), dtype=np.int64)
    bt = rng.integers(0, 10**6, size=(2, S, R), dtype=np.int64)
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    out = sf.sf_exposure_gain(flat[1:].view(T, S, R), torch.from_numpy(bt).to(DEV), 5)
    torch.cuda.synchronize()
    o = oracle.exposure_gain(d, bt, 5)
    for k in GAIN_KEYS:
        np.testing.assert_array_equal(out[k].cpu().numpy(), o[k], err_msg=k)


# ----------------------------------------------------------------------------
# lag over the median rank (Sec. 4)

def assert_lag_equal(sf, d):
    lag, inc = sf.sf_frontier_lag(torch.from_numpy(np.ascontiguousarray(d)).to(DEV))
    torch.cuda.synchronize()
    ol, oi = oracle.frontier_lag(d)
    np.testing.assert_array_equal(lag.cpu().numpy(), ol)
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)


@pytest.mark.parametrize("R", [1, 2, 3, 7, 64, 65, 127, 128, 129, 256, 300, 512, 513, 1000,
                               1024, 2047, 4096, 5000, 8192, 10001, 16384])
def test_lag_rank_sweep(sf, R):
    rng = np.random.Generator(np.random.PCG64(R + 7))
    T = max(2, min(40, 200000 // (R * 6)))
    for hi in (3, 10**6, 1 << 40):               # ties, moderate, wide range (6 radix passes)
        d = rng.integers(0, hi + 1, size=(T, 6, R), dtype=np.int64)
        d[0] = 5                                 # a step where every prefix is equal
        if R > 2:
            d[1, 2, R // 3] += 1 << 44           # one outlier rank
        print("case R=%d hi=%d T=%d" % (R, hi, T), flush=True)
        assert_lag_equal(sf, d)


@pytest.mark.parametrize("R", [1024, 2048, 4096, 8192, 16384])
def test_narrow_pass_hand_over(sf, R):
    """At 1024 to 16384 ranks the raw spread, and at 8192 and 16384 the lag,
    run on 32-bit values and hand a step whose values leave 32 bits to the
    64-bit kernel:
    a duration of 2^32 or more, a rebased prefix that carries past 2^32 at
    a later stage, an overflow at the last stage only, neighbours that stay
    narrow, and every step handed over; all against the oracle."""
    rng = np.random.Generator(np.random.PCG64(R + 23))
    T, S = 10, 5
    d = rng.integers(0, 10**7, size=(T, S, R), dtype=np.int64)
    d[2, 2, R // 3] = (1 << 32) + 5              # a duration past 32 bits
    d[4, 0, 7] = 3 * 10**9                       # the prefix spread carries at stage 1
    d[4, 1, 7] = 3 * 10**9
    d[6, S - 1, R - 1] = 1 << 33                 # the last stage only
    d[8, :4, 5] = 10**9                          # 4e9 after four stages: still narrow
    d[9, 0, 0] = (1 << 32) - 1                   # the largest narrow duration
    print("case R=%d mixed" % R, flush=True)
    assert_lag_equal(sf, d)
    assert_spread_equal(sf, d, 3)
    wide = rng.integers(1 << 32, 1 << 40, size=(3, 2, R), dtype=np.int64)
    print("case R=%d all handed over" % R, flush=True)
    assert_lag_equal(sf, wide)
    assert_spread_equal(sf, wide, 2)



@pytest.mark.parametrize("R", [16385, 16386, 20000, 32767, 32768, 40000, 65536])
def test_lag_spread_past_16384_ranks(sf, R):
    """More ranks than a step holds in 64-bit registers: up to 32768 the
    32-bit pass with 32 values per lane (partial last tile for R below it)
    and the streaming 64-bit kernel for the steps it hands over; odd R and
    more than 32768 ranks the streaming kernel alone.  Tie-heavy and wide
    values, and steps forced past 32 bits (a duration of 2^32 + 5, a prefix
    spread past 2^32 at a later stage) next to steps that stay narrow."""
    rng = np.random.Generator(np.random.PCG64(R))
    T, S = 5, 4
    for hi in (3, 10**8):
        d = rng.integers(0, hi, size=(T, S, R), dtype=np.int64)
        if hi > 3:
            d[1, 2, R // 3] = (1 << 32) + 5
            d[3, :, R - 1] = [1 << 30, 1 << 31, 1 << 31, 5]
        print("case R=%d hi=%d" % (R, hi), flush=True)
        dd = torch.from_numpy(d).to(DEV)
        lag, inc = sf.sf_frontier_lag(dd)
        sp, wsp = sf.sf_rank_spread(dd, 2)
        torch.cuda.synchronize()
        ol, oi = oracle.frontier_lag(d)
        np.testing.assert_array_equal(lag.cpu().numpy(), ol)
        np.testing.assert_array_equal(inc.cpu().numpy(), oi)
        osp, owsp = oracle.rank_spread(d, 2)
        np.testing.assert_array_equal(sp.cpu().numpy(), osp)
        np.testing.assert_array_equal(wsp.cpu().numpy(), owsp)


@pytest.mark.parametrize("R", [4096, 16384])
def test_lag_spread_misaligned_large(sf, R):
    """A base 8 bytes past 16-byte alignment takes the 8-byte-load shapes
    (64-bit, full tiles) at the rank counts whose aligned calls take the
    32-bit pass; wide and narrow values alike."""
    rng = np.random.Generator(np.random.PCG64(R + 29))
    T, S = 6, 3
    d = rng.integers(0, 10**7, size=(T, S, R), dtype=np.int64)
    d[2, 1, 5] = 1 << 35
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    dd = flat[1:].view(T, S, R)
    print("case R=%d misaligned" % R, flush=True)
    lag, inc = sf.sf_frontier_lag(dd)
    sp, wsp = sf.sf_rank_spread(dd, 4)
    torch.cuda.synchronize()
    ol, oi = oracle.frontier_lag(d)
    osp, owsp = oracle.rank_spread(d, 4)
    np.testing.assert_array_equal(lag.cpu().numpy(), ol)
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(sp.cpu().numpy(), osp)
    np.testing.assert_array_equal(wsp.cpu().numpy(), owsp)


@pytest.mark.parametrize("S", [1, 2, 12, 100, 512])
def test_lag_stage_sweep(sf, S):
    rng = np.random.Generator(np.random.PCG64(S + 11))
    for R in (9, 1030):
        T = max(2, min(16, 100000 // (R * S)))
        d = rng.integers(0, 10**7, size=(T, S, R), dtype=np.int64)
        assert_lag_equal(sf, d)


def test_lag_stall_and_odd_base(sf):
    import pins
    lag, inc = sf.sf_frontier_lag(torch.from_numpy(pins.stall_case()).to(DEV))
    torch.cuda.synchronize()
    assert lag.cpu().numpy()[0].tolist() == [30 * pins.MS, 30 * pins.MS, 0, 0, 0, 0]
    T, S, R = 7, 5, 402
    d = synth.random_durations(T, S, R, seed=3, hi=10**5)
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    lag, inc = sf.sf_frontier_lag(flat[1:].view(T, S, R))
    torch.cuda.synchronize()
    ol, oi = oracle.frontier_lag(d)
    np.testing.assert_array_equal(lag.cpu().numpy(), ol)
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)


# ----------------------------------------------------------------------------
# raw rank spread (Sec. 6.2)

def _spread_fn(sf):
    def f(d, window):
        sp, wsp = sf.sf_rank_spread(torch.from_numpy(np.ascontiguousarray(d)).to(DEV), window)
        torch.cuda.synchronize()
        return sp.cpu().numpy(), wsp.cpu().numpy()
    return f


def assert_spread_equal(sf, d, window):
    sp, wsp = _spread_fn(sf)(d, window)
    osp, owsp = oracle.rank_spread(d, window)
    np.testing.assert_array_equal(sp, osp)
    np.testing.assert_array_equal(wsp, owsp)


@pytest.mark.parametrize("R", [1, 2, 3, 7, 64, 127, 128, 129, 256, 300, 513, 1000, 1024, 2047,
                               4096, 5000, 8192, 10001, 16384])
def test_spread_rank_sweep(sf, R):
    rng = np.random.Generator(np.random.PCG64(R + 17))
    T = max(2, min(40, 200000 // (R * 6)))
    for hi in (3, 10**6, 1 << 40):
        d = rng.integers(0, hi + 1, size=(T, 6, R), dtype=np.int64)
        d[0] = 5                                 # a step where every duration is equal
        if R > 2:
            d[1, 2, R // 3] += 1 << 44           # one outlier rank
        print("case R=%d hi=%d T=%d" % (R, hi, T), flush=True)
        assert_spread_equal(sf, d, 7)


def test_spread_pins_and_layouts(sf):
    import pins
    f = _spread_fn(sf)
    pins.pin_spread_stall(f)
    pins.pin_spread_invariants(f)
    pins.pin_spread_first_boundary_is_lag(
        f, lambda d: tuple(x.cpu().numpy() for x in sf.sf_frontier_lag(torch.from_numpy(d).to(DEV))))
    for S in (1, 12, 512):
        d = synth.random_durations(3, S, 33, seed=S, hi=10**6)
        assert_spread_equal(sf, d, 2)
    T, S, R = 7, 5, 402                          # 8-byte aligned base: 8-byte loads
    d = synth.random_durations(T, S, R, seed=4, hi=10**5)
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    sp, wsp = sf.sf_rank_spread(flat[1:].view(T, S, R), 3)
    torch.cuda.synchronize()
    osp, owsp = oracle.rank_spread(d, 3)
    np.testing.assert_array_equal(sp.cpu().numpy(), osp)
    np.testing.assert_array_equal(wsp.cpu().numpy(), owsp)


# ----------------------------------------------------------------------------
# per-rank window median, the baseline of Eq. (4)

def _median_fn(sf):
    def f(d, window):
        m = sf.sf_window_median(torch.from_numpy(np.ascontiguousarray(d)).to(DEV), window)
        torch.cuda.synchronize()
        return m.cpu().numpy()
    return f


def assert_median_equal(sf, d, window):
    np.testing.assert_array_equal(_median_fn(sf)(d, window), oracle.window_median(d, window))


@pytest.mark.parametrize("window", [1, 2, 3, 64, 100, 127, 128, 129, 250, 256, 257, 500, 512, 513,
                                    1000, 1024, 1025, 2048])
def test_median_window_sweep(sf, window):
    rng = np.random.Generator(np.random.PCG64(window + 23))
    T = 2 * window + window // 3 + 1             # a ragged last window
    for R, hi in ((16, 3), (33, 10**6), (5, 1 << 40)):
        d = rng.integers(0, hi + 1, size=(T, 3, R), dtype=np.int64)
        d[:, 1, 0] = 9                           # a constant series
        d[min(T - 1, 3), 2, R // 2] += 1 << 44   # an outlier step
        print("case window=%d R=%d hi=%d T=%d" % (window, R, hi, T), flush=True)
        assert_median_equal(sf, d, window)


@pytest.mark.parametrize("R", [1, 2, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256,
                               257, 1000, 4097])
def test_median_rank_sweep(sf, R):
    """Rank counts at the edges of every tile width (32 ranks for windows
    of up to 1024 steps, 64 up to 512, 128 up to 256, 256 up to 128), odd
    counts (8-byte loads) and a partial last tile."""
    for window, T in ((100, 250), (200, 410), (400, 800), (1000, 1100)):
        d = synth.random_durations(T, 2, R, seed=R + window, hi=10**7)
        print("case R=%d window=%d T=%d" % (R, window, T), flush=True)
        assert_median_equal(sf, d, window)


@pytest.mark.parametrize("window", [100, 250, 1000])
def test_median_warm_start_edges(sf, window):
    """The warm start of the window median (a column's median bracketed
    around the same rank's median of the window before, or in a unit's
    first window around a median already found in the tile) must give the
    oracle's median whether the guess lands inside its bracket, just past
    its edge or far off, and when the bracket holds too many values: window
    scales that drift by 0 to 60% from one window to the next, ranks whose
    scales differ 50-fold inside one tile, constant columns and columns of
    mass ties (every value in the bracket), values next to 2^32 (no bracket
    fits below 2^32), zeros, and a ragged last window."""
    rng = np.random.Generator(np.random.PCG64(window))
    R, S = 96, 3
    shifts = [0.0, 0.004, -0.008, 0.012, 0.02, -0.03, 0.05, 0.5, -0.6, 1e-4]
    scale = np.cumprod([1.0] + [1.0 + x for x in shifts])   # one per window
    W = len(scale)
    T = window * (W - 1) + window // 2 + 1                   # ragged last window
    w_of_t = np.minimum(np.arange(T) // window, W - 1)
    noise = 1.0 + 0.1 * rng.standard_normal((T, S, R))
    d = np.rint(2e7 * scale[w_of_t][:, None, None] * noise).clip(1, None).astype(np.int64)
    d[:, :, R // 2:] *= 50                                   # a 50-fold scale change inside tile 1
    d[:, 1, 5] = 5_000_000                                   # a constant column
    ties = rng.random((T, R)) < 0.5
    d[:, 1, 40:60] = np.where(ties[:, 40:60], 7_000_000, d[:, 1, 40:60])  # mass ties at the median
    d[:, 2, R - 1] = (1 << 32) - 1 - rng.integers(0, 1000, size=T)        # next to 2^32
    d[:, 2, 0] = 0                                           # zeros
    d[:, 2, 1] = rng.integers(0, 3, size=T)                  # medians of 0, 1 or 2
    print("case window=%d T=%d R=%d" % (window, T, R), flush=True)
    assert_median_equal(sf, d, window)


def test_median_wide_and_narrow_tiles_mixed(sf):
    """Tiles whose values all fit 32 bits next to tiles with one value of
    2^32 or more (resolved in 64 bits from global memory): per stage, per
    window and per 32-rank tile, on all four tile widths."""
    for window, T, R in ((1000, 2000, 96), (500, 1000, 192), (250, 500, 384), (100, 200, 768)):
        d = synth.random_durations(T, 3, R, seed=window, hi=10**9)
        d[window + 7, 1, R // 2] = (1 << 32) + 5     # window 1, stage 1, a middle tile
        d[3, 0, R - 1] = (1 << 32) - 1               # the largest 32-bit value: narrow
        d[window - 1, 2, 0] = 1 << 45                # window 0, stage 2, tile 0
        print("case window=%d T=%d R=%d" % (window, T, R), flush=True)
        assert_median_equal(sf, d, window)


def test_median_pins_and_layouts(sf):
    import pins
    f = _median_fn(sf)
    for pin in pins.MEDIAN_PINS:
        pin(f)
    T, S, R = 40, 3, 30                          # 8-byte aligned base, even R
    d = synth.random_durations(T, S, R, seed=5, hi=10**8)
    flat = torch.zeros(T * S * R + 1, dtype=torch.int64, device=DEV)
    flat[1:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    m = sf.sf_window_median(flat[1:].view(T, S, R), 16)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(m.cpu().numpy(), oracle.window_median(d, 16))
    assert_median_equal(sf, synth.random_durations(5, 512, 3, seed=6, hi=100), 2)


def test_median_feeds_gain(sf):
    """The window median as the baseline of the direct-exposure gain."""
    d = synth.random_durations(60, 6, 40, seed=7, hi=10**7)
    dd = torch.from_numpy(d).to(DEV)
    m = sf.sf_window_median(dd, 20)
    out = sf.sf_exposure_gain(dd, m, 20)
    torch.cuda.synchronize()
    o = oracle.exposure_gain(d, oracle.window_median(d, 20), 20)
    for k in GAIN_KEYS:
        np.testing.assert_array_equal(out[k].cpu().numpy(), o[k])


# ----------------------------------------------------------------------------
# the checked frontier pass: outputs of sf_frontier, plus the data contract

def checked(sf, d, status=None):
    inc, lead, st = sf.sf_frontier_checked(torch.from_numpy(np.ascontiguousarray(d)).to(DEV),
                                           status=status)
    torch.cuda.synchronize()
    return inc.cpu().numpy(), lead.cpu().numpy(), int(st.cpu()[0])


@pytest.mark.parametrize("R", [1, 3, 8, 16, 31, 64, 100, 128, 255, 256, 511, 512, 1000, 1024,
                               2047, 2048, 4095, 4096, 5000, 16384])
def test_checked_rank_sweep(sf, R):
    """Every launch shape: clean data gives sf_frontier's outputs and a
    clear status; one violation at the last step, stage and rank is seen."""
    T, S = 5, 4
    d = synth.random_durations(T, S, R, seed=R + 3, hi=10**9)
    oi, ol = oracle.frontier(d)
    inc, lead, st = checked(sf, d)
    np.testing.assert_array_equal(inc, oi)
    np.testing.assert_array_equal(lead, ol)
    assert st == oracle.range_status(d) == 0
    for bad in (-1, 1 << 47, np.iinfo(np.int64).min):
        e = d.copy()
        e[T - 1, S - 1, R - 1] = bad
        assert checked(sf, e)[2] == oracle.range_status(e) == sf.SF_ERANGE, (R, bad)


def test_checked_prefix_bound(sf):
    """A prefix of 2^47 - 1 passes and the same prefix reaching 2^47 is
    flagged, on a rank in the middle of a several-tile row; the status word
    collects across calls and is never cleared by the library."""
    T, S, R = 3, 5, 3001
    lim = 1 << 47
    d = np.zeros((T, S, R), dtype=np.int64)
    d[1, :, 1777] = [lim // 4, lim // 4, lim // 4, lim // 8, lim // 8 - 1]
    assert checked(sf, d)[2] == oracle.range_status(d) == 0
    oi, ol = oracle.frontier(d)
    inc, lead, _ = checked(sf, d)
    np.testing.assert_array_equal(inc, oi)
    np.testing.assert_array_equal(lead, ol)
    e = d.copy()
    e[1, 4, 1777] += 1
    st = torch.zeros((1,), dtype=torch.int32, device=DEV)
    assert checked(sf, e, st)[2] == oracle.range_status(e) == sf.SF_ERANGE
    assert checked(sf, d, st)[2] == sf.SF_ERANGE          # kept, not cleared
    for pin in (pins_range_edges_gpu,):
        pin(sf)


def pins_range_edges_gpu(sf):
    import pins
    pins.pin_range_edges(lambda d: checked(sf, d)[2])
    pins.pin_range_library(lambda d: checked(sf, d)[2])


def test_median_window_longer_than_input(sf):
    """A window longer than the input is one window of all T steps: on the
    tiled kernel up to 1024 steps and on the column-streaming one above."""
    for T, window, R in ((300, 1024, 20), (1000, 5000, 33), (1, 7, 5), (129, 10**9, 2),
                         (1025, 5000, 4), (3001, 4000, 7)):
        d = synth.random_durations(T, 3, R, seed=T + R, hi=10**8)
        assert_median_equal(sf, d, window)


def test_entry_points_on_a_side_stream(sf):
    """Every entry point enqueues on the stream it is given (a default-
    priority side stream here) and gives the same results there."""
    d = synth.random_durations(40, 6, 300, seed=9, hi=10**7)
    dd = torch.from_numpy(d).to(DEV)
    oi, ol = oracle.frontier(d)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        inc, lead = sf.sf_frontier(dd, stream=side)
        cinc, clead, st = sf.sf_frontier_checked(dd, stream=side)
        ev = sf.sf_frontier_evidence(dd, stream=side)
        lag, laginc = sf.sf_frontier_lag(dd, stream=side)
        sp, wsp = sf.sf_rank_spread(dd, 8, stream=side)
        med = sf.sf_window_median(dd, 8, stream=side)
        gain = sf.sf_exposure_gain(dd, med, 8, stream=side)
        ex, cnt, top2 = sf.sf_window_summary(inc, lead, R=300, window=8, stream=side)
        le, letop2 = sf.sf_window_lead_exposed(inc, lead, R=300, window=8, stream=side)
        swc, elc = sf.sf_window_leader_switches(ev["leader"], ev["gap"], ev["ties"], 8, 10**5,
                                                stream=side)
        order, size = sf.sf_route(ex, stream=side)
    side.synchronize()
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(lead.cpu().numpy(), ol)
    np.testing.assert_array_equal(cinc.cpu().numpy(), oi)
    assert int(st.cpu()[0]) == 0
    np.testing.assert_array_equal(ev["gap"].cpu().numpy(), oracle.frontier_evidence(d)["gap"])
    np.testing.assert_array_equal(lag.cpu().numpy(), oracle.frontier_lag(d)[0])
    np.testing.assert_array_equal(sp.cpu().numpy(), oracle.rank_spread(d, 8)[0])
    om = oracle.window_median(d, 8)
    np.testing.assert_array_equal(med.cpu().numpy(), om)
    np.testing.assert_array_equal(gain["gain"].cpu().numpy(), oracle.exposure_gain(d, om, 8)["gain"])
    oe, oc, ot = oracle.window_summary(oi, ol, 300, 8)
    np.testing.assert_array_equal(ex.cpu().numpy(), oe)
    np.testing.assert_array_equal(top2.cpu().numpy(), ot)
    ole, olt = oracle.window_lead_exposed(oi, ol, 300, 8)
    np.testing.assert_array_equal(le.cpu().numpy(), ole)
    np.testing.assert_array_equal(letop2.cpu().numpy(), olt)
    oev = oracle.frontier_evidence(d)
    osw, oel = oracle.window_leader_switches(oev["lead"], oev["gap"], oev["ties"], 8, 10**5)
    np.testing.assert_array_equal(swc.cpu().numpy(), osw)
    np.testing.assert_array_equal(elc.cpu().numpy(), oel)
    oo, os_ = oracle.route(oe)
    np.testing.assert_array_equal(order.cpu().numpy(), oo)


def test_side_stream_outside_stream_context(sf):
    """Calls given a side stream while torch's current stream is another
    one: the status word the binding allocates is cleared on the side
    stream before the checked pass (so a violation is reported, not erased),
    and outputs the binding allocates belong to that stream."""
    T, S, R = 64, 5, 777
    d = synth.random_durations(T, S, R, seed=31, hi=10**8)
    d[T - 1, S - 1, R - 1] = -5  # outside the data contract
    dd = torch.from_numpy(d).to(DEV)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    # long work on the current stream first, so an unordered clear there
    # would land after the side stream's kernel
    big = torch.ones((1 << 26,), dtype=torch.int64, device=DEV)
    for _ in range(20):
        big.mul_(1)
    _, _, st = sf.sf_frontier_checked(dd, stream=side)
    inc, lead = sf.sf_frontier(dd, stream=side)
    side.synchronize()
    assert int(st.cpu()[0]) == oracle.range_status(d) == sf.SF_ERANGE
    torch.cuda.synchronize()
    clean = np.abs(d)
    dc = torch.from_numpy(clean).to(DEV)
    torch.cuda.synchronize()
    for _ in range(20):
        big.mul_(1)
    i2, l2, st2 = sf.sf_frontier_checked(dc, stream=side)
    side.synchronize()
    assert int(st2.cpu()[0]) == 0
    oi, ol = oracle.frontier(clean)
    np.testing.assert_array_equal(i2.cpu().numpy(), oi)
    np.testing.assert_array_equal(l2.cpu().numpy(), ol)
    torch.cuda.synchronize()
