"""The entry points inside a captured HIP graph: they allocate nothing, set
no memory with memset and never synchronise, so a sequence of calls can be
captured once and replayed.  Each replay here follows eager work that
refills the input in place, and every replay is checked against the oracle
on that replay's data."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
DEV = "cuda:0"


@pytest.fixture(scope="module")
def sf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_06751_amd import stagefrontier
    return stagefrontier


def test_captured_path_replays(sf):
    T, S, R, window = 40, 6, 300, 8
    W = sf.sf_num_windows(T, window)
    d_in = torch.empty((T, S, R), dtype=torch.int64, device=DEV)
    out = {
        "inc": torch.empty((T, S), dtype=torch.int64, device=DEV),
        "lead": torch.empty((T, S), dtype=torch.int32, device=DEV),
        "ex": torch.empty((W, S), dtype=torch.int64, device=DEV),
        "cnt": torch.empty((W, S, R), dtype=torch.int32, device=DEV),
        "top2": torch.empty((W, 2, 2), dtype=torch.int32, device=DEV),
        "le": torch.empty((W, S, R), dtype=torch.int64, device=DEV),
        "letop2": torch.empty((W, 2, 2), dtype=torch.int32, device=DEV),
        "ev": {k: torch.empty((T, S), dtype=torch.int32 if k in ("leader", "ties") else torch.int64,
                              device=DEV) for k in sf.EVIDENCE_FIELDS},
        "sw": torch.empty((W, S), dtype=torch.int32, device=DEV),
        "el": torch.empty((W, S), dtype=torch.int32, device=DEV),
        "lag": torch.empty((T, S), dtype=torch.int64, device=DEV),
        "laginc": torch.empty((T, S), dtype=torch.int64, device=DEV),
        "med": torch.empty((W, S, R), dtype=torch.int64, device=DEV),
        "gain": torch.empty((T, S), dtype=torch.int64, device=DEV),
        "mk": torch.empty((T,), dtype=torch.int64, device=DEV),
        "wgain": torch.empty((W, S), dtype=torch.int64, device=DEV),
        "wmk": torch.empty((W,), dtype=torch.int64, device=DEV),
    }

    def path(stream):
        sf.sf_frontier(d_in, out["inc"], out["lead"], stream=stream)
        sf.sf_window_summary(out["inc"], out["lead"], R, window, out["ex"], out["cnt"], out["top2"],
                             stream=stream)
        sf.sf_window_lead_exposed(out["inc"], out["lead"], R, window, out["le"], out["letop2"],
                                  stream=stream)
        sf.sf_frontier_evidence(d_in, out["ev"], stream=stream)
        sf.sf_window_leader_switches(out["ev"]["leader"], out["ev"]["gap"], out["ev"]["ties"], window,
                                     1000, out["sw"], out["el"], stream=stream)
        sf.sf_frontier_lag(d_in, out["lag"], out["laginc"], stream=stream)
        sf.sf_window_median(d_in, window, out["med"], stream=stream)
        sf.sf_exposure_gain(d_in, out["med"], window,
                            {"gain": out["gain"], "makespan": out["mk"],
                             "window_gain": out["wgain"], "window_makespan": out["wmk"]},
                            stream=stream)

    # warm up on a side stream (as graph capture requires), then capture
    d_in.copy_(torch.from_numpy(synth.random_durations(T, S, R, seed=70, hi=10**6)))
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        path(side)
    torch.cuda.current_stream(DEV).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        path(torch.cuda.current_stream(DEV))
    torch.cuda.synchronize()

    for rep, hi in enumerate([3, 10**6, 10**9]):
        d = synth.random_durations(T, S, R, seed=80 + rep, hi=hi)
        d_in.copy_(torch.from_numpy(d))            # eager work between replays
        out["inc"].fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print("replay %d hi=%d" % (rep, hi), flush=True)
        oi, ol = oracle.frontier(d)
        oe, oc, ot = oracle.window_summary(oi, ol, R, window)
        olag, olaginc = oracle.frontier_lag(d)
        om = oracle.window_median(d, window)
        og = oracle.exposure_gain(d, om, window)
        np.testing.assert_array_equal(out["inc"].cpu().numpy(), oi)
        np.testing.assert_array_equal(out["lead"].cpu().numpy(), ol)
        np.testing.assert_array_equal(out["ex"].cpu().numpy(), oe)
        np.testing.assert_array_equal(out["cnt"].cpu().numpy(), oc)
        np.testing.assert_array_equal(out["top2"].cpu().numpy(), ot)
        ole, olt = oracle.window_lead_exposed(oi, ol, R, window)
        np.testing.assert_array_equal(out["le"].cpu().numpy(), ole)
        np.testing.assert_array_equal(out["letop2"].cpu().numpy(), olt)
        oev = oracle.frontier_evidence(d)
        np.testing.assert_array_equal(out["ev"]["gap"].cpu().numpy(), oev["gap"])
        osw, oel = oracle.window_leader_switches(oev["lead"], oev["gap"], oev["ties"], window, 1000)
        np.testing.assert_array_equal(out["sw"].cpu().numpy(), osw)
        np.testing.assert_array_equal(out["el"].cpu().numpy(), oel)
        np.testing.assert_array_equal(out["lag"].cpu().numpy(), olag)
        np.testing.assert_array_equal(out["laginc"].cpu().numpy(), olaginc)
        np.testing.assert_array_equal(out["med"].cpu().numpy(), om)
        np.testing.assert_array_equal(out["gain"].cpu().numpy(), og["gain"])
        np.testing.assert_array_equal(out["wgain"].cpu().numpy(), og["window_gain"])


def test_captured_narrow_pass_replays(sf):
    """The lag and the raw spread at 16384 ranks (the 32-bit pass plus the
    64-bit pass over the steps it hands over, two launches) captured once
    and replayed on inputs that hand over no step, some steps, then none
    again: the hand-over goes through the output itself, so every replay
    must stand alone."""
    T, S, R, window = 5, 3, 16384, 2
    W = sf.sf_num_windows(T, window)
    d_in = torch.empty((T, S, R), dtype=torch.int64, device=DEV)
    lag = torch.empty((T, S), dtype=torch.int64, device=DEV)
    laginc = torch.empty((T, S), dtype=torch.int64, device=DEV)
    sp = torch.empty((T, S), dtype=torch.int64, device=DEV)
    wsp = torch.empty((W, S), dtype=torch.int64, device=DEV)

    def path(stream):
        sf.sf_frontier_lag(d_in, lag, laginc, stream=stream)
        sf.sf_rank_spread(d_in, window, sp, wsp, stream=stream)

    def data(seed, wide_steps):
        d = synth.random_durations(T, S, R, seed=seed, hi=10**7)
        for t in wide_steps:
            d[t, 1, 100 + t] = (1 << 32) + t       # a duration past 32 bits
        return d

    d_in.copy_(torch.from_numpy(data(90, [])))
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        path(side)
    torch.cuda.current_stream(DEV).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        path(torch.cuda.current_stream(DEV))
    torch.cuda.synchronize()

    for rep, wide_steps in enumerate([[], [1, 4], [], [0, 1, 2, 3, 4], []]):
        d = data(91 + rep, wide_steps)
        d_in.copy_(torch.from_numpy(d))            # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        print("replay %d handed over %s" % (rep, wide_steps), flush=True)
        olag, olaginc = oracle.frontier_lag(d)
        osp, owsp = oracle.rank_spread(d, window)
        np.testing.assert_array_equal(lag.cpu().numpy(), olag)
        np.testing.assert_array_equal(laginc.cpu().numpy(), olaginc)
        np.testing.assert_array_equal(sp.cpu().numpy(), osp)
        np.testing.assert_array_equal(wsp.cpu().numpy(), owsp)
