"""The five full-size workloads, run exactly as the benchmark runs them
(the 16384-rank workload in two step-axis chunks), against the oracle over
every step and every window: bit-exact."""
import os
import time
from concurrent.futures import ThreadPoolExecutor

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


def log(msg):
    print("[%s] %s" % (time.strftime("%H:%M:%S"), msg), flush=True)


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_full_parity(sf, name):
    wl = synth.WORKLOADS[name]
    T, S, R = wl.T, wl.S, wl.R
    dev = torch.device("cuda:0")
    log("workload %s: T=%d S=%d R=%d window=%d chunks=%d (%.2f GB)"
        % (name, T, S, R, wl.window, wl.chunks, wl.input_bytes / 1e9))
    d = torch.empty((T, S, R), dtype=torch.int64, device=dev)
    oi = np.empty((T, S), dtype=np.int64)
    ol = np.empty((T, S), dtype=np.int32)
    bounds = wl.chunk_bounds()
    buf = np.empty((max(t1 - t0 for t0, t1 in bounds), S, R), dtype=np.int64)
    for t0, t1 in bounds:
        x = buf[: t1 - t0]
        synth.generate(wl, t0, t1, out=x)
        d[t0:t1].copy_(torch.from_numpy(x))
        oi[t0:t1], ol[t0:t1] = oracle.frontier(x)
        log("chunk [%d, %d) generated, copied, oracle done" % (t0, t1))
    del buf
    oe, oc, ot = oracle.window_summary(oi, ol, R, wl.window)

    inc = torch.empty((T, S), dtype=torch.int64, device=dev)
    lead = torch.empty((T, S), dtype=torch.int32, device=dev)
    for t0, t1 in bounds:
        sf.sf_frontier(d[t0:t1], inc[t0:t1], lead[t0:t1])
    ex, cnt, top2 = sf.sf_window_summary(inc, lead, R, wl.window)
    le, letop2 = sf.sf_window_lead_exposed(inc, lead, R, wl.window)
    torch.cuda.synchronize()
    log("gpu done")
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(lead.cpu().numpy(), ol)
    np.testing.assert_array_equal(ex.cpu().numpy(), oe)
    np.testing.assert_array_equal(cnt.cpu().numpy(), oc)
    np.testing.assert_array_equal(top2.cpu().numpy(), ot)
    ole, olt = oracle.window_lead_exposed(oi, ol, R, wl.window)
    np.testing.assert_array_equal(le.cpu().numpy(), ole)
    np.testing.assert_array_equal(letop2.cpu().numpy(), olt)
    # the tie workload exercises what it is meant to: every injected tie
    # that lands on the frontier (both ranks at the step's largest prefix;
    # the others were overtaken by a third rank or a later injection) is led
    # by the lower of its two ranks, and nearly all of them do land
    if wl.tie_frac:
        P_ties = 0
        injected = [e for e in synth.injections(wl) if e[1] == "tie"]
        assert len(injected) == round(wl.tie_frac * T * S)
        for t, kind, (s, r1, r2, _) in injected:
            x = synth.generate(wl, t, t + 1)[0]
            P = x[: s + 1].sum(axis=0)
            if P[r1] == P[r2] == P.max():
                assert ol[t, s] == min(r1, r2) == np.flatnonzero(P == P.max())[0], (t, s, r1, r2)
                P_ties += 1
        log("%d of %d injected ties are frontier ties" % (P_ties, len(injected)))
        assert P_ties >= 2300
    log("parity ok: %s" % name)
    del d, inc, lead, ex, cnt, top2, le, letop2
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_evidence_full_parity(sf, name):
    """sf_frontier_evidence over every step of every workload (per chunk)."""
    wl = synth.WORKLOADS[name]
    T, S, R = wl.T, wl.S, wl.R
    dev = torch.device("cuda:0")
    log("evidence %s" % name)
    bounds = wl.chunk_bounds()
    n_max = max(t1 - t0 for t0, t1 in bounds)
    d = torch.empty((n_max, S, R), dtype=torch.int64, device=dev)
    buf = np.empty((n_max, S, R), dtype=np.int64)
    keys = {"increment": "inc", "leader": "lead", "gap": "gap", "ties": "ties",
            "stage_max": "stage_max", "stage_sum": "stage_sum"}
    for t0, t1 in bounds:
        n = t1 - t0
        synth.generate(wl, t0, t1, out=buf[:n])
        d[:n].copy_(torch.from_numpy(buf[:n]))
        out = sf.sf_frontier_evidence(d[:n])
        o = oracle.frontier_evidence(buf[:n])
        torch.cuda.synchronize()
        for gk, ok in keys.items():
            np.testing.assert_array_equal(out[gk].cpu().numpy(), o[ok], err_msg=gk)
        # leader switches of the chunk's windows (chunks are window-aligned)
        for min_gap in (0, 10**6):
            sw, el = sf.sf_window_leader_switches(out["leader"], out["gap"], out["ties"], wl.window,
                                                  min_gap)
            osw, oel = oracle.window_leader_switches(o["lead"], o["gap"], o["ties"], wl.window,
                                                     min_gap)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(sw.cpu().numpy(), osw)
            np.testing.assert_array_equal(el.cpu().numpy(), oel)
        log("evidence and switches chunk [%d, %d) ok" % (t0, t1))
    del d, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_ingest_and_route(sf, name):
    """Ingest of the workload's per-rank buffers (first steps, up to 2000)
    against the oracle, and the routing set of all its windows."""
    wl = synth.WORKLOADS[name]
    T, S, R = wl.T, wl.S, wl.R
    n = min(T, 2000 if R <= 1024 else 400)
    d0 = synth.generate(wl, 0, n)
    x = d0[:, :-1, :].transpose(2, 0, 1).copy()        # per-rank [R][n][S-1]
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    w = d0.sum(axis=1).T.copy() + rng.integers(-10**6, 10**6, size=(R, n), dtype=np.int64)
    gd, go = sf.sf_ingest(torch.from_numpy(x).to("cuda:0"), torch.from_numpy(w).to("cuda:0"))
    torch.cuda.synchronize()
    od, oo = oracle.ingest(x, w)
    np.testing.assert_array_equal(gd.cpu().numpy(), od)
    np.testing.assert_array_equal(go.cpu().numpy(), oo)
    log("ingest ok: %s, %d steps" % (name, n))
    # routing set over every window of the workload (exposed totals from
    # the oracle's own pass over the generated steps)
    ex = np.empty((wl.num_windows, S), dtype=np.int64)
    for w0 in range(0, T, wl.window * max(1, 2000 // wl.window)):
        t1 = min(T, w0 + wl.window * max(1, 2000 // wl.window))
        oi, ol = oracle.frontier(synth.generate(wl, w0, t1))
        e, _, _ = oracle.window_summary(oi, ol, R, wl.window)
        ex[w0 // wl.window: w0 // wl.window + len(e)] = e
    go2, gs2 = sf.sf_route(torch.from_numpy(ex).to("cuda:0"))
    torch.cuda.synchronize()
    oo2, os2 = oracle.route(ex)
    np.testing.assert_array_equal(go2.cpu().numpy(), oo2)
    np.testing.assert_array_equal(gs2.cpu().numpy(), os2)
    log("route ok: %s, %d windows, sizes %s" % (name, len(ex), np.bincount(os2).tolist()))


def host_threads() -> int:
    """Oracle worker threads: the CPU share of the box (at most 16)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(16, n))


def whole_input(wl):
    """The workload's full [T, S, R] input on the host and in HBM."""
    x = synth.generate(wl)
    d = torch.from_numpy(x).to("cuda:0")
    return x, d


def window_ranges(wl, per=1):
    """[t0, t1) of runs of `per` whole windows covering all steps."""
    step = wl.window * per
    return [(t0, min(wl.T, t0 + step)) for t0 in range(0, wl.T, step)]


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_lag_spread_full(sf, name):
    """The lag over the median rank and the raw rank spread over every step
    of every workload, in the launch configuration the benchmark times (the
    16384-rank workload as two chunk launches), against the oracle run on
    disjoint step ranges (lag) and whole windows (spread) over the host's
    cores: every output bit-exact."""
    wl = synth.WORKLOADS[name]
    T, S, R = wl.T, wl.S, wl.R
    log("lag/spread %s: T=%d S=%d R=%d" % (name, T, S, R))
    x, d = whole_input(wl)
    lag = torch.empty((T, S), dtype=torch.int64, device="cuda:0")
    linc = torch.empty_like(lag)
    sp = torch.empty_like(lag)
    W = wl.num_windows
    wsp = torch.empty((W, S), dtype=torch.int64, device="cuda:0")
    for t0, t1 in wl.chunk_bounds():
        w0, w1 = t0 // wl.window, -(-t1 // wl.window)
        sf.sf_frontier_lag(d[t0:t1], lag[t0:t1], linc[t0:t1])
        sf.sf_rank_spread(d[t0:t1], wl.window, sp[t0:t1], wsp[w0:w1])
    torch.cuda.synchronize()
    log("gpu done")
    nth = host_threads()
    cuts = [T * k // (4 * nth) for k in range(4 * nth + 1)]
    with ThreadPoolExecutor(max_workers=nth) as pool:
        lag_parts = list(pool.map(lambda ab: oracle.frontier_lag(x[ab[0]:ab[1]]),
                                  [(a, b) for a, b in zip(cuts, cuts[1:]) if b > a]))
        log("oracle lag done")
        sp_parts = list(pool.map(lambda ab: oracle.rank_spread(x[ab[0]:ab[1]], wl.window),
                                 window_ranges(wl)))
        log("oracle spread done")
    np.testing.assert_array_equal(lag.cpu().numpy(), np.concatenate([p[0] for p in lag_parts]))
    np.testing.assert_array_equal(linc.cpu().numpy(), np.concatenate([p[1] for p in lag_parts]))
    np.testing.assert_array_equal(sp.cpu().numpy(), np.concatenate([p[0] for p in sp_parts]))
    np.testing.assert_array_equal(wsp.cpu().numpy(), np.concatenate([p[1] for p in sp_parts]))
    log("lag and spread ok: %s, all %d steps" % (name, T))
    del d, lag, linc, sp, wsp
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_median_gain_full(sf, name):
    """The per-rank window median of every window, stage and rank of every
    workload, and the direct-exposure gain of Eq. (4) over every step with
    that median as the baseline (the chain the benchmark times, chunk by
    chunk), against the oracle run window by window over the host's cores:
    every output bit-exact."""
    wl = synth.WORKLOADS[name]
    T, S, R = wl.T, wl.S, wl.R
    log("median/gain %s: T=%d S=%d R=%d window=%d" % (name, T, S, R, wl.window))
    x, d = whole_input(wl)
    W = wl.num_windows
    med = torch.empty((W, S, R), dtype=torch.int64, device="cuda:0")
    shapes = {"gain": (T, S), "makespan": (T,), "window_gain": (W, S), "window_makespan": (W,)}
    g = {k: torch.empty(v, dtype=torch.int64, device="cuda:0") for k, v in shapes.items()}
    for t0, t1 in wl.chunk_bounds():
        w0, w1 = t0 // wl.window, -(-t1 // wl.window)
        sf.sf_window_median(d[t0:t1], wl.window, med[w0:w1])
        sf.sf_exposure_gain(d[t0:t1], med[w0:w1], wl.window,
                            {"gain": g["gain"][t0:t1], "makespan": g["makespan"][t0:t1],
                             "window_gain": g["window_gain"][w0:w1],
                             "window_makespan": g["window_makespan"][w0:w1]})
    torch.cuda.synchronize()
    log("gpu done")

    def one_window(ab):
        t0, t1 = ab
        xs = x[t0:t1]
        om = oracle.window_median(xs, wl.window)
        return om, oracle.exposure_gain(xs, om, wl.window)

    with ThreadPoolExecutor(max_workers=host_threads()) as pool:
        parts = list(pool.map(one_window, window_ranges(wl)))
    log("oracle done")
    np.testing.assert_array_equal(med.cpu().numpy(), np.concatenate([p[0] for p in parts]))
    for k in shapes:
        np.testing.assert_array_equal(g[k].cpu().numpy(), np.concatenate([p[1][k] for p in parts]),
                                      err_msg=k)
    log("window median and gain ok: %s, all %d windows" % (name, W))
    del d, med, g
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_gain_no_stall_baseline(sf, name):
    """The direct-exposure gain of Eq. (4) on sampled step ranges of every
    workload, with the recipe's no-stall stage medians as the baseline."""
    wl = synth.WORKLOADS[name]
    S, R = wl.S, wl.R
    n = min(wl.T, 600 if R <= 1024 else 60)
    base = np.array([b * synth.MS for b in wl.base_ms], dtype=np.int64)
    for t0 in sorted({0, wl.T // 2, wl.T - n}):
        x = synth.generate(wl, t0, t0 + n)
        W = -(-n // wl.window)
        bt = np.broadcast_to(base.reshape(1, S, 1), (W, S, R)).copy()
        out = sf.sf_exposure_gain(torch.from_numpy(x).to("cuda:0"), torch.from_numpy(bt).to("cuda:0"),
                                  wl.window)
        torch.cuda.synchronize()
        o = oracle.exposure_gain(x, bt, wl.window)
        for k in ("gain", "makespan", "window_gain", "window_makespan"):
            np.testing.assert_array_equal(out[k].cpu().numpy(), o[k], err_msg=k)
    log("gain ok: %s (%d steps x 3 ranges)" % (name, n))
