"""Seeded random shapes through every entry point, against the oracle: step,
stage and rank counts drawn across the launch-shape boundaries, tie-heavy
and wide values, misaligned bases and chunked step axes (bit-exact)."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
DEV = "cuda:0"


@pytest.fixture(scope="module")
def sf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_06751_amd import stagefrontier
    return stagefrontier


def device_copy(d, offset):
    """d on the GPU, starting `offset` int64 elements into its allocation."""
    flat = torch.zeros(d.size + offset, dtype=torch.int64, device=DEV)
    flat[offset:] = torch.from_numpy(d.reshape(-1)).to(DEV)
    return flat[offset:].view(*d.shape)


def case(seed):
    rng = np.random.Generator(np.random.PCG64(1000 + seed))
    T = int(rng.integers(1, 300))
    S = int(rng.integers(1, 40))
    R = int(np.exp(rng.uniform(0, np.log(5000))))
    hi = [3, 1000, 10**9][seed % 3]
    d = rng.integers(0, hi + 1, size=(T, S, R), dtype=np.int64)
    window = int(rng.integers(1, T + 2))
    offset = int(rng.integers(0, 2))
    return d, window, offset


@pytest.mark.parametrize("seed", range(60))
def test_random_shape(sf, seed):
    d, window, offset = case(seed)
    T, S, R = d.shape
    print("case seed=%d T=%d S=%d R=%d window=%d offset=%d" % (seed, T, S, R, window, offset),
          flush=True)
    dd = device_copy(d, offset)
    oi, ol = oracle.frontier(d)

    # the path, in two chunks along the step axis
    cut = T // 2
    inc = torch.empty((T, S), dtype=torch.int64, device=DEV)
    lead = torch.empty((T, S), dtype=torch.int32, device=DEV)
    for t0, t1 in ((0, cut), (cut, T)):
        if t1 > t0:
            sf.sf_frontier(dd[t0:t1], inc[t0:t1], lead[t0:t1])
    ex, cnt, top2 = sf.sf_window_summary(inc, lead, R, window)
    le, letop2 = sf.sf_window_lead_exposed(inc, lead, R, window)
    cinc, clead, st = sf.sf_frontier_checked(dd)
    ev = sf.sf_frontier_evidence(dd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(inc.cpu().numpy(), oi)
    np.testing.assert_array_equal(lead.cpu().numpy(), ol)
    np.testing.assert_array_equal(cinc.cpu().numpy(), oi)
    np.testing.assert_array_equal(clead.cpu().numpy(), ol)
    assert int(st.cpu()[0]) == oracle.range_status(d) == 0
    oe, oc, ot = oracle.window_summary(oi, ol, R, window)
    np.testing.assert_array_equal(ex.cpu().numpy(), oe)
    np.testing.assert_array_equal(cnt.cpu().numpy(), oc)
    np.testing.assert_array_equal(top2.cpu().numpy(), ot)
    ole, olt = oracle.window_lead_exposed(oi, ol, R, window)
    np.testing.assert_array_equal(le.cpu().numpy(), ole)
    np.testing.assert_array_equal(letop2.cpu().numpy(), olt)
    oev = oracle.frontier_evidence(d)
    for k, ok in (("gap", "gap"), ("ties", "ties"), ("stage_max", "stage_max"),
                  ("stage_sum", "stage_sum")):
        np.testing.assert_array_equal(ev[k].cpu().numpy(), oev[ok], err_msg=k)
    min_gap = [0, 2, 10**6][seed % 3]
    swc, elc = sf.sf_window_leader_switches(ev["leader"], ev["gap"], ev["ties"], window, min_gap)
    torch.cuda.synchronize()
    osw, oel = oracle.window_leader_switches(oev["lead"], oev["gap"], oev["ties"], window, min_gap)
    np.testing.assert_array_equal(swc.cpu().numpy(), osw)
    np.testing.assert_array_equal(elc.cpu().numpy(), oel)

    # the selects
    lag, laginc = sf.sf_frontier_lag(dd)
    sp, wsp = sf.sf_rank_spread(dd, window)
    torch.cuda.synchronize()
    ol_, oli = oracle.frontier_lag(d)
    np.testing.assert_array_equal(lag.cpu().numpy(), ol_)
    np.testing.assert_array_equal(laginc.cpu().numpy(), oli)
    osp, owsp = oracle.rank_spread(d, window)
    np.testing.assert_array_equal(sp.cpu().numpy(), osp)
    np.testing.assert_array_equal(wsp.cpu().numpy(), owsp)
    med = sf.sf_window_median(dd, window)
    torch.cuda.synchronize()
    om = oracle.window_median(d, window)
    np.testing.assert_array_equal(med.cpu().numpy(), om)
    g = sf.sf_exposure_gain(dd, med, window)
    torch.cuda.synchronize()
    og = oracle.exposure_gain(d, om, window)
    for k in ("gain", "makespan", "window_gain", "window_makespan"):
        np.testing.assert_array_equal(g[k].cpu().numpy(), og[k], err_msg=k)
