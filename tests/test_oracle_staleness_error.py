"""Pins for the oracle's exact memories (``x_mem``) and the staleness-error
measurement of MSPipe-S (Sec. 3.3, App. E.2).

* s = 0: a fetch is never stale, so the exact memories equal the fetched ones
  bit for bit (closed form);
* s > 0: the exact memories at iteration i equal the committed state of a
  second oracle run to iteration i-1 and flushed (every write set applied),
  a different code path (the queue's commit) from the one that builds x_mem;
* the errors: zero at s = 0; positive at s > 0 over the stale nodes; the
  mitigation changes only the stale rows, so the two errors over U differ
  exactly by the stale rows' contribution.
"""
import numpy as np

from oracle.staleness_error import staleness_errors, summarize
from workloads import make_weights, make_workload


def test_exact_equals_fetched_without_staleness(orc):
    wl = make_workload("tiny", E=4000, s=0)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    o = orc.Oracle(wl, w, s=0)
    for _ in range(wl.n_iters):
        r = o.step()
        np.testing.assert_array_equal(r.x_mem, r.f_mem)


def test_exact_equals_flushed_state(orc):
    wl = make_workload("tiny", E=5000, s=3)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    a = orc.Oracle(wl, w, s=3)
    checked = 0
    for i in range(wl.n_iters):
        r = a.step()
        if i in (1, 4, 9, 17):
            b = orc.Oracle(wl, w, s=3)
            for _ in range(i):
                b.step(want="light")
            b.flush()
            np.testing.assert_array_equal(r.x_mem, b.state()["mem"][r.U])
            checked += int((r.x_mem != r.f_mem).any(axis=1).sum())
    assert checked > 0   # the stale fetches really differ from the exact rows


def test_staleness_errors(orc):
    wl = make_workload("tiny", E=6000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    mit = dict(p=0.9, lam=0.5, K=4)
    rows = staleness_errors(orc, wl, w, 0, mit, 30)
    assert all(r[3] == 0.0 for r in rows)   # no staleness, no error
    rows = staleness_errors(orc, wl, w, 2, mit, 30)
    t = summarize(rows)
    assert t["stale"] > 0 and t["fetch_stale"] > 0
    for (_, _, ns, fu, mu, fs, ms) in rows:
        # rows outside the stale set are unchanged: the squared errors over U
        # differ by the stale rows' squared errors only
        assert abs((fu ** 2 - fs ** 2) - (mu ** 2 - ms ** 2)) <= 1e-9 * max(1.0, fu ** 2)
