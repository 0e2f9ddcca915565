"""The oracle resumed from a saved state with pending write sets (Eq. 2: a
read at iteration i sees exactly the writes of iterations <= i-1-s) equals
the run that was not interrupted, bit for bit.  The saved state is built from
independent oracle runs: the committed tables are a run through iteration
j-1-s, flushed; the pending write set of iteration k (j-s <= k <= j-1) is
the rows whose version is k after a run through k, flushed."""
import dataclasses

import numpy as np
import pytest

from workloads import make_weights, make_workload


def _run(orc, wl, w, n):
    o = orc.Oracle(wl, w)
    res = [o.step() for _ in range(n)]
    return o, res


@pytest.mark.parametrize("s,j", [(0, 5), (1, 6), (2, 9), (3, 4)])
def test_resume_with_pending_write_sets(orc, s, j):
    wl = make_workload("tiny", E=3000, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    n = 6
    _, straight = _run(orc, wl, w, j + n)
    first = j - s   # the pending write sets: iterations first .. j-1
    base, _ = _run(orc, wl, w, first)
    base.flush()
    T = base.state()
    pending = []
    for k in range(first, j):
        ok, _ = _run(orc, wl, w, k + 1)
        ok.flush()
        Tk = ok.state()
        sel = np.flatnonzero(Tk["ver"] == k)
        pending.append((k, sel.astype(np.int32), Tk["mem"][sel], Tk["mem_ts"][sel],
                        Tk["mail"][sel], Tk["mail_ts"][sel]))
    o = orc.Oracle(wl, w)
    o.set_state(j, T["mem"], T["mem_ts"], T["mail"], T["mail_ts"], T["ver"], pending=pending)
    for i in range(j, j + n):
        r = o.step()
        want = straight[i]
        for f in dataclasses.fields(r):
            a, b = getattr(r, f.name), getattr(want, f.name)
            if isinstance(a, np.ndarray):
                assert np.array_equal(a, b), (i, f.name)
            else:
                assert a == b, (i, f.name)


def test_pending_sets_must_grow(orc):
    wl = make_workload("tiny", E=3000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    o = orc.Oracle(wl, w)
    z = np.zeros((0, wl.M)), np.zeros(0)
    empty = (np.zeros(0, np.int32), z[0], z[1], np.zeros((0, wl.D_m)), z[1])
    with pytest.raises(AssertionError):
        o.set_state(5, np.zeros((wl.N, wl.M)), np.zeros(wl.N), np.zeros((wl.N, wl.D_m)),
                    np.zeros(wl.N), np.full(wl.N, -1, np.int32),
                    pending=[(4,) + empty, (3,) + empty])
