"""Minimal-staleness bound of MSPipe (Sec. 3.2): the stage start/end time model
(Eq. 3 and Eq. 4) and the per-iteration minimal staleness k_i (constraints
C1-C3).

TEST INFRASTRUCTURE: the plain reference the library's solver
(``tgm_min_staleness``) is checked against.  Pure Python loops over small
inputs; no code is shared with the library.

Stages, numbered as in the paper: 1 sample, 2 feature fetch, 3 memory fetch,
4 MTGNN compute, 5 memory update.  Iterations are numbered 1..n; "iteration 0"
ends every stage at time 0 (nothing runs before the first iteration).

Readings (the paper leaves these open):
* C1 is read as the definition of the delayed fetch: iteration i's memory
  fetch starts at max(b_i^(3), e_{i-k}^(5)), once the update of iteration i-k
  is done.  C2 then requires that start plus tau^(3) to be no later than
  b_i^(4), which is e_{i-k}^(5) <= b_i^(4) - tau^(3) (b_i^(3) + tau^(3) <= b_i^(4)
  holds by Eq. 3).
* k_i ranges over 1 <= k < min(i, k_max) (C3).  If that range is empty
  (i <= 1, or k_max <= 1), iteration i is a warm-up iteration: it does not
  wait (App. D), reported as k_i = 0.  If no k in the range meets C2, k_i is
  the largest one, min(i, k_max) - 1, and the fetch stalls the compute stage
  by e_{i-k}^(5) + tau^(3) - b_i^(4).
"""
from __future__ import annotations


def stage_times(tau, n):
    """b[i][j], e[i][j] for i = 0..n and j = 1..5 (index 0 unused), by Eq. 3-4."""
    assert len(tau) == 5 and all(t >= 0 for t in tau)
    T = [0.0] + [float(t) for t in tau]           # T[j] = tau^(j)
    b = [[0.0] * 6 for _ in range(n + 1)]
    e = [[0.0] * 6 for _ in range(n + 1)]
    for i in range(1, n + 1):
        for j in range(1, 6):
            if j == 1:
                b[i][j] = e[i - 1][1]
            elif j == 2:
                b[i][j] = max(e[i][1], e[i - 1][3])   # waits for the previous memory fetch
            else:
                b[i][j] = max(e[i][j - 1], e[i - 1][j])
            e[i][j] = b[i][j] + T[j]
    return b, e


def min_staleness(tau, n, k_max):
    """Per iteration i = 1..n: (k_i, fetch start, stall).  See the readings above."""
    b, e = stage_times(tau, n)
    t3 = float(tau[2])
    out = []
    for i in range(1, n + 1):
        hi = min(i, k_max)          # k < hi
        if hi <= 1:
            out.append((0, b[i][3], 0.0))   # warm-up: no wait
            continue
        k = None
        for kk in range(1, hi):
            if e[i - kk][5] <= b[i][4] - t3:
                k = kk
                break
        if k is None:
            k = hi - 1
        start = max(b[i][3], e[i - k][5])
        out.append((k, start, max(0.0, start + t3 - b[i][4])))
    return out
