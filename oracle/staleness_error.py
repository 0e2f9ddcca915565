"""Staleness error of the fetched memories, with and without MSPipe-S.

TEST INFRASTRUCTURE: runs the fp64 oracle only (no GPU code).

Sec. 5.5 (error reduction) and App. E.2 compare, per iteration i, the
Frobenius distance between the memories a stale fetch returns and the exact
memories, ||s~ - s||_F, with the distance after the similarity-based
mitigation, ||s^ - s||_F.  The exact memories are those a fetch without
staleness would read at the same point of the same run: the committed state
with every write set of iterations <= i-1 applied (the oracle's ``x_mem``).
Only stale nodes are changed by the mitigation, so the distance is reported
over the whole node set and over the stale nodes alone.

    python -m oracle.staleness_error --workload wiki --s 1 --p 0.99 --iters 120
"""
from __future__ import annotations

import argparse
import sys

import numpy as np


def staleness_errors(orc, wl, w, s: int, mitigation: dict, iters: int, first: int = 0,
                     init: dict | None = None):
    """Per iteration: (i, n_U, n_stale, err_fetch_U, err_mitig_U, err_fetch_stale,
    err_mitig_stale), from one mitigated run at staleness s."""
    o = orc.Oracle(wl, w, s=s, mitigation=mitigation)
    if init is not None:
        o.set_state(first, **init)
    out = []
    for _ in range(iters):
        r = o.step(want="all")
        if r is None:
            break
        st = r.m_stale
        fro = lambda a, b: float(np.linalg.norm(a - b))
        out.append((r.iter, r.n_U, len(st), fro(r.f_mem, r.x_mem), fro(r.m_mem, r.x_mem),
                    fro(r.f_mem[st], r.x_mem[st]), fro(r.m_mem[st], r.x_mem[st])))
    return out


def summarize(rows):
    """Totals over iterations: sqrt of summed squares, so the figures are the
    Frobenius norms of the stacked per-iteration differences."""
    a = np.array([r[3:] for r in rows]) if rows else np.zeros((0, 4))
    tot = np.sqrt((a ** 2).sum(axis=0)) if len(a) else np.zeros(4)
    return dict(iters=len(rows), stale=int(sum(r[2] for r in rows)),
                fetch_U=tot[0], mitig_U=tot[1], fetch_stale=tot[2], mitig_stale=tot[3])


def main(argv=None):
    import os
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import oracle as orc
    from workloads import make_weights, make_workload

    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="wiki")
    ap.add_argument("--s", type=int, default=None)
    ap.add_argument("--p", type=float, default=0.99)
    ap.add_argument("--lam", type=float, default=0.95)
    ap.add_argument("--K", type=int, default=10)
    ap.add_argument("--iters", type=int, default=120)
    args = ap.parse_args(argv)
    orc.build(force=False)
    wl = make_workload(args.workload)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    s = wl.s if args.s is None else args.s
    mit = dict(p=args.p, lam=args.lam, K=args.K)
    rows = staleness_errors(orc, wl, w, s, mit, args.iters)
    t = summarize(rows)
    print(f"{wl.name} s={s} p={args.p} lambda={args.lam} K={args.K}: {t['iters']} iterations, "
          f"{t['stale']} stale fetches")
    print(f"  ||s~ - s||_F over U      {t['fetch_U']:.6g}")
    print(f"  ||s^ - s||_F over U      {t['mitig_U']:.6g}")
    print(f"  ||s~ - s||_F stale nodes {t['fetch_stale']:.6g}")
    print(f"  ||s^ - s||_F stale nodes {t['mitig_stale']:.6g}")


if __name__ == "__main__":
    main()
