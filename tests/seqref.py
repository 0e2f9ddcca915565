"""Straight-line model of the memory-module stage for tiny streams.

Used only to pin the oracle.  It is written differently from the oracle on
purpose, so that a mistake in one is unlikely to be repeated in the other:

* sampling is a brute-force scan over every event;
* the snapshot of iteration i is rebuilt from scratch each iteration by
  replaying the write sets of iterations 0 .. i-1-s onto the initial state
  (the staleness rule of Eq. 2 with the paper's k = s + 1);
* the memory updater is ``torch.nn.GRUCell`` in fp64;
* attention is ``torch.nn.functional.scaled_dot_product_attention`` in fp64;
* the latest-message reduce is ``max`` over (t, e, role) tuples.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F


def brute_sample(src, dst, t, v, tq, nb):
    cands = [e for e in range(len(src)) if (src[e] == v or dst[e] == v) and t[e] < tq]
    cands.sort(key=lambda e: (t[e], e), reverse=True)
    cands = cands[:nb]
    nbr = [int(dst[e]) if src[e] == v else int(src[e]) for e in cands]
    return nbr, cands, [float(t[e]) for e in cands]


def run(wl, w, s, n_iters=None, init=None, first_batch=0):
    N, M, D_e, D_t, H, nb, B = wl.N, wl.M, wl.D_e, wl.D_t, wl.H, wl.nb, wl.B
    D_m = 2 * M + D_e
    d_h = M // H
    src, dst, t, neg = wl.src, wl.dst, wl.t, wl.neg
    f = wl.efeat if D_e > 0 else np.zeros((wl.E, 0), np.float32)
    tt = lambda a: torch.as_tensor(np.asarray(a, dtype=np.float64))

    gru = torch.nn.GRUCell(D_m + D_t, M).double()
    with torch.no_grad():
        gru.weight_ih.copy_(tt(w.W_ih)); gru.weight_hh.copy_(tt(w.W_hh))
        gru.bias_ih.copy_(tt(w.b_ih)); gru.bias_hh.copy_(tt(w.b_hh))
    omega, beta = tt(w.omega), tt(w.beta)
    phi = lambda dt: torch.cos(omega * float(dt) + beta)
    Wq, bq, Wk, bk = tt(w.W_q), tt(w.b_q), tt(w.W_k), tt(w.b_k)
    Wv, bv, Wo, bo = tt(w.W_v), tt(w.b_v), tt(w.W_o), tt(w.b_o)

    if init is None:
        init = dict(mem=np.zeros((N, M)), mem_ts=np.zeros(N), mail=np.zeros((N, D_m)),
                    mail_ts=np.zeros(N), ver=-np.ones(N, np.int64))
    writes = []      # list of dicts node -> row tuple, index = iteration
    out = []
    n_it = (wl.n_iters - first_batch) if n_iters is None else n_iters
    for i in range(n_it):
        st = {k: np.array(v, copy=True) for k, v in init.items()}
        for j in range(0, i - s):          # iterations 0 .. i-1-s
            for node, (m, mts, ml, mlts) in writes[j].items():
                st["mem"][node] = m; st["mem_ts"][node] = mts
                st["mail"][node] = ml; st["mail_ts"][node] = mlts; st["ver"][node] = j
        lo, hi = wl.batch(first_batch + i)
        roots = list(src[lo:hi]) + list(dst[lo:hi]) + list(neg[lo:hi])
        rts = list(t[lo:hi]) * 3
        samp = [brute_sample(src, dst, t, int(v), tq, nb) for v, tq in zip(roots, rts)]
        U = sorted(set(int(v) for v in roots) | set(u for sm in samp for u in sm[0]))
        pos = {u: k for k, u in enumerate(U)}
        snew = {}
        new_mem_ts = {}
        with torch.no_grad():
            for u in U:
                if st["ver"][u] >= 0:
                    x = torch.cat([tt(st["mail"][u]), phi(st["mail_ts"][u] - st["mem_ts"][u])])
                    snew[u] = gru(x[None], tt(st["mem"][u])[None])[0].numpy()
                    new_mem_ts[u] = st["mail_ts"][u]
                else:
                    snew[u] = np.array(st["mem"][u], copy=True)
                    new_mem_ts[u] = st["mem_ts"][u]
            hs = []
            for (v, tq, (nbr, eids, nts)) in zip(roots, rts, samp):
                sv = tt(snew[int(v)])
                q = F.linear(torch.cat([sv, phi(0.0)]), Wq, bq)
                if len(nbr) == 0:
                    a = torch.zeros(M, dtype=torch.float64)
                else:
                    kap = torch.stack([torch.cat([tt(snew[u]), tt(f[e]), phi(tq - te)])
                                       for u, e, te in zip(nbr, eids, nts)])
                    K = F.linear(kap, Wk, bk)
                    V = F.linear(kap, Wv, bv)
                    qh = q.view(H, 1, d_h)
                    Kh = K.view(-1, H, d_h).transpose(0, 1).contiguous()
                    Vh = V.view(-1, H, d_h).transpose(0, 1).contiguous()
                    a = F.scaled_dot_product_attention(qh, Kh, Vh).reshape(M)
                hs.append(torch.relu(F.linear(torch.cat([a, sv]), Wo, bo)).numpy())
        cands = {}
        for e in range(lo, hi):
            for role, node in ((0, int(src[e])), (1, int(dst[e]))):
                key = (float(t[e]), e, role)
                if node not in cands or key > cands[node]:
                    cands[node] = key
        W = {}
        winner = np.full(len(U), -1, np.int64)
        for node, (_, e, role) in cands.items():
            other = int(dst[e]) if role == 0 else int(src[e])
            mail = np.concatenate([snew[node], snew[other], f[e].astype(np.float64)])
            W[node] = (snew[node], new_mem_ts[node], mail, float(t[e]))
            winner[pos[node]] = 2 * e + role
        writes.append(W)
        out.append(dict(
            roots=np.array(roots), nbr=[sm[0] for sm in samp], eid=[sm[1] for sm in samp],
            nts=[sm[2] for sm in samp], U=np.array(U),
            f_mem=np.array([st["mem"][u] for u in U]), f_mem_ts=np.array([st["mem_ts"][u] for u in U]),
            f_mail=np.array([st["mail"][u] for u in U]),
            f_mail_ts=np.array([st["mail_ts"][u] for u in U]),
            f_ver=np.array([st["ver"][u] for u in U]),
            s_new=np.array([snew[u] for u in U]), new_mem_ts=np.array([new_mem_ts[u] for u in U]),
            h=np.array(hs), winner=winner))
    # final state: every write set applied
    st = {k: np.array(v, copy=True) for k, v in init.items()}
    for j, Wj in enumerate(writes):
        for node, (m, mts, ml, mlts) in Wj.items():
            st["mem"][node] = m; st["mem_ts"][node] = mts
            st["mail"][node] = ml; st["mail_ts"][node] = mlts; st["ver"][node] = j
    return out, st
