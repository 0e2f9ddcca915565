"""Pins for the oracle's APAN family (readings R32-R35): a mailbox of the K
latest mails per node, each mail delivered to its node and (propagation) to
the node's sampled neighbours, an attention over the mailbox feeding the
GRU, the updated memory as the embedding.

* reduction to TGN -- with one mail per mailbox and no propagation, the
  attention over a single mail returns that mail, so every updated memory
  and every table must equal the TGN oracle's bit for bit (the TGN oracle is
  pinned on its own);
* brute-force mailboxes -- every delivery of a run enumerated here from the
  events and the (pinned) sampler, in (t, e, role, slot) order; each node's
  committed mailbox must hold the last K of its deliveries: their times,
  edge features and memory parts exactly;
* closed forms -- W_k = 0 makes every score of a mailbox equal, so the
  aggregate is the mean of the mails; the update is then torch's fp64
  GRUCell of [mean || phi(newest - memory time)].
"""
import dataclasses

import numpy as np
import pytest

from workloads import make_weights, make_workload


def _run(orc, wl, w, s=None, n=None):
    o = orc.Oracle(wl, w, s=s)
    res = []
    for _ in range(wl.n_iters if n is None else n):
        res.append(o.step())
    return o, res


@pytest.mark.parametrize("s", [0, 2])
def test_one_mail_without_propagation_is_tgn(orc, s):
    wl = make_workload("tiny", E=4000, s=s)
    wt = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    wa = make_weights(wl.M, wl.D_e, wl.D_t, beta="random", model="apan", K_mb=1,
                      propagate=False)
    wa = dataclasses.replace(wa, W_ih=wt.W_ih, W_hh=wt.W_hh, b_ih=wt.b_ih, b_hh=wt.b_hh)
    ot, rt = _run(orc, wl, wt, s=s)
    oa, ra = _run(orc, wl, wa, s=s)
    for a, t in zip(ra, rt):
        assert np.array_equal(a.s_new, t.s_new)
        assert np.array_equal(a.new_mem_ts, t.new_mem_ts)
        assert np.array_equal(a.h, a.s_new[a.root_pos])
        assert np.array_equal(a.f_mb_cnt > 0, t.f_ver >= 0)
    ot.flush()
    oa.flush()
    st, sa = ot.state(), oa.state()
    for k in ("mem", "mem_ts", "ver"):
        assert np.array_equal(st[k], sa[k]), k
    mb, ts, cnt = oa.mailbox()
    has = st["ver"] >= 0
    assert np.array_equal(cnt > 0, has)
    assert np.array_equal(mb[has, 0], st["mail"][has])
    assert np.array_equal(ts[has, 0], st["mail_ts"][has])


def test_mailboxes_match_brute_force(orc):
    wl = make_workload("tiny", E=3000, s=0)
    K = 3
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=K, propagate=True)
    o, res = _run(orc, wl, w, s=0)
    o.flush()
    mb, ts, cnt = o.mailbox()
    M, D_e = wl.M, wl.D_e
    deliveries = {v: [] for v in range(wl.N)}
    for r in res:
        lo, hi = wl.batch(r.iter)
        b = hi - lo
        roots = np.concatenate([wl.src[lo:hi], wl.dst[lo:hi]])
        rts = np.concatenate([wl.t[lo:hi], wl.t[lo:hi]])
        nbr, _, _, c = orc.sample(wl.N, wl.src, wl.dst, wl.t, roots, rts, wl.nb)
        pos = {int(u): k for k, u in enumerate(r.U)}
        for k in range(b):
            e = lo + k
            for role in (0, 1):
                v = int(wl.src[e] if role == 0 else wl.dst[e])
                other = int(wl.dst[e] if role == 0 else wl.src[e])
                rr = role * b + k
                msg = np.concatenate([r.s_new[pos[v]], r.s_new[pos[other]],
                                      np.asarray(wl.efeat[e], np.float64)])
                for wv in [v] + [int(x) for x in nbr[rr, :c[rr]]]:
                    deliveries[wv].append((float(wl.t[e]), msg))
    checked = 0
    for v in range(wl.N):
        want = deliveries[v][-K:]
        assert cnt[v] == len(want), v
        for j, (t, msg) in enumerate(want):
            assert ts[v, j] == t
            assert np.array_equal(mb[v, j], msg)
            checked += 1
    assert checked > 1000 and (cnt == K).sum() > 100


def test_zero_key_weights_average_the_mailbox(orc):
    torch = pytest.importorskip("torch")
    wl = make_workload("tiny", E=3000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=4, beta="random")
    w = dataclasses.replace(w, W_k=np.zeros_like(w.W_k))
    _, res = _run(orc, wl, w, s=1)
    cell = torch.nn.GRUCell(wl.D_m + wl.D_t, wl.M).double()
    with torch.no_grad():
        for name in ("weight_ih", "weight_hh", "bias_ih", "bias_hh"):
            src = {"weight_ih": w.W_ih, "weight_hh": w.W_hh, "bias_ih": w.b_ih,
                   "bias_hh": w.b_hh}[name]
            getattr(cell, name).copy_(torch.from_numpy(np.asarray(src, np.float64)))
    om, be = np.asarray(w.omega), np.asarray(w.beta)
    n = 0
    for r in res[5:]:
        for k in np.flatnonzero(r.f_mb_cnt >= 2)[:20]:
            c = r.f_mb_cnt[k]
            mean = r.f_mb[k, :c].mean(axis=0)
            tref = r.f_mb_ts[k, c - 1]
            x = np.concatenate([mean, np.cos(om * (tref - r.f_mem_ts[k]) + be)])
            with torch.no_grad():
                want = cell(torch.from_numpy(x)[None],
                            torch.from_numpy(r.f_mem[k].copy())[None])[0].numpy()
            np.testing.assert_allclose(r.s_new[k], want, rtol=0, atol=1e-12)
            assert r.new_mem_ts[k] == tref
            n += 1
    assert n > 50


def test_scores_follow_the_age_of_each_mail(orc):
    """A weight set under which the attention reduces to a scalar function of
    each mail's age: W_q = 0 and b_q = e_0 make the query e_0; W_k holds only
    3 at the first time-code column, whose phase is beta_0 = pi/2 (omega_0 =
    1), so the score of mail j is 3 cos(age_j + pi/2) / sqrt(M) =
    -3 sin(age_j) / sqrt(M) with age_j = t_newest - t_j (the sign of the age
    matters).  The aggregate is the softmax of those scores over the mails."""
    torch = pytest.importorskip("torch")
    wl = make_workload("tiny", E=3000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=4, beta="random")
    beta = np.array(w.beta, np.float64)
    beta[0] = np.pi / 2
    Wk = np.zeros_like(w.W_k)
    Wk[0, wl.D_m] = 3.0
    bq = np.zeros_like(w.b_q)
    bq[0] = 1.0
    w = dataclasses.replace(w, beta=beta, W_q=np.zeros_like(w.W_q), b_q=bq, W_k=Wk,
                            b_k=np.zeros_like(w.b_k))
    assert np.asarray(w.omega)[0] == 1.0
    _, res = _run(orc, wl, w, s=1)
    cell = torch.nn.GRUCell(wl.D_m + wl.D_t, wl.M).double()
    with torch.no_grad():
        for name, src in (("weight_ih", w.W_ih), ("weight_hh", w.W_hh), ("bias_ih", w.b_ih),
                          ("bias_hh", w.b_hh)):
            getattr(cell, name).copy_(torch.from_numpy(np.asarray(src, np.float64)))
    n = 0
    for r in res[5:]:
        for k in np.flatnonzero(r.f_mb_cnt >= 3)[:20]:
            c = r.f_mb_cnt[k]
            t = r.f_mb_ts[k, :c]
            sc = -3.0 * np.sin(t[-1] - t) / np.sqrt(wl.M)
            al = np.exp(sc - sc.max())
            al /= al.sum()
            agg = (al[:, None] * r.f_mb[k, :c]).sum(axis=0)
            x = np.concatenate([agg, np.cos(np.asarray(w.omega) * (t[-1] - r.f_mem_ts[k]) +
                                            beta)])
            with torch.no_grad():
                want = cell(torch.from_numpy(x)[None],
                            torch.from_numpy(r.f_mem[k].copy())[None])[0].numpy()
            np.testing.assert_allclose(r.s_new[k], want, rtol=0, atol=1e-12)
            n += 1
    assert n > 50


def test_loaded_state_continues_the_run(orc):
    """set_state + set_mailbox at iteration j from a run's flushed tables:
    with s = 0 (every write set committed before the next fetch) the loaded
    oracle must continue exactly as the run itself; a mailbox loaded in the
    wrong order or with dropped counts changes the next attention."""
    wl = make_workload("tiny", E=4000, s=0)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random", model="apan", K_mb=4)
    j = 6
    a, _ = _run(orc, wl, w, s=0, n=j)
    a.flush()
    st = a.state()
    mb, mb_ts, cnt = a.mailbox()
    assert (cnt == 4).sum() > 0 and ((cnt > 0) & (cnt < 4)).sum() > 0
    b = orc.Oracle(wl, w, s=0)
    b.set_state(j, **st)
    b.set_mailbox(mb, mb_ts, cnt)
    for _ in range(4):
        ra, rb = a.step(), b.step()
        for k in ("f_mem", "f_mb", "f_mb_ts", "f_mb_cnt", "s_new", "h"):
            assert np.array_equal(getattr(ra, k), getattr(rb, k)), k
    # the same mails in reverse order: different scores, different updates
    c = orc.Oracle(wl, w, s=0)
    c.set_state(j, **st)
    rev = np.array(mb)
    rts = np.array(mb_ts)
    for v in np.nonzero(cnt > 1)[0]:
        rev[v, :cnt[v]] = mb[v, :cnt[v]][::-1]
        rts[v, :cnt[v]] = mb_ts[v, :cnt[v]][::-1]
    c.set_mailbox(rev, rts, cnt)
    a2 = orc.Oracle(wl, w, s=0)
    a2.set_state(j, **st)
    a2.set_mailbox(mb, mb_ts, cnt)
    assert not np.array_equal(c.step().s_new, a2.step().s_new)
    with pytest.raises(ValueError):
        c.set_mailbox(mb, mb_ts, np.full_like(cnt, 5))
