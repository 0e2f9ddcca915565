"""Pins for the oracle's staleness mitigation (MSPipe-S, Sec. 3.3).

* gamma          -- numpy's inverted-CDF quantile (the nearest-rank definition);
* stale set, Omega and the blended rows -- re-derived by brute force in Python
  on tiny streams: neighbour sets from a scan over every event, similarity as
  Python set intersections, Omega by a plain sort;
* closed forms   -- lambda = 1 changes nothing; lambda = 0 with K = 1 copies the
  most similar node's memory; p = 1 leaves no node stale;
* invariants     -- every mitigated coordinate lies between the smallest and
  largest of the blended memories; a stale node without mail carries its
  mitigated memory through the memory update unchanged.
"""
import numpy as np
import pytest

from workloads import custom_workload, make_weights, make_workload


def _run(orc, wl, w, s, mit, iters):
    o = orc.Oracle(wl, w, s=s, mitigation=mit)
    out = []
    for _ in range(iters):
        r = o.step()
        if r is None:
            break
        out.append(r)
    return out


def _neighbour_sets(wl, ids, T):
    """Distinct other endpoints of each node's nb most recent events with t < T,
    by a scan over every event (ties in t to the larger event id)."""
    src, dst, t = wl.src, wl.dst, wl.t
    before = np.nonzero(t < T)[0]
    sets = []
    for v in ids:
        ev = [e for e in before if src[e] == v or dst[e] == v]
        ev.sort(key=lambda e: (t[e], e), reverse=True)
        nbrs = set()
        for e in ev[:wl.nb]:
            nbrs.add(int(dst[e]) if src[e] == v else int(src[e]))
        sets.append(nbrs)
    return sets


def _brute_force(wl, r, p, lam, K):
    T = wl.t[r.iter * wl.B]
    dt = T - r.f_mem_ts
    gamma = float(np.quantile(dt, p, method="inverted_cdf"))
    stale = [k for k in range(r.n_U) if dt[k] > gamma]
    active = [k for k in range(r.n_U) if dt[k] < gamma]
    sets = _neighbour_sets(wl, r.U, T)
    mem = r.f_mem.copy()
    omega = []
    for v in stale:
        cand = []
        for u in active:
            sim = len(sets[v] & sets[u])
            if sim > 0:
                cand.append((-sim, -r.f_mem_ts[u], int(r.U[u]), u))
        cand.sort()
        om = [c[3] for c in cand[:K]]
        omega.append(om + [-1] * (K - len(om)))
        if om:
            mem[v] = lam * r.f_mem[v] + (1 - lam) * r.f_mem[om].mean(axis=0)
    return gamma, np.array(stale, np.int32), np.array(omega, np.int32).reshape(-1, K), mem


@pytest.mark.parametrize("p", [0.0, 0.3, 0.5, 0.9, 0.99, 1.0])
@pytest.mark.parametrize("n", [1, 2, 7, 100, 1001])
def test_quantile_is_nearest_rank(orc, p, n):
    x = np.random.default_rng(n).integers(0, 50, n).astype(np.float64)   # many ties
    assert orc.quantile_nearest_rank(x, p) == np.quantile(x, p, method="inverted_cdf")


@pytest.fixture(scope="module")
def tiny_mitigated(orc):
    wl = make_workload("tiny", E=6000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    mit = dict(p=0.9, lam=0.95, K=4)
    return wl, w, mit, _run(orc, wl, w, 2, mit, 30)


def test_mitigation_matches_brute_force(tiny_mitigated):
    wl, _, mit, res = tiny_mitigated
    checked = 0
    for r in res[14::5]:   # iterations with stale nodes
        gamma, stale, omega, mem = _brute_force(wl, r, mit["p"], mit["lam"], mit["K"])
        assert r.m_gamma == gamma
        np.testing.assert_array_equal(r.m_stale, stale)
        np.testing.assert_array_equal(r.m_omega, omega)
        np.testing.assert_allclose(r.m_mem, mem, rtol=0, atol=1e-13)
        checked += len(stale)
    assert checked > 100


def test_mitigation_on_a_hand_built_stream(orc):
    # batch 0 gives every node mail; batch 1 updates and writes them all, so at
    # batch 2 (T = 20, s = 0) the memory times are 0:2 1:4 2:6 3:5 4:4 5:6 and
    # the gaps 18 16 14 15 16 14.  p = 0.8 over six nodes: gamma = the 5th
    # smallest = 16, node 0 alone is stale, nodes 2, 3, 5 are active.
    # Neighbour sets at T (nb = 4): N(0) = {3,4,5}, N(2) = {1,3,4},
    # N(3) = {1,2,4}, N(5) = {0,1,2}: common with N(0) 2, 1, 0 -> Omega = (2, 3)
    ev = [(0, 3, 1.0), (0, 4, 2.0), (1, 3, 3.0), (1, 4, 4.0), (2, 3, 5.0), (2, 5, 6.0),
          (0, 5, 7.0), (1, 2, 8.0), (3, 4, 9.0), (1, 3, 10.0), (2, 4, 11.0), (5, 1, 12.0),
          (0, 1, 20.0), (3, 4, 21.0)]
    src = np.array([e[0] for e in ev])
    dst = np.array([e[1] for e in ev])
    t = np.array([e[2] for e in ev])
    wl = custom_workload("hand", 6, src, dst, t, dst.copy(), None, M=4, D_t=4, H=1, nb=4,
                         B=6, s=0)
    w = make_weights(4, 0, 4, seed=3)
    mit = dict(p=0.8, lam=0.25, K=2)
    r = _run(orc, wl, w, 0, mit, 3)[2]
    np.testing.assert_array_equal(r.U, np.arange(6))
    np.testing.assert_array_equal(r.f_mem_ts, [2, 4, 6, 5, 4, 6])
    assert r.m_gamma == 16.0
    assert r.m_stale.tolist() == [0]
    assert r.m_omega.tolist() == [[2, 3]]
    want = 0.25 * r.f_mem[0] + 0.75 * (r.f_mem[2] + r.f_mem[3]) / 2
    np.testing.assert_allclose(r.m_mem[0], want, rtol=0, atol=1e-15)
    assert np.abs(r.f_mem[[0, 2, 3]]).min(axis=1).max() > 0    # real memories were blended
    gamma, stale, omega, mem = _brute_force(wl, r, mit["p"], mit["lam"], mit["K"])
    assert (gamma, stale.tolist(), omega.tolist()) == (16.0, [0], [[2, 3]])


def test_lambda_one_changes_nothing(orc):
    wl = make_workload("tiny", E=5000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    res = _run(orc, wl, w, 2, dict(p=0.9, lam=1.0, K=4), 20)
    assert sum(len(r.m_stale) for r in res) > 0
    for r in res:
        np.testing.assert_array_equal(r.m_mem, r.f_mem)


def test_lambda_zero_k_one_copies_most_similar(orc):
    wl = make_workload("tiny", E=5000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    res = _run(orc, wl, w, 2, dict(p=0.9, lam=0.0, K=1), 20)
    n = 0
    for r in res:
        for v, om in zip(r.m_stale, r.m_omega):
            if om[0] >= 0:
                np.testing.assert_array_equal(r.m_mem[v], r.f_mem[om[0]])
                n += 1
    assert n > 0


def test_quantile_one_leaves_no_stale_node(orc):
    wl = make_workload("tiny", E=5000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    for r in _run(orc, wl, w, 2, dict(p=1.0, lam=0.5, K=4), 20):
        assert len(r.m_stale) == 0
        np.testing.assert_array_equal(r.m_mem, r.f_mem)


def test_mitigated_rows_are_convex_blends(tiny_mitigated):
    _, _, _, res = tiny_mitigated
    for r in res:
        for v, om in zip(r.m_stale, r.m_omega):
            rows = [r.f_mem[v]] + [r.f_mem[u] for u in om if u >= 0]
            lo, hi = np.min(rows, axis=0), np.max(rows, axis=0)
            assert np.all(r.m_mem[v] >= lo - 1e-15) and np.all(r.m_mem[v] <= hi + 1e-15)
        other = np.setdiff1d(np.arange(r.n_U), r.m_stale)
        np.testing.assert_array_equal(r.m_mem[other], r.f_mem[other])


def test_update_consumes_mitigated_memory(tiny_mitigated):
    # a node without mail keeps its (mitigated) memory through the update
    _, _, _, res = tiny_mitigated
    n = 0
    for r in res:
        for v in r.m_stale:
            if r.f_ver[v] < 0:
                np.testing.assert_array_equal(r.s_new[v], r.m_mem[v])
                n += 1
    assert n > 0


def test_update_of_stale_node_with_mail_reads_blended_memory(orc):
    """Sec. 3.3's second equation: the memory update of a stale node takes the
    blended memory as its previous state.  For every stale node with mail the
    oracle's s' must equal an independent fp64 GRU (torch's GRUCell, with the
    input [mail || cos(omega (mail_ts - mem_ts) + beta)] formed here in numpy)
    of the blended row, and differ from the same GRU of the row as fetched."""
    torch = pytest.importorskip("torch")
    wl = make_workload("tiny", E=6000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    res = _run(orc, wl, w, 2, dict(p=0.9, lam=0.5, K=4), 30)
    M = wl.M
    cell = torch.nn.GRUCell(wl.D_m + wl.D_t, M).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(np.asarray(w.W_ih, np.float64)))
        cell.weight_hh.copy_(torch.from_numpy(np.asarray(w.W_hh, np.float64)))
        cell.bias_ih.copy_(torch.from_numpy(np.asarray(w.b_ih, np.float64)))
        cell.bias_hh.copy_(torch.from_numpy(np.asarray(w.b_hh, np.float64)))
    omega, beta = np.asarray(w.omega, np.float64), np.asarray(w.beta, np.float64)
    n = 0
    for r in res:
        for v in r.m_stale:
            if r.f_ver[v] < 0 or np.array_equal(r.m_mem[v], r.f_mem[v]):
                continue
            phi = np.cos(omega * (r.f_mail_ts[v] - r.f_mem_ts[v]) + beta)
            x = torch.from_numpy(np.concatenate([r.f_mail[v], phi]))[None]
            with torch.no_grad():
                blended = cell(x, torch.from_numpy(r.m_mem[v].copy())[None])[0].numpy()
                fetched = cell(x, torch.from_numpy(r.f_mem[v].copy())[None])[0].numpy()
            np.testing.assert_allclose(r.s_new[v], blended, rtol=0, atol=1e-12)
            assert np.abs(r.s_new[v] - fetched).max() > 1e-6
            n += 1
    assert n > 20
