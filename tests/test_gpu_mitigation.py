"""GPU staleness mitigation (MSPipe-S, Sec. 3.3) through the C ABI against the
fp64 oracle, which applies the same readings.

Bit-exact: gamma, the stale positions and their Omega (positions in the node
set), and every index, time and version the stage produces.  Floating point:
the mitigated fetched memories and everything downstream (s', h, the committed
tables) within |gpu - oracle| <= 1e-5 + 1e-4 |oracle|.
"""
import dataclasses

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from test_gpu_parity import (compare_state, compare_step, exact, gdelt_prefix,  # noqa: E402
                             sparse_features, synthetic_state, tie_heavy, window_rows)
from workloads import make_weights, make_workload  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2402_15113_amd import tgm
    tgm.lib()   # fails loudly when the library is missing


def run_mitigated(orc, wl, w, mit, n_iters=None, s=None, first=0, init=None, gpu_efeat=None):
    """GPU stage (Stage.step: fetch, tgm_mitigate, update, embed) and oracle
    side by side; returns the number of stale nodes seen."""
    from paper_2402_15113_amd.stage import Stage
    s = wl.s if s is None else s
    efeat = wl.efeat if gpu_efeat is None else gpu_efeat
    st = Stage(wl.N, wl.src, wl.dst, wl.t, wl.neg, efeat, w, M=wl.M, D_t=wl.D_t, H=wl.H,
               nb=wl.nb, B=wl.B, s=s, mitigation=mit)
    o = orc.Oracle(wl, w, s=s, mitigation=mit)
    if init is not None:
        st.load_state(first, **init)
        o.set_state(first, **init)
    n = (wl.n_iters - first) if n_iters is None else n_iters
    seen = 0
    for k in range(n):
        i = first + k
        print(f"[mitigation] {wl.name} s={s} {mit} iter {i}", flush=True)
        st.step(i)
        r = o.step(want="all")
        gamma, stale, omega = st.mitigation_result()
        assert gamma == r.m_gamma, (gamma, r.m_gamma)
        exact("stale", stale, r.m_stale)
        exact("omega", omega, r.m_omega)
        seen += len(stale)
        # the fetch buffer holds the mitigated rows on the GPU side
        compare_step(st.outputs(), dataclasses.replace(r, f_mem=r.m_mem))
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()
    return seen


@pytest.mark.parametrize("s,mit", [(2, dict(p=0.9, lam=0.95, K=4)),
                                   (0, dict(p=0.75, lam=0.0, K=16)),
                                   (1, dict(p=0.5, lam=0.3, K=1))])
def test_mitigation_tiny_full_run(orc, s, mit):
    wl = make_workload("tiny", s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    assert run_mitigated(orc, wl, w, mit) > 0


@pytest.mark.parametrize("seed,kw,mit", [
    (0, {}, dict(p=0.6, lam=0.5, K=3)),
    (1, dict(nb=1, s=0), dict(p=0.3, lam=0.0, K=2)),
    (2, dict(D_e=0, s=3), dict(p=0.0, lam=0.9, K=5)),   # p = 0: gamma is the smallest gap
    (3, dict(nb=12, B=5), dict(p=1.0, lam=0.5, K=4)),   # p = 1: nothing is stale
    (4, dict(nb=20, s=1), dict(p=0.5, lam=0.25, K=16))])   # the widest neighbour sets
def test_mitigation_tie_heavy(orc, seed, kw, mit):
    # integer times over a short span: many equal gaps, equal memory times and
    # equal common-neighbour counts
    wl = tie_heavy(seed, **kw)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    run_mitigated(orc, wl, w, mit)


def test_mitigation_wiki_window(orc):
    # early in a stream the never-updated nodes share the largest gap (T - 0),
    # so a p = 0.99 tail would tie with gamma and leave nothing stale: p = 0.6
    wl = make_workload("wiki", E=36_000)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    assert run_mitigated(orc, wl, w, dict(p=0.6, lam=0.95, K=10)) > 0


def test_mitigation_reddit_from_synthetic_state(orc):
    """A mid-run window of the REDDIT-shaped stream from a seeded state: many
    distinct memory times, so the p = 0.99 tail is populated."""
    wl = make_workload("reddit", E=60_000)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    j = 80
    assert run_mitigated(orc, wl, w, dict(p=0.99, lam=0.95, K=10), n_iters=4, first=j,
                         init=synthetic_state(wl, j, 5)) > 0


def test_mitigation_gdelt_window(orc):
    """GDELT-shaped batches 20,000 .. 20,001 (B 4000, node sets near 16,682) from
    a seeded state on the graph of their first 80 M events."""
    j, n = 20_000, 2
    wl = gdelt_prefix((j + n) * 4000)
    rows = window_rows(orc, wl, j, n)
    host, dev = sparse_features(wl, rows)
    wl = dataclasses.replace(wl, efeat=host)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    assert run_mitigated(orc, wl, w, dict(p=0.99, lam=0.95, K=10), n_iters=n, first=j,
                         init=synthetic_state(wl, j, 11), gpu_efeat=dev) > 0
    del dev
    torch.cuda.empty_cache()


def test_mitigation_pipelined_equals_sequential():
    """The executor (mitigation set on the state) and Stage.step give
    bit-identical results."""
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("wiki", E=30_000)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    mit = dict(p=0.6, lam=0.9, K=8)
    n = wl.n_iters
    a = from_workload(wl, w, mitigation=mit)
    a.run(0, 17)
    a.run(17, n - 17)
    b = from_workload(wl, w, mitigation=mit)
    for i in range(n):
        b.step(i)
    oa, ob = a.outputs(), b.outputs()
    for k in oa:
        assert np.array_equal(np.asarray(oa[k]), np.asarray(ob[k])), k
    ra, rb = a.mitigation_result(), b.mitigation_result()
    assert ra[0] == rb[0] and np.array_equal(ra[1], rb[1]) and np.array_equal(ra[2], rb[2])
    assert len(ra[1]) > 0
    a.flush()
    b.flush()
    sa, sb = a.state(), b.state()
    for k in sa:
        assert np.array_equal(sa[k], sb[k]), k
    a.close()
    b.close()


def test_mitigation_argument_errors():
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=2_000)
    st = from_workload(wl, make_weights(wl.M, wl.D_e, wl.D_t))
    for args in ((0, 10, 4), (100, 0, 4), (100, 65, 4), (100, 10, 0), (100, 10, 17)):
        with pytest.raises(tgm.TgmError) as e:
            tgm.tgm_mitigator_create(*args)
        assert e.value.code == tgm.TGM_EINVAL
    mt = tgm.tgm_mitigator_create(st.cap, wl.nb, 4)
    st.step(0)
    call = lambda **kw: tgm.tgm_mitigate(
        mt, st.g, kw.get("first", 0), st.nodes, st.n_nodes, kw.get("cap", st.cap), st.f_mem,
        st.f_mem_ts, wl.M, kw.get("p", 0.9), kw.get("lam", 0.5), stream=st.stream)
    for kw, code in ((dict(p=1.5), tgm.TGM_EINVAL), (dict(p=-0.1), tgm.TGM_EINVAL),
                     (dict(lam=2.0), tgm.TGM_EINVAL), (dict(first=wl.E), tgm.TGM_ERANGE),
                     (dict(cap=st.cap + 1), tgm.TGM_ESIZE)):
        with pytest.raises(tgm.TgmError) as e:
            call(**kw)
        assert e.value.code == code, kw
    call()   # valid
    torch.cuda.synchronize()
    tgm.tgm_mitigator_destroy(mt)
    st.close()
