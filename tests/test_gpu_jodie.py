"""The JODIE model family on the GPU (RNN updater in the GRU kernel's
pipeline, time-projection embedding) against the fp64 oracle through the
C ABI, sequential and pipelined.  Bit-exact: indices, versions, times,
winners.  Floating point within |gpu - oracle| <= 1e-5 + 1e-4 |oracle|."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from test_gpu_parity import compare_state, compare_step, run_pair, tie_heavy  # noqa: E402
from workloads import make_weights, make_workload  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2402_15113_amd import tgm
    tgm.lib()


def _w(wl, seed=0):
    return make_weights(wl.M, wl.D_e, wl.D_t, seed=seed, model="jodie")


@pytest.mark.parametrize("s", [0, 2])
def test_jodie_tiny_full_run(orc, s):
    wl = make_workload("tiny", s=s)
    run_pair(orc, wl, _w(wl), s=s)


@pytest.mark.parametrize("seed,kw", [(0, {}), (1, dict(nb=1, s=0)), (2, dict(D_e=0, s=3)),
                                     (4, dict(M=36, H=3, D_e=17, D_t=23, B=11, nb=10))])
def test_jodie_tie_heavy(orc, seed, kw):
    wl = tie_heavy(seed, **kw)
    run_pair(orc, wl, _w(wl, seed))


def test_jodie_wiki_window(orc):
    wl = make_workload("wiki", E=36_000)
    run_pair(orc, wl, _w(wl), check_every=7)


@pytest.mark.parametrize("name,s,E", [("tiny", 2, None), ("wiki", 1, 36_000)])
def test_jodie_pipelined_run(orc, name, s, E):
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload(name, E=E, s=s)
    w = _w(wl)
    st = from_workload(wl, w)
    o = orc.Oracle(wl, w)
    n = wl.n_iters
    print(f"[jodie] pipelined {name} s={s} iters 0..{n - 1}", flush=True)
    st.run(0, n)
    for i in range(n):
        r = o.step(want="all" if i == n - 1 else "light")
    compare_step(st.outputs(), r)
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()


def test_jodie_pipelined_equals_sequential():
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("wiki", E=30_000)
    w = _w(wl)
    n = wl.n_iters
    a = from_workload(wl, w)
    a.run(0, 20)
    a.run(20, n - 20)
    b = from_workload(wl, w)
    for i in range(n):
        b.step(i)
    oa, ob = a.outputs(), b.outputs()
    for k in oa:
        assert np.array_equal(np.asarray(oa[k]), np.asarray(ob[k])), k
    a.close()
    b.close()


def test_model_family_argument_errors():
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=2_000)
    j = from_workload(wl, _w(wl))
    t = from_workload(wl, make_weights(wl.M, wl.D_e, wl.D_t))
    for st in (j, t):
        st.step(0)
    b = j.sets[0]
    with pytest.raises(tgm.TgmError) as e:   # attention on a JODIE model
        tgm.tgm_embed(j.m, j.g, 3 * wl.B, wl.nb, b.root_pos, b.root_ts, b.nbr_pos, b.eid, b.nts,
                      b.cnt, j.mem_new, b.n_nodes, j.cap, j.h, stream=j.stream)
    assert e.value.code == tgm.TGM_EINVAL
    with pytest.raises(tgm.TgmError) as e:   # the projection on a TGN model
        tgm.tgm_embed_projection(t.m, 3 * wl.B, b.root_pos, b.root_ts, t.mem_new, t.new_mem_ts,
                                 b.n_nodes, t.cap, t.h, stream=t.stream)
    assert e.value.code == tgm.TGM_EINVAL
    with pytest.raises(tgm.TgmError) as e:   # R beyond max_roots
        tgm.tgm_embed_projection(j.m, 3 * wl.B + 1, b.root_pos, b.root_ts, j.mem_new,
                                 j.new_mem_ts, b.n_nodes, j.cap, j.h, stream=j.stream)
    assert e.value.code == tgm.TGM_ESIZE
    torch.cuda.synchronize()
    j.close()
    t.close()


def test_jodie_with_mitigation_pipelined_equals_sequential(orc):
    """The mitigation acts on fetched memories, so it composes with either
    family: the executor and Stage.step agree bit for bit, and the sequential
    run matches the oracle."""
    from paper_2402_15113_amd.stage import from_workload
    from test_gpu_mitigation import run_mitigated
    wl = make_workload("tiny", s=2)
    w = _w(wl)
    mit = dict(p=0.8, lam=0.9, K=4)
    assert run_mitigated(orc, wl, w, mit) > 0
    a, b = from_workload(wl, w, mitigation=mit), from_workload(wl, w, mitigation=mit)
    n = wl.n_iters
    a.run(0, n)
    for i in range(n):
        b.step(i)
    oa, ob = a.outputs(), b.outputs()
    for k in oa:
        assert np.array_equal(np.asarray(oa[k]), np.asarray(ob[k])), k
    a.close()
    b.close()
