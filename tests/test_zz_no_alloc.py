"""tgm_mitigate_noalloc, the entry point for callers that cannot allocate
device memory, against tgm_mitigate (the same mitigation with a mitigator
handle's work space).  Two calls in a row, the second on a smaller input (a
smaller node set and cap, other nb and K), each compared bit for bit with
tgm_mitigate on the same fetched memories; the library's allocation count
does not move across either call.  The work space is one fixed array per GPU
that every call shares, so the second call also shows that nothing left by
the first one leaks into it."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from workloads import make_weights, make_workload  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2402_15113_amd import tgm
    tgm.lib()


def _fetched(wl, w, it):
    """A stage run sequentially through iteration it-1, then the sample and the
    fetch of iteration it (the mitigation's input)."""
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    st = from_workload(wl, w)
    for i in range(it):
        st.step(i)
    lo, hi = st.batch(it)
    S = st.sets[0]
    tgm.tgm_sample_nodes(st.g, lo, hi - lo, st.nb, S.root, S.root_ts, S.nbr, S.eid, S.nts, S.cnt,
                         S.nodes, S.n_nodes, st.cap, S.root_pos, S.nbr_pos, stream=st.stream)
    tgm.tgm_fetch_memory(st.st, it, S.nodes, S.n_nodes, st.cap, st.f_mem, st.f_mem_ts, st.f_mail,
                         st.f_mail_ts, st.f_ver, stream=st.stream)
    return st, lo, S


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_equals_mitigate(order):
    from paper_2402_15113_amd import tgm
    cases = [("wiki", dict(E=60_000), 40, dict(p=0.6, lam=0.5, nb=10, K=10)),
             ("tiny", dict(E=6000, s=2), 20, dict(p=0.7, lam=0.25, nb=3, K=4))]
    caps = []
    for name, kw, it, m in cases:
        wl = make_workload(name, **kw)
        wl.nb = m["nb"]
        w = make_weights(wl.M, wl.D_e, wl.D_t)
        st, lo, S = _fetched(wl, w, it)
        n = int(S.n_nodes.item())
        print(f"[noalloc] {name} iter {it}: cap {st.cap}, {n} nodes, {m}", flush=True)
        caps.append((st.cap, n))
        ref = st.f_mem.clone()
        out = st.f_mem.clone()
        mt = tgm.tgm_mitigator_create(st.cap, m["nb"], m["K"])
        tgm.tgm_mitigate(mt, st.g, lo, S.nodes, S.n_nodes, st.cap, ref, st.f_mem_ts, wl.M,
                         m["p"], m["lam"], stream=st.stream)
        torch.cuda.synchronize()
        before = tgm.alloc_count()
        tgm.tgm_mitigate_noalloc(st.g, lo, S.nodes, S.n_nodes, st.cap, out, st.f_mem_ts, wl.M,
                                 m["nb"], m["K"], m["p"], m["lam"], stream=st.stream)
        torch.cuda.synchronize()
        assert tgm.alloc_count() == before
        assert tgm.last_device_error() == tgm.TGM_OK
        changed = (ref != st.f_mem).any(dim=1)
        assert int(changed.sum()) > 0, "no stale node was blended"
        assert torch.equal(out, ref)
        print(f"[noalloc] {name}: {int(changed.sum())} rows blended, equal", flush=True)
        tgm.tgm_mitigator_destroy(mt)
        st.close()
    assert caps[1][0] < caps[0][0] and caps[1][1] < caps[0][1]


def test_noalloc_rejects_sizes_beyond_its_limit():
    from paper_2402_15113_amd import tgm
    wl = make_workload("tiny", E=3000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    st, lo, S = _fetched(wl, w, 3)

    def code(**kw):
        a = dict(cap=st.cap, nb=wl.nb, K=4)
        a.update(kw)
        with pytest.raises(tgm.TgmError) as e:
            tgm.tgm_mitigate_noalloc(st.g, lo, S.nodes, S.n_nodes, a["cap"], st.f_mem,
                                     st.f_mem_ts, wl.M, a["nb"], a["K"], 0.5, 0.5,
                                     stream=st.stream)
        return e.value.code

    assert code(cap=tgm.MITIGATE_NOALLOC_MAX_NODES + 1) == tgm.TGM_ESIZE
    assert code(nb=65) == tgm.TGM_EINVAL
    assert code(K=17) == tgm.TGM_EINVAL
    torch.cuda.synchronize()
    assert tgm.last_device_error() == tgm.TGM_OK
    st.close()
