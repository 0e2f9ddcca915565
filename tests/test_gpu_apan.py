"""The APAN family on the GPU (tgm_apan_step) against the fp64 oracle, every
iteration: the node set, the fetched memories and mailboxes (times and
counts exactly, rows within 1e-5 + 1e-4 |oracle|), the new memories and
their times, the embeddings; then the flushed tables and mailboxes."""
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


def apan_state(wl, j, K, seed):
    """Seeded committed tables at iteration j: memories, times and versions,
    and mailboxes whose mails are older than batch j."""
    from test_gpu_parity import synthetic_state
    from workloads import synthetic_mailbox
    st = synthetic_state(wl, j, seed)
    mb, mb_ts, cnt = synthetic_mailbox(wl.N, K, wl.D_m, wl.t[wl.batch(j)[0] - 1], seed + 1)
    return st, (mb, mb_ts, cnt)


def apan_pair(orc, wl, w, n=None, s=None, first=0, init=None, efeat=None):
    from paper_2402_15113_amd.stage import ApanStage
    from test_gpu_parity import close, exact
    st = ApanStage(wl, w, s=s, efeat=efeat)
    o = orc.Oracle(wl, w, s=s)
    if init is not None:
        tab, (mb, mb_ts, cnt) = init
        st.load_state(first, tab["mem"], tab["mem_ts"], tab["ver"], mb, mb_ts, cnt)
        o.set_state(first, **tab)
        o.set_mailbox(mb, mb_ts, cnt)
    n = (wl.n_iters - first) if n is None else n
    for i in range(first, first + n):
        print(f"[apan] {wl.name} K={w.K_mb} propagate={w.propagate} s={st.s} iter {i}",
              flush=True)
        st.step(i)
        g, r = st.outputs(), o.step()
        assert g["n_U"] == r.n_U
        exact("U", g["U"], r.U)
        exact("root_pos", g["root_pos"], r.root_pos)
        exact("f_ver", g["f_ver"], r.f_ver)
        exact("f_mem_ts", g["f_mem_ts"], r.f_mem_ts)
        exact("f_mb_cnt", g["f_mb_cnt"], r.f_mb_cnt)
        for p in range(r.n_U):
            c = r.f_mb_cnt[p]
            exact("f_mb_ts", g["f_mb_ts"][p, :c], r.f_mb_ts[p, :c])
        mask = np.arange(w.K_mb)[None, :] < r.f_mb_cnt[:, None]
        close("f_mb", g["f_mb"][mask], r.f_mb[mask])
        close("f_mem", g["f_mem"], r.f_mem)
        exact("new_mem_ts", g["new_mem_ts"], r.new_mem_ts)
        close("s_new", g["s_new"], r.s_new)
        close("h", g["h"], r.h)
    st.flush()
    o.flush()
    gs = st.state()
    os_ = o.state()
    exact("ver", gs["ver"], os_["ver"])
    exact("mem_ts", gs["mem_ts"], os_["mem_ts"])
    close("mem", gs["mem"], os_["mem"])
    mb, mb_ts, cnt = o.mailbox()
    exact("mb_cnt", gs["mb_cnt"], cnt)
    mask = np.arange(w.K_mb)[None, :] < cnt[:, None]
    exact("mb_ts", gs["mb_ts"][mask], mb_ts[mask])
    close("mb", gs["mb"][mask], mb[mask])
    st.close()


@pytest.mark.parametrize("s,K,prop", [(0, 4, True), (2, 4, True), (1, 1, False),
                                      (2, 16, True), (1, 3, False)])
def test_apan_tiny(orc, s, K, prop):
    wl = make_workload("tiny", E=6000, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=K, propagate=prop, beta="random")
    apan_pair(orc, wl, w, s=s)


def test_apan_tie_heavy_odd_dims(orc):
    from test_gpu_parity import tie_heavy
    for seed, kw in ((4, dict(M=36, H=3, D_e=17, D_t=23, B=11, nb=10)),
                     (2, dict(D_e=0, s=3)), (3, dict(nb=64, B=5, M=20, H=4, D_t=1))):
        wl = tie_heavy(seed, **kw)
        w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=5, seed=seed, beta="random")
        apan_pair(orc, wl, w)


def test_apan_wiki_window(orc):
    wl = make_workload("wiki", E=24 * 600)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=10)
    apan_pair(orc, wl, w)


def test_apan_lastfm_window(orc):
    wl = make_workload("lastfm", E=12 * 2000)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=10)
    apan_pair(orc, wl, w)


def test_apan_wiki_from_loaded_state(orc):
    """A mid-run WIKI window from seeded tables and mailboxes (s = 2: the
    loaded tables plus the window's own write sets from i - 3 on)."""
    wl = make_workload("wiki", E=60_000)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=10)
    apan_pair(orc, wl, w, n=6, first=60, init=apan_state(wl, 60, 10, 7))


def test_apan_gdelt_window(orc):
    """GDELT-shaped batches 20,000 .. 20,001 (B 4000, node sets near all 16,682
    nodes, mailboxes of 10 mails of 386 values) from seeded tables on the
    graph of their first 80 M events."""
    import dataclasses
    from test_gpu_parity import gdelt_prefix, sparse_features, window_rows
    j, n = 20_000, 2
    wl = gdelt_prefix((j + n) * 4000)
    rows = window_rows(orc, wl, j, n)
    host, dev = sparse_features(wl, rows)
    wl = dataclasses.replace(wl, efeat=host)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=10)
    apan_pair(orc, wl, w, n=n, first=j, init=apan_state(wl, j, 10, 11), efeat=dev)
    del dev
    torch.cuda.empty_cache()


def test_apan_reset_repeats_the_run():
    from paper_2402_15113_amd.stage import ApanStage
    wl = make_workload("wiki", E=24 * 400)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=6)
    st = ApanStage(wl, w)
    outs = []
    for rep in range(2):
        if rep:
            st.reset()
        for i in range(wl.n_iters):
            st.step(i)
        st.flush()
        outs.append((st.outputs(), st.state()))
    (o1, s1), (o2, s2) = outs
    for k in o1:
        assert np.array_equal(np.asarray(o1[k]), np.asarray(o2[k])), k
    for k in s1:
        assert np.array_equal(s1[k], s2[k]), k
    st.close()


def test_apan_protocol_and_limits():
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import ApanStage
    wl = make_workload("tiny", E=2000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="apan", K_mb=4)
    st = ApanStage(wl, w)
    st.step(0)
    with pytest.raises(tgm.TgmError) as e:   # not the next iteration
        st.step(2)
    assert e.value.code == tgm.TGM_EORDER
    st.close()
    with pytest.raises(tgm.TgmError) as e:
        tgm.tgm_apan_create(wl.N, wl.M, wl.D_e, wl.D_t, wl.nb, 17, True, 1, wl.B, 100, w)
    assert e.value.code == tgm.TGM_EINVAL
    torch.cuda.synchronize()
    assert tgm.last_device_error() == tgm.TGM_OK
