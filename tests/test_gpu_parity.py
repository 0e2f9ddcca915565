"""GPU path (libtgm through its C ABI) against the fp64 oracle.

Bit-exact: roots, sampled neighbours / event ids / times / counts, the node
set and every position map, fetched versions and timestamps, new memory
timestamps, latest-message winners, committed versions and timestamps.
Floating point (fetched memory and mail, updated memory s', embeddings h,
committed tables): |gpu - oracle| <= 1e-5 + 1e-4 |oracle| element-wise
(fp32 vs fp64).
"""
import dataclasses
import time

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from workloads import (CONFIGS, FEAT_CHUNK, custom_workload, edge_feature_rows,  # noqa: E402
                       make_weights, make_workload)

ATOL, RTOL = 1e-5, 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2402_15113_amd import tgm
    tgm.lib()   # fails loudly when the library is missing


def close(name, g, o):
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    assert g.shape == o.shape, (name, g.shape, o.shape)
    err = np.abs(g - o)
    bad = err > ATOL + RTOL * np.abs(o)
    if bad.any():
        k = np.unravel_index(np.argmax(err - (ATOL + RTOL * np.abs(o))), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{bad.size} outside tolerance; worst at "
                             f"{k}: gpu {g[k]!r} oracle {o[k]!r}")
    return float(err.max()) if err.size else 0.0


def exact(name, g, o):
    g, o = np.asarray(g), np.asarray(o)
    assert g.shape == o.shape, (name, g.shape, o.shape)
    if not np.array_equal(g, o):
        k = np.argwhere(g != o)[0]
        raise AssertionError(f"{name}: {int((g != o).sum())} mismatches; first at {tuple(k)}: "
                             f"gpu {g[tuple(k)]!r} oracle {o[tuple(k)]!r}")


def compare_step(go, r, close_fn=None):
    """go: Stage.outputs(); r: oracle StepResult of the same iteration;
    close_fn replaces close for the floating-point fields."""
    cf = close_fn or close
    assert go["iter"] == r.iter and go["b"] == r.b
    exact("root", go["root"], r.root)
    exact("root_ts", go["root_ts"], r.root_ts)
    exact("cnt", go["cnt"], r.cnt)
    exact("nbr", go["nbr"], r.nbr)
    exact("eid", go["eid"], r.eid)
    exact("nts", go["nts"], r.nts)
    assert go["n_U"] == r.n_U
    exact("U", go["U"], r.U)
    exact("root_pos", go["root_pos"], r.root_pos)
    exact("nbr_pos", go["nbr_pos"], r.nbr_pos)
    exact("f_ver", go["f_ver"], r.f_ver)
    exact("f_mem_ts", go["f_mem_ts"], r.f_mem_ts)
    exact("f_mail_ts", go["f_mail_ts"], r.f_mail_ts)
    exact("new_mem_ts", go["new_mem_ts"], r.new_mem_ts)
    exact("winner", go["winner"], r.winner)
    e = {}
    e["f_mem"] = cf("f_mem", go["f_mem"], r.f_mem)
    e["f_mail"] = cf("f_mail", go["f_mail"], r.f_mail)
    e["s_new"] = cf("s_new", go["s_new"], r.s_new)
    e["h"] = cf("h", go["h"], r.h)
    return e


def compare_state(gs, os_):
    exact("ver", gs["ver"], os_["ver"])
    exact("mem_ts", gs["mem_ts"], os_["mem_ts"])
    exact("mail_ts", gs["mail_ts"], os_["mail_ts"])
    close("mem", gs["mem"], os_["mem"])
    close("mail", gs["mail"], os_["mail"])


def run_pair(orc, wl, w, n_iters=None, s=None, first=0, init=None, check_every=1,
             gpu_efeat=None):
    """Run the GPU stage and the oracle side by side over iterations
    first .. first + n_iters - 1 and compare every check_every-th step, then the
    flushed tables.  gpu_efeat (a device tensor) replaces wl.efeat on the GPU
    side only; it must hold the same values wherever either side reads."""
    from paper_2402_15113_amd.stage import Stage, from_workload
    if gpu_efeat is None:
        st = from_workload(wl, w, s=s)
    else:
        st = Stage(wl.N, wl.src, wl.dst, wl.t, wl.neg, gpu_efeat, w, M=wl.M, D_t=wl.D_t,
                   H=wl.H, nb=wl.nb, B=wl.B, s=wl.s if s is None else s)
    o = orc.Oracle(wl, w, s=s)
    if init is not None:
        st.load_state(first, **init)
        o.set_state(first, **init)
    n = (wl.n_iters - first) if n_iters is None else n_iters
    worst = {}
    for k in range(n):
        i = first + k
        print(f"[parity] {wl.name} s={st.s} iter {i}", flush=True)
        st.step(i)
        want = (k % check_every == 0) or k == n - 1
        r = o.step(want="all" if want else "light")
        if want:
            for key, v in compare_step(st.outputs(), r).items():
                worst[key] = max(worst.get(key, 0.0), v)
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()
    return worst


@pytest.mark.parametrize("s", [0, 2])
def test_tiny_full_run(orc, s):
    wl = make_workload("tiny", s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    worst = run_pair(orc, wl, w)
    print("worst abs errors", worst)


def test_tiny_ragged_tail(orc):
    wl = make_workload("tiny", E=19_937, s=1)   # last batch holds 137 events
    assert wl.E % wl.B != 0
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    run_pair(orc, wl, w)


def tie_heavy(seed, N=13, E=300, span=40, D_e=3, B=7, M=8, D_t=5, H=2, nb=3, s=1):
    r = np.random.default_rng(seed)
    src = r.integers(0, N, E)
    dst = r.integers(0, N, E)
    dst[::9] = src[::9]   # self-loops
    t = np.sort(r.integers(0, span, E)).astype(np.float64)
    neg = r.integers(0, N, E)
    f = r.standard_normal((E, D_e)).astype(np.float32) if D_e else None
    return custom_workload(f"ties{seed}", N, src, dst, t, neg, f, M=M, D_t=D_t, H=H, nb=nb, B=B,
                           s=s, seed=seed)


@pytest.mark.parametrize("seed,kw", [(0, {}), (1, dict(nb=1, s=0)), (2, dict(D_e=0, s=3)),
                                     (3, dict(nb=64, B=5, M=20, H=4, D_t=1)),
                                     (4, dict(M=36, H=3, D_e=17, D_t=23, B=11, nb=10))])
def test_tie_heavy_edge_cases(orc, seed, kw):
    """Integer timestamps with many ties, self-loops, roots without history,
    dims that are not multiples of the 16-wide MFMA tiles, nb = 1 and 64."""
    wl = tie_heavy(seed, **kw)
    w = make_weights(wl.M, wl.D_e, wl.D_t, seed=seed, beta="random")
    run_pair(orc, wl, w)


@pytest.mark.parametrize("seed,kw", [
    (20, dict(M=128, H=2, D_e=256, D_t=128, nb=10, B=9)),   # the documented maxima
    (21, dict(M=112, H=2, D_e=96, D_t=16, nb=16, B=6)),     # largest folded shape
    (25, dict(M=112, H=7, D_e=40, D_t=16, nb=16, B=6)),     # 5 roots x 7 heads > 16: unfolded
    (22, dict(M=16, H=1, D_e=1, D_t=1, nb=17, B=4)),        # smallest dims, nb past 16
    (23, dict(M=64, H=4, D_e=0, D_t=100, nb=2, B=13, s=0)),
    (24, dict(M=100, H=2, D_e=172, D_t=100, nb=10, B=8, s=2))])
def test_shape_limits(orc, seed, kw):
    """Shapes at the limits the model header states (M <= 128, D_e <= 256,
    D_e + D_t <= 384, nb <= 64), the boundary of the folded attention (nb <=
    16, M <= 112) and the smallest dims."""
    wl = tie_heavy(seed, N=29, E=240, **kw)
    w = make_weights(wl.M, wl.D_e, wl.D_t, seed=seed, beta="random")
    run_pair(orc, wl, w)


def test_wiki_full_run(orc):
    """The bench workload (WIKI-shaped, B = 600, s = 1), every batch."""
    wl = make_workload("wiki")
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    worst = run_pair(orc, wl, w, check_every=8)
    print("worst abs errors", worst)


def test_lastfm_no_edge_features_window(orc):
    """LastFM-shaped: D_e = 0, heavy repetition (latest-message reduce and
    write-set conflicts), B = 2000, s = 2: first 64 batches."""
    wl = make_workload("lastfm")
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    run_pair(orc, wl, w, n_iters=64)


@pytest.mark.parametrize("s", [1, 2, 4])
def test_reddit_window(orc, s):
    """REDDIT-shaped, first 32 batches."""
    wl = make_workload("reddit", s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    run_pair(orc, wl, w, n_iters=32)


def test_mid_run_window_from_synthetic_state(orc):
    """A window in the middle of the REDDIT-shaped stream (batches 560..575),
    both sides started from the same seeded synthetic state."""
    wl = make_workload("reddit", s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    j = 560
    r = np.random.default_rng(7)
    N, M, D_m = wl.N, wl.M, wl.D_m
    lo, _ = wl.batch(j)
    mem_ts = np.floor(r.uniform(0, wl.t[lo - 1], N))
    init = dict(mem=r.uniform(-1, 1, (N, M)).astype(np.float32).astype(np.float64),
                mem_ts=mem_ts,
                mail=r.standard_normal((N, D_m)).astype(np.float32).astype(np.float64),
                mail_ts=np.minimum(mem_ts + np.floor(r.exponential(3600, N)), wl.t[lo - 1]),
                ver=np.where(r.random(N) < 0.9, r.integers(0, j - 2, N), -1).astype(np.int32))
    run_pair(orc, wl, w, n_iters=16, first=j, init=init)


@pytest.mark.parametrize("name,s,E", [("tiny", 0, None), ("tiny", 2, None), ("wiki", 1, 36_000),
                                      ("lastfm", 2, 60_000)])
def test_pipelined_run(orc, name, s, E):
    """Stage.run (prefetch of i+1 on a second stream beside compute(i)) against
    the oracle: the last iteration's outputs and the flushed tables."""
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload(name, E=E, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    st = from_workload(wl, w)
    o = orc.Oracle(wl, w)
    n = wl.n_iters
    print(f"[parity] pipelined {name} s={s} iters 0..{n - 1}", flush=True)
    st.run(0, n)
    for i in range(n):
        r = o.step(want="all" if i == n - 1 else "light")
    compare_step(st.outputs(), r)
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()


def test_pipelined_equals_sequential():
    """Stage.run and Stage.step give bit-identical results (the same kernels;
    only the streams differ), including across a run split in two."""
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("wiki", E=30_000)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
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
    a.flush()
    b.flush()
    sa, sb = a.state(), b.state()
    for k in sa:
        assert np.array_equal(sa[k], sb[k]), k
    a.close()
    b.close()


# ------------------------------------------------------------------ GDELT-shaped
# The full stream has 191,290,882 events and a 142 GB edge-feature table.  It
# is generated once per session without features; the tests below read only
# the feature rows they need (the rows of the events the oracle's sampler picks
# and of the batch events), which both sides receive as a zero table with
# those rows filled.
_GDELT = {}


def gdelt_stream():
    if "wl" not in _GDELT:
        print("[parity] generating the GDELT-shaped stream (191,290,882 events)", flush=True)
        t0 = time.time()
        _GDELT["wl"] = make_workload("gdelt", with_features=False)
        print(f"[parity] generated in {time.time() - t0:.0f} s", flush=True)
    return _GDELT["wl"]


def gdelt_prefix(E):
    """The first E events (all a batch < E / B can see: sampling is strictly
    earlier and events are time-sorted)."""
    full = gdelt_stream()
    return dataclasses.replace(full, src=full.src[:E], dst=full.dst[:E], t=full.t[:E],
                               neg=full.neg[:E])


def window_rows(orc, wl, first, n):
    """Feature rows read by batches first .. first + n - 1: the batch events and
    the events the oracle's sampler picks for their roots."""
    roots, rts = [], []
    for i in range(first, first + n):
        a, b = wl.batch(i)
        roots += [wl.src[a:b], wl.dst[a:b], wl.neg[a:b]]
        rts += [wl.t[a:b]] * 3
    _, eid, _, _ = orc.sample(wl.N, wl.src, wl.dst, wl.t, np.concatenate(roots),
                              np.concatenate(rts), wl.nb)
    lo, hi = wl.batch(first)[0], wl.batch(first + n - 1)[1]
    return np.unique(np.concatenate([eid[eid >= 0].ravel().astype(np.int64),
                                     np.arange(lo, hi, dtype=np.int64)]))


def sparse_features(wl, rows):
    """Host table [E x D_e] that is zero except `rows` (untouched pages stay
    unallocated), and the same table on the device."""
    from concurrent.futures import ThreadPoolExecutor
    E_full = CONFIGS[wl.name]["E"]
    host = np.zeros((wl.E, wl.D_e), dtype=np.float32)

    def fill(c):
        lo = int(c) * FEAT_CHUNK
        hi = min(lo + FEAT_CHUNK, wl.E)
        sel = rows[(rows >= lo) & (rows < hi)]
        host[sel] = edge_feature_rows(wl.seed, E_full, wl.D_e, lo, hi)[sel - lo]

    with ThreadPoolExecutor(8) as ex:
        list(ex.map(fill, np.unique(rows // FEAT_CHUNK)))
    dev = torch.zeros((wl.E, wl.D_e), dtype=torch.float32, device="cuda")
    dev[torch.from_numpy(rows).cuda()] = torch.from_numpy(host[rows]).cuda()
    return host, dev


def synthetic_state(wl, j, seed):
    """A seeded memory state standing in for the one iteration j would see."""
    r = np.random.default_rng(seed)
    N, M, D_m = wl.N, wl.M, wl.D_m
    lo, _ = wl.batch(j)
    mem_ts = np.floor(r.uniform(0, wl.t[lo - 1], N))
    return dict(mem=r.uniform(-1, 1, (N, M)).astype(np.float32).astype(np.float64),
                mem_ts=mem_ts,
                mail=r.standard_normal((N, D_m)).astype(np.float32).astype(np.float64),
                mail_ts=np.minimum(mem_ts + np.floor(r.exponential(3600, N)), wl.t[lo - 1]),
                ver=np.where(r.random(N) < 0.9, r.integers(0, j - 2, N), -1).astype(np.int32))


def test_gdelt_first_batches(orc):
    """GDELT-shaped stream at full model size (D_e 186, B 4000, s 4): the first
    4 batches from the initial state."""
    wl = gdelt_prefix(4 * 4000)
    wl = dataclasses.replace(wl, efeat=edge_feature_rows(wl.seed, CONFIGS["gdelt"]["E"],
                                                          wl.D_e, 0, wl.E))
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    run_pair(orc, wl, w, n_iters=4)


def test_gdelt_mid_run_window(orc):
    """GDELT-shaped stream, batches 20,000 .. 20,003 on the real graph of their
    first 80,016,000 events (80 M-event history, 59.5 GB feature table on the
    device), both sides started from the same seeded synthetic state."""
    j, n = 20_000, 4
    wl = gdelt_prefix((j + n) * 4000)
    rows = window_rows(orc, wl, j, n)
    print(f"[parity] gdelt window: {len(rows)} feature rows", flush=True)
    host, dev = sparse_features(wl, rows)
    wl = dataclasses.replace(wl, efeat=host)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    run_pair(orc, wl, w, n_iters=n, first=j, init=synthetic_state(wl, j, 11), gpu_efeat=dev)
    del dev
    torch.cuda.empty_cache()


def test_gdelt_sampler_full_graph(orc):
    """The whole GDELT-shaped graph (191 M events, 382 M adjacency records): the
    sampler at a random sample of (node, time) roots against the oracle's."""
    from paper_2402_15113_amd import tgm
    wl = gdelt_stream()
    dev = torch.device("cuda:0")
    T = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
    src, dst, t, neg = (T(wl.src, torch.int32), T(wl.dst, torch.int32), T(wl.t, torch.float64),
                        T(wl.neg, torch.int32))
    g = tgm.tgm_graph_create(wl.N, src, dst, t, neg, None)
    r = np.random.default_rng(5)
    R, nb = 8192, 10
    deg = np.bincount(np.concatenate([wl.src[:1 << 24], wl.dst[:1 << 24]]), minlength=wl.N)
    hot = np.argsort(deg)[-50:]
    root = np.where(r.random(R) < 0.5, r.choice(hot, R), r.integers(0, wl.N, R)).astype(np.int32)
    rts = np.where(r.random(R) < 0.5, wl.t[r.integers(0, wl.E, R)],
                   r.uniform(-5, wl.t[-1] + 5, R))
    nbr, eid, nts, cnt = (torch.empty((R, nb), dtype=torch.int32, device=dev),
                          torch.empty((R, nb), dtype=torch.int32, device=dev),
                          torch.empty((R, nb), dtype=torch.float64, device=dev),
                          torch.empty(R, dtype=torch.int32, device=dev))
    tgm.tgm_sample(g, T(root, torch.int32), T(rts, torch.float64), R, nb, nbr, eid, nts, cnt)
    torch.cuda.synchronize()
    onbr, oeid, onts, ocnt = orc.sample(wl.N, wl.src, wl.dst, wl.t, root, rts, nb)
    exact("cnt", cnt.cpu().numpy(), ocnt)
    exact("nbr", nbr.cpu().numpy(), onbr)
    exact("eid", eid.cpu().numpy(), oeid)
    exact("nts", nts.cpu().numpy(), onts)
    _, _, _, n_adj = tgm.tgm_graph_info(g)
    assert n_adj == 2 * wl.E - int((wl.src == wl.dst).sum())
    tgm.tgm_graph_destroy(g)
    del src, dst, t, neg
    torch.cuda.empty_cache()


def test_sampler_full_size_sampled_roots(orc):
    """REDDIT-shaped full graph (672k events, max degree ~184k): the sampler
    at a random sample of (node, time) roots against the oracle's sampler."""
    from paper_2402_15113_amd import tgm
    wl = make_workload("reddit", with_features=False)
    dev = torch.device("cuda:0")
    T = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
    src, dst, t, neg = (T(wl.src, torch.int32), T(wl.dst, torch.int32), T(wl.t, torch.float64),
                        T(wl.neg, torch.int32))
    g = tgm.tgm_graph_create(wl.N, src, dst, t, neg, None)
    r = np.random.default_rng(3)
    R, nb = 4096, 10
    # half hot nodes (high degree), half uniform; times on and between event times
    deg = np.bincount(np.concatenate([wl.src, wl.dst]), minlength=wl.N)
    hot = np.argsort(deg)[-50:]
    root = np.where(r.random(R) < 0.5, r.choice(hot, R), r.integers(0, wl.N, R)).astype(np.int32)
    rts = np.where(r.random(R) < 0.5, wl.t[r.integers(0, wl.E, R)],
                   r.uniform(-5, wl.t[-1] + 5, R))
    nbr, eid, nts, cnt = (torch.empty((R, nb), dtype=torch.int32, device=dev),
                          torch.empty((R, nb), dtype=torch.int32, device=dev),
                          torch.empty((R, nb), dtype=torch.float64, device=dev),
                          torch.empty(R, dtype=torch.int32, device=dev))
    tgm.tgm_sample(g, T(root, torch.int32), T(rts, torch.float64), R, nb, nbr, eid, nts, cnt)
    torch.cuda.synchronize()
    onbr, oeid, onts, ocnt = orc.sample(wl.N, wl.src, wl.dst, wl.t, root, rts, nb)
    exact("cnt", cnt.cpu().numpy(), ocnt)
    exact("nbr", nbr.cpu().numpy(), onbr)
    exact("eid", eid.cpu().numpy(), oeid)
    exact("nts", nts.cpu().numpy(), onts)
    _, _, _, n_adj = tgm.tgm_graph_info(g)
    assert n_adj == 2 * wl.E - int((wl.src == wl.dst).sum())
    tgm.tgm_graph_destroy(g)


def test_deterministic_rerun():
    """Two runs of the same stream are bit-identical (no fp atomics)."""
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=6000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    outs = []
    for _ in range(2):
        st = from_workload(wl, w)
        for i in range(wl.n_iters):
            st.step(i)
        o = st.outputs()
        st.flush()
        outs.append((o, st.state()))
        st.close()
    (a, sa), (b, sb) = outs
    for k in ("h", "s_new", "f_mail"):
        assert np.array_equal(a[k], b[k]), k
    for k in sa:
        assert np.array_equal(sa[k], sb[k]), k


def test_protocol_errors():
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=2000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    st = from_workload(wl, w)
    st.step(0)
    st.step(1)
    with pytest.raises(tgm.TgmError) as ei:   # iteration 1 again: not the next update
        st.step(1)
    assert ei.value.code == tgm.TGM_EORDER
    with pytest.raises(tgm.TgmError) as ei:   # fetch at 4 needs the update of 2
        tgm.tgm_fetch_memory(st.st, 4, st.nodes, st.n_nodes, st.cap, st.f_mem, st.f_mem_ts,
                             st.f_mail, st.f_mail_ts, st.f_ver)
    assert ei.value.code == tgm.TGM_EORDER
    with pytest.raises(tgm.TgmError) as ei:
        tgm.tgm_sample(st.g, st.root, st.root_ts, 3, 0, st.nbr, st.eid, st.nts, st.cnt)
    assert ei.value.code == tgm.TGM_EINVAL
    with pytest.raises(tgm.TgmError) as ei:
        tgm.tgm_node_set(st.g, st.root, 3 * wl.B, st.nbr, wl.nb, st.nodes, st.n_nodes, 5,
                         st.root_pos, st.nbr_pos)
    assert ei.value.code == tgm.TGM_ESIZE
    torch.cuda.synchronize()
    assert tgm.last_device_error() == tgm.TGM_OK
    st.close()


def test_graph_create_rejects_bad_content():
    from paper_2402_15113_amd import tgm
    dev = torch.device("cuda:0")
    src = torch.tensor([0, 1, 2], dtype=torch.int32, device=dev)
    dst = torch.tensor([1, 2, 5], dtype=torch.int32, device=dev)   # 5 >= N
    t = torch.tensor([0.0, 1.0, 2.0], dtype=torch.float64, device=dev)
    with pytest.raises(tgm.TgmError) as ei:
        tgm.tgm_graph_create(4, src, dst, t, src, None)
    assert ei.value.code == tgm.TGM_ERANGE
    dst = torch.tensor([1, 2, 3], dtype=torch.int32, device=dev)
    t = torch.tensor([0.0, 2.0, 1.0], dtype=torch.float64, device=dev)   # unsorted
    with pytest.raises(tgm.TgmError) as ei:
        tgm.tgm_graph_create(4, src, dst, t, src, None)
    assert ei.value.code == tgm.TGM_ERANGE


def test_sample_batch_equals_roots_then_sample():
    """tgm_sample_batch == tgm_batch_roots followed by tgm_sample, bit for bit."""
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("lastfm", E=60_000)   # no edge features
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    st = from_workload(wl, w)
    dev = st.dev
    for i in (0, 7, wl.n_iters - 1):
        lo, hi = wl.batch(i)
        b = hi - lo
        R, nb = 3 * b, wl.nb
        tgm.tgm_sample_batch(st.g, lo, b, nb, st.root, st.root_ts, st.nbr, st.eid, st.nts, st.cnt)
        root2 = torch.empty(R, dtype=torch.int32, device=dev)
        rts2 = torch.empty(R, dtype=torch.float64, device=dev)
        nbr2 = torch.empty((R, nb), dtype=torch.int32, device=dev)
        eid2 = torch.empty((R, nb), dtype=torch.int32, device=dev)
        nts2 = torch.empty((R, nb), dtype=torch.float64, device=dev)
        cnt2 = torch.empty(R, dtype=torch.int32, device=dev)
        tgm.tgm_batch_roots(st.g, lo, b, root2, rts2)
        tgm.tgm_sample(st.g, root2, rts2, R, nb, nbr2, eid2, nts2, cnt2)
        torch.cuda.synchronize()
        for a, c in ((st.root[:R], root2), (st.root_ts[:R], rts2), (st.nbr[:R], nbr2),
                     (st.eid[:R], eid2), (st.nts[:R], nts2), (st.cnt[:R], cnt2)):
            assert torch.equal(a, c)
    st.close()


def test_sample_nodes_equals_sample_batch_then_node_set():
    """tgm_sample_nodes (sampler-made node marks) == tgm_sample_batch followed
    by tgm_node_set, bit for bit, including on a graph with a self-loop-heavy,
    tie-heavy stream."""
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    for wl in (make_workload("wiki", E=40_000), make_workload("lastfm", E=60_000)):
        w = make_weights(wl.M, wl.D_e, wl.D_t)
        st = from_workload(wl, w)
        dev, nb, cap = st.dev, wl.nb, st.cap
        for i in (0, 3, wl.n_iters - 1):
            lo, hi = wl.batch(i)
            b = hi - lo
            R = 3 * b
            print(f"[parity] sample_nodes {wl.name} iter {i} b={b}", flush=True)
            tgm.tgm_sample_nodes(st.g, lo, b, nb, st.root, st.root_ts, st.nbr, st.eid, st.nts,
                                 st.cnt, st.nodes, st.n_nodes, cap, st.root_pos, st.nbr_pos)
            z = lambda shape, dt: torch.full(shape, -7, dtype=dt, device=dev)
            root2, rts2 = z((R,), torch.int32), z((R,), torch.float64)
            nbr2, eid2 = z((R, nb), torch.int32), z((R, nb), torch.int32)
            nts2, cnt2 = z((R, nb), torch.float64), z((R,), torch.int32)
            nodes2, n2 = z((cap,), torch.int32), z((1,), torch.int32)
            rp2, np2 = z((R,), torch.int32), z((R, nb), torch.int32)
            tgm.tgm_sample_batch(st.g, lo, b, nb, root2, rts2, nbr2, eid2, nts2, cnt2)
            tgm.tgm_node_set(st.g, root2, R, nbr2, nb, nodes2, n2, cap, rp2, np2)
            torch.cuda.synchronize()
            n = int(n2.item())
            assert int(st.n_nodes.item()) == n
            for a, c in ((st.root[:R], root2), (st.root_ts[:R], rts2), (st.nbr[:R], nbr2),
                         (st.eid[:R], eid2), (st.nts[:R], nts2), (st.cnt[:R], cnt2),
                         (st.nodes[:n], nodes2[:n]), (st.root_pos[:R], rp2),
                         (st.nbr_pos[:R], np2)):
                assert torch.equal(a, c)
        st.close()


@pytest.mark.parametrize("s", [1, 3])
def test_fetch_ahead_order(orc, s):
    """With s >= 1 the fetch of iteration i+1 may be issued before the update of
    iteration i (the prefetch that staleness allows); results are unchanged."""
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=4000, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    st = from_workload(wl, w)
    o = orc.Oracle(wl, w)
    bufs = []
    dev = st.dev
    for i in range(wl.n_iters):
        # iteration i: sample + node set + fetch into its own buffers
        lo, hi = wl.batch(i)
        b = hi - lo
        R, nb, cap = 3 * b, wl.nb, st.cap
        z = lambda shape, dt: torch.zeros(shape, dtype=dt, device=dev)
        B = dict(root=z(R, torch.int32), rts=z(R, torch.float64), nbr=z((R, nb), torch.int32),
                 eid=z((R, nb), torch.int32), nts=z((R, nb), torch.float64),
                 cnt=z(R, torch.int32), nodes=z(cap, torch.int32), n=z(1, torch.int32),
                 rpos=z(R, torch.int32), npos=z((R, nb), torch.int32),
                 mem=z((cap, wl.M), torch.float32), mts=z(cap, torch.float64),
                 mail=z((cap, wl.D_m), torch.float32), lts=z(cap, torch.float64),
                 ver=z(cap, torch.int32), new=z((cap, wl.M), torch.float32),
                 h=z((R, wl.M), torch.float32), lo=lo, b=b)
        tgm.tgm_sample_batch(st.g, lo, b, nb, B["root"], B["rts"], B["nbr"], B["eid"], B["nts"],
                             B["cnt"])
        tgm.tgm_node_set(st.g, B["root"], R, B["nbr"], nb, B["nodes"], B["n"], cap, B["rpos"],
                         B["npos"])
        tgm.tgm_fetch_memory(st.st, i, B["nodes"], B["n"], cap, B["mem"], B["mts"], B["mail"],
                             B["lts"], B["ver"])
        bufs.append(B)
        if i >= 1:   # the update of the previous iteration, after this fetch
            j = i - 1
            P = bufs[j]
            tgm.tgm_update_memory(st.st, st.m, st.g, j, P["nodes"], P["n"], cap, P["mem"],
                                  P["mts"], P["mail"], P["lts"], P["ver"], P["lo"], P["b"],
                                  P["rpos"][:P["b"]], P["rpos"][P["b"]:2 * P["b"]], P["new"])
            tgm.tgm_embed(st.m, st.g, 3 * P["b"], nb, P["rpos"], P["rts"], P["npos"], P["eid"],
                          P["nts"], P["cnt"], P["new"], P["n"], cap, P["h"])
            r = o.step()
            torch.cuda.synchronize()
            n = int(P["n"].item())
            exact("f_ver", P["ver"][:n].cpu().numpy(), r.f_ver)
            close("h", P["h"][:3 * P["b"]].cpu().numpy(), r.h)
            bufs[j] = None
    j = wl.n_iters - 1
    P = bufs[j]
    tgm.tgm_update_memory(st.st, st.m, st.g, j, P["nodes"], P["n"], st.cap, P["mem"], P["mts"],
                          P["mail"], P["lts"], P["ver"], P["lo"], P["b"], P["rpos"][:P["b"]],
                          P["rpos"][P["b"]:2 * P["b"]], P["new"])
    o.step()
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()
