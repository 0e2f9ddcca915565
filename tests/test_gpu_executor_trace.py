"""Every iteration of the pipelined executor (tgm_stage_run, the benchmarked
path) against the fp64 oracle.

tgm_stage_run fuses each attention launch with the next iteration's gather
(k_attn_agg_gather; for JODIE k_tproj_gather) and the staging with the node
projections.  Its optional per-iteration copies of h and of the new memories
s' let the embeddings and memories of every iteration be compared element by
element (|gpu - oracle| <= 1e-5 + 1e-4 |oracle|), not only the last one and
the flushed tables.  Windows (Eq. 2 and Alg. 1 define what each must
reproduce): the whole WIKI-shaped stream; the first 64 LastFM-shaped
batches; the first 32 REDDIT-shaped batches at s = 1, 2, 4 and batches
560..591 of a run from the start; GDELT-shaped batches 48..63 of a run from
the start, and a GDELT-shaped window at batch 20,000 from a seeded state.
Also: the executor allocates nothing (tgm_alloc_count does not move).
"""
import dataclasses

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


def projection_close(name, g, r, w):
    """JODIE's embedding h = s' * f with f = 1 + w_t (t - ts') formed exactly in
    fp64 (reading R27): an error e in s' reaches h as |f| e, so h is held to
    the s' tolerance scaled by |f| (1e-5 |f| + 1e-4 |h|).  f can reach ~80 on
    the GDELT-shaped stream, where memory times lag the query by up to 2.5
    years."""
    from test_gpu_parity import ATOL, RTOL
    f = 1.0 + np.asarray(w.w_t, np.float64)[None, :] * \
        (r.root_ts - r.new_mem_ts[r.root_pos])[:, None]
    g = np.asarray(g, np.float64)
    err = np.abs(g - r.h)
    tol = ATOL * np.maximum(1.0, np.abs(f)) + RTOL * np.abs(r.h)
    bad = err > tol
    if bad.any():
        k = np.unravel_index(np.argmax(err - tol), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{bad.size} outside tolerance; worst at "
                             f"{k}: gpu {g[k]!r} oracle {r.h[k]!r} f {f[k]!r}")
    return float(err.max()) if err.size else 0.0


def traced_pair(orc, wl, w, first, n, *, s=None, init=None, gpu_efeat=None, skip_to=None,
                mitigation=None):
    """GPU: the executor over iterations first .. first+n-1 (from the state
    `init`, or from the start); iterations before `skip_to` run untraced.
    Oracle: the same iterations from the same start.  Compares h and s' of
    every iteration from skip_to on, then the flushed tables."""
    from paper_2402_15113_amd.stage import Stage, from_workload
    from test_gpu_parity import close, compare_state
    skip_to = first if skip_to is None else skip_to
    if gpu_efeat is None:
        st = from_workload(wl, w, s=s, mitigation=mitigation)
    else:
        st = Stage(wl.N, wl.src, wl.dst, wl.t, wl.neg, gpu_efeat, w, M=wl.M, D_t=wl.D_t,
                   H=wl.H, nb=wl.nb, B=wl.B, s=wl.s if s is None else s, mitigation=mitigation)
    o = orc.Oracle(wl, w, s=s, mitigation=mitigation)
    if init is not None:
        st.load_state(first, **init)
        o.set_state(first, **init)
    if skip_to > first:
        st.run(first, skip_to - first)
    print(f"[trace] {wl.name} s={st.s} iters {skip_to}..{first + n - 1}", flush=True)
    h_tr, s_tr = st.run(skip_to, first + n - skip_to, trace=True)
    torch.cuda.synchronize()
    worst = {"h": 0.0, "s_new": 0.0}
    for i in range(first, first + n):
        r = o.step(want="all" if i >= skip_to else "light")
        if i < skip_to:
            continue
        k = i - skip_to
        h = h_tr[k, :r.R].cpu().numpy()
        sn = s_tr[k, :r.n_U].cpu().numpy()
        worst["s_new"] = max(worst["s_new"], close(f"s_new[{i}]", sn, r.s_new))
        if getattr(w, "kind", "tgn") == "jodie":
            worst["h"] = max(worst["h"], projection_close(f"h[{i}]", h, r, w))
        else:
            worst["h"] = max(worst["h"], close(f"h[{i}]", h, r.h))
    del h_tr, s_tr
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()
    print(f"[trace] worst abs errors {worst}", flush=True)
    return worst


@pytest.mark.parametrize("model", ["tgn", "jodie"])
def test_wiki_every_iteration(orc, model):
    """The whole WIKI-shaped stream (263 batches, s = 1), every iteration."""
    wl = make_workload("wiki")
    w = make_weights(wl.M, wl.D_e, wl.D_t, model=model)
    traced_pair(orc, wl, w, 0, wl.n_iters)


@pytest.mark.parametrize("model", ["tgn", "jodie"])
def test_lastfm_every_iteration(orc, model):
    """LastFM-shaped (D_e = 0, B = 2000, heavy repetition, s = 2): batches 0..63."""
    wl = make_workload("lastfm", E=64 * 2000)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model=model)
    traced_pair(orc, wl, w, 0, 64)


@pytest.mark.parametrize("s", [1, 2, 4])
def test_reddit_first_32(orc, s):
    wl = make_workload("reddit", E=32 * 600, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    traced_pair(orc, wl, w, 0, 32)


def test_reddit_mid_run_from_the_start(orc):
    """REDDIT-shaped, s = 2: both sides run from the initial state through
    batch 591; batches 560..591 are compared every iteration."""
    wl = make_workload("reddit", E=592 * 600, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    traced_pair(orc, wl, w, 0, 592, skip_to=560)


def test_mitigated_every_iteration(orc):
    """MSPipe-S on (p = 0.9, lambda = 0.5, K = 4) under the executor, tiny stream."""
    wl = make_workload("tiny", E=8000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    traced_pair(orc, wl, w, 0, wl.n_iters, mitigation=dict(p=0.9, lam=0.5, K=4))


@pytest.mark.parametrize("model", ["tgn", "jodie"])
def test_gdelt_window_every_iteration(orc, model):
    """GDELT-shaped (D_e 186, B 4000, s 4): batches 20,000..20,007 on the graph
    of their first 80,032,000 events, from a seeded state."""
    from test_gpu_parity import gdelt_prefix, sparse_features, synthetic_state, window_rows
    j, n = 20_000, 8
    wl = gdelt_prefix((j + n) * 4000)
    rows = window_rows(orc, wl, j, n)
    print(f"[trace] gdelt window: {len(rows)} feature rows", flush=True)
    host, dev = sparse_features(wl, rows)
    wl = dataclasses.replace(wl, efeat=host)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model=model)
    traced_pair(orc, wl, w, j, n, init=synthetic_state(wl, j, 11), gpu_efeat=dev)
    del dev
    torch.cuda.empty_cache()


def test_gdelt_from_the_start(orc):
    """GDELT-shaped (D_e 186, B 4000, s 4): both sides run from the initial
    state through batch 63 (the GPU with the executor); batches 48..63 are
    compared every iteration.  The state the window starts from is each side's
    own: the GPU's after its 48 pipelined batches."""
    from test_gpu_parity import gdelt_prefix
    from workloads import CONFIGS, edge_feature_rows
    wl = gdelt_prefix(64 * 4000)
    wl = dataclasses.replace(wl, efeat=edge_feature_rows(wl.seed, CONFIGS["gdelt"]["E"],
                                                          wl.D_e, 0, wl.E))
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    traced_pair(orc, wl, w, 0, 64, skip_to=48)


@pytest.mark.parametrize("model,mit", [("tgn", None), ("jodie", None),
                                       ("tgn", dict(p=0.7, lam=0.9, K=4))])
def test_executor_allocates_nothing(model, mit):
    """tgm_stage_run allocates no device memory, on its first run with a state
    or a mitigator, and after (tgm_alloc_count: every allocation of the library
    goes through one counted wrapper)."""
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("wiki", E=30_000)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model=model)
    st = from_workload(wl, w, mitigation=mit)
    torch.cuda.synchronize()
    before = tgm.alloc_count()
    st.run(0, 20)
    st.run(20, wl.n_iters - 20)
    torch.cuda.synchronize()
    assert tgm.alloc_count() == before
    st.close()


def test_executor_rejects_too_many_sample_sets():
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=4000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    st = from_workload(wl, w)
    st.run(0, 2)
    sb, fb = st._bufs
    big = (tgm.SampleBuffers * 18)(*([sb[0]] * 18))
    with pytest.raises(tgm.TgmError) as e:
        tgm.tgm_stage_run(st.g, st.st, st.m, 2, 2, st.B, st.nb, st.cap, big, fb, st.mem_new,
                          st.new_mem_ts, None, st.h, st.stream, st.pre_stream)
    assert e.value.code == tgm.TGM_ESIZE
    st.close()
