"""Checkpoint and resume of the versioned state (tgm_state_save /
tgm_state_restore): a run stopped after iteration k-1, saved, and resumed in
a fresh state from the checkpoint gives bit for bit the outputs and final
tables of the run that was not stopped (which the parity tests compare with
the oracle).  With s > 0 the checkpoint holds staged write sets that no fetch
has needed yet, so the resumed run commits them itself."""
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


def _same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), k


@pytest.mark.parametrize("s,k,model,mit", [(0, 7, "tgn", None), (2, 9, "tgn", None),
                                           (3, 1, "tgn", None), (2, 11, "jodie", None),
                                           (1, 10, "tgn", dict(p=0.7, lam=0.9, K=4))])
def test_resume_equals_uninterrupted_sequential(s, k, model, mit):
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=6000, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model=model)
    n = wl.n_iters
    print(f"[ckpt] tiny s={s} {model} mitigation={mit} stop after {k}, iters {n}", flush=True)

    def from_workload_(wl, w):
        return from_workload(wl, w, mitigation=mit)

    a = from_workload_(wl, w)
    want = []
    for i in range(n):
        a.step(i)
        if i >= k:
            want.append(a.outputs())
    a.flush()
    final = a.state()
    a.close()
    b = from_workload_(wl, w)
    for i in range(k):
        b.step(i)
    ck = b.save_checkpoint()
    b.close()
    c = from_workload_(wl, w)
    c.restore_checkpoint(ck)
    for i in range(k, n):
        c.step(i)
        _same(c.outputs(), want[i - k])
    c.flush()
    _same(c.state(), final)
    c.close()


@pytest.mark.parametrize("name,s,E,k", [("tiny", 2, None, 13), ("wiki", 1, 30_000, 24)])
def test_resume_equals_uninterrupted_pipelined(name, s, E, k):
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload(name, E=E, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    n = wl.n_iters
    print(f"[ckpt] pipelined {name} s={s} stop after {k}, iters {n}", flush=True)
    a = from_workload(wl, w)
    a.run(0, n)
    out = a.outputs()
    a.flush()
    final = a.state()
    a.close()
    b = from_workload(wl, w)
    b.run(0, k)
    ck = b.save_checkpoint()
    b.close()
    c = from_workload(wl, w)
    c.restore_checkpoint(ck)
    c.run(k, n - k)
    _same(c.outputs(), out)
    c.flush()
    _same(c.state(), final)
    c.close()


def test_checkpoint_argument_errors():
    from paper_2402_15113_amd import tgm
    from paper_2402_15113_amd.stage import from_workload
    wl = make_workload("tiny", E=3000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    a = from_workload(wl, w)
    for i in range(4):
        a.step(i)
    ck = a.save_checkpoint()
    assert ck.nbytes == tgm.tgm_state_checkpoint_bytes(a.st)

    def code(fn):
        with pytest.raises(tgm.TgmError) as e:
            fn()
        return e.value.code

    assert code(lambda: tgm.tgm_state_save(a.st, stream=a.stream, nbytes=ck.nbytes - 8)) == \
        tgm.TGM_ESIZE
    assert code(lambda: a.restore_checkpoint(ck[:-8])) == tgm.TGM_ESIZE
    bad = ck.copy()
    bad[0] ^= 1                                   # magic
    assert code(lambda: a.restore_checkpoint(bad)) == tgm.TGM_EINVAL
    bad = ck.copy().view(np.int64)
    bad[8] = bad[7] - 1                           # staged before committed
    assert code(lambda: a.restore_checkpoint(bad.view(np.uint8))) == tgm.TGM_EINVAL
    other = from_workload(wl, w, s=2)             # another staleness
    assert code(lambda: other.restore_checkpoint(ck)) == tgm.TGM_EINVAL
    other.close()
    # a failed restore leaves the state as it was: the run continues
    a.step(4)
    a.restore_checkpoint(ck)                      # and a good one rewinds it
    a.step(4)
    torch.cuda.synchronize()
    a.close()


@pytest.mark.parametrize("name,s,E,j,n", [("tiny", 2, 6000, 15, 12), ("wiki", 3, 40_000, 40, 12)])
def test_window_resumed_from_gpu_checkpoint(orc, name, s, E, j, n):
    """A parity window that starts mid-run from a GPU checkpoint: the GPU runs
    iterations 0..j-1 (pipelined), saves, and a fresh state restored from the
    checkpoint runs j..j+n-1.  The oracle runs 0..j+n-1 on its own (it takes
    no input from the GPU) and every step of the window is compared.  The
    checkpoint's content is checked too: its committed tables with its pending
    write sets applied in order equal the tables of a separate oracle run
    through j-1 and flushed."""
    from ckpt_format import parse
    from paper_2402_15113_amd.stage import from_workload
    from test_gpu_parity import close, compare_state, compare_step, exact
    wl = make_workload(name, E=E, s=s)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    a = from_workload(wl, w)
    a.run(0, j)
    raw = a.save_checkpoint()
    a.close()
    ck = parse(raw)
    print(f"[ckpt] {name} s={s}: resume at {ck['next_iter']} with "
          f"{len(ck['pending'])} pending write sets", flush=True)
    assert ck["next_iter"] == j and len(ck["pending"]) == s
    # the checkpoint's tables, flushed by hand, against the oracle's
    mem, mem_ts, mail, mail_ts, ver = (ck[k].copy() for k in ("mem", "mem_ts", "mail",
                                                               "mail_ts", "ver"))
    for it, node, wm, wmt, wml, wmlt in ck["pending"]:
        mem[node], mem_ts[node], mail[node], mail_ts[node], ver[node] = wm, wmt, wml, wmlt, it
    ref = orc.Oracle(wl, w)
    for i in range(j):
        ref.step(want="light")
    ref.flush()
    rs = ref.state()
    exact("ver", ver, rs["ver"])
    exact("mem_ts", mem_ts, rs["mem_ts"])
    exact("mail_ts", mail_ts, rs["mail_ts"])
    close("mem", mem, rs["mem"])
    close("mail", mail, rs["mail"])
    del ref
    # the resumed run against an oracle that ran from the start
    st = from_workload(wl, w)
    st.restore_checkpoint(raw)
    o = orc.Oracle(wl, w)
    for i in range(j):
        o.step(want="light")
    for i in range(j, j + n):
        st.step(i)
        compare_step(st.outputs(), o.step(want="all"))
    st.flush()
    o.flush()
    compare_state(st.state(), o.state())
    st.close()
