"""Pins for the oracle's JODIE model family: an RNN memory updater and the time
projection embedding h = s' * (1 + w_t (t - ts')).

* RNN cell   -- torch fp64 RNNCell (tanh) and a hand-worked step;
* projection -- closed forms: w_t = 0 or a query at the memory's time gives
                s'; a one-element case by hand;
* the stage  -- a JODIE run's embeddings are the projections of the updated
                memories of the roots (re-derived from the run's own outputs);
                its update is the RNN cell on the GRU's input (a node without
                mail keeps its memory); and it shares sampling, node sets and
                the latest-message winners with TGN on the same stream.
"""
import numpy as np
import pytest
import torch

from workloads import make_weights, make_workload


@pytest.mark.parametrize("seed", range(3))
def test_rnn_matches_torch_rnncell(orc, seed):
    M, D_x = 8, 13
    r = np.random.default_rng(seed)
    W_ih, W_hh = r.uniform(-1, 1, (M, D_x)), r.uniform(-1, 1, (M, M))
    b_ih, b_hh = r.uniform(-1, 1, M), r.uniform(-1, 1, M)
    x, h = r.standard_normal(D_x), r.uniform(-1, 1, M)
    cell = torch.nn.RNNCell(D_x, M, nonlinearity="tanh").double()
    with torch.no_grad():
        for p, v in ((cell.weight_ih, W_ih), (cell.weight_hh, W_hh), (cell.bias_ih, b_ih),
                     (cell.bias_hh, b_hh)):
            p.copy_(torch.from_numpy(v))
        want = cell(torch.from_numpy(x)[None], torch.from_numpy(h)[None])[0].numpy()
    np.testing.assert_allclose(orc.rnn_cell(W_ih, W_hh, b_ih, b_hh, x, h), want,
                               rtol=0, atol=1e-14)


def test_rnn_hand_worked_step(orc):
    # M = 2, D_x = 1: pre-activations 0.5*2 + 0.1 + (0.3*1 - 0.2*(-1)) + 0.0 = 1.6
    # and -1*2 + 0 + (0*1 + 1*(-1)) + 0.5 = -2.5
    W_ih = np.array([[0.5], [-1.0]])
    W_hh = np.array([[0.3, -0.2], [0.0, 1.0]])
    b_ih, b_hh = np.array([0.1, 0.0]), np.array([0.0, 0.5])
    out = orc.rnn_cell(W_ih, W_hh, b_ih, b_hh, np.array([2.0]), np.array([1.0, -1.0]))
    np.testing.assert_allclose(out, [np.tanh(1.6), np.tanh(-2.5)], rtol=0, atol=1e-15)


def test_time_projection_closed_forms(orc):
    s = np.array([1.5, -2.0, 0.25])
    w = np.array([0.1, -0.3, 2.0])
    np.testing.assert_array_equal(orc.time_projection(np.zeros(3), s, 4.0, 9.0), s)
    np.testing.assert_array_equal(orc.time_projection(w, s, 7.0, 7.0), s)
    # one element: 1.5 * (1 + 0.1 * (9 - 4)) = 2.25
    assert orc.time_projection(w[:1], s[:1], 4.0, 9.0)[0] == 2.25


@pytest.fixture(scope="module")
def jodie_run(orc):
    wl = make_workload("tiny", E=5000, s=2)
    w = make_weights(wl.M, wl.D_e, wl.D_t, model="jodie")
    o = orc.Oracle(wl, w)
    return wl, w, [o.step() for _ in range(wl.n_iters)]


def test_embeddings_are_projections(orc, jodie_run):
    wl, w, res = jodie_run
    for r in res:
        p = r.root_pos
        d = r.root_ts - r.new_mem_ts[p]
        want = r.s_new[p] * (1.0 + w.w_t.astype(np.float64)[None, :] * d[:, None])
        np.testing.assert_allclose(r.h, want, rtol=0, atol=1e-13)


def test_update_is_the_rnn_cell(orc, jodie_run):
    wl, w, res = jodie_run
    checked = 0
    for r in res[3:12]:
        for k in range(0, r.n_U, 7):
            if r.f_ver[k] < 0:
                np.testing.assert_array_equal(r.s_new[k], r.f_mem[k])   # no mail: kept
                continue
            x = np.concatenate([r.f_mail[k], orc.time_encode(w.omega, w.beta,
                                                            r.f_mail_ts[k] - r.f_mem_ts[k])])
            want = orc.rnn_cell(w.W_ih, w.W_hh, w.b_ih, w.b_hh, x, r.f_mem[k])
            np.testing.assert_allclose(r.s_new[k], want, rtol=0, atol=1e-13)
            checked += 1
    assert checked > 50


def test_jodie_differs_from_tgn_only_in_the_model(orc):
    # the same stream: identical samples and node sets, different memories
    wl = make_workload("tiny", E=3000, s=1)
    a = orc.Oracle(wl, make_weights(wl.M, wl.D_e, wl.D_t))
    b = orc.Oracle(wl, make_weights(wl.M, wl.D_e, wl.D_t, model="jodie"))
    for _ in range(5):
        ra, rb = a.step(), b.step()
        np.testing.assert_array_equal(ra.U, rb.U)
        np.testing.assert_array_equal(ra.nbr, rb.nbr)
        np.testing.assert_array_equal(ra.winner, rb.winner)
    assert not np.allclose(ra.s_new, rb.s_new)
