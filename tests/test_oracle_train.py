"""Pins for the oracle's training step (loss, gradient, optimizer).

* torch fp64 autograd -- the same iteration's forward written with torch ops
  (GRUCell, masked multi-head attention, the link predictor,
  binary_cross_entropy_with_logits) from the oracle's fetched rows; autograd's
  gradient of every parameter must equal the oracle's (the gradient is derived
  by autograd, not retyped);
* finite differences -- central differences of the oracle's own loss, with
  one weight moved up and down for one iteration, against its gradient;
* closed forms -- a zero output layer gives loss 2 log 2 and zero gradients
  below it; SGD moves theta by exactly -lr g; Adam's first step moves each
  coordinate by -lr g / (|g| + eps).
"""
import math

import numpy as np
import pytest

from workloads import make_predictor, make_weights, make_workload

torch = pytest.importorskip("torch")


def _oracle(orc, wl, w, P, s=None, opt="sgd", lr=0.0, mitigation=None):
    return orc.Oracle(wl, w, s=s, mitigation=mitigation,
                      training=dict(predictor=P, opt=opt, lr=lr))


def _torch_iteration(wl, w, P, r):
    """Forward of iteration r (an oracle StepResult) in torch fp64, from the
    rows it fetched; returns (loss, {name: tensor}, s_new, h)."""
    T = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    prm = {k: T(getattr(w, k)) for k in ("W_ih", "W_hh", "b_ih", "b_hh", "W_q", "b_q", "W_k",
                                         "b_k", "W_v", "b_v", "W_o", "b_o")}
    prm.update(W_src=T(P.W_src), W_dst=T(P.W_dst), b_p=T(P.b_p), w_out=T(P.w_out),
               b_out=T([P.b_out]))
    M, H, D_e, nb = wl.M, wl.H, wl.D_e, wl.nb
    om = torch.tensor(np.asarray(w.omega, np.float64))
    be = torch.tensor(np.asarray(w.beta, np.float64))
    phi = lambda dt: torch.cos(dt[..., None] * om + be)
    cell = torch.nn.GRUCell(wl.D_m + wl.D_t, M).double()
    fmem = torch.tensor(r.m_mem if r.m_mem is not None else r.f_mem)
    x = torch.cat([torch.tensor(r.f_mail), phi(torch.tensor(r.f_mail_ts - r.f_mem_ts))], dim=1)
    gru = torch.func.functional_call(cell, {"weight_ih": prm["W_ih"], "weight_hh": prm["W_hh"],
                                            "bias_ih": prm["b_ih"], "bias_hh": prm["b_hh"]},
                                     (x, fmem))
    has = torch.tensor(r.f_ver >= 0)[:, None]
    s_new = torch.where(has, gru, fmem)
    R = r.R
    rp = torch.tensor(r.root_pos.astype(np.int64))
    npos = torch.tensor(np.maximum(r.nbr_pos, 0).astype(np.int64))
    valid = torch.tensor(r.nbr_pos >= 0)
    sv = s_new[rp]
    xq = torch.cat([sv, phi(torch.zeros(R, dtype=torch.float64))], dim=1)
    q = xq @ prm["W_q"].T + prm["b_q"]
    f = np.zeros((R, nb, D_e))
    if D_e:
        f[r.nbr_pos >= 0] = np.asarray(wl.efeat, np.float64)[r.eid[r.nbr_pos >= 0]]
    dt = torch.tensor(r.root_ts[:, None] - np.where(r.nbr_pos >= 0, r.nts, 0.0))
    kap = torch.cat([s_new[npos], torch.tensor(f), phi(dt)], dim=2) * valid[..., None]
    K = kap @ prm["W_k"].T + prm["b_k"]
    V = kap @ prm["W_v"].T + prm["b_v"]
    dh = M // H
    sc = (q.view(R, 1, H, dh) * K.view(R, nb, H, dh)).sum(-1) / math.sqrt(dh)
    sc = sc.masked_fill(~valid[..., None], float("-inf"))
    al = torch.softmax(sc, dim=1)
    al = torch.where(valid.any(dim=1)[:, None, None], al, torch.zeros_like(al))
    a = (al[..., None] * V.view(R, nb, H, dh)).sum(1).reshape(R, M)
    pre = torch.cat([a, sv], dim=1) @ prm["W_o"].T + prm["b_o"]
    h = torch.relu(pre)
    b = r.b
    zp = h[:b] @ prm["W_src"].T + h[b:2 * b] @ prm["W_dst"].T + prm["b_p"]
    zn = h[:b] @ prm["W_src"].T + h[2 * b:] @ prm["W_dst"].T + prm["b_p"]
    sp = torch.relu(zp) @ prm["w_out"] + prm["b_out"]
    sn = torch.relu(zn) @ prm["w_out"] + prm["b_out"]
    bce = torch.nn.functional.binary_cross_entropy_with_logits
    loss = bce(sp, torch.ones(b, dtype=torch.float64), reduction="sum") / b + \
        bce(sn, torch.zeros(b, dtype=torch.float64), reduction="sum") / b
    return loss, prm, s_new, h, pre


@pytest.mark.parametrize("name,kw,s,first,mit", [
    ("tiny", dict(E=3000), 0, 6, None),
    ("tiny", dict(E=3000), 2, 9, None),
    ("tiny", dict(E=4000), 2, 12, dict(p=0.8, lam=0.6, K=3)),
    ("lastfm", dict(E=8000, B=400), 2, 8, None),   # no edge features, heavy repetition
])
def test_gradient_equals_torch_autograd(orc, name, kw, s, first, mit):
    wl = make_workload(name, s=s, **kw)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    P = make_predictor(wl.M, seed=3)
    o = _oracle(orc, wl, w, P, s=s, mitigation=mit)
    for _ in range(first):
        o.step(want="light")
    r = o.step()
    loss, prm, s_new, h, _ = _torch_iteration(wl, w, P, r)
    np.testing.assert_allclose(s_new.detach().numpy(), r.s_new, rtol=0, atol=1e-12)
    np.testing.assert_allclose(h.detach().numpy(), r.h, rtol=0, atol=1e-12)
    assert abs(loss.item() - r.loss) < 1e-12
    loss.backward()
    got = o.split(r.grad)
    for k, t in prm.items():
        ref = t.grad.numpy().ravel()
        np.testing.assert_allclose(got[k], ref, rtol=1e-9, atol=1e-13, err_msg=k)
        if k not in ("b_out",):
            assert np.abs(ref).max() > 0, k   # every tensor takes part


def test_gradient_matches_finite_differences(orc):
    """Central differences of the oracle's loss at iteration j (s = 0, so the
    flushed state after j-1 is what iteration j reads) for a spread of
    coordinates of every parameter tensor."""
    import dataclasses
    wl = make_workload("tiny", E=2400, s=0)
    wl = dataclasses.replace(wl, N=60, src=wl.src % 60, dst=wl.dst % 60, neg=wl.neg % 60, B=40,
                             M=6, D_t=4, H=2, nb=4, efeat=wl.efeat[:, :5], D_e=5)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random", seed=4)
    P = make_predictor(wl.M, seed=5)
    j = 20
    base = _oracle(orc, wl, w, P, s=0)
    for _ in range(j):
        base.step(want="light")
    base.flush()
    st = base.state()

    def at(w_, P_):
        o = _oracle(orc, wl, w_, P_, s=0)
        o.set_state(j, **st)
        return o.step()

    r0 = at(w, P)
    g = base.split(r0.grad)
    rng = np.random.default_rng(0)
    delta = 2.0 ** -14
    checked = 0
    for name in g:
        src = P if name in ("W_src", "W_dst", "b_p", "w_out", "b_out") else w
        arr = np.atleast_1d(np.asarray(getattr(src, name), np.float32))
        for idx in rng.choice(arr.size, size=min(4, arr.size), replace=False):
            def moved(d):
                a = arr.copy().ravel()
                a[idx] = np.float32(a[idx] + d)
                a = a.reshape(arr.shape)
                if src is P:
                    P2 = dataclasses.replace(P, **{name: float(a[0]) if name == "b_out" else a})
                    return at(w, P2).loss
                return at(dataclasses.replace(w, **{name: a}), P).loss
            fd = (moved(delta) - moved(-delta)) / (2 * delta)
            an = g[name][idx]
            assert abs(fd - an) <= 1e-3 * abs(an) + 1e-8, (name, idx, fd, an)
            checked += 1
    assert checked >= 60


def test_zero_output_layer_closed_form(orc):
    """w_out = 0, b_out = 0: every score is 0, the loss is 2 log 2, b_out's
    gradient is (1/b) sum (sigma(0) - 1 + sigma(0)) = 0 and nothing below the
    output layer gets a gradient; w_out's is (1/b) sum (ReLU(z_neg) - ReLU(z_pos)) / 2."""
    import dataclasses
    wl = make_workload("tiny", E=2000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    P = dataclasses.replace(make_predictor(wl.M), w_out=np.zeros(wl.M, np.float32), b_out=0.0)
    o = _oracle(orc, wl, w, P, s=1)
    for _ in range(4):
        o.step(want="light")
    r = o.step()
    assert abs(r.loss - 2 * math.log(2)) < 1e-13   # 2b terms of log 2, summed
    g = o.split(r.grad)
    assert g["b_out"][0] == 0.0
    for k, v in g.items():
        if k != "w_out" and k != "b_out":
            assert not np.any(v), k
    b = r.b
    h = r.h
    Ws = np.asarray(P.W_src, np.float64)
    Wd = np.asarray(P.W_dst, np.float64)
    zp = h[:b] @ Ws.T + h[b:2 * b] @ Wd.T + P.b_p
    zn = h[:b] @ Ws.T + h[2 * b:] @ Wd.T + P.b_p
    want = (np.maximum(zn, 0) - np.maximum(zp, 0)).sum(0) / (2 * b)
    np.testing.assert_allclose(g["w_out"], want, rtol=1e-12, atol=1e-15)


def test_sgd_and_adam_steps(orc):
    wl = make_workload("tiny", E=2000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t)
    P = make_predictor(wl.M)
    for opt, lr in (("sgd", 0.05), ("adam", 1e-3)):
        o = _oracle(orc, wl, w, P, s=1, opt=opt, lr=lr)
        before = o.params()
        r = o.step()
        if opt == "sgd":
            assert np.array_equal(r.params, before - lr * r.grad)
        else:   # first Adam step: m_hat = g, v_hat = g^2
            np.testing.assert_allclose(r.params - before,
                                       -lr * r.grad / (np.abs(r.grad) + 1e-8),
                                       rtol=1e-9, atol=1e-16)
        # the next iteration runs with the new weights
        r2 = o.step()
        assert not np.array_equal(r2.params, r.params)


def test_relu_margin_is_the_smallest_pre_activation(orc):
    """The reported margin equals the smallest |z| of the predictor and |o| of
    the output projection, recomputed here from the torch forward."""
    wl = make_workload("tiny", E=3000, s=1)
    w = make_weights(wl.M, wl.D_e, wl.D_t, beta="random")
    P = make_predictor(wl.M, seed=3)
    o = _oracle(orc, wl, w, P, s=1)
    for _ in range(5):
        o.step(want="light")
    r = o.step()
    _, prm, s_new, h, pre = _torch_iteration(wl, w, P, r)
    b = r.b
    with torch.no_grad():
        hh = torch.tensor(r.h)
        zp = hh[:b] @ prm["W_src"].T + hh[b:2 * b] @ prm["W_dst"].T + prm["b_p"]
        zn = hh[:b] @ prm["W_src"].T + hh[2 * b:] @ prm["W_dst"].T + prm["b_p"]
    m = min(zp.abs().min().item(), zn.abs().min().item(), pre.detach().abs().min().item())
    assert abs(r.relu_margin - m) <= 1e-12 * max(m, 1e-300) + 1e-15
