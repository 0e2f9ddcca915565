"""fp64 CPU oracle for the memory-module stage (test infrastructure).

TEST INFRASTRUCTURE ONLY: the yardstick the GPU library is checked against.
Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU path;
the arithmetic lives in ``tgm_oracle.c`` (plain C, fp64) and this module only
marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tgm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_i32p = C.POINTER(C.c_int32)
_i64p = C.POINTER(C.c_int64)
_f64p = C.POINTER(C.c_double)
_f32p = C.POINTER(C.c_float)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, OpenMP over independent units)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


class _Desc(C.Structure):
    _fields_ = [("N", C.c_int), ("E", C.c_int64),
                ("src", _i32p), ("dst", _i32p), ("neg", _i32p), ("t", _f64p),
                ("efeat", _f32p),
                ("D_e", C.c_int), ("M", C.c_int), ("D_t", C.c_int), ("H", C.c_int),
                ("nb", C.c_int), ("B", C.c_int), ("s", C.c_int),
                ("W_ih", _f32p), ("W_hh", _f32p), ("b_ih", _f32p), ("b_hh", _f32p),
                ("omega", _f64p), ("beta", _f64p),
                ("W_q", _f32p), ("b_q", _f32p), ("W_k", _f32p), ("b_k", _f32p),
                ("W_v", _f32p), ("b_v", _f32p), ("W_o", _f32p), ("b_o", _f32p),
                ("kind", C.c_int), ("w_t", _f32p), ("K_mb", C.c_int), ("propagate", C.c_int)]

KINDS = {"tgn": 0, "jodie": 1, "apan": 2}


class _StepOut(C.Structure):
    _fields_ = [("iter", C.c_int64), ("b", C.c_int32), ("R", C.c_int32), ("n_U", C.c_int32),
                ("pad_", C.c_int32),
                ("root", _i32p), ("root_ts", _f64p), ("nbr", _i32p), ("eid", _i32p),
                ("nts", _f64p), ("cnt", _i32p), ("U", _i32p), ("root_pos", _i32p),
                ("nbr_pos", _i32p), ("f_mem", _f64p), ("f_mem_ts", _f64p), ("f_mail", _f64p),
                ("f_mail_ts", _f64p), ("f_ver", _i32p), ("s_new", _f64p),
                ("new_mem_ts", _f64p), ("h", _f64p), ("winner", _i64p),
                ("m_mem", _f64p), ("m_stale", _i32p), ("m_omega", _i32p), ("m_gamma", C.c_double),
                ("m_n_stale", C.c_int32), ("m_pad", C.c_int32), ("x_mem", _f64p),
                ("loss", C.c_double), ("grad", _f64p), ("params", _f64p),
                ("relu_margin", C.c_double), ("f_mb", _f64p), ("f_mb_ts", _f64p),
                ("f_mb_cnt", _i32p)]

OPTIMIZERS = {"sgd": 0, "adam": 1}
# the parameter vector's tensors, in order (orc_param_sizes)
PARAM_NAMES = ("W_ih", "W_hh", "b_ih", "b_hh", "W_q", "b_q", "W_k", "b_k", "W_v", "b_v", "W_o",
               "b_o", "W_src", "W_dst", "b_p", "w_out", "b_out")


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = C.CDLL(_LIB)
        L.orc_time_encode.argtypes = [C.c_int, _f64p, _f64p, C.c_double, _f64p]
        L.orc_gru_cell.argtypes = [C.c_int, C.c_int, _f64p, _f64p, _f64p, _f64p, _f64p, _f64p,
                                   _f64p]
        L.orc_embed_one.argtypes = [C.c_int] * 4 + [_f64p] * 10 + [_f64p, C.c_double, C.c_int,
                                                                    _f64p, _f64p, _f64p, _f64p]
        L.orc_sample.argtypes = [C.c_int, C.c_int64, _i32p, _i32p, _f64p, C.c_int, _i32p, _f64p,
                                 C.c_int, _i32p, _i32p, _f64p, _i32p]
        L.orc_sample.restype = C.c_int
        L.orc_create.argtypes = [C.POINTER(_Desc)]
        L.orc_create.restype = C.c_void_p
        L.orc_destroy.argtypes = [C.c_void_p]
        L.orc_flush.argtypes = [C.c_void_p]
        L.orc_set_state.argtypes = [C.c_void_p, C.c_int64, _f64p, _f64p, _f64p, _f64p, _i32p]
        L.orc_get_state.argtypes = [C.c_void_p, _f64p, _f64p, _f64p, _f64p, _i32p]
        L.orc_push_wset.argtypes = [C.c_void_p, C.c_int64, C.c_int, _i32p, _f64p, _f64p, _f64p,
                                    _f64p]
        L.orc_push_wset.restype = C.c_int
        L.orc_next_iter.argtypes = [C.c_void_p]
        L.orc_next_iter.restype = C.c_int64
        L.orc_step.argtypes = [C.c_void_p, C.POINTER(_StepOut)]
        L.orc_step.restype = C.c_int
        L.orc_set_mitigation.argtypes = [C.c_void_p, C.c_int, C.c_double, C.c_double, C.c_int]
        L.orc_set_mitigation.restype = C.c_int
        L.orc_rnn_cell.argtypes = [C.c_int, C.c_int] + [_f64p] * 7
        L.orc_time_projection.argtypes = [C.c_int, _f64p, _f64p, C.c_double, C.c_double, _f64p]
        L.orc_quantile_nearest_rank.argtypes = [C.c_int, _f64p, C.c_double]
        L.orc_quantile_nearest_rank.restype = C.c_double
        L.orc_set_training.argtypes = [C.c_void_p, C.c_int, C.c_double, C.c_double, C.c_double,
                                       C.c_double, _f32p, _f32p, _f32p, _f32p, C.c_float]
        L.orc_set_training.restype = C.c_int
        L.orc_param_count.argtypes = [C.c_void_p]
        L.orc_param_count.restype = C.c_int64
        L.orc_param_sizes.argtypes = [C.c_void_p, _i64p]
        L.orc_get_params.argtypes = [C.c_void_p, _f64p]
        L.orc_get_mailbox.argtypes = [C.c_void_p, _f64p, _f64p, _i32p]
        L.orc_set_mailbox.argtypes = [C.c_void_p, _f64p, _f64p, _i32p]
        L.orc_set_mailbox.restype = C.c_int
        L.orc_set_threads.argtypes = [C.c_int]
        L.orc_set_threads.restype = C.c_int
        _lib = L
    return _lib


def set_threads(n: int = 0) -> int:
    """Threads of the oracle's OpenMP loops (n < 1: unchanged); returns the
    count in use."""
    return int(lib().orc_set_threads(int(n)))


def _p(a, typ):
    if a is None:
        return C.cast(None, typ)
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(typ)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# Building blocks (used by the pins)
# ---------------------------------------------------------------------------

def time_encode(omega, beta, dt) -> np.ndarray:
    omega, beta = _f64(omega), _f64(beta)
    out = np.empty(len(omega))
    lib().orc_time_encode(len(omega), _p(omega, _f64p), _p(beta, _f64p), float(dt),
                          _p(out, _f64p))
    return out


def rnn_cell(W_ih, W_hh, b_ih, b_hh, x, h) -> np.ndarray:
    W_ih, W_hh, b_ih, b_hh, x, h = map(_f64, (W_ih, W_hh, b_ih, b_hh, x, h))
    M = h.shape[0]
    D_x = x.shape[0]
    assert W_ih.shape == (M, D_x) and W_hh.shape == (M, M)
    out = np.empty(M)
    lib().orc_rnn_cell(M, D_x, *(_p(a, _f64p) for a in (W_ih, W_hh, b_ih, b_hh, x, h)),
                       _p(out, _f64p))
    return out


def time_projection(w_t, s, ts, tq) -> np.ndarray:
    w_t, s = _f64(w_t), _f64(s)
    out = np.empty(len(s))
    lib().orc_time_projection(len(s), _p(w_t, _f64p), _p(s, _f64p), float(ts), float(tq),
                              _p(out, _f64p))
    return out


def gru_cell(W_ih, W_hh, b_ih, b_hh, x, h) -> np.ndarray:
    W_ih, W_hh, b_ih, b_hh, x, h = map(_f64, (W_ih, W_hh, b_ih, b_hh, x, h))
    M = h.shape[0]
    D_x = x.shape[0]
    assert W_ih.shape == (3 * M, D_x) and W_hh.shape == (3 * M, M)
    out = np.empty(M)
    lib().orc_gru_cell(M, D_x, *(_p(a, _f64p) for a in (W_ih, W_hh, b_ih, b_hh, x, h)),
                       _p(out, _f64p))
    return out


def embed_one(w, H, s_v, tq, s_u, f, nts) -> np.ndarray:
    """Embedding of one root from explicit neighbour rows (``w`` a Weights)."""
    s_v = _f64(s_v)
    M = s_v.shape[0]
    s_u = _f64(s_u).reshape(-1, M)
    cnt = s_u.shape[0]
    D_t = len(w.omega)
    D_e = w.W_k.shape[1] - M - D_t
    f = _f64(f).reshape(cnt, D_e) if D_e > 0 else np.zeros((cnt, 0))
    nts = _f64(nts).reshape(cnt)
    ws = [_f64(x) for x in (w.omega, w.beta, w.W_q, w.b_q, w.W_k, w.b_k, w.W_v, w.b_v,
                             w.W_o, w.b_o)]
    out = np.empty(M)
    lib().orc_embed_one(M, D_e, D_t, H, *(_p(x, _f64p) for x in ws), _p(s_v, _f64p), float(tq),
                        cnt, _p(np.ascontiguousarray(s_u), _f64p),
                        _p(np.ascontiguousarray(f), _f64p), _p(nts, _f64p), _p(out, _f64p))
    return out


def sample(N, src, dst, t, root, root_ts, nb):
    src = np.ascontiguousarray(src, dtype=np.int32)
    dst = np.ascontiguousarray(dst, dtype=np.int32)
    t = _f64(t)
    root = np.ascontiguousarray(root, dtype=np.int32)
    root_ts = _f64(root_ts)
    R = len(root)
    nbr = np.empty((R, nb), np.int32)
    eid = np.empty((R, nb), np.int32)
    nts = np.empty((R, nb), np.float64)
    cnt = np.empty(R, np.int32)
    rc = lib().orc_sample(N, len(src), _p(src, _i32p), _p(dst, _i32p), _p(t, _f64p), R,
                          _p(root, _i32p), _p(root_ts, _f64p), nb, _p(nbr, _i32p),
                          _p(eid, _i32p), _p(nts, _f64p), _p(cnt, _i32p))
    assert rc == 0
    return nbr, eid, nts, cnt


def quantile_nearest_rank(x, p) -> float:
    """The ceil(p n)-th smallest of the n values x (the staleness threshold of
    the mitigation, Sec. 3.3)."""
    x = _f64(x)
    return float(lib().orc_quantile_nearest_rank(len(x), _p(x, _f64p), float(p)))


# ---------------------------------------------------------------------------
# Stateful driver
# ---------------------------------------------------------------------------

@dataclass
class StepResult:
    iter: int
    b: int
    R: int
    n_U: int
    root: np.ndarray
    root_ts: np.ndarray
    nbr: np.ndarray
    eid: np.ndarray
    nts: np.ndarray
    cnt: np.ndarray
    U: np.ndarray
    root_pos: np.ndarray
    nbr_pos: np.ndarray
    f_mem: np.ndarray
    f_mem_ts: np.ndarray
    f_mail: np.ndarray
    f_mail_ts: np.ndarray
    f_ver: np.ndarray
    s_new: np.ndarray
    new_mem_ts: np.ndarray
    h: np.ndarray
    winner: np.ndarray
    # staleness mitigation (None when off): mitigated fetched memories, stale
    # positions in U, their Omega as positions [n_stale x K] (-1 padded), gamma
    m_mem: np.ndarray | None = None
    m_stale: np.ndarray | None = None
    m_omega: np.ndarray | None = None
    m_gamma: float | None = None
    # the exact memories of U: committed state plus every write set of
    # iterations <= i-1 (what a fetch without staleness would read here)
    x_mem: np.ndarray | None = None
    # training (None when off): the loss, the gradient of the parameter
    # vector and the parameters after the optimizer step
    loss: float | None = None
    grad: np.ndarray | None = None
    params: np.ndarray | None = None
    # the smallest |pre-activation| of the ReLUs on the gradient's path
    relu_margin: float | None = None
    # APAN: the fetched mailboxes, oldest mail first
    f_mb: np.ndarray | None = None
    f_mb_ts: np.ndarray | None = None
    f_mb_cnt: np.ndarray | None = None


class Oracle:
    """Runs the stage iteration by iteration on a workload (``workloads.Workload``)."""

    def __init__(self, wl, w, s: int | None = None, mitigation: dict | None = None,
                 training: dict | None = None):
        """``mitigation=dict(p=.., lam=.., K=..)`` enables the MSPipe-S step
        (Sec. 3.3) between the fetch and the memory update.
        ``training=dict(predictor=P, opt="sgd"|"adam", lr=.., beta1=..,
        beta2=.., eps=..)`` adds the training step (link-prediction loss,
        gradient, optimizer) after each iteration; P a
        ``workloads.Predictor``."""
        self.wl = wl
        self.mitigation = mitigation
        self.s = wl.s if s is None else s
        self.M, self.D_m, self.N, self.nb, self.B = wl.M, wl.D_m, wl.N, wl.nb, wl.B
        self._keep = []

        def keep(a, dt):
            a = np.ascontiguousarray(a, dtype=dt)
            self._keep.append(a)
            return a

        d = _Desc()
        d.N, d.E = wl.N, wl.E
        d.src = _p(keep(wl.src, np.int32), _i32p)
        d.dst = _p(keep(wl.dst, np.int32), _i32p)
        d.neg = _p(keep(wl.neg, np.int32), _i32p)
        d.t = _p(keep(wl.t, np.float64), _f64p)
        d.efeat = _p(keep(wl.efeat, np.float32), _f32p) if wl.D_e > 0 else C.cast(None, _f32p)
        d.D_e, d.M, d.D_t, d.H, d.nb, d.B, d.s = (wl.D_e, wl.M, wl.D_t, wl.H, wl.nb, wl.B,
                                                  self.s)
        for name in ("W_ih", "W_hh", "b_ih", "b_hh", "W_q", "b_q", "W_k", "b_k", "W_v", "b_v",
                     "W_o", "b_o", "w_t"):
            a = getattr(w, name, None)
            setattr(d, name, _p(keep(a, np.float32), _f32p) if a is not None else
                    C.cast(None, _f32p))
        d.kind = KINDS[getattr(w, "kind", "tgn")]
        self.K_mb = int(getattr(w, "K_mb", 0) or 0)
        d.K_mb = self.K_mb
        d.propagate = 1 if getattr(w, "propagate", False) else 0
        d.omega = _p(keep(w.omega, np.float64), _f64p)
        d.beta = _p(keep(w.beta, np.float64), _f64p)
        self._desc = d
        h = lib().orc_create(C.byref(d))
        if not h:
            raise ValueError("oracle: invalid description")
        self._h = h
        if mitigation is not None:
            rc = lib().orc_set_mitigation(h, 1, float(mitigation["p"]), float(mitigation["lam"]),
                                          int(mitigation["K"]))
            if rc != 0:
                raise ValueError("oracle: invalid mitigation parameters")
        self.training = training
        self.n_params = 0
        if training is not None:
            P = training["predictor"]
            pw = [keep(getattr(P, k), np.float32) for k in ("W_src", "W_dst", "b_p", "w_out")]
            rc = lib().orc_set_training(
                h, OPTIMIZERS[training.get("opt", "adam")], float(training.get("lr", 1e-4)),
                float(training.get("beta1", 0.9)), float(training.get("beta2", 0.999)),
                float(training.get("eps", 1e-8)), *(_p(a, _f32p) for a in pw),
                float(P.b_out))
            if rc != 0:
                raise ValueError("oracle: invalid training parameters")
            self.n_params = int(lib().orc_param_count(h))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().orc_destroy(h)
            self._h = None

    @property
    def next_iter(self) -> int:
        return int(lib().orc_next_iter(self._h))

    def step(self, want: str = "all") -> StepResult | None:
        """Run the next iteration; ``want='light'`` skips the big float outputs."""
        B, nb, N, M, D_m = self.B, self.nb, self.N, self.M, self.D_m
        R = 3 * B
        o = _StepOut()
        arrs = dict(root=np.empty(R, np.int32), root_ts=np.empty(R), nbr=np.empty(R * nb, np.int32),
                    eid=np.empty(R * nb, np.int32), nts=np.empty(R * nb), cnt=np.empty(R, np.int32),
                    U=np.empty(N, np.int32), root_pos=np.empty(R, np.int32),
                    nbr_pos=np.empty(R * nb, np.int32), f_mem_ts=np.empty(N),
                    f_mail_ts=np.empty(N), f_ver=np.empty(N, np.int32), new_mem_ts=np.empty(N),
                    winner=np.empty(N, np.int64))
        if want == "all":
            arrs.update(f_mem=np.empty(N * M), f_mail=np.empty(N * D_m + 1),
                        s_new=np.empty(N * M), h=np.empty(R * M), x_mem=np.empty(N * M))
        mit = self.mitigation
        if mit is not None:
            K = int(mit["K"])
            arrs.update(m_mem=np.empty(N * M), m_stale=np.empty(N, np.int32),
                        m_omega=np.empty(N * K, np.int32))
        if self.n_params:
            arrs.update(grad=np.empty(self.n_params), params=np.empty(self.n_params))
        Kmb = self.K_mb
        if Kmb:
            arrs.update(f_mb=np.empty(N * Kmb * D_m + 1), f_mb_ts=np.empty(N * Kmb),
                        f_mb_cnt=np.empty(N, np.int32))
        for k, fld in _StepOut._fields_:
            if k in arrs:
                setattr(o, k, _p(arrs[k], fld))
        rc = lib().orc_step(self._h, C.byref(o))
        if rc == -2:
            return None
        assert rc == 0
        R, nU = o.R, o.n_U
        g = lambda k, n, shape=None: (arrs[k][:n].reshape(shape) if shape else arrs[k][:n]) \
            if k in arrs else None
        return StepResult(
            iter=o.iter, b=o.b, R=R, n_U=nU, root=g("root", R), root_ts=g("root_ts", R),
            nbr=g("nbr", R * nb, (R, nb)), eid=g("eid", R * nb, (R, nb)),
            nts=g("nts", R * nb, (R, nb)), cnt=g("cnt", R), U=g("U", nU),
            root_pos=g("root_pos", R), nbr_pos=g("nbr_pos", R * nb, (R, nb)),
            f_mem=g("f_mem", nU * M, (nU, M)), f_mem_ts=g("f_mem_ts", nU),
            f_mail=g("f_mail", nU * D_m, (nU, D_m)), f_mail_ts=g("f_mail_ts", nU),
            f_ver=g("f_ver", nU), s_new=g("s_new", nU * M, (nU, M)),
            new_mem_ts=g("new_mem_ts", nU), h=g("h", R * M, (R, M)), winner=g("winner", nU),
            m_mem=g("m_mem", nU * M, (nU, M)), m_stale=g("m_stale", o.m_n_stale),
            m_omega=(arrs["m_omega"][:o.m_n_stale * int(mit["K"])].reshape(-1, int(mit["K"]))
                     if mit is not None else None),
            m_gamma=o.m_gamma if mit is not None else None,
            x_mem=g("x_mem", nU * M, (nU, M)),
            loss=o.loss if self.n_params else None,
            grad=arrs["grad"] if self.n_params else None,
            params=arrs["params"] if self.n_params else None,
            relu_margin=o.relu_margin if self.n_params else None,
            f_mb=arrs["f_mb"][:nU * Kmb * D_m].reshape(nU, Kmb, D_m) if Kmb else None,
            f_mb_ts=arrs["f_mb_ts"][:nU * Kmb].reshape(nU, Kmb) if Kmb else None,
            f_mb_cnt=arrs["f_mb_cnt"][:nU] if Kmb else None)

    def flush(self):
        lib().orc_flush(self._h)

    def mailbox(self):
        """APAN: the committed mailboxes (rows [N x K_mb x D_m], times
        [N x K_mb], counts [N]), oldest mail first."""
        N, K, D_m = self.N, self.K_mb, self.D_m
        mb, ts, cnt = np.empty(N * K * D_m + 1), np.empty(N * K), np.empty(N, np.int32)
        lib().orc_get_mailbox(self._h, _p(mb, _f64p), _p(ts, _f64p), _p(cnt, _i32p))
        return mb[:N * K * D_m].reshape(N, K, D_m), ts.reshape(N, K), cnt

    def set_mailbox(self, mb, mb_ts, mb_cnt):
        """APAN: replace the committed mailboxes (the layouts of mailbox();
        after set_state, which empties the queue of write sets)."""
        mb, mb_ts = _f64(mb), _f64(mb_ts)
        cnt = np.ascontiguousarray(mb_cnt, dtype=np.int32)
        N, K, D_m = self.N, self.K_mb, self.D_m
        assert mb.size == N * K * D_m and mb_ts.size == N * K and cnt.size == N
        if lib().orc_set_mailbox(self._h, _p(mb, _f64p), _p(mb_ts, _f64p), _p(cnt, _i32p)) != 0:
            raise ValueError("orc_set_mailbox: not an APAN model, or a count outside [0, K_mb]")

    def param_sizes(self) -> list:
        sz = np.zeros(len(PARAM_NAMES), np.int64)
        lib().orc_param_sizes(self._h, _p(sz, _i64p))
        return [int(x) for x in sz]

    def split(self, vec) -> dict:
        """The tensors of a parameter vector, by name (flat)."""
        out, o = {}, 0
        for name, n in zip(PARAM_NAMES, self.param_sizes()):
            out[name] = vec[o:o + n]
            o += n
        return out

    def params(self) -> np.ndarray:
        out = np.empty(self.n_params)
        lib().orc_get_params(self._h, _p(out, _f64p))
        return out

    def state(self):
        N, M, D_m = self.N, self.M, self.D_m
        mem, mem_ts = np.empty((N, M)), np.empty(N)
        mail, mail_ts = np.empty((N, D_m)), np.empty(N)
        ver = np.empty(N, np.int32)
        lib().orc_get_state(self._h, _p(mem, _f64p), _p(mem_ts, _f64p),
                            _p(mail, _f64p) if D_m else C.cast(None, _f64p),
                            _p(mail_ts, _f64p), _p(ver, _i32p))
        return dict(mem=mem, mem_ts=mem_ts, mail=mail, mail_ts=mail_ts, ver=ver)

    def set_state(self, it, mem, mem_ts, mail, mail_ts, ver, pending=()):
        """Committed tables at iteration `it`, then the pending write sets of
        a saved state: (iteration, node, mem, mem_ts, mail, mail_ts) each, in
        iteration order (Eq. 2: a read at i applies those of iteration
        <= i-1-s)."""
        mem, mem_ts, mail, mail_ts = map(_f64, (mem, mem_ts, mail, mail_ts))
        ver = np.ascontiguousarray(ver, dtype=np.int32)
        lib().orc_set_state(self._h, int(it), _p(mem, _f64p), _p(mem_ts, _f64p),
                            _p(mail, _f64p), _p(mail_ts, _f64p), _p(ver, _i32p))
        for j, node, wm, wmt, wl, wlt in pending:
            node = np.ascontiguousarray(node, dtype=np.int32)
            wm, wmt, wl, wlt = map(_f64, (wm, wmt, wl, wlt))
            assert lib().orc_push_wset(self._h, int(j), len(node), _p(node, _i32p),
                                       _p(wm, _f64p), _p(wmt, _f64p), _p(wl, _f64p),
                                       _p(wlt, _f64p)) == 0
