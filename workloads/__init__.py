"""Seeded synthetic temporal-graph workloads for the memory-module stage.

This module only draws inputs: event streams, negative destinations, edge
features, model weights and time-encoding frequencies.  It holds none of the
method's arithmetic and is shared, unchanged, by the fp64 oracle (tests,
CPU baseline) and by the GPU path (tests, bench).

Every random tensor comes from its own counter-based Philox-4x32-10 stream
(Salmon et al., SC'11) keyed by (seed, tensor name, chunk), so a tensor can
be regenerated piecewise without storing it.

The five workloads stand in for the paper's public datasets (Tab. of dataset
statistics in Sec. 5: WIKI, REDDIT, LastFM, GDELT) with the shapes, sizes and
structure the experiments use: bipartite user-item streams with heavy-tailed
activity, timestamps sorted ascending, one negative destination per positive
event, fixed 10-neighbour sampling and memory dimension 100 (Sec. 5,
training settings).  No dataset item is reproduced.
"""
from __future__ import annotations

import hashlib
import math
import os
from dataclasses import dataclass, field

import numpy as np

__all__ = ["Workload", "Weights", "Predictor", "CONFIGS", "FEAT_CHUNK", "make_workload",
           "make_weights", "make_predictor", "edge_feature_rows", "config_names"]

# Rows per independently keyed chunk of the edge-feature stream.
FEAT_CHUNK = 1 << 16
_FEAT_CHUNK = FEAT_CHUNK


def _key(seed: int, name: str, chunk: int = 0) -> np.ndarray:
    h = hashlib.sha256(f"{seed}/{name}/{chunk}".encode()).digest()
    return np.frombuffer(h[:16], dtype=np.uint64).copy()


def _rng(seed: int, name: str, chunk: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=_key(seed, name, chunk)))


@dataclass
class Workload:
    """One temporal event stream plus the dimensions of the model run on it."""
    name: str
    N: int
    src: np.ndarray          # int32[E]
    dst: np.ndarray          # int32[E]
    t: np.ndarray            # float64[E], ascending; events ordered by (t, index)
    neg: np.ndarray          # int32[E], one negative destination per event
    efeat: np.ndarray | None  # float32[E, D_e], None when D_e == 0
    D_e: int
    M: int                   # memory dimension
    D_t: int                 # time-encoding dimension
    H: int                   # attention heads
    nb: int                  # neighbours per root
    B: int                   # batch size (events)
    s: int                   # staleness: a read at iteration i sees writes <= i-1-s
    seed: int
    meta: dict = field(default_factory=dict)

    @property
    def E(self) -> int:
        return int(self.src.shape[0])

    @property
    def D_m(self) -> int:
        return 2 * self.M + self.D_e

    @property
    def D_x(self) -> int:
        return self.D_m + self.D_t

    @property
    def n_iters(self) -> int:
        return (self.E + self.B - 1) // self.B

    def batch(self, i: int) -> tuple[int, int]:
        lo = i * self.B
        return lo, min(self.E, lo + self.B)


@dataclass
class Weights:
    """Model parameters, row-major.  fp32 except the time encoding (fp64).
    TGN: a GRU updater and attention.  JODIE: an RNN updater ([M, D_x] and
    [M, M] weights, [M] biases) and the time projection w_t [M]; no attention
    weights.  APAN: the GRU updater, fed by an attention over the node's
    mailbox (W_q [M, M + D_t], W_k [M, D_m + D_t] and their biases)."""
    W_ih: np.ndarray  # [3M, D_x]  gate order r, z, n   (JODIE: [M, D_x])
    W_hh: np.ndarray  # [3M, M]                        (JODIE: [M, M])
    b_ih: np.ndarray  # [3M]                           (JODIE: [M])
    b_hh: np.ndarray  # [3M]                           (JODIE: [M])
    omega: np.ndarray  # float64[D_t]
    beta: np.ndarray   # float64[D_t]
    W_q: np.ndarray | None = None   # [d_a, M + D_t]
    b_q: np.ndarray | None = None
    W_k: np.ndarray | None = None   # [d_a, M + D_e + D_t]
    b_k: np.ndarray | None = None
    W_v: np.ndarray | None = None   # [d_a, M + D_e + D_t]
    b_v: np.ndarray | None = None
    W_o: np.ndarray | None = None   # [M, d_a + M]
    b_o: np.ndarray | None = None   # [M]
    kind: str = "tgn"               # "tgn", "jodie" or "apan"
    w_t: np.ndarray | None = None   # [M] JODIE's time projection
    K_mb: int = 0                   # APAN: mails per mailbox
    propagate: bool = False         # APAN: mails also go to the sampled neighbours


# ---------------------------------------------------------------------------
# Workload definitions
# ---------------------------------------------------------------------------

CONFIGS = {
    # name: (description, builder kwargs)
    "tiny": dict(N=1000, E=20_000, D_e=16, M=32, D_t=32, H=2, B=200, s=0),
    "wiki": dict(N=9227, E=157_474, D_e=172, M=100, D_t=100, H=2, B=600, s=1),
    "reddit": dict(N=10_984, E=672_447, D_e=172, M=100, D_t=100, H=2, B=600, s=1),
    "lastfm": dict(N=1980, E=1_293_103, D_e=0, M=100, D_t=100, H=2, B=2000, s=2),
    "gdelt": dict(N=16_682, E=191_290_882, D_e=186, M=100, D_t=100, H=2, B=4000, s=4),
}


def config_names() -> list[str]:
    return list(CONFIGS)


def _inverse_cdf(c: np.ndarray, u: np.ndarray) -> np.ndarray:
    """min(#{k : c[k] <= u}, n - 1) for every u (c non-decreasing, c[-1] == 1):
    the inverse-CDF draw, as searchsorted(c, u, side='right'), run over blocks
    of u on several threads (searchsorted releases the GIL; the result does not
    depend on the split)."""
    from concurrent.futures import ThreadPoolExecutor
    n = len(c)
    out = np.empty(len(u), dtype=np.int64)
    step = 1 << 22

    def block(lo):
        out[lo:lo + step] = np.searchsorted(c, u[lo:lo + step], side="right")

    if len(u) <= step:
        block(0)
    else:
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(block, range(0, len(u), step)))
    np.minimum(out, n - 1, out=out)
    return out


def _bounded_zipf(rng: np.random.Generator, n: int, a: float, size: int) -> np.ndarray:
    """Ranks 0..n-1 with P(rank k) proportional to (k+1)^-a."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-a)
    c = np.cumsum(w)
    c /= c[-1]
    return _inverse_cdf(c, rng.random(size))


def _weighted_choice(rng: np.random.Generator, w: np.ndarray, size: int) -> np.ndarray:
    c = np.cumsum(w.astype(np.float64))
    c /= c[-1]
    return _inverse_cdf(c, rng.random(size))


def _sorted_int_seconds(rng: np.random.Generator, E: int, span: int) -> np.ndarray:
    return np.sort(rng.integers(0, span, size=E)).astype(np.float64)


def _events_tiny(seed, N, E):
    src = _rng(seed, "src").integers(0, N, size=E)
    dst = _rng(seed, "dst").integers(0, N, size=E)
    t = np.sort(_rng(seed, "t").random(E) * 1e6)
    neg = _rng(seed, "neg").integers(0, N, size=E)
    return src, dst, t, neg, {"graph": "uniform src/dst, t ~ U[0,1e6) continuous"}


def _events_wiki(seed, N, E):
    n_user, n_item = 8227, 1000
    assert N == n_user + n_item
    perm = _rng(seed, "user_perm").permutation(n_user)
    src = perm[_bounded_zipf(_rng(seed, "src"), n_user, 1.2, E)]
    dst = n_user + _rng(seed, "dst").integers(0, n_item, size=E)
    t = _sorted_int_seconds(_rng(seed, "t"), E, 30 * 86400)
    neg = n_user + _rng(seed, "neg").integers(0, n_item, size=E)
    return src, dst, t, neg, {"graph": "bipartite 8227 users Zipf(1.2) x 1000 items uniform, "
                                       "integer seconds over 30 days"}


def _events_reddit(seed, N, E):
    n_user, n_item = 10_000, 984
    assert N == n_user + n_item
    # Chung-Lu endpoints: Pareto(1.1) weights on each side => degree tail ~ d^-2.1
    wu = _rng(seed, "user_w").pareto(1.1, n_user) + 1.0
    wi = _rng(seed, "item_w").pareto(1.1, n_item) + 1.0
    src = _weighted_choice(_rng(seed, "src"), wu, E)
    dst = n_user + _weighted_choice(_rng(seed, "dst"), wi, E)
    t = _sorted_int_seconds(_rng(seed, "t"), E, 30 * 86400)
    neg = n_user + _rng(seed, "neg").integers(0, n_item, size=E)
    return src, dst, t, neg, {"graph": "bipartite Chung-Lu, Pareto(1.1) weights both sides, "
                                       "integer seconds over 30 days"}


def _events_lastfm(seed, N, E):
    n_hot = 99
    perm = _rng(seed, "perm").permutation(N)
    hot, cold = perm[:n_hot], perm[n_hot:]

    def endpoint(name):
        r = _rng(seed, name)
        is_hot = r.random(E) < 0.6
        h = hot[r.integers(0, n_hot, size=E)]
        c = cold[r.integers(0, len(cold), size=E)]
        return np.where(is_hot, h, c)

    src, dst = endpoint("src"), endpoint("dst")
    t = _sorted_int_seconds(_rng(seed, "t"), E, 30 * 86400)
    neg = _rng(seed, "neg").integers(0, N, size=E)
    return src, dst, t, neg, {"graph": "unipartite, 99 hot nodes take each endpoint w.p. 0.6, "
                                       "integer seconds over 30 days"}


def _events_gdelt(seed, N, E):
    # Bursty arrivals: Poisson counts with a Gamma(0.5) rate per 15-minute window.
    span = int(2.5 * 365 * 86400)
    win = 900
    n_win = span // win
    rate = _rng(seed, "rate").gamma(0.5, 1.0, size=n_win)
    p = rate / rate.sum()
    counts = _rng(seed, "counts").multinomial(E, p)
    r = _rng(seed, "t")
    base = np.repeat(np.arange(n_win, dtype=np.int64) * win, counts)
    t = np.sort(base + r.integers(0, win, size=E)).astype(np.float64)
    src = _bounded_zipf(_rng(seed, "src"), N, 1.0, E)
    dst = _bounded_zipf(_rng(seed, "dst"), N, 1.0, E)
    perm = _rng(seed, "perm").permutation(N)
    src, dst = perm[src], perm[dst]
    neg = _rng(seed, "neg").integers(0, N, size=E)
    return src, dst, t, neg, {"graph": "unipartite Zipf(1.0) endpoints, Gamma(0.5)-modulated "
                                       "Poisson arrivals per 15 min over 2.5 years"}


_BUILDERS = {"tiny": _events_tiny, "wiki": _events_wiki, "reddit": _events_reddit,
             "lastfm": _events_lastfm, "gdelt": _events_gdelt}


def edge_feature_rows(seed: int, E: int, D_e: int, lo: int, hi: int) -> np.ndarray:
    """Rows [lo, hi) of the N(0,1) fp32 edge-feature table of a stream of E events."""
    assert 0 <= lo <= hi <= E
    out = np.empty((hi - lo, D_e), dtype=np.float32)
    if D_e == 0 or hi == lo:
        return out
    c0, c1 = lo // _FEAT_CHUNK, (hi - 1) // _FEAT_CHUNK
    for c in range(c0, c1 + 1):
        base = c * _FEAT_CHUNK
        n = min(_FEAT_CHUNK, E - base)
        block = _rng(seed, "efeat", c).standard_normal((n, D_e), dtype=np.float32)
        a, b = max(lo, base), min(hi, base + n)
        out[a - lo:b - lo] = block[a - base:b - base]
    return out


def make_workload(name: str, *, E: int | None = None, s: int | None = None,
                  seed: int = 0, with_features: bool = True, **overrides) -> Workload:
    """Build one named workload.  ``E`` truncates the stream to its first E events
    (the prefix of the full stream, so windows of a large workload stay
    consistent), ``s`` overrides the staleness."""
    cfg = dict(CONFIGS[name])
    cfg.update(overrides)
    E_full = cfg.pop("E")
    N = cfg.pop("N")
    src, dst, t, neg, meta = _BUILDERS[name](seed, N, E_full)
    if E is not None:
        assert 0 < E <= E_full
        src, dst, t, neg = src[:E], dst[:E], t[:E], neg[:E]
    E_used = len(src)
    D_e = cfg["D_e"]
    efeat = None
    if D_e > 0 and with_features:
        efeat = edge_feature_rows(seed, E_full, D_e, 0, E_used)
    if s is not None:
        cfg["s"] = s
    return Workload(name=name, N=N, src=np.ascontiguousarray(src, dtype=np.int32),
                    dst=np.ascontiguousarray(dst, dtype=np.int32),
                    t=np.ascontiguousarray(t, dtype=np.float64),
                    neg=np.ascontiguousarray(neg, dtype=np.int32), efeat=efeat,
                    nb=10, seed=seed, meta=meta, **cfg)


def custom_workload(name, N, src, dst, t, neg, efeat, *, M, D_t, H, nb, B, s, seed=0):
    """Wrap a hand-built stream (used by small tests)."""
    D_e = 0 if efeat is None else int(efeat.shape[1])
    return Workload(name=name, N=N, src=np.ascontiguousarray(src, dtype=np.int32),
                    dst=np.ascontiguousarray(dst, dtype=np.int32),
                    t=np.ascontiguousarray(t, dtype=np.float64),
                    neg=np.ascontiguousarray(neg, dtype=np.int32),
                    efeat=None if efeat is None else np.ascontiguousarray(efeat, dtype=np.float32),
                    D_e=D_e, M=M, D_t=D_t, H=H, nb=nb, B=B, s=s, seed=seed)


@dataclass
class Predictor:
    """Link-predictor weights: z = W_src h_u + W_dst h_v + b_p,
    score = w_out . ReLU(z) + b_out (fp32)."""
    W_src: np.ndarray
    W_dst: np.ndarray
    b_p: np.ndarray
    w_out: np.ndarray
    b_out: float


def make_predictor(M: int, *, seed: int = 0) -> Predictor:
    """U(+-1/sqrt(fan_in)) fp32 predictor weights (fan_in 2M for the first
    layer, which sees both endpoints, M for the output)."""
    r = lambda n: _rng(seed, "p/" + n)
    return Predictor(W_src=_uniform(r("W_src"), (M, M), 2 * M),
                     W_dst=_uniform(r("W_dst"), (M, M), 2 * M),
                     b_p=_uniform(r("b_p"), (M,), 2 * M),
                     w_out=_uniform(r("w_out"), (M,), M),
                     b_out=float(_uniform(r("b_out"), (1,), M)[0]))


def _uniform(rng, shape, fan_in):
    bound = 1.0 / math.sqrt(fan_in)
    return rng.uniform(-bound, bound, size=shape).astype(np.float32)


def make_weights(M: int, D_e: int, D_t: int, *, seed: int = 0,
                 beta: str = "zero", model: str = "tgn", K_mb: int = 10,
                 propagate: bool = True) -> Weights:
    """U(+-1/sqrt(fan_in)) fp32 weights; time-encoding frequencies
    omega_d = 10^(-9 d / (D_t - 1)) and phases beta (zero, or U(0, 2pi) when
    ``beta='random'``) in fp64.  ``model='jodie'``: an RNN updater and a time
    projection w_t ~ U(+-1/sqrt(M)) scaled by 1e-5 per time unit (the
    streams' gaps reach 1e6).  ``model='apan'``: the GRU and the mailbox
    attention, K_mb mails per mailbox, mails propagated to the neighbours
    when ``propagate``."""
    D_m = 2 * M + D_e
    D_x = D_m + D_t
    d_a = M
    D_kv = M + D_e + D_t
    r = lambda n: _rng(seed, "w/" + n)
    d = np.arange(D_t, dtype=np.float64)
    omega = 10.0 ** (-9.0 * d / max(D_t - 1, 1))
    if beta == "zero":
        b = np.zeros(D_t)
    elif beta == "random":
        b = r("beta").uniform(0.0, 2.0 * math.pi, size=D_t)
    else:
        raise ValueError(beta)
    if model == "jodie":
        return Weights(
            W_ih=_uniform(r("W_ih1"), (M, D_x), D_x),
            W_hh=_uniform(r("W_hh1"), (M, M), M),
            b_ih=_uniform(r("b_ih1"), (M,), M),
            b_hh=_uniform(r("b_hh1"), (M,), M),
            omega=omega, beta=b, kind="jodie",
            w_t=(_uniform(r("w_t"), (M,), M) * np.float32(1e-5)).astype(np.float32))
    if model == "apan":
        D_mk = D_m + D_t
        return Weights(
            W_ih=_uniform(r("W_ih"), (3 * M, D_x), D_x),
            W_hh=_uniform(r("W_hh"), (3 * M, M), M),
            b_ih=_uniform(r("b_ih"), (3 * M,), M),
            b_hh=_uniform(r("b_hh"), (3 * M,), M),
            omega=omega, beta=b, kind="apan",
            W_q=_uniform(r("W_q"), (d_a, M + D_t), M + D_t),
            b_q=_uniform(r("b_q"), (d_a,), M + D_t),
            W_k=_uniform(r("W_kmb"), (d_a, D_mk), D_mk),
            b_k=_uniform(r("b_kmb"), (d_a,), D_mk),
            K_mb=K_mb, propagate=propagate)
    if model != "tgn":
        raise ValueError(model)
    return Weights(
        W_ih=_uniform(r("W_ih"), (3 * M, D_x), D_x),
        W_hh=_uniform(r("W_hh"), (3 * M, M), M),
        b_ih=_uniform(r("b_ih"), (3 * M,), M),
        b_hh=_uniform(r("b_hh"), (3 * M,), M),
        omega=omega, beta=b,
        W_q=_uniform(r("W_q"), (d_a, M + D_t), M + D_t),
        b_q=_uniform(r("b_q"), (d_a,), M + D_t),
        W_k=_uniform(r("W_k"), (d_a, D_kv), D_kv),
        b_k=_uniform(r("b_k"), (d_a,), D_kv),
        W_v=_uniform(r("W_v"), (d_a, D_kv), D_kv),
        b_v=_uniform(r("b_v"), (d_a,), D_kv),
        W_o=_uniform(r("W_o"), (M, d_a + M), d_a + M),
        b_o=_uniform(r("b_o"), (M,), d_a + M),
    )


def synthetic_mailbox(N: int, K: int, D_m: int, t_end: float, seed: int = 0):
    """A seeded APAN mailbox state (rows [N x K x D_m] and times [N x K],
    oldest mail first, zero past the count; counts [N]): 70 % of the nodes hold
    K mails, the rest 0 .. K-1; mail rows N(0, 1) rounded to fp32; each
    mailbox's times are non-decreasing whole seconds before t_end."""
    r = np.random.default_rng(seed)
    cnt = np.where(r.random(N) < 0.7, K, r.integers(0, K, N)).astype(np.int32)
    used = np.arange(K)[None, :] < cnt[:, None]
    mb = r.standard_normal((N, K, D_m)).astype(np.float32).astype(np.float64) * used[:, :, None]
    ts = np.sort(np.floor(r.uniform(0, max(t_end, 1.0), (N, K))), axis=1) * used
    return mb, ts, cnt
