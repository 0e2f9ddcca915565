"""Runs the per-batch memory-module stage through libtgm.

``Stage`` owns the library handles and every per-batch device buffer
(allocated once, through torch).  Iteration i is tgm_sample_nodes (roots,
sampling, node set), tgm_fetch_memory (state as of iteration i-1-s),
tgm_update_memory (GRU, latest-message reduce, staged write-back) and
tgm_embed.

``step(i)`` issues the four calls on one stream.  ``run(i0, n)`` hands
iterations i0 .. i0+n-1 to the library's pipelined executor
(tgm_stage_run): the sample and node set, which depend on the event stream
only, run a chunk of iterations ahead on a second stream (the prefetch of
Sec. 3.1), into sample buffer set (i - i0) % nsb.  Results are identical to
``step`` (tested).  The class holds no arithmetic of the method: all of it
runs in the library's kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import tgm

# sample and node-set buffers of one batch (``Stage.<name>`` reads the set of
# the last iteration)
_SAMPLE_BUFFERS = ("root", "root_ts", "nbr", "eid", "nts", "cnt", "nodes", "n_nodes", "root_pos",
                   "nbr_pos")
_SETS = 16   # sample buffer sets of the pipelined executor: chunks of up to 8 iterations


class _Sample:
    """Sample and node-set buffers of one batch."""

    def __init__(self, dev, R, nb, cap):
        i32, f64 = torch.int32, torch.float64
        z = lambda shape, dt: torch.zeros(shape, dtype=dt, device=dev)
        self.root, self.root_ts = z(R, i32), z(R, f64)
        self.nbr, self.eid, self.nts = z((R, nb), i32), z((R, nb), i32), z((R, nb), f64)
        self.cnt = z(R, i32)
        self.nodes, self.n_nodes = z(cap, i32), z(1, i32)
        self.root_pos, self.nbr_pos = z(R, i32), z((R, nb), i32)


class Stage:
    def __init__(self, N, src, dst, t, neg, efeat, weights, *, M, D_t, H, nb, B, s,
                 device="cuda", stream=None, mitigation=None, training=None):
        """src, dst, t, neg: numpy or torch arrays of the event stream; efeat
        [E x D_e] fp32 or None; weights a ``workloads.Weights``;
        ``mitigation=dict(p=.., lam=.., K=..)`` turns on the similarity-based
        staleness mitigation (Sec. 3.3) of every fetch;
        ``training=dict(predictor=P, opt="adam"|"sgd", lr=..)`` adds the
        training step (loss, gradient, optimizer) after every iteration."""
        dev = torch.device(device)
        self.dev = dev
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        self.pre_stream = torch.cuda.Stream(dev)   # default priority
        T = lambda a, dt: a.to(dev, dt).contiguous() if torch.is_tensor(a) else \
            torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
        self.src = T(src, torch.int32)
        self.dst = T(dst, torch.int32)
        self.t = T(t, torch.float64)
        self.neg = T(neg, torch.int32)
        self.efeat = None if efeat is None else T(efeat, torch.float32)
        self.N, self.E = int(N), int(self.src.numel())
        self.D_e = 0 if efeat is None else int(self.efeat.shape[1])
        self.M, self.D_t, self.H, self.nb, self.B, self.s = M, D_t, H, nb, B, s
        self.D_m = 2 * M + self.D_e
        self.n_iters = (self.E + B - 1) // B
        R = 3 * B
        self.cap = min(self.N, R * (nb + 1))
        st = self.stream
        self.g = tgm.tgm_graph_create(self.N, self.src, self.dst, self.t, self.neg, self.efeat,
                                      stream=st)
        self.st = tgm.tgm_state_create(self.N, M, self.D_m, s, B, stream=st)
        self.kind = getattr(weights, "kind", "tgn")   # "tgn" or "jodie"
        self.m = tgm.tgm_model_create(M, self.D_e, D_t, H, nb, self.cap, R, weights, stream=st)
        self.sets = [_Sample(dev, R, nb, self.cap) for _ in range(_SETS)]
        z = lambda shape, dt: torch.zeros(shape, dtype=dt, device=dev)
        cap = self.cap
        self.f_mem, self.f_mem_ts = z((cap, M), torch.float32), z(cap, torch.float64)
        self.f_mail, self.f_mail_ts = z((cap, self.D_m), torch.float32), z(cap, torch.float64)
        self.f_ver = z(cap, torch.int32)
        self.mem_new, self.new_mem_ts = z((self.cap, M), torch.float32), z(self.cap, torch.float64)
        self.winner = z(self.cap, torch.int64)
        self.h = z((R, M), torch.float32)
        self.want_winner = True
        self.mit = None
        self.mitigation = mitigation
        if mitigation is not None:
            self.mit = tgm.tgm_mitigator_create(self.cap, nb, int(mitigation["K"]))
            tgm.tgm_state_set_mitigation(self.st, self.mit, mitigation["p"], mitigation["lam"])
        self.tr = None
        self.training = training
        if training is not None:
            kw = {k: training[k] for k in ("opt", "lr", "beta1", "beta2", "eps") if k in training}
            self.tr = tgm.tgm_trainer_create(self.m, weights, training["predictor"], stream=st,
                                             **kw)
            self.n_params, self.param_sizes, _ = tgm.tgm_trainer_info(self.tr)
            self.loss = z(1, torch.float32)
            self.loss_log = z(self.n_iters, torch.float32)
            tgm.tgm_state_set_training(self.st, self.tr, self.loss_log)
        self.last = None      # (iteration, batch size) of the last issued iteration
        self._set = 0         # its sample buffer set
        self._bufs = None

    def __getattr__(self, name):
        if name in _SAMPLE_BUFFERS and "sets" in self.__dict__:
            return getattr(self.sets[self.__dict__.get("_set", 0)], name)
        raise AttributeError(name)

    def close(self):
        for fn, h in ((tgm.tgm_trainer_destroy, "tr"), (tgm.tgm_model_destroy, "m"),
                      (tgm.tgm_state_destroy, "st"),
                      (tgm.tgm_mitigator_destroy, "mit"), (tgm.tgm_graph_destroy, "g")):
            if self.__dict__.get(h) is not None:
                fn(self.__dict__[h])
                self.__dict__[h] = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def batch(self, i):
        lo = i * self.B
        return lo, min(self.E, lo + self.B)

    def step(self, i: int):
        """Enqueue iteration i on the main stream (no synchronisation)."""
        lo, hi = self.batch(i)
        n = hi - lo
        b, st = self.sets[0], self.stream
        tgm.tgm_sample_nodes(self.g, lo, n, self.nb, b.root, b.root_ts, b.nbr, b.eid, b.nts,
                             b.cnt, b.nodes, b.n_nodes, self.cap, b.root_pos, b.nbr_pos, stream=st)
        tgm.tgm_fetch_memory(self.st, i, b.nodes, b.n_nodes, self.cap, self.f_mem, self.f_mem_ts,
                             self.f_mail, self.f_mail_ts, self.f_ver, stream=st)
        if self.mit is not None:
            mit = self.mitigation
            tgm.tgm_mitigate(self.mit, self.g, lo, b.nodes, b.n_nodes, self.cap, self.f_mem,
                             self.f_mem_ts, self.M, mit["p"], mit["lam"], stream=st)
        tgm.tgm_update_memory(self.st, self.m, self.g, i, b.nodes, b.n_nodes, self.cap,
                              self.f_mem, self.f_mem_ts, self.f_mail, self.f_mail_ts, self.f_ver,
                              lo, n, b.root_pos[:n], b.root_pos[n:2 * n], self.mem_new,
                              self.new_mem_ts, self.winner if self.want_winner else None,
                              stream=st)
        if self.kind == "jodie":
            tgm.tgm_embed_projection(self.m, 3 * n, b.root_pos, b.root_ts, self.mem_new,
                                     self.new_mem_ts, b.n_nodes, self.cap, self.h, stream=st)
        else:
            tgm.tgm_embed(self.m, self.g, 3 * n, self.nb, b.root_pos, b.root_ts, b.nbr_pos,
                          b.eid, b.nts, b.cnt, self.mem_new, b.n_nodes, self.cap, self.h,
                          stream=st)
        if self.tr is not None and not getattr(self, "_train_off", False):
            sb, fb = self._structs()
            tgm.tgm_train_step(self.tr, self.m, self.g, n, sb[0], fb, self.mem_new, self.h,
                               self.cap, loss=self.loss_log[i:i + 1], stream=st)
        self.last, self._set = (i, n), 0

    def set_training(self, on: bool):
        """Turns the training step after every iteration on or off (a stage
        made with ``training``)."""
        assert self.tr is not None, "the stage was made without training"
        self._train_off = not on
        tgm.tgm_state_set_training(self.st, self.tr if on else None,
                                   self.loss_log if on else None)

    def _structs(self):
        if self._bufs is None:
            sb = (tgm.SampleBuffers * len(self.sets))(
                *[tgm.buffers(tgm.SampleBuffers, **vars(b)) for b in self.sets])
            fb = tgm.buffers(tgm.FetchBuffers, mem=self.f_mem, mem_ts=self.f_mem_ts,
                             mail=self.f_mail, mail_ts=self.f_mail_ts, ver=self.f_ver)
            self._bufs = (sb, fb)
        return self._bufs

    def train_state(self):
        """Host copies of the trainer's parameter vector, the gradient of the
        last step and the per-iteration losses so far (synchronises)."""
        params = torch.empty(self.n_params, dtype=torch.float32, device=self.dev)
        grad = torch.empty_like(params)
        tgm.tgm_trainer_read(self.tr, params, grad, stream=self.stream)
        torch.cuda.synchronize(self.dev)
        return dict(params=params.cpu().numpy(), grad=grad.cpu().numpy(),
                    loss=self.loss_log.cpu().numpy())

    def run(self, i0: int, n: int, trace: bool = False):
        """Enqueue iterations i0 .. i0+n-1 through the library's pipelined
        executor (tgm_stage_run).  Ordered after everything issued before on
        the main stream; the main stream ends after the last iteration.  With
        trace=True returns device tensors (h [n x 3B x M], s_new [n x cap x M])
        holding every iteration's embeddings and new memories."""
        if n <= 0:
            return None
        sb, fb = self._structs()
        h_tr = s_tr = None
        if trace:
            h_tr = torch.zeros((n, 3 * self.B, self.M), dtype=torch.float32, device=self.dev)
            s_tr = torch.zeros((n, self.cap, self.M), dtype=torch.float32, device=self.dev)
        tgm.tgm_stage_run(self.g, self.st, self.m, i0, n, self.B, self.nb, self.cap, sb, fb,
                          self.mem_new, self.new_mem_ts,
                          self.winner if self.want_winner else None, self.h, self.stream,
                          self.pre_stream, h_trace=h_tr, s_trace=s_tr)
        last = i0 + n - 1
        lo, hi = self.batch(last)
        self.last, self._set = (last, hi - lo), (n - 1) % len(self.sets)
        return (h_tr, s_tr) if trace else None

    # ------------------------------------------------------------ read-back
    def outputs(self):
        """Host copies of the last iteration's outputs (synchronises)."""
        torch.cuda.synchronize(self.dev)
        i, b = self.last
        s = self.sets[self._set]
        R = 3 * b
        n = int(s.n_nodes.item())
        c = lambda x: x.cpu().numpy()
        return dict(iter=i, b=b, R=R, n_U=n, root=c(s.root[:R]), root_ts=c(s.root_ts[:R]),
                    nbr=c(s.nbr[:R]), eid=c(s.eid[:R]), nts=c(s.nts[:R]),
                    cnt=c(s.cnt[:R]), U=c(s.nodes[:n]), root_pos=c(s.root_pos[:R]),
                    nbr_pos=c(s.nbr_pos[:R]), f_mem=c(self.f_mem[:n]),
                    f_mem_ts=c(self.f_mem_ts[:n]), f_mail=c(self.f_mail[:n]),
                    f_mail_ts=c(self.f_mail_ts[:n]), f_ver=c(self.f_ver[:n]),
                    s_new=c(self.mem_new[:n]), new_mem_ts=c(self.new_mem_ts[:n]),
                    winner=c(self.winner[:n]), h=c(self.h[:R]))

    def mitigation_result(self):
        """Host copies of the last mitigation: gamma, stale positions, Omega
        positions [n_stale x K] (synchronises)."""
        K = int(self.mitigation["K"])
        dev = self.dev
        gamma = torch.zeros(1, dtype=torch.float64, device=dev)
        ns = torch.zeros(1, dtype=torch.int32, device=dev)
        stale = torch.zeros(self.cap, dtype=torch.int32, device=dev)
        omega = torch.zeros(self.cap * K, dtype=torch.int32, device=dev)
        tgm.tgm_mitigator_read(self.mit, gamma, ns, stale, omega, stream=self.stream)
        torch.cuda.synchronize(dev)
        n = int(ns.item())
        return (float(gamma.item()), stale[:n].cpu().numpy(),
                omega[:n * K].view(n, K).cpu().numpy())

    def flush(self):
        tgm.tgm_state_flush(self.st, stream=self.stream)

    def state(self):
        N, M, D_m, dev = self.N, self.M, self.D_m, self.dev
        mem = torch.empty((N, M), dtype=torch.float32, device=dev)
        mail = torch.empty((N, D_m), dtype=torch.float32, device=dev)
        mem_ts = torch.empty(N, dtype=torch.float64, device=dev)
        mail_ts = torch.empty(N, dtype=torch.float64, device=dev)
        ver = torch.empty(N, dtype=torch.int32, device=dev)
        tgm.tgm_state_read(self.st, mem, mem_ts, mail, mail_ts, ver, stream=self.stream)
        torch.cuda.synchronize(dev)
        return dict(mem=mem.cpu().numpy(), mem_ts=mem_ts.cpu().numpy(), mail=mail.cpu().numpy(),
                    mail_ts=mail_ts.cpu().numpy(), ver=ver.cpu().numpy())

    def reset(self):
        """The initial state again; the next iteration is 0."""
        tgm.tgm_state_reset(self.st, stream=self.stream)

    def load_state(self, it, mem, mem_ts, mail, mail_ts, ver):
        dev = self.dev
        T = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
        self._loaded = [T(mem, torch.float32), T(mem_ts, torch.float64),
                        T(mail, torch.float32), T(mail_ts, torch.float64), T(ver, torch.int32)]
        tgm.tgm_state_load(self.st, it, *self._loaded, stream=self.stream)
        torch.cuda.synchronize(dev)


    def save_checkpoint(self):
        """The versioned state's checkpoint (host uint8 array: committed
        tables, staged write sets, protocol counters) after the work issued
        so far on the stage's stream."""
        return tgm.tgm_state_save(self.st, stream=self.stream)

    def restore_checkpoint(self, buf):
        """Continue from a checkpoint of a stage with the same N, M, D_m, s
        and batch size: the next step or run takes the iteration after the
        checkpoint's last update."""
        tgm.tgm_state_restore(self.st, buf, stream=self.stream)


class ApanStage:
    """The APAN family through libtgm: tgm_sample_nodes, then tgm_apan_step
    (fetch with the mailboxes, mailbox attention and GRU, identity
    embedding, staged write set with the propagated mails) per iteration."""

    def __init__(self, wl, w, *, s=None, device="cuda", stream=None, efeat=None):
        """``efeat``: a device edge-feature table to use instead of the
        workload's host one."""
        dev = torch.device(device)
        self.dev, self.wl = dev, wl
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        T = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
        self.src, self.dst = T(wl.src, torch.int32), T(wl.dst, torch.int32)
        self.t, self.neg = T(wl.t, torch.float64), T(wl.neg, torch.int32)
        if efeat is not None:
            self.efeat = efeat
        else:
            self.efeat = None if wl.efeat is None else T(wl.efeat, torch.float32)
        self.N, self.M, self.nb, self.B = wl.N, wl.M, wl.nb, wl.B
        self.s = wl.s if s is None else s
        self.K = int(w.K_mb)
        self.D_m = 2 * wl.M + wl.D_e
        R = 3 * wl.B
        self.cap = min(self.N, R * (self.nb + 1))
        st = self.stream
        self.g = tgm.tgm_graph_create(self.N, self.src, self.dst, self.t, self.neg, self.efeat,
                                      stream=st)
        self.a = tgm.tgm_apan_create(self.N, wl.M, wl.D_e, wl.D_t, self.nb, self.K, w.propagate,
                                     self.s, wl.B, self.cap, w, stream=st)
        self.sb = _Sample(dev, R, self.nb, self.cap)
        self._sbs = tgm.buffers(tgm.SampleBuffers, **vars(self.sb))
        z = lambda shape, dt: torch.zeros(shape, dtype=dt, device=dev)
        self.mem_new, self.new_mem_ts = z((self.cap, wl.M), torch.float32), z(self.cap,
                                                                              torch.float64)
        self.h = z((R, wl.M), torch.float32)
        self.last = None

    def step(self, i: int):
        lo = i * self.B
        n = min(self.B, self.wl.E - lo)
        b = self.sb
        tgm.tgm_sample_nodes(self.g, lo, n, self.nb, b.root, b.root_ts, b.nbr, b.eid, b.nts,
                             b.cnt, b.nodes, b.n_nodes, self.cap, b.root_pos, b.nbr_pos,
                             stream=self.stream)
        tgm.tgm_apan_step(self.a, self.g, i, self._sbs, self.cap, self.mem_new, self.new_mem_ts,
                          self.h, stream=self.stream)
        self.last = (i, n)

    def run(self, i0: int, n: int):
        """Iterations i0 .. i0 + n - 1, one after another on the stream."""
        for i in range(i0, i0 + n):
            self.step(i)

    def reset(self):
        tgm.tgm_apan_reset(self.a, stream=self.stream)

    def load_state(self, it, mem, mem_ts, ver, mb, mb_ts, mb_cnt):
        """Committed tables at iteration ``it`` (host arrays or device
        tensors, the layouts of ``state()``); the next step is ``it``."""
        dev = self.dev

        def T(a, dt):
            if isinstance(a, torch.Tensor):
                return a.to(dev, dt).contiguous()
            return torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
        keep = (T(mem, torch.float32), T(mem_ts, torch.float64), T(ver, torch.int32),
                T(mb, torch.float32), T(mb_ts, torch.float64), T(mb_cnt, torch.int32))
        tgm.tgm_apan_load(self.a, it, *keep, stream=self.stream)
        self.stream.synchronize()

    def outputs(self):
        """Host copies of the last iteration's node set, fetched rows and
        mailboxes (oldest first), new memories and embeddings (synchronises)."""
        i, n = self.last
        dev, C, M, K, D_m = self.dev, self.cap, self.M, self.K, self.D_m
        e = lambda shape, dt: torch.empty(shape, dtype=dt, device=dev)
        f_mem, f_ts, f_ver = e((C, M), torch.float32), e(C, torch.float64), e(C, torch.int32)
        f_mb, f_mbt, f_cnt = e((C, K, D_m), torch.float32), e((C, K), torch.float64), \
            e(C, torch.int32)
        tgm.tgm_apan_fetched(self.a, f_mem, f_ts, f_ver, f_mb, f_mbt, f_cnt, stream=self.stream)
        torch.cuda.synchronize(dev)
        nU = int(self.sb.n_nodes.item())
        R = 3 * n
        c = lambda x: x.cpu().numpy()
        return dict(iter=i, b=n, n_U=nU, U=c(self.sb.nodes[:nU]), root_pos=c(self.sb.root_pos[:R]),
                    f_mem=c(f_mem[:nU]), f_mem_ts=c(f_ts[:nU]), f_ver=c(f_ver[:nU]),
                    f_mb=c(f_mb[:nU]), f_mb_ts=c(f_mbt[:nU]), f_mb_cnt=c(f_cnt[:nU]),
                    s_new=c(self.mem_new[:nU]), new_mem_ts=c(self.new_mem_ts[:nU]),
                    h=c(self.h[:R]))

    def flush(self):
        tgm.tgm_apan_flush(self.a, stream=self.stream)

    def counts(self):
        """Sizes of the last iteration (synchronises): events, roots, valid
        sampled slots, node-set size, nodes with mail, fetched mails."""
        i, n = self.last
        torch.cuda.synchronize(self.dev)
        nU = int(self.sb.n_nodes.item())
        R = 3 * n
        cnt = torch.empty(self.cap, dtype=torch.int32, device=self.dev)
        tgm.tgm_apan_fetched(self.a, mb_cnt=cnt, stream=self.stream)
        c = cnt[:nU]
        return dict(b=n, R=R, slots=int(self.sb.cnt[:R].sum().item()), n_U=nU,
                    n_mail=int((c > 0).sum().item()), n_mails=int(c.sum().item()))

    def device_state(self):
        """The committed tables as device tensors (mem, mem_ts, ver, mb, mb_ts,
        mb_cnt: the arguments of ``load_state``); ordered on the stream."""
        dev, N, M, K, D_m = self.dev, self.N, self.M, self.K, self.D_m
        e = lambda shape, dt: torch.empty(shape, dtype=dt, device=dev)
        mem, mem_ts, ver = e((N, M), torch.float32), e(N, torch.float64), e(N, torch.int32)
        mb, mb_ts, cnt = e((N, K, D_m), torch.float32), e((N, K), torch.float64), \
            e(N, torch.int32)
        tgm.tgm_apan_read(self.a, mem, mem_ts, ver, mb, mb_ts, cnt, stream=self.stream)
        return mem, mem_ts, ver, mb, mb_ts, cnt

    def state(self):
        mem, mem_ts, ver, mb, mb_ts, cnt = self.device_state()
        torch.cuda.synchronize(self.dev)
        c = lambda x: x.cpu().numpy()
        return dict(mem=c(mem), mem_ts=c(mem_ts), ver=c(ver), mb=c(mb), mb_ts=c(mb_ts),
                    mb_cnt=c(cnt))

    def close(self):
        if self.__dict__.get("a") is not None:
            tgm.tgm_apan_destroy(self.a)
            self.a = None
        if self.__dict__.get("g") is not None:
            tgm.tgm_graph_destroy(self.g)
            self.g = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def from_workload(wl, w, *, s=None, device="cuda", stream=None, mitigation=None,
                  training=None) -> Stage:
    return Stage(wl.N, wl.src, wl.dst, wl.t, wl.neg, wl.efeat, w, M=wl.M, D_t=wl.D_t, H=wl.H,
                 nb=wl.nb, B=wl.B, s=wl.s if s is None else s, device=device, stream=stream,
                 mitigation=mitigation, training=training)


# ------------------------------------------------------- staleness bound
# The paper's five stages (Sec. 3.2) as this library's kernels on the
# sequential path (one call per stage).  Edge features are read inside the
# attention kernel, so the feature fetch has no kernel of its own; the
# mitigation belongs to the memory fetch (Sec. 3.3).
STAGE_KERNELS = {1: ("k_sample_batch", "k_ns_mark", "k_ns_pos"), 2: (),
                 3: ("k_gather_state", "k_mit_prep", "k_mit_select", "k_mit_omega",
                     "k_mit_final"),
                 4: ("k_phi", "k_gru", "k_gru_w", "k_node_proj", "k_attn_agg", "k_attn_fold",
                     "k_attn", "k_tproj"),
                 5: ("k_stage", "k_commit")}


def stage_durations_us(profile: dict, iters: int) -> list:
    """Per-iteration durations (µs) of the five stages from a per-kernel
    profile ({kernel: (launches, total ms)}, template instances folded into
    their kernel) taken over `iters` sequential steps."""
    folded = {}
    for name, (launches, ms) in profile.items():
        base = name.split("<")[0].lstrip("(")
        n0, m0 = folded.get(base, (0, 0.0))
        folded[base] = (n0 + launches, m0 + ms)
    return [sum(folded.get(k, (0, 0.0))[1] for k in STAGE_KERNELS[j]) * 1e3 / iters
            for j in range(1, 6)]


def minimal_staleness(tau_us, k_max: int = 16, n: int = 64) -> dict:
    """The minimal staleness of Sec. 3.2 (Eq. 3-4, C1-C3) for the stage
    durations tau_us, by the library's host solver, in steady state (the last
    of n iterations).  The paper's k corresponds to s = k - 1 here: a fetch at
    iteration i reads the write sets of iterations up to i - 1 - s."""
    k, _, stall, _, _ = tgm.tgm_min_staleness(list(tau_us), n, k_max)
    return {"tau_us": dict(zip(("sample", "feature_fetch", "memory_fetch", "compute",
                                "memory_update"), (float(t) for t in tau_us))),
            "k_min": int(k[-1]), "s_equivalent": int(k[-1]) - 1,
            "stall_free": bool(stall[-1] == 0.0), "k_max": k_max}



def calibrate_staleness(stage: Stage, first: int = 0, *, warm: int = 3, iters: int = 12,
                        k_max: int = 16) -> dict:
    """The online half of the bound (Sec. 3.2; App. D.1 profiles a few
    iterations before training): `warm` untimed sequential steps of `stage`
    from batch `first` on, then `iters` profiled ones, their kernel durations
    mapped to the five stages, and the steady-state minimal staleness solved
    from them.  Adds "s", the staleness this library's state takes for it
    (k_min - 1).  The steps advance the stage's state, so the run that uses
    the result is built afresh with that s: calibrate on a stage of its own."""
    for i in range(first, first + warm):
        stage.step(i)
    torch.cuda.synchronize()
    tgm.tgm_profile_reset()
    tgm.tgm_profile_enable(True)
    try:
        for i in range(first + warm, first + warm + iters):
            stage.step(i)
        torch.cuda.synchronize()
    finally:
        tgm.tgm_profile_enable(False)
    res = minimal_staleness(stage_durations_us(tgm.tgm_profile_read(), iters), k_max=k_max)
    res["s"] = max(res["k_min"] - 1, 0)
    res["calibration"] = {"first": first, "warm": warm, "iters": iters}
    return res
