"""Runs the per-batch memory-module stage through libtgm.

``Stage`` owns the library handles and every per-batch device buffer
(allocated once, through torch), and issues, for iteration i, the calls
tgm_sample_nodes (roots + sampling + node set) -> tgm_fetch_memory ->
tgm_update_memory -> tgm_embed on one stream.  It holds no arithmetic of the
method: all of it runs in the library's kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import tgm


class Stage:
    def __init__(self, N, src, dst, t, neg, efeat, weights, *, M, D_t, H, nb, B, s,
                 device="cuda", stream=None):
        """src, dst, t, neg: numpy or torch arrays of the event stream; efeat
        [E x D_e] fp32 or None; weights a ``workloads.Weights``."""
        dev = torch.device(device)
        self.dev = dev
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
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
        self.m = tgm.tgm_model_create(M, self.D_e, D_t, H, nb, self.cap, R, weights, stream=st)
        i32, f64, f32 = torch.int32, torch.float64, torch.float32
        z = lambda shape, dt: torch.zeros(shape, dtype=dt, device=dev)
        cap = self.cap
        self.root, self.root_ts = z(R, i32), z(R, f64)
        self.nbr, self.eid, self.nts = z((R, nb), i32), z((R, nb), i32), z((R, nb), f64)
        self.cnt = z(R, i32)
        self.nodes, self.n_nodes = z(cap, i32), z(1, i32)
        self.root_pos, self.nbr_pos = z(R, i32), z((R, nb), i32)
        self.f_mem, self.f_mem_ts = z((cap, M), f32), z(cap, f64)
        self.f_mail, self.f_mail_ts = z((cap, self.D_m), f32), z(cap, f64)
        self.f_ver = z(cap, i32)
        self.mem_new, self.new_mem_ts = z((cap, M), f32), z(cap, f64)
        self.winner = z(cap, torch.int64)
        self.h = z((R, M), f32)
        self.want_winner = True
        self.last = None

    def close(self):
        for fn, h in ((tgm.tgm_model_destroy, "m"), (tgm.tgm_state_destroy, "st"),
                      (tgm.tgm_graph_destroy, "g")):
            if getattr(self, h, None) is not None:
                fn(getattr(self, h))
                setattr(self, h, None)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def batch(self, i):
        lo = i * self.B
        return lo, min(self.E, lo + self.B)

    def step(self, i: int):
        """Enqueue iteration i (no synchronisation)."""
        lo, hi = self.batch(i)
        b = hi - lo
        R = 3 * b
        nb, cap, st = self.nb, self.cap, self.stream
        tgm.tgm_sample_nodes(self.g, lo, b, nb, self.root, self.root_ts, self.nbr, self.eid,
                             self.nts, self.cnt, self.nodes, self.n_nodes, cap, self.root_pos,
                             self.nbr_pos, stream=st)
        tgm.tgm_fetch_memory(self.st, i, self.nodes, self.n_nodes, cap, self.f_mem,
                             self.f_mem_ts, self.f_mail, self.f_mail_ts, self.f_ver, stream=st)
        tgm.tgm_update_memory(self.st, self.m, self.g, i, self.nodes, self.n_nodes, cap,
                              self.f_mem, self.f_mem_ts, self.f_mail, self.f_mail_ts, self.f_ver,
                              lo, b, self.root_pos[:b], self.root_pos[b:2 * b], self.mem_new,
                              self.new_mem_ts, self.winner if self.want_winner else None,
                              stream=st)
        tgm.tgm_embed(self.m, self.g, R, nb, self.root_pos, self.root_ts, self.nbr_pos,
                      self.eid, self.nts, self.cnt, self.mem_new, self.n_nodes, cap, self.h,
                      stream=st)
        self.last = (i, b)

    def outputs(self):
        """Host copies of the last iteration's outputs (synchronises)."""
        torch.cuda.synchronize(self.dev)
        i, b = self.last
        R, nb = 3 * b, self.nb
        n = int(self.n_nodes.item())
        c = lambda x: x.cpu().numpy()
        return dict(iter=i, b=b, R=R, n_U=n, root=c(self.root[:R]), root_ts=c(self.root_ts[:R]),
                    nbr=c(self.nbr[:R]), eid=c(self.eid[:R]), nts=c(self.nts[:R]),
                    cnt=c(self.cnt[:R]), U=c(self.nodes[:n]), root_pos=c(self.root_pos[:R]),
                    nbr_pos=c(self.nbr_pos[:R]), f_mem=c(self.f_mem[:n]),
                    f_mem_ts=c(self.f_mem_ts[:n]), f_mail=c(self.f_mail[:n]),
                    f_mail_ts=c(self.f_mail_ts[:n]), f_ver=c(self.f_ver[:n]),
                    s_new=c(self.mem_new[:n]), new_mem_ts=c(self.new_mem_ts[:n]),
                    winner=c(self.winner[:n]), h=c(self.h[:R]))

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

    def load_state(self, it, mem, mem_ts, mail, mail_ts, ver):
        dev = self.dev
        T = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
        self._loaded = [T(mem, torch.float32), T(mem_ts, torch.float64),
                        T(mail, torch.float32), T(mail_ts, torch.float64), T(ver, torch.int32)]
        tgm.tgm_state_load(self.st, it, *self._loaded, stream=self.stream)
        torch.cuda.synchronize(dev)


def from_workload(wl, w, *, s=None, device="cuda", stream=None) -> Stage:
    return Stage(wl.N, wl.src, wl.dst, wl.t, wl.neg, wl.efeat, w, M=wl.M, D_t=wl.D_t, H=wl.H,
                 nb=wl.nb, B=wl.B, s=wl.s if s is None else s, device=device, stream=stream)
