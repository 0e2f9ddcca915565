"""ctypes binding of libtgm (include/tgm.h), function for function.

Argument marshalling only: device arrays are torch tensors on the GPU (passed
by data pointer), streams are torch streams.  Every computation happens in
the library's HIP kernels.  A missing library is an error, never a fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtgm.so")

TGM_OK, TGM_EINVAL, TGM_ERANGE, TGM_EORDER, TGM_ESIZE, TGM_EDEVICE, TGM_ENOMEM = \
    0, -1, -2, -3, -4, -5, -6
MAX_SAMPLE_SETS = 16                     # TGM_MAX_SAMPLE_SETS
MITIGATE_NOALLOC_MAX_NODES = 32768       # TGM_MITIGATE_NOALLOC_MAX_NODES

# Every exported symbol of include/tgm.h
SYMBOLS = ["tgm_status_str", "tgm_last_device_error", "tgm_version", "tgm_alloc_count",
           "tgm_graph_create",
           "tgm_graph_destroy", "tgm_graph_info", "tgm_batch_roots", "tgm_sample", "tgm_sample_batch",
           "tgm_node_set", "tgm_sample_nodes", "tgm_state_create", "tgm_state_destroy", "tgm_state_reset",
           "tgm_state_flush", "tgm_state_read", "tgm_state_load", "tgm_state_checkpoint_bytes",
           "tgm_state_save", "tgm_state_restore", "tgm_fetch_memory",
           "tgm_model_create", "tgm_model_destroy", "tgm_update_memory", "tgm_embed",
           "tgm_stage_run", "tgm_mitigator_create", "tgm_mitigator_destroy", "tgm_mitigate",
           "tgm_mitigator_read", "tgm_state_set_mitigation", "tgm_min_staleness",
           "tgm_mitigate_noalloc", "tgm_trainer_create", "tgm_trainer_destroy",
           "tgm_trainer_info", "tgm_trainer_read", "tgm_train_step", "tgm_state_set_training",
           "tgm_apan_create", "tgm_apan_destroy", "tgm_apan_step", "tgm_apan_flush",
           "tgm_apan_reset", "tgm_apan_load",
           "tgm_apan_read", "tgm_apan_fetched",
           "tgm_embed_projection",
           "tgm_profile_enable", "tgm_profile_reset", "tgm_profile_count", "tgm_profile_get"]


class TgmError(RuntimeError):
    def __init__(self, fn, code):
        self.code = code
        super().__init__(f"{fn}: {status_str(code)} ({code})")


class SampleBuffers(C.Structure):
    _fields_ = [(name, C.c_void_p) for name in (
        "root", "root_ts", "nbr", "eid", "nts", "cnt", "nodes", "n_nodes", "root_pos", "nbr_pos")]


class FetchBuffers(C.Structure):
    _fields_ = [(name, C.c_void_p) for name in ("mem", "mem_ts", "mail", "mail_ts", "ver")]


class ModelDesc(C.Structure):
    _fields_ = [("M", C.c_int32), ("D_e", C.c_int32), ("D_t", C.c_int32), ("H", C.c_int32),
                ("nb", C.c_int32), ("max_nodes", C.c_int32), ("max_roots", C.c_int32),
                ("kind", C.c_int32)]


TGM_MODEL_TGN, TGM_MODEL_JODIE = 0, 1
MODEL_KINDS = {"tgn": TGM_MODEL_TGN, "jodie": TGM_MODEL_JODIE}


_fp = C.POINTER(C.c_float)
_dp = C.POINTER(C.c_double)


class Weights(C.Structure):
    _fields_ = [("W_ih", _fp), ("W_hh", _fp), ("b_ih", _fp), ("b_hh", _fp),
                ("omega", _dp), ("beta", _dp),
                ("W_q", _fp), ("b_q", _fp), ("W_k", _fp), ("b_k", _fp), ("W_v", _fp),
                ("b_v", _fp), ("W_o", _fp), ("b_o", _fp), ("w_t", _fp)]


class ApanDesc(C.Structure):
    _fields_ = [("N", C.c_int32), ("M", C.c_int32), ("D_e", C.c_int32), ("D_t", C.c_int32),
                ("nb", C.c_int32), ("K_mb", C.c_int32), ("propagate", C.c_int32),
                ("s", C.c_int32), ("max_batch", C.c_int32), ("max_nodes", C.c_int32)]


class Predictor(C.Structure):
    _fields_ = [("W_src", _fp), ("W_dst", _fp), ("b_p", _fp), ("w_out", _fp),
                ("b_out", C.c_float)]


class Optimizer(C.Structure):
    _fields_ = [("kind", C.c_int32), ("lr", C.c_float), ("beta1", C.c_float),
                ("beta2", C.c_float), ("eps", C.c_float)]


TGM_OPT_SGD, TGM_OPT_ADAM = 0, 1
OPTIMIZERS = {"sgd": TGM_OPT_SGD, "adam": TGM_OPT_ADAM}
N_PARAM_TENSORS = 17   # TGM_N_PARAM_TENSORS

_lib = None
V, I32, I64, P = C.c_void_p, C.c_int32, C.c_int64, C.c_void_p


def lib():
    """Load libtgm.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = C.CDLL(LIB_PATH)
        L.tgm_status_str.argtypes = [I32]
        L.tgm_status_str.restype = C.c_char_p
        L.tgm_last_device_error.restype = I32
        L.tgm_version.restype = I32
        sig = {
            "tgm_graph_create": [I32, I64, P, P, P, P, P, I32, V, C.POINTER(V)],
            "tgm_graph_destroy": [V],
            "tgm_graph_info": [V, P, P, P, P],
            "tgm_batch_roots": [V, I64, I32, P, P, V],
            "tgm_sample": [V, P, P, I32, I32, P, P, P, P, V],
            "tgm_sample_batch": [V, I64, I32, I32, P, P, P, P, P, P, V],
            "tgm_node_set": [V, P, I32, P, I32, P, P, I32, P, P, V],
            "tgm_sample_nodes": [V, I64, I32, I32, P, P, P, P, P, P, P, P, I32, P, P, V],
            "tgm_state_create": [I32, I32, I32, I32, I32, V, C.POINTER(V)],
            "tgm_state_destroy": [V],
            "tgm_state_reset": [V, V],
            "tgm_state_flush": [V, V],
            "tgm_state_read": [V, P, P, P, P, P, V],
            "tgm_state_load": [V, I64, P, P, P, P, P, V],
            "tgm_state_checkpoint_bytes": [V, C.POINTER(C.c_size_t)],
            "tgm_state_save": [V, P, C.c_size_t, V],
            "tgm_state_restore": [V, P, C.c_size_t, V],
            "tgm_fetch_memory": [V, I64, P, P, I32, P, P, P, P, P, V],
            "tgm_model_create": [C.POINTER(ModelDesc), C.POINTER(Weights), V, C.POINTER(V)],
            "tgm_model_destroy": [V],
            "tgm_update_memory": [V, V, V, I64, P, P, I32, P, P, P, P, P, I64, I32, P, P, P, P, P,
                                  V],
            "tgm_embed": [V, V, I32, I32, P, P, P, P, P, P, P, P, I32, P, V],
            "tgm_stage_run": [V, V, V, I64, I64, I32, I32, I32, C.POINTER(SampleBuffers), I32,
                              C.POINTER(FetchBuffers), P, P, P, P, P, P, V, V],
            "tgm_alloc_count": [C.POINTER(I64)],
            "tgm_trainer_create": [V, C.POINTER(Weights), C.POINTER(Predictor),
                                   C.POINTER(Optimizer), V, C.POINTER(V)],
            "tgm_trainer_destroy": [V],
            "tgm_trainer_info": [V, C.POINTER(I64), C.POINTER(I64), C.POINTER(I64)],
            "tgm_trainer_read": [V, P, P, P, V],
            "tgm_train_step": [V, V, V, I32, C.POINTER(SampleBuffers), C.POINTER(FetchBuffers),
                               P, P, I32, P, V],
            "tgm_state_set_training": [V, V, P, I64],
            "tgm_apan_create": [C.POINTER(ApanDesc), C.POINTER(Weights), V, C.POINTER(V)],
            "tgm_apan_destroy": [V],
            "tgm_apan_step": [V, V, I64, C.POINTER(SampleBuffers), I32, P, P, P, V],
            "tgm_apan_flush": [V, V],
            "tgm_apan_reset": [V, V],
            "tgm_apan_load": [V, I64, P, P, P, P, P, P, V],
            "tgm_apan_read": [V, P, P, P, P, P, P, V],
            "tgm_apan_fetched": [V, P, P, P, P, P, P, V],
            "tgm_mitigator_create": [I32, I32, I32, C.POINTER(V)],
            "tgm_mitigator_destroy": [V],
            "tgm_mitigate": [V, V, I64, P, P, I32, P, P, I32, C.c_double, C.c_float, V],
            "tgm_mitigate_noalloc": [V, I64, P, P, I32, P, P, I32, I32, I32, C.c_double,
                                     C.c_float, V],
            "tgm_mitigator_read": [V, P, P, P, P, V],
            "tgm_state_set_mitigation": [V, V, C.c_double, C.c_float],
            "tgm_min_staleness": [P, I64, I32, P, P, P, P, P],
            "tgm_embed_projection": [V, I32, P, P, P, P, P, I32, P, V],
        }
        sig["tgm_profile_enable"] = [I32]
        sig["tgm_profile_reset"] = []
        sig["tgm_profile_count"] = []
        sig["tgm_profile_get"] = [I32, C.POINTER(C.c_char_p), C.POINTER(I64),
                                  C.POINTER(C.c_double)]
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = I32
        _lib = L
    return _lib


def status_str(code: int) -> str:
    return lib().tgm_status_str(int(code)).decode()


def _check(fn, rc):
    if rc != TGM_OK:
        raise TgmError(fn, rc)


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    return C.c_void_p(t.data_ptr())


def _s(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def last_device_error() -> int:
    return lib().tgm_last_device_error()


def version() -> int:
    return lib().tgm_version()


def tgm_profile_enable(on: bool):
    _check("tgm_profile_enable", lib().tgm_profile_enable(1 if on else 0))


def tgm_profile_reset():
    _check("tgm_profile_reset", lib().tgm_profile_reset())


def tgm_profile_read() -> dict:
    """{kernel name: (launches, total ms)}; synchronises the recorded events."""
    L = lib()
    out = {}
    for k in range(L.tgm_profile_count()):
        name, n, ms = C.c_char_p(), C.c_int64(), C.c_double()
        _check("tgm_profile_get", L.tgm_profile_get(k, C.byref(name), C.byref(n), C.byref(ms)))
        out[name.value.decode()] = (n.value, ms.value)
    return out


# ------------------------------------------------------------------ graph
def tgm_graph_create(N, src, dst, t, neg, efeat, stream=None):
    E = int(src.numel())
    D_e = 0 if efeat is None else int(efeat.shape[1])
    h = V()
    _check("tgm_graph_create", lib().tgm_graph_create(N, E, _p(src), _p(dst), _p(t), _p(neg),
                                                      _p(efeat), D_e, _s(stream), C.byref(h)))
    return h


def tgm_graph_destroy(g):
    _check("tgm_graph_destroy", lib().tgm_graph_destroy(g))


def tgm_graph_info(g):
    N, E, D_e, n_adj = C.c_int32(), C.c_int64(), C.c_int32(), C.c_int64()
    _check("tgm_graph_info", lib().tgm_graph_info(g, C.byref(N), C.byref(E), C.byref(D_e),
                                                  C.byref(n_adj)))
    return N.value, E.value, D_e.value, n_adj.value


def tgm_batch_roots(g, first_event, b, root, root_ts, stream=None):
    _check("tgm_batch_roots", lib().tgm_batch_roots(g, first_event, b, _p(root), _p(root_ts),
                                                    _s(stream)))


def tgm_sample(g, root, root_ts, R, nb, nbr, eid, nts, cnt, stream=None):
    _check("tgm_sample", lib().tgm_sample(g, _p(root), _p(root_ts), R, nb, _p(nbr), _p(eid),
                                          _p(nts), _p(cnt), _s(stream)))


def tgm_sample_batch(g, first_event, b, nb, root, root_ts, nbr, eid, nts, cnt, stream=None):
    _check("tgm_sample_batch", lib().tgm_sample_batch(g, first_event, b, nb, _p(root),
                                                      _p(root_ts), _p(nbr), _p(eid), _p(nts),
                                                      _p(cnt), _s(stream)))


def tgm_node_set(g, root, R, nbr, nb, nodes, n_nodes, cap, root_pos, nbr_pos, stream=None):
    _check("tgm_node_set", lib().tgm_node_set(g, _p(root), R, _p(nbr), nb, _p(nodes),
                                              _p(n_nodes), cap, _p(root_pos), _p(nbr_pos),
                                              _s(stream)))


def tgm_sample_nodes(g, first_event, b, nb, root, root_ts, nbr, eid, nts, cnt, nodes, n_nodes, cap,
                     root_pos, nbr_pos, stream=None):
    _check("tgm_sample_nodes", lib().tgm_sample_nodes(
        g, first_event, b, nb, _p(root), _p(root_ts), _p(nbr), _p(eid), _p(nts), _p(cnt),
        _p(nodes), _p(n_nodes), cap, _p(root_pos), _p(nbr_pos), _s(stream)))


# ------------------------------------------------------------------ state
def tgm_state_create(N, M, D_m, s, max_batch, stream=None):
    h = V()
    _check("tgm_state_create", lib().tgm_state_create(N, M, D_m, s, max_batch, _s(stream),
                                                      C.byref(h)))
    return h


def tgm_state_destroy(st):
    _check("tgm_state_destroy", lib().tgm_state_destroy(st))


def tgm_state_reset(st, stream=None):
    _check("tgm_state_reset", lib().tgm_state_reset(st, _s(stream)))


def tgm_state_flush(st, stream=None):
    _check("tgm_state_flush", lib().tgm_state_flush(st, _s(stream)))


def tgm_state_read(st, mem, mem_ts, mail, mail_ts, ver, stream=None):
    _check("tgm_state_read", lib().tgm_state_read(st, _p(mem), _p(mem_ts), _p(mail),
                                                  _p(mail_ts), _p(ver), _s(stream)))


def tgm_state_load(st, it, mem, mem_ts, mail, mail_ts, ver, stream=None):
    _check("tgm_state_load", lib().tgm_state_load(st, it, _p(mem), _p(mem_ts), _p(mail),
                                                  _p(mail_ts), _p(ver), _s(stream)))


def tgm_state_checkpoint_bytes(st) -> int:
    n = C.c_size_t(0)
    _check("tgm_state_checkpoint_bytes", lib().tgm_state_checkpoint_bytes(st, C.byref(n)))
    return n.value


def tgm_state_save(st, stream=None, nbytes=None):
    """The state's checkpoint as a host uint8 array (after the work already on
    `stream`; returns once it is copied)."""
    import numpy as np
    n = tgm_state_checkpoint_bytes(st) if nbytes is None else nbytes
    buf = np.zeros(n, dtype=np.uint8)
    _check("tgm_state_save", lib().tgm_state_save(st, buf.ctypes.data, n, _s(stream)))
    return buf


def tgm_state_restore(st, buf, stream=None):
    """Load a checkpoint (a contiguous host uint8 array) into st."""
    import numpy as np
    buf = np.ascontiguousarray(buf, dtype=np.uint8)
    _check("tgm_state_restore", lib().tgm_state_restore(st, buf.ctypes.data, buf.nbytes,
                                                        _s(stream)))


def tgm_fetch_memory(st, it, nodes, n_nodes, cap, mem, mem_ts, mail, mail_ts, ver, stream=None):
    _check("tgm_fetch_memory", lib().tgm_fetch_memory(st, it, _p(nodes), _p(n_nodes), cap,
                                                      _p(mem), _p(mem_ts), _p(mail), _p(mail_ts),
                                                      _p(ver), _s(stream)))


def buffers(struct, **tensors):
    """A SampleBuffers / FetchBuffers holding the device pointers of the named tensors."""
    return struct(*[tensors[f].data_ptr() for f, _ in struct._fields_])


def tgm_stage_run(g, st, m, i0, n, B, nb, cap, sample_bufs, fetch_bufs, mem_new, new_mem_ts,
                  winner, h, stream, prefetch_stream, h_trace=None, s_trace=None):
    """sample_bufs: a (SampleBuffers * nsb) array; fetch_bufs: a FetchBuffers;
    h_trace [n x 3B x M] and s_trace [n x cap x M] optional per-iteration
    copies of h and mem_new."""
    _check("tgm_stage_run", lib().tgm_stage_run(
        g, st, m, i0, n, B, nb, cap, sample_bufs, len(sample_bufs), C.byref(fetch_bufs),
        _p(mem_new), _p(new_mem_ts), _p(winner), _p(h), _p(h_trace), _p(s_trace), _s(stream),
        _s(prefetch_stream)))


def alloc_count() -> int:
    """Device allocations the library has made in this process so far."""
    c = I64()
    _check("tgm_alloc_count", lib().tgm_alloc_count(C.byref(c)))
    return int(c.value)


# ------------------------------------------------------------- mitigation
def tgm_mitigator_create(max_nodes, nb, K):
    h = V()
    _check("tgm_mitigator_create", lib().tgm_mitigator_create(max_nodes, nb, K, C.byref(h)))
    return h


def tgm_mitigator_destroy(mt):
    _check("tgm_mitigator_destroy", lib().tgm_mitigator_destroy(mt))


def tgm_mitigate(mt, g, first_event, nodes, n_nodes, cap, mem, mem_ts, M, p, lam, stream=None):
    _check("tgm_mitigate", lib().tgm_mitigate(mt, g, first_event, _p(nodes), _p(n_nodes), cap,
                                              _p(mem), _p(mem_ts), M, float(p), float(lam),
                                              _s(stream)))


def tgm_mitigate_noalloc(g, first_event, nodes, n_nodes, cap, mem, mem_ts, M, nb, K, p, lam,
                         stream=None):
    _check("tgm_mitigate_noalloc", lib().tgm_mitigate_noalloc(
        g, first_event, _p(nodes), _p(n_nodes), cap, _p(mem), _p(mem_ts), M, nb, K, float(p),
        float(lam), _s(stream)))


def tgm_mitigator_read(mt, gamma, n_stale, stale, omega, stream=None):
    _check("tgm_mitigator_read", lib().tgm_mitigator_read(mt, _p(gamma), _p(n_stale), _p(stale),
                                                          _p(omega), _s(stream)))


def tgm_state_set_mitigation(st, mt, p=1.0, lam=1.0):
    _check("tgm_state_set_mitigation", lib().tgm_state_set_mitigation(st, mt, float(p),
                                                                      float(lam)))


# ------------------------------------------------------------- staleness bound
def tgm_min_staleness(tau, n, k_max):
    """Host solver of the minimal-staleness bound: returns (k, fetch_start,
    stall, b, e) for iterations 1..n as numpy arrays (b, e: [n x 5])."""
    import numpy as np
    t = np.ascontiguousarray(tau, dtype=np.float64)
    if t.shape != (5,):
        raise ValueError("tau holds the five stage durations")
    n = int(n)
    k = np.zeros(max(n, 1), np.int32)
    fs, st = np.zeros(max(n, 1)), np.zeros(max(n, 1))
    b, e = np.zeros((max(n, 1), 5)), np.zeros((max(n, 1), 5))
    _check("tgm_min_staleness", lib().tgm_min_staleness(
        t.ctypes.data, n, int(k_max), k.ctypes.data, fs.ctypes.data, st.ctypes.data,
        b.ctypes.data, e.ctypes.data))
    return k[:n], fs[:n], st[:n], b[:n], e[:n]


# ------------------------------------------------------------------ model
def _weights_struct(w, keep):
    def arr(name, dt):
        v = getattr(w, name, None)
        if v is None:
            return None
        a = np.ascontiguousarray(v, dtype=dt)
        keep[name] = a
        return a.ctypes.data_as(_fp if dt == np.float32 else _dp)

    ws = Weights()
    for name in ("W_ih", "W_hh", "b_ih", "b_hh", "W_q", "b_q", "W_k", "b_k", "W_v", "b_v",
                 "W_o", "b_o", "w_t"):
        setattr(ws, name, arr(name, np.float32))
    ws.omega = arr("omega", np.float64)
    ws.beta = arr("beta", np.float64)
    return ws


def tgm_trainer_create(m, w, pred, opt="adam", lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8,
                       stream=None):
    """``w`` the model's numpy weights (workloads.Weights), ``pred`` a
    workloads.Predictor."""
    keep = {}
    ws = _weights_struct(w, keep)
    pa = {k: np.ascontiguousarray(getattr(pred, k), dtype=np.float32)
          for k in ("W_src", "W_dst", "b_p", "w_out")}
    ps = Predictor(*[pa[k].ctypes.data_as(_fp) for k in ("W_src", "W_dst", "b_p", "w_out")],
                   float(pred.b_out))
    os_ = Optimizer(OPTIMIZERS[opt], float(lr), float(beta1), float(beta2), float(eps))
    h = V()
    _check("tgm_trainer_create", lib().tgm_trainer_create(m, C.byref(ws), C.byref(ps),
                                                          C.byref(os_), _s(stream), C.byref(h)))
    return h


def tgm_apan_create(N, M, D_e, D_t, nb, K_mb, propagate, s, max_batch, max_nodes, w,
                    stream=None):
    """``w`` the APAN weights (workloads.make_weights(model='apan'))."""
    keep = {}
    ws = _weights_struct(w, keep)
    d = ApanDesc(N, M, D_e, D_t, nb, K_mb, 1 if propagate else 0, s, max_batch, max_nodes)
    h = V()
    _check("tgm_apan_create", lib().tgm_apan_create(C.byref(d), C.byref(ws), _s(stream),
                                                    C.byref(h)))
    return h


def tgm_apan_destroy(a):
    _check("tgm_apan_destroy", lib().tgm_apan_destroy(a))


def tgm_apan_step(a, g, it, sample_bufs, cap, mem_new, new_mem_ts, h, stream=None):
    _check("tgm_apan_step", lib().tgm_apan_step(a, g, it, C.byref(sample_bufs), cap,
                                                _p(mem_new), _p(new_mem_ts), _p(h),
                                                _s(stream)))


def tgm_apan_flush(a, stream=None):
    _check("tgm_apan_flush", lib().tgm_apan_flush(a, _s(stream)))


def tgm_apan_reset(a, stream=None):
    _check("tgm_apan_reset", lib().tgm_apan_reset(a, _s(stream)))


def tgm_apan_load(a, it, mem, mem_ts, ver, mb, mb_ts, mb_cnt, stream=None):
    _check("tgm_apan_load", lib().tgm_apan_load(a, it, _p(mem), _p(mem_ts), _p(ver), _p(mb),
                                                _p(mb_ts), _p(mb_cnt), _s(stream)))


def tgm_apan_read(a, mem=None, mem_ts=None, ver=None, mb=None, mb_ts=None, mb_cnt=None,
                  stream=None):
    _check("tgm_apan_read", lib().tgm_apan_read(a, _p(mem), _p(mem_ts), _p(ver), _p(mb),
                                                _p(mb_ts), _p(mb_cnt), _s(stream)))


def tgm_apan_fetched(a, mem=None, mem_ts=None, ver=None, mb=None, mb_ts=None, mb_cnt=None,
                     stream=None):
    _check("tgm_apan_fetched", lib().tgm_apan_fetched(a, _p(mem), _p(mem_ts), _p(ver), _p(mb),
                                                      _p(mb_ts), _p(mb_cnt), _s(stream)))


def tgm_trainer_destroy(tr):
    _check("tgm_trainer_destroy", lib().tgm_trainer_destroy(tr))


def tgm_trainer_info(tr):
    """(n_params, [sizes of the 17 tensors], optimizer steps taken)."""
    n, st = I64(), I64()
    sz = (I64 * N_PARAM_TENSORS)()
    _check("tgm_trainer_info", lib().tgm_trainer_info(tr, C.byref(n), sz, C.byref(st)))
    return int(n.value), [int(x) for x in sz], int(st.value)


def tgm_trainer_read(tr, params=None, grad=None, loss=None, stream=None):
    _check("tgm_trainer_read", lib().tgm_trainer_read(tr, _p(params), _p(grad), _p(loss),
                                                      _s(stream)))


def tgm_train_step(tr, m, g, b, sample_bufs, fetch_bufs, mem_new, h, cap, loss=None,
                   stream=None):
    _check("tgm_train_step", lib().tgm_train_step(tr, m, g, b, C.byref(sample_bufs),
                                                  C.byref(fetch_bufs), _p(mem_new), _p(h), cap,
                                                  _p(loss), _s(stream)))


def tgm_state_set_training(st, tr, loss_log=None):
    n = 0 if loss_log is None else int(loss_log.numel())
    _check("tgm_state_set_training", lib().tgm_state_set_training(st, tr, _p(loss_log), n))


def tgm_model_create(M, D_e, D_t, H, nb, max_nodes, max_roots, w, stream=None):
    """``w`` holds numpy weights (fp32; omega and beta fp64), see workloads.Weights."""
    kind = MODEL_KINDS[getattr(w, "kind", "tgn")]
    d = ModelDesc(M, D_e, D_t, H, nb, max_nodes, max_roots, kind)
    keep = {}

    def arr(name, dt):
        v = getattr(w, name, None)
        if v is None:
            return None
        a = np.ascontiguousarray(v, dtype=dt)
        keep[name] = a
        return a.ctypes.data_as(_fp if dt == np.float32 else _dp)

    ws = Weights()
    for name in ("W_ih", "W_hh", "b_ih", "b_hh", "W_q", "b_q", "W_k", "b_k", "W_v", "b_v",
                 "W_o", "b_o", "w_t"):
        setattr(ws, name, arr(name, np.float32))
    ws.omega = arr("omega", np.float64)
    ws.beta = arr("beta", np.float64)
    h = V()
    _check("tgm_model_create", lib().tgm_model_create(C.byref(d), C.byref(ws), _s(stream),
                                                      C.byref(h)))
    return h


def tgm_model_destroy(m):
    _check("tgm_model_destroy", lib().tgm_model_destroy(m))


def tgm_update_memory(st, m, g, it, nodes, n_nodes, cap, mem, mem_ts, mail, mail_ts, ver,
                      first_event, b, src_pos, dst_pos, mem_new, new_mem_ts=None, winner=None,
                      stream=None):
    _check("tgm_update_memory", lib().tgm_update_memory(
        st, m, g, it, _p(nodes), _p(n_nodes), cap, _p(mem), _p(mem_ts), _p(mail), _p(mail_ts),
        _p(ver), first_event, b, _p(src_pos), _p(dst_pos), _p(mem_new), _p(new_mem_ts),
        _p(winner), _s(stream)))


def tgm_embed_projection(m, R, root_pos, root_ts, mem_new, new_mem_ts, n_nodes, cap, h,
                         stream=None):
    _check("tgm_embed_projection", lib().tgm_embed_projection(
        m, R, _p(root_pos), _p(root_ts), _p(mem_new), _p(new_mem_ts), _p(n_nodes), cap, _p(h),
        _s(stream)))


def tgm_embed(m, g, R, nb, root_pos, root_ts, nbr_pos, eid, nts, cnt, mem_new, n_nodes, cap, h,
              stream=None):
    _check("tgm_embed", lib().tgm_embed(m, g, R, nb, _p(root_pos), _p(root_ts), _p(nbr_pos),
                                        _p(eid), _p(nts), _p(cnt), _p(mem_new), _p(n_nodes), cap,
                                        _p(h), _s(stream)))
