"""Reads a state checkpoint (the host buffer of tgm_state_save) into numpy
arrays: the committed tables, and the pending write sets as the oracle takes
them (Oracle.set_state(..., pending=...)).  The layout is the one
include/tgm.h documents: an int64 header (magic, format, N, M, D_m, s,
max_batch, committed through, staged through, last fetch, slots), an int64
(iteration, b, staged) triple per ring slot, then 8-byte-aligned sections:
mem, mem_ts, mail, mail_ts, ver, and the ring's r_flag, r_node, r_mem,
r_mail, r_mem_ts, r_mail_ts (2 max_batch rows per slot)."""
import numpy as np

MAGIC = 0x74676D2D636B7074
HEADER = 11


def parse(buf):
    buf = np.ascontiguousarray(buf, dtype=np.uint8)
    h = buf[:8 * HEADER].view(np.int64)
    assert int(h[0]) == MAGIC and int(h[1]) == 1
    N, M, D_m, s, max_batch, committed, staged, last_fetch, slots = (int(x) for x in h[2:11])
    meta = buf[8 * HEADER:8 * (HEADER + 3 * slots)].view(np.int64).reshape(slots, 3)
    rows = slots * 2 * max_batch
    off = 8 * (HEADER + 3 * slots)
    out = {}
    for name, dt, n in (("mem", np.float32, N * M), ("mem_ts", np.float64, N),
                        ("mail", np.float32, N * D_m), ("mail_ts", np.float64, N),
                        ("ver", np.int32, N), ("r_flag", np.int32, rows),
                        ("r_node", np.int32, rows), ("r_mem", np.float32, rows * M),
                        ("r_mail", np.float32, rows * D_m), ("r_mem_ts", np.float64, rows),
                        ("r_mail_ts", np.float64, rows)):
        nbytes = n * np.dtype(dt).itemsize
        out[name] = buf[off:off + nbytes].view(dt).copy()
        off += (nbytes + 7) & ~7
    assert off <= buf.nbytes
    pending = []
    for it in range(committed + 1, staged + 1):
        j = it % slots
        assert int(meta[j, 0]) == it and int(meta[j, 2]) == 1
        b = int(meta[j, 1])
        lo = j * 2 * max_batch
        sel = lo + np.flatnonzero(out["r_flag"][lo:lo + 2 * b] != 0)
        pending.append((it, out["r_node"][sel],
                        out["r_mem"].reshape(rows, M)[sel].astype(np.float64),
                        out["r_mem_ts"][sel],
                        out["r_mail"].reshape(rows, D_m)[sel].astype(np.float64),
                        out["r_mail_ts"][sel]))
    return dict(N=N, M=M, D_m=D_m, s=s, next_iter=staged + 1, last_fetch=last_fetch,
                mem=out["mem"].reshape(N, M).astype(np.float64), mem_ts=out["mem_ts"],
                mail=out["mail"].reshape(N, D_m).astype(np.float64), mail_ts=out["mail_ts"],
                ver=out["ver"], pending=pending)
