"""The sampler's search through the graph's sparse time index (the time of
every 64th adjacency record): lists whose first record and length fall on,
just before and just after multiples of 64, a hub list long enough for two
rounds of the index search, timestamps in long runs of ties, and queries at
every distinct event time, just below and just above them, before the first
and after the last.  Bit-exact against the oracle's sampler (Sec. 5: the nb
most recent strictly earlier events)."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _stream(seed):
    """Events sorted by time.  Node 0 is the hub (about 9,000 events, well
    past 64 x 64 records); nodes 1..12 get list lengths around 64 k, so the
    lists' first records land at many offsets modulo 64."""
    r = np.random.default_rng(seed)
    N = 16
    src, dst = [], []
    for v, L in zip(range(1, 13), (63, 64, 65, 127, 128, 129, 1, 2, 191, 192, 193, 0)):
        for _ in range(L):
            src.append(v)
            dst.append(int(r.integers(13, N)))   # partners among 13..15
    for _ in range(9000):
        src.append(0)
        dst.append(int(r.integers(13, N)))
    for _ in range(37):   # self-loops: one incidence each
        v = int(r.integers(0, N))
        src.append(v)
        dst.append(v)
    E = len(src)
    order = r.permutation(E)
    src = np.asarray(src, np.int32)[order]
    dst = np.asarray(dst, np.int32)[order]
    # times in runs of ties: 300 distinct values
    t = np.sort(r.integers(0, 300, E)).astype(np.float64) * 0.5
    neg = r.integers(0, N, E).astype(np.int32)
    return N, src, dst, t, neg


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("nb", [1, 10, 64])
def test_index_search_against_oracle(orc, seed, nb):
    from paper_2402_15113_amd import tgm
    N, src, dst, t, neg = _stream(seed)
    dev = torch.device("cuda:0")
    T = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)
    g = tgm.tgm_graph_create(N, T(src, torch.int32), T(dst, torch.int32), T(t, torch.float64),
                             T(neg, torch.int32), None)
    times = np.unique(t)
    q = np.concatenate([times, times - 0.25, times + 0.25, [-1.0, t[-1] + 1.0]])
    root = np.repeat(np.arange(N, dtype=np.int32), len(q))
    rts = np.tile(q, N)
    R = len(root)
    out = [torch.empty((R, nb), dtype=torch.int32, device=dev),
           torch.empty((R, nb), dtype=torch.int32, device=dev),
           torch.empty((R, nb), dtype=torch.float64, device=dev),
           torch.empty(R, dtype=torch.int32, device=dev)]
    print(f"sampler index: seed {seed} nb {nb} roots {R}", flush=True)
    tgm.tgm_sample(g, T(root, torch.int32), T(rts, torch.float64), R, nb, *out)
    torch.cuda.synchronize()
    onbr, oeid, onts, ocnt = orc.sample(N, src, dst, t, root, rts, nb)
    np.testing.assert_array_equal(out[3].cpu().numpy(), ocnt)
    np.testing.assert_array_equal(out[0].cpu().numpy(), onbr)
    np.testing.assert_array_equal(out[1].cpu().numpy(), oeid)
    np.testing.assert_array_equal(out[2].cpu().numpy(), onts)
    # the hub's list needs two rounds of the index search, and every list
    # length around 64 k occurs
    _, _, _, n_adj = tgm.tgm_graph_info(g)
    assert n_adj == 2 * len(src) - int((src == dst).sum())
    assert (ocnt[root == 0] == nb).any()
    tgm.tgm_graph_destroy(g)
