// Event graph, batch roots, temporal sampler and node set.
#include <hipcub/hipcub.hpp>

#include <climits>

#include "common.h"

using namespace tgm;

namespace {

// ------------------------------------------------------------ graph build
// Checks ids in [0, N) and t non-decreasing.  bad[0]: id out of range,
// bad[1]: time out of order.
__global__ void k_validate(int64_t E, int32_t N, const int32_t *__restrict__ src,
                           const int32_t *__restrict__ dst, const int32_t *__restrict__ neg,
                           const double *__restrict__ t, int32_t *bad)
{
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t a = src[e], b = dst[e], c = neg[e];
        if (a < 0 || a >= N || b < 0 || b >= N || c < 0 || c >= N)
            atomicOr(&bad[0], 1);
        if (e + 1 < E && !(t[e] <= t[e + 1]))
            atomicOr(&bad[1], 1);
    }
}

// Incidence 2e is (src[e], e); incidence 2e + 1 is (dst[e], e), or the
// sentinel key N for a self-loop so that it sorts past every list.
__global__ void k_incidences(int64_t E, int32_t N, const int32_t *__restrict__ src,
                             const int32_t *__restrict__ dst, int32_t *__restrict__ key,
                             int32_t *__restrict__ val)
{
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < E;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t a = src[e], b = dst[e];
        key[2 * e] = a;
        key[2 * e + 1] = (a == b) ? N : b;
        val[2 * e] = (int32_t)e;
        val[2 * e + 1] = (int32_t)e;
    }
}

// off[v] = first position whose (sorted) key is >= v, for v in [0, N].
__global__ void k_offsets(int64_t n, int32_t N, const int32_t *__restrict__ key,
                          int64_t *__restrict__ off)
{
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k <= n;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t prev = (k == 0) ? -1 : key[k - 1];
        const int32_t cur = (k == n) ? N + 1 : key[k];
        for (int32_t v = prev + 1; v <= cur && v <= N; ++v)
            off[v] = k;
    }
}

__global__ void k_adj_records(int64_t n, const int32_t *__restrict__ key,
                              const int32_t *__restrict__ val, const int32_t *__restrict__ src,
                              const int32_t *__restrict__ dst, const double *__restrict__ t,
                              AdjRec *__restrict__ adj)
{
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < n;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t v = key[k], e = val[k];
        AdjRec r;
        r.ts = t[e];
        r.eid = e;
        r.nbr = (src[e] == v) ? dst[e] : src[e];
        adj[k] = r;
    }
}

// The sparse time index: tix[j] = time of adjacency record 64 j.
__global__ void k_time_index(int64_t n_tix, const AdjRec *__restrict__ adj,
                             double *__restrict__ tix)
{
    for (int64_t j = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; j < n_tix;
         j += (int64_t)gridDim.x * blockDim.x)
        tix[j] = adj[j * kWave].ts;
}

int grid_for(int64_t n, int block)
{
    int64_t g = cdiv(n, block);
    if (g > 65536)
        g = 65536;
    return (int)(g < 1 ? 1 : g);
}

// ------------------------------------------------------------ batch roots
__global__ void k_batch_roots(int64_t first, int32_t b, const int32_t *__restrict__ src,
                              const int32_t *__restrict__ dst, const int32_t *__restrict__ neg,
                              const double *__restrict__ t, int32_t *__restrict__ root,
                              double *__restrict__ root_ts)
{
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= b)
        return;
    const int64_t e = first + k;
    const double te = t[e];
    root[k] = src[e];
    root[b + k] = dst[e];
    root[2 * b + k] = neg[e];
    root_ts[k] = te;
    root_ts[b + k] = te;
    root_ts[2 * b + k] = te;
}

// ------------------------------------------------------------ sampler
// One wavefront per root: recent_end() finds the end of the root's strictly
// earlier events, then lanes j < nb read entries p-1-j: the nb most recent
// strictly earlier events, newest first.
__device__ __forceinline__ void sample_one(const int64_t *__restrict__ off,
                                           const AdjRec *__restrict__ adj,
                                           const double *__restrict__ tix, int r, int32_t v,
                                           double tq, int32_t N, int32_t nb,
                                           int32_t *__restrict__ nbr, int32_t *__restrict__ eid,
                                           double *__restrict__ nts, int32_t *__restrict__ cnt,
                                           int32_t *__restrict__ stamp = nullptr,
                                           int32_t epoch = 0)
{
    const int lane = threadIdx.x & 63;
    if (stamp && v >= 0 && v < N && lane == 0)   // node-set mark of the root (see k_ns_mark)
        stamp[v] = epoch;
    int64_t base;
    const int64_t p = recent_end(off, adj, tix, v, tq, N, &base);
    const int64_t avail = p - base;
    const int c = avail < nb ? (int)avail : nb;
    if (lane < nb) {
        const int64_t o = (int64_t)r * nb + lane;
        if (lane < c) {
            const AdjRec a = adj[p - 1 - lane];
            nbr[o] = a.nbr;
            eid[o] = a.eid;
            nts[o] = a.ts;
            if (stamp)   // adjacency ids are in [0, N): checked at graph creation
                stamp[a.nbr] = epoch;
        } else {
            nbr[o] = -1;
            eid[o] = -1;
            nts[o] = 0.0;
        }
    }
    if (lane == 0)
        cnt[r] = c;
}

__global__ __launch_bounds__(256) void k_sample(const int64_t *__restrict__ off,
                                                const AdjRec *__restrict__ adj,
                                                const double *__restrict__ tix,
                                                const int32_t *__restrict__ root,
                                                const double *__restrict__ root_ts, int32_t R,
                                                int32_t N, int32_t nb, int32_t *__restrict__ nbr,
                                                int32_t *__restrict__ eid,
                                                double *__restrict__ nts,
                                                int32_t *__restrict__ cnt)
{
    const int r = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    if (r >= R)
        return;
    sample_one(off, adj, tix, r, root[r], root_ts[r], N, nb, nbr, eid, nts, cnt);
}

// Roots of a batch and their sampling in one pass: wavefront r takes root r
// of src[batch] ++ dst[batch] ++ neg[batch] straight from the event arrays.
__global__ __launch_bounds__(256) void k_sample_batch(
    const int64_t *__restrict__ off, const AdjRec *__restrict__ adj,
    const double *__restrict__ tix, int64_t first, int32_t b,
    const int32_t *__restrict__ src, const int32_t *__restrict__ dst,
    const int32_t *__restrict__ neg, const double *__restrict__ t, int32_t N, int32_t nb,
    int32_t *__restrict__ root, double *__restrict__ root_ts, int32_t *__restrict__ nbr,
    int32_t *__restrict__ eid, double *__restrict__ nts, int32_t *__restrict__ cnt,
    int32_t *__restrict__ stamp, int32_t epoch)
{
    const int r = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    if (r >= 3 * b)
        return;
    const int third = r / b, k = r - third * b;
    const int64_t e = first + k;
    const int32_t v = third == 0 ? src[e] : (third == 1 ? dst[e] : neg[e]);
    const double tq = t[e];
    if ((threadIdx.x & 63) == 0) {
        root[r] = v;
        root_ts[r] = tq;
    }
    sample_one(off, adj, tix, r, v, tq, N, nb, nbr, eid, nts, cnt, stamp, epoch);
}

// ------------------------------------------------------------ node set
// Two launches.  k_ns_mark stamps every valid root and neighbour id into the
// graph's per-node stamp array with this call's epoch (plain stores: all
// writers of one id write the same value, so no atomics and no clearing).
// In k_ns_pos every workgroup turns the stamps into a membership bitmap
// (one ballot per 64 ids), scans its word popcounts (which numbers the
// members in id order: sorted and deduplicated in one pass), writes its share
// of U and maps its slice of roots and neighbours to their positions.  The
// bitmap is rebuilt per workgroup because it is small (N/8 bytes) and L2-hot;
// that replaces a grid-wide barrier.
constexpr int kNsThreads = 1024;
constexpr int kNsWaves = kNsThreads / kWave;
constexpr int kNsIds = 2;                          // ids per thread in k_ns_pos
constexpr int kNsIdsPerBlock = kNsThreads * kNsIds;
constexpr int kNsScan = 8;                         // stamp loads in flight per thread
constexpr int kNsMaxWords = 1 << 13;               // 2^19 node ids

__global__ __launch_bounds__(256) void k_fill_i32(int32_t *__restrict__ p, int32_t n, int32_t v)
{
    const int k = blockIdx.x * 256 + threadIdx.x;
    if (k < n)
        p[k] = v;
}

__global__ __launch_bounds__(256) void k_ns_mark(int32_t N, const int32_t *__restrict__ root,
                                                 int32_t R, const int32_t *__restrict__ nbr,
                                                 int32_t total, int32_t *__restrict__ stamp,
                                                 int32_t epoch)
{
    const int k = blockIdx.x * 256 + threadIdx.x;
    if (k >= total)
        return;
    const int32_t x = k < R ? root[k] : nbr[k - R];
    if (x >= 0 && x < N)
        stamp[x] = epoch;
}

__global__ __launch_bounds__(kNsThreads) void k_ns_pos(
    int32_t N, const int32_t *__restrict__ stamp, int32_t epoch,
    const int32_t *__restrict__ root, int32_t R, const int32_t *__restrict__ nbr, int32_t total,
    int32_t *__restrict__ nodes, int32_t *__restrict__ n_nodes, int32_t *__restrict__ root_pos,
    int32_t *__restrict__ nbr_pos)
{
    extern __shared__ uint64_t ns_mask[];                 // [NW] membership words
    const int NW = (N + 63) >> 6;
    uint32_t *pre = reinterpret_cast<uint32_t *>(ns_mask + NW);   // [NW] exclusive prefix
    __shared__ uint32_t wave_tot[kNsWaves];
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // this workgroup's ids, loaded first so their latency hides behind the scan
    const int k0 = blockIdx.x * kNsIdsPerBlock + tid;
    int32_t x[kNsIds];
#pragma unroll
    for (int u = 0; u < kNsIds; ++u) {
        const int k = k0 + u * kNsThreads;
        x[u] = k < R ? root[k] : (k < total ? nbr[k - R] : -1);
    }

    // 1. membership words: kNsScan coalesced stamp loads in flight per thread,
    // then one ballot per 64 ids (wave w of round u covers word 16 u + w)
    for (int base = 0; base < NW * kWave; base += kNsScan * kNsThreads) {
        int32_t f[kNsScan];
#pragma unroll
        for (int u = 0; u < kNsScan; ++u) {
            const int id = base + u * kNsThreads + tid;
            f[u] = id < N ? stamp[id] : 0;
        }
#pragma unroll
        for (int u = 0; u < kNsScan; ++u) {
            const int w = (base >> 6) + u * kNsWaves + wave;
            const uint64_t m = __ballot(f[u] == epoch);
            if (w < NW && lane == 0)
                ns_mask[w] = m;
        }
    }
    __syncthreads();

    // 2. exclusive prefix of the word popcounts: contiguous word ranges per
    // thread, a shuffle scan per wave, then the wave totals
    const int per = (NW + kNsThreads - 1) / kNsThreads;
    const int wa = min(NW, tid * per), wz = min(NW, wa + per);
    uint32_t sum = 0;
    for (int w = wa; w < wz; ++w)
        sum += (uint32_t)__popcll(ns_mask[w]);
    uint32_t inc = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o, kWave);
        if (lane >= o)
            inc += y;
    }
    if (lane == kWave - 1)
        wave_tot[wave] = inc;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int v = 0; v < kNsWaves; ++v) {
        const uint32_t t = wave_tot[v];
        before += v < wave ? t : 0u;
        all += t;
    }
    uint32_t run = before + inc - sum;
    for (int w = wa; w < wz; ++w) {
        pre[w] = run;
        run += (uint32_t)__popcll(ns_mask[w]);
    }
    __syncthreads();

    // 3. this workgroup's share of U: one wave per membership word
    for (int w = blockIdx.x * kNsWaves + wave; w < NW; w += gridDim.x * kNsWaves) {
        const uint64_t m = ns_mask[w];
        if ((m >> lane) & 1ull)
            nodes[pre[w] + (uint32_t)__popcll(m & ((1ull << lane) - 1ull))] = w * kWave + lane;
    }
    if (blockIdx.x == 0 && tid == 0)
        *n_nodes = (int32_t)all;

    // 4. positions of this workgroup's roots and neighbours (-1 for ids
    // outside [0, N), which are not members)
#pragma unroll
    for (int u = 0; u < kNsIds; ++u) {
        const int k = k0 + u * kNsThreads;
        if (k < total) {
            const int32_t v = x[u];
            int32_t q = -1;
            if (v >= 0 && v < N) {
                const int w = v >> 6;
                q = (int32_t)(pre[w] +
                              (uint32_t)__popcll(ns_mask[w] & ((1ull << (v & 63)) - 1ull)));
            }
            if (k < R)
                root_pos[k] = q;
            else
                nbr_pos[k - R] = q;
        }
    }
}

}  // namespace

// ======================================================================== API

extern "C" tgm_status_t tgm_graph_create(int32_t N, int64_t E, const int32_t *src,
                                         const int32_t *dst, const double *t,
                                         const int32_t *neg, const float *efeat, int32_t D_e,
                                         void *stream, tgm_graph_t *out)
{
    if (!out || N <= 0 || E < 0 || D_e < 0 || 2 * E >= (int64_t)INT_MAX)
        return TGM_EINVAL;
    if (E > 0 && (!src || !dst || !t || !neg))
        return TGM_EINVAL;
    if ((D_e > 0) != (efeat != nullptr) && E > 0)
        return TGM_EINVAL;
    *out = nullptr;
    hipStream_t s = as_stream(stream);
    tgm_graph *g = new tgm_graph();
    g->N = N;
    g->E = E;
    g->D_e = D_e;
    g->src = src;
    g->dst = dst;
    g->t = t;
    g->neg = neg;
    g->efeat = efeat;

    const int64_t n2 = 2 * E;
    int32_t *bad = nullptr, *key = nullptr, *val = nullptr, *key2 = nullptr, *val2 = nullptr;
    void *tmp = nullptr;
    size_t tmp_bytes = 0;
    tgm_status_t st = TGM_OK;
    auto fail = [&](tgm_status_t code) {
        st = code;
    };
    do {
        if (dev_malloc(&g->off, sizeof(int64_t) * (N + 1)) != hipSuccess) { fail(TGM_ENOMEM); break; }
        if (dev_malloc(&bad, sizeof(int32_t) * 2) != hipSuccess) { fail(TGM_ENOMEM); break; }
        if (dev_malloc(&g->ns_stamp, sizeof(int32_t) * N) != hipSuccess) { fail(TGM_ENOMEM); break; }
        if (hipMemsetAsync(g->ns_stamp, 0, sizeof(int32_t) * N, s) != hipSuccess) { fail(TGM_EDEVICE); break; }
        if (hipMemsetAsync(bad, 0, sizeof(int32_t) * 2, s) != hipSuccess) { fail(TGM_EDEVICE); break; }
        if (E == 0) {
            if (hipMemsetAsync(g->off, 0, sizeof(int64_t) * (N + 1), s) != hipSuccess) { fail(TGM_EDEVICE); break; }
            if (hipStreamSynchronize(s) != hipSuccess) { fail(TGM_EDEVICE); break; }
            break;
        }
        hipLaunchKernelGGL(k_validate, dim3(grid_for(E, 256)), dim3(256), 0, s, E, N, src, dst,
                           neg, t, bad);
        int32_t hbad[2] = {0, 0};
        if (hipMemcpyAsync(hbad, bad, sizeof(hbad), hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) { fail(TGM_EDEVICE); break; }
        if (hbad[0] || hbad[1]) { fail(TGM_ERANGE); break; }

        if (dev_malloc(&key, sizeof(int32_t) * n2) != hipSuccess ||
            dev_malloc(&val, sizeof(int32_t) * n2) != hipSuccess ||
            dev_malloc(&key2, sizeof(int32_t) * n2) != hipSuccess ||
            dev_malloc(&val2, sizeof(int32_t) * n2) != hipSuccess) { fail(TGM_ENOMEM); break; }
        hipLaunchKernelGGL(k_incidences, dim3(grid_for(E, 256)), dim3(256), 0, s, E, N, src, dst,
                           key, val);
        int bits = 1;
        while ((1ll << bits) <= (int64_t)N)
            ++bits;
        // LSD radix sort is stable: within a node, incidences keep event order
        if (hipcub::DeviceRadixSort::SortPairs(nullptr, tmp_bytes, key, key2, val, val2, (int)n2,
                                               0, bits, s) != hipSuccess) { fail(TGM_EDEVICE); break; }
        if (dev_malloc(&tmp, tmp_bytes) != hipSuccess) { fail(TGM_ENOMEM); break; }
        if (hipcub::DeviceRadixSort::SortPairs(tmp, tmp_bytes, key, key2, val, val2, (int)n2, 0,
                                               bits, s) != hipSuccess) { fail(TGM_EDEVICE); break; }
        hipLaunchKernelGGL(k_offsets, dim3(grid_for(n2 + 1, 256)), dim3(256), 0, s, n2, N, key2,
                           g->off);
        int64_t n_adj = 0;
        if (hipMemcpyAsync(&n_adj, g->off + N, sizeof(int64_t), hipMemcpyDeviceToHost, s) !=
                hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) { fail(TGM_EDEVICE); break; }
        g->n_adj = n_adj;
        if (dev_malloc(&g->adj, sizeof(AdjRec) * (n_adj > 0 ? n_adj : 1)) != hipSuccess) { fail(TGM_ENOMEM); break; }
        const int64_t n_tix = cdiv(n_adj, kWave);
        if (dev_malloc(&g->tix, sizeof(double) * (n_tix > 0 ? n_tix : 1)) != hipSuccess) { fail(TGM_ENOMEM); break; }
        if (n_adj > 0) {
            hipLaunchKernelGGL(k_adj_records, dim3(grid_for(n_adj, 256)), dim3(256), 0, s, n_adj,
                               key2, val2, src, dst, t, g->adj);
            hipLaunchKernelGGL(k_time_index, dim3(grid_for(n_tix, 256)), dim3(256), 0, s, n_tix,
                               g->adj, g->tix);
        }
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) { fail(TGM_EDEVICE); break; }
    } while (0);
    hipFree(bad);
    hipFree(key);
    hipFree(val);
    hipFree(key2);
    hipFree(val2);
    hipFree(tmp);
    if (st != TGM_OK) {
        tgm_graph_destroy(g);
        return st;
    }
    *out = g;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_graph_destroy(tgm_graph_t g)
{
    if (!g)
        return TGM_EINVAL;
    hipFree(g->off);
    hipFree(g->adj);
    hipFree(g->tix);
    hipFree(g->ns_stamp);
    delete g;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_graph_info(tgm_graph_t g, int32_t *N, int64_t *E, int32_t *D_e,
                                       int64_t *n_adj)
{
    if (!g)
        return TGM_EINVAL;
    if (N) *N = g->N;
    if (E) *E = g->E;
    if (D_e) *D_e = g->D_e;
    if (n_adj) *n_adj = g->n_adj;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_batch_roots(tgm_graph_t g, int64_t first_event, int32_t b,
                                        int32_t *root, double *root_ts, void *stream)
{
    if (!g || b < 0 || first_event < 0 || first_event + b > g->E)
        return TGM_EINVAL;
    if (b == 0)
        return TGM_OK;
    if (!root || !root_ts)
        return TGM_EINVAL;
    TGM_LAUNCH(k_batch_roots, dim3(cdiv(b, 256)), dim3(256), 0, as_stream(stream),
                       first_event, b, g->src, g->dst, g->neg, g->t, root, root_ts);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_sample(tgm_graph_t g, const int32_t *root, const double *root_ts,
                                   int32_t R, int32_t nb, int32_t *nbr, int32_t *eid,
                                   double *nts, int32_t *cnt, void *stream)
{
    if (!g || R < 0 || nb < 1 || nb > kWave)
        return TGM_EINVAL;
    if (R == 0)
        return TGM_OK;
    if (!root || !root_ts || !nbr || !eid || !nts || !cnt)
        return TGM_EINVAL;
    const int per_block = 256 / kWave;
    TGM_LAUNCH(k_sample, dim3(cdiv(R, per_block)), dim3(256), 0, as_stream(stream),
                       g->off, g->adj, g->tix, root, root_ts, R, g->N, nb, nbr, eid, nts, cnt);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_sample_batch(tgm_graph_t g, int64_t first_event, int32_t b,
                                         int32_t nb, int32_t *root, double *root_ts,
                                         int32_t *nbr, int32_t *eid, double *nts, int32_t *cnt,
                                         void *stream)
{
    if (!g || b < 0 || first_event < 0 || first_event + b > g->E || nb < 1 || nb > kWave)
        return TGM_EINVAL;
    if (b == 0)
        return TGM_OK;
    if (!root || !root_ts || !nbr || !eid || !nts || !cnt)
        return TGM_EINVAL;
    const int per_block = 256 / kWave;
    TGM_LAUNCH(k_sample_batch, dim3(cdiv(3 * (int64_t)b, per_block)), dim3(256), 0,
               as_stream(stream), g->off, g->adj, g->tix, first_event, b, g->src, g->dst, g->neg, g->t,
               g->N, nb, root, root_ts, nbr, eid, nts, cnt, nullptr, 0);
    return TGM_OK;
}

namespace {

tgm_status_t ns_check(tgm_graph_t g, int32_t R, int32_t nb, const int32_t *root,
                      const int32_t *nbr, const int32_t *nodes, const int32_t *n_nodes,
                      int32_t cap, const int32_t *root_pos, const int32_t *nbr_pos)
{
    if (!g || R < 0 || nb < 0 || !n_nodes || (int64_t)R * (nb + 1) > INT32_MAX)
        return TGM_EINVAL;
    const int64_t need = std::min<int64_t>(g->N, (int64_t)R * (nb + 1));
    if (cap < need)
        return TGM_ESIZE;
    if ((R > 0 && (!root || !nodes || !root_pos)) || ((int64_t)R * nb > 0 && (!nbr || !nbr_pos)))
        return TGM_EINVAL;
    if (((g->N + 63) >> 6) > kNsMaxWords)
        return TGM_EINVAL;
    return TGM_OK;
}

// The epoch of a new node set (stamps of older sets never equal it).
tgm_status_t ns_next_epoch(tgm_graph_t g, hipStream_t s, int32_t *epoch)
{
    if (g->ns_epoch == INT32_MAX) {   // stamps restart from zero
        TGM_LAUNCH(k_fill_i32, dim3(cdiv(g->N, 256)), dim3(256), 0, s, g->ns_stamp, g->N, 0);
        g->ns_epoch = 0;
    }
    *epoch = ++g->ns_epoch;
    return TGM_OK;
}

// Ranking of the ids stamped with `epoch`: U, its size and the positions.
tgm_status_t ns_rank(tgm_graph_t g, const int32_t *root, int32_t R, const int32_t *nbr,
                     int32_t nb, int32_t *nodes, int32_t *n_nodes, int32_t *root_pos,
                     int32_t *nbr_pos, int32_t epoch, hipStream_t s)
{
    const int NW = (g->N + 63) >> 6;
    const size_t lds = (sizeof(uint64_t) + sizeof(uint32_t)) * NW;
    static bool lds_opt_in = false;
    if (!lds_opt_in) {
        TGM_HIP(hipFuncSetAttribute((const void *)k_ns_pos,
                                    hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)((sizeof(uint64_t) + sizeof(uint32_t)) * kNsMaxWords)));
        lds_opt_in = true;
    }
    const int32_t total = (int32_t)((int64_t)R * (nb + 1));
    TGM_LAUNCH(k_ns_pos, dim3((unsigned)std::max<int64_t>(1, cdiv(total, kNsIdsPerBlock))),
               dim3(kNsThreads), lds, s, g->N, g->ns_stamp, epoch, root, R, nbr, total, nodes,
               n_nodes, root_pos, nbr_pos);
    return TGM_OK;
}

}  // namespace

extern "C" tgm_status_t tgm_node_set(tgm_graph_t g, const int32_t *root, int32_t R,
                                     const int32_t *nbr, int32_t nb, int32_t *nodes,
                                     int32_t *n_nodes, int32_t cap, int32_t *root_pos,
                                     int32_t *nbr_pos, void *stream)
{
    tgm_status_t st = ns_check(g, R, nb, root, nbr, nodes, n_nodes, cap, root_pos, nbr_pos);
    if (st != TGM_OK)
        return st;
    hipStream_t s = as_stream(stream);
    int32_t epoch = 0;
    if ((st = ns_next_epoch(g, s, &epoch)) != TGM_OK)
        return st;
    const int32_t total = (int32_t)((int64_t)R * (nb + 1));
    if (total > 0)
        TGM_LAUNCH(k_ns_mark, dim3(cdiv(total, 256)), dim3(256), 0, s, g->N, root, R, nbr, total,
                   g->ns_stamp, epoch);
    return ns_rank(g, root, R, nbr, nb, nodes, n_nodes, root_pos, nbr_pos, epoch, s);
}

extern "C" tgm_status_t tgm_sample_nodes(tgm_graph_t g, int64_t first_event, int32_t b,
                                         int32_t nb, int32_t *root, double *root_ts,
                                         int32_t *nbr, int32_t *eid, double *nts, int32_t *cnt,
                                         int32_t *nodes, int32_t *n_nodes, int32_t cap,
                                         int32_t *root_pos, int32_t *nbr_pos, void *stream)
{
    if (!g || b < 0 || first_event < 0 || first_event + b > g->E || nb < 1 || nb > kWave)
        return TGM_EINVAL;
    if (b > 0 && (!root || !root_ts || !nbr || !eid || !nts || !cnt))
        return TGM_EINVAL;
    const int32_t R = 3 * b;
    tgm_status_t st = ns_check(g, R, nb, root, nbr, nodes, n_nodes, cap, root_pos, nbr_pos);
    if (st != TGM_OK)
        return st;
    hipStream_t s = as_stream(stream);
    int32_t epoch = 0;
    if ((st = ns_next_epoch(g, s, &epoch)) != TGM_OK)
        return st;
    if (b > 0) {   // the sampler stamps every root and neighbour it writes
        const int per_block = 256 / kWave;
        TGM_LAUNCH(k_sample_batch, dim3(cdiv(3 * (int64_t)b, per_block)), dim3(256), 0, s, g->off,
                   g->adj, g->tix, first_event, b, g->src, g->dst, g->neg, g->t, g->N, nb, root,
                   root_ts, nbr, eid, nts, cnt, g->ns_stamp, epoch);
    }
    return ns_rank(g, root, R, nbr, nb, nodes, n_nodes, root_pos, nbr_pos, epoch, s);
}
