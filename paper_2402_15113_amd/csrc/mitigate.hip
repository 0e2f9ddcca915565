// Similarity-based staleness mitigation (MSPipe-S, Sec. 4.3) of the fetched
// memories of a batch, between the fetch and the memory update.  For the
// fetched node set U (positions p < n, memory times mem_ts):
//   gap       dt_p = T - mem_ts_p, T the time of the batch's first event;
//   gamma     the nearest-rank quantile: the ceil(p_q n)-th smallest gap;
//   stale     dt > gamma; active: dt < gamma;
//   N(u)      the distinct other endpoints of u's nb most recent events
//             before T (the sampler's temporal neighbourhood);
//   Omega(v)  the K active nodes with the most common neighbours (at least
//             one), then the fresher memory, then the smaller id;
//   s_v      <- lambda s_v + (1 - lambda) mean_{u in Omega(v)} s_u  (in place;
//             a stale row is never a source: sources are active).
// Three launches: k_mit_prep (one wavefront per node: gap and sorted distinct
// neighbour set), k_mit_select (one workgroup: a radix select of gamma over
// the order-preserving 64-bit keys of the gaps, then the stale positions in
// order), k_mit_omega (one workgroup per stale node: its neighbour set in an
// LDS hash set, every active node probed against it, a per-thread top-K, a
// wave-merge of the sorted lists, the blend).  Integer decisions only; the
// gaps are formed exactly as the oracle forms them (one fp64 subtraction).
#include <hip/hip_runtime.h>

#include "common.h"

using namespace tgm;

struct tgm_mitigator {
    int32_t cap = 0, nb = 0, nbp = 0, K = 0;
    double *dt = nullptr;        // [cap] gaps
    int32_t *nset = nullptr;     // [cap x nbp] sorted distinct neighbour ids
    int32_t *ncnt = nullptr;     // [cap]
    double *gamma = nullptr;     // [1]
    int32_t *n_stale = nullptr;  // [1]
    int32_t *stale = nullptr;    // [cap] stale positions, ascending
    int32_t *omega = nullptr;    // [cap x K] Omega positions, -1 padded
};

namespace {

constexpr int kMitMaxK = 16;
constexpr int kMitHash = 256;          // LDS hash slots (>= 4 nb)
constexpr int kMitThreads = 256;       // k_mit_omega
constexpr int kMitSelThreads = 1024;   // k_mit_select

// ---------------------------------------------------------------- prep
// One wavefront per fetched node: its gap and its sorted distinct neighbour
// set.  Lane j < c holds the j-th most recent neighbour; duplicates and ranks
// come from a loop over the c lanes with readlane (c <= nb <= 64).
__global__ __launch_bounds__(256) void k_mit_prep(const int64_t *__restrict__ off,
                                                  const AdjRec *__restrict__ adj, int32_t N,
                                                  const double *__restrict__ t, int64_t first,
                                                  const int32_t *__restrict__ nodes,
                                                  const int32_t *__restrict__ n_nodes,
                                                  int32_t cap, const double *__restrict__ mem_ts,
                                                  int32_t nb, int32_t nbp,
                                                  double *__restrict__ dt,
                                                  int32_t *__restrict__ nset,
                                                  int32_t *__restrict__ ncnt)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int n = min(*n_nodes, cap);
    if (p >= n)
        return;   // whole wavefronts
    const int lane = threadIdx.x & 63;
    const double T = t[first];
    const int32_t v = nodes[p];
    int64_t base;
    const int64_t end = recent_end(off, adj, v, T, N, &base);
    const int c = end - base < nb ? (int)(end - base) : nb;
    const int32_t w = lane < c ? adj[end - 1 - lane].nbr : INT32_MAX;
    bool dup = false;   // an earlier lane holds the same id
    int less = 0;       // distinct ids below w
    for (int i = 0; i < c; ++i) {
        const int32_t x = __builtin_amdgcn_readlane(w, i);
        bool first_of_x = true;   // x is the first lane holding its value
        for (int k = 0; k < i; ++k)
            first_of_x = first_of_x && __builtin_amdgcn_readlane(w, k) != x;
        dup = dup || (i < lane && x == w);
        less += (first_of_x && x < w) ? 1 : 0;
    }
    if (lane < c && !dup)
        nset[(int64_t)p * nbp + less] = w;
    const uint64_t firsts = __ballot(lane < c && !dup);
    if (lane == 0) {
        ncnt[p] = __popcll(firsts);
        dt[p] = T - mem_ts[p];
    }
}

// ---------------------------------------------------------------- select
__device__ __forceinline__ uint64_t order_key(double x)
{
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

__device__ __forceinline__ double key_value(uint64_t k)
{
    const uint64_t u = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
    return __longlong_as_double((long long)u);
}

// One workgroup: gamma = the rank-th smallest gap (rank = ceil(pq n) in fp64,
// clamped to [1, n]) by an 8-pass radix select on 8-bit digits, most
// significant first; then the positions with dt > gamma, ascending.
__global__ __launch_bounds__(kMitSelThreads) void k_mit_select(
    const double *__restrict__ dt, const int32_t *__restrict__ n_nodes, int32_t cap, double pq,
    double *__restrict__ gamma_out, int32_t *__restrict__ stale, int32_t *__restrict__ n_stale)
{
    __shared__ uint32_t hist[256];
    __shared__ uint64_t s_prefix;
    __shared__ int s_krem;
    __shared__ int s_wsum[kMitSelThreads / kWave];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nw = blockDim.x >> 6;
    const int n = min(*n_nodes, cap);
    if (n <= 0) {
        if (tid == 0) {
            *n_stale = 0;
            *gamma_out = 0.0;
        }
        return;
    }
    long long rank = (long long)ceil(pq * (double)n);
    rank = rank < 1 ? 1 : (rank > n ? n : rank);
    int krem = (int)(rank - 1);
    uint64_t prefix = 0, mask = 0;
    for (int pass = 7; pass >= 0; --pass) {
        const int sh = 8 * pass;
        for (int i = tid; i < 256; i += blockDim.x)
            hist[i] = 0;
        __syncthreads();
        for (int i = tid; i < n; i += blockDim.x) {
            const uint64_t k = order_key(dt[i]);
            if ((k & mask) == prefix)
                atomicAdd(&hist[(k >> sh) & 255], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            // lane l holds bins 4l .. 4l + 3; a wave scan finds the bin of krem
            uint32_t b[4];
            uint32_t sum = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                b[j] = hist[4 * lane + j];
                sum += b[j];
            }
            uint32_t incl = sum;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const uint32_t y = __shfl_up(incl, o, kWave);
                if (lane >= o)
                    incl += y;
            }
            const uint32_t excl = incl - sum;
            if (excl <= (uint32_t)krem && (uint32_t)krem < incl) {
                uint32_t cum = excl;
                int bin = 4 * lane + 3;
                bool found = false;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (!found) {
                        if ((uint32_t)krem < cum + b[j]) {
                            bin = 4 * lane + j;
                            found = true;
                        } else {
                            cum += b[j];
                        }
                    }
                }
                s_prefix = prefix | ((uint64_t)bin << sh);
                s_krem = krem - (int)cum;
            }
        }
        __syncthreads();
        prefix = s_prefix;
        krem = s_krem;
        mask |= 255ull << sh;
        __syncthreads();
    }
    const double gamma = key_value(prefix);
    // stale positions in order, one block of blockDim.x positions at a time
    int base = 0;
    for (int b0 = 0; b0 < n; b0 += blockDim.x) {
        const int i = b0 + tid;
        const bool f = i < n && dt[i] > gamma;
        const uint64_t bal = __ballot(f);
        const int in_wave = __popcll(bal & ((1ull << lane) - 1));
        if (lane == 0)
            s_wsum[wave] = __popcll(bal);
        __syncthreads();
        int before = 0, total = 0;
        for (int k = 0; k < nw; ++k) {
            before += k < wave ? s_wsum[k] : 0;
            total += s_wsum[k];
        }
        if (f)
            stale[base + before + in_wave] = i;
        base += total;
        __syncthreads();
    }
    if (tid == 0) {
        *n_stale = base;
        *gamma_out = gamma;
    }
}

// ---------------------------------------------------------------- omega
struct Cand {
    int sim;
    double mts;
    int32_t id, pos;
};

// more common neighbours, then the fresher memory, then the smaller id
__device__ __forceinline__ bool better(const Cand &a, const Cand &b)
{
    if (a.sim != b.sim)
        return a.sim > b.sim;
    if (a.mts != b.mts)
        return a.mts > b.mts;
    return a.id < b.id;
}

__device__ __forceinline__ int hash_slot(int32_t w) { return (int)(((uint32_t)w * 2654435761u) >> 24); }

__device__ __forceinline__ bool hash_has(const int32_t *hs, int32_t w)
{
    for (int k = 0, s = hash_slot(w); k < kMitHash; ++k, s = (s + 1) & (kMitHash - 1)) {
        const int32_t x = hs[s];
        if (x == w)
            return true;
        if (x < 0)
            return false;
    }
    return false;
}

// One workgroup per stale node (blocks past the count exit).
__global__ __launch_bounds__(kMitThreads) void k_mit_omega(
    const int32_t *__restrict__ nodes, const int32_t *__restrict__ n_nodes, int32_t cap,
    const double *__restrict__ dt, const double *__restrict__ mem_ts,
    const int32_t *__restrict__ nset, const int32_t *__restrict__ ncnt, int32_t nbp,
    const double *__restrict__ gamma_p, const int32_t *__restrict__ stale,
    const int32_t *__restrict__ n_stale, int32_t K, float lambda, float *__restrict__ mem,
    int32_t M, int32_t *__restrict__ omega)
{
    __shared__ int32_t hs[kMitHash];
    // each thread's sorted list: similarity and position (mem_ts and the id
    // are read back through the position)
    __shared__ int c_sim[kMitThreads * kMitMaxK];
    __shared__ int32_t c_pos[kMitThreads * kMitMaxK];
    __shared__ int32_t r_pos[kMitMaxK];
    __shared__ int s_m;
    const int q = blockIdx.x;
    if (q >= *n_stale)
        return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int n = min(*n_nodes, cap);
    const double gamma = *gamma_p;
    const int v = stale[q];
    for (int i = tid; i < kMitHash; i += blockDim.x)
        hs[i] = -1;
    __syncthreads();
    if (tid < ncnt[v]) {   // distinct ids: each is inserted once
        const int32_t w = nset[(int64_t)v * nbp + tid];
        for (int s = hash_slot(w);; s = (s + 1) & (kMitHash - 1))
            if (atomicCAS(&hs[s], -1, w) == -1)
                break;
    }
    __syncthreads();
    // this thread's best K candidates, sorted best first (sim 0 = empty)
    Cand top[kMitMaxK];
#pragma unroll
    for (int j = 0; j < kMitMaxK; ++j)
        top[j] = Cand{0, 0.0, 0, -1};
    for (int u = tid; u < n; u += blockDim.x) {
        if (!(dt[u] < gamma))
            continue;
        const int c = ncnt[u];
        int sim = 0;
        for (int j = 0; j < c; ++j)
            sim += hash_has(hs, nset[(int64_t)u * nbp + j]) ? 1 : 0;
        if (sim == 0)
            continue;
        Cand x{sim, mem_ts[u], nodes[u], u};
        // insertion into the sorted list: entries worse than x move down one
#pragma unroll
        for (int j = 0; j < kMitMaxK; ++j) {
            if (j < K && (top[j].sim == 0 || better(x, top[j]))) {
                const Cand y = top[j];
                top[j] = x;
                x = y;
            }
        }
    }
#pragma unroll
    for (int j = 0; j < kMitMaxK; ++j) {
        const int o = tid * kMitMaxK + j;
        c_sim[o] = j < K ? top[j].sim : 0;
        c_pos[o] = top[j].pos;
    }
    __syncthreads();
    if (tid < kWave) {
        // lane l merges the sorted lists of threads 4l .. 4l + 3 (heads h[i]);
        // each round the wave takes its best head
        int h[4] = {0, 0, 0, 0};
        int m = 0;
        for (int r = 0; r < K; ++r) {
            Cand best{0, 0.0, 0, -1};
            int bi = -1;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int o = (4 * lane + i) * kMitMaxK + h[i];
                if (h[i] < K && c_sim[o] > 0) {
                    const int32_t ps = c_pos[o];
                    const Cand x{c_sim[o], mem_ts[ps], nodes[ps], ps};
                    if (bi < 0 || better(x, best)) {
                        best = x;
                        bi = i;
                    }
                }
            }
            // wave arg-best: the winner is unique (ids are distinct)
            Cand wb = best;
            int wl = bi >= 0 ? lane : -1;
#pragma unroll
            for (int o = kWave / 2; o >= 1; o >>= 1) {
                Cand y;
                y.sim = __shfl_xor(wb.sim, o, kWave);
                y.mts = __shfl_xor(wb.mts, o, kWave);
                y.id = __shfl_xor(wb.id, o, kWave);
                y.pos = __shfl_xor(wb.pos, o, kWave);
                const int yl = __shfl_xor(wl, o, kWave);
                if (yl >= 0 && (wl < 0 || better(y, wb))) {
                    wb = y;
                    wl = yl;
                }
            }
            if (wl < 0)
                break;   // no candidate left anywhere (uniform)
            if (lane == wl)
                ++h[bi];
            if (lane == 0)
                r_pos[r] = wb.pos;
            m = r + 1;
        }
        if (lane == 0)
            s_m = m;
    }
    __syncthreads();
    const int m = s_m;
    if (omega && tid < K)
        omega[(int64_t)q * K + tid] = tid < m ? r_pos[tid] : -1;
    if (m > 0) {
        const float rest = 1.0f - lambda;
        for (int c = tid; c < M; c += blockDim.x) {
            float acc = 0.f;
            for (int j = 0; j < m; ++j)
                acc += mem[(int64_t)r_pos[j] * M + c];
            mem[(int64_t)v * M + c] = lambda * mem[(int64_t)v * M + c] + rest * (acc / (float)m);
        }
    }
}

}  // namespace

// ======================================================================== API

extern "C" tgm_status_t tgm_mitigator_create(int32_t max_nodes, int32_t nb, int32_t K,
                                             tgm_mitigator_t *out)
{
    if (!out)
        return TGM_EINVAL;
    *out = nullptr;
    if (max_nodes <= 0 || nb < 1 || nb > 64 || K < 1 || K > kMitMaxK)
        return TGM_EINVAL;
    tgm_mitigator *mt = new tgm_mitigator();
    mt->cap = max_nodes;
    mt->nb = nb;
    mt->nbp = round_up(nb, 4);
    mt->K = K;
    const size_t c = (size_t)max_nodes;
    if (hipMalloc((void **)&mt->dt, sizeof(double) * c) != hipSuccess ||
        hipMalloc((void **)&mt->nset, sizeof(int32_t) * c * mt->nbp) != hipSuccess ||
        hipMalloc((void **)&mt->ncnt, sizeof(int32_t) * c) != hipSuccess ||
        hipMalloc((void **)&mt->gamma, sizeof(double)) != hipSuccess ||
        hipMalloc((void **)&mt->n_stale, sizeof(int32_t)) != hipSuccess ||
        hipMalloc((void **)&mt->stale, sizeof(int32_t) * c) != hipSuccess ||
        hipMalloc((void **)&mt->omega, sizeof(int32_t) * c * K) != hipSuccess) {
        tgm_mitigator_destroy(mt);
        return TGM_ENOMEM;
    }
    *out = mt;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_mitigator_destroy(tgm_mitigator_t mt)
{
    if (!mt)
        return TGM_EINVAL;
    (void)hipFree(mt->dt);
    (void)hipFree(mt->nset);
    (void)hipFree(mt->ncnt);
    (void)hipFree(mt->gamma);
    (void)hipFree(mt->n_stale);
    (void)hipFree(mt->stale);
    (void)hipFree(mt->omega);
    delete mt;
    return TGM_OK;
}

tgm_status_t tgm::mitigate_launch(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                                  const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                                  float *mem, const double *mem_ts, int32_t M, double p,
                                  float lambda, hipStream_t s)
{
    if (!mt || !g || !nodes || !n_nodes || !mem || !mem_ts || M <= 0 || cap < 0)
        return TGM_EINVAL;
    if (!(p >= 0.0 && p <= 1.0) || !(lambda >= 0.0f && lambda <= 1.0f))
        return TGM_EINVAL;
    if (first_event < 0 || first_event >= g->E)
        return TGM_ERANGE;
    if (cap > mt->cap)
        return TGM_ESIZE;
    if (cap == 0)
        return TGM_OK;
    TGM_LAUNCH(k_mit_prep, dim3((unsigned)cdiv(cap, 4)), dim3(256), 0, s, g->off, g->adj, g->N,
               g->t, first_event, nodes, n_nodes, cap, mem_ts, mt->nb, mt->nbp, mt->dt,
               mt->nset, mt->ncnt);
    TGM_LAUNCH(k_mit_select, dim3(1), dim3(kMitSelThreads), 0, s, mt->dt, n_nodes, cap, p,
               mt->gamma, mt->stale, mt->n_stale);
    // at most n - ceil(p n) + 1 <= cap (1 - p) + 1 nodes are stale
    const int64_t grid = std::min<int64_t>(cap, (int64_t)std::floor(cap * (1.0 - p)) + 1);
    TGM_LAUNCH(k_mit_omega, dim3((unsigned)grid), dim3(kMitThreads), 0, s, nodes, n_nodes, cap,
               mt->dt, mem_ts, mt->nset, mt->ncnt, mt->nbp, mt->gamma, mt->stale, mt->n_stale,
               mt->K, lambda, mem, M, mt->omega);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_mitigate(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                                     const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                                     float *mem, const double *mem_ts, int32_t M, double p,
                                     float lambda, void *stream)
{
    return tgm::mitigate_launch(mt, g, first_event, nodes, n_nodes, cap, mem, mem_ts, M, p,
                                lambda, as_stream(stream));
}

extern "C" tgm_status_t tgm_mitigator_read(tgm_mitigator_t mt, double *gamma, int32_t *n_stale,
                                           int32_t *stale, int32_t *omega, void *stream)
{
    if (!mt)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t c = (size_t)mt->cap;
    if (gamma)
        TGM_HIP(hipMemcpyAsync(gamma, mt->gamma, sizeof(double), hipMemcpyDeviceToDevice, s));
    if (n_stale)
        TGM_HIP(hipMemcpyAsync(n_stale, mt->n_stale, sizeof(int32_t), hipMemcpyDeviceToDevice,
                               s));
    if (stale)
        TGM_HIP(hipMemcpyAsync(stale, mt->stale, sizeof(int32_t) * c, hipMemcpyDeviceToDevice, s));
    if (omega)
        TGM_HIP(hipMemcpyAsync(omega, mt->omega, sizeof(int32_t) * c * mt->K,
                               hipMemcpyDeviceToDevice, s));
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_set_mitigation(tgm_state_t st, tgm_mitigator_t mt, double p,
                                                 float lambda)
{
    if (!st || (mt && (!(p >= 0.0 && p <= 1.0) || !(lambda >= 0.0f && lambda <= 1.0f))))
        return TGM_EINVAL;
    st->mit = mt;
    st->mit_p = p;
    st->mit_lambda = lambda;
    return TGM_OK;
}
