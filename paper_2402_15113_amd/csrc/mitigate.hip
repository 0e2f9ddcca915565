// Similarity-based staleness mitigation (MSPipe-S, Sec. 3.3) of the fetched
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
// Three launches:
//   k_mit_prep    one wavefront per node: its sorted distinct neighbour set
//                 (padded with INT32_MAX).  It depends on the graph and the
//                 node set only, so the pipelined executor runs it on its
//                 sampling stream, into one slot per sample buffer set;
//   k_mit_select  one workgroup: gamma by a radix select over the
//                 order-preserving 64-bit keys of the gaps (held in
//                 registers, eight digit passes), then the stale positions
//                 in order;
//   k_mit_omega   work items (stale node, chunk of the node set) over a
//                 fixed grid: the stale node's neighbour set in an LDS hash
//                 set, every active node's set of the chunk probed against it,
//                 per-thread sorted lists merged into the top-K; with one
//                 chunk per node, Omega and the blend;
//   k_mit_final   with several chunks per node: each stale node's chunk
//                 lists merged into Omega, and the blend (the launch boundary
//                 orders the lists; no device-wide fence is needed).
// Integer decisions only; each gap is formed where it is used, by the one fp64
// subtraction the oracle makes.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.h"

using namespace tgm;

struct tgm_mitigator {
    int32_t cap = 0, nb = 0, nbp = 0, K = 0;
    int32_t nslots = 0;          // neighbour-set slots (0: tgm_mitigate; 1..: the executor's)
    int32_t *nset = nullptr;     // [nslots x cap x nbp] sorted distinct neighbour ids
    int32_t *ncnt = nullptr;     // [nslots x cap]
    double *gamma = nullptr;     // [1]
    int32_t *n_stale = nullptr;  // [1]
    int32_t *stale = nullptr;    // [cap] stale positions, ascending
    int32_t *omega = nullptr;    // [cap x K] Omega positions, -1 padded
    int2 *part = nullptr;        // [kMitOmegaGrid x kMitMaxK] chunk top-K lists of k_mit_omega
};

namespace {

constexpr int kMitMaxK = 16;
constexpr int kMitThreads = 256;           // k_mit_omega
constexpr int kMitSelThreads = 1024;       // k_mit_select
constexpr int kMitSelRegs = 20;            // gaps per k_mit_select thread in registers
constexpr int kMitHashBits = 10;
constexpr int kMitHash = 1 << kMitHashBits;   // LDS hash slots (16 per possible id)
constexpr int kMitPerThread = 4;           // nodes a k_mit_omega thread takes per round
constexpr int kMitChunk = 1024;             // nodes of one k_mit_omega round (256 x 4)
constexpr int kMitMaxChunks = 64;           // chunk lists of one stale node (64 x 16 entries)
static_assert(kMitChunk == kMitThreads * kMitPerThread, "a round is one node per thread slot");
static_assert(kMitMaxChunks * kMitMaxK <= kMitChunk, "the chunk lists fit the round entries");
constexpr int kMitOmegaGrid = 1024;         // k_mit_omega workgroups

constexpr int kMitMaxNodes = 1 << 20;
static_assert(TGM_MITIGATE_NOALLOC_MAX_NODES * (64 + 1 + 1 + 16) * 4 +
                  kMitOmegaGrid * kMitMaxK * 8 + 8 * 256 <= TGM_MITIGATE_NOALLOC_BYTES,
              "the no-allocation work space fits its largest call");

// ---------------------------------------------------------------- prep
// One wavefront per fetched node: its sorted distinct neighbour set before T,
// the time of event `first`.  Lane j < c holds the j-th most recent
// neighbour; duplicates and ranks come from a loop over the c lanes with
// readlane (c <= nb <= 64).
__global__ __launch_bounds__(256) void k_mit_prep(const int64_t *__restrict__ off,
                                                  const AdjRec *__restrict__ adj,
                                                  const double *__restrict__ tix, int32_t N,
                                                  const double *__restrict__ t, int64_t first,
                                                  const int32_t *__restrict__ nodes,
                                                  const int32_t *__restrict__ n_nodes,
                                                  int32_t cap, int32_t nb, int32_t nbp,
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
    const int64_t end = recent_end(off, adj, tix, v, T, N, &base);
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
    const int d = __popcll(__ballot(lane < c && !dup));
    if (lane >= d && lane < nbp)
        nset[(int64_t)p * nbp + lane] = INT32_MAX;   // padding: never an id
    if (lane == 0)
        ncnt[p] = d;
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

// Inclusive prefix sum over the 64 lanes of a wavefront: shifts by 1, 2, 4
// and 8 within each row of 16 lanes, then row 0's total into row 1 and row
// 2's into row 3 (row_bcast:15), then rows 0-1's total into rows 2 and 3
// (row_bcast:31).  Lanes without a source add 0.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v)
{
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);
    return v;
}

// Adds the keys of this round (one per thread; `in` marks those that count)
// to the histogram of the digit (k >> sh) & dmask.  The bins of the wave's
// first two remaining lanes take one atomic each (the leading digits of gaps
// are few); the rest one per lane.
__device__ __forceinline__ void hist_add(uint32_t *hist, uint64_t k, bool in, int sh,
                                         uint32_t dmask)
{
    const int lane = threadIdx.x & 63;
    const int bin = (int)((k >> sh) & dmask);
    uint64_t act = __ballot(in);
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        if (act == 0)
            break;
        const int lead = __builtin_ctzll(act);
        const int first = __builtin_amdgcn_readlane(bin, lead);
        const uint64_t same = __ballot(in && bin == first);
        if (lane == lead)
            atomicAdd(&hist[first], (uint32_t)__popcll(same));
        in = in && bin != first;
        act &= ~same;
    }
    if (in)
        atomicAdd(&hist[bin], 1u);
}

// One workgroup: gamma = the rank-th smallest gap (rank = ceil(pq n) in fp64,
// clamped to [1, n]) by a radix select over the order-preserving 64-bit keys
// of the gaps, most significant byte first (eight passes).  The keys stay in
// registers (kMitSelRegs per thread; read again from global memory each pass
// when n is larger).  A pass adds the digits of the keys that match the
// prefix found so far to a 256-bin LDS histogram; after one barrier every
// wave reads the whole histogram (four bins a lane), scans the lane sums with
// DPP and finds the bin that holds the rank, so no second barrier is needed.
// Three histogram buffers rotate: the one a pass clears was last read two
// passes before, by waves that have all passed the barrier since.  Then the
// positions with dt > gamma, ascending.
__global__ __launch_bounds__(kMitSelThreads) void k_mit_select(
    const double *__restrict__ t, int64_t first, const double *__restrict__ mem_ts,
    const int32_t *__restrict__ n_nodes, int32_t cap, double pq, double *__restrict__ gamma_out,
    int32_t *__restrict__ stale, int32_t *__restrict__ n_stale)
{
    constexpr int R = kMitSelRegs;
    constexpr int T = kMitSelThreads;
    __shared__ __align__(16) uint32_t hist[3][256];
    __shared__ int s_wsum[2][T / kWave];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = min(*n_nodes, cap);
    if (n <= 0) {
        if (tid == 0) {
            *n_stale = 0;
            *gamma_out = 0.0;
        }
        return;
    }
    const double T0 = t[first];
    auto gap = [&](int i) { return T0 - mem_ts[i]; };
    const bool in_regs = n <= R * T;
    const int rounds = (n + T - 1) / T;
    uint64_t kr[R];   // this thread's keys tid + j T (when in_regs)
    if (in_regs) {
        // every load issued before the first use; indices clamped to the
        // buffer (cap), not to n, so they need not wait for the count (mem_ts
        // holds cap entries)
        double x[R];
#pragma unroll
        for (int j = 0; j < R; ++j)
            x[j] = mem_ts[min(tid + j * T, cap - 1)];
#pragma unroll
        for (int j = 0; j < R; ++j)
            kr[j] = order_key(T0 - x[j]);
    }
    if (tid < 256)
        hist[0][tid] = 0;
    long long rank = (long long)ceil(pq * (double)n);
    rank = rank < 1 ? 1 : (rank > n ? n : rank);
    {
        // gamma is the largest gap when at least n - rank + 1 gaps equal it;
        // then no gap exceeds it and nothing is stale (two barriers instead
        // of the eight passes)
        uint64_t km = 0;
        if (in_regs) {
#pragma unroll
            for (int j = 0; j < R; ++j)
                if (j < rounds && tid + j * T < n)
                    km = kr[j] > km ? kr[j] : km;
        } else {
            for (int i = tid; i < n; i += T) {
                const uint64_t k = order_key(gap(i));
                km = k > km ? k : km;
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const uint64_t y = (uint64_t)__shfl_xor((long long)km, o, kWave);
            km = y > km ? y : km;
        }
        __shared__ uint64_t s_km[T / kWave];
        __shared__ int s_kc[T / kWave];
        if (lane == 0)
            s_km[wave] = km;
        __syncthreads();
        for (int w = 0; w < T / kWave; ++w)
            km = s_km[w] > km ? s_km[w] : km;
        int cnt = 0;
        if (in_regs) {
#pragma unroll
            for (int j = 0; j < R; ++j)
                if (j < rounds)
                    cnt += __popcll(__ballot(tid + j * T < n && kr[j] == km));
        } else {
            for (int b0 = 0; b0 < n; b0 += T) {   // whole waves per round
                const int i = b0 + tid;
                cnt += __popcll(__ballot(i < n && order_key(gap(min(i, n - 1))) == km));
            }
        }
        if (lane == 0)
            s_kc[wave] = cnt;
        __syncthreads();
        int total = 0;
        for (int w = 0; w < T / kWave; ++w)
            total += s_kc[w];
        if ((long long)total >= (long long)n - rank + 1) {   // uniform
            if (tid == 0) {
                *n_stale = 0;
                *gamma_out = key_value(km);
            }
            return;
        }
    }
    uint32_t krem = (uint32_t)(rank - 1);   // keys below the target among those matching
    uint64_t prefix = 0, mask = 0;
    for (int pass = 0; pass < 8; ++pass) {
        const int sh = 56 - 8 * pass;
        uint32_t *H = hist[pass % 3];
        if (tid < 256)
            hist[(pass + 1) % 3][tid] = 0;   // the next pass's buffer
        if (pass == 0)
            __syncthreads();   // hist[0] is clear
        if (in_regs) {
#pragma unroll
            for (int j = 0; j < R; ++j) {
                if (j < rounds)   // uniform
                    hist_add(H, kr[j], tid + j * T < n && (kr[j] & mask) == prefix, sh, 255u);
            }
        } else {
            for (int b0 = 0; b0 < n; b0 += T) {   // whole waves per round
                const int i = b0 + tid;
                const uint64_t k = i < n ? order_key(gap(i)) : 0;
                hist_add(H, k, i < n && (k & mask) == prefix, sh, 255u);
            }
        }
        __syncthreads();
        // every wave: lane l holds bins 4l .. 4l + 3
        const uint4 c = reinterpret_cast<const uint4 *>(H)[lane];
        const uint32_t a0 = c.x, a1 = a0 + c.y, a2 = a1 + c.z, sum = a2 + c.w;
        const uint32_t incl = wave_incl_scan(sum);
        const uint32_t excl = incl - sum;
        // the one lane whose bins hold the rank
        const int L = __builtin_ctzll(__ballot(excl <= krem && krem < incl));
        const uint32_t r = krem - excl;   // meaningful on lane L
        const uint32_t j = (r >= a0 ? 1u : 0u) + (r >= a1 ? 1u : 0u) + (r >= a2 ? 1u : 0u);
        const uint32_t below = excl + (j == 0 ? 0u : (j == 1 ? a0 : (j == 2 ? a1 : a2)));
        const uint32_t bin = (uint32_t)__builtin_amdgcn_readlane((int)(4 * lane + j), L);
        krem -= (uint32_t)__builtin_amdgcn_readlane((int)below, L);
        prefix |= (uint64_t)bin << sh;
        mask |= 255ull << sh;
    }
    // stale positions in order (key > prefix  <=>  dt > gamma); the wave
    // counts alternate between two buffers, one barrier a round
    int base = 0;
    for (int j = 0; j < rounds; ++j) {
        const int i = tid + j * T;
        uint64_t k = 0;
        if (in_regs) {
#pragma unroll
            for (int jj = 0; jj < R; ++jj)
                k = jj == j ? kr[jj] : k;
        } else {
            k = order_key(gap(min(i, n - 1)));
        }
        const bool f = i < n && k > prefix;
        const uint64_t bal = __ballot(f);
        const int in_wave = __popcll(bal & ((1ull << lane) - 1));
        int *ws = s_wsum[j & 1];
        if (lane == 0)
            ws[wave] = __popcll(bal);
        __syncthreads();
        int before = 0, total = 0;
        for (int w = 0; w < T / kWave; ++w) {
            before += w < wave ? ws[w] : 0;
            total += ws[w];
        }
        if (f)
            stale[base + before + in_wave] = i;
        base += total;
    }
    if (tid == 0) {
        *n_stale = base;
        *gamma_out = key_value(prefix);
    }
}

// ---------------------------------------------------------------- omega
struct Cand {
    int sim;
    double mts;
    int32_t id, pos;
};

// more common neighbours, then the fresher memory, then the smaller id.  An
// empty entry (similarity 0) loses to every candidate, so no separate "first
// candidate" test is needed: the comparisons below use `better` alone (with a
// short-circuit first-candidate test, the compiler kept the old position
// while taking the other fields of a new best).
__device__ __forceinline__ bool better(const Cand &a, const Cand &b)
{
    if (a.sim != b.sim)
        return a.sim > b.sim;
    if (a.mts != b.mts)
        return a.mts > b.mts;
    return a.id < b.id;
}

__device__ __forceinline__ int hash_slot(int32_t w)
{
    return (int)(((uint32_t)w * 2654435761u) >> (32 - kMitHashBits));
}

// Whether w (not in slot `from - 1`) is further along its probe sequence.
__device__ __forceinline__ int hash_walk(const int32_t *hs, int32_t w, int from)
{
    for (int k = 1, s = from; k < kMitHash; ++k, s = (s + 1) & (kMitHash - 1)) {
        const int32_t x = hs[s];
        if (x == w)
            return 1;
        if (x < 0)
            return 0;
    }
    return 0;
}

// One step of the wave arg-best: the candidate that DPP control CTRL brings
// in (rows ROWS only; a lane with no source sees its own) replaces the lane's
// when better.
template <int CTRL, int ROWS>
__device__ __forceinline__ void best_step(Cand &b, int &bl)
{
    const long long m = __double_as_longlong(b.mts);
    const int mlo = (int)m, mhi = (int)(m >> 32);
    Cand y;
    y.sim = __builtin_amdgcn_update_dpp(b.sim, b.sim, CTRL, ROWS, 0xF, false);
    const int lo = __builtin_amdgcn_update_dpp(mlo, mlo, CTRL, ROWS, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(mhi, mhi, CTRL, ROWS, 0xF, false);
    y.mts = __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
    y.id = __builtin_amdgcn_update_dpp(b.id, b.id, CTRL, ROWS, 0xF, false);
    y.pos = __builtin_amdgcn_update_dpp(b.pos, b.pos, CTRL, ROWS, 0xF, false);
    const int yl = __builtin_amdgcn_update_dpp(bl, bl, CTRL, ROWS, 0xF, false);
    if (better(y, b)) {
        b = y;
        bl = yl;
    }
}

// The wave's best candidate and its lane, on every lane: a running best
// within each row of 16 lanes (shifts by 1, 2, 4, 8), the rows joined into
// lane 63 by the two row broadcasts, then read from lane 63.
__device__ __forceinline__ void wave_best(Cand &b, int &bl)
{
    best_step<0x111, 0xF>(b, bl);
    best_step<0x112, 0xF>(b, bl);
    best_step<0x114, 0xF>(b, bl);
    best_step<0x118, 0xF>(b, bl);
    best_step<0x142, 0xA>(b, bl);
    best_step<0x143, 0xC>(b, bl);
    const long long m = __double_as_longlong(b.mts);
    const int lo = __builtin_amdgcn_readlane((int)m, 63);
    const int hi = __builtin_amdgcn_readlane((int)(m >> 32), 63);
    b.mts = __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
    b.sim = __builtin_amdgcn_readlane(b.sim, 63);
    b.id = __builtin_amdgcn_readlane(b.id, 63);
    b.pos = __builtin_amdgcn_readlane(b.pos, 63);
    bl = __builtin_amdgcn_readlane(bl, 63);
}

// Candidate lists in LDS: entry arrays of similarity (0 = end of a list),
// memory time, id and position.
struct Lists {
    int *sim;
    double *mts;
    int32_t *id, *pos;
};

// Wave 0 merges nl sorted lists of the entry arrays (entry h of list l at
// l * ls + h * es, at most len entries) and one more list at `xb` of xl
// entries into the best K.  Returns their count m on every lane; lane j < m
// holds the j-th in *mine.  Lane i owns lists i, i + 64, i + 128 and i + 192
// (nl <= 256), so the heads of neighbouring lanes sit side by side when the
// lists are interleaved (es = the list count); lane 63 also owns the extra
// list.  Each lane keeps its five heads in registers; each round the wave
// takes its best head with the DPP arg-best, and only the winning lane reads
// the next entry of that list.
__device__ int merge_lists(const Lists &L, int nl, int ls, int es, int len, int xb, int xl, int K,
                           Cand *mine)
{
    const int lane = threadIdx.x & 63;
    int h[5] = {0, 0, 0, 0, 0};
    Cand hd[5];
    // entry h[i] of owned list i, or an empty entry (similarity 0)
    auto head = [&](int i) {
        const int l = lane + kWave * i;
        const bool own = i < 4 ? (l < nl && h[i] < len) : (lane == 63 && h[4] < xl);
        const int o = i < 4 ? l * ls + h[i] * es : xb + h[4];
        Cand x{0, 0.0, 0, -1};
        if (own && L.sim[o] > 0)
            x = Cand{L.sim[o], L.mts[o], L.id[o], L.pos[o]};
        return x;
    };
#pragma unroll
    for (int i = 0; i < 5; ++i)
        hd[i] = head(i);
    int m = 0;
    for (int r = 0; r < K; ++r) {
        Cand best = hd[0];
        int bi = 0;
#pragma unroll
        for (int i = 1; i < 5; ++i)
            if (better(hd[i], best)) {   // empties lose
                best = hd[i];
                bi = i;
            }
        // the winner is unique (positions are distinct)
        Cand wb = best;
        int wl = best.sim > 0 ? lane : -1;
        wave_best(wb, wl);   // an empty lane's entry has similarity 0
        if (wl < 0)
            break;   // no candidate left anywhere (uniform)
        if (lane == wl) {
#pragma unroll
            for (int i = 0; i < 5; ++i)
                if (i == bi) {
                    ++h[i];
                    hd[i] = head(i);
                }
        }
        if (lane == r)
            *mine = wb;
        m = r + 1;
    }
    return m;
}

// Work items (stale node q, chunk c of the node set), q-major, strided over a
// fixed grid.  An item probes the neighbour set of every active node of its
// chunk against the stale node's (an LDS hash set), 1024 nodes at a time
// (kMitPerThread per thread, each thread keeping its best few sorted), and
// merges the thread lists into a running top-K.  With one chunk that is
// Omega, which the workgroup writes and blends; otherwise the chunk lists go
// to `part` for k_mit_final.  No workgroup waits for another.
template <int NBP>   // padded neighbour-set width: 4 (nb <= 4), 12 (<= 12) or 64
__global__ __launch_bounds__(kMitThreads) void k_mit_omega(
    const int32_t *__restrict__ nodes, const int32_t *__restrict__ n_nodes, int32_t cap,
    const double *__restrict__ t, int64_t first, const double *__restrict__ mem_ts,
    const int32_t *__restrict__ nset, const int32_t *__restrict__ ncnt,
    const double *__restrict__ gamma_p, const int32_t *__restrict__ stale,
    const int32_t *__restrict__ n_stale, int2 *__restrict__ part, int32_t K, float lambda,
    float *__restrict__ mem, int32_t M, int32_t *__restrict__ omega)
{
    typedef int __attribute__((ext_vector_type(4))) i4;
    constexpr int P = kMitPerThread;
    constexpr int U = NBP > 16 ? 1 : P;   // nodes in flight per thread
    constexpr int kSub = kMitThreads * P;  // nodes per round
    // entries: [0, kSub) thread lists (P each), then the running list
    constexpr int kE = kSub + kMitMaxK;
    __shared__ int32_t hs[kMitHash];
    __shared__ int e_sim[kE];
    __shared__ double e_mts[kE];
    __shared__ int32_t e_id[kE], e_pos[kE];
    __shared__ int s_m;
    const Lists L{e_sim, e_mts, e_id, e_pos};
    const int RB = kSub;   // the running list
    const int tid = threadIdx.x;
    const int n = min(*n_nodes, cap);
    const int ns = *n_stale;
    // chunks per stale node: one per 1024-node round, at most kMitMaxChunks,
    // and no more items than kMitOmegaGrid unless every stale node is one item
    const int nsub = (n + kSub - 1) / kSub;
    int nce = min(min(nsub, kMitMaxChunks), max(1, kMitOmegaGrid / max(ns, 1)));
    const int chunk = (nsub + nce - 1) / nce * kSub;
    nce = (n + chunk - 1) / chunk;   // chunks that hold nodes
    const int items = ns * nce;
    const double gamma = *gamma_p;
    const double T0 = t[first];
    const int KP = K < P ? K : P;   // per-thread list length
    for (int item = blockIdx.x; item < items; item += gridDim.x) {
        const int q = item / nce, c = item % nce;
        const int v = stale[q];
        for (int i = tid; i < kMitHash; i += blockDim.x)
            hs[i] = -1;
        if (tid == 0)
            s_m = 0;
        __syncthreads();
        if (tid < ncnt[v]) {   // distinct ids: each is inserted once
            const int32_t w = nset[(int64_t)v * NBP + tid];
            for (int sl = hash_slot(w);; sl = (sl + 1) & (kMitHash - 1))
                if (atomicCAS(&hs[sl], -1, w) == -1)
                    break;
        }
        __syncthreads();
        const int lo = c * chunk, hi = min(n, lo + chunk);
        for (int sub = lo; sub < hi; sub += kSub) {
            // this thread's best candidates among its P nodes, best first
            Cand top[P];
#pragma unroll
            for (int j = 0; j < P; ++j)
                top[j] = Cand{0, 0.0, 0, -1};
#pragma unroll
            for (int x0 = 0; x0 < P; x0 += U) {
                i4 row[U][NBP / 4];
                double g[U];
#pragma unroll
                for (int x = 0; x < U; ++x) {
                    const int u = min(sub + tid + (x0 + x) * kMitThreads, hi - 1);   // in range
                    g[x] = T0 - mem_ts[u];   // the gap
#pragma unroll
                    for (int e = 0; e < NBP / 4; ++e)
                        row[x][e] = reinterpret_cast<const i4 *>(nset + (int64_t)u * NBP)[e];
                }
#pragma unroll
                for (int x = 0; x < U; ++x) {
                    const int u = sub + tid + (x0 + x) * kMitThreads;
                    // first probes of every id together; one that meets another
                    // id walks on (rare: at most 64 of kMitHash slots are taken)
                    int32_t y[NBP];
#pragma unroll
                    for (int e = 0; e < NBP; ++e)
                        y[e] = hs[hash_slot(row[x][e / 4][e % 4])];
                    int sim = 0;
#pragma unroll
                    for (int e = 0; e < NBP; ++e) {
                        const int32_t w = row[x][e / 4][e % 4];
                        if (w != INT32_MAX) {
                            if (y[e] == w)
                                ++sim;
                            else if (y[e] >= 0)
                                sim += hash_walk(hs, w, (hash_slot(w) + 1) & (kMitHash - 1));
                        }
                    }
                    // active nodes only (v is not); a common neighbour at least
                    if (u >= hi || !(g[x] < gamma) || sim == 0)
                        continue;
                    Cand z{sim, mem_ts[u], nodes[u], u};
#pragma unroll
                    for (int j = 0; j < P; ++j) {   // sorted insertion
                        if (j < KP && better(z, top[j])) {   // empties lose
                            const Cand t = top[j];
                            top[j] = z;
                            z = t;
                        }
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < P; ++j) {
                const int o = j * kMitThreads + tid;   // entry j of every list together
                e_sim[o] = j < KP ? top[j].sim : 0;
                e_mts[o] = top[j].mts;
                e_id[o] = top[j].id;
                e_pos[o] = top[j].pos;
            }
            __syncthreads();
            if (tid < kWave) {   // the new running list, written after the merge's reads
                Cand w;
                const int m = merge_lists(L, kMitThreads, 1, kMitThreads, P, RB, s_m, K, &w);
                if (tid < m) {
                    e_sim[RB + tid] = w.sim;
                    e_mts[RB + tid] = w.mts;
                    e_id[RB + tid] = w.id;
                    e_pos[RB + tid] = w.pos;
                }
                if (tid == 0)
                    s_m = m;
            }
            __syncthreads();
        }
        if (nce > 1) {   // the chunk's list, for k_mit_final
            int2 *mine = part + ((int64_t)q * nce + c) * K;   // q nce < kMitOmegaGrid
            if (tid < K)
                mine[tid] = tid < s_m ? make_int2(e_sim[RB + tid], e_pos[RB + tid])
                                      : make_int2(0, -1);
            __syncthreads();   // s_m is reused
            continue;
        }
        const int m = s_m;
        if (omega && tid < K)
            omega[(int64_t)q * K + tid] = tid < m ? e_pos[RB + tid] : -1;
        if (m > 0) {
            const float rest = 1.0f - lambda;
            for (int cc = tid; cc < M; cc += blockDim.x) {
                float acc = 0.f;
                for (int j = 0; j < m; ++j)
                    acc += mem[(int64_t)e_pos[RB + j] * M + cc];
                mem[(int64_t)v * M + cc] =
                    lambda * mem[(int64_t)v * M + cc] + rest * (acc / (float)m);
            }
        }
        __syncthreads();   // the entries and s_m are reused
    }
}

}  // namespace

// ======================================================================== API

namespace {


}  // namespace

extern "C" tgm_status_t tgm_mitigator_create(int32_t max_nodes, int32_t nb, int32_t K,
                                             tgm_mitigator_t *out)
{
    if (!out)
        return TGM_EINVAL;
    *out = nullptr;
    if (max_nodes <= 0 || max_nodes > kMitMaxNodes || nb < 1 || nb > 64 || K < 1 || K > kMitMaxK)
        return TGM_EINVAL;
    tgm_mitigator *mt = new tgm_mitigator();
    mt->cap = max_nodes;
    mt->nb = nb;
    mt->nbp = nb <= 4 ? 4 : (nb <= 12 ? 12 : 64);   // the widths k_mit_omega reads
    mt->K = K;
    const size_t c = (size_t)max_nodes;
    if (dev_malloc((void **)&mt->gamma, sizeof(double)) != hipSuccess ||
        dev_malloc((void **)&mt->n_stale, sizeof(int32_t)) != hipSuccess ||
        dev_malloc((void **)&mt->stale, sizeof(int32_t) * c) != hipSuccess ||
        dev_malloc((void **)&mt->omega, sizeof(int32_t) * c * K) != hipSuccess ||
        dev_malloc((void **)&mt->part, sizeof(int2) * kMitOmegaGrid * kMitMaxK) != hipSuccess ||
        tgm::mitigate_reserve(mt, 1) != TGM_OK) {
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
    (void)hipFree(mt->nset);
    (void)hipFree(mt->ncnt);
    (void)hipFree(mt->gamma);
    (void)hipFree(mt->n_stale);
    (void)hipFree(mt->stale);
    (void)hipFree(mt->omega);
    (void)hipFree(mt->part);
    delete mt;
    return TGM_OK;
}

int32_t tgm::mitigate_slots(tgm_mitigator_t mt) { return mt ? mt->nslots : 0; }

tgm_status_t tgm::mitigate_reserve(tgm_mitigator_t mt, int32_t nslots)
{
    if (!mt || nslots < 1)
        return TGM_EINVAL;
    if (nslots <= mt->nslots)
        return TGM_OK;
    // the sets of earlier calls need not survive: a run fills its slots first
    if (mt->nslots > 0 && hipDeviceSynchronize() != hipSuccess)
        return TGM_EDEVICE;
    (void)hipFree(mt->nset);
    (void)hipFree(mt->ncnt);
    mt->nset = nullptr;
    mt->ncnt = nullptr;
    mt->nslots = 0;
    const size_t c = (size_t)mt->cap * nslots;
    if (dev_malloc((void **)&mt->nset, sizeof(int32_t) * c * mt->nbp) != hipSuccess ||
        dev_malloc((void **)&mt->ncnt, sizeof(int32_t) * c) != hipSuccess)
        return TGM_ENOMEM;
    mt->nslots = nslots;
    return TGM_OK;
}

namespace {

// Stale nodes q, strided over the grid, when k_mit_omega split each one's
// node set over several chunks (the same nce as there): the nce chunk lists
// of q merged into Omega (wave 0), written, and the blend.
__global__ __launch_bounds__(kMitThreads) void k_mit_final(
    const int32_t *__restrict__ nodes, const int32_t *__restrict__ n_nodes, int32_t cap,
    const double *__restrict__ mem_ts, const int32_t *__restrict__ stale,
    const int32_t *__restrict__ n_stale, const int2 *__restrict__ part, int32_t K, float lambda,
    float *__restrict__ mem, int32_t M, int32_t *__restrict__ omega)
{
    constexpr int kE = kMitMaxChunks * kMitMaxK;
    __shared__ int e_sim[kE];
    __shared__ double e_mts[kE];
    __shared__ int32_t e_id[kE], e_pos[kE];
    __shared__ int32_t s_pos[kMitMaxK];
    __shared__ int s_m;
    const Lists L{e_sim, e_mts, e_id, e_pos};
    const int tid = threadIdx.x;
    const int n = min(*n_nodes, cap);
    const int ns = *n_stale;
    constexpr int kSub = kMitThreads * kMitPerThread;
    const int nsub = (n + kSub - 1) / kSub;
    int nce = min(min(nsub, kMitMaxChunks), max(1, kMitOmegaGrid / max(ns, 1)));
    const int chunk = (nsub + nce - 1) / nce * kSub;
    nce = (n + chunk - 1) / chunk;
    if (nce <= 1)
        return;   // k_mit_omega finished every stale node (uniform)
    for (int q = blockIdx.x; q < ns; q += gridDim.x) {
        for (int i = tid; i < nce * K; i += blockDim.x) {
            const int2 e = part[(int64_t)q * nce * K + i];
            const int ps = e.y < 0 ? 0 : e.y;
            e_sim[i] = e.x;
            e_mts[i] = mem_ts[ps];
            e_id[i] = nodes[ps];
            e_pos[i] = e.y;
        }
        __syncthreads();
        if (tid < kWave) {
            Cand w;
            const int m = merge_lists(L, nce, K, 1, K, 0, 0, K, &w);
            if (tid < m)
                s_pos[tid] = w.pos;
            if (tid == 0)
                s_m = m;
        }
        __syncthreads();
        const int m = s_m;
        if (omega && tid < K)
            omega[(int64_t)q * K + tid] = tid < m ? s_pos[tid] : -1;
        if (m > 0) {
            const int v = stale[q];
            const float rest = 1.0f - lambda;
            for (int cc = tid; cc < M; cc += blockDim.x) {
                float acc = 0.f;
                for (int j = 0; j < m; ++j)
                    acc += mem[(int64_t)s_pos[j] * M + cc];
                mem[(int64_t)v * M + cc] =
                    lambda * mem[(int64_t)v * M + cc] + rest * (acc / (float)m);
            }
        }
        __syncthreads();   // the entries and s_m are reused
    }
}

// The work space one mitigation reads and writes: a mitigator's (one of its
// neighbour-set slots), or the fixed per-device array of
// tgm_mitigate_noalloc.
struct MitWork {
    int32_t nb = 0, nbp = 0, K = 0;
    int32_t *nset = nullptr, *ncnt = nullptr;   // [cap x nbp], [cap]
    double *gamma = nullptr;
    int32_t *n_stale = nullptr, *stale = nullptr, *omega = nullptr;
    int2 *part = nullptr;
};

MitWork work_of(const tgm_mitigator *mt, int32_t slot)
{
    MitWork w;
    const int64_t o = (int64_t)slot * mt->cap;
    w.nb = mt->nb;
    w.nbp = mt->nbp;
    w.K = mt->K;
    w.nset = mt->nset + o * mt->nbp;
    w.ncnt = mt->ncnt + o;
    w.gamma = mt->gamma;
    w.n_stale = mt->n_stale;
    w.stale = mt->stale;
    w.omega = mt->omega;
    w.part = mt->part;
    return w;
}

tgm_status_t prep_launch(const MitWork &w, tgm_graph_t g, int64_t first_event,
                         const int32_t *nodes, const int32_t *n_nodes, int32_t cap, hipStream_t s)
{
    if (cap == 0)
        return TGM_OK;
    TGM_LAUNCH(k_mit_prep, dim3((unsigned)cdiv(cap, 4)), dim3(256), 0, s, g->off, g->adj, g->tix, g->N,
               g->t, first_event, nodes, n_nodes, cap, w.nb, w.nbp, w.nset, w.ncnt);
    return TGM_OK;
}

tgm_status_t blend_launch(const MitWork &w, tgm_graph_t g, int64_t first_event,
                          const int32_t *nodes, const int32_t *n_nodes, int32_t cap, float *mem,
                          const double *mem_ts, int32_t M, double p, float lambda, hipStream_t s)
{
    if (cap == 0)
        return TGM_OK;
    TGM_LAUNCH(k_mit_select, dim3(1), dim3(kMitSelThreads), 0, s, g->t, first_event, mem_ts,
               n_nodes, cap, p, w.gamma, w.stale, w.n_stale);
    // at most n - ceil(p n) + 1 <= cap (1 - p) + 1 nodes are stale, each in
    // at most ceil(cap / kMitChunk) items; a fixed grid strides over the items
    const int64_t slots = std::min<int64_t>(cap, (int64_t)std::floor(cap * (1.0 - p)) + 1);
    const dim3 grid((unsigned)std::min<int64_t>(slots * cdiv(cap, kMitChunk), kMitOmegaGrid));
    if (w.nbp == 4)
        TGM_LAUNCH(k_mit_omega<4>, grid, dim3(kMitThreads), 0, s, nodes, n_nodes, cap, g->t,
                   first_event, mem_ts, w.nset, w.ncnt, w.gamma, w.stale, w.n_stale, w.part,
                   w.K, lambda, mem, M, w.omega);
    else if (w.nbp == 12)
        TGM_LAUNCH(k_mit_omega<12>, grid, dim3(kMitThreads), 0, s, nodes, n_nodes, cap, g->t,
                   first_event, mem_ts, w.nset, w.ncnt, w.gamma, w.stale, w.n_stale, w.part,
                   w.K, lambda, mem, M, w.omega);
    else
        TGM_LAUNCH(k_mit_omega<64>, grid, dim3(kMitThreads), 0, s, nodes, n_nodes, cap, g->t,
                   first_event, mem_ts, w.nset, w.ncnt, w.gamma, w.stale, w.n_stale, w.part,
                   w.K, lambda, mem, M, w.omega);
    // the stale nodes whose node set k_mit_omega split over several chunks
    TGM_LAUNCH(k_mit_final, dim3((unsigned)std::min<int64_t>(slots, kMitOmegaGrid)),
               dim3(kMitThreads), 0, s, nodes, n_nodes, cap, mem_ts, w.stale, w.n_stale, w.part,
               w.K, lambda, mem, M, w.omega);
    return TGM_OK;
}

}  // namespace

tgm_status_t tgm::mitigate_prep_launch(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                                       const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                                       int32_t slot, hipStream_t s)
{
    if (!mt || !g || !nodes || !n_nodes || cap < 0 || slot < 0 || slot >= mt->nslots)
        return TGM_EINVAL;
    if (first_event < 0 || first_event >= g->E)
        return TGM_ERANGE;
    if (cap > mt->cap)
        return TGM_ESIZE;
    return prep_launch(work_of(mt, slot), g, first_event, nodes, n_nodes, cap, s);
}

tgm_status_t tgm::mitigate_launch(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                                  const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                                  float *mem, const double *mem_ts, int32_t M, double p,
                                  float lambda, int32_t slot, hipStream_t s)
{
    if (!mt || !g || !nodes || !n_nodes || !mem || !mem_ts || M <= 0 || cap < 0 || slot < 0 ||
        slot >= mt->nslots)
        return TGM_EINVAL;
    if (!(p >= 0.0 && p <= 1.0) || !(lambda >= 0.0f && lambda <= 1.0f))
        return TGM_EINVAL;
    if (first_event < 0 || first_event >= g->E)
        return TGM_ERANGE;
    if (cap > mt->cap)
        return TGM_ESIZE;
    return blend_launch(work_of(mt, slot), g, first_event, nodes, n_nodes, cap, mem, mem_ts, M,
                        p, lambda, s);
}

extern "C" tgm_status_t tgm_mitigate(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                                     const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                                     float *mem, const double *mem_ts, int32_t M, double p,
                                     float lambda, void *stream)
{
    // slot 0: the neighbour sets of this call
    if (!mem || !mem_ts || M <= 0)
        return TGM_EINVAL;
    if (!(p >= 0.0 && p <= 1.0) || !(lambda >= 0.0f && lambda <= 1.0f))
        return TGM_EINVAL;
    TGM_TRY_STATUS(tgm::mitigate_prep_launch(mt, g, first_event, nodes, n_nodes, cap, 0,
                                             as_stream(stream)));
    return tgm::mitigate_launch(mt, g, first_event, nodes, n_nodes, cap, mem, mem_ts, M, p,
                                lambda, 0, as_stream(stream));
}

// ------------------------------------------------- the allocation-free variant
// tgm_mitigate_noalloc keeps its work space in this array.  Each GPU the
// library runs on holds its own copy until the process ends.  Host code never
// passes the array's name to a kernel or a copy (on the host it is a stand-in,
// not a device address): it looks up each device's address once, with that
// device current, and uses that.
namespace {

constexpr int32_t kNoallocMaxNodes = TGM_MITIGATE_NOALLOC_MAX_NODES;
constexpr size_t kNoallocBytes = TGM_MITIGATE_NOALLOC_BYTES;
constexpr int kMaxDevices = 64;

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The work space of one call, carved from the array in this order.
size_t noalloc_layout(int32_t cap, int32_t nbp, int32_t K, char *base, MitWork *w)
{
    size_t o = 0;
    auto take = [&](size_t bytes) {
        char *p = base ? base + o : nullptr;
        o = align256(o + bytes);
        return p;
    };
    const size_t c = (size_t)cap;
    void *nset = take(sizeof(int32_t) * c * nbp);
    void *ncnt = take(sizeof(int32_t) * c);
    void *gamma = take(sizeof(double));
    void *n_stale = take(sizeof(int32_t));
    void *stale = take(sizeof(int32_t) * c);
    void *omega = take(sizeof(int32_t) * c * K);
    void *part = take(sizeof(int2) * kMitOmegaGrid * kMitMaxK);
    if (w) {
        w->nset = (int32_t *)nset;
        w->ncnt = (int32_t *)ncnt;
        w->gamma = (double *)gamma;
        w->n_stale = (int32_t *)n_stale;
        w->stale = (int32_t *)stale;
        w->omega = (int32_t *)omega;
        w->part = (int2 *)part;
    }
    return o;
}

}  // namespace

static __device__ __align__(256) char scratch[TGM_MITIGATE_NOALLOC_BYTES];

namespace {

std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up on the first call on
// that device (hipGetSymbolAddress, with the device current) and kept.
tgm_status_t static_scratch_ptr(char **out)
{
    int dev = -1;
    TGM_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices)
        return TGM_EDEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            record_error(e != hipSuccess ? e : hipErrorInvalidSymbol);
            return TGM_EDEVICE;
        }
        g_scratch_ptr[dev] = (char *)p;
    }
    *out = g_scratch_ptr[dev];
    return TGM_OK;
}

}  // namespace

extern "C" tgm_status_t tgm_mitigate_noalloc(tgm_graph_t g, int64_t first_event,
                                             const int32_t *nodes, const int32_t *n_nodes,
                                             int32_t cap, float *mem, const double *mem_ts,
                                             int32_t M, int32_t nb, int32_t K, double p,
                                             float lambda, void *stream)
{
    if (!g || !nodes || !n_nodes || !mem || !mem_ts || M <= 0 || cap < 0)
        return TGM_EINVAL;
    if (nb < 1 || nb > 64 || K < 1 || K > kMitMaxK)
        return TGM_EINVAL;
    if (!(p >= 0.0 && p <= 1.0) || !(lambda >= 0.0f && lambda <= 1.0f))
        return TGM_EINVAL;
    if (first_event < 0 || first_event >= g->E)
        return TGM_ERANGE;
    if (cap > kNoallocMaxNodes)
        return TGM_ESIZE;
    MitWork w;
    w.nb = nb;
    w.nbp = nb <= 4 ? 4 : (nb <= 12 ? 12 : 64);
    w.K = K;
    if (noalloc_layout(cap, w.nbp, K, nullptr, nullptr) > kNoallocBytes)
        return TGM_ESIZE;
    if (cap == 0)
        return TGM_OK;
    char *base = nullptr;
    TGM_TRY_STATUS(static_scratch_ptr(&base));
    noalloc_layout(cap, w.nbp, K, base, &w);
    // k_mit_select clears the per-stale-node counters k_mit_omega needs at
    // zero; everything else is written before it is read within the call
    hipStream_t s = as_stream(stream);
    TGM_TRY_STATUS(prep_launch(w, g, first_event, nodes, n_nodes, cap, s));
    return blend_launch(w, g, first_event, nodes, n_nodes, cap, mem, mem_ts, M, p, lambda, s);
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
    // the executor's neighbour-set slots (one per sample buffer set), made
    // here so that a run allocates nothing
    if (mt)
        TGM_TRY_STATUS(tgm::mitigate_reserve(mt, 1 + TGM_MAX_SAMPLE_SETS));
    st->mit = mt;
    st->mit_p = p;
    st->mit_lambda = lambda;
    return TGM_OK;
}
