// Internal declarations shared by the libtgm translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "tgm.h"

namespace tgm {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---------------------------------------------------------------- errors
void record_error(hipError_t e);

#define TGM_HIP(call)                                  \
    do {                                               \
        hipError_t e_ = (call);                        \
        if (e_ != hipSuccess) {                        \
            ::tgm::record_error(e_);                   \
            return TGM_EDEVICE;                        \
        }                                              \
    } while (0)

#define TGM_TRY_STATUS(call)                           \
    do {                                               \
        const tgm_status_t st_ = (call);               \
        if (st_ != TGM_OK)                             \
            return st_;                                \
    } while (0)

#define TGM_LAUNCHED()                                 \
    do {                                               \
        hipError_t e_ = hipGetLastError();             \
        if (e_ != hipSuccess) {                        \
            ::tgm::record_error(e_);                   \
            return TGM_EDEVICE;                        \
        }                                              \
    } while (0)

inline hipStream_t as_stream(void *s) { return reinterpret_cast<hipStream_t>(s); }

// Every device allocation of the library goes through dev_malloc, which counts
// it (tgm_alloc_count), so a caller can check that a call allocated nothing.
void count_alloc();
template <class T>
inline hipError_t dev_malloc(T **p, size_t bytes)
{
    count_alloc();
    return hipMalloc((void **)p, bytes);
}

// Per-kernel timing (tgm_profile_*): prof_begin returns -1 when disabled.
int prof_begin(const char *kernel, hipStream_t s);
void prof_end(int id, hipStream_t s);

// Launch a kernel, timed when profiling is on, and check the launch.
#define TGM_LAUNCH(kern, grid, block, lds, s, ...)                       \
    do {                                                                 \
        const int pid_ = ::tgm::prof_begin(#kern, s);                    \
        hipLaunchKernelGGL(kern, grid, block, lds, s, __VA_ARGS__);      \
        ::tgm::prof_end(pid_, s);                                        \
        TGM_LAUNCHED();                                                  \
    } while (0)

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int32_t round_up(int32_t a, int32_t b) { return (int32_t)cdiv(a, b) * b; }

// ---------------------------------------------------------------- handles
// One adjacency entry: an event touching the node, with its time and the
// other endpoint.  16 bytes, so the k entries a sampler reads are one
// contiguous 16k-byte run.
struct AdjRec {
    double ts;
    int32_t eid;
    int32_t nbr;
};

}  // namespace tgm

struct tgm_graph {
    int32_t N = 0;
    int64_t E = 0;
    int32_t D_e = 0;
    const int32_t *src = nullptr, *dst = nullptr, *neg = nullptr;
    const double *t = nullptr;
    const float *efeat = nullptr;
    int64_t *off = nullptr;           // [N + 1]
    tgm::AdjRec *adj = nullptr;       // [n_adj]
    double *tix = nullptr;            // [cdiv(n_adj, 64)] time of record 64 j
    int64_t n_adj = 0;
    int32_t *ns_stamp = nullptr;      // [N] node-set epoch stamps (scratch of tgm_node_set)
    int32_t ns_epoch = 0;             // epoch of the last tgm_node_set call
};

struct tgm_state {
    int32_t N = 0, M = 0, D_m = 0, s = 0, max_batch = 0;
    // committed tables
    float *mem = nullptr, *mail = nullptr;
    double *mem_ts = nullptr, *mail_ts = nullptr;
    int32_t *ver = nullptr;
    // ring of s + 1 staged write sets, each indexed by candidate c in [0, 2b):
    // candidate c is (event first + c/2, role c%2)
    int32_t *r_flag = nullptr, *r_node = nullptr;
    float *r_mem = nullptr, *r_mail = nullptr;
    double *r_mem_ts = nullptr, *r_mail_ts = nullptr;
    struct Slot {
        int64_t iter = -1;
        int32_t b = 0;
        bool staged = false;
    };
    std::vector<Slot> ring;
    int64_t committed_through = -1;   // all writes <= this are in the tables
    int64_t staged_through = -1;      // last iteration whose update was issued
    int64_t last_fetch = INT64_MIN;
    // [N] latest candidate per node-set position, as the key (tag << 32) | c
    // of the update call that wrote it (tags start at 1, so zero is stale)
    uint64_t *win = nullptr;
    uint32_t win_tag = 0;             // tag of the last update call
    // the pipelined executor's latest-message reduce, run beside each sample
    // on the prefetch stream: one [xwin_cap] key array per sample buffer set,
    // keyed with a tag that grows with every reduced iteration
    uint64_t *xwin = nullptr;
    int32_t xwin_slots = 0, xwin_cap = 0;
    uint32_t xwin_tag = 0;
    // the executor's cross-stream events (sampled chunk and computed chunk by
    // parity, start), made at creation so that a run creates nothing
    hipEvent_t run_ev[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
    // training step after every iteration of the executor (off when null):
    // iteration i's loss goes to loss_log[i % loss_log_len] when a log is set
    struct tgm_trainer *trainer = nullptr;
    float *loss_log = nullptr;
    int64_t loss_log_len = 0;
    // staleness mitigation applied by the pipelined executor after each fetch
    // (tgm_state_set_mitigation; off when mit is null)
    struct tgm_mitigator *mit = nullptr;
    double mit_p = 1.0;
    float mit_lambda = 1.0f;
    size_t ring_rows() const { return 2 * (size_t)max_batch; }
};

struct tgm_model {
    int32_t M = 0, D_e = 0, D_t = 0, H = 0, nb = 0, max_nodes = 0, max_roots = 0;
    int32_t D_m = 0, D_x = 0;
    // GRU: packed B operands and biases
    int32_t KXC = 0, KHC = 0, MB = 0;   // 16-wide chunks of D_x, M and hidden blocks
    tgm::f4 *gru_bx = nullptr;           // [3][KXC][MB][64]
    // the GRU with one hidden block's weights resident in LDS (when the shapes
    // fit) and its time-encoding input [max_nodes x D_t], formed per call
    bool gru_w = false;
    float *phi = nullptr;
    tgm::f4 *gru_bh = nullptr;           // [3][KHC][MB][64]
    float *gru_bias = nullptr;           // [4][MB*16]: b_ir+b_hr, b_iz+b_hz, b_in, b_hn
    double *omega = nullptr, *beta = nullptr;
    // node projections P = s' [W_q^s; W_k^s; W_v^s]^T
    int32_t PC = 0, PNB = 0;             // chunks of M, 16-col blocks of 3M
    tgm::f4 *proj_b = nullptr;
    float *P = nullptr;                  // [max_nodes x PNB*16]
    // attention: per-slot part [efeat || phi] -> [K | V]
    int32_t KFC = 0, KVNB = 0;           // chunks of D_e + D_t, 16-col blocks of 2M
    tgm::f4 *kv_b = nullptr;
    float *pbias = nullptr;   // [PNB*16] bias of the node projection: c_q | b_k | b_v | 0
    // attention with the query folded into the key weights (when the shapes fit)
    bool fold = false;
    // attention by aggregation of the slot rows (when the shapes fit; it
    // reads the folded attention's packed operands)
    bool agg = false;
    int32_t VNB = 0, DC = 0;             // 16-col blocks of M, 16-wide chunks of M
    tgm::f4 *v_b = nullptr;              // [KFC(+pad)][VNB][64]: V part of the slot weights
    tgm::f4 *uk_a = nullptr;             // [DC][KFC][64]: W_k^t as A fragments
    // output projection
    int32_t OC = 0, ONB = 0;             // chunks of 2M, 16-col blocks of M
    tgm::f4 *out_b = nullptr;
    float *b_o = nullptr;
    // model family; JODIE's time projection and a [max_nodes] buffer of new
    // memory times for the executor when its caller passes none
    int32_t kind = TGM_MODEL_TGN;
    float *w_t = nullptr;
    double *nts = nullptr;
};

namespace tgm {

// ---------------------------------------------------------------- device
// v_mfma_f32_16x16x4_f32: lane l supplies A[l%16][l/16] and B[l/16][l%16];
// the 4 results of lane l are C[4*(l/16) + v][l%16], v = 0..3.
__device__ __forceinline__ f4 mfma_16x16x4(float a, float b, f4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// 16 consecutive k of one 16x16 output block.  Lane l holds a = A[row][k0 + 4q
// .. +3] and b = B[k0 + 4q .. +3][col] with q = l/16, row = col = l%16; the
// four instructions each cover the k-slice {k0 + 4q + j}.
__device__ __forceinline__ f4 mfma_k16(f4 a, f4 b, f4 c)
{
    c = mfma_16x16x4(a.x, b.x, c);
    c = mfma_16x16x4(a.y, b.y, c);
    c = mfma_16x16x4(a.z, b.z, c);
    c = mfma_16x16x4(a.w, b.w, c);
    return c;
}

// Cosine time encoding cos(omega * dt + beta).  Time gaps reach 1e8 s, where
// an fp32 phase is off by whole radians, so the phase is formed and reduced to
// a fraction of a turn in fp64 (to within ~2e-8 rad for |phase| <= 1e8).  The
// cosine of the reduced angle uses the symmetries of cos to fold the angle into
// [0, pi/2] (x = 2 pi h, h in [0, 1/4]; beyond a quarter turn
// cos(2 pi h) = -cos(2 pi (1/2 - h))) and then the Taylor series of cos through
// the x^12 term, whose truncation error on [0, pi/2] is below
// (pi/2)^14 / 14! < 1e-8; fp32 rounding keeps the total within ~2e-7.
__device__ __forceinline__ float cos_turns(float f)   // cos(2 pi f), |f| <= 1/2
{
    float h = fabsf(f);
    const bool flip = h > 0.25f;
    h = flip ? 0.5f - h : h;
    const float x = h * 6.28318530717958648f;
    const float x2 = x * x;
    // 1 - x^2/2! + x^4/4! - ... + x^12/12!, Horner in x^2
    float p = 2.08767569878680989792e-9f;         //  1/12!
    p = fmaf(p, x2, -2.75573192239858906526e-7f);  // -1/10!
    p = fmaf(p, x2, 2.48015873015873015873e-5f);   //  1/8!
    p = fmaf(p, x2, -1.38888888888888888889e-3f);  // -1/6!
    p = fmaf(p, x2, 4.16666666666666666667e-2f);   //  1/4!
    p = fmaf(p, x2, -0.5f);                        // -1/2!
    p = fmaf(p, x2, 1.0f);
    return flip ? -p : p;
}

__device__ __forceinline__ float time_enc(double omega, double beta, double dt)
{
    const double ph = fma(omega, dt, beta);
    const double rev = ph * 0.15915494309189535;   // phase in turns: ph / (2 pi)
    return cos_turns((float)(rev - rint(rev)));    // [-1/2, 1/2] turn, exact in fp64
}

// Software pipelining: a loop loads the next k-chunk's operand while it
// multiplies the current one.  Left alone, the compiler sinks such a load to
// its use in the next iteration (and waits for it there); consuming the
// registers here, after the iteration's MFMAs have been issued, keeps the load
// one iteration ahead.
__device__ __forceinline__ void keep_loaded(const f4 &a) { asm volatile("" ::"v"(a)); }
// Keeps the scheduler from moving instructions across this point (used right
// after the prefetch loads so they are issued before the iteration's MFMAs).
__device__ __forceinline__ void issue_fence() { __builtin_amdgcn_sched_barrier(0); }

// A workgroup barrier that orders LDS accesses only: each wave waits for its
// own LDS operations (lgkmcnt), not for its global loads still in flight,
// which __syncthreads (a release fence over every address space) also waits
// for.  For exchanges through LDS while the next operands stream in.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Reductions over one 16-lane DPP row (lanes 16i .. 16i + 15) with row-local
// DPP moves: swaps inside quads (quad_perm [1,0,3,2], then [2,3,0,1]), then the
// half-row and row mirrors.  Each step combines a lane with its partner's equal
// partial (a+b and b+a round alike), so every lane of the row ends with the
// same value.  Only the row's own lanes are read: other rows may be inactive.
template <int CTRL>
__device__ __forceinline__ float dpp_row(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

__device__ __forceinline__ float row16_max(float v)
{
    v = fmaxf(v, dpp_row<kDppXor1>(v));
    v = fmaxf(v, dpp_row<kDppXor2>(v));
    v = fmaxf(v, dpp_row<kDppHalfMirror>(v));
    return fmaxf(v, dpp_row<kDppMirror>(v));
}

__device__ __forceinline__ float row16_sum(float v)
{
    v += dpp_row<kDppXor1>(v);
    v += dpp_row<kDppXor2>(v);
    v += dpp_row<kDppHalfMirror>(v);
    return v + dpp_row<kDppMirror>(v);
}

// One wavefront: the adjacency list of v is sorted by (t, e); returns p, the
// first entry with ts >= tq, so that [*base, p) are v's strictly earlier
// events.  An id outside [0, N) has an empty list.
//
// tix[j] is the time of adjacency record 64 j (the graph's sparse time index,
// 8 bytes per 64 records).  The records 64 j inside v's list are searched
// first in tix, whose entries for one list are contiguous: a 64-ary search
// where each round lane l probes the last entry of the l-th of 64 equal
// segments, and the ballot's popcount names the segment that holds the
// boundary.  With c of those records earlier than tq, every record before
// the c-th is earlier and the (c+1)-th is not, so the boundary lies in one
// window of at most 64 records (from the c-th such record, or from the list's
// start when c = 0, up to the next one or the list's end), counted with one
// more ballot.
__device__ __forceinline__ int64_t recent_end(const int64_t *__restrict__ off,
                                              const AdjRec *__restrict__ adj,
                                              const double *__restrict__ tix, int32_t v,
                                              double tq, int32_t N, int64_t *base)
{
    const int lane = threadIdx.x & 63;
    const bool ok = v >= 0 && v < N;
    const int64_t b0 = ok ? off[v] : 0, e0 = ok ? off[v + 1] : 0;
    *base = b0;
    // indexed records 64 j with b0 <= 64 j < e0: j in [j0, j1)
    const int64_t j0 = (b0 + kWave - 1) >> 6;
    const int64_t j1 = e0 > b0 ? max(j0, ((e0 - 1) >> 6) + 1) : j0;
    int64_t lo = j0, hi = j1;
    while (hi - lo > kWave) {
        const int64_t step = (hi - lo + kWave - 1) / kWave;
        const int64_t probe = lo + (int64_t)(lane + 1) * step - 1;
        const bool below = probe < hi && tix[probe] < tq;
        const int c = __popcll(__ballot(below));
        const int64_t nlo = lo + (int64_t)c * step;
        const int64_t nhi = nlo + step < hi ? nlo + step : hi;
        lo = nlo;
        hi = nhi;
    }
    {
        const int64_t idx = lo + lane;
        const bool below = idx < hi && tix[idx] < tq;
        lo += __popcll(__ballot(below));
    }
    // lo - j0 indexed records are earlier than tq
    const int64_t ws = lo > j0 ? (lo - 1) << 6 : b0;
    const int64_t we = min(lo > j0 ? ws + kWave : (j0 << 6), e0);
    const int64_t idx = ws + lane;
    const bool below = idx < we && adj[idx].ts < tq;
    return ws + __popcll(__ballot(below));
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o, kWave);
    return v;
}

// Copy `n` floats with one wavefront; 16-byte accesses when both rows allow it.
__device__ __forceinline__ void wave_copy_row(float *__restrict__ dst,
                                              const float *__restrict__ src, int n, int lane)
{
    if (((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 15) == 0 &&
        (n & 3) == 0) {
        const f4 *s4 = reinterpret_cast<const f4 *>(src);
        f4 *d4 = reinterpret_cast<f4 *>(dst);
        for (int k = lane; k < (n >> 2); k += kWave)
            d4[k] = s4[k];
    } else if (((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) & 7) ==
                   0 &&
               (n & 1) == 0) {
        const f2 *s2 = reinterpret_cast<const f2 *>(src);
        f2 *d2 = reinterpret_cast<f2 *>(dst);
        for (int k = lane; k < (n >> 1); k += kWave)
            d2[k] = s2[k];
    } else {
        for (int k = lane; k < n; k += kWave)
            dst[k] = src[k];
    }
}

// Two rows copied by one wavefront with every load issued before the first
// store (lane l holds elements l + 64 u; clamped indices keep the loads
// unconditional and in range; n1 >= 1, n2 >= 0).  The rows must fit U1 and
// U2 chunks of 64 elements.
template <int U1, int U2>
__device__ __forceinline__ void copy2_rows_regs(float *__restrict__ d1,
                                                const float *__restrict__ s1, int n1,
                                                float *__restrict__ d2,
                                                const float *__restrict__ s2, int n2, int lane)
{
    float a[U1], b[U2];
#pragma unroll
    for (int u = 0; u < U1; ++u)
        a[u] = s1[min(lane + kWave * u, n1 - 1)];
#pragma unroll
    for (int u = 0; u < U2; ++u)
        b[u] = n2 > 0 ? s2[min(lane + kWave * u, n2 - 1)] : 0.f;
#pragma unroll
    for (int u = 0; u < U1; ++u)
        if (lane + kWave * u < n1)
            d1[lane + kWave * u] = a[u];
#pragma unroll
    for (int u = 0; u < U2; ++u)
        if (lane + kWave * u < n2)
            d2[lane + kWave * u] = b[u];
}

// The same with V1- and V2-wide vector accesses (row lengths multiples of
// the widths, every row aligned to them; n2 >= V2): lane l holds vectors
// l + 64 u of each row.
template <int V1, int V2, int U1, int U2>
__device__ __forceinline__ void copy2_rows_vec(float *__restrict__ d1,
                                               const float *__restrict__ s1, int n1,
                                               float *__restrict__ d2,
                                               const float *__restrict__ s2, int n2, int lane)
{
    typedef float v1_t __attribute__((ext_vector_type(V1)));
    typedef float v2_t __attribute__((ext_vector_type(V2)));
    const int m1 = n1 / V1, m2 = n2 / V2;
    const v1_t *a1 = reinterpret_cast<const v1_t *>(s1);
    const v2_t *a2 = reinterpret_cast<const v2_t *>(s2);
    v1_t a[U1];
    v2_t b[U2];
#pragma unroll
    for (int u = 0; u < U1; ++u)
        a[u] = a1[min(lane + kWave * u, m1 - 1)];
#pragma unroll
    for (int u = 0; u < U2; ++u)
        b[u] = a2[min(lane + kWave * u, m2 - 1)];
#pragma unroll
    for (int u = 0; u < U1; ++u)
        if (lane + kWave * u < m1)
            reinterpret_cast<v1_t *>(d1)[lane + kWave * u] = a[u];
#pragma unroll
    for (int u = 0; u < U2; ++u)
        if (lane + kWave * u < m2)
            reinterpret_cast<v2_t *>(d2)[lane + kWave * u] = b[u];
}

// Whether rows of n floats at p and q allow w-wide vector accesses
__device__ __forceinline__ bool rows_vec_ok(const void *p, const void *q, int n, int w)
{
    return n % w == 0 &&
           ((reinterpret_cast<uintptr_t>(p) | reinterpret_cast<uintptr_t>(q)) & (4 * w - 1)) == 0;
}

// Copies rows (s1 -> d1, n1 floats) and (s2 -> d2, n2 floats) with one
// wavefront: loads first when the rows are short enough (vector accesses
// when the rows allow them), else row by row.
__device__ __forceinline__ void wave_copy_2rows(float *d1, const float *s1, int n1, float *d2,
                                                const float *s2, int n2, int lane)
{
    if (n1 >= 4 && n1 <= 4 * kWave && rows_vec_ok(d1, s1, n1, 4) && n2 >= 4 &&
        n2 <= 8 * kWave && rows_vec_ok(d2, s2, n2, 4)) {
        copy2_rows_vec<4, 4, 1, 2>(d1, s1, n1, d2, s2, n2, lane);
    } else if (n1 >= 4 && n1 <= 4 * kWave && rows_vec_ok(d1, s1, n1, 4) && n2 >= 2 &&
               n2 <= 8 * kWave && rows_vec_ok(d2, s2, n2, 2)) {
        copy2_rows_vec<4, 2, 1, 4>(d1, s1, n1, d2, s2, n2, lane);
    } else if (n1 <= 2 * kWave && n2 <= 8 * kWave) {
        copy2_rows_regs<2, 8>(d1, s1, n1, d2, s2, n2, lane);
    } else if (n1 <= 4 * kWave && n2 <= 16 * kWave) {
        copy2_rows_regs<4, 16>(d1, s1, n1, d2, s2, n2, lane);
    } else {
        wave_copy_row(d1, s1, n1, lane);
        wave_copy_row(d2, s2, n2, lane);
    }
}

// One fetch's gather: rows nodes[0 .. min(*n_nodes, cap)) of the committed
// tables into the caller's buffers (see tgm_fetch_memory).
struct GatherPlan {
    const int32_t *nodes = nullptr, *n_nodes = nullptr;
    int32_t cap = 0, M = 0, D_m = 0;
    const float *mem = nullptr, *mail = nullptr;
    const double *mem_ts = nullptr, *mail_ts = nullptr;
    const int32_t *ver = nullptr;
    float *o_mem = nullptr, *o_mail = nullptr;
    double *o_mem_ts = nullptr, *o_mail_ts = nullptr;
    int32_t *o_ver = nullptr;
    // optional: the GRU's time input phi(mail_ts - mem_ts) of each fetched
    // node ([cap x D_t], zero for a node without mail), formed by the gather
    const double *omega = nullptr, *beta = nullptr;
    int32_t D_t = 0;
    float *o_phi = nullptr;
    // o_mem == nullptr: phi alone, no rows copied (the executor's GRU then
    // reads the committed tables in place; see tgm_stage_run)
    void phi_only() { o_mem = nullptr; o_mail = nullptr; o_mem_ts = o_mail_ts = nullptr; o_ver = nullptr; }
};

// Row p of a gather, copied by one wavefront.  Every load of the node's two
// rows and three scalars is issued before the first store: one wavefront
// keeps up to 2.5 KB in flight, which the HBM latency needs (with a load and
// its store per round trip, a node's rows took several round trips).  Lane l
// holds elements l + 64 u of a row (4-byte loads, 256 contiguous bytes per
// instruction); indices past the row are clamped to its last element, so
// every load is unconditional and in range.  UM and UD bound the 64-element
// chunks of the two rows.
template <int UM, int UD>
__device__ __forceinline__ void gather_row_regs(const GatherPlan &g, int p, int lane)
{
    const int32_t v = g.nodes[p];
    const int M = g.M, D = g.D_m;
    const float *sm = g.mem + (int64_t)v * M, *sd = g.mail + (int64_t)v * D;
    float a[UM], b[UD];
#pragma unroll
    for (int u = 0; u < UM; ++u)
        a[u] = sm[min(lane + kWave * u, M - 1)];
#pragma unroll
    for (int u = 0; u < UD; ++u)
        b[u] = D > 0 ? sd[min(lane + kWave * u, D - 1)] : 0.f;
    double mts = 0.0, lts = 0.0;
    int32_t ver = 0;
    if (lane == 0) {
        mts = g.mem_ts[v];
        lts = g.mail_ts[v];
        ver = g.ver[v];
    }
    float *dm = g.o_mem + (int64_t)p * M, *dd = g.o_mail + (int64_t)p * D;
#pragma unroll
    for (int u = 0; u < UM; ++u)
        if (lane + kWave * u < M)
            dm[lane + kWave * u] = a[u];
#pragma unroll
    for (int u = 0; u < UD; ++u)
        if (lane + kWave * u < D)
            dd[lane + kWave * u] = b[u];
    if (lane == 0) {
        g.o_mem_ts[p] = mts;
        g.o_mail_ts[p] = lts;
        g.o_ver[p] = ver;
    }
}

__device__ __forceinline__ void gather_row(const GatherPlan &g, int p, int lane);

// Rows p0 .. p0 + NPW - 1 (those below n) of a gather, copied by one
// wavefront: lane j < NPW loads node id j, then every row load of the NPW
// nodes is issued (up to 10 KB in flight) before the first store.  Positions
// past n reuse the last node's rows for their (discarded) loads.
constexpr int kGatherNPW = 4;   // nodes per wavefront

template <int UM, int UD>
__device__ __forceinline__ void gather_rows_regs(const GatherPlan &g, int p0, int n, int lane)
{
    constexpr int NPW = kGatherNPW;
    const int M = g.M, D = g.D_m;
    const int32_t vid = g.nodes[min(p0 + (lane < NPW ? lane : 0), n - 1)];
    float a[NPW][UM], b[NPW][UD];
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
        const int32_t v = __builtin_amdgcn_readlane(vid, j);
        const float *sm = g.mem + (int64_t)v * M, *sd = g.mail + (int64_t)v * D;
#pragma unroll
        for (int u = 0; u < UM; ++u)
            a[j][u] = sm[min(lane + kWave * u, M - 1)];
#pragma unroll
        for (int u = 0; u < UD; ++u)
            b[j][u] = D > 0 ? sd[min(lane + kWave * u, D - 1)] : 0.f;
    }
    double mts = 0.0, lts = 0.0;
    int32_t ver = 0;
    if (lane < NPW) {
        mts = g.mem_ts[vid];
        lts = g.mail_ts[vid];
        ver = g.ver[vid];
    }
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
        const int p = p0 + j;
        if (p >= n)
            break;   // uniform
        float *dm = g.o_mem + (int64_t)p * M, *dd = g.o_mail + (int64_t)p * D;
#pragma unroll
        for (int u = 0; u < UM; ++u)
            if (lane + kWave * u < M)
                dm[lane + kWave * u] = a[j][u];
#pragma unroll
        for (int u = 0; u < UD; ++u)
            if (lane + kWave * u < D)
                dd[lane + kWave * u] = b[j][u];
    }
    if (lane < NPW && p0 + lane < n) {
        g.o_mem_ts[p0 + lane] = mts;
        g.o_mail_ts[p0 + lane] = lts;
        g.o_ver[p0 + lane] = ver;
    }
}

// The same with VM- and VD-wide vector accesses to the memory and mail rows
// (both row lengths multiples of their width, every row base aligned to it):
// lane l holds vectors l + 64 u, so one instruction moves 64 VM (or VD)
// floats of a row.  UM and UD bound the 64-vector chunks of the two rows.
template <int VM, int VD, int UM, int UD, int NPW>
__device__ __forceinline__ void gather_rows_vec(const GatherPlan &g, int p0, int n, int lane)
{
    typedef float vm_t __attribute__((ext_vector_type(VM)));
    typedef float vd_t __attribute__((ext_vector_type(VD)));
    const int NM = g.M / VM, ND = g.D_m / VD;   // vectors per row
    const int32_t vid = g.nodes[min(p0 + (lane < NPW ? lane : 0), n - 1)];
    vm_t a[NPW][UM];
    vd_t b[NPW][UD];
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
        const int32_t v = __builtin_amdgcn_readlane(vid, j);
        const vm_t *sm = reinterpret_cast<const vm_t *>(g.mem + (int64_t)v * g.M);
        const vd_t *sd = reinterpret_cast<const vd_t *>(g.mail + (int64_t)v * g.D_m);
#pragma unroll
        for (int u = 0; u < UM; ++u)
            a[j][u] = sm[min(lane + kWave * u, NM - 1)];
#pragma unroll
        for (int u = 0; u < UD; ++u)
            b[j][u] = sd[min(lane + kWave * u, ND - 1)];
    }
    double mts = 0.0, lts = 0.0;
    int32_t ver = 0;
    if (lane < NPW) {
        mts = g.mem_ts[vid];
        lts = g.mail_ts[vid];
        ver = g.ver[vid];
    }
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
        const int p = p0 + j;
        if (p >= n)
            break;   // uniform
        vm_t *dm = reinterpret_cast<vm_t *>(g.o_mem + (int64_t)p * g.M);
        vd_t *dd = reinterpret_cast<vd_t *>(g.o_mail + (int64_t)p * g.D_m);
#pragma unroll
        for (int u = 0; u < UM; ++u)
            if (lane + kWave * u < NM)
                dm[lane + kWave * u] = a[j][u];
#pragma unroll
        for (int u = 0; u < UD; ++u)
            if (lane + kWave * u < ND)
                dd[lane + kWave * u] = b[j][u];
    }
    if (lane < NPW && p0 + lane < n) {
        g.o_mem_ts[p0 + lane] = mts;
        g.o_mail_ts[p0 + lane] = lts;
        g.o_ver[p0 + lane] = ver;
    }
}

// Whether every row of the four row arrays starts at a multiple of w floats
// (w = 2 or 4): row lengths multiples of w, bases aligned to 4 w bytes.
__device__ __forceinline__ bool gather_aligned(const GatherPlan &g, int wm, int wd)
{
    const uintptr_t am = reinterpret_cast<uintptr_t>(g.mem) | reinterpret_cast<uintptr_t>(g.o_mem);
    const uintptr_t ad = reinterpret_cast<uintptr_t>(g.mail) |
                         reinterpret_cast<uintptr_t>(g.o_mail);
    return g.M % wm == 0 && (am & (4 * wm - 1)) == 0 && g.D_m % wd == 0 &&
           (ad & (4 * wd - 1)) == 0;
}

// Rows p0 .. p0 + kGatherNPW - 1 (those below n) of a gather by one wavefront
// (VEC: vector accesses where the rows allow them; the launches that carry
// the gather beside another kernel's blocks keep the 4-byte ones, which need
// fewer registers).
// phi of the fetched nodes p0 .. p0 + kGatherNPW - 1 (those below n), when the
// plan asks for it: cos(omega_d (mail_ts - mem_ts) + beta_d) for a node with
// mail, zero otherwise (the node's times and version as the gather copies
// them)
// The time inputs phi of positions p0 .. p0 + NPW - 1 (those below n), one
// wavefront: every load first (the nodes' times and versions; the stores
// below could alias them, so loads after a store would wait for it), then the
// codes.
template <int NPW>
__device__ __forceinline__ void phi_rows(const GatherPlan &g, int p0, int n, int lane)
{
    double dt[NPW];
    bool has[NPW];
#pragma unroll
    for (int j = 0; j < NPW; ++j) {
        const int32_t v = g.nodes[min(p0 + j, n - 1)];
        dt[j] = g.mail_ts[v] - g.mem_ts[v];
        has[j] = g.ver[v] >= 0;
    }
    for (int d0 = 0; d0 < g.D_t; d0 += kWave) {
        const int d = d0 + lane;
        const int dc = min(d, g.D_t - 1);
        const double om = g.omega[dc], be = g.beta[dc];
#pragma unroll
        for (int j = 0; j < NPW; ++j)
            if (p0 + j < n && d < g.D_t)
                g.o_phi[(int64_t)(p0 + j) * g.D_t + d] = has[j] ? time_enc(om, be, dt[j]) : 0.f;
    }
}

__device__ __forceinline__ void gather_phi(const GatherPlan &g, int p0, int n, int lane)
{
    if (g.o_phi)
        phi_rows<kGatherNPW>(g, p0, n, lane);
}

template <bool VEC = false>
__device__ __forceinline__ void gather_rows(const GatherPlan &g, int p0, int n, int lane)
{
    gather_phi(g, p0, n, lane);
    if (!g.o_mem)   // phi only: the GRU reads the committed rows in place
        return;
    if (VEC && g.M > 0 && g.M <= 4 * kWave && g.D_m > 0 && g.D_m <= 16 * kWave &&
        gather_aligned(g, 4, 4)) {
        gather_rows_vec<4, 4, 1, 4, kGatherNPW>(g, p0, n, lane);
    } else if (VEC && g.M > 0 && g.M <= 4 * kWave && g.D_m > 0 && g.D_m <= 8 * kWave &&
               gather_aligned(g, 4, 2)) {
        gather_rows_vec<4, 2, 1, 4, kGatherNPW>(g, p0, n, lane);
    } else if (g.M <= 2 * kWave && g.D_m <= 8 * kWave) {
        gather_rows_regs<2, 8>(g, p0, n, lane);
    } else {
        for (int j = 0; j < kGatherNPW && p0 + j < n; ++j)
            gather_row(g, p0 + j, lane);
    }
}

__device__ __forceinline__ void gather_row(const GatherPlan &g, int p, int lane)
{
    if (g.M <= 2 * kWave && g.D_m <= 8 * kWave) {
        gather_row_regs<2, 8>(g, p, lane);
    } else if (g.M <= 4 * kWave && g.D_m <= 16 * kWave) {
        gather_row_regs<4, 16>(g, p, lane);
    } else {
        const int32_t v = g.nodes[p];
        wave_copy_row(g.o_mem + (int64_t)p * g.M, g.mem + (int64_t)v * g.M, g.M, lane);
        wave_copy_row(g.o_mail + (int64_t)p * g.D_m, g.mail + (int64_t)v * g.D_m, g.D_m, lane);
        if (lane == 0) {
            g.o_mem_ts[p] = g.mem_ts[v];
            g.o_mail_ts[p] = g.mail_ts[v];
            g.o_ver[p] = g.ver[v];
        }
    }
}

// A fetch spread over the nblk workgroups (of `waves` wavefronts) that follow
// other work in a launch; b is this workgroup's index among them.  Rows:
// kGatherNPW nodes per wavefront at a time; phi only: kPhiNPW.
constexpr int kPhiNPW = 8;   // enough wavefronts for a small node set, and loads enough in flight
__device__ __forceinline__ void gather_blocks(const GatherPlan &g, int b, int nblk, int waves,
                                              int wave, int lane)
{
    const int n = min(*g.n_nodes, g.cap);
    if (g.o_mem) {
        for (int p = (b * waves + wave) * kGatherNPW; p < n; p += nblk * waves * kGatherNPW)
            gather_rows(g, p, n, lane);
    } else if (g.o_phi) {
        for (int p = (b * waves + wave) * kPhiNPW; p < n; p += nblk * waves * kPhiNPW)
            phi_rows<kPhiNPW>(g, p, n, lane);
    }
}

// Block-wide gather of `rows` rows of `n` floats into LDS: row r of the
// destination (stride `lds_stride` floats, starting at column `col0`) is
// src[off[r] .. off[r] + n), or zeros when off[r] < 0.  `off` lives in LDS.
// Every thread issues up to kStageUnroll loads before its stores, so a block's
// row gathers are in flight together instead of one dependent row at a time.
constexpr int kStageUnroll = 8;

template <int W>
struct VecOf;
template <>
struct VecOf<4> { typedef f4 T; };
template <>
struct VecOf<2> { typedef f2 T; };
template <>
struct VecOf<1> { typedef float T; };

template <int W>
__device__ __forceinline__ void stage_rows_w(float *__restrict__ lds, int lds_stride, int col0,
                                             const float *__restrict__ src,
                                             const int64_t *__restrict__ off, int rows, int n)
{
    typedef typename VecOf<W>::T V;
    const int per_row = n / W;
    const int total = rows * per_row;
    const int nt = blockDim.x;
    for (int base = threadIdx.x; base < total; base += nt * kStageUnroll) {
        V v[kStageUnroll];
#pragma unroll
        for (int u = 0; u < kStageUnroll; ++u) {
            const int idx = base + u * nt;
            if (idx < total) {
                const int r = idx / per_row, c = idx - r * per_row;
                const int64_t o = off[r];
                v[u] = o >= 0 ? *reinterpret_cast<const V *>(src + o + (int64_t)c * W) : V(0);
            }
        }
#pragma unroll
        for (int u = 0; u < kStageUnroll; ++u) {
            const int idx = base + u * nt;
            if (idx < total) {
                const int r = idx / per_row, c = idx - r * per_row;
                *reinterpret_cast<V *>(lds + r * lds_stride + col0 + c * W) = v[u];
            }
        }
    }
}

// Rows staged by one wavefront: up to RMAX rows of n floats, lanes across the
// columns in W-float vectors (n <= 64 * W * CMAX).  load() issues every load
// of the wave's rows at once (no per-element index division); store() writes
// them to LDS.  Rows with off < 0, and columns past n, are zero.  src must
// hold at least W elements (the dead lanes read its first vector).
template <int W, int RMAX, int CMAX>
struct WaveRows {
    typedef typename VecOf<W>::T V;
    V v[RMAX][CMAX];

    // Branch-free: a dead lane reads src[0], and the value is only masked in
    // store(), so no load is waited for before the first store.
    __device__ __forceinline__ void load(const float *__restrict__ src, const int64_t (&off)[RMAX],
                                         int n, int lane)
    {
        const int nv = n / W;
#pragma unroll
        for (int i = 0; i < RMAX; ++i)
#pragma unroll
            for (int c = 0; c < CMAX; ++c) {
                const int cc = lane + kWave * c;
                const bool ok = off[i] >= 0 && cc < nv;
                v[i][c] = *reinterpret_cast<const V *>(src + (ok ? off[i] + (int64_t)cc * W : 0));
            }
    }

    // row i goes to LDS row lrow[i] (skipped when lrow[i] < 0); off must be the
    // offsets given to load()
    __device__ __forceinline__ void store(float *__restrict__ lds, int stride, int col0,
                                          const int (&lrow)[RMAX], const int64_t (&off)[RMAX],
                                          int n, int lane) const
    {
        const int nv = n / W;
#pragma unroll
        for (int i = 0; i < RMAX; ++i)
#pragma unroll
            for (int c = 0; c < CMAX; ++c) {
                const int cc = lane + kWave * c;
                if (lrow[i] >= 0 && cc < nv)
                    *reinterpret_cast<V *>(lds + lrow[i] * stride + col0 + cc * W) =
                        off[i] >= 0 ? v[i][c] : V(0);
            }
    }
};

// `ld` is the source row stride in floats (every off[r] is a multiple of it).
__device__ __forceinline__ void stage_rows(float *__restrict__ lds, int lds_stride, int col0,
                                           const float *__restrict__ src, int64_t ld,
                                           const int64_t *__restrict__ off, int rows, int n)
{
    const bool a16 = (reinterpret_cast<uintptr_t>(src) & 15) == 0;
    const bool a8 = (reinterpret_cast<uintptr_t>(src) & 7) == 0;
    if (a16 && (n & 3) == 0 && (ld & 3) == 0 && (col0 & 3) == 0 && (lds_stride & 3) == 0)
        stage_rows_w<4>(lds, lds_stride, col0, src, off, rows, n);
    else if (a8 && (n & 1) == 0 && (ld & 1) == 0 && (col0 & 1) == 0 && (lds_stride & 1) == 0)
        stage_rows_w<2>(lds, lds_stride, col0, src, off, rows, n);
    else
        stage_rows_w<1>(lds, lds_stride, col0, src, off, rows, n);
}

// ---------------------------------------------------------------- host
// Pack the B operand of C = A * W^T (W is n_out x K, row stride ldw, columns
// [c0, c0 + K)) for mfma_k16: out[((kc * NB + nb) * 64 + lane) * 4 + j] =
// W[16 nb + lane%16][c0 + 16 kc + 4 (lane/16) + j], zero outside.
std::vector<float> pack_b(const float *W, int n_out, int ldw, int c0, int K, int KC, int NB);

tgm_status_t upload(void *dst, const void *src, size_t bytes);

// Host side of tgm_fetch_memory: argument and protocol checks, the commits
// the fetch needs (enqueued on s), and the gather to run, in *plan.
tgm_status_t fetch_plan(tgm_state_t st, int64_t iter, const int32_t *nodes,
                        const int32_t *n_nodes, int32_t cap, float *mem, double *mem_ts,
                        float *mail, double *mail_ts, int32_t *ver, hipStream_t s,
                        GatherPlan *plan);
// The gather of a plan as its own launch.
tgm_status_t launch_gather(const GatherPlan &plan, hipStream_t s);

// The compute of iteration `iter` for the pipelined executor, with the fetch
// of iteration iter + 1 into the same fetch buffers when next_sb (its sample
// buffers) is given, in three launches on s: the GRU (with the
// latest-message reduce); the staging of the write set fused with the node
// projections; the attention fused with the next fetch's gather, which needs
// only the staging's commits.  Same results as tgm_update_memory and
// tgm_embed of iter followed by tgm_fetch_memory of iter + 1.
// inplace: this iteration's fetch formed phi only (GatherPlan::phi_only),
// and its GRU reads the committed tables in place at the node set's rows
// (they still hold exactly the write sets through iter - 1 - s: the next
// commit comes with this iteration's staging); next_inplace: the same for the
// fetch of iter + 1 made here.  next_ready (may be NULL): s waits for it
// right before the launch that carries the next fetch (the event of the
// next iteration's sample on another stream).
// Makes a fetch plan form the GRU's phi input of the model m as well (when
// the model's GRU reads it precomputed).
void phi_plan(const tgm_model *m, GatherPlan *plan);

tgm_status_t compute_iteration(tgm_state_t st, tgm_model_t m, tgm_graph_t g, int64_t iter,
                               const tgm_sample_buffers &sb, const tgm_fetch_buffers &fb,
                               int32_t cap, int64_t first_event, int32_t b, int32_t nb,
                               float *mem_new, double *new_mem_ts, int64_t *winner, float *h,
                               const tgm_sample_buffers *next_sb, int32_t mit_slot,
                               uint64_t *xwin, uint64_t xtag, hipStream_t s,
                               bool inplace = false, bool next_inplace = false,
                               hipEvent_t next_ready = nullptr);

// The executor's latest-message reduce of an iteration, on the prefetch
// stream beside its sample: exec_latest_launch reduces the 2b candidates of
// the batch into key array `slot` (one of the TGM_MAX_SAMPLE_SETS arrays of N
// entries made with the state) under a fresh tag and returns the array and
// the tag, which compute_iteration's staging then reads.
tgm_status_t exec_latest_launch(tgm_state_t st, int32_t slot, int32_t b, const int32_t *src_pos,
                                const int32_t *dst_pos, const int32_t *n_nodes, hipStream_t s,
                                uint64_t **win, uint64_t *tag);

// The mitigation of tgm_mitigate in two parts.  mitigate_prep_launch writes
// the neighbour sets of a node set into slot `slot` (it needs the graph and
// the node set only); mitigate_launch selects the stale nodes and blends their
// fetched memories with the sets of that slot.  Slot 0 belongs to
// tgm_mitigate; mitigate_reserve makes slots 0 .. nslots - 1 (it may allocate,
// and drops the contents of existing slots).
tgm_status_t mitigate_reserve(tgm_mitigator_t mt, int32_t nslots);
int32_t mitigate_slots(tgm_mitigator_t mt);

// The trained weights of a TGN model, plain row-major device arrays (the
// layouts of tgm_weights).  model_repack rebuilds every packed operand the
// model's kernels read from them (after an optimizer step).
struct ModelParams {
    const float *W_ih, *W_hh, *b_ih, *b_hh, *W_q, *b_q, *W_k, *b_k, *W_v, *b_v, *W_o, *b_o;
};
tgm_status_t model_repack(tgm_model_t m, const ModelParams &w, hipStream_t s);

// C[m x n] = op(A) op(B) (+ bias[n]) (+ C when accumulate), fp32 MFMA, no
// split of the reduction (the GEMM of the training step; op as there).  With
// m_live (device, may be NULL) only the rows below min(m, *m_live) are
// computed; the rest of C is left as it was.
tgm_status_t gemm_f32(bool ta, bool tb, int m, int n, int k, const float *A, int lda,
                      const float *B, int ldb, float *C, int ldc, const float *bias,
                      bool accumulate, hipStream_t s, const int32_t *m_live = nullptr);

// The training step of one iteration (tgm_train_step) on stream s, from the
// iteration's sample and fetch buffers, new memories and embeddings.
tgm_status_t train_step_launch(tgm_trainer_t tr, tgm_model_t m, tgm_graph_t g, int32_t b,
                               const tgm_sample_buffers &sb, const tgm_fetch_buffers &fb,
                               const float *mem_new, const float *h, int32_t cap, float *loss_out,
                               hipStream_t s);
tgm_status_t mitigate_prep_launch(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                                  const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                                  int32_t slot, hipStream_t s);
tgm_status_t mitigate_launch(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                             const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                             float *mem, const double *mem_ts, int32_t M, double p, float lambda,
                             int32_t slot, hipStream_t s);

}  // namespace tgm
