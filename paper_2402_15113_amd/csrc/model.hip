// Memory update (GRU + latest-message reduce + staged write-back) and the
// attention embedding.  The dense contractions run on fp32 MFMA
// (v_mfma_f32_16x16x4_f32); everything else is vector code.
#include <algorithm>
#include <cmath>
#include <utility>

#include "common.h"

using namespace tgm;

namespace {

constexpr int kMaxWaves = 8;
constexpr int kCUs = 256;      // compute units of an MI355X
constexpr int kAttMaxCB = 2;   // K|V column blocks per wave
constexpr int kAttMaxRB = 5;   // 16-row slot blocks per workgroup

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + expf(-x)); }

// ------------------------------------------------------------------ GRU
// The work is nrb x MB equal tasks (16-row block rb, 16-wide hidden block hb).
// Persistent grid of kGruGrid workgroups: workgroup w takes a contiguous range
// of tasks (ranges are dealt so that the ranges of one XCD are adjacent, and
// the tasks of one row block mostly meet in one L2) and walks it in rounds of
// at most 4 kGruSlots tasks spanning at most 2 row blocks:
//   the rows' GRU inputs [mail || phi(mail_ts - mem_ts) | mem] are staged in
//   LDS with all their loads in flight together; tasks j and j + 4 q of the
//   round go to wavefronts j and j + 4, which split the reduction (k) range in
//   two halves and stream the weights of their half for each of their tasks,
//   two chunks ahead of the multiply (longer ranges take fewer rounds);
//   each accumulates r and z over [x | h] and n in its x part and its h part
//   (which the reset gate scales); the two halves swap partial sums through
//   LDS, and the lower half applies the gates to the wave's first task, the
//   upper half to its second.
// The hb = 0 tasks also write the new memory timestamps.  The same launch
// runs the batch's latest-message reduce (latest_reduce) first.
constexpr int kGruWaves = 8;
constexpr int kGruGrid = 256;
constexpr int kGruRows = 32;   // rows staged per round (2 row blocks)
constexpr int kGruSlots = 2;   // tasks per wave pair and round (rounds of 4 kGruSlots tasks)

struct GruArgs {
    const int32_t *n_nodes;
    // set (k_gru_w only): mem, mail, mem_ts, mail_ts and ver are the committed
    // tables, read at row nodes[p] for position p of the node set
    const int32_t *nodes;
    const float *mem, *mail;
    const double *mem_ts, *mail_ts;
    const int32_t *ver;
    const f4 *bx, *bh;
    const float *bias;
    const double *omega, *beta;
    int M, D_m, D_t, KXC, KHC, MB;
    float *mem_new;
    double *new_mem_ts;
    // latest-message reduce of the batch (see latest_reduce)
    int32_t n_cand;
    const int32_t *src_pos, *dst_pos;
    uint64_t *win;
    uint64_t tag;   // (update tag) << 32
};

// The weights of k-chunk c (chunks [0, KXC) are the x part, the rest the h
// part) for hidden block hb: gates r, z, n.
struct GruW {
    const f4 *bx, *bh;
    int64_t kstep, gx, gh;
    int KXC, last;   // last: the highest chunk that may be loaded

    // G = 3 gates (GRU: r, z, n) or 1 (the RNN cell: its single gate sits in
    // w[2], where the GRU keeps n)
    template <int G>
    __device__ __forceinline__ void load(int c, int hb, int lane, f4 (&w)[3]) const
    {
        c = c < last ? c : last;
        const bool x = c < KXC;
        const f4 *p = (x ? bx + (int64_t)c * kstep : bh + (int64_t)(c - KXC) * kstep) +
                      (int64_t)hb * kWave + lane;
        const int64_t gs = x ? gx : gh;
        if (G == 3) {
            w[0] = p[0];
            w[1] = p[gs];
            w[2] = p[2 * gs];
        } else {
            w[2] = p[0];
        }
    }
};

template <int G>
__device__ __forceinline__ void gru_mma(const float *arow, int c, int KXC, const f4 (&w)[3],
                                        f4 &ar, f4 &az, f4 &anx, f4 &anh)
{
    const f4 a = *reinterpret_cast<const f4 *>(arow + c * 16);
    if (G == 3) {
        ar = mfma_k16(a, w[0], ar);
        az = mfma_k16(a, w[1], az);
    }
    if (c < KXC)
        anx = mfma_k16(a, w[2], anx);
    else
        anh = mfma_k16(a, w[2], anh);
}

// Rows of one round held in registers between their load and their LDS
// store: wave w takes rows w + 8 i.
template <int W, int CM, int CH>
struct GruRows {
    static constexpr int RR = kGruRows / kGruWaves;
    WaveRows<W, RR, CM> xm;
    WaveRows<W, RR, CH> xh;
    int64_t offm[RR], offh[RR];
    int lr[RR], vv[RR];
    double mt[RR], lt[RR];

    __device__ __forceinline__ void load(const GruArgs &g, int row0, int nrows, int wave,
                                         int lane)
    {
#pragma unroll
        for (int i = 0; i < RR; ++i) {
            const int r = wave + kGruWaves * i;
            const bool live = r < nrows;
            const int p = row0 + (live ? r : 0);   // branch-free: dead rows read the first row
            lr[i] = r;
            vv[i] = g.ver[p];
            mt[i] = g.mem_ts[p];
            lt[i] = g.mail_ts[p];
            offm[i] = live ? (int64_t)p * g.D_m : -1;
            offh[i] = live ? (int64_t)p * g.M : -1;
        }
        xm.load(g.mail, offm, g.D_m, lane);
        xh.load(g.mem, offh, g.M, lane);
    }

    __device__ __forceinline__ void store(const GruArgs &g, float *A, int *s_has, double *s_nts,
                                          int SA, int KX, const double *s_om,
                                          const double *s_be, int nrows, int lane) const
    {
        const int D_m = g.D_m, D_t = g.D_t, M = g.M;
        bool has[RR];
        double dt[RR];
#pragma unroll
        for (int i = 0; i < RR; ++i) {
            has[i] = lr[i] < nrows && vv[i] >= 0;
            dt[i] = lt[i] - mt[i];
        }
        for (int d = lane; d < D_t; d += kWave) {
            const double om = s_om[d], be = s_be[d];
#pragma unroll
            for (int i = 0; i < RR; ++i)
                A[lr[i] * SA + D_m + d] = has[i] ? time_enc(om, be, dt[i]) : 0.f;
        }
        const int padx = KX - D_m - D_t, padh = SA - 4 - KX - M;
#pragma unroll
        for (int i = 0; i < RR; ++i) {
            float *row = A + lr[i] * SA;
            for (int k = lane; k < padx; k += kWave)
                row[D_m + D_t + k] = 0.f;
            for (int k = lane; k < padh; k += kWave)
                row[KX + M + k] = 0.f;
            if (lane == 0) {
                s_has[lr[i]] = has[i];
                s_nts[lr[i]] = has[i] ? lt[i] : mt[i];
            }
        }
        xm.store(A, SA, 0, lr, offm, D_m, lane);
        xh.store(A, SA, KX, lr, offh, M, lane);
    }
};

// Latest-message reduce.  Candidate c = 2 (e - first) + role is the message
// of event first + c/2 to its source (role 0) or destination (role 1).  The
// stream is sorted by (t, e), so the candidate order is the (t, e, role)
// order and the latest message of a node is its largest c: an integer max,
// exact and order-independent.  The slot of a node holds the 64-bit key
// (tag << 32) | c, with a tag that grows with every update call, so a max
// over keys needs no reset between calls: a key of an older call is smaller
// than any key of this one.  Candidates of one wavefront that hit the same
// node are first reduced with lane shuffles (the wave's candidates are
// consecutive, so a node's last lane in the wave holds its wave maximum); only
// that lane issues the atomic.  Thread c of the grid takes candidates c,
// c + (grid threads), ... (a multiple of 64 apart: a wave's candidates stay
// consecutive).
__device__ __forceinline__ void latest_reduce(const GruArgs &g, int n)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
         c - lane < g.n_cand; c += stride) {   // the whole wave past the candidates: done
        int p = c < g.n_cand ? ((c & 1) ? g.dst_pos[c >> 1] : g.src_pos[c >> 1]) : -1;
        const bool live = p >= 0 && p < n;   // positions outside the node set are dropped
        if (!live)
            p = -1 - lane;
        // is there a later lane in this wave with the same position?
        bool later = false;
        for (int o = 1; o < kWave; ++o) {
            const int q = __shfl(p, (lane + o) & (kWave - 1), kWave);
            later |= (lane + o < kWave) && q == p;
        }
        if (live && !later)
            atomicMax(reinterpret_cast<unsigned long long *>(g.win + p),
                      (unsigned long long)(g.tag | (uint64_t)c));
    }
}

// The latest-message reduce on its own (the executor runs it on the prefetch
// stream): only the reduce fields of g are read.
__global__ __launch_bounds__(256) void k_latest(GruArgs g)
{
    latest_reduce(g, *g.n_nodes);
}

template <int W, int CM, int CH, int NG>
__device__ __forceinline__ void gru_body(const GruArgs &g, float *lds, int *s_has,
                                         double *s_nts)
{
    const int n = *g.n_nodes;
    latest_reduce(g, n);
    const int M = g.M, MB = g.MB, D_t = g.D_t, KXC = g.KXC, KHC = g.KHC;
    const int KC = KXC + KHC;
    const int KX = KXC * 16, SA = KC * 16 + 4;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    constexpr int S = kGruSlots;
    float *A = lds;                                              // [kGruRows][SA]
    f4 *red = reinterpret_cast<f4 *>(lds + kGruRows * SA);       // [4 S tasks][4][64]
    double *s_om = reinterpret_cast<double *>(red + 4 * S * 4 * kWave);
    double *s_be = s_om + D_t;

    // this workgroup's task range: range c = (w % 8) * (G / 8) + w / 8, so the
    // ranges of one XCD are adjacent
    const int64_t T = (int64_t)((n + 15) >> 4) * MB;
    const int G = gridDim.x;
    const int c = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
    const int64_t t0 = T * c / G, t1 = T * (c + 1) / G;
    if (t0 >= t1)
        return;

    GruW gw;
    gw.bx = g.bx;
    gw.bh = g.bh;
    gw.kstep = (int64_t)MB * kWave;
    gw.gx = (int64_t)KXC * gw.kstep;
    gw.gh = (int64_t)KHC * gw.kstep;
    gw.KXC = KXC;
    const int j = wave & 3, half = wave >> 2;
    const int kc0 = half ? KC / 2 : 0, kc1 = half ? KC : KC / 2;
    gw.last = kc1 - 1;
    const float *arow0 = A + (lane & 15) * SA + 4 * (lane >> 4);
    const int MP = MB * 16;
    GruRows<W, CM, CH> rows;

    // round geometry: tasks [t, te), rows [row0, row0 + nrows)
    auto round_end = [&](int64_t t) {
        const int64_t rb_a = t / MB;
        return std::min<int64_t>(std::min<int64_t>(t + 4 * S, t1), (rb_a + 2) * MB);
    };
    auto round_rows = [&](int64_t t, int64_t te) {
        const int rb_a = (int)(t / MB);
        return std::min(kGruRows, std::min<int>(n - rb_a * 16,
                                                (int)(((te - 1) / MB - rb_a + 1) * 16)));
    };

    // the first round's rows go out before the time-encoding constants are
    // set up
    int64_t t = t0;
    int64_t te = round_end(t);
    rows.load(g, (int)(t / MB) * 16, round_rows(t, te), wave, lane);
    for (int d = tid; d < D_t; d += blockDim.x) {
        s_om[d] = g.omega[d];
        s_be[d] = g.beta[d];
    }
    for (;;) {
        const int rb_a = (int)(t / MB);
        const int row0 = rb_a * 16;
        const int nrows = round_rows(t, te);
        // slot q of this wave pair: task t + j + 4 q of the round
        bool live[S];
        int hb[S], lrow0[S];
#pragma unroll
        for (int q = 0; q < S; ++q) {
            const int64_t tj = t + j + 4 * q;
            live[q] = tj < te;
            const int rb = live[q] ? (int)(tj / MB) : rb_a;
            hb[q] = live[q] ? (int)(tj - (int64_t)rb * MB) : 0;
            lrow0[q] = (rb - rb_a) * 16;
        }
        // the first two weight chunks load while the rows are staged
        f4 w0[S][3], w1[S][3], w2[S][3];
#pragma unroll
        for (int q = 0; q < S; ++q)
            if (live[q]) {
                gw.load<NG>(kc0, hb[q], lane, w0[q]);
                gw.load<NG>(kc0 + 1, hb[q], lane, w1[q]);
            }
        __syncthreads();   // s_om is written; the previous round is done with LDS
        rows.store(g, A, s_has, s_nts, SA, KX, s_om, s_be, nrows, lane);
        __syncthreads();

        f4 ar[S], az[S], anx[S], anh[S];
#pragma unroll
        for (int q = 0; q < S; ++q)
            ar[q] = az[q] = anx[q] = anh[q] = f4{0, 0, 0, 0};
        if (live[0]) {
            // three weight sets rotate: chunk c + 2 loads while chunk c
            // multiplies; each chunk serves the wave's live slots
            for (int cc = kc0; cc < kc1; cc += 3) {
#pragma unroll
                for (int q = 0; q < S; ++q)
                    if (live[q])
                        gw.load<NG>(cc + 2, hb[q], lane, w2[q]);
                issue_fence();
#pragma unroll
                for (int q = 0; q < S; ++q)
                    if (live[q])
                        gru_mma<NG>(arow0 + lrow0[q] * SA, cc, KXC, w0[q], ar[q], az[q], anx[q],
                                    anh[q]);
#pragma unroll
                for (int q = 0; q < S; ++q)
                    if (live[q])
                        gw.load<NG>(cc + 3, hb[q], lane, w0[q]);
                issue_fence();
                if (cc + 1 < kc1)
#pragma unroll
                    for (int q = 0; q < S; ++q)
                        if (live[q])
                            gru_mma<NG>(arow0 + lrow0[q] * SA, cc + 1, KXC, w1[q], ar[q], az[q],
                                        anx[q], anh[q]);
#pragma unroll
                for (int q = 0; q < S; ++q)
                    if (live[q])
                        gw.load<NG>(cc + 4, hb[q], lane, w1[q]);
                issue_fence();
                if (cc + 2 < kc1)
#pragma unroll
                    for (int q = 0; q < S; ++q)
                        if (live[q])
                            gru_mma<NG>(arow0 + lrow0[q] * SA, cc + 2, KXC, w2[q], ar[q], az[q],
                                        anx[q], anh[q]);
            }
            // swap partial sums: slot 0 is finished by the lower half and slot
            // 1 by the upper half, each handing the other its sums
            const int give = half ? 0 : 1;
            if (live[give]) {
                f4 *rw = red + ((j + 4 * give) * 4) * kWave + lane;
                rw[0] = give ? ar[1] : ar[0];
                rw[kWave] = give ? az[1] : az[0];
                rw[2 * kWave] = give ? anx[1] : anx[0];
                rw[3 * kWave] = give ? anh[1] : anh[0];
            }
        }
        const int64_t tn = te;
        const int64_t ten = tn < t1 ? round_end(tn) : tn;
        if (tn < t1)   // the next round's rows, in flight during the epilogue
            rows.load(g, (int)(tn / MB) * 16, round_rows(tn, ten), wave, lane);
        __syncthreads();
        {
            const int q = half;   // the slot this wave finishes
            if (live[q]) {
                // lane holds values v = 0..3 of rows 4 (lane / 16) + v, column
                // hb 16 + lane % 16
                const f4 *rq = red + ((j + 4 * q) * 4) * kWave + lane;
                const f4 sr = (q ? ar[1] : ar[0]) + rq[0], sz = (q ? az[1] : az[0]) + rq[kWave];
                const f4 snx = (q ? anx[1] : anx[0]) + rq[2 * kWave];
                const f4 snh = (q ? anh[1] : anh[0]) + rq[3 * kWave];
                const int hbq = q ? hb[1] : hb[0], lrq = q ? lrow0[1] : lrow0[0];
                const int col = hbq * 16 + (lane & 15);
                const int colc = col < M ? col : 0;
                const float b_r = g.bias[colc], b_z = g.bias[MP + colc];
                const float b_nx = g.bias[2 * MP + colc], b_nh = g.bias[3 * MP + colc];
                if (col < M) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int lr = lrq + 4 * (lane >> 4) + v;
                        const int p = row0 + lr;
                        if (p < n) {
                            const float h = A[lr * SA + KX + col];
                            float o = h;
                            if (s_has[lr]) {
                                if (NG == 3) {
                                    const float r = sigmoidf_(sr[v] + b_r);
                                    const float z = sigmoidf_(sz[v] + b_z);
                                    const float nn = tanhf(snx[v] + b_nx + r * (snh[v] + b_nh));
                                    o = (1.0f - z) * nn + z * h;
                                } else {   // the RNN cell
                                    o = tanhf((snx[v] + b_nx) + (snh[v] + b_nh));
                                }
                            }
                            g.mem_new[(int64_t)p * M + col] = o;
                        }
                    }
                }
                if (hbq == 0 && g.new_mem_ts && lane < 16 && row0 + lrq + lane < n)
                    g.new_mem_ts[row0 + lrq + lane] = s_nts[lrq + lane];
            }
        }
        if (tn >= t1)
            break;
        t = tn;
        te = ten;
    }
}

// NG = 3: the GRU cell; NG = 1: the RNN cell (JODIE), same pipeline.
template <int NG>
__global__ __launch_bounds__(64 * kGruWaves) void k_gru(GruArgs g)
{
    extern __shared__ float lds[];
    __shared__ int s_has[kGruRows];
    __shared__ double s_nts[kGruRows];
    const bool al = ((reinterpret_cast<uintptr_t>(g.mail) | reinterpret_cast<uintptr_t>(g.mem)) &
                     15) == 0 &&
                    (g.D_m & 3) == 0 && (g.M & 3) == 0;   // 16-byte rows: vector loads
    if (al)
        gru_body<4, 2, 1, NG>(g, lds, s_has, s_nts);   // D_m <= 512, M <= 256
    else
        gru_body<1, 8, 2, NG>(g, lds, s_has, s_nts);
}

// ------------------------------------------------------------------ GRU, weights resident
// The same cell as k_gru with the operands the other way round: workgroup b
// owns hidden block hb = b % MB, keeps that block's weight fragments (all k
// chunks, every gate) in LDS for the whole launch, and streams the rows of
// its range of 16-row blocks through them.  Wavefronts j and j + 4 (one SIMD)
// split the k range of a row block in two halves, as in k_gru; the four
// pairs take the range's row blocks four at a time.  The A operand comes
// straight from the fetched rows in global memory (mail || phi | mem), kGwDepth
// chunks ahead of the multiply, where phi(mail_ts - mem_ts) was formed once
// per node by k_phi.  After a row block the two halves swap the partial sums
// of two of the four rows each lane holds and apply the gates to the other
// two.
#ifndef GW_DEPTH
#define GW_DEPTH 4
#endif
constexpr int kGwDepth = GW_DEPTH;   // A chunks in flight per wavefront
#ifndef GW_J
#define GW_J 4
#endif
constexpr int kGwJ = GW_J;              // row blocks per step (wavefront pairs)
constexpr int kGwWaves = 2 * kGwJ;
constexpr int kGwBufs = kGwJ <= 4 ? 2 : 1;   // swap areas (alternating between steps)
// k-chunks of k_gru_w's weights: KC rounded up to a multiple of 2 kGwDepth
__host__ __device__ constexpr int gw_chunks(int KC)
{
    return (KC + 2 * kGwDepth - 1) / (2 * kGwDepth) * (2 * kGwDepth);
}

// phi[p][d] = cos(omega_d (mail_ts - mem_ts) + beta_d) for the nodes of the
// set that hold mail (zero otherwise): the time part of the GRU input.
__global__ __launch_bounds__(256) void k_phi(const int32_t *__restrict__ n_nodes, int32_t cap,
                                             int D_t, const double *__restrict__ mem_ts,
                                             const double *__restrict__ mail_ts,
                                             const int32_t *__restrict__ ver,
                                             const double *__restrict__ omega,
                                             const double *__restrict__ beta,
                                             float *__restrict__ phi)
{
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int n = min(*n_nodes, cap);
    if (i >= (int64_t)n * D_t)
        return;
    const int p = (int)(i / D_t), d = (int)(i - (int64_t)p * D_t);
    phi[i] = ver[p] >= 0 ? time_enc(omega[d], beta[d], mail_ts[p] - mem_ts[p]) : 0.f;
}

// A fragment of k-chunk c for row p (lane holds k = 16 c + 4 (lane / 16) + 0..3),
// as two 8-byte pairs: x chunks from the mail row and phi (D_m and D_t even,
// so a pair never straddles a boundary), h chunks from the memory row.  Past
// each part the pair is read from the row's start instead: the packed weights
// are zero there, and every value read is finite, so those products add zero.
// Only addresses are selected: a select on a loaded value would make the
// compiler wait for the load where the select is.
struct GwA {
    f2 lo, hi;
};

__device__ __forceinline__ GwA gw_a(const GruArgs &g, const float *mrow, const float *frow,
                                    const float *hrow, int c, int lane)
{
    // global address space spelled out: a pointer picked by a select would
    // otherwise be loaded as a flat address, which the LDS counter also counts
    typedef const f2 __attribute__((address_space(1))) *gf2;
    const int KXC = g.KXC, D_m = g.D_m, D_x = g.D_m + g.D_t;
    const float *s0, *s1;
    // a chunk wholly inside one part of the row (the test is the same in
    // every lane) takes one address; only the chunks that straddle a part's
    // end choose per lane
    if (c < KXC) {
        const int k0 = 16 * c, k = k0 + 4 * (lane >> 4), k1 = k + 2;
        if (k0 + 16 <= D_m) {
            s0 = mrow + k;
            s1 = s0 + 2;
        } else if (k0 >= D_m && k0 + 16 <= D_x) {
            s0 = frow + (k - D_m);
            s1 = s0 + 2;
        } else {
            s0 = k < D_m ? mrow + k : (k < D_x ? frow + (k - D_m) : mrow);
            s1 = k1 < D_m ? mrow + k1 : (k1 < D_x ? frow + (k1 - D_m) : mrow);
        }
    } else {
        const int k0 = 16 * (c - KXC), k = k0 + 4 * (lane >> 4);
        if (k0 + 16 <= g.M) {
            s0 = hrow + k;
            s1 = s0 + 2;
        } else {
            s0 = k < g.M ? hrow + k : hrow;
            s1 = k < g.M ? hrow + k + 2 : hrow;
        }
    }
    return GwA{*(gf2)(s0), *(gf2)(s1)};
}

template <int NG>
__global__ __launch_bounds__(64 * kGwWaves) void k_gru_w(GruArgs g, const float *phi)
{
    extern __shared__ float lds[];
    const int n = *g.n_nodes;
    latest_reduce(g, n);
    const int M = g.M, MB = g.MB, KXC = g.KXC, KC = g.KXC + g.KHC, D_t = g.D_t;
    const int KCP = gw_chunks(KC);   // with zero chunks: each half a whole number of ring rounds
    // workgroup b runs on XCD b % 8; its slot counts XCD-major (the 32 slots
    // of XCD 0 first), and slots [r MB, (r + 1) MB) take the MB blocks of
    // row range r, so a range's rows are read by at most two XCDs' L2s
    const int G = (int)gridDim.x;
    const int slot = ((int)blockIdx.x & 7) * (G >> 3) + ((int)blockIdx.x >> 3);
    const int R = G / MB;   // row-block ranges
    const int hb = slot % MB, r = slot / MB;
    const int nrb = (n + 15) >> 4;
    const int rb0 = (int)((int64_t)nrb * r / R), rb1 = (int)((int64_t)nrb * (r + 1) / R);
    if (r >= R || rb0 >= rb1)
        return;
    const int tid = threadIdx.x, lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int j = wave % kGwJ, half = wave / kGwJ;
    const int kc0 = half ? KCP / 2 : 0, kc1 = half ? KCP : KCP / 2;
    f4 *W = reinterpret_cast<f4 *>(lds);   // [KCP][NG][64] fragments of block hb
    f2 *red = reinterpret_cast<f2 *>(W + (int64_t)KCP * NG * kWave);   // [bufs][J][2][4][64]

    // the rows of this pair's first block, then the weights of block hb
    const int steps = (rb1 - rb0 + kGwJ - 1) / kGwJ;
    int rb = rb0 + j;
    const int vm = half ? 2 : 0;   // the two of a lane's four rows this wave finishes
    // Position p of the node set reads row p of the fetched rows, or (g.nodes
    // set) the committed tables' row of node nodes[p]: the ids of a step's
    // epilogue rows load a step ahead, those of its A rows two steps ahead
    // (the step before reads the A rows' first chunks).  phi stays by
    // position.
    auto node_of = [&](int p) -> int { return g.nodes ? g.nodes[p] : p; };
    auto a_pos = [&](int b) { return min(min(b, rb1 - 1) * 16 + (lane & 15), n - 1); };
    auto e_pos = [&](int b, int u) {
        return min(min(b, rb1 - 1) * 16 + 4 * (lane >> 4) + vm + u, n - 1);
    };
    auto rows_of = [&](int p, int v, const float *&mrow, const float *&frow, const float *&hrow) {
        mrow = g.mail + (int64_t)v * g.D_m;   // rows past n repeat the last
        frow = phi + (int64_t)p * D_t;
        hrow = g.mem + (int64_t)v * M;
    };
    const float *mrow, *frow, *hrow;
    {
        const int p = a_pos(rb);
        rows_of(p, node_of(p), mrow, frow, hrow);
    }
    int ve[2] = {node_of(e_pos(rb, 0)), node_of(e_pos(rb, 1))};
    int va1 = node_of(a_pos(rb + kGwJ));   // the A rows' ids of the next step
    GwA ring[kGwDepth];
#pragma unroll
    for (int q = 0; q < kGwDepth; ++q)
        ring[q] = gw_a(g, mrow, frow, hrow, min(kc0 + q, kc1 - 1), lane);
    {
        // sixteen fragments per thread in flight before their LDS stores
        const int64_t kstep = (int64_t)MB * kWave;
        const int64_t gx = (int64_t)KXC * kstep, gh = (int64_t)g.KHC * kstep;
        const int total = KCP * NG * kWave;
        for (int i0 = 0; i0 < total; i0 += 16 * (int)blockDim.x) {
            f4 v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int i = min(i0 + u * (int)blockDim.x + tid, KC * NG * kWave - 1);
                const int l = i & (kWave - 1), cq = i >> 6, c = cq / NG, q = cq - c * NG;
                const bool x = c < KXC;
                const f4 *src = (x ? g.bx + (int64_t)c * kstep
                                   : g.bh + (int64_t)(c - KXC) * kstep) +
                                (int64_t)hb * kWave + l;
                v[u] = src[q * (x ? gx : gh)];
            }
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int i = i0 + u * (int)blockDim.x + tid;
                if (i < total)
                    W[i] = i < KC * NG * kWave ? v[u] : f4{0, 0, 0, 0};   // padding chunks
            }
        }
    }
    const int MP = MB * 16;
    const int col = hb * 16 + (lane & 15);
    const int colc = col < M ? col : 0;
    const float b_r = g.bias[colc], b_z = g.bias[MP + colc];
    const float b_nx = g.bias[2 * MP + colc], b_nh = g.bias[3 * MP + colc];
    lds_barrier();   // the weights are in LDS; the A chunks stay in flight

    for (int st = 0; st < steps; ++st, rb += kGwJ) {
        const bool live = rb < rb1;
        // the epilogue's inputs of this wave's two rows, in flight during the
        // multiply, and the next step's row ids
        float h2[2];
        int has2[2];
        double nts2[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int v = ve[u];
            h2[u] = g.mem[(int64_t)v * M + colc];
            has2[u] = g.ver[v] >= 0;
            nts2[u] = has2[u] ? g.mail_ts[v] : g.mem_ts[v];
        }
        // the next step's A rows (their ids loaded a step ago), and the ids
        // of the step after
        const float *mrow_n, *frow_n, *hrow_n;
        rows_of(a_pos(rb + kGwJ), va1, mrow_n, frow_n, hrow_n);
        va1 = node_of(a_pos(rb + 2 * kGwJ));
#pragma unroll
        for (int u = 0; u < 2; ++u)
            ve[u] = node_of(e_pos(rb + kGwJ, u));
        f4 ar = {0, 0, 0, 0}, az = ar, anx = ar, anh = ar;
        if (live) {
            // chunk c multiplies from ring slot (c - kc0) % kGwDepth, which
            // then loads chunk c + kGwDepth, or past kc1 the next row block's
            // chunk kc0 + (c + kGwDepth - kc1) (kc1 - kc0 is a multiple of
            // kGwDepth, so that chunk lands in its slot; after the last block
            // the rows repeat the range's last); the B fragments of chunk c + 1
            // are read from LDS before chunk c multiplies
            f4 bw[3], bn[3];
            auto b_read = [&](int c, f4(&b)[3]) {
                const f4 *wb = W + (int64_t)min(c, kc1 - 1) * NG * kWave + lane;
#pragma unroll
                for (int q = 0; q < NG; ++q)
                    b[q] = wb[q * kWave];
            };
            b_read(kc0, bw);
            for (int c0 = kc0; c0 < kc1; c0 += kGwDepth) {
#pragma unroll
                for (int q = 0; q < kGwDepth; ++q) {
                    const int c = c0 + q;
                    {
                        const f4 a = {ring[q].lo[0], ring[q].lo[1], ring[q].hi[0],
                                      ring[q].hi[1]};
                        b_read(c + 1, bn);
                        if (NG == 3) {
                            ar = mfma_k16(a, bw[0], ar);
                            az = mfma_k16(a, bw[1], az);
                            if (c < KXC)
                                anx = mfma_k16(a, bw[2], anx);
                            else
                                anh = mfma_k16(a, bw[2], anh);
                        } else {
                            if (c < KXC)
                                anx = mfma_k16(a, bw[0], anx);
                            else
                                anh = mfma_k16(a, bw[0], anh);
                        }
                        const int cn = c + kGwDepth;
                        const bool nx = cn >= kc1;
                        ring[q] = gw_a(g, nx ? mrow_n : mrow, nx ? frow_n : frow,
                                       nx ? hrow_n : hrow, nx ? kc0 + (cn - kc1) : cn, lane);
#pragma unroll
                        for (int u = 0; u < NG; ++u)
                            bw[u] = bn[u];
                    }
                    issue_fence();
                }
            }
        }
        mrow = mrow_n;
        frow = frow_n;
        hrow = hrow_n;
        // values v = 0..3 of rows 4 (lane / 16) + v: the lower half keeps v =
        // 0, 1 and hands over v = 2, 3; the upper half the reverse
        // (with two swap areas they alternate between steps, so a step's sums
        // never land where the previous step's are still being read; with one,
        // a second barrier follows the reads)
        f2 *rs = red + (kGwBufs == 2 ? (st & 1) : 0) * (kGwJ * 2 * 4 * kWave);
        f2 *rw = rs + ((j * 2 + half) * 4) * kWave + lane;
        const int vo = half ? 0 : 2;
        if (live) {
            rw[0] = f2{ar[vo], ar[vo + 1]};
            rw[kWave] = f2{az[vo], az[vo + 1]};
            rw[2 * kWave] = f2{anx[vo], anx[vo + 1]};
            rw[3 * kWave] = f2{anh[vo], anh[vo + 1]};
        }
        lds_barrier();   // the next block's A chunks stay in flight
        f2 pr = {0, 0}, pz = pr, pnx = pr, pnh = pr;
        if (live) {
            const f2 *ro = rs + ((j * 2 + (half ^ 1)) * 4) * kWave + lane;
            pr = ro[0];
            pz = ro[kWave];
            pnx = ro[2 * kWave];
            pnh = ro[3 * kWave];
        }
        if (kGwBufs == 1)
            lds_barrier();   // every read of the swap area done before the next writes
        if (live) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int v = vm + u;
                const int p = rb * 16 + 4 * (lane >> 4) + v;
                if (p < n && col < M) {
                    const float h = h2[u];
                    float o = h;
                    if (has2[u]) {
                        if (NG == 3) {
                            const float rr = sigmoidf_(ar[v] + pr[u] + b_r);
                            const float z = sigmoidf_(az[v] + pz[u] + b_z);
                            const float nn =
                                tanhf(anx[v] + pnx[u] + b_nx + rr * (anh[v] + pnh[u] + b_nh));
                            o = (1.0f - z) * nn + z * h;
                        } else {   // the RNN cell
                            o = tanhf((anx[v] + pnx[u] + b_nx) + (anh[v] + pnh[u] + b_nh));
                        }
                    }
                    g.mem_new[(int64_t)p * M + col] = o;
                    if (hb == 0 && g.new_mem_ts && (lane & 15) == 0)
                        g.new_mem_ts[p] = nts2[u];
                }
            }
        }
    }
}

// LDS of k_gru_w: the weight fragments of one hidden block and the swap area
size_t gru_w_lds(const tgm_model *m, int NG)
{
    return (size_t)gw_chunks(m->KXC + m->KHC) * NG * kWave * 16 +
           kGwBufs * kGwJ * 2 * 4 * kWave * 8;
}

// Shapes k_gru_w handles: 8-byte pairs of the mail row, phi and the memory
// row; the weights of a hidden block within the LDS
bool gru_w_fits(const tgm_model *m, int NG)
{
    return m->D_m % 2 == 0 && m->D_t % 2 == 0 && m->M % 4 == 0 && m->MB <= kGruGrid &&
           gru_w_lds(m, NG) <= 160 * 1024;
}

// JODIE's embedding: the time projection h[r] = s'[p] * (1 + w_t (t_r - ts'[p]))
// of root r's updated memory (p = root_pos[r]), in fp64, one thread per
// element of h.  A position outside the node set yields a zero row.
struct TprojArgs {
    int32_t R = 0, M = 0;
    const int32_t *root_pos = nullptr, *n_nodes = nullptr;
    const double *root_ts = nullptr, *nts = nullptr;
    const float *mem_new = nullptr, *w_t = nullptr;
    float *h = nullptr;
};

__device__ __forceinline__ void tproj_elem(const TprojArgs &a, int64_t i, int n)
{
    const int r = (int)(i / a.M), c = (int)(i - (int64_t)r * a.M);
    const int p = a.root_pos[r];
    float o = 0.f;
    if (p >= 0 && p < n) {
        const double d = a.root_ts[r] - a.nts[p];
        o = (float)((double)a.mem_new[(int64_t)p * a.M + c] * (1.0 + (double)a.w_t[c] * d));
    }
    a.h[i] = o;
}

__global__ __launch_bounds__(256) void k_tproj(TprojArgs a)
{
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i < (int64_t)a.R * a.M)
        tproj_elem(a, i, *a.n_nodes);
}

// The projection and the gather of the next fetch in one launch: the last
// n_tp blocks project, the others gather (kGatherNPW nodes per wavefront).
__global__ __launch_bounds__(256) void k_tproj_gather(TprojArgs a, int n_tp, GatherPlan gp)
{
    // the gather's blocks come first: their row copies are the longer chains,
    // and the projection's small blocks fill the CUs around them
    const int n_gather = (int)gridDim.x - n_tp;
    if ((int)blockIdx.x >= n_gather) {
        const int64_t i = (blockIdx.x - n_gather) * (int64_t)blockDim.x + threadIdx.x;
        if (i < (int64_t)a.R * a.M)
            tproj_elem(a, i, *a.n_nodes);
        return;
    }
    gather_blocks(gp, (int)blockIdx.x, n_gather, blockDim.x >> 6, threadIdx.x >> 6,
                  threadIdx.x & 63);
}

// Stage the write set of iteration i, and commit an older one, in one launch.
// Wavefronts c < n_cand each take one candidate of iteration i: the winning
// candidate of its node writes the node's new memory, its message
// [s'_self || s'_other || efeat[e]] and the timestamps -- into the ring slot of
// iteration i, or straight into the tables when the staleness is 0.
// Wavefronts n_cand <= c < n_cand + n_commit copy the flagged rows of the ring
// slot of iteration c_iter (= i - s) into the tables: every fetch up to
// iteration i has already been issued, and the next one needs exactly the
// writes through i - s.
struct StageArgs {
    int32_t n_cand, n_commit;
    int64_t first, iter, c_iter;
    int M, D_m, D_e;
    bool direct;
    const int32_t *n_nodes, *src, *dst, *src_pos, *dst_pos, *ver;
    const uint64_t *win;
    uint64_t tag;   // (update tag) << 32
    const double *t, *mem_ts, *mail_ts;
    // the new memory times of the node set (written by the GRU launch), read
    // instead of ver / mem_ts / mail_ts when set (the GRU read the tables in
    // place, and no fetched rows exist)
    const double *nts_new;
    const float *efeat, *mem_new;
    // destination ring slot of iteration i
    int32_t *r_flag, *r_node;
    float *r_mem, *r_mail;
    double *r_mem_ts, *r_mail_ts;
    // ring slot committed in this launch
    const int32_t *c_flag, *c_node;
    const float *c_mem, *c_mail;
    const double *c_mem_ts, *c_mail_ts;
    // committed tables
    float *mem, *mail;
    double *t_mem_ts, *t_mail_ts;
    int32_t *t_ver;
};

// Wavefront work item c of a staging launch (see StageArgs).
__device__ __forceinline__ void stage_wave(const StageArgs &g, int c, int lane)
{
    const int M = g.M, D_m = g.D_m, D_e = g.D_e;
    if (c >= g.n_cand) {
        const int k = c - g.n_cand;
        if (k >= g.n_commit || !g.c_flag[k])
            return;
        const int32_t v = g.c_node[k];
        double mts = 0.0, lts = 0.0;
        if (lane == 0) {
            mts = g.c_mem_ts[k];
            lts = g.c_mail_ts[k];
        }
        wave_copy_2rows(g.mem + (int64_t)v * M, g.c_mem + (int64_t)k * M, M,
                        g.mail + (int64_t)v * D_m, g.c_mail + (int64_t)k * D_m, D_m, lane);
        if (lane == 0) {
            g.t_mem_ts[v] = mts;
            g.t_mail_ts[v] = lts;
            g.t_ver[v] = (int32_t)g.c_iter;
        }
        return;
    }
    const int k = c >> 1, role = c & 1;
    const int n = *g.n_nodes;
    const int p = role ? g.dst_pos[k] : g.src_pos[k];
    const int q = role ? g.src_pos[k] : g.dst_pos[k];
    if (p < 0 || p >= n || q < 0 || q >= n || g.win[p] != (g.tag | (uint64_t)c)) {
        if (lane == 0 && !g.direct)
            g.r_flag[c] = 0;
        return;
    }
    const int64_t e = g.first + k;
    const int32_t w = role ? g.dst[e] : g.src[e];
    const float *sp = g.mem_new + (int64_t)p * M;
    float *dm = g.direct ? g.mem + (int64_t)w * M : g.r_mem + (int64_t)c * M;
    float *ml = g.direct ? g.mail + (int64_t)w * D_m : g.r_mail + (int64_t)c * D_m;
    const float *sq = g.mem_new + (int64_t)q * M, *fe = g.efeat + e * D_e;
    if (M % 4 == 0 && M <= 4 * kWave && D_e % 2 == 0 && D_m <= 8 * kWave &&
        ((reinterpret_cast<uintptr_t>(sp) | reinterpret_cast<uintptr_t>(sq) |
          reinterpret_cast<uintptr_t>(dm)) & 15) == 0 &&
        ((reinterpret_cast<uintptr_t>(ml) | reinterpret_cast<uintptr_t>(fe)) & 7) == 0) {
        // vector accesses: the memory row in 16-byte, the message
        // [s'_p || s'_q || efeat] in 8-byte pieces (pair i of the message
        // comes from s'_p, s'_q or the feature row); every load first
        const int m4 = M / 4, h2 = M / 2, n2 = D_m / 2;
        const f4 a = reinterpret_cast<const f4 *>(sp)[min(lane, m4 - 1)];
        f2 b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = min(lane + kWave * u, n2 - 1);
            const float *src = i < h2 ? sp + 2 * i : (i < M ? sq + 2 * (i - h2) : fe + 2 * (i - M));
            b[u] = *reinterpret_cast<const f2 *>(src);
        }
        if (lane < m4)
            reinterpret_cast<f4 *>(dm)[lane] = a;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (lane + kWave * u < n2)
                reinterpret_cast<f2 *>(ml)[lane + kWave * u] = b[u];
    } else if (M <= 2 * kWave && D_e <= 4 * kWave) {
        // every load before the first store: s'_p, s'_q and the feature row
        // (lane l holds elements l + 64 u, clamped indices)
        float a[2], bq[2], f[4];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            a[u] = sp[min(lane + kWave * u, M - 1)];
            bq[u] = sq[min(lane + kWave * u, M - 1)];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            f[u] = D_e > 0 ? fe[min(lane + kWave * u, D_e - 1)] : 0.f;
#pragma unroll
        for (int u = 0; u < 2; ++u)
            if (lane + kWave * u < M) {
                dm[lane + kWave * u] = a[u];
                ml[lane + kWave * u] = a[u];
                ml[M + lane + kWave * u] = bq[u];
            }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (lane + kWave * u < D_e)
                ml[2 * M + lane + kWave * u] = f[u];
    } else {
        wave_copy_row(dm, sp, M, lane);
        wave_copy_row(ml, sp, M, lane);
        wave_copy_row(ml + M, g.mem_new + (int64_t)q * M, M, lane);
        if (D_e > 0)
            wave_copy_row(ml + 2 * M, g.efeat + e * D_e, D_e, lane);
    }
    if (lane == 0) {
        const double mts =
            g.nts_new ? g.nts_new[p] : (g.ver[p] >= 0 ? g.mail_ts[p] : g.mem_ts[p]);
        if (g.direct) {
            g.t_mem_ts[w] = mts;
            g.t_mail_ts[w] = g.t[e];
            g.t_ver[w] = (int32_t)g.iter;
        } else {
            g.r_flag[c] = 1;
            g.r_node[c] = w;
            g.r_mem_ts[c] = mts;
            g.r_mail_ts[c] = g.t[e];
        }
    }
}

__global__ __launch_bounds__(256) void k_stage(StageArgs g)
{
    stage_wave(g, (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6),
               threadIdx.x & 63);
}

__global__ void k_fill_u64(uint64_t *__restrict__ p, int32_t n)
{
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < n)
        p[k] = 0;
}

__global__ void k_winner_out(const int32_t *__restrict__ n_nodes, int32_t cap, int64_t first,
                             const uint64_t *__restrict__ win, uint64_t tag,
                             int64_t *__restrict__ winner)
{
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= cap || p >= *n_nodes)
        return;
    const uint64_t key = win[p];
    winner[p] = (key >> 32) == (tag >> 32) ? 2 * first + (int64_t)(key & 0xffffffffu) : -1;
}

// ------------------------------------------------------------------ embed
// Node projections P[p] = s'_p [W_q^s; W_k^s; W_v^s]^T: the memory part of the
// query, key and value projections depends only on the node, so it is
// computed once per node of the set instead of once per slot.
constexpr int kProjMaxPC = 8;   // k-chunks of the node projection (K = M <= 128)

// Persistent over 16-row tiles.  The PNB column blocks are split into CS
// contiguous groups of at most nw blocks (launched with nw = 4..8 waves):
// workgroup b takes group b % CS of tiles b / CS, b / CS + nblk / CS, ...,
// so a node set of few tiles still spreads over CS times as many CUs.  Wave w
// owns block w of its group and keeps that block's weights in registers,
// loaded once while the first tile's rows are in flight; the next tile's rows
// load while a tile multiplies.  Two accumulators alternate over the k steps.
// PCM: the k-chunks held in registers (PC <= PCM).
template <int W, int C, int PCM>
__device__ __forceinline__ void node_proj_body(int n, const float *__restrict__ mem_new, int M,
                                               int PC, const f4 *__restrict__ pb, int PNB,
                                               int CS, const float *__restrict__ pbias,
                                               float *__restrict__ P, float *lds, int bid,
                                               int nblk)
{
    const int K = PC * 16, SA = K + 4, ldP = PNB * 16;
    const int nw = blockDim.x >> 6;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int per = (PNB + CS - 1) / CS;
    const int lo = (bid % CS) * per, hi = min(PNB, lo + per);
    const bool has_cb = lo + wave < hi;
    const int cb = has_cb ? lo + wave : lo;
    const float *arow = lds + (lane & 15) * SA + 4 * (lane >> 4);

    // rows of tile row0: wave w takes rows w + nw i (nw >= 4)
    int64_t off[4];
    int lr[4];
    auto rows_of = [&](int row0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wave + nw * i;
            lr[i] = r < 16 ? r : -1;
            off[i] = (r < 16 && row0 + r < n) ? (int64_t)(row0 + r) * M : -1;
        }
    };
    const int tstep = (nblk / CS) * 16;
    int row0 = (bid / CS) * 16;
    WaveRows<W, 4, C> x;
    rows_of(row0);
    x.load(mem_new, off, M, lane);
    f4 w[PCM];
    const int64_t kstep = (int64_t)PNB * kWave;
#pragma unroll
    for (int kc = 0; kc < PCM; ++kc)   // chunks past PC reload chunk 0, unused
        w[kc] = pb[(int64_t)(kc < PC ? kc : 0) * kstep + (int64_t)cb * kWave + lane];
    const float e0 = pbias[cb * 16 + (lane & 15)];
    for (;;) {
        __syncthreads();   // the previous tile is done with LDS
        x.store(lds, SA, 0, lr, off, M, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (lr[i] >= 0)
                for (int k = M + lane; k < K; k += kWave)
                    lds[lr[i] * SA + k] = 0.f;
        __syncthreads();
        const int next = row0 + tstep;
        if (next < n) {
            rows_of(next);
            x.load(mem_new, off, M, lane);
        }
        if (has_cb) {
            f4 c0 = {0, 0, 0, 0}, c1 = c0;
#pragma unroll
            for (int kc = 0; kc < PCM; ++kc) {
                if (kc < PC) {
                    const f4 a = *reinterpret_cast<const f4 *>(arow + kc * 16);
                    c0 = mfma_16x16x4(a[0], w[kc][0], c0);
                    c1 = mfma_16x16x4(a[1], w[kc][1], c1);
                    c0 = mfma_16x16x4(a[2], w[kc][2], c0);
                    c1 = mfma_16x16x4(a[3], w[kc][3], c1);
                }
            }
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int r = row0 + 4 * (lane >> 4) + v;
                if (r < n)
                    P[(int64_t)r * ldP + cb * 16 + (lane & 15)] = (c0[v] + c1[v]) + e0;
            }
        }
        if (next >= n)
            break;
        row0 = next;
    }
}

struct ProjArgs {
    const int32_t *n_nodes;
    const float *mem_new;
    int M, PC, PNB, CS;   // CS: column groups of the node projection
    const f4 *pb;
    const float *pbias;
    float *P;
};

// Block bid of nblk node-projection blocks.  LEAN: the caller has checked
// lean_proj() (M % 4 == 0, 16-byte aligned rows, at most 7 k-chunks), so only
// the variant with seven weight chunks in registers is compiled in.
template <bool LEAN>
__device__ __forceinline__ void node_proj_block(const ProjArgs &a, float *lds, int bid, int nblk)
{
    const int n = *a.n_nodes;
    if ((bid / a.CS) * 16 >= n || bid >= (nblk / a.CS) * a.CS)
        return;
    if (LEAN)
        node_proj_body<4, 1, kProjMaxPC - 1>(n, a.mem_new, a.M, a.PC, a.pb, a.PNB, a.CS, a.pbias,
                                             a.P, lds, bid, nblk);
    else if ((a.M & 3) == 0 && (reinterpret_cast<uintptr_t>(a.mem_new) & 15) == 0)
        node_proj_body<4, 1, kProjMaxPC>(n, a.mem_new, a.M, a.PC, a.pb, a.PNB, a.CS, a.pbias, a.P,
                                         lds, bid, nblk);
    else
        node_proj_body<1, 2, kProjMaxPC>(n, a.mem_new, a.M, a.PC, a.pb, a.PNB, a.CS, a.pbias, a.P,
                                         lds, bid, nblk);
}

bool lean_proj(const ProjArgs &a)
{
    return (a.M & 3) == 0 && (reinterpret_cast<uintptr_t>(a.mem_new) & 15) == 0 &&
           a.PC <= kProjMaxPC - 1;
}

__global__ __launch_bounds__(512) void k_node_proj(ProjArgs a)
{
    extern __shared__ float lds[];
    node_proj_block<false>(a, lds, blockIdx.x, gridDim.x);
}

// The staging of a write set and the node projections in one launch: blocks
// [0, n_proj) project, the rest stage (one wavefront per staging item).  The
// lean variant is held to 80 VGPRs (six waves per SIMD), so a CU that holds
// two projection workgroups has room for a staging workgroup beside them.
template <bool LEAN>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(LEAN ? 6 : 1))) void k_stage_proj(StageArgs sa, ProjArgs pa, int n_proj)
{
    extern __shared__ float lds[];
    if ((int)blockIdx.x < n_proj) {
        node_proj_block<LEAN>(pa, lds, blockIdx.x, n_proj);
        return;
    }
    const int waves = blockDim.x >> 6;
    stage_wave(sa, ((int)blockIdx.x - n_proj) * waves + (int)(threadIdx.x >> 6), threadIdx.x & 63);
}

struct AttnArgs {
    int R, nb, RT, RBa, M, H, D_e, D_t;
    int64_t E;
    const int32_t *n_nodes;
    const int32_t *root_pos, *nbr_pos, *eid, *cnt;
    const double *root_ts, *nts;
    const float *P;
    int ldP;
    const float *efeat;
    const double *omega, *beta;
    const f4 *kv_b;
    int KFC, KVNB;
    const float *pbias;   // c_q | b_k | b_v: the rows of P carry it already
    const f4 *v_b, *uk_a;     // folded attention: V weights, W_k^t fragments
    int VNB, DC;              // 16-col blocks of M, 16-wide chunks of M
    const f4 *out_b;
    int OC, ONB;
    const float *b_o;
    const float *mem_new;
    float *h;
};

// Attention embedding of RT roots per workgroup (their RT*nb slots fill RBa
// 16-row MFMA blocks):
//  1. metadata of the slots and roots, and the time-encoding constants, to LDS
//     (one round of loads);
//  2. each slot's [efeat[eid] || phi(t_root - t_slot)] row, the roots' query
//     and s'_v rows to LDS (one round of loads, all in flight together);
//  3. one MFMA GEMM gives the per-slot part of K and V for all heads; its
//     accumulators start from the neighbour's node projection plus the bias,
//     and the (row block, column block) tiles are dealt out evenly over the
//     waves; K and V go back to LDS;
//  4. scores, softmax and the weighted sum of V: for nb <= 16 two 16-lane rows
//     per (root, head) with row-local DPP reductions; otherwise one thread per
//     score, one wave per softmax and one thread per output;
//  5. the output projection ReLU(W_o [a || s'_v] + b_o) as a second MFMA GEMM
//     whose weights were fetched before step 4.
constexpr int kAttMaxSlots = kAttMaxRB * 16;
constexpr int kAttMaxOC = 16;   // 16-wide k-chunks of the output projection (2M <= 256)
constexpr int kAttPre = 6;      // time-code k-chunks whose weights are preloaded

template <int RB>   // 16-row slot blocks per workgroup (3..5)
__device__ __forceinline__ void attn_block(const AttnArgs &g, float *lds, int bid)
{
    __shared__ int s_np[kAttMaxSlots];         // neighbour's node-set position, -1 if none
    __shared__ int64_t s_qoff[kAttMaxSlots], s_voff[kAttMaxSlots];
    __shared__ int s_cnt[kAttMaxSlots];
    __shared__ int64_t s_eoff[kAttMaxSlots];   // edge-feature row offset, -1 if none
    __shared__ double s_dt[kAttMaxSlots];      // t_root - t_slot
    __shared__ int s_ok[kAttMaxSlots];         // slot holds a sampled neighbour
    const int r0 = bid * g.RT;
    const int nroots = min(g.RT, g.R - r0);
    if (nroots <= 0)
        return;
    const int M = g.M, nb = g.nb, D_e = g.D_e, D_t = g.D_t, H = g.H;
    const int n = *g.n_nodes;   // positions and event ids are bounds-checked
    const int RA = RB * 16;
    const int KF = g.KFC * 16, SA = KF + 4;
    const int SKV = g.KVNB * 16 + 4;
    const int ORB = (g.RT + 15) / 16;
    const int SAO = g.OC * 16 + 4;
    float *A = lds;                                   // [RA][SA], then K|V [RA][SKV]
    float *Q = lds + RA * (SA > SKV ? SA : SKV);      // [RT][M]
    float *AO = Q + g.RT * M;                         // [ORB*16][SAO]: [a || s'_v]
    float *S = AO + ORB * 16 * SAO;   // scores, then weights: [RT*H*nb], or [RT*H][16] for nb <= 16
    // [D_t] fp64 frequencies and phases, at an 8-byte aligned float offset
    double *s_om = reinterpret_cast<double *>(
        lds + (((S - lds) + H * max(RA, g.RT * 16) + 1) & ~(int64_t)1));
    double *s_be = s_om + D_t;
    const int nw = blockDim.x >> 6;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform

    // GEMM tiles of this wave: column blocks cb0 = wave and cb1 = wave + nw
    // (cb1 = cb0 when past the last block: the copy computes and stores the same
    // values) over all RB row blocks, so each A fragment read from LDS feeds
    // both column blocks.
    const int cb0 = wave, cb1 = wave + nw < g.KVNB ? wave + nw : wave;
    const bool has_tiles = cb0 < g.KVNB;

    // A wave's loads complete in issue order, so they are issued in the order
    // they are consumed: the weights of the chunks made of time codes only
    // (they do not depend on the batch: issued first, they arrive with the
    // metadata), the metadata, the edge-feature rows (consumed after the
    // time-code chunks), then, once the GEMM runs, the query and s'_v rows and
    // the accumulator seeds (consumed at its end).
    const int P1 = min(D_t / 16, kAttPre);   // k-chunks of time codes only
    const int64_t kstep = (int64_t)g.KVNB * kWave;
    const f4 *p0 = g.kv_b + (int64_t)(has_tiles ? cb0 : 0) * kWave + lane;
    const int64_t o1 = (int64_t)(cb1 - cb0) * kWave;
    f4 bpre[kAttPre][2];
#pragma unroll
    for (int kc = 0; kc < kAttPre; ++kc) {   // chunks past P1 are loaded and unused
        bpre[kc][0] = p0[kc * kstep];
        bpre[kc][1] = p0[kc * kstep + o1];
    }
    issue_fence();

    // 1. metadata of the roots and of the slots and the time-encoding constants
    // in one round of loads (branch-free: indices clamped, results masked; the
    // launch has at least ORB * 16 and RA threads), and the zero parts of the
    // output projection's input: columns [0, M) of rows without a root, the
    // padding [2M, ..)
    {
        const int rr = min(tid, nroots - 1);
        const int sr = min(tid, RA - 1);
        const int r = sr / nb, j = sr - r * nb;
        const int rc = min(r, nroots - 1);
        const int64_t sl = (int64_t)(r0 + rc) * nb + j;
        const int dd = min(tid, max(D_t - 1, 0));
        const int pv = g.root_pos[r0 + rr];
        const int c_root = g.cnt[r0 + rr];
        const int c_slot = g.cnt[r0 + rc];
        const int64_t e = g.eid[sl];
        const int q = g.nbr_pos[sl];
        const double t_root = g.root_ts[r0 + rc];
        const double t_slot = g.nts[sl];
        const double om = g.omega[dd], be = g.beta[dd];
        if (tid < ORB * 16) {
            const bool ok = tid < nroots && pv >= 0 && pv < n;
            s_qoff[tid] = ok ? (int64_t)pv * g.ldP : -1;
            s_voff[tid] = ok ? (int64_t)pv * M : -1;
            s_cnt[tid] = tid < nroots ? c_root : 0;
        }
        if (tid < RA) {
            const bool ok = r < nroots && j < c_slot;
            s_ok[sr] = ok;
            s_dt[sr] = r < nroots ? t_root - t_slot : 0.0;
            s_eoff[sr] = (ok && D_e > 0 && e >= 0 && e < g.E) ? e * D_e : -1;
            s_np[sr] = (ok && q >= 0 && q < n) ? q : -1;
        }
        if (tid < D_t) {
            s_om[tid] = om;
            s_be[tid] = be;
        }
        for (int d = tid + blockDim.x; d < D_t; d += blockDim.x) {
            s_om[d] = g.omega[d];
            s_be[d] = g.beta[d];
        }
    }
    {
        const int w2 = g.OC * 16 - M;
        for (int idx = tid; idx < ORB * 16 * w2; idx += blockDim.x) {
            const int r = idx / w2, c = idx - r * w2;
            if (c >= M || r >= nroots)
                AO[r * SAO + (c < M ? c : M + c)] = 0.f;
        }
    }
    __syncthreads();

    // 2. the edge-feature rows of the slots (to registers; wave w stages slot
    // rows w + kMaxWaves i, the launch has kMaxWaves waves), then the time codes
    // phi(t_root - t_slot) in columns [0, D_t) while they are in flight
    constexpr int RPW = 2 * RB;   // RB * 16 / kMaxWaves
    int64_t eoff[RPW];
    int lr[RPW];
    double dts[RPW];
    bool oks[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        lr[i] = wave + kMaxWaves * i;
        eoff[i] = s_eoff[lr[i]];
        dts[i] = s_dt[lr[i]];
        oks[i] = s_ok[lr[i]] != 0;
    }
    const bool vec_e = D_e > 0 && g.E > 0 && (reinterpret_cast<uintptr_t>(g.efeat) & 15) == 0 &&
                       (D_e & 3) == 0 && (D_t & 3) == 0;
    // issued on every path (the other paths read P[0] and drop it), so the
    // waits below count the same loads on every path
    int64_t eoffv[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i)
        eoffv[i] = vec_e ? eoff[i] : -1;
    WaveRows<4, RPW, 1> xf;
    xf.load(vec_e ? g.efeat : g.P, eoffv, D_e, lane);
    issue_fence();
    // (the RPW rows of a column are independent chains) and the zero padding
    // past D_t + D_e
    for (int d = lane; d < D_t; d += kWave) {
        const double om = s_om[d], be = s_be[d];
#pragma unroll
        for (int i = 0; i < RPW; ++i)
            A[lr[i] * SA + d] = oks[i] ? time_enc(om, be, dts[i]) : 0.f;
    }
    for (int k = D_t + D_e + lane; k < KF; k += kWave)
#pragma unroll
        for (int i = 0; i < RPW; ++i)
            A[lr[i] * SA + k] = 0.f;
    __syncthreads();

    // 3. per-slot K|V GEMM over [phi || efeat]: first the time-code chunks
    // (weights in registers, so no wait on the loads still in flight), then the
    // edge-feature rows go to LDS and the remaining chunks stream their weights
    f4 acc[2][RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        acc[0][rb] = f4{0, 0, 0, 0};
        acc[1][rb] = f4{0, 0, 0, 0};
    }
    const float *arow = A + (lane & 15) * SA + 4 * (lane >> 4);
// one k-chunk: the RB A fragments, then the MFMAs k-slice-major over the
// 2 x RB independent accumulators
#define TGM_ATT_MMA(KC, B0, B1)                                                              \
    {                                                                                       \
        f4 a_[RB];                                                                          \
        _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                                   \
            a_[rb] = *reinterpret_cast<const f4 *>(arow + rb * 16 * SA + (KC) * 16);        \
        _Pragma("unroll") for (int j = 0; j < 4; ++j)                                       \
        {                                                                                   \
            _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                               \
            {                                                                               \
                acc[0][rb] = mfma_16x16x4(a_[rb][j], (B0)[j], acc[0][rb]);                  \
                acc[1][rb] = mfma_16x16x4(a_[rb][j], (B1)[j], acc[1][rb]);                  \
            }                                                                               \
        }                                                                                   \
    }
    if (has_tiles && P1 > 0)
        TGM_ATT_MMA(0, bpre[0][0], bpre[0][1])
    issue_fence();
    // query rows (the node projection carries the folded bias c_q; a root
    // without a position gets c_q alone) and s'_v rows: two vectors per thread
    // (branch-free), stored before the second part of the GEMM; the rest after
    // the GEMM
    const bool qv4 = (M & 3) == 0 && (reinterpret_cast<uintptr_t>(g.mem_new) & 15) == 0;
    const int M4 = qv4 ? M >> 2 : 0, M4c = qv4 ? M >> 2 : 1;
    const int nq4 = nroots * M4, nv4 = ORB * 16 * M4;
    f4 qreg[2], vreg[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = tid + u * blockDim.x;
        const int rq = i < nq4 ? i / M4c : 0, cq = i < nq4 ? i - rq * M4c : 0;
        const int rv = i < nv4 ? i / M4c : 0, cv = i < nv4 ? i - rv * M4c : 0;
        const int64_t oq = s_qoff[rq], ov = s_voff[rv];
        qreg[u] = *reinterpret_cast<const f4 *>(oq >= 0 && qv4 ? g.P + oq + 4 * cq
                                                               : g.pbias + 4 * cq);
        vreg[u] = *reinterpret_cast<const f4 *>(ov >= 0 && qv4 ? g.mem_new + ov + 4 * cv
                                                               : g.mem_new);
    }
    // seeds: the neighbour's row of P (node projection plus bias), or the bias
    // alone for a slot without a neighbour; columns past 2M read column 0
    f4 seed[2][RB];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int c = (i ? cb1 : cb0) * 16 + (lane & 15);
        const int col = M + (c < 2 * M ? c : 0);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int np = s_np[rb * 16 + 4 * (lane >> 4) + v];
                seed[i][rb][v] = *(np >= 0 ? g.P + (int64_t)np * g.ldP + col : g.pbias + col);
            }
    }
    issue_fence();
    if (has_tiles) {
#pragma unroll
        for (int kc = 1; kc < kAttPre; ++kc)
            if (kc < P1)
                TGM_ATT_MMA(kc, bpre[kc][0], bpre[kc][1])
    }
    // the weights of chunks P1 and P1 + 1 (the packed weights carry two zero
    // chunks past the end), then the edge-feature rows to columns [D_t, D_t + D_e)
    // (no chunk read so far touches them)
    const f4 *pk = p0 + P1 * kstep;
    f4 x0 = pk[0], x1 = pk[o1];
    // the output projection's weights, used in step 5 (unconditional: the
    // packed weights hold kAttMaxOC chunks, zero past OC; waves beyond ONB
    // load the last block and compute nothing)
    f4 ob[kAttMaxOC];
    const int ocb = wave;
    const float bo = g.b_o[min(ocb * 16 + (lane & 15), M - 1)];
    {
        const f4 *ob0 = g.out_b + (int64_t)min(ocb, g.ONB - 1) * kWave + lane;
#pragma unroll
        for (int kc = 0; kc < kAttMaxOC; ++kc)
            ob[kc] = ob0[(int64_t)kc * g.ONB * kWave];
    }
    issue_fence();
    // the query rows and the [. || s'_v] rows of the output projection's input
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = tid + u * blockDim.x;
        if (i < nq4) {
            const int r = i / M4c, c = i - r * M4c;
            *reinterpret_cast<f4 *>(Q + r * M + 4 * c) = qreg[u];
        }
        if (i < nv4) {
            const int r = i / M4c, c = i - r * M4c;
            *reinterpret_cast<f4 *>(AO + r * SAO + M + 4 * c) =
                s_voff[r] >= 0 ? vreg[u] : f4{0, 0, 0, 0};
        }
    }
    if (vec_e) {
        xf.store(A, SA, D_t, lr, eoffv, D_e, lane);
    } else if (D_e > 0) {   // unaligned or empty edge features: plain copies
        for (int i = 0; i < RPW; ++i)
            for (int k = lane; k < D_e; k += kWave)
                A[lr[i] * SA + D_t + k] = eoff[i] >= 0 ? g.efeat[eoff[i] + k] : 0.f;
    }
    __syncthreads();
    if (has_tiles) {
        // two register sets of weights alternate (chunk kc + 1 loads while kc
        // multiplies)
        int kc = P1;
        for (; kc + 1 < g.KFC; kc += 2) {
            const f4 *q = pk + kstep;
            const f4 y0 = q[0], y1 = q[o1];
            issue_fence();
            TGM_ATT_MMA(kc, x0, x1)
            pk += 2 * kstep;
            x0 = pk[0];
            x1 = pk[o1];
            issue_fence();
            TGM_ATT_MMA(kc + 1, y0, y1)
        }
        if (kc < g.KFC) {
            TGM_ATT_MMA(kc, x0, x1)
        }
#undef TGM_ATT_MMA
        // K|V = GEMM + seed
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
                acc[i][rb] += seed[i][rb];
    }
    // query and s'_v vectors past the first two per thread (none of this
    // touches the slot rows)
    if (qv4) {
        for (int i = tid + 2 * blockDim.x; i < max(nq4, nv4); i += blockDim.x) {
            const int r = i / M4c, c = i - r * M4c;
            if (i < nq4)
                *reinterpret_cast<f4 *>(Q + r * M + 4 * c) =
                    *reinterpret_cast<const f4 *>(s_qoff[r] >= 0 ? g.P + s_qoff[r] + 4 * c
                                                                 : g.pbias + 4 * c);
            if (i < nv4)
                *reinterpret_cast<f4 *>(AO + r * SAO + M + 4 * c) =
                    s_voff[r] >= 0 ? *reinterpret_cast<const f4 *>(g.mem_new + s_voff[r] + 4 * c)
                                   : f4{0, 0, 0, 0};
        }
    } else {     // scalar path
        for (int i = tid; i < ORB * 16 * M; i += blockDim.x) {
            const int r = i / M, k = i - r * M;
            if (r < nroots)
                Q[r * M + k] = s_qoff[r] >= 0 ? g.P[s_qoff[r] + k] : g.pbias[k];
            AO[r * SAO + M + k] = s_voff[r] >= 0 ? g.mem_new[s_voff[r] + k] : 0.f;
        }
    }
    __syncthreads();   // every read of the slot rows is done

    // K|V over the slot rows
    float *KV = A;
    if (has_tiles) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int col = (i ? cb1 : cb0) * 16 + (lane & 15);
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    KV[(rb * 16 + 4 * (lane >> 4) + v) * SKV + col] = acc[i][rb][v];
        }
    }
    __syncthreads();

    // 4. attention
    const int d_h = M / H;
    const float scale = 1.0f / sqrtf((float)d_h);
    if (nb <= 16) {
        // two 16-lane rows per (root, head), h = bit 4 of the lane: lane j of
        // both rows scores slot j over alternate pairs of the head's dimensions
        // and a swap of the rows adds the halves (in one order on both); the
        // softmax reductions stay inside the row (DPP); the row with h = 0
        // writes the 16 weights (zero past c) to S, and both rows read them
        // back (same wave: LDS is in order) for the weighted sum of V, whose
        // d_h outputs they share
        const int j = lane & 15, h = (lane >> 4) & 1;
        const int npair = nroots * H;
        const bool pairs = (d_h & 1) == 0;   // 8-byte aligned dimension pairs
        for (int pr = wave * 2 + (lane >> 5); pr < npair; pr += nw * 2) {
            const int r = pr / H, eta = pr - r * H;
            const int c = s_cnt[r];
            const float *qr = Q + r * M + eta * d_h;
            const float *kr = KV + (r * nb + min(j, nb - 1)) * SKV + eta * d_h;
            float d0 = 0.f, d1 = 0.f;
            if (pairs) {
                int d = 2 * h;
                for (; d + 13 < d_h; d += 16) {   // four pairs, loads issued together
                    float2 q2[4], k2[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        q2[t] = *reinterpret_cast<const float2 *>(qr + d + 4 * t);
                        k2[t] = *reinterpret_cast<const float2 *>(kr + d + 4 * t);
                    }
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        d0 += q2[t].x * k2[t].x;
                        d1 += q2[t].y * k2[t].y;
                    }
                }
                for (; d < d_h; d += 4) {
                    const float2 q2 = *reinterpret_cast<const float2 *>(qr + d);
                    const float2 k2 = *reinterpret_cast<const float2 *>(kr + d);
                    d0 += q2.x * k2.x;
                    d1 += q2.y * k2.y;
                }
            } else {
                for (int d = h; d < d_h; d += 2)
                    d0 += qr[d] * kr[d];
            }
            const float part = d0 + d1;
            const float other = __shfl_xor(part, 16, kWave);
            const float dot = h ? other + part : part + other;
            const float sc = j < c ? dot * scale : -INFINITY;
            const float mx = row16_max(sc);
            const float e = j < c ? expf(sc - mx) : 0.f;
            const float den = row16_sum(e);
            float *al = S + pr * 16;
            if (h == 0)
                al[j] = j < c ? e / den : 0.f;
            float alv[16];
#pragma unroll
            for (int jj = 0; jj < 16; ++jj)
                alv[jj] = al[jj];
            const float *vr = KV + r * nb * SKV + M + eta * d_h;
            float *ar = AO + r * SAO + eta * d_h;
            for (int k = j + 16 * h; k < d_h; k += 32) {
                float a0 = 0.f, a1 = 0.f;
#pragma unroll
                for (int jj = 0; jj < 16; jj += 2) {
                    a0 += alv[jj] * vr[min(jj, nb - 1) * SKV + k];
                    a1 += alv[jj + 1] * vr[min(jj + 1, nb - 1) * SKV + k];
                }
                ar[k] = a0 + a1;   // 0 when the root has no neighbours
            }
        }
    } else {
        // scores (one thread per (root, head, slot)), softmax (one wave per
        // (root, head): lane j holds slot j, reductions over lanes) and the
        // weighted sum of V (one thread per output)
        const int nsc = nroots * H * nb;
        for (int idx = tid; idx < nsc; idx += blockDim.x) {
            const int r = idx / (H * nb), rem = idx - r * (H * nb);
            const int eta = rem / nb, j = rem - eta * nb;
            float sc = -INFINITY;
            if (j < s_cnt[r]) {
                const float *qr = Q + r * M + eta * d_h;
                const float *kr = KV + (r * nb + j) * SKV + eta * d_h;
                float dot = 0.f;
                for (int d = 0; d < d_h; ++d)
                    dot += qr[d] * kr[d];
                sc = dot * scale;
            }
            S[idx] = sc;
        }
        __syncthreads();
        for (int pr = wave; pr < nroots * H; pr += nw) {
            const int c = s_cnt[pr / H];
            float *sr = S + pr * nb;
            const float sc = lane < c ? sr[lane] : -INFINITY;
            float mx = sc;
#pragma unroll
            for (int o = kWave / 2; o >= 1; o >>= 1)
                mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
            const float e = lane < c ? expf(sc - mx) : 0.f;
            float den = e;
#pragma unroll
            for (int o = kWave / 2; o >= 1; o >>= 1)
                den += __shfl_xor(den, o, kWave);
            if (lane < c)
                sr[lane] = e / den;
        }
        __syncthreads();
        for (int idx = tid; idx < nroots * M; idx += blockDim.x) {
            const int r = idx / M, k = idx - r * M;
            const int eta = k / d_h;
            const float *al = S + (r * H + eta) * nb;
            const int c = s_cnt[r];
            float a = 0.f;
            for (int j = 0; j < c; ++j)
                a += al[j] * KV[(r * nb + j) * SKV + M + k];
            AO[r * SAO + k] = a;   // 0 when the root has no neighbours
        }
    }
    __syncthreads();

    // 5. h = ReLU(W_o [a || s'_v] + b_o): the row block's fragments first (chunks
    // past OC re-read the last one against zero weights), then four accumulators
    // over the chunks
    if (ocb < g.ONB) {
        const float *orow = AO + (lane & 15) * SAO + 4 * (lane >> 4);
        const int col = ocb * 16 + (lane & 15);
        const int OC = g.OC;
        for (int orb = 0; orb < ORB; ++orb) {
            f4 af[kAttMaxOC];
#pragma unroll
            for (int kc = 0; kc < kAttMaxOC; ++kc)
                af[kc] = *reinterpret_cast<const f4 *>(orow + orb * 16 * SAO + min(kc, OC - 1) * 16);
            f4 ac[4] = {{0, 0, 0, 0}, {0, 0, 0, 0}, {0, 0, 0, 0}, {0, 0, 0, 0}};
#pragma unroll
            for (int kc = 0; kc < kAttMaxOC; ++kc)
                if (kc < OC)
                    ac[kc & 3] = mfma_k16(af[kc], ob[kc], ac[kc & 3]);
            if (col < M) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int r = orb * 16 + 4 * (lane >> 4) + v;
                    if (r < nroots)
                        g.h[(int64_t)(r0 + r) * M + col] =
                            fmaxf((ac[0][v] + ac[1][v]) + (ac[2][v] + ac[3][v]) + bo, 0.f);
                }
            }
        }
    }
}

template <int RB>
__global__ __launch_bounds__(512) void k_attn(AttnArgs g)
{
    extern __shared__ float lds[];
    attn_block<RB>(g, lds, blockIdx.x);
}

// The attention and the gather of the next iteration's fetch in one launch:
// blocks [0, n_attn) embed; the rest (dispatched after them, on the CUs the
// attention leaves free) gather one node row per wavefront.
template <int RB>
__global__ __launch_bounds__(512) void k_attn_gather(AttnArgs g, int n_attn, GatherPlan gp)
{
    extern __shared__ float lds[];
    if ((int)blockIdx.x < n_attn) {
        attn_block<RB>(g, lds, blockIdx.x);
        return;
    }
    gather_blocks(gp, (int)blockIdx.x - n_attn, (int)gridDim.x - n_attn, blockDim.x >> 6,
                  threadIdx.x >> 6, threadIdx.x & 63);
}

// ---------------------------------------------------------------------------
// Attention with the query folded into the key weights.  Each score is
//   q_r,eta . K_s,eta = sum_k a_s[k] U[k][(r, eta)] + seedK_s,eta . q_r,eta
// with a_s = [phi || efeat] the slot row, seedK_s the neighbour's key part of
// P (node projection plus b_k) and U[k][(r, eta)] = sum_{d in head eta}
// W_k[d][k] q_r[d] (Eq. 1's emb() restated by associativity).  K itself
// is never formed: the per-slot GEMM produces V (VNB column blocks) and one
// block of 16 score columns (n = r * H + eta, RT * H <= 16) instead of the
// 2M columns of K | V.  Roles of the kMaxWaves wavefronts:
//   * wave w < VNB: V column block w over all RB row blocks;
//   * wave VNB (the score wave): the score block, first the seedK . q part
//     (K = M, operands straight from P), then [phi || efeat] x U;
//   * waves on SIMDs (wave % 4) other than the score wave's: the U GEMM
//     (KFC row blocks of 16 k, K = M, weights W_k^t preloaded).
// A wave's loads complete in issue order, so each issues what it consumes
// first before the edge-feature rows (the slow, HBM-bound loads).
constexpr int kAttUT = 3;   // U tiles per wavefront
constexpr int kAttDC = 7;   // 16-wide chunks of M (M <= 112)
constexpr int kAttFoldOC = 2 * kAttDC;   // 16-wide chunks of [a || s'_v]

template <int RB>   // 16-row slot blocks per workgroup (3..5)
__device__ __forceinline__ void attn_fold_block(const AttnArgs &g, float *lds, int bid)
{
    __shared__ int s_np[kAttMaxSlots];         // neighbour's node-set position, -1 if none
    __shared__ int64_t s_qoff[kAttMaxSlots], s_voff[kAttMaxSlots];
    __shared__ int s_cnt[kAttMaxSlots];
    __shared__ int64_t s_eoff[kAttMaxSlots];   // edge-feature row offset, -1 if none
    __shared__ double s_dt[kAttMaxSlots];      // t_root - t_slot
    __shared__ int s_ok[kAttMaxSlots];         // slot holds a sampled neighbour
    const int r0 = bid * g.RT;
    const int nroots = min(g.RT, g.R - r0);
    if (nroots <= 0)
        return;
    const int M = g.M, nb = g.nb, D_e = g.D_e, D_t = g.D_t, H = g.H;
    const int n = *g.n_nodes;   // positions and event ids are bounds-checked
    const int KFC = g.KFC, VNB = g.VNB, DC = g.DC;
    const int RA = RB * 16;
    const int KF = KFC * 16, SA = KF + 4, SV = VNB * 16 + 4;
    const int ORB = (g.RT + 15) / 16;
    const int SAO = g.OC * 16 + 4;
    const int d_h = M / H;
    float *A = lds;                                             // [RA][SA], then V [RA][SV]
    f4 *U = reinterpret_cast<f4 *>(A + RA * SA);                // [KFC][64] B fragments
    float *AO = reinterpret_cast<float *>(U + KFC * kWave);     // [ORB*16][SAO]: [a || s'_v]
    float *S = AO + ORB * 16 * SAO;                             // [RA][H] scores
    float *Wt = S + RA * H;                                     // [RT*H][16] weights
    double *s_om = reinterpret_cast<double *>(
        lds + (((Wt - lds) + g.RT * H * 16 + 1) & ~(int64_t)1));
    double *s_be = s_om + D_t;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
    const bool is_v = wave < VNB, is_s = wave == VNB;
    int ui = -1, NU = 0;   // this wave's index among the U waves, their number
    for (int w = 0; w < kMaxWaves; ++w)
        if ((w & 3) != (VNB & 3)) {
            if (w == wave)
                ui = NU;
            ++NU;
        }

    // 0. the W_k^t fragments of this wave's U tiles (they do not depend on the
    // batch; indices clamped).  Loads issued inside a role's branch are only
    // waited for inside it, before any later load is: the wait counts stay
    // exact on every path.
    f4 ua[kAttUT][kAttDC];
    if (ui >= 0) {
#pragma unroll
        for (int t = 0; t < kAttUT; ++t) {
            const int kb = min(ui + NU * t, KFC - 1);
#pragma unroll
            for (int dc = 0; dc < kAttDC; ++dc)
                ua[t][dc] = g.uk_a[((int64_t)min(dc, DC - 1) * KFC + kb) * kWave + lane];
        }
    }
    issue_fence();

    // 1. metadata of the roots and of the slots and the time-encoding constants
    // in one round of loads, by the two waves on the score wave's SIMD (the U
    // waves' weight loads stay in flight meanwhile; branch-free: indices
    // clamped, results masked; RA and ORB * 16 are at most 128), and the zero
    // parts of the output projection's input: columns [0, M) of rows without a
    // root, the padding [2M, ..)
    if (ui < 0) {
        const int mt = (wave > 3 ? 64 : 0) + lane;   // 0 .. 127
        const int rr = min(mt, nroots - 1);
        const int sr = min(mt, RA - 1);
        const int r = sr / nb, j = sr - r * nb;
        const int rc = min(r, nroots - 1);
        const int64_t sl = (int64_t)(r0 + rc) * nb + j;
        const int dd = min(mt, max(D_t - 1, 0));
        const int pv_ = g.root_pos[r0 + rr];
        const int c_root = g.cnt[r0 + rr];
        const int c_slot = g.cnt[r0 + rc];
        const int64_t e = g.eid[sl];
        const int q = g.nbr_pos[sl];
        const double t_root = g.root_ts[r0 + rc];
        const double t_slot = g.nts[sl];
        const double om = g.omega[dd], be = g.beta[dd];
        if (mt < ORB * 16) {
            const bool ok = mt < nroots && pv_ >= 0 && pv_ < n;
            s_qoff[mt] = ok ? (int64_t)pv_ * g.ldP : -1;
            s_voff[mt] = ok ? (int64_t)pv_ * M : -1;
            s_cnt[mt] = mt < nroots ? c_root : 0;
        }
        if (mt < RA) {
            const bool ok = r < nroots && j < c_slot;
            s_ok[sr] = ok;
            s_dt[sr] = r < nroots ? t_root - t_slot : 0.0;
            s_eoff[sr] = (ok && D_e > 0 && e >= 0 && e < g.E) ? e * D_e : -1;
            s_np[sr] = (ok && q >= 0 && q < n) ? q : -1;
        }
        if (mt < D_t) {
            s_om[mt] = om;
            s_be[mt] = be;
        }
        for (int d = mt + 128; d < D_t; d += 128) {
            s_om[d] = g.omega[d];
            s_be[d] = g.beta[d];
        }
    }
    {
        const int w2 = g.OC * 16 - M;
        for (int idx = tid; idx < ORB * 16 * w2; idx += blockDim.x) {
            const int rw = idx / w2, c = idx - rw * w2;
            if (c >= M || rw >= nroots)
                AO[rw * SAO + (c < M ? c : M + c)] = 0.f;
        }
    }
    __syncthreads();

    // 2. query fragments (every wave: the B operand of the U GEMM and of the
    // score wave's seed part): lane l holds q_r[d] of column n = l % 16
    // (r = n / H, eta = n % H) for d = 16 dc + 4 (l / 16) + j, zero outside
    // head eta, past M and for a column without a root; a root without a
    // position has the folded bias c_q as its query
    const int cn = lane & 15, cr = cn / H, ceta = cn - cr * H;
    f4 bq[kAttDC];
    {
        const int64_t qo = cr < nroots ? s_qoff[cr] : -1;
        const float *qrow = qo >= 0 ? g.P + qo : g.pbias;
#pragma unroll
        for (int dc = 0; dc < kAttDC; ++dc)
            bq[dc] = *reinterpret_cast<const f4 *>(qrow + min(16 * dc + 4 * (lane >> 4), M - 4));
    }
    issue_fence();
    // the score wave's seed part: K = M over the neighbours' key rows of P (or
    // b_k for a slot without one)
    f4 acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
        acc[rb] = f4{0, 0, 0, 0};
    // (masked where first used, after the loads that must not wait for it)
    auto mask_q = [&]() {
        const int lo = ceta * d_h, hi = cr < nroots ? lo + d_h : lo;
#pragma unroll
        for (int dc = 0; dc < kAttDC; ++dc)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d = 16 * dc + 4 * (lane >> 4) + j;
                if (!(d >= lo && d < hi))
                    bq[dc][j] = 0.f;
            }
    };
    constexpr int RPW = 2 * RB;   // slot rows staged per wave (RB * 16 / kMaxWaves)
    int64_t eoff[RPW];
    int lr[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        lr[i] = wave + kMaxWaves * i;
        eoff[i] = s_eoff[lr[i]];
    }
    const bool vec_e = D_e > 0 && g.E > 0 && (reinterpret_cast<uintptr_t>(g.efeat) & 15) == 0 &&
                       (D_e & 3) == 0 && (D_t & 3) == 0;
    int64_t eoffv[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i)
        eoffv[i] = vec_e ? eoff[i] : -1;
    WaveRows<4, RPW, 1> xf;
    const int P1 = min(D_t / 16, kAttPre);   // k-chunks of time codes only
    const int64_t vstep = (int64_t)VNB * kWave;
    const f4 *pv = g.v_b + (int64_t)(is_v ? wave : 0) * kWave + lane;
    f4 bpre[kAttPre];
    // the time codes phi(t_root - t_slot) in columns [0, D_t), computed while
    // the P rows are in flight (the RPW rows of a column are independent
    // chains), and the zero padding past D_t + D_e; inlined into each role's
    // branch below, so that role-specific registers never share live ranges
    auto time_codes = [&]() {
        double dts[RPW];
        bool oks[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            dts[i] = s_dt[lr[i]];
            oks[i] = s_ok[lr[i]] != 0;
        }
        for (int d = lane; d < D_t; d += kWave) {
            const double om = s_om[d], be = s_be[d];
#pragma unroll
            for (int i = 0; i < RPW; ++i)
                A[lr[i] * SA + d] = oks[i] ? time_enc(om, be, dts[i]) : 0.f;
        }
        for (int k = D_t + D_e + lane; k < KF; k += kWave)
#pragma unroll
            for (int i = 0; i < RPW; ++i)
                A[lr[i] * SA + k] = 0.f;
    };
    if (is_s) {
        // the neighbours' key rows: every row's loads in flight together
        f4 sa[RB][kAttDC];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const int np = s_np[rb * 16 + (lane & 15)];
            const float *row = (np >= 0 ? g.P + (int64_t)np * g.ldP : g.pbias) + M;
#pragma unroll
            for (int dc = 0; dc < kAttDC; ++dc)
                sa[rb][dc] =
                    *reinterpret_cast<const f4 *>(row + min(16 * dc + 4 * (lane >> 4), M - 4));
        }
        issue_fence();
        time_codes();
        mask_q();
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int dc = 0; dc < kAttDC; ++dc)   // bq is zero past M
                acc[rb] = mfma_k16(sa[rb][dc], bq[dc], acc[rb]);
    } else if (ui >= 0) {
        time_codes();
        mask_q();
        // U tiles kb = ui + NU t: U[16 kb .. +16][n] -> LDS
        f4 au[kAttUT];
#pragma unroll
        for (int t = 0; t < kAttUT; ++t)
            au[t] = f4{0, 0, 0, 0};
#pragma unroll
        for (int dc = 0; dc < kAttDC; ++dc)   // bq is zero past M
#pragma unroll
            for (int t = 0; t < kAttUT; ++t)
                au[t] = mfma_k16(ua[t][dc], bq[dc], au[t]);
#pragma unroll
        for (int t = 0; t < kAttUT; ++t) {
            const int kb = ui + NU * t;
            if (kb < KFC)
                U[kb * kWave + lane] = au[t];
        }
    } else {
        time_codes();
    }
    // then the loads consumed in step 3 (after the fragments above, whose waits
    // they would otherwise join): the V weights of the chunks made of time
    // codes only, and the edge-feature rows
    if (is_v) {
#pragma unroll
        for (int kc = 0; kc < kAttPre; ++kc)   // chunks past P1 are loaded and unused
            bpre[kc] = pv[kc * vstep];
    }
    xf.load(vec_e ? g.efeat : g.P, eoffv, D_e, lane);
    issue_fence();
    __syncthreads();

    // 3. the per-slot GEMM over [phi || efeat]: the time-code chunks first (V
    // weights in registers, U in LDS: no wait on the rows in flight), then the
    // edge-feature rows go to LDS and the remaining chunks follow
    const float *arow = A + (lane & 15) * SA + 4 * (lane >> 4);
// one k-chunk against the B fragment b: the RB A fragments, then the MFMAs
#define TGM_FOLD_MMA(KC, B)                                                                 \
    {                                                                                       \
        f4 a_[RB];                                                                          \
        _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                                   \
            a_[rb] = *reinterpret_cast<const f4 *>(arow + rb * 16 * SA + (KC) * 16);        \
        _Pragma("unroll") for (int j = 0; j < 4; ++j)                                       \
        {                                                                                   \
            _Pragma("unroll") for (int rb = 0; rb < RB; ++rb)                               \
                acc[rb] = mfma_16x16x4(a_[rb][j], (B)[j], acc[rb]);                          \
        }                                                                                   \
    }
    if (is_v && P1 > 0) {
        TGM_FOLD_MMA(0, bpre[0])
    } else if (is_s && P1 > 0) {
        const f4 ub = U[lane];
        TGM_FOLD_MMA(0, ub)
    }
    issue_fence();
    // s'_v rows of the output projection's input (two vectors per thread,
    // branch-free; the rest after the GEMM) and the V seeds: the neighbour's
    // value row of P, or b_v alone for a slot without a neighbour
    const bool v4 = (M & 3) == 0 && (reinterpret_cast<uintptr_t>(g.mem_new) & 15) == 0;
    const int M4 = v4 ? M >> 2 : 0, M4c = v4 ? M >> 2 : 1;
    const int nv4 = ORB * 16 * M4;
    f4 vreg[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = tid + u * blockDim.x;
        const int rv = i < nv4 ? i / M4c : 0, cv = i < nv4 ? i - rv * M4c : 0;
        const int64_t ov = s_voff[rv];
        vreg[u] = *reinterpret_cast<const f4 *>(ov >= 0 && v4 ? g.mem_new + ov + 4 * cv
                                                              : g.mem_new);
    }
    f4 seed[RB];
    {
        const int c = (is_v ? wave : 0) * 16 + (lane & 15);
        const int col = 2 * M + (c < M ? c : 0);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int np = s_np[rb * 16 + 4 * (lane >> 4) + v];
                seed[rb][v] = *(np >= 0 ? g.P + (int64_t)np * g.ldP + col : g.pbias + col);
            }
    }
    issue_fence();
    if (is_v) {
#pragma unroll
        for (int kc = 1; kc < kAttPre; ++kc)
            if (kc < P1)
                TGM_FOLD_MMA(kc, bpre[kc])
    } else if (is_s) {
        for (int kc = 1; kc < P1; ++kc) {
            const f4 ub = U[kc * kWave + lane];
            TGM_FOLD_MMA(kc, ub)
        }
    }
    // the V weights of chunk P1 (the packed weights carry two zero chunks past
    // the end), the edge-feature rows to columns [D_t, D_t + D_e) and the s'_v
    // rows, then the output projection's weights (unconditional: the packed
    // weights hold kAttMaxOC >= kAttFoldOC chunks, zero past OC; waves beyond
    // ONB load the last block and compute nothing)
    const f4 *pk = pv + P1 * vstep;
    f4 x = pk[0];
    if (vec_e) {
        xf.store(A, SA, D_t, lr, eoffv, D_e, lane);
    } else if (D_e > 0) {   // unaligned edge features: plain copies
        for (int i = 0; i < RPW; ++i)
            for (int k = lane; k < D_e; k += kWave)
                A[lr[i] * SA + D_t + k] = eoff[i] >= 0 ? g.efeat[eoff[i] + k] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int i = tid + u * blockDim.x;
        if (i < nv4) {
            const int r = i / M4c, c = i - r * M4c;
            *reinterpret_cast<f4 *>(AO + r * SAO + M + 4 * c) =
                s_voff[r] >= 0 ? vreg[u] : f4{0, 0, 0, 0};
        }
    }
    f4 ob[kAttFoldOC];
    const int ocb = wave;
    const float bo = g.b_o[min(ocb * 16 + (lane & 15), M - 1)];
    {
        const f4 *ob0 = g.out_b + (int64_t)min(ocb, g.ONB - 1) * kWave + lane;
#pragma unroll
        for (int kc = 0; kc < kAttFoldOC; ++kc)
            ob[kc] = ob0[(int64_t)kc * g.ONB * kWave];
    }
    issue_fence();
    __syncthreads();
    if (is_v) {
        // two register sets of weights alternate (chunk kc + 1 loads while kc
        // multiplies)
        int kc = P1;
        for (; kc + 1 < KFC; kc += 2) {
            const f4 y = pk[vstep];
            issue_fence();
            TGM_FOLD_MMA(kc, x)
            pk += 2 * vstep;
            x = pk[0];
            issue_fence();
            TGM_FOLD_MMA(kc + 1, y)
        }
        if (kc < KFC)
            TGM_FOLD_MMA(kc, x)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
            acc[rb] += seed[rb];
    } else if (is_s) {
#pragma unroll 2
        for (int kc = P1; kc < KFC; ++kc) {
            const f4 ub = U[kc * kWave + lane];
            TGM_FOLD_MMA(kc, ub)
        }
    }
#undef TGM_FOLD_MMA
    // s'_v vectors past the first two per thread (none of this touches the
    // slot rows)
    if (v4) {
        for (int i = tid + 2 * blockDim.x; i < nv4; i += blockDim.x) {
            const int r = i / M4c, c = i - r * M4c;
            *reinterpret_cast<f4 *>(AO + r * SAO + M + 4 * c) =
                s_voff[r] >= 0 ? *reinterpret_cast<const f4 *>(g.mem_new + s_voff[r] + 4 * c)
                               : f4{0, 0, 0, 0};
        }
    } else {
        for (int i = tid; i < ORB * 16 * M; i += blockDim.x) {
            const int r = i / M, k = i - r * M;
            AO[r * SAO + M + k] = s_voff[r] >= 0 ? g.mem_new[s_voff[r] + k] : 0.f;
        }
    }
    __syncthreads();   // every read of the slot rows is done

    // V over the slot rows; the score wave keeps score (s, eta) of slot s's own
    // root r(s) = s / nb, held by the lane of column n = r(s) * H + eta
    float *Vs = A;
    const float scale = 1.0f / sqrtf((float)d_h);
    if (is_v) {
        const int col = wave * 16 + (lane & 15);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                Vs[(rb * 16 + 4 * (lane >> 4) + v) * SV + col] = acc[rb][v];
    } else if (is_s) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int s = rb * 16 + 4 * (lane >> 4) + v;
                if (s / nb == cr && cr < nroots)
                    S[s * H + ceta] = acc[rb][v] * scale;
            }
    }
    __syncthreads();

    // 4. softmax and the weighted sum of V: two 16-lane rows per (root, head),
    // h = bit 4 of the lane; lane j holds slot j's score, the reductions stay
    // inside the row (DPP); the row with h = 0 writes the 16 weights (zero past
    // c) and both rows read them back (same wave: LDS is in order) and share
    // the head's d_h outputs
    {
        const int nw = blockDim.x >> 6;
        const int j = lane & 15, h = (lane >> 4) & 1;
        const int npair = nroots * H;
        for (int pr = wave * 2 + (lane >> 5); pr < npair; pr += nw * 2) {
            const int r = pr / H, eta = pr - r * H;
            const int c = s_cnt[r];
            const float sc = j < c ? S[(r * nb + min(j, nb - 1)) * H + eta] : -INFINITY;
            const float mx = row16_max(sc);
            const float e = j < c ? expf(sc - mx) : 0.f;
            const float den = row16_sum(e);
            float *al = Wt + pr * 16;
            if (h == 0)
                al[j] = j < c ? e / den : 0.f;
            float alv[16];
#pragma unroll
            for (int jj = 0; jj < 16; ++jj)
                alv[jj] = al[jj];
            const float *vr = Vs + r * nb * SV + eta * d_h;
            float *ar = AO + r * SAO + eta * d_h;
            for (int k = j + 16 * h; k < d_h; k += 32) {
                float a0 = 0.f, a1 = 0.f;
#pragma unroll
                for (int jj = 0; jj < 16; jj += 2) {
                    a0 += alv[jj] * vr[min(jj, nb - 1) * SV + k];
                    a1 += alv[jj + 1] * vr[min(jj + 1, nb - 1) * SV + k];
                }
                ar[k] = a0 + a1;   // 0 when the root has no neighbours
            }
        }
    }
    __syncthreads();

    // 5. h = ReLU(W_o [a || s'_v] + b_o): the row block's fragments first (chunks
    // past OC re-read the last one against zero weights), then four accumulators
    if (ocb < g.ONB) {
        const float *orow = AO + (lane & 15) * SAO + 4 * (lane >> 4);
        const int col = ocb * 16 + (lane & 15);
        const int OC = g.OC;
        for (int orb = 0; orb < ORB; ++orb) {
            f4 af[kAttFoldOC];
#pragma unroll
            for (int kc = 0; kc < kAttFoldOC; ++kc)
                af[kc] = *reinterpret_cast<const f4 *>(orow + orb * 16 * SAO + min(kc, OC - 1) * 16);
            f4 ac[4] = {{0, 0, 0, 0}, {0, 0, 0, 0}, {0, 0, 0, 0}, {0, 0, 0, 0}};
#pragma unroll
            for (int kc = 0; kc < kAttFoldOC; ++kc)
                if (kc < OC)
                    ac[kc & 3] = mfma_k16(af[kc], ob[kc], ac[kc & 3]);
            if (col < M) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int r = orb * 16 + 4 * (lane >> 4) + v;
                    if (r < nroots)
                        g.h[(int64_t)(r0 + r) * M + col] =
                            fmaxf((ac[0][v] + ac[1][v]) + (ac[2][v] + ac[3][v]) + bo, 0.f);
                }
            }
        }
    }
}

template <int RB>
__global__ __launch_bounds__(512) void k_attn_fold(AttnArgs g)
{
    extern __shared__ float lds[];
    attn_fold_block<RB>(g, lds, blockIdx.x);
}

template <int RB>
__global__ __launch_bounds__(512) void k_attn_fold_gather(AttnArgs g, int n_attn, GatherPlan gp)
{
    extern __shared__ float lds[];
    if ((int)blockIdx.x < n_attn) {
        attn_fold_block<RB>(g, lds, blockIdx.x);
        return;
    }
    gather_blocks(gp, (int)blockIdx.x - n_attn, (int)gridDim.x - n_attn, blockDim.x >> 6,
                  threadIdx.x >> 6, threadIdx.x & 63);
}

// ---------------------------------------------------------------------------
// Attention by aggregation.  The value projection is linear, so for root r
// and head eta, with weights alpha_s over the root's slots s,
//   o_r,eta = sum_s alpha_s (W_v,a a_s + seedV_s)_eta
//           = (W_v,a abar_r,eta)_eta + (sum_s alpha_s seedV_s)_eta,
//   abar_r,eta = sum_s alpha_s a_s,
// and each score is (a_s . U_r,eta + seedK_s . q_r,eta) / sqrt(d_h) with
// U_r,eta = W_k,a^t q_r,eta (Eq. 1's emb() restated by linearity; a_s =
// [phi || efeat] the slot row, seedK_s / seedV_s the neighbour's key / value
// part of P, the node projection plus the bias).  The per-slot work is one dot
// product and one axpy of a_s per head, on the VALU; the GEMMs run once per
// (root, head) row: U, the value projection of the aggregates and the output
// projection, each a single 16-row MFMA block per workgroup (RT roots, RT H
// <= 16 rows, row n = root * H + head).
// Wavefront w owns root r0 + w; phases, separated by barriers:
//   1. every wave: the query fragments of all RT roots, then its U tiles (16
//      columns of k each) -> LDS Us, and its 16-slot block of the seed part
//      seedK_s . q (K = M, the neighbours' key rows of P) -> LDS Sk; its own
//      root's slot metadata and slot rows a_s, in registers (lane l holds
//      columns l + 64 i);
//   2. scores (wave reductions), softmax, abar -> LDS As; the aggregate of the
//      value seeds and s'_r -> LDS AO;
//   3. value GEMM, wave cb taking column block cb; a column is kept for the
//      row of its own head and added into AO;
//   4. output GEMM h = ReLU(W_o [o || s'_r] + b_o).
// LDS: 2 x 16 rows of the slot-row width and 16 rows of [o || s'_r], about
// 53 KB at the GDELT-shaped sizes, so that two workgroups share a CU.
constexpr int kAggCols = 5;     // slot-row columns per lane (KF <= 320)
constexpr int kAggTCols = 2;    // of them time codes (D_t <= 128)
constexpr int kAggDC = 7;       // 16-wide chunks of M (M <= 112)
constexpr int kAggUT = 3;       // U tiles per wave (KFC <= 24)
constexpr int kAggMaxH = 4;
constexpr int kAggMaxKC = 24;   // k-chunks of the value GEMM (KFC) and of the output one (OC)
constexpr int kAggRing = 8;     // weight chunks in flight per wave in those GEMMs

// Sum over the wavefront, the same in every lane: DPP sums inside each 16-lane
// row, then the four row sums (lanes 0, 16, 32, 48) read as scalars and added
// in that order.
__device__ __forceinline__ float wave_sum_rows(float v)
{
    v = row16_sum(v);
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

// One GEMM of a 16-row A block in LDS (k-chunks of 16 columns) against packed
// B chunks (kc * bstep apart): the first kAggRing chunks are already in `ring`
// (loaded by the caller before the barrier that publishes A); a slot is
// refilled with the chunk kAggRing further on right after its MFMAs are
// issued (indices clamped: the last rounds reload the last chunk).
__device__ __forceinline__ f4 agg_gemm(const float *arow, const f4 *pw, int64_t bstep, int KC,
                                       f4 (&ring)[kAggRing])
{
    f4 acc = f4{0, 0, 0, 0};
    int kc0 = 0;
    for (; kc0 + kAggRing <= KC; kc0 += kAggRing) {
#pragma unroll
        for (int i = 0; i < kAggRing; ++i) {
            const f4 a = *reinterpret_cast<const f4 *>(arow + 16 * (kc0 + i));
            acc = mfma_k16(a, ring[i], acc);
            ring[i] = pw[min(kc0 + kAggRing + i, KC - 1) * bstep];
        }
    }
#pragma unroll
    for (int i = 0; i < kAggRing; ++i)
        if (kc0 + i < KC) {
            const f4 a = *reinterpret_cast<const f4 *>(arow + 16 * (kc0 + i));
            acc = mfma_k16(a, ring[i], acc);
        }
    return acc;
}

__device__ __forceinline__ void agg_ring_load(const f4 *pw, int64_t bstep, int KC,
                                              f4 (&ring)[kAggRing])
{
#pragma unroll
    for (int i = 0; i < kAggRing; ++i)
        ring[i] = pw[min(i, KC - 1) * bstep];
}

template <int NBM>   // slots per root held in registers (nb <= NBM)
__device__ __forceinline__ void attn_agg_block(const AttnArgs &g, float *lds, int bid)
{
    const int RT = g.RT;
    const int r0 = bid * RT;
    const int nroots = min(RT, g.R - r0);
    if (nroots <= 0)
        return;
    const int M = g.M, nb = g.nb, D_e = g.D_e, D_t = g.D_t, H = g.H;
    const int KFC = g.KFC, DC = g.DC, VNB = g.VNB, OC = g.OC, ONB = g.ONB;
    const int KF = D_t + D_e;
    const int KFP = KFC * 16 + 4, SAO = OC * 16 + 4;
    const int d_h = M / H;
    const int n = *g.n_nodes;   // positions and event ids are bounds-checked
    float *Us = lds;              // [16][KFP]: U rows (r, eta)
    float *As = Us + 16 * KFP;    // [16][KFP]: abar rows (r, eta)
    float *AO = As + 16 * KFP;    // [16][SAO]: [o || s'_r || 0]
    float *Sk = AO + 16 * SAO;    // [RT nb][H]: seedK_s . q_r(s),eta
    const int tid = threadIdx.x, lane = tid & 63, q4 = 4 * (lane >> 4);
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int cn = lane & 15, cr = cn / H, ce = cn - cr * H;
    const bool own = wave < nroots;
    const int r = r0 + min(wave, nroots - 1);
    const bool seeds = wave * 16 < nroots * nb;   // this wave has a 16-slot seed block

    // 1a. loads that depend on nothing: the first U tile's W_k,a^t fragments,
    // then the indices: the query columns' roots, the seed block's slots, the
    // own root's slots (lane j < nb: slot j)
    f4 ua[kAggDC];
#pragma unroll
    for (int dc = 0; dc < kAggDC; ++dc)
        ua[dc] = g.uk_a[((int64_t)min(dc, DC - 1) * KFC + min(wave, KFC - 1)) * kWave + lane];
    const int qpos = g.root_pos[r0 + min(cr, nroots - 1)];
    const int sr = wave * 16 + cn;
    const int sw = min(sr / nb, nroots - 1), sj = sr - (sr / nb) * nb;
    const int spos = g.nbr_pos[(int64_t)(r0 + sw) * nb + sj];
    const int c = own ? g.cnt[r] : 0;
    const int pv = g.root_pos[r];
    const double t_root = g.root_ts[r];
    int my_e = -1, my_np = -1;
    double my_dt = 0.0;
    if (lane < nb) {
        const int64_t sl = (int64_t)r * nb + lane;
        const int64_t e = g.eid[sl];
        const int q = g.nbr_pos[sl];
        my_e = (lane < c && D_e > 0 && e >= 0 && e < g.E) ? (int)e : -1;
        my_np = (lane < c && q >= 0 && q < n) ? q : -1;
        my_dt = t_root - g.nts[sl];
    }
    const bool pv_ok = own && pv >= 0 && pv < n;
    issue_fence();

    // 1b. query fragments (B operand of the U and seed GEMMs): lane l holds q of
    // column n = l % 16 (root n / H, head n % H) for d = 16 dc + 4 (l / 16) + j,
    // zero outside the head, past M and for a column without a root
    f4 bq[kAggDC];
    {
        const bool ok = cr < nroots && qpos >= 0 && qpos < n;
        const float *qrow = ok ? g.P + (int64_t)qpos * g.ldP : g.pbias;
#pragma unroll
        for (int dc = 0; dc < kAggDC; ++dc)
            bq[dc] = *reinterpret_cast<const f4 *>(qrow + min(16 * dc + q4, M - 4));
    }
    issue_fence();
    {
        const int lo = ce * d_h, hi = cr < nroots ? lo + d_h : lo;
#pragma unroll
        for (int dc = 0; dc < kAggDC; ++dc)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int d = 16 * dc + q4 + j;
                if (!(dc < DC && d >= lo && d < hi))
                    bq[dc][j] = 0.f;
            }
    }
    // 1c. U tiles kb = wave + 8 t: U^t[16 kb .. +16][n] = W_k,a^t q_n; the next
    // tile's fragments load while this one multiplies
#pragma unroll
    for (int t = 0; t < kAggUT; ++t) {
        const int kb = wave + kMaxWaves * t;
        if (kb < KFC) {
            f4 cur[kAggDC];
#pragma unroll
            for (int dc = 0; dc < kAggDC; ++dc)
                cur[dc] = ua[dc];
            if (kb + kMaxWaves < KFC) {
#pragma unroll
                for (int dc = 0; dc < kAggDC; ++dc)
                    ua[dc] = g.uk_a[((int64_t)min(dc, DC - 1) * KFC + kb + kMaxWaves) * kWave +
                                    lane];
            }
            issue_fence();
            f4 acc = f4{0, 0, 0, 0};
#pragma unroll
            for (int dc = 0; dc < kAggDC; ++dc)   // bq is zero past M
                acc = mfma_k16(cur[dc], bq[dc], acc);
#pragma unroll
            for (int v = 0; v < 4; ++v)
                Us[cn * KFP + 16 * kb + q4 + v] = acc[v];
        }
    }
    // 1d. the seed part of the scores: rows = the workgroup's slots (root
    // s / nb, slot s % nb), A = the neighbours' key rows of P (b_k for a slot
    // without one); kept for the slot's own root
    f4 sa[kAggDC];
    {
        const float *krow = ((spos >= 0 && spos < n) ? g.P + (int64_t)spos * g.ldP : g.pbias) + M;
#pragma unroll
        for (int dc = 0; dc < kAggDC; ++dc)
            sa[dc] = *reinterpret_cast<const f4 *>(krow + min(16 * dc + q4, M - 4));
    }
    issue_fence();
    if (seeds) {
        f4 acc = f4{0, 0, 0, 0};
#pragma unroll
        for (int dc = 0; dc < kAggDC; ++dc)
            acc = mfma_k16(sa[dc], bq[dc], acc);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int srow = wave * 16 + q4 + v;
            if (srow < nroots * nb && cr == srow / nb)
                Sk[srow * H + ce] = acc[v];
        }
    }
    // 1e. the own root's slot rows: edge features (HBM), then the time codes
    // phi(t_root - t_slot) computed while those are in flight
    float xs[NBM][kAggCols];   // slot j's columns lane + 64 i
#pragma unroll
    for (int j = 0; j < NBM; ++j) {
        // the slot's event id, the same in every lane (a scalar base address)
        const int ej = __builtin_amdgcn_readfirstlane(__shfl(my_e, j, kWave));
        const float *erow = g.efeat + (int64_t)max(ej, 0) * D_e - D_t;
#pragma unroll
        for (int i = 0; i < kAggCols; ++i) {
            const int k = lane + kWave * i;
            float x = 0.f;
            if (j < c && ej >= 0 && k >= D_t && k < KF)
                x = erow[k];
            xs[j][i] = x;
        }
    }
    issue_fence();
    {
        double om[kAggTCols], be[kAggTCols];
#pragma unroll
        for (int i = 0; i < kAggTCols; ++i) {
            const int k = min(lane + kWave * i, max(D_t - 1, 0));
            om[i] = D_t > 0 ? g.omega[k] : 0.0;
            be[i] = D_t > 0 ? g.beta[k] : 0.0;
        }
#pragma unroll
        for (int j = 0; j < NBM; ++j) {
            const double dtj = __shfl(my_dt, j, kWave);
#pragma unroll
            for (int i = 0; i < kAggTCols; ++i)
                if (lane + kWave * i < D_t)
                    xs[j][i] = j < c ? time_enc(om[i], be[i], dtj) : 0.f;
        }
    }
    __syncthreads();

    // 2. scores, softmax, aggregates (own root); the value seeds of the lane's
    // columns d = lane, lane + 64 and s'_r load first
    const float scale = 1.0f / sqrtf((float)d_h);
    f4 ring[kAggRing];
    if (own) {
        float vs[NBM][2];
#pragma unroll
        for (int j = 0; j < NBM; ++j) {
            const int npj = __shfl(my_np, j, kWave);
            const float *vrow = (npj >= 0 ? g.P + (int64_t)npj * g.ldP : g.pbias) + 2 * M;
#pragma unroll
            for (int u = 0; u < 2; ++u)
                vs[j][u] = (j < c && lane + kWave * u < M) ? vrow[lane + kWave * u] : 0.f;
        }
        float sr_[2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
            sr_[u] = (pv_ok && lane + kWave * u < M) ? g.mem_new[(int64_t)pv * M + lane + kWave * u]
                                                      : 0.f;
        issue_fence();
        float sv[2] = {0.f, 0.f};   // sum_j alpha_j,head(d) seedV_j[d]
#pragma unroll
        for (int eta = 0; eta < kAggMaxH; ++eta) {
            if (eta < H) {
                float uu[kAggCols];
#pragma unroll
                for (int i = 0; i < kAggCols; ++i)
                    uu[i] = lane + kWave * i < KFC * 16
                                ? Us[(wave * H + eta) * KFP + lane + kWave * i] : 0.f;
                float al[NBM];
                float mx = -INFINITY;
#pragma unroll
                for (int j = 0; j < NBM; ++j) {
                    float part = 0.f;
#pragma unroll
                    for (int i = 0; i < kAggCols; ++i)
                        part = fmaf(xs[j][i], uu[i], part);
                    const float seed = Sk[(wave * nb + min(j, nb - 1)) * H + eta];
                    const float scj = (wave_sum_rows(part) + seed) * scale;
                    al[j] = j < c ? scj : -INFINITY;
                    mx = fmaxf(mx, al[j]);
                }
                float den = 0.f;
#pragma unroll
                for (int j = 0; j < NBM; ++j) {
                    al[j] = j < c ? __expf(al[j] - mx) : 0.f;
                    den += al[j];
                }
                const float inv = c > 0 ? 1.0f / den : 0.f;   // no slots: no weights
#pragma unroll
                for (int j = 0; j < NBM; ++j)
                    al[j] *= inv;
                // abar_eta over the lane's columns (zero past KF: xs is)
#pragma unroll
                for (int i = 0; i < kAggCols; ++i) {
                    float a = 0.f;
#pragma unroll
                    for (int j = 0; j < NBM; ++j)
                        a = fmaf(al[j], xs[j][i], a);
                    if (lane + kWave * i < KFC * 16)
                        As[(wave * H + eta) * KFP + lane + kWave * i] = a;
                }
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int d = lane + kWave * u;
                    if (d < M && d / d_h == eta) {
#pragma unroll
                        for (int j = 0; j < NBM; ++j)
                            sv[u] = fmaf(al[j], vs[j][u], sv[u]);
                    }
                }
            }
        }
        // [sum alpha seedV || s'_r || 0]
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int d = lane + kWave * u;
            if (d < M) {
                AO[wave * SAO + d] = sv[u];
                AO[wave * SAO + M + d] = sr_[u];
            }
        }
        for (int k = 2 * M + lane; k < OC * 16; k += kWave)
            AO[wave * SAO + k] = 0.f;
    }
    // the value GEMM's first weight chunks load across the barrier
    const f4 *pwv = g.v_b + (int64_t)min(wave, VNB - 1) * kWave + lane;
    const int64_t vstep = (int64_t)VNB * kWave;
    if (wave < VNB)
        agg_ring_load(pwv, vstep, KFC, ring);
    __syncthreads();

    // 3. value GEMM: [RT H x KF] abar rows x W_v,a^t, column block wave
    if (wave < VNB) {
        const f4 acc = agg_gemm(As + cn * KFP + q4, pwv, vstep, KFC, ring);
        const int col = wave * 16 + cn;
        if (col < M) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = q4 + v, rr = row / H, ee = row - rr * H;
                if (rr < nroots && col / d_h == ee)
                    AO[rr * SAO + col] += acc[v];
            }
        }
    }
    const f4 *pwo = g.out_b + (int64_t)min(wave, ONB - 1) * kWave + lane;
    const int64_t ostep = (int64_t)ONB * kWave;
    if (wave < ONB)
        agg_ring_load(pwo, ostep, OC, ring);
    __syncthreads();

    // 4. h = ReLU(W_o [o || s'_r] + b_o), column block wave
    if (wave < ONB) {
        const f4 acc = agg_gemm(AO + cn * SAO + q4, pwo, ostep, OC, ring);
        const int col = wave * 16 + cn;
        if (col < M) {
            const float bo = g.b_o[col];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = q4 + v;
                if (row < nroots)
                    g.h[(int64_t)(r0 + row) * M + col] = fmaxf(acc[v] + bo, 0.f);
            }
        }
    }
}

template <int NBM>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(NBM <= 10 ? 4 : 2))) void k_attn_agg(AttnArgs g)
{
    extern __shared__ float lds[];
    attn_agg_block<NBM>(g, lds, blockIdx.x);
}

// with the gather of the next iteration's fetch on the blocks past n_attn
// (dispatched last: they take the CUs the attention's tail leaves free)
template <int NBM>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(NBM <= 10 ? 4 : 2))) void k_attn_agg_gather(
    AttnArgs g, int n_attn, GatherPlan gp)
{
    extern __shared__ float lds[];
    if ((int)blockIdx.x < n_attn) {
        attn_agg_block<NBM>(g, lds, blockIdx.x);
        return;
    }
    gather_blocks(gp, (int)blockIdx.x - n_attn, (int)gridDim.x - n_attn, blockDim.x >> 6,
                  threadIdx.x >> 6, threadIdx.x & 63);
}

// q bias folded at creation: c_q = W_q^t phi(0) + b_q with phi(0)_d = cos(beta_d).
__global__ void k_fold_q_bias(int M, int D_t, const float *__restrict__ W_q, const float *b_q,
                              const double *__restrict__ beta, float *c_q)   // may alias b_q
{
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= M)
        return;
    double acc = b_q[k];
    for (int d = 0; d < D_t; ++d)
        acc += (double)W_q[(int64_t)k * (M + D_t) + M + d] * cos(beta[d]);
    c_q[k] = (float)acc;
}

bool attn_lds_opt_in(int bytes, int fold_bytes, int agg_bytes)
{
    if (agg_bytes > 0) {
        const void *fa[] = {(const void *)k_attn_agg<4>, (const void *)k_attn_agg<10>,
                            (const void *)k_attn_agg<16>, (const void *)k_attn_agg_gather<4>,
                            (const void *)k_attn_agg_gather<10>,
                            (const void *)k_attn_agg_gather<16>};
        for (const void *f : fa)
            if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, agg_bytes) !=
                hipSuccess)
                return false;
    }
    const void *fn[] = {(const void *)k_attn<3>, (const void *)k_attn<4>, (const void *)k_attn<5>,
                        (const void *)k_attn_gather<3>, (const void *)k_attn_gather<4>,
                        (const void *)k_attn_gather<5>};
    for (const void *f : fn)
        if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) !=
            hipSuccess)
            return false;
    if (fold_bytes <= 0)
        return true;
    const void *ff[] = {(const void *)k_attn_fold<3>, (const void *)k_attn_fold<4>,
                        (const void *)k_attn_fold<5>, (const void *)k_attn_fold_gather<3>,
                        (const void *)k_attn_fold_gather<4>,
                        (const void *)k_attn_fold_gather<5>};
    for (const void *f : ff)
        if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, fold_bytes) !=
            hipSuccess)
            return false;
    return true;
}

int waves_for(int blocks) { return blocks < kMaxWaves ? (blocks < 1 ? 1 : blocks) : kMaxWaves; }

size_t gru_lds(const tgm_model *m)
{
    return sizeof(float) * (kGruRows * ((m->KXC + m->KHC) * 16 + 4) +
                            4 * kGruSlots * 4 * kWave * 4) +
           2 * sizeof(double) * m->D_t;
}

size_t proj_lds(const tgm_model *m) { return sizeof(float) * 16 * (m->PC * 16 + 4); }

int attn_roots(const tgm_model *m, int *RBa)
{
    // slots of RT roots fill at most 5 MFMA row blocks; for 1 <= nb <= 64 this
    // gives 3 <= RBa <= 5 (the instantiations of k_attn)
    int rb = 5;
    int RT = (16 * rb) / m->nb;
    if (RT < 1)
        RT = 1;
    *RBa = (int)cdiv((int64_t)RT * m->nb, 16);
    return RT;
}

size_t attn_lds(const tgm_model *m)
{
    int RBa;
    const int RT = attn_roots(m, &RBa);
    const int RA = RBa * 16;
    const int SA = m->KFC * 16 + 4, SKV = m->KVNB * 16 + 4;
    const int ORB = (RT + 15) / 16;
    const size_t before_s = (size_t)RA * (SA > SKV ? SA : SKV) + (size_t)RT * m->M +
                            (size_t)ORB * 16 * (m->OC * 16 + 4);
    const size_t om =
        (before_s + (size_t)m->H * std::max(RA, 16 * RT) + 1) & ~(size_t)1;   // as in k_attn
    return sizeof(float) * om + 2 * sizeof(double) * m->D_t;
}

// LDS of k_attn_fold (the layout in attn_fold_block)
size_t attn_fold_lds(const tgm_model *m)
{
    int RBa;
    const int RT = attn_roots(m, &RBa);
    const size_t RA = (size_t)RBa * 16, SA = (size_t)m->KFC * 16 + 4;
    const size_t ORB = (size_t)(RT + 15) / 16, SAO = (size_t)m->OC * 16 + 4;
    const size_t fl = RA * SA + (size_t)m->KFC * kWave * 4 + ORB * 16 * SAO + RA * m->H +
                      (size_t)RT * m->H * 16;
    return sizeof(float) * ((fl + 1) & ~(size_t)1) + 2 * sizeof(double) * m->D_t;
}

// Shapes the folded attention handles: rows of 16 lanes hold a root's slots,
// one 16-column score block (RT * H <= 16), V blocks and the score wave within
// kMaxWaves, the U tiles within kAttUT per U wave, V within the slot-row region
bool attn_fold_fits(const tgm_model *m)
{
    int RBa;
    const int RT = attn_roots(m, &RBa);
    const int DC = (int)cdiv(m->M, 16);
    int nu = 0;
    for (int w = 0; w < kMaxWaves; ++w)
        nu += (w & 3) != (DC & 3);
    return m->nb <= 16 && m->M % 4 == 0 && DC <= kAttDC && DC + 1 <= kMaxWaves &&
           RT * m->H <= 16 && m->KFC <= kAttUT * nu && DC <= m->KFC &&
           attn_fold_lds(m) <= 160 * 1024;
}

// Roots per workgroup of the attention by aggregation: one per wavefront,
// RT H <= 16 (one 16-row MFMA block of (root, head) rows)
int attn_agg_roots(const tgm_model *m) { return std::min(kMaxWaves, 16 / std::max(m->H, 1)); }

size_t attn_agg_lds(const tgm_model *m)
{
    return sizeof(float) * (2 * 16 * ((size_t)m->KFC * 16 + 4) + 16 * ((size_t)m->OC * 16 + 4) +
                            (size_t)attn_agg_roots(m) * m->nb * m->H);
}

// Shapes the attention by aggregation handles: slots and time codes within
// the registers of a lane, M within 8 column blocks (one per wave) and two
// columns per lane, the U tiles within kAggUT per wave
bool attn_agg_fits(const tgm_model *m)
{
    const int KF = m->D_e + m->D_t;
    return m->nb >= 1 && m->nb <= 16 && m->M % 4 == 0 && m->M <= 112 && m->H >= 1 &&
           m->H <= kAggMaxH && m->M % m->H == 0 && KF >= 1 && KF <= kAggCols * kWave &&
           m->D_t <= kAggTCols * kWave && m->KFC <= kAggUT * kMaxWaves &&
           m->VNB <= kMaxWaves && m->ONB <= kMaxWaves && m->DC <= kAggDC &&
           m->OC <= kAggMaxKC && m->KFC <= kAggMaxKC &&
           attn_agg_lds(m) <= 64 * 1024;
}

}  // namespace

// ======================================================================== API

namespace {

// The JODIE part of tgm_model_create: the RNN cell's operands in the GRU
// kernel's layout (one gate block, in the slot of the GRU's n gate, and its
// biases b_ih, b_hh in the n slots), the time encoding, the time projection
// and the executor's buffer of new memory times.
// The resident-weight GRU when the shapes fit: its phi buffer and LDS opt-in.
tgm_status_t gru_w_setup(tgm_model *m, int NG)
{
    m->gru_w = gru_w_fits(m, NG);
    if (!m->gru_w)
        return TGM_OK;
    if (dev_malloc((void **)&m->phi,
                   sizeof(float) * std::max<size_t>(1, (size_t)m->max_nodes * m->D_t)) !=
        hipSuccess)
        return TGM_ENOMEM;
    const void *f = NG == 1 ? (const void *)k_gru_w<1> : (const void *)k_gru_w<3>;
    if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)gru_w_lds(m, NG)) != hipSuccess)
        return TGM_EINVAL;
    return TGM_OK;
}

tgm_status_t create_jodie(tgm_model *m, const tgm_model_desc *d, const tgm_weights *w)
{
    const int M = m->M, D_x = m->D_x, D_t = m->D_t, MP = m->MB * 16;
    auto bx = pack_b(w->W_ih, M, D_x, 0, D_x, m->KXC, m->MB);
    auto bh = pack_b(w->W_hh, M, M, 0, M, m->KHC, m->MB);
    bx.resize(bx.size() + 2 * (size_t)m->MB * kWave * 4, 0.f);   // two zero chunks past the end
    bh.resize(bh.size() + 2 * (size_t)m->MB * kWave * 4, 0.f);
    std::vector<float> bias(4 * (size_t)MP, 0.f);
    for (int k = 0; k < M; ++k) {
        bias[2 * MP + k] = w->b_ih[k];
        bias[3 * MP + k] = w->b_hh[k];
    }
    auto alloc = [](void **p, size_t bytes) {
        return dev_malloc(p, bytes ? bytes : 16) == hipSuccess;
    };
    if (!alloc((void **)&m->gru_bx, bx.size() * 4) || !alloc((void **)&m->gru_bh, bh.size() * 4) ||
        !alloc((void **)&m->gru_bias, bias.size() * 4) ||
        !alloc((void **)&m->omega, sizeof(double) * D_t) ||
        !alloc((void **)&m->beta, sizeof(double) * D_t) || !alloc((void **)&m->w_t, 4 * M) ||
        !alloc((void **)&m->nts, sizeof(double) * (size_t)d->max_nodes))
        return TGM_ENOMEM;
    TGM_TRY_STATUS(upload(m->gru_bx, bx.data(), bx.size() * 4));
    TGM_TRY_STATUS(upload(m->gru_bh, bh.data(), bh.size() * 4));
    TGM_TRY_STATUS(upload(m->gru_bias, bias.data(), bias.size() * 4));
    if (D_t > 0) {
        TGM_TRY_STATUS(upload(m->omega, w->omega, sizeof(double) * D_t));
        TGM_TRY_STATUS(upload(m->beta, w->beta, sizeof(double) * D_t));
    }
    TGM_TRY_STATUS(upload(m->w_t, w->w_t, 4 * M));
    if (hipFuncSetAttribute((const void *)k_gru<1>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)gru_lds(m)) != hipSuccess)
        return TGM_EINVAL;
    return gru_w_setup(m, 1);
}

}  // namespace

extern "C" tgm_status_t tgm_model_destroy(tgm_model_t m)
{
    if (!m)
        return TGM_EINVAL;
    hipFree(m->gru_bx);
    hipFree(m->gru_bh);
    hipFree(m->gru_bias);
    hipFree(m->omega);
    hipFree(m->beta);
    hipFree(m->proj_b);
    hipFree(m->P);
    hipFree(m->kv_b);
    hipFree(m->v_b);
    hipFree(m->uk_a);
    hipFree(m->pbias);
    hipFree(m->out_b);
    hipFree(m->b_o);
    hipFree(m->w_t);
    hipFree(m->nts);
    hipFree(m->phi);
    delete m;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_model_create(const tgm_model_desc *d, const tgm_weights *w,
                                         void *stream, tgm_model_t *out)
{
    if (!d || !w || !out)
        return TGM_EINVAL;
    *out = nullptr;
    const int M = d->M, D_e = d->D_e, D_t = d->D_t, H = d->H, nb = d->nb;
    // limits of the kernels' tiling: K|V column blocks fit kMaxWaves * kAttMaxCB
    // wavefront slots (M <= 128), a wavefront stages rows of at most 256 edge
    // features (so D_m <= 512); LDS bounds D_e + D_t (checked below)
    if (M <= 0 || D_e < 0 || D_t < 0 || H <= 0 || M % H != 0 || nb < 1 || nb > 64 ||
        d->max_nodes <= 0 || d->max_roots < 0 || 2 * M > 16 * kMaxWaves * kAttMaxCB ||
        D_e > 256)
        return TGM_EINVAL;
    if (!w->W_ih || !w->W_hh || !w->b_ih || !w->b_hh || (D_t > 0 && (!w->omega || !w->beta)))
        return TGM_EINVAL;
    if (d->kind == TGM_MODEL_JODIE ? !w->w_t
                                   : (!w->W_q || !w->b_q || !w->W_k || !w->b_k || !w->W_v ||
                                      !w->b_v || !w->W_o || !w->b_o))
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    tgm_model *m = new tgm_model();
    m->M = M; m->D_e = D_e; m->D_t = D_t; m->H = H; m->nb = nb;
    m->max_nodes = d->max_nodes; m->max_roots = d->max_roots;
    m->D_m = 2 * M + D_e;
    m->D_x = m->D_m + D_t;
    m->KXC = (int)cdiv(m->D_x, 16);
    m->KHC = (int)cdiv(M, 16);
    m->MB = (int)cdiv(M, 16);
    m->PC = m->KHC;
    m->PNB = (int)cdiv(3 * M, 16);
    m->KFC = (int)cdiv(D_e + D_t > 0 ? D_e + D_t : 1, 16);
    m->KVNB = (int)cdiv(2 * M, 16);
    m->OC = (int)cdiv(2 * M, 16);
    m->ONB = (int)cdiv(M, 16);
    m->VNB = m->DC = (int)cdiv(M, 16);
    m->kind = d->kind;
    if (d->kind == TGM_MODEL_JODIE) {
        const tgm_status_t st = create_jodie(m, d, w);
        if (st != TGM_OK) {
            tgm_model_destroy(m);
            return st;
        }
        *out = m;
        return TGM_OK;
    }
    if (d->kind != TGM_MODEL_TGN) {
        tgm_model_destroy(m);
        return TGM_EINVAL;
    }
    m->fold = attn_fold_fits(m);
    m->agg = attn_agg_fits(m);

    // GRU operands
    const int D_x = m->D_x, MP = m->MB * 16;
    std::vector<float> bx, bh;
    for (int gte = 0; gte < 3; ++gte) {
        auto px = pack_b(w->W_ih + (size_t)gte * M * D_x, M, D_x, 0, D_x, m->KXC, m->MB);
        auto ph = pack_b(w->W_hh + (size_t)gte * M * M, M, M, 0, M, m->KHC, m->MB);
        bx.insert(bx.end(), px.begin(), px.end());
        bh.insert(bh.end(), ph.begin(), ph.end());
    }
    std::vector<float> bias(4 * (size_t)MP, 0.f);
    for (int k = 0; k < M; ++k) {
        bias[k] = w->b_ih[k] + w->b_hh[k];
        bias[MP + k] = w->b_ih[M + k] + w->b_hh[M + k];
        bias[2 * MP + k] = w->b_ih[2 * M + k];
        bias[3 * MP + k] = w->b_hh[2 * M + k];
    }
    // node projections: rows of [W_q^s; W_k^s; W_v^s] (3M x M)
    const int Dq = M + D_t, Dkv = M + D_e + D_t;
    std::vector<float> wp((size_t)3 * M * M);
    for (int n = 0; n < M; ++n)
        for (int k = 0; k < M; ++k) {
            wp[(size_t)n * M + k] = w->W_q[(size_t)n * Dq + k];
            wp[(size_t)(M + n) * M + k] = w->W_k[(size_t)n * Dkv + k];
            wp[(size_t)(2 * M + n) * M + k] = w->W_v[(size_t)n * Dkv + k];
        }
    auto pb = pack_b(wp.data(), 3 * M, M, 0, M, m->PC, m->PNB);
    // per-slot part of [K | V]: columns M .. M + D_e + D_t of W_k and W_v
    const int KF = D_e + D_t;
    std::vector<float> wkv((size_t)2 * M * (KF > 0 ? KF : 1), 0.f);
    for (int n = 0; n < M; ++n)
        for (int k = 0; k < KF; ++k) {
            // slot row order [phi || efeat]: column k < D_t is time code k, the
            // rest edge feature k - D_t (W's own order is [s || efeat || phi])
            const int src = k < D_t ? M + D_e + k : M + k - D_t;
            wkv[(size_t)n * KF + k] = w->W_k[(size_t)n * Dkv + src];
            wkv[(size_t)(M + n) * KF + k] = w->W_v[(size_t)n * Dkv + src];
        }
    auto kvb = pack_b(wkv.data(), 2 * M, KF, 0, KF, m->KFC, m->KVNB);
    // folded attention: the V rows alone, and W_k^t [KF x M] as A fragments
    std::vector<float> vb, uka;
    if (m->fold || m->agg) {
        vb = pack_b(wkv.data() + (size_t)M * (KF > 0 ? KF : 1), M, KF, 0, KF, m->KFC, m->VNB);
        vb.resize((size_t)std::max(m->KFC + 2, kAttPre) * m->VNB * kWave * 4, 0.f);
        std::vector<float> wkt((size_t)(KF > 0 ? KF : 1) * M, 0.f);
        for (int d = 0; d < M; ++d)
            for (int k = 0; k < KF; ++k)
                wkt[(size_t)k * M + d] = wkv[(size_t)d * KF + k];
        uka = pack_b(wkt.data(), KF, M, 0, M, m->DC, m->KFC);
    }
    auto ob = pack_b(w->W_o, M, 2 * M, 0, 2 * M, m->OC, m->ONB);
    // two zero k-chunks past the end of every packed operand: the kernels
    // load chunks kc + 1 and kc + 2 while multiplying chunk kc
    bx.resize(bx.size() + 2 * (size_t)m->MB * kWave * 4, 0.f);
    bh.resize(bh.size() + 2 * (size_t)m->MB * kWave * 4, 0.f);
    pb.resize(pb.size() + 2 * (size_t)m->PNB * kWave * 4, 0.f);
    // (and at least kAttPre chunks: k_attn preloads that many)
    kvb.resize((size_t)std::max(m->KFC + 2, kAttPre) * m->KVNB * kWave * 4, 0.f);
    // (k_attn loads kAttMaxOC chunks)
    ob.resize((size_t)std::max(m->OC + 2, kAttMaxOC) * m->ONB * kWave * 4, 0.f);

    float *wq_dev = nullptr;
    tgm_status_t st = TGM_OK;
    do {
        auto alloc = [&](void **p, size_t bytes) {
            return dev_malloc(p, bytes ? bytes : 16) == hipSuccess;
        };
        if (!alloc((void **)&m->gru_bx, bx.size() * 4) || !alloc((void **)&m->gru_bh, bh.size() * 4) ||
            !alloc((void **)&m->gru_bias, bias.size() * 4) ||
            !alloc((void **)&m->omega, sizeof(double) * D_t) ||
            !alloc((void **)&m->beta, sizeof(double) * D_t) ||
            !alloc((void **)&m->proj_b, pb.size() * 4) ||
            !alloc((void **)&m->P, sizeof(float) * (size_t)d->max_nodes * m->PNB * 16) ||
            !alloc((void **)&m->kv_b, kvb.size() * 4) ||
            ((m->fold || m->agg) && (!alloc((void **)&m->v_b, vb.size() * 4) ||
                         !alloc((void **)&m->uk_a, uka.size() * 4))) ||
            !alloc((void **)&m->pbias, sizeof(float) * m->PNB * 16) ||
            !alloc((void **)&m->out_b, ob.size() * 4) || !alloc((void **)&m->b_o, 4 * M) ||
            !alloc((void **)&wq_dev, sizeof(float) * (size_t)M * Dq)) {
            st = TGM_ENOMEM;
            break;
        }
        if ((st = upload(m->gru_bx, bx.data(), bx.size() * 4)) != TGM_OK) break;
        if ((st = upload(m->gru_bh, bh.data(), bh.size() * 4)) != TGM_OK) break;
        if ((st = upload(m->gru_bias, bias.data(), bias.size() * 4)) != TGM_OK) break;
        if (D_t > 0) {
            if ((st = upload(m->omega, w->omega, sizeof(double) * D_t)) != TGM_OK) break;
            if ((st = upload(m->beta, w->beta, sizeof(double) * D_t)) != TGM_OK) break;
        }
        if ((st = upload(m->proj_b, pb.data(), pb.size() * 4)) != TGM_OK) break;
        if ((st = upload(m->kv_b, kvb.data(), kvb.size() * 4)) != TGM_OK) break;
        if (m->fold || m->agg) {
            if ((st = upload(m->v_b, vb.data(), vb.size() * 4)) != TGM_OK) break;
            if ((st = upload(m->uk_a, uka.data(), uka.size() * 4)) != TGM_OK) break;
        }
        {   // b_q (folded into c_q in place below), b_k, b_v, zero padding
            std::vector<float> pbias((size_t)m->PNB * 16, 0.f);
            std::copy(w->b_q, w->b_q + M, pbias.begin());
            std::copy(w->b_k, w->b_k + M, pbias.begin() + M);
            std::copy(w->b_v, w->b_v + M, pbias.begin() + 2 * M);
            if ((st = upload(m->pbias, pbias.data(), pbias.size() * 4)) != TGM_OK) break;
        }
        if ((st = upload(m->out_b, ob.data(), ob.size() * 4)) != TGM_OK) break;
        if ((st = upload(m->b_o, w->b_o, 4 * M)) != TGM_OK) break;
        if ((st = upload(wq_dev, w->W_q, sizeof(float) * (size_t)M * Dq)) != TGM_OK) break;
        hipLaunchKernelGGL(k_fold_q_bias, dim3(cdiv(M, 64)), dim3(64), 0, s, M, D_t, wq_dev,
                           m->pbias, m->beta, m->pbias);
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
            st = TGM_EDEVICE;
            break;
        }
        // large LDS footprints need an explicit opt-in
        if (hipFuncSetAttribute((const void *)k_gru<3>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)gru_lds(m)) != hipSuccess ||
            hipFuncSetAttribute((const void *)k_node_proj,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)proj_lds(m)) != hipSuccess ||
            !attn_lds_opt_in((int)attn_lds(m), m->fold ? (int)attn_fold_lds(m) : 0,
                             m->agg ? (int)attn_agg_lds(m) : 0)) {
            st = TGM_EINVAL;   // dimensions beyond the LDS of one workgroup
            break;
        }
        if ((st = gru_w_setup(m, 3)) != TGM_OK)
            break;
    } while (0);
    hipFree(wq_dev);
    if (st != TGM_OK) {
        tgm_model_destroy(m);
        return st;
    }
    *out = m;
    return TGM_OK;
}

namespace {

// Host side of tgm_update_memory: the checks, the GRU launch (with the
// latest-message reduce) on s, the staging launch's arguments (*sa, *n_items
// wavefront items) and the protocol bookkeeping.  *tag is the call's key tag.
tgm_status_t update_begin(tgm_state_t st, tgm_model_t m, tgm_graph_t g, int64_t iter,
                          const int32_t *n_nodes, int32_t cap, const float *mem,
                          const double *mem_ts, const float *mail, const double *mail_ts,
                          const int32_t *ver, int64_t first_event, int32_t b,
                          const int32_t *src_pos, const int32_t *dst_pos, float *mem_new,
                          double *new_mem_ts, hipStream_t s, StageArgs *sa, int *n_items,
                          uint64_t *tag_out, uint64_t *ext_win = nullptr, uint64_t ext_tag = 0,
                          bool phi_ready = false, const int32_t *inplace_nodes = nullptr)
{
    if (!st || !m || !g || !n_nodes || cap < 0 || b < 0 || first_event < 0 ||
        first_event + b > g->E)
        return TGM_EINVAL;
    if (inplace_nodes && (!m->gru_w || !phi_ready || !new_mem_ts))
        return TGM_EINVAL;   // only the resident-weights GRU reads the tables in place
    if (m->M != st->M || m->D_m != st->D_m || g->D_e != m->D_e || g->N != st->N)
        return TGM_EINVAL;
    if (b > st->max_batch)
        return TGM_ESIZE;
    if (cap > m->max_nodes || cap > st->N)
        return TGM_ESIZE;
    if (cap > 0 && (!mem || !mem_ts || !mail || !mail_ts || !ver || !mem_new))
        return TGM_EINVAL;
    if (b > 0 && (!src_pos || !dst_pos || cap == 0))
        return TGM_EINVAL;
    if (iter != st->staged_through + 1)
        return TGM_EORDER;
    const int slots = st->s + 1;
    if (iter - slots > st->committed_through)
        return TGM_EORDER;   // the slot still holds an uncommitted write set
    // the keys of this update's latest-message reduce: the state's array, or
    // one the executor reduced already (ext_win; the GRU then skips the reduce)
    uint64_t *win = ext_win ? ext_win : st->win;
    uint64_t tag = ext_tag;
    if (!ext_win) {
        if (st->win_tag == UINT32_MAX) {   // keys restart from zero
            TGM_LAUNCH(k_fill_u64, dim3(cdiv(st->N, 256)), dim3(256), 0, s, st->win, st->N);
            st->win_tag = 0;
        }
        tag = (uint64_t)(++st->win_tag) << 32;
    }
    const int n_cand = 2 * b;
    if (cap > 0) {
        GruArgs ga;
        ga.n_nodes = n_nodes; ga.nodes = nullptr; ga.mem = mem; ga.mail = mail;
        ga.mem_ts = mem_ts; ga.mail_ts = mail_ts; ga.ver = ver;
        if (inplace_nodes) {   // the committed tables, read in place
            ga.nodes = inplace_nodes; ga.mem = st->mem; ga.mail = st->mail;
            ga.mem_ts = st->mem_ts; ga.mail_ts = st->mail_ts; ga.ver = st->ver;
        }
        ga.bx = m->gru_bx; ga.bh = m->gru_bh;
        ga.bias = m->gru_bias; ga.omega = m->omega; ga.beta = m->beta; ga.M = m->M;
        ga.D_m = m->D_m; ga.D_t = m->D_t; ga.KXC = m->KXC; ga.KHC = m->KHC; ga.MB = m->MB;
        ga.mem_new = mem_new; ga.new_mem_ts = new_mem_ts;
        ga.n_cand = ext_win ? 0 : n_cand; ga.src_pos = src_pos; ga.dst_pos = dst_pos;
        ga.win = win; ga.tag = tag;
        const bool jodie = m->kind == TGM_MODEL_JODIE;
        const bool w_ok = m->gru_w &&
                          ((reinterpret_cast<uintptr_t>(ga.mem) |
                            reinterpret_cast<uintptr_t>(ga.mail)) & 7) == 0;
        if (inplace_nodes && (!w_ok || !phi_ready || !new_mem_ts))
            return TGM_EINVAL;   // only the resident-weights GRU reads in place
        if (w_ok) {
            // phi once per node (unless the fetch formed it), then MB hidden
            // blocks x (kGruGrid / MB) row ranges (kGruGrid % MB workgroups idle)
            if (m->D_t > 0 && !phi_ready)
                TGM_LAUNCH(k_phi, dim3((unsigned)cdiv((int64_t)cap * m->D_t, 256)), dim3(256), 0,
                           s, n_nodes, cap, m->D_t, mem_ts, mail_ts, ver, m->omega, m->beta,
                           m->phi);
            const dim3 grid((unsigned)kGruGrid);
            if (jodie)
                TGM_LAUNCH(k_gru_w<1>, grid, dim3(64 * kGwWaves), gru_w_lds(m, 1), s, ga,
                           m->phi);
            else
                TGM_LAUNCH(k_gru_w<3>, grid, dim3(64 * kGwWaves), gru_w_lds(m, 3), s, ga,
                           m->phi);
        } else if (jodie) {
            // persistent: the node set's tasks are split over kGruGrid workgroups
            TGM_LAUNCH(k_gru<1>, dim3(kGruGrid), dim3(64 * kGruWaves), gru_lds(m), s, ga);
        } else {
            TGM_LAUNCH(k_gru<3>, dim3(kGruGrid), dim3(64 * kGruWaves), gru_lds(m), s, ga);
        }
    }
    const size_t base = (size_t)(iter % slots) * st->ring_rows();
    // the write set of iteration iter - s is committed by the staging launch
    // when it is the next one due (s = 0: the current write set goes to the
    // tables)
    const bool direct = st->s == 0;
    const int64_t cj = iter - st->s;
    const tgm_state::Slot &cs = st->ring[((cj % slots) + slots) % slots];
    const bool fuse = !direct && cj >= 0 && cj == st->committed_through + 1 && cs.staged &&
                      cs.iter == cj;
    const int n_commit = fuse ? 2 * cs.b : 0;
    const size_t cbase = (size_t)(((cj % slots) + slots) % slots) * st->ring_rows();
    StageArgs &a = *sa;
    a.n_cand = n_cand; a.n_commit = n_commit;
    a.first = first_event; a.iter = iter; a.c_iter = cj;
    a.M = m->M; a.D_m = m->D_m; a.D_e = m->D_e; a.direct = direct;
    a.n_nodes = n_nodes; a.src = g->src; a.dst = g->dst; a.src_pos = src_pos;
    a.dst_pos = dst_pos; a.win = win; a.tag = tag; a.ver = ver;
    a.t = g->t; a.mem_ts = mem_ts; a.mail_ts = mail_ts; a.efeat = g->efeat;
    a.nts_new = inplace_nodes ? new_mem_ts : nullptr;
    a.mem_new = mem_new;
    a.r_flag = st->r_flag + base; a.r_node = st->r_node + base;
    a.r_mem = st->r_mem + base * st->M; a.r_mail = st->r_mail + base * st->D_m;
    a.r_mem_ts = st->r_mem_ts + base; a.r_mail_ts = st->r_mail_ts + base;
    a.c_flag = st->r_flag + cbase; a.c_node = st->r_node + cbase;
    a.c_mem = st->r_mem + cbase * st->M; a.c_mail = st->r_mail + cbase * st->D_m;
    a.c_mem_ts = st->r_mem_ts + cbase; a.c_mail_ts = st->r_mail_ts + cbase;
    a.mem = st->mem; a.mail = st->mail; a.t_mem_ts = st->mem_ts; a.t_mail_ts = st->mail_ts;
    a.t_ver = st->ver;
    *n_items = n_cand + n_commit;
    *tag_out = tag;
    if (fuse) {
        st->ring[cj % slots].staged = false;
        st->committed_through = cj;
    }
    if (direct) {
        st->committed_through = iter;
    } else {
        tgm_state::Slot &sl = st->ring[iter % slots];
        sl.iter = iter;
        sl.b = b;
        sl.staged = true;
    }
    st->staged_through = iter;
    return TGM_OK;
}

tgm_status_t update_winner(const uint64_t *win, const int32_t *n_nodes, int32_t cap,
                           int64_t first_event, uint64_t tag, int64_t *winner, hipStream_t s)
{
    if (winner && cap > 0)
        TGM_LAUNCH(k_winner_out, dim3(cdiv(cap, 256)), dim3(256), 0, s, n_nodes, cap,
                   first_event, win, tag, winner);
    return TGM_OK;
}

// Checks of tgm_embed and the arguments of its two launches.
tgm_status_t embed_plan(tgm_model_t m, tgm_graph_t g, int32_t R, int32_t nb,
                        const int32_t *root_pos, const double *root_ts, const int32_t *nbr_pos,
                        const int32_t *eid, const double *nts, const int32_t *cnt,
                        const float *mem_new, const int32_t *n_nodes, int32_t cap, float *h,
                        ProjArgs *pa, int *proj_grid, int *proj_waves, AttnArgs *aa)
{
    if (!m || !g || R < 0 || nb != m->nb || !n_nodes || cap < 0 || g->D_e != m->D_e ||
        m->kind != TGM_MODEL_TGN)
        return TGM_EINVAL;
    if (R > m->max_roots || cap > m->max_nodes)
        return TGM_ESIZE;
    if (R == 0)
        return TGM_OK;
    if (!root_pos || !root_ts || !nbr_pos || !eid || !nts || !cnt || !mem_new || !h || cap == 0)
        return TGM_EINVAL;
    // persistent grid: at most the tiles of the largest node set; every wave
    // owns up to three column blocks
    // column groups of at most kMaxWaves blocks, one block per wave; a grid of
    // up to 512 workgroups, a multiple of the group count
    const int CS = (int)cdiv(m->PNB, kMaxWaves);
    *proj_waves = std::max<int>(4, (int)cdiv(m->PNB, CS));
    *proj_grid = (int)std::min<int64_t>(cdiv(cap, 16) * CS, 512 / CS * CS);
    pa->CS = CS;
    pa->n_nodes = n_nodes; pa->mem_new = mem_new; pa->M = m->M; pa->PC = m->PC;
    pa->PNB = m->PNB; pa->pb = m->proj_b; pa->pbias = m->pbias; pa->P = m->P;
    AttnArgs &a = *aa;
    a.R = R; a.nb = nb; a.RT = attn_roots(m, &a.RBa); a.M = m->M; a.H = m->H;
    if (m->agg)
        a.RT = attn_agg_roots(m);
    a.E = g->E; a.n_nodes = n_nodes;
    a.D_e = m->D_e; a.D_t = m->D_t;
    a.root_pos = root_pos; a.nbr_pos = nbr_pos; a.eid = eid; a.cnt = cnt;
    a.root_ts = root_ts; a.nts = nts;
    a.P = m->P; a.ldP = m->PNB * 16;
    a.efeat = g->efeat; a.omega = m->omega; a.beta = m->beta;
    a.kv_b = m->kv_b; a.KFC = m->KFC; a.KVNB = m->KVNB;
    a.pbias = m->pbias;
    a.v_b = m->v_b; a.uk_a = m->uk_a; a.VNB = m->VNB; a.DC = m->DC;
    a.out_b = m->out_b; a.OC = m->OC; a.ONB = m->ONB; a.b_o = m->b_o;
    a.mem_new = mem_new; a.h = h;
    return a.RBa >= 3 && a.RBa <= 5 ? TGM_OK : TGM_EINVAL;
}

// The attention launch, with the gather of `next` in the same launch when
// given (extra blocks after the attention's).
tgm_status_t launch_attn(const tgm_model *m, const AttnArgs &a, const GatherPlan *next,
                         hipStream_t s)
{
    const int n_attn = (int)cdiv(a.R, a.RT);
    const dim3 block(64 * kMaxWaves);
    if (m->agg) {
        const size_t lds = attn_agg_lds(m);
        const int nbm = a.nb <= 4 ? 4 : a.nb <= 10 ? 10 : 16;
        if (next && next->cap > 0) {
            // one gather block per CU after the attention's blocks
            const dim3 grid(n_attn + kCUs);
            switch (nbm) {
            case 4: TGM_LAUNCH(k_attn_agg_gather<4>, grid, block, lds, s, a, n_attn, *next); break;
            case 10: TGM_LAUNCH(k_attn_agg_gather<10>, grid, block, lds, s, a, n_attn, *next); break;
            default: TGM_LAUNCH(k_attn_agg_gather<16>, grid, block, lds, s, a, n_attn, *next); break;
            }
            return TGM_OK;
        }
        const dim3 grid(n_attn);
        switch (nbm) {
        case 4: TGM_LAUNCH(k_attn_agg<4>, grid, block, lds, s, a); break;
        case 10: TGM_LAUNCH(k_attn_agg<10>, grid, block, lds, s, a); break;
        default: TGM_LAUNCH(k_attn_agg<16>, grid, block, lds, s, a); break;
        }
        return TGM_OK;
    }
    const size_t lds = m->fold ? attn_fold_lds(m) : attn_lds(m);
    // the gather rides along when the attention's last round of blocks
    // leaves CUs free: its blocks are dispatched after the attention's, hold
    // one CU each (they carry the attention's LDS size) and fill that round;
    // otherwise it is its own launch
    const int spare = (kCUs - n_attn % kCUs) % kCUs;
    if (next && next->cap > 0 && spare < 8) {
        TGM_TRY_STATUS(launch_gather(*next, s));
        next = nullptr;
    }
    if (next && next->cap > 0) {
        const int n_gather = spare;
        const dim3 grid(n_attn + n_gather);
        if (m->fold) {
            switch (a.RBa) {
            case 3: TGM_LAUNCH(k_attn_fold_gather<3>, grid, block, lds, s, a, n_attn, *next); break;
            case 4: TGM_LAUNCH(k_attn_fold_gather<4>, grid, block, lds, s, a, n_attn, *next); break;
            default: TGM_LAUNCH(k_attn_fold_gather<5>, grid, block, lds, s, a, n_attn, *next); break;
            }
            return TGM_OK;
        }
        switch (a.RBa) {
        case 3: TGM_LAUNCH(k_attn_gather<3>, grid, block, lds, s, a, n_attn, *next); break;
        case 4: TGM_LAUNCH(k_attn_gather<4>, grid, block, lds, s, a, n_attn, *next); break;
        default: TGM_LAUNCH(k_attn_gather<5>, grid, block, lds, s, a, n_attn, *next); break;
        }
        return TGM_OK;
    }
    const dim3 grid(n_attn);
    if (m->fold) {
        switch (a.RBa) {
        case 3: TGM_LAUNCH(k_attn_fold<3>, grid, block, lds, s, a); break;
        case 4: TGM_LAUNCH(k_attn_fold<4>, grid, block, lds, s, a); break;
        default: TGM_LAUNCH(k_attn_fold<5>, grid, block, lds, s, a); break;
        }
        return TGM_OK;
    }
    switch (a.RBa) {
    case 3: TGM_LAUNCH(k_attn<3>, grid, block, lds, s, a); break;
    case 4: TGM_LAUNCH(k_attn<4>, grid, block, lds, s, a); break;
    default: TGM_LAUNCH(k_attn<5>, grid, block, lds, s, a); break;
    }
    return TGM_OK;
}

}  // namespace

extern "C" tgm_status_t tgm_update_memory(tgm_state_t st, tgm_model_t m, tgm_graph_t g,
                                          int64_t iter, const int32_t *nodes,
                                          const int32_t *n_nodes, int32_t cap, const float *mem,
                                          const double *mem_ts, const float *mail,
                                          const double *mail_ts, const int32_t *ver,
                                          int64_t first_event, int32_t b, const int32_t *src_pos,
                                          const int32_t *dst_pos, float *mem_new,
                                          double *new_mem_ts, int64_t *winner, void *stream)
{
    (void)nodes;
    const hipStream_t s = as_stream(stream);
    StageArgs sa;
    int n_items = 0;
    uint64_t tag = 0;
    tgm_status_t rc = update_begin(st, m, g, iter, n_nodes, cap, mem, mem_ts, mail, mail_ts, ver,
                                   first_event, b, src_pos, dst_pos, mem_new, new_mem_ts, s, &sa,
                                   &n_items, &tag);
    if (rc != TGM_OK)
        return rc;
    if (n_items > 0)
        TGM_LAUNCH(k_stage, dim3(cdiv(n_items, 4)), dim3(256), 0, s, sa);
    return update_winner(st->win, n_nodes, cap, first_event, tag, winner, s);
}

extern "C" tgm_status_t tgm_embed(tgm_model_t m, tgm_graph_t g, int32_t R, int32_t nb,
                                  const int32_t *root_pos, const double *root_ts,
                                  const int32_t *nbr_pos, const int32_t *eid, const double *nts,
                                  const int32_t *cnt, const float *mem_new,
                                  const int32_t *n_nodes, int32_t cap, float *h, void *stream)
{
    const hipStream_t s = as_stream(stream);
    ProjArgs pa;
    AttnArgs aa;
    int proj_grid = 0, proj_waves = 0;
    const tgm_status_t rc = embed_plan(m, g, R, nb, root_pos, root_ts, nbr_pos, eid, nts, cnt,
                                       mem_new, n_nodes, cap, h, &pa, &proj_grid, &proj_waves,
                                       &aa);
    if (rc != TGM_OK || R == 0)
        return rc;
    TGM_LAUNCH(k_node_proj, dim3(proj_grid), dim3(64 * proj_waves), proj_lds(m), s, pa);
    return launch_attn(m, aa, nullptr, s);
}

namespace {

tgm_status_t tproj_plan(tgm_model_t m, int32_t R, const int32_t *root_pos,
                        const double *root_ts, const float *mem_new, const double *new_mem_ts,
                        const int32_t *n_nodes, int32_t cap, float *h, TprojArgs *a)
{
    if (!m || m->kind != TGM_MODEL_JODIE || R < 0 || cap < 0 || !n_nodes)
        return TGM_EINVAL;
    if (R > m->max_roots || cap > m->max_nodes)
        return TGM_ESIZE;
    if (R > 0 && (!root_pos || !root_ts || !mem_new || !new_mem_ts || !h || cap == 0))
        return TGM_EINVAL;
    a->R = R; a->M = m->M; a->root_pos = root_pos; a->n_nodes = n_nodes;
    a->root_ts = root_ts; a->nts = new_mem_ts; a->mem_new = mem_new; a->w_t = m->w_t; a->h = h;
    return TGM_OK;
}

}  // namespace

extern "C" tgm_status_t tgm_embed_projection(tgm_model_t m, int32_t R, const int32_t *root_pos,
                                             const double *root_ts, const float *mem_new,
                                             const double *new_mem_ts, const int32_t *n_nodes,
                                             int32_t cap, float *h, void *stream)
{
    TprojArgs a;
    TGM_TRY_STATUS(tproj_plan(m, R, root_pos, root_ts, mem_new, new_mem_ts, n_nodes, cap, h, &a));
    if (R > 0)
        TGM_LAUNCH(k_tproj, dim3((unsigned)cdiv((int64_t)R * m->M, 256)), dim3(256), 0,
                   as_stream(stream), a);
    return TGM_OK;
}

void tgm::phi_plan(const tgm_model *m, GatherPlan *plan)
{
    if (!m || !plan || !m->gru_w || m->D_t == 0)
        return;
    plan->omega = m->omega;
    plan->beta = m->beta;
    plan->D_t = m->D_t;
    plan->o_phi = m->phi;
}

tgm_status_t tgm::compute_iteration(tgm_state_t st, tgm_model_t m, tgm_graph_t g, int64_t iter,
                                    const tgm_sample_buffers &sb, const tgm_fetch_buffers &fb,
                                    int32_t cap, int64_t first_event, int32_t b, int32_t nb,
                                    float *mem_new, double *new_mem_ts, int64_t *winner,
                                    float *h, const tgm_sample_buffers *next_sb,
                                    int32_t mit_slot, uint64_t *xwin, uint64_t xtag,
                                    hipStream_t s, bool inplace, bool next_inplace,
                                    hipEvent_t next_ready)
{
    if (st && st->mit)   // the mitigation of this iteration's fetched memories
        TGM_TRY_STATUS(mitigate_launch(st->mit, g, first_event, sb.nodes, sb.n_nodes, cap,
                                       fb.mem, fb.mem_ts, st->M, st->mit_p, st->mit_lambda,
                                       mit_slot, s));
    StageArgs sa;
    int n_items = 0;
    uint64_t tag = 0;
    const bool jodie = m && m->kind == TGM_MODEL_JODIE;
    // JODIE's projection reads the new memory times: the model's buffer
    // stands in when the caller keeps none
    double *nts = jodie && !new_mem_ts ? m->nts : new_mem_ts;
    if (inplace && st && st->mit)
        return TGM_EINVAL;   // the mitigation blends fetched rows
    tgm_status_t rc = update_begin(st, m, g, iter, sb.n_nodes, cap, fb.mem, fb.mem_ts, fb.mail,
                                   fb.mail_ts, fb.ver, first_event, b, sb.root_pos,
                                   sb.root_pos + b, mem_new, nts, s, &sa, &n_items, &tag,
                                   xwin, xtag, true,   // every executor fetch forms phi
                                   inplace ? sb.nodes : nullptr);
    if (rc != TGM_OK)
        return rc;
    if (jodie) {
        // RNN, staging, then the projection with the next fetch's gather
        TprojArgs ta;
        const int32_t R = 3 * b;
        TGM_TRY_STATUS(tproj_plan(m, R, sb.root_pos, sb.root_ts, mem_new, nts, sb.n_nodes, cap,
                                  h, &ta));
        GatherPlan next_plan;
        bool has_next = false;
        if (next_sb) {
            TGM_TRY_STATUS(fetch_plan(st, iter + 1, next_sb->nodes, next_sb->n_nodes, cap,
                                      fb.mem, fb.mem_ts, fb.mail, fb.mail_ts, fb.ver, s,
                                      &next_plan));
            phi_plan(m, &next_plan);
            if (next_inplace)
                next_plan.phi_only();
            has_next = next_plan.cap > 0;
        }
        if (n_items > 0)
            TGM_LAUNCH(k_stage, dim3((unsigned)cdiv(n_items, 4)), dim3(256), 0, s, sa);
        TGM_TRY_STATUS(update_winner(sa.win, sb.n_nodes, cap, first_event, tag, winner, s));
        const int n_tp = (int)cdiv((int64_t)R * m->M, 256);
        if (next_ready)
            TGM_HIP(hipStreamWaitEvent(s, next_ready, 0));
        if (has_next)
            TGM_LAUNCH(k_tproj_gather, dim3((unsigned)(n_tp + kCUs)), dim3(256), 0, s, ta, n_tp,
                       next_plan);
        else if (R > 0)
            TGM_LAUNCH(k_tproj, dim3((unsigned)n_tp), dim3(256), 0, s, ta);
        return TGM_OK;
    }
    ProjArgs pa;
    AttnArgs aa;
    int proj_grid = 0, proj_waves = 0;
    const int32_t R = 3 * b;
    rc = embed_plan(m, g, R, nb, sb.root_pos, sb.root_ts, sb.nbr_pos, sb.eid, sb.nts, sb.cnt,
                    mem_new, sb.n_nodes, cap, h, &pa, &proj_grid, &proj_waves, &aa);
    if (rc != TGM_OK)
        return rc;
    // the fetch of iteration iter + 1, planned after this update's protocol
    // step (so the commit it needs is the one this staging launch makes)
    GatherPlan next_plan;
    const GatherPlan *next = nullptr;
    if (next_sb) {
        rc = fetch_plan(st, iter + 1, next_sb->nodes, next_sb->n_nodes, cap, fb.mem, fb.mem_ts,
                        fb.mail, fb.mail_ts, fb.ver, s, &next_plan);
        if (rc != TGM_OK)
            return rc;
        phi_plan(m, &next_plan);
        if (next_inplace)
            next_plan.phi_only();
        next = &next_plan;
    }
    // staging items ride in blocks after the projection's
    const int n_stage_blocks = (int)cdiv(n_items, proj_waves);
    if ((R > 0 || n_items > 0) && lean_proj(pa))
        TGM_LAUNCH(k_stage_proj<true>, dim3((R > 0 ? proj_grid : 0) + n_stage_blocks),
                   dim3(64 * proj_waves), proj_lds(m), s, sa, pa, R > 0 ? proj_grid : 0);
    else if (R > 0 || n_items > 0)
        TGM_LAUNCH(k_stage_proj<false>, dim3((R > 0 ? proj_grid : 0) + n_stage_blocks),
                   dim3(64 * proj_waves), proj_lds(m), s, sa, pa, R > 0 ? proj_grid : 0);
    TGM_TRY_STATUS(update_winner(sa.win, sb.n_nodes, cap, first_event, tag, winner, s));
    if (next_ready)
        TGM_HIP(hipStreamWaitEvent(s, next_ready, 0));
    if (R > 0)
        return launch_attn(m, aa, next, s);
    return next ? launch_gather(*next, s) : TGM_OK;
}

tgm_status_t tgm::exec_latest_launch(tgm_state_t st, int32_t slot, int32_t b,
                                     const int32_t *src_pos, const int32_t *dst_pos,
                                     const int32_t *n_nodes, hipStream_t s, uint64_t **win,
                                     uint64_t *tag)
{
    if (!st || slot < 0 || slot >= st->xwin_slots || b < 0 || !n_nodes || !win || !tag)
        return TGM_EINVAL;
    if (st->xwin_tag == UINT32_MAX) {   // keys restart from zero in every array
        const int64_t n = (int64_t)st->xwin_slots * st->xwin_cap;
        TGM_LAUNCH(k_fill_u64, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, st->xwin, (int32_t)n);
        st->xwin_tag = 0;
    }
    *tag = (uint64_t)(++st->xwin_tag) << 32;
    *win = st->xwin + (size_t)slot * st->xwin_cap;
    const int n_cand = 2 * b;
    if (n_cand == 0)
        return TGM_OK;
    if (!src_pos || !dst_pos)
        return TGM_EINVAL;
    GruArgs ga{};
    ga.n_nodes = n_nodes;
    ga.n_cand = n_cand;
    ga.src_pos = src_pos;
    ga.dst_pos = dst_pos;
    ga.win = *win;
    ga.tag = *tag;
    TGM_LAUNCH(k_latest, dim3((unsigned)cdiv(n_cand, 256)), dim3(256), 0, s, ga);
    return TGM_OK;
}

// ------------------------------------------------------------------ repack
// After a training step the plain weights have changed: every operand the
// kernels read in a packed layout is rebuilt from them on the device, in the
// layouts tgm_model_create builds on the host (the zero padding past the data
// chunks stays as it was).
namespace {

// Source of element (n, k) of a packed B operand: row n of up to three row
// blocks of `rows` rows each (W[b], leading dimension ldw[b]); with perm_Dt
// >= 0 the column k is read from the slot-row order [phi || efeat] of
// columns of [s || efeat || phi]; with trans the roles of n and k swap.
struct PackSrc {
    const float *W[3];
    int ldw[3];
    int rows;
    int perm_M, perm_De, perm_Dt;
    int trans;
};

__device__ __forceinline__ float pack_src(const PackSrc &p, int n, int k)
{
    int r = n, c = k;
    if (p.trans) {
        r = k;
        c = n;
    }
    const int blk = r / p.rows, rr = r - blk * p.rows;
    if (p.perm_Dt >= 0)
        c = c < p.perm_Dt ? p.perm_M + p.perm_De + c : p.perm_M + c - p.perm_Dt;
    return p.W[blk][(int64_t)rr * p.ldw[blk] + c];
}

// out[((kc NB + nb) 64 + lane) 4 + j] = src(16 nb + lane % 16, 16 kc + 4 (lane / 16) + j),
// zero outside [0, n_out) x [0, K): the layout of pack_b
__global__ __launch_bounds__(256) void k_pack(PackSrc p, int n_out, int K, int KC, int NB,
                                              float *__restrict__ out)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= (int64_t)KC * NB * kWave * 4)
        return;
    const int j = (int)(t & 3), lane = (int)((t >> 2) & 63);
    const int64_t blk = t >> 8;
    const int nb = (int)(blk % NB), kc = (int)(blk / NB);
    const int k = 16 * kc + 4 * (lane >> 4) + j, n = 16 * nb + (lane & 15);
    out[t] = (k < K && n < n_out) ? pack_src(p, n, k) : 0.f;
}

// GRU biases [4][MP]: b_ir + b_hr, b_iz + b_hz, b_in, b_hn (JODIE: 0, 0, b_ih, b_hh)
__global__ void k_pack_gru_bias(int M, int MP, int gates, const float *__restrict__ b_ih,
                                const float *__restrict__ b_hh, float *__restrict__ out)
{
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= M)
        return;
    if (gates == 3) {
        out[k] = b_ih[k] + b_hh[k];
        out[MP + k] = b_ih[M + k] + b_hh[M + k];
        out[2 * MP + k] = b_ih[2 * M + k];
        out[3 * MP + k] = b_hh[2 * M + k];
    } else {
        out[2 * MP + k] = b_ih[k];
        out[3 * MP + k] = b_hh[k];
    }
}

__global__ void k_copy_f32(const float *__restrict__ src, float *__restrict__ dst, int n)
{
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < n)
        dst[k] = src[k];
}

tgm_status_t pack_launch(const PackSrc &p, int n_out, int K, int KC, int NB, void *out,
                         hipStream_t s)
{
    const int64_t n = (int64_t)KC * NB * kWave * 4;
    if (n > 0)
        TGM_LAUNCH(k_pack, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, p, n_out, K, KC, NB,
                   (float *)out);
    return TGM_OK;
}

PackSrc plain_src(const float *W, int ldw, int rows)
{
    PackSrc p{};
    p.W[0] = p.W[1] = p.W[2] = W;
    p.ldw[0] = p.ldw[1] = p.ldw[2] = ldw;
    p.rows = rows > 0 ? rows : 1;
    p.perm_Dt = -1;
    return p;
}

}  // namespace

tgm_status_t tgm::model_repack(tgm_model_t m, const ModelParams &w, hipStream_t s)
{
    if (!m || m->kind != TGM_MODEL_TGN)
        return TGM_EINVAL;
    const int M = m->M, D_e = m->D_e, D_t = m->D_t, D_x = m->D_x, MP = m->MB * 16;
    const int Dq = M + D_t, Dkv = M + D_e + D_t, KF = D_e + D_t;
    // GRU: one packed operand per gate, in gate order
    const int64_t gx = (int64_t)m->KXC * m->MB * kWave * 4, gh = (int64_t)m->KHC * m->MB * kWave * 4;
    for (int gte = 0; gte < 3; ++gte) {
        TGM_TRY_STATUS(pack_launch(plain_src(w.W_ih + (int64_t)gte * M * D_x, D_x, M), M, D_x,
                                   m->KXC, m->MB, (float *)m->gru_bx + gte * gx, s));
        TGM_TRY_STATUS(pack_launch(plain_src(w.W_hh + (int64_t)gte * M * M, M, M), M, M, m->KHC,
                                   m->MB, (float *)m->gru_bh + gte * gh, s));
    }
    TGM_LAUNCH(k_pack_gru_bias, dim3((unsigned)cdiv(M, 128)), dim3(128), 0, s, M, MP, 3, w.b_ih,
               w.b_hh, m->gru_bias);
    // node projections: rows of [W_q^s; W_k^s; W_v^s]
    {
        PackSrc p{};
        p.W[0] = w.W_q;
        p.W[1] = w.W_k;
        p.W[2] = w.W_v;
        p.ldw[0] = Dq;
        p.ldw[1] = p.ldw[2] = Dkv;
        p.rows = M;
        p.perm_Dt = -1;
        TGM_TRY_STATUS(pack_launch(p, 3 * M, M, m->PC, m->PNB, m->proj_b, s));
    }
    // per-slot part of [K | V] in the slot-row column order [phi || efeat]
    PackSrc kv{};
    kv.W[0] = w.W_k;
    kv.W[1] = kv.W[2] = w.W_v;
    kv.ldw[0] = kv.ldw[1] = kv.ldw[2] = Dkv;
    kv.rows = M;
    kv.perm_M = M;
    kv.perm_De = D_e;
    kv.perm_Dt = D_t;
    if (KF > 0)
        TGM_TRY_STATUS(pack_launch(kv, 2 * M, KF, m->KFC, m->KVNB, m->kv_b, s));
    if ((m->fold || m->agg) && KF > 0) {
        PackSrc v = kv;
        v.W[0] = w.W_v;
        TGM_TRY_STATUS(pack_launch(v, M, KF, m->KFC, m->VNB, m->v_b, s));
        PackSrc u = kv;   // W_k^t [KF x M]: element (kf, d) = W_k[d][perm(kf)]
        u.trans = 1;
        TGM_TRY_STATUS(pack_launch(u, KF, M, m->DC, m->KFC, m->uk_a, s));
    }
    TGM_TRY_STATUS(pack_launch(plain_src(w.W_o, 2 * M, M), M, 2 * M, m->OC, m->ONB, m->out_b, s));
    // biases of the node projection: c_q = W_q^t phi(0) + b_q, then b_k, b_v
    hipLaunchKernelGGL(k_fold_q_bias, dim3((unsigned)cdiv(M, 64)), dim3(64), 0, s, M, D_t, w.W_q,
                       w.b_q, m->beta, m->pbias);
    TGM_LAUNCHED();
    TGM_LAUNCH(k_copy_f32, dim3((unsigned)cdiv(M, 128)), dim3(128), 0, s, w.b_k, m->pbias + M, M);
    TGM_LAUNCH(k_copy_f32, dim3((unsigned)cdiv(M, 128)), dim3(128), 0, s, w.b_v,
               m->pbias + 2 * M, M);
    TGM_LAUNCH(k_copy_f32, dim3((unsigned)cdiv(M, 128)), dim3(128), 0, s, w.b_o, m->b_o, M);
    return TGM_OK;
}
