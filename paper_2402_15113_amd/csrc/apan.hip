// APAN, the third model family of the paper's experiments (Sec. 5; App. B:
// an RNN memory updater with an attention mechanism and asynchronous
// propagation).  Per node a mailbox of the K latest mails (a ring of K rows
// and times, its head and count); the mails an event generates for its two
// endpoints go to the endpoints and to their sampled neighbours; a node's
// memory update attends over its mailbox and feeds the aggregate to a GRU;
// the embedding is the updated memory.  Mail deliveries and memory writes of
// iteration i form its write set, committed before the fetch of iteration
// i + s + 1 (Eq. 2), as for the other families.
//
// One call per iteration (tgm_apan_step): commit the due write sets, gather
// the node set's memories and mailboxes, the attention and the GRU, the
// embeddings, and the staging of the iteration's write set.  The deliveries
// of an iteration are radix-sorted by (node, delivery index); the index is
// monotone in (t, e, role, slot), so each node's segment is in mail order and
// its last K entries are the ones its mailbox keeps.
#include <hip/hip_runtime.h>

#include <hipcub/hipcub.hpp>

#include <algorithm>
#include <cmath>
#include <vector>

#include "common.h"

using namespace tgm;

namespace {

constexpr int kApanMaxK = 16;

struct ApanRows {   // the node set's rows and the staging work space
    const int32_t *nodes, *n_nodes;
    int cap, M, D_m, D_t, K;
    const float *mem, *mb;          // tables [N x M], [N x K x D_m]
    const double *mem_ts, *mb_ts;   // [N], [N x K]
    const int32_t *ver, *mb_head, *mb_cnt;
    float *f_mem, *f_mb;            // fetched [cap x M], [cap x K x D_m] (oldest first)
    double *f_mem_ts, *f_mb_ts;     // [cap], [cap x K]
    int32_t *f_ver, *f_cnt;         // [cap]
};

// Gather of the node set, one wavefront per node: memory, its time and
// version, and the mailbox's mails oldest first.
__global__ __launch_bounds__(256) void k_apan_gather(ApanRows a)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    const int n = min(*a.n_nodes, a.cap);
    if (p >= n)
        return;
    const int v = a.nodes[p], M = a.M, D_m = a.D_m, K = a.K;
    wave_copy_row(a.f_mem + (int64_t)p * M, a.mem + (int64_t)v * M, M, lane);
    const int cnt = a.mb_cnt[v], head = a.mb_head[v];
    for (int j = 0; j < cnt; ++j) {
        const int slot = ((head - cnt + j) % K + K) % K;
        wave_copy_row(a.f_mb + ((int64_t)p * K + j) * D_m, a.mb + ((int64_t)v * K + slot) * D_m,
                      D_m, lane);
        if (lane == 0)
            a.f_mb_ts[(int64_t)p * K + j] = a.mb_ts[(int64_t)v * K + slot];
    }
    if (lane == 0) {
        a.f_mem_ts[p] = a.mem_ts[v];
        a.f_ver[p] = a.ver[v];
        a.f_cnt[p] = cnt;
    }
}

// Xq[p] = [f_mem[p] || phi(0)], one wavefront per node (rows past n zero)
__global__ __launch_bounds__(256) void k_apan_query_rows(const int32_t *__restrict__ n_nodes,
                                                         int cap, int M, int D_t,
                                                         const float *__restrict__ f_mem,
                                                         const double *__restrict__ omega,
                                                         const double *__restrict__ beta,
                                                         float *__restrict__ Xq)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (p >= cap)
        return;
    float *x = Xq + (int64_t)p * (M + D_t);
    if (p >= min(*n_nodes, cap)) {
        for (int k = lane; k < M + D_t; k += kWave)
            x[k] = 0.f;
        return;
    }
    for (int k = lane; k < M; k += kWave)
        x[k] = f_mem[(int64_t)p * M + k];
    for (int d = lane; d < D_t; d += kWave)
        x[M + d] = time_enc(omega[d], beta[d], 0.0);
}

// The mailbox attention, one wavefront per node with mail: u = W_k^t q has
// been formed for the node (u [cap x (D_m + D_t)], qb = q . b_k), so the
// score of mail j is (u . [mail_j || phi(t_newest - t_j)] + qb) / sqrt(M).
// Writes the GRU input row X[p] = [sum_j alpha_j mail_j || phi(t_newest -
// mem_ts)] and t_newest; nodes without mail get a zero row.
struct AttnArgs2 {
    const int32_t *n_nodes;
    int cap, M, D_m, D_t, K;
    float scale;
    const float *u, *qb, *f_mb;
    const double *f_mb_ts, *f_mem_ts, *omega, *beta;
    const int32_t *f_cnt;
    float *X;          // [cap x (D_m + D_t)]
    double *t_new;     // [cap]
};

__global__ __launch_bounds__(256) void k_apan_attn(AttnArgs2 a)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (p >= a.cap)
        return;
    const int D_m = a.D_m, D_t = a.D_t, D_x = D_m + D_t, K = a.K;
    float *x = a.X + (int64_t)p * D_x;
    const int cnt = p < min(*a.n_nodes, a.cap) ? a.f_cnt[p] : 0;
    if (cnt == 0) {
        for (int k = lane; k < D_x; k += kWave)
            x[k] = 0.f;
        if (lane == 0)
            a.t_new[p] = p < min(*a.n_nodes, a.cap) ? a.f_mem_ts[p] : 0.0;
        return;
    }
    const float *u = a.u + (int64_t)p * D_x;
    const float *rows = a.f_mb + (int64_t)p * K * D_m;
    const double *ts = a.f_mb_ts + (int64_t)p * K;
    const double tref = ts[cnt - 1];
    // every mail's partial score at once: per element of u, the loads of all
    // the node's mails are in flight together (each lane sums its elements
    // in the same order as a mail-by-mail loop would)
    float part[kApanMaxK];
#pragma unroll
    for (int j = 0; j < kApanMaxK; ++j)
        part[j] = 0.f;
    for (int k = lane; k < D_m; k += kWave) {
        const float uk = u[k];
#pragma unroll
        for (int j = 0; j < kApanMaxK; ++j)
            if (j < cnt)
                part[j] += uk * rows[(int64_t)j * D_m + k];
    }
    for (int d = lane; d < D_t; d += kWave) {
        const float ud = u[D_m + d];
        const double om = a.omega[d], be = a.beta[d];
#pragma unroll
        for (int j = 0; j < kApanMaxK; ++j)
            if (j < cnt)
                part[j] += ud * time_enc(om, be, tref - ts[j]);
    }
    const float qb = a.qb[p];
    float mine = -INFINITY;   // lane j < cnt: the score of mail j
#pragma unroll
    for (int j = 0; j < kApanMaxK; ++j)
        if (j < cnt) {
            const float sc = (wave_sum(part[j]) + qb) * a.scale;
            if (lane == j)
                mine = sc;
        }
    float mx = mine;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    const float ex = lane < cnt ? expf(mine - mx) : 0.f;
    const float al = ex / wave_sum(ex);
    float alv[kApanMaxK];   // every lane holds every weight (shuffles in uniform flow)
#pragma unroll
    for (int j = 0; j < kApanMaxK; ++j)
        alv[j] = __shfl(al, j < cnt ? j : 0, kWave);
    for (int k = lane; k < D_m; k += kWave) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < kApanMaxK; ++j)
            if (j < cnt)
                acc += alv[j] * rows[(int64_t)j * D_m + k];
        x[k] = acc;
    }
    for (int d = lane; d < D_t; d += kWave)
        x[D_m + d] = time_enc(a.omega[d], a.beta[d], tref - a.f_mem_ts[p]);
    if (lane == 0)
        a.t_new[p] = tref;
}

// q . b_k per node (the common part of every score), one wavefront per node
__global__ __launch_bounds__(256) void k_apan_qb(const int32_t *__restrict__ n_nodes, int cap,
                                                 int M, const float *__restrict__ Q,
                                                 const float *__restrict__ b_k,
                                                 float *__restrict__ qb)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (p >= min(*n_nodes, cap))
        return;
    float acc = 0.f;
    for (int k = lane; k < M; k += kWave)
        acc += Q[(int64_t)p * M + k] * b_k[k];
    acc = wave_sum(acc);
    if (lane == 0)
        qb[p] = acc;
}

// The GRU cell from the gate pre-activations Gx = X W_ih^t + b_ih and
// Gh = mem W_hh^t + b_hh, one thread per (node, unit); nodes without mail
// keep their memory.
__global__ __launch_bounds__(256) void k_apan_gru(const int32_t *__restrict__ n_nodes, int cap,
                                                  int M, const int32_t *__restrict__ f_cnt,
                                                  const float *__restrict__ Gx,
                                                  const float *__restrict__ Gh,
                                                  const float *__restrict__ f_mem,
                                                  float *__restrict__ s_new)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= (int64_t)cap * M)
        return;
    const int p = (int)(t / M), j = (int)(t % M);
    if (p >= min(*n_nodes, cap))
        return;
    const float h = f_mem[(int64_t)p * M + j];
    if (f_cnt[p] == 0) {
        s_new[(int64_t)p * M + j] = h;
        return;
    }
    const int64_t o = (int64_t)p * 3 * M;
    const float r = 1.f / (1.f + expf(-(Gx[o + j] + Gh[o + j])));
    const float z = 1.f / (1.f + expf(-(Gx[o + M + j] + Gh[o + M + j])));
    const float n = tanhf(Gx[o + 2 * M + j] + r * Gh[o + 2 * M + j]);
    s_new[(int64_t)p * M + j] = (1.f - z) * n + z * h;
}

// h[r] = s_new[root_pos[r]] (the embedding is the updated memory)
__global__ __launch_bounds__(256) void k_apan_embed(int R, int M,
                                                    const int32_t *__restrict__ root_pos,
                                                    const float *__restrict__ s_new,
                                                    float *__restrict__ h)
{
    const int r = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    if (r >= R)
        return;
    wave_copy_row(h + (int64_t)r * M, s_new + (int64_t)root_pos[r] * M, M, threadIdx.x & 63);
}

// ------------------------------------------------------------- staging
// Delivery d = ((k 2 + role)(nb + 1) + slot) of batch event k: the mail of
// endpoint v (role 0: src, 1: dst) to v (slot 0) or to its neighbour in
// sampled slot (slot - 1) of root role b + k.  Key (node << 32) | d; empty
// or unused deliveries get the largest key.
__global__ __launch_bounds__(256) void k_apan_keys(int32_t b, int nb, int propagate,
                                                   const int32_t *__restrict__ root,
                                                   const int32_t *__restrict__ nbr,
                                                   const int32_t *__restrict__ cnt,
                                                   uint64_t *__restrict__ keys)
{
    const int64_t d = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int per = nb + 1;
    if (d >= (int64_t)2 * b * per)
        return;
    const int slot = (int)(d % per), kr = (int)(d / per), role = kr & 1, k = kr >> 1;
    const int r = role * b + k;
    int32_t w = -1;
    if (slot == 0)
        w = root[r];
    else if (propagate && slot - 1 < cnt[r])
        w = nbr[(int64_t)r * nb + slot - 1];
    keys[d] = w < 0 ? ~(uint64_t)0 : ((uint64_t)(uint32_t)w << 32) | (uint64_t)d;
}

// Segment bounds by node id over the sorted keys
__global__ __launch_bounds__(256) void k_apan_bounds(int64_t n, const uint64_t *__restrict__ keys,
                                                     int32_t N, int32_t *__restrict__ seg,
                                                     int32_t *__restrict__ seg_end)
{
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= n || keys[i] == ~(uint64_t)0)
        return;
    const int32_t w = (int32_t)(keys[i] >> 32);
    if (w < 0 || w >= N)
        return;
    if (i == 0 || (keys[i - 1] >> 32) != (keys[i] >> 32))
        seg[w] = (int32_t)i;
    if (i == n - 1 || (keys[i + 1] >> 32) != (keys[i] >> 32))
        seg_end[w] = (int32_t)(i + 1);
}

struct StageArgs2 {
    int32_t b, nb, M, D_e, D_m, K, N;
    int64_t first;
    const uint64_t *keys;       // sorted
    const int32_t *seg, *seg_end;
    const int32_t *root_pos;    // [3b]
    const float *s_new, *efeat;
    const double *t;
    // the slot's delivery rows, indexed by sorted position
    int32_t *d_node, *d_rank, *d_keep;   // d_keep: count kept for the node, 0 = dropped
    float *d_mail;
    double *d_t;
};

// One wavefront per sorted delivery: rows that the node's mailbox keeps (the
// last K of its segment) are written with their rank among the kept ones.
__global__ __launch_bounds__(256) void k_apan_stage_mail(StageArgs2 a, int64_t n)
{
    const int64_t i = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (i >= n)
        return;
    const uint64_t key = a.keys[i];
    if (key == ~(uint64_t)0) {
        if (lane == 0)
            a.d_keep[i] = 0;
        return;
    }
    const int32_t w = (int32_t)(key >> 32);
    const int64_t lo = a.seg[w], hi = a.seg_end[w];
    const int64_t keep_from = max(lo, hi - a.K);
    if (i < keep_from) {
        if (lane == 0)
            a.d_keep[i] = 0;
        return;
    }
    const int64_t d = (int64_t)(key & 0xffffffffu);
    const int per = a.nb + 1;
    const int kr = (int)(d / per), role = kr & 1, k = kr >> 1;
    const int pv = a.root_pos[role * a.b + k], po = a.root_pos[(1 - role) * a.b + k];
    const int M = a.M, D_e = a.D_e;
    float *row = a.d_mail + i * a.D_m;
    wave_copy_row(row, a.s_new + (int64_t)pv * M, M, lane);
    wave_copy_row(row + M, a.s_new + (int64_t)po * M, M, lane);
    if (D_e > 0)
        wave_copy_row(row + 2 * M, a.efeat + (a.first + k) * D_e, D_e, lane);
    if (lane == 0) {
        a.d_node[i] = w;
        a.d_rank[i] = (int32_t)(i - keep_from);
        a.d_keep[i] = (int32_t)(hi - keep_from);
        a.d_t[i] = a.t[a.first + k];
    }
}

// Memory rows of the batch's endpoints, by node-set position: flag[p] = 1 and
// the new memory for every position that is a source or destination.
__global__ __launch_bounds__(256) void k_apan_stage_mem(int32_t b, int M,
                                                        const int32_t *__restrict__ root_pos,
                                                        const int32_t *__restrict__ nodes,
                                                        const float *__restrict__ s_new,
                                                        const double *__restrict__ new_ts,
                                                        int32_t *__restrict__ flag,
                                                        int32_t *__restrict__ node,
                                                        float *__restrict__ r_mem,
                                                        double *__restrict__ r_ts)
{
    // one wavefront per endpoint occurrence; all occurrences of a node write
    // the same values (plain stores)
    const int e = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (e >= 2 * b)
        return;
    const int p = root_pos[e];
    wave_copy_row(r_mem + (int64_t)p * M, s_new + (int64_t)p * M, M, lane);
    if (lane == 0) {
        flag[p] = 1;
        node[p] = nodes[p];
        r_ts[p] = new_ts[p];
    }
}

__global__ __launch_bounds__(256) void k_apan_clear_flags(int32_t *__restrict__ flag, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        flag[i] = 0;
}

// ------------------------------------------------------------- commit
__global__ __launch_bounds__(256) void k_apan_commit_mem(int cap, int M, int64_t iter,
                                                         const int32_t *__restrict__ flag,
                                                         const int32_t *__restrict__ node,
                                                         const float *__restrict__ r_mem,
                                                         const double *__restrict__ r_ts,
                                                         float *__restrict__ mem,
                                                         double *__restrict__ mem_ts,
                                                         int32_t *__restrict__ ver)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (p >= cap || !flag[p])
        return;
    const int v = node[p];
    wave_copy_row(mem + (int64_t)v * M, r_mem + (int64_t)p * M, M, lane);
    if (lane == 0) {
        mem_ts[v] = r_ts[p];
        ver[v] = (int32_t)iter;
    }
}

// kept mails into the ring at head + rank (heads are updated after)
__global__ __launch_bounds__(256) void k_apan_commit_mail(int64_t n, int D_m, int K,
                                                          const int32_t *__restrict__ d_node,
                                                          const int32_t *__restrict__ d_rank,
                                                          const int32_t *__restrict__ d_keep,
                                                          const float *__restrict__ d_mail,
                                                          const double *__restrict__ d_t,
                                                          const int32_t *__restrict__ head,
                                                          float *__restrict__ mb,
                                                          double *__restrict__ mb_ts)
{
    const int64_t i = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (i >= n || d_keep[i] == 0)
        return;
    const int v = d_node[i];
    const int slot = (head[v] + d_rank[i]) % K;
    wave_copy_row(mb + ((int64_t)v * K + slot) * D_m, d_mail + i * D_m, D_m, lane);
    if (lane == 0)
        mb_ts[(int64_t)v * K + slot] = d_t[i];
}

__global__ __launch_bounds__(256) void k_apan_commit_heads(int64_t n, int K,
                                                           const int32_t *__restrict__ d_node,
                                                           const int32_t *__restrict__ d_rank,
                                                           const int32_t *__restrict__ d_keep,
                                                           int32_t *__restrict__ head,
                                                           int32_t *__restrict__ cnt)
{
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= n || d_keep[i] == 0 || d_rank[i] != d_keep[i] - 1)
        return;
    const int v = d_node[i], k = d_keep[i];
    head[v] = (head[v] + k) % K;
    cnt[v] = min(K, cnt[v] + k);
}

// The committed mailboxes oldest first, one wavefront per node; rows past the
// count are zero.
__global__ __launch_bounds__(256) void k_apan_read_mb(int32_t N, int K, int D_m,
                                                      const float *__restrict__ mb,
                                                      const double *__restrict__ mb_ts,
                                                      const int32_t *__restrict__ head,
                                                      const int32_t *__restrict__ cnt,
                                                      float *__restrict__ out,
                                                      double *__restrict__ out_ts)
{
    const int v = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (v >= N)
        return;
    const int c = cnt[v], hd = head[v];
    for (int j = 0; j < K; ++j) {
        float *dst = out + ((int64_t)v * K + j) * D_m;
        if (j < c) {
            const int slot = ((hd - c + j) % K + K) % K;
            wave_copy_row(dst, mb + ((int64_t)v * K + slot) * D_m, D_m, lane);
            if (lane == 0)
                out_ts[(int64_t)v * K + j] = mb_ts[(int64_t)v * K + slot];
        } else {
            for (int k = lane; k < D_m; k += kWave)
                dst[k] = 0.f;
            if (lane == 0)
                out_ts[(int64_t)v * K + j] = 0.0;
        }
    }
}

// Mailboxes given oldest first with their counts into the rings: mail j at
// slot j, head = count mod K; counts are clamped to [0, K].
__global__ __launch_bounds__(256) void k_apan_load_mb(int32_t N, int K, int D_m,
                                                      const float *__restrict__ in,
                                                      const double *__restrict__ in_ts,
                                                      const int32_t *__restrict__ in_cnt,
                                                      float *__restrict__ mb,
                                                      double *__restrict__ mb_ts,
                                                      int32_t *__restrict__ head,
                                                      int32_t *__restrict__ cnt)
{
    const int v = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (v >= N)
        return;
    const int c = min(max(in_cnt[v], 0), K);
    for (int j = 0; j < c; ++j) {
        wave_copy_row(mb + ((int64_t)v * K + j) * D_m, in + ((int64_t)v * K + j) * D_m, D_m,
                      lane);
        if (lane == 0)
            mb_ts[(int64_t)v * K + j] = in_ts[(int64_t)v * K + j];
    }
    if (lane == 0) {
        head[v] = c % K;
        cnt[v] = c;
    }
}

__global__ void k_apan_init(int32_t N, int M, int K, int D_m, float *__restrict__ mem,
                            double *__restrict__ mem_ts, int32_t *__restrict__ ver,
                            float *__restrict__ mb, double *__restrict__ mb_ts,
                            int32_t *__restrict__ head, int32_t *__restrict__ cnt)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (int64_t k = t0; k < (int64_t)N * M; k += stride)
        mem[k] = 0.f;
    for (int64_t k = t0; k < (int64_t)N * K * D_m; k += stride)
        mb[k] = 0.f;
    for (int64_t k = t0; k < (int64_t)N * K; k += stride)
        mb_ts[k] = 0.0;
    for (int64_t k = t0; k < N; k += stride) {
        mem_ts[k] = 0.0;
        ver[k] = -1;
        head[k] = 0;
        cnt[k] = 0;
    }
}

}  // namespace

struct tgm_apan {
    int32_t N = 0, M = 0, D_e = 0, D_t = 0, D_m = 0, D_x = 0, nb = 0, K = 0, s = 0;
    int32_t max_batch = 0, max_nodes = 0, propagate = 1;
    // weights (plain, device)
    float *W_ih = nullptr, *W_hh = nullptr, *b_ih = nullptr, *b_hh = nullptr;
    float *W_q = nullptr, *b_q = nullptr, *W_k = nullptr, *b_k = nullptr;
    double *omega = nullptr, *beta = nullptr;
    // committed tables
    float *mem = nullptr, *mb = nullptr;
    double *mem_ts = nullptr, *mb_ts = nullptr;
    int32_t *ver = nullptr, *head = nullptr, *cnt = nullptr;
    // fetched rows of the last step and the updater's work space
    float *f_mem = nullptr, *f_mb = nullptr, *Xq = nullptr, *Q = nullptr, *U = nullptr,
          *qb = nullptr, *X = nullptr, *Gx = nullptr, *Gh = nullptr;
    double *f_mem_ts = nullptr, *f_mb_ts = nullptr, *t_new = nullptr;
    int32_t *f_ver = nullptr, *f_cnt = nullptr;
    // staging: keys, sort, segments
    uint64_t *keys = nullptr, *keys_sorted = nullptr;
    int32_t *seg = nullptr, *seg_end = nullptr;
    void *sort_tmp = nullptr;
    size_t sort_bytes = 0;
    // ring of s + 1 write sets: memory rows by node-set position, mail rows
    // by sorted delivery position
    struct Slot {
        int64_t iter = -1;
        int64_t n_del = 0;
        bool staged = false;
    };
    std::vector<Slot> ring;
    int32_t *r_flag = nullptr, *r_node = nullptr;
    float *r_mem = nullptr;
    double *r_ts = nullptr;
    int32_t *d_node = nullptr, *d_rank = nullptr, *d_keep = nullptr;
    float *d_mail = nullptr;
    double *d_t = nullptr;
    int64_t committed_through = -1, staged_through = -1;
    int64_t max_del() const { return 2 * (int64_t)max_batch * (nb + 1); }
};

namespace {

tgm_status_t apan_commit_through(tgm_apan *a, int64_t target, hipStream_t s)
{
    const int slots = a->s + 1;
    for (int64_t j = a->committed_through + 1; j <= target; ++j) {
        tgm_apan::Slot &sl = a->ring[j % slots];
        if (!sl.staged || sl.iter != j)
            return TGM_EORDER;
        const int64_t r = j % slots;
        const int64_t cap = a->max_nodes, md = a->max_del();
        TGM_LAUNCH(k_apan_commit_mem, dim3((unsigned)cdiv(cap * kWave, 256)), dim3(256), 0, s,
                   (int)cap, a->M, j, a->r_flag + r * cap, a->r_node + r * cap,
                   a->r_mem + r * cap * a->M, a->r_ts + r * cap, a->mem, a->mem_ts, a->ver);
        if (sl.n_del > 0) {
            TGM_LAUNCH(k_apan_commit_mail, dim3((unsigned)cdiv(sl.n_del * kWave, 256)),
                       dim3(256), 0, s, sl.n_del, a->D_m, a->K, a->d_node + r * md,
                       a->d_rank + r * md, a->d_keep + r * md, a->d_mail + r * md * a->D_m,
                       a->d_t + r * md, a->head, a->mb, a->mb_ts);
            TGM_LAUNCH(k_apan_commit_heads, dim3((unsigned)cdiv(sl.n_del, 256)), dim3(256), 0,
                       s, sl.n_del, a->K, a->d_node + r * md, a->d_rank + r * md,
                       a->d_keep + r * md, a->head, a->cnt);
        }
        sl.staged = false;
        a->committed_through = j;
    }
    return TGM_OK;
}

}  // namespace

// ======================================================================== API

extern "C" tgm_status_t tgm_apan_destroy(tgm_apan_t a)
{
    if (!a)
        return TGM_EINVAL;
    void *bufs[] = {a->W_ih, a->W_hh, a->b_ih, a->b_hh, a->W_q, a->b_q, a->W_k, a->b_k,
                    a->omega, a->beta, a->mem, a->mb, a->mem_ts, a->mb_ts, a->ver, a->head,
                    a->cnt, a->f_mem, a->f_mb, a->Xq, a->Q, a->U, a->qb, a->X, a->Gx, a->Gh,
                    a->f_mem_ts, a->f_mb_ts, a->t_new, a->f_ver, a->f_cnt, a->keys,
                    a->keys_sorted, a->seg, a->seg_end, a->sort_tmp, a->r_flag, a->r_node,
                    a->r_mem, a->r_ts, a->d_node, a->d_rank, a->d_keep, a->d_mail, a->d_t};
    for (void *b : bufs)
        (void)hipFree(b);
    delete a;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_apan_create(const tgm_apan_desc *d, const tgm_weights *w,
                                        void *stream, tgm_apan_t *out)
{
    if (!out)
        return TGM_EINVAL;
    *out = nullptr;
    if (!d || !w || d->N <= 0 || d->M <= 0 || d->M > 128 || d->D_e < 0 || d->D_e > 256 ||
        d->D_t < 0 || d->nb < 1 || d->nb > 64 || d->K_mb < 1 || d->K_mb > kApanMaxK ||
        d->s < 0 || d->max_batch <= 0 || d->max_nodes <= 0)
        return TGM_EINVAL;
    if (!w->W_ih || !w->W_hh || !w->b_ih || !w->b_hh || !w->W_q || !w->b_q || !w->W_k ||
        !w->b_k || (d->D_t > 0 && (!w->omega || !w->beta)))
        return TGM_EINVAL;
    tgm_apan *a = new tgm_apan();
    a->N = d->N;
    a->M = d->M;
    a->D_e = d->D_e;
    a->D_t = d->D_t;
    a->D_m = 2 * d->M + d->D_e;
    a->D_x = a->D_m + d->D_t;
    a->nb = d->nb;
    a->K = d->K_mb;
    a->s = d->s;
    a->max_batch = d->max_batch;
    a->max_nodes = d->max_nodes;
    a->propagate = d->propagate != 0;
    a->ring.resize(d->s + 1);
    const int64_t N = a->N, M = a->M, K = a->K, D_m = a->D_m, D_x = a->D_x, D_t = a->D_t;
    const int64_t C = a->max_nodes, MD = a->max_del(), slots = d->s + 1;
    tgm_status_t st = TGM_OK;
    auto alloc = [&](auto **ptr, int64_t count) {
        if (st == TGM_OK &&
            dev_malloc(ptr, sizeof(**ptr) * (size_t)std::max<int64_t>(count, 1)) != hipSuccess)
            st = TGM_ENOMEM;
    };
    alloc(&a->W_ih, 3 * M * D_x);
    alloc(&a->W_hh, 3 * M * M);
    alloc(&a->b_ih, 3 * M);
    alloc(&a->b_hh, 3 * M);
    alloc(&a->W_q, M * (M + D_t));
    alloc(&a->b_q, M);
    alloc(&a->W_k, M * D_x);
    alloc(&a->b_k, M);
    alloc(&a->omega, D_t);
    alloc(&a->beta, D_t);
    alloc(&a->mem, N * M);
    alloc(&a->mb, N * K * D_m);
    alloc(&a->mem_ts, N);
    alloc(&a->mb_ts, N * K);
    alloc(&a->ver, N);
    alloc(&a->head, N);
    alloc(&a->cnt, N);
    alloc(&a->f_mem, C * M);
    alloc(&a->f_mb, C * K * D_m);
    alloc(&a->Xq, C * (M + D_t));
    alloc(&a->Q, C * M);
    alloc(&a->U, C * D_x);
    alloc(&a->qb, C);
    alloc(&a->X, C * D_x);
    alloc(&a->Gx, C * 3 * M);
    alloc(&a->Gh, C * 3 * M);
    alloc(&a->f_mem_ts, C);
    alloc(&a->f_mb_ts, C * K);
    alloc(&a->t_new, C);
    alloc(&a->f_ver, C);
    alloc(&a->f_cnt, C);
    alloc(&a->keys, MD);
    alloc(&a->keys_sorted, MD);
    alloc(&a->seg, N);
    alloc(&a->seg_end, N);
    alloc(&a->r_flag, slots * C);
    alloc(&a->r_node, slots * C);
    alloc(&a->r_mem, slots * C * M);
    alloc(&a->r_ts, slots * C);
    alloc(&a->d_node, slots * MD);
    alloc(&a->d_rank, slots * MD);
    alloc(&a->d_keep, slots * MD);
    alloc(&a->d_mail, slots * MD * D_m);
    alloc(&a->d_t, slots * MD);
    if (st == TGM_OK) {
        size_t bytes = 0;
        if (hipcub::DeviceRadixSort::SortKeys(nullptr, bytes, a->keys, a->keys_sorted, (int)MD, 0,
                                              64) != hipSuccess)
            st = TGM_EDEVICE;
        a->sort_bytes = bytes;
        alloc((char **)&a->sort_tmp, (int64_t)bytes);
    }
    hipStream_t s = as_stream(stream);
    if (st == TGM_OK) {
        const struct {
            void *dst;
            const void *src;
            size_t bytes;
        } up[] = {{a->W_ih, w->W_ih, 4 * (size_t)(3 * M * D_x)}, {a->W_hh, w->W_hh, 4 * (size_t)(3 * M * M)},
                  {a->b_ih, w->b_ih, 4 * (size_t)(3 * M)}, {a->b_hh, w->b_hh, 4 * (size_t)(3 * M)},
                  {a->W_q, w->W_q, 4 * (size_t)(M * (M + D_t))}, {a->b_q, w->b_q, 4 * (size_t)M},
                  {a->W_k, w->W_k, 4 * (size_t)(M * D_x)}, {a->b_k, w->b_k, 4 * (size_t)M},
                  {a->omega, w->omega, 8 * (size_t)D_t}, {a->beta, w->beta, 8 * (size_t)D_t}};
        for (const auto &u : up)
            if (st == TGM_OK && u.bytes > 0)
                st = upload(u.dst, u.src, u.bytes);
    }
    if (st == TGM_OK) {
        hipLaunchKernelGGL(k_apan_init, dim3(1024), dim3(256), 0, s, a->N, a->M, a->K, a->D_m,
                           a->mem, a->mem_ts, a->ver, a->mb, a->mb_ts, a->head, a->cnt);
        hipLaunchKernelGGL(k_apan_clear_flags, dim3((unsigned)cdiv(slots * C, 256)), dim3(256), 0,
                           s, a->r_flag, (int)(slots * C));
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
            st = TGM_EDEVICE;
    }
    if (st != TGM_OK) {
        tgm_apan_destroy(a);
        return st;
    }
    *out = a;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_apan_step(tgm_apan_t a, tgm_graph_t g, int64_t iter,
                                      const tgm_sample_buffers *sb, int32_t cap, float *mem_new,
                                      double *new_mem_ts, float *h, void *stream)
{
    if (!a || !g || !sb || !mem_new || !h || cap < 0)
        return TGM_EINVAL;
    if (!sb->root || !sb->root_pos || !sb->nbr || !sb->cnt || !sb->nodes || !sb->n_nodes)
        return TGM_EINVAL;
    if (g->N != a->N || g->D_e != a->D_e || (a->D_e > 0 && !g->efeat))
        return TGM_EINVAL;
    if (cap > a->max_nodes)
        return TGM_ESIZE;
    if (iter != a->staged_through + 1)
        return TGM_EORDER;
    const int64_t lo = iter * (int64_t)a->max_batch;
    if (lo >= g->E || iter < 0)
        return TGM_ERANGE;
    const int32_t b = (int32_t)std::min<int64_t>(a->max_batch, g->E - lo);
    const int M = a->M, D_m = a->D_m, D_t = a->D_t, D_x = a->D_x, K = a->K, nb = a->nb;
    const int R = 3 * b;
    hipStream_t s = as_stream(stream);
    // the write sets a fetch at iter sees: <= iter - 1 - s (Eq. 2)
    TGM_TRY_STATUS(apan_commit_through(a, iter - 1 - a->s, s));
    ApanRows ar{sb->nodes, sb->n_nodes, cap, M, D_m, D_t, K, a->mem, a->mb, a->mem_ts,
                a->mb_ts, a->ver, a->head, a->cnt, a->f_mem, a->f_mb, a->f_mem_ts,
                a->f_mb_ts, a->f_ver, a->f_cnt};
    if (cap > 0) {
        TGM_LAUNCH(k_apan_gather, dim3((unsigned)cdiv((int64_t)cap * kWave, 256)), dim3(256), 0,
                   s, ar);
        // the mailbox attention: q, u = q W_k, q . b_k, then scores and the
        // aggregate per node
        TGM_LAUNCH(k_apan_query_rows, dim3((unsigned)cdiv((int64_t)cap * kWave, 256)),
                   dim3(256), 0, s, sb->n_nodes, cap, M, D_t, a->f_mem, a->omega, a->beta,
                   a->Xq);
        TGM_TRY_STATUS(gemm_f32(false, true, cap, M, M + D_t, a->Xq, M + D_t, a->W_q, M + D_t,
                                a->Q, M, a->b_q, false, s, sb->n_nodes));
        TGM_TRY_STATUS(gemm_f32(false, false, cap, D_x, M, a->Q, M, a->W_k, D_x, a->U, D_x,
                                nullptr, false, s, sb->n_nodes));
        TGM_LAUNCH(k_apan_qb, dim3((unsigned)cdiv((int64_t)cap * kWave, 256)), dim3(256), 0, s,
                   sb->n_nodes, cap, M, a->Q, a->b_k, a->qb);
        AttnArgs2 aa{sb->n_nodes, cap, M, D_m, D_t, K, 1.f / sqrtf((float)M), a->U, a->qb,
                     a->f_mb, a->f_mb_ts, a->f_mem_ts, a->omega, a->beta, a->f_cnt, a->X,
                     a->t_new};
        TGM_LAUNCH(k_apan_attn, dim3((unsigned)cdiv((int64_t)cap * kWave, 256)), dim3(256), 0, s,
                   aa);
        // the GRU on [aggregate || phi(t_newest - mem_ts)]
        TGM_TRY_STATUS(gemm_f32(false, true, cap, 3 * M, D_x, a->X, D_x, a->W_ih, D_x, a->Gx,
                                3 * M, a->b_ih, false, s, sb->n_nodes));
        TGM_TRY_STATUS(gemm_f32(false, true, cap, 3 * M, M, a->f_mem, M, a->W_hh, M, a->Gh,
                                3 * M, a->b_hh, false, s, sb->n_nodes));
        TGM_LAUNCH(k_apan_gru, dim3((unsigned)cdiv((int64_t)cap * M, 256)), dim3(256), 0, s,
                   sb->n_nodes, cap, M, a->f_cnt, a->Gx, a->Gh, a->f_mem, mem_new);
        if (new_mem_ts)
            TGM_HIP(hipMemcpyAsync(new_mem_ts, a->t_new, sizeof(double) * cap,
                                   hipMemcpyDeviceToDevice, s));
    }
    if (R > 0)
        TGM_LAUNCH(k_apan_embed, dim3((unsigned)cdiv((int64_t)R * kWave, 256)), dim3(256), 0, s,
                   R, M, sb->root_pos, mem_new, h);
    // the write set of iter: memory rows of the endpoints, mail deliveries
    const int slots = a->s + 1;
    tgm_apan::Slot &sl = a->ring[iter % slots];
    if (sl.staged)
        return TGM_EORDER;   // cannot happen: commits run ahead of the ring
    const int64_t r = iter % slots, C = a->max_nodes, MD = a->max_del();
    TGM_LAUNCH(k_apan_clear_flags, dim3((unsigned)cdiv(C, 256)), dim3(256), 0, s,
               a->r_flag + r * C, (int)C);
    if (b > 0)
        TGM_LAUNCH(k_apan_stage_mem, dim3((unsigned)cdiv((int64_t)2 * b * kWave, 256)),
                   dim3(256), 0, s, b, M, sb->root_pos, sb->nodes, mem_new, a->t_new,
                   a->r_flag + r * C, a->r_node + r * C, a->r_mem + r * C * M, a->r_ts + r * C);
    const int64_t n_del = (int64_t)2 * b * (nb + 1);
    if (n_del > 0) {
        TGM_LAUNCH(k_apan_keys, dim3((unsigned)cdiv(n_del, 256)), dim3(256), 0, s, b, nb,
                   a->propagate, sb->root, sb->nbr, sb->cnt, a->keys);
        size_t bytes = a->sort_bytes;
        TGM_HIP(hipcub::DeviceRadixSort::SortKeys(a->sort_tmp, bytes, a->keys, a->keys_sorted,
                                                  (int)n_del, 0, 64, s));
        TGM_LAUNCH(k_apan_bounds, dim3((unsigned)cdiv(n_del, 256)), dim3(256), 0, s, n_del,
                   a->keys_sorted, a->N, a->seg, a->seg_end);
        StageArgs2 sa{b, nb, M, a->D_e, D_m, K, a->N, lo, a->keys_sorted, a->seg, a->seg_end,
                      sb->root_pos, mem_new, g->efeat, g->t, a->d_node + r * MD,
                      a->d_rank + r * MD, a->d_keep + r * MD, a->d_mail + r * MD * D_m,
                      a->d_t + r * MD};
        TGM_LAUNCH(k_apan_stage_mail, dim3((unsigned)cdiv(n_del * kWave, 256)), dim3(256), 0, s,
                   sa, n_del);
    }
    sl.iter = iter;
    sl.n_del = n_del;
    sl.staged = true;
    a->staged_through = iter;
    return TGM_OK;
}

namespace {

void apan_restart(tgm_apan *a, int64_t iter)
{
    for (tgm_apan::Slot &sl : a->ring)
        sl = tgm_apan::Slot{};
    a->committed_through = iter - 1;
    a->staged_through = iter - 1;
}

}  // namespace

extern "C" tgm_status_t tgm_apan_reset(tgm_apan_t a, void *stream)
{
    if (!a)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    TGM_LAUNCH(k_apan_init, dim3(1024), dim3(256), 0, s, a->N, a->M, a->K, a->D_m, a->mem,
               a->mem_ts, a->ver, a->mb, a->mb_ts, a->head, a->cnt);
    apan_restart(a, 0);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_apan_load(tgm_apan_t a, int64_t iter, const float *mem,
                                      const double *mem_ts, const int32_t *ver, const float *mb,
                                      const double *mb_ts, const int32_t *mb_cnt, void *stream)
{
    if (!a || iter < 0 || !mem || !mem_ts || !ver || !mb || !mb_ts || !mb_cnt)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t N = a->N, M = a->M;
    TGM_HIP(hipMemcpyAsync(a->mem, mem, 4 * N * M, hipMemcpyDeviceToDevice, s));
    TGM_HIP(hipMemcpyAsync(a->mem_ts, mem_ts, 8 * N, hipMemcpyDeviceToDevice, s));
    TGM_HIP(hipMemcpyAsync(a->ver, ver, 4 * N, hipMemcpyDeviceToDevice, s));
    TGM_LAUNCH(k_apan_load_mb, dim3((unsigned)cdiv((int64_t)N * kWave, 256)), dim3(256), 0, s,
               a->N, a->K, a->D_m, mb, mb_ts, mb_cnt, a->mb, a->mb_ts, a->head, a->cnt);
    apan_restart(a, iter);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_apan_flush(tgm_apan_t a, void *stream)
{
    if (!a)
        return TGM_EINVAL;
    return apan_commit_through(a, a->staged_through, as_stream(stream));
}

extern "C" tgm_status_t tgm_apan_read(tgm_apan_t a, float *mem, double *mem_ts, int32_t *ver,
                                      float *mb, double *mb_ts, int32_t *mb_cnt, void *stream)
{
    if (!a || (!mb) != (!mb_ts))
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t N = a->N, M = a->M;
    if (mem)
        TGM_HIP(hipMemcpyAsync(mem, a->mem, 4 * N * M, hipMemcpyDeviceToDevice, s));
    if (mem_ts)
        TGM_HIP(hipMemcpyAsync(mem_ts, a->mem_ts, 8 * N, hipMemcpyDeviceToDevice, s));
    if (ver)
        TGM_HIP(hipMemcpyAsync(ver, a->ver, 4 * N, hipMemcpyDeviceToDevice, s));
    if (mb_cnt)
        TGM_HIP(hipMemcpyAsync(mb_cnt, a->cnt, 4 * N, hipMemcpyDeviceToDevice, s));
    if (mb)
        TGM_LAUNCH(k_apan_read_mb, dim3((unsigned)cdiv((int64_t)N * kWave, 256)), dim3(256), 0,
                   s, a->N, a->K, a->D_m, a->mb, a->mb_ts, a->head, a->cnt, mb, mb_ts);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_apan_fetched(tgm_apan_t a, float *mem, double *mem_ts, int32_t *ver,
                                         float *mb, double *mb_ts, int32_t *mb_cnt, void *stream)
{
    if (!a)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t C = a->max_nodes, M = a->M, K = a->K, D_m = a->D_m;
    if (mem)
        TGM_HIP(hipMemcpyAsync(mem, a->f_mem, 4 * C * M, hipMemcpyDeviceToDevice, s));
    if (mem_ts)
        TGM_HIP(hipMemcpyAsync(mem_ts, a->f_mem_ts, 8 * C, hipMemcpyDeviceToDevice, s));
    if (ver)
        TGM_HIP(hipMemcpyAsync(ver, a->f_ver, 4 * C, hipMemcpyDeviceToDevice, s));
    if (mb)
        TGM_HIP(hipMemcpyAsync(mb, a->f_mb, 4 * C * K * D_m, hipMemcpyDeviceToDevice, s));
    if (mb_ts)
        TGM_HIP(hipMemcpyAsync(mb_ts, a->f_mb_ts, 8 * C * K, hipMemcpyDeviceToDevice, s));
    if (mb_cnt)
        TGM_HIP(hipMemcpyAsync(mb_cnt, a->f_cnt, 4 * C, hipMemcpyDeviceToDevice, s));
    return TGM_OK;
}
