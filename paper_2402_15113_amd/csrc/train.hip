// Training step after the stage: the link-prediction loss of the batch, its
// gradient with respect to every weight of the model and of the predictor,
// the optimizer step, and the repack of the model's operands (Sec. 5,
// training settings: link prediction on equal numbers of positive and
// negative pairs; App. C.2: the loss and backward steps of the training
// stage).
//
// Every reduction has a fixed order, so results are bit-reproducible: the
// weight gradients are MFMA GEMMs whose long reduction dimension (slots,
// roots, nodes) is split over workgroups into partial sums that a second
// launch adds in split order; the gradient of each node's updated memory
// gathers its contributions (the roots and neighbour slots that read it)
// after a radix sort of (node, contributor) keys.
#include <hip/hip_runtime.h>

#include <hipcub/hipcub.hpp>

#include <algorithm>
#include <cmath>

#include "common.h"

using namespace tgm;

namespace {

// ------------------------------------------------------------------ GEMM
// C[m x n] = op(A)[m x k] op(B)[k x n] (+ bias[n]) (+ C when accumulate),
// row-major.  op(A)(i, kk) = ta ? A[kk lda + i] : A[i lda + kk];
// op(B)(kk, j) = tb ? B[j ldb + kk] : B[kk ldb + j].  A workgroup of 4
// wavefronts takes a 64 x 64 tile (32 x 32 per wavefront, v_mfma 16x16x4)
// over the k range of its split (blockIdx.z); with several splits each
// writes its partial tile to `part` and k_gemm_reduce adds them in order.
// The k range goes in steps of kGK2 = 32 through two LDS buffers: the next
// step's elements load into registers while the current step multiplies,
// and one barrier per step hands the buffers over.  Within a split every
// accumulator takes its k in increasing order, 16 at a time.
constexpr int kGT = 64, kGK = 16, kGK2 = 32, kGPad = 4;
constexpr int kMaxSplits = 64;

struct GemmArgs {
    int m, n, k;
    const float *A;
    int lda;
    const float *B;
    int ldb;
    float *C;
    int ldc;
    const float *bias;
    int accumulate;
    int splits, kchunk;
    float *part;
    const int32_t *m_live;   // rows at or past *m_live are skipped (NULL: none)
};

// Element u of this thread's share of a 64 x kGK2 operand tile: (row, kk) of
// the tile, laid out so that consecutive threads read consecutive addresses.
template <bool T>
__device__ __forceinline__ void gemm_elem(int tid, int u, int &r, int &kk)
{
    const int e = tid + u * 256;
    if (T) {   // element (r, kk) at X[kk ld + r]: rows contiguous
        r = e & (kGT - 1);
        kk = e >> 6;
    } else {   // element (r, kk) at X[r ld + kk]: k contiguous
        r = e >> 5;
        kk = e & (kGK2 - 1);
    }
}

template <bool TA, bool TB>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g)
{
    __shared__ __align__(16) float As[2][kGT][kGK2 + kGPad];
    __shared__ __align__(16) float Bs[2][kGT][kGK2 + kGPad];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m0 = blockIdx.y * kGT, n0 = blockIdx.x * kGT, z = blockIdx.z;
    if (g.m_live && m0 >= *g.m_live)
        return;   // the whole tile is past the live rows
    const int k_lo = z * g.kchunk, k_hi = min(g.k, k_lo + g.kchunk);
    const int wr = (wave >> 1) * 32, wc = (wave & 1) * 32;
    const int q = lane >> 4, rl = lane & 15;
    // the tile's elements of one k step, loaded branch-free (clamped
    // addresses; the zero mask is applied where they are stored)
    constexpr int NE = kGT * kGK2 / 256;
    float ra[NE], rb[NE];
    auto load = [&](int k0) {
#pragma unroll
        for (int u = 0; u < NE; ++u) {
            int i, kk;
            gemm_elem<TA>(tid, u, i, kk);
            const int gi = min(m0 + i, g.m - 1), gk = min(k0 + kk, g.k - 1);
            ra[u] = TA ? g.A[(int64_t)gk * g.lda + gi] : g.A[(int64_t)gi * g.lda + gk];
            int j, kb;
            gemm_elem<!TB>(tid, u, j, kb);
            const int gj = min(n0 + j, g.n - 1), gkb = min(k0 + kb, g.k - 1);
            rb[u] = TB ? g.B[(int64_t)gj * g.ldb + gkb] : g.B[(int64_t)gkb * g.ldb + gj];
        }
    };
    auto store = [&](int k0, int buf) {
#pragma unroll
        for (int u = 0; u < NE; ++u) {
            int i, kk;
            gemm_elem<TA>(tid, u, i, kk);
            As[buf][i][kk] = (m0 + i < g.m && k0 + kk < k_hi) ? ra[u] : 0.f;
            int j, kb;
            gemm_elem<!TB>(tid, u, j, kb);
            Bs[buf][j][kb] = (n0 + j < g.n && k0 + kb < k_hi) ? rb[u] : 0.f;
        }
    };
    f4 acc[2][2];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
            acc[bi][bj] = f4{0.f, 0.f, 0.f, 0.f};
    if (k_lo < k_hi) {
        load(k_lo);
        store(k_lo, 0);
        __syncthreads();
    }
    int buf = 0;
    for (int k0 = k_lo; k0 < k_hi; k0 += kGK2, buf ^= 1) {
        const bool more = k0 + kGK2 < k_hi;
        if (more)
            load(k0 + kGK2);
#pragma unroll
        for (int h = 0; h < kGK2 / kGK; ++h) {
#pragma unroll
            for (int bi = 0; bi < 2; ++bi) {
                const f4 a = *reinterpret_cast<const f4 *>(&As[buf][wr + bi * 16 + rl][16 * h + 4 * q]);
#pragma unroll
                for (int bj = 0; bj < 2; ++bj) {
                    const f4 bv =
                        *reinterpret_cast<const f4 *>(&Bs[buf][wc + bj * 16 + rl][16 * h + 4 * q]);
                    acc[bi][bj] = mfma_k16(a, bv, acc[bi][bj]);
                }
            }
        }
        if (more) {
            store(k0 + kGK2, buf ^ 1);
            __syncthreads();
        }
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = m0 + wr + bi * 16 + 4 * q + v, col = n0 + wc + bj * 16 + rl;
                if (row >= g.m || col >= g.n)
                    continue;
                float x = acc[bi][bj][v];
                if (g.splits > 1) {
                    g.part[((int64_t)z * g.m + row) * g.n + col] = x;
                } else {
                    if (g.bias)
                        x += g.bias[col];
                    float *c = g.C + (int64_t)row * g.ldc + col;
                    *c = g.accumulate ? *c + x : x;
                }
            }
}

__global__ __launch_bounds__(256) void k_gemm_reduce(GemmArgs g)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= (int64_t)g.m * g.n)
        return;
    const int row = (int)(t / g.n), col = (int)(t % g.n);
    float x = 0.f;
    for (int z = 0; z < g.splits; ++z)
        x += g.part[((int64_t)z * g.m + row) * g.n + col];
    if (g.bias)
        x += g.bias[col];
    float *c = g.C + (int64_t)row * g.ldc + col;
    *c = g.accumulate ? *c + x : x;
}

// ------------------------------------------------------------- predictor
// One wavefront per event e < b (lanes over the hidden units j < M <= 128):
// z+ = Zs[e] + Zd[e] + b_p, z- = Zs[e] + Zd[b + e] + b_p, the two scores, the
// event's loss, and the gradients of the scores (dsc) and pre-activations.
struct PredArgs {
    int b, M;
    const float *Zs, *Zd;        // [b x M], [2b x M]
    const float *b_p, *w_out, *b_out;
    float *dZsrc, *dZdst, *act;  // [b x M], [2b x M], [2b x M]
    float *dsc, *lossv;          // [2b], [b]
};

__device__ __forceinline__ float softplusf(float x)
{
    return x > 0.f ? x + log1pf(expf(-x)) : log1pf(expf(x));
}
__device__ __forceinline__ float sigmoidf(float x) { return 1.f / (1.f + expf(-x)); }

__global__ __launch_bounds__(256) void k_pred(PredArgs a)
{
    const int e = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (e >= a.b)
        return;
    const int M = a.M, b = a.b;
    float zp[2], zn[2], sp = 0.f, sn = 0.f;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int j = lane + 64 * u;
        zp[u] = zn[u] = 0.f;
        if (j < M) {
            const float zs = a.Zs[(int64_t)e * M + j] + a.b_p[j];
            zp[u] = zs + a.Zd[(int64_t)e * M + j];
            zn[u] = zs + a.Zd[(int64_t)(b + e) * M + j];
            sp += a.w_out[j] * fmaxf(zp[u], 0.f);
            sn += a.w_out[j] * fmaxf(zn[u], 0.f);
        }
    }
    sp = wave_sum(sp) + a.b_out[0];
    sn = wave_sum(sn) + a.b_out[0];
    const float dsp = (sigmoidf(sp) - 1.f) / (float)b, dsn = sigmoidf(sn) / (float)b;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int j = lane + 64 * u;
        if (j >= M)
            continue;
        const float dzp = zp[u] > 0.f ? dsp * a.w_out[j] : 0.f;
        const float dzn = zn[u] > 0.f ? dsn * a.w_out[j] : 0.f;
        a.dZsrc[(int64_t)e * M + j] = dzp + dzn;
        a.dZdst[(int64_t)e * M + j] = dzp;
        a.dZdst[(int64_t)(b + e) * M + j] = dzn;
        a.act[(int64_t)e * M + j] = fmaxf(zp[u], 0.f);
        a.act[(int64_t)(b + e) * M + j] = fmaxf(zn[u], 0.f);
    }
    if (lane == 0) {
        a.dsc[e] = dsp;
        a.dsc[b + e] = dsn;
        a.lossv[e] = softplusf(-sp) + softplusf(sn);
    }
}

// loss = (1/b) sum of the events' losses, in a fixed order (one workgroup)
__global__ __launch_bounds__(256) void k_loss(const float *__restrict__ lossv, int b,
                                              float *__restrict__ out)
{
    __shared__ float part[256];
    float x = 0.f;
    for (int e = threadIdx.x; e < b; e += 256)
        x += lossv[e];
    part[threadIdx.x] = x;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w)
            part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        *out = part[0] / (float)b;
}

// ------------------------------------------------------------- attention
// Rows of the attention's inputs, one wavefront per row: Xq[r] = [s'_v ||
// phi(0)] for the R roots, then kap[sl] = [s'_u || efeat[eid] || phi(t - t')]
// for the R nb slots (zero for slots past the root's count).
struct RowArgs {
    int R, nb, M, D_e, D_t;
    const int32_t *root_pos, *nbr_pos, *eid, *cnt;
    const double *root_ts, *nts, *omega, *beta;
    const float *s_new, *efeat;
    float *Xq, *kap;
};

__global__ __launch_bounds__(256) void k_att_rows(RowArgs a)
{
    const int64_t w = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    const int M = a.M, D_e = a.D_e, D_t = a.D_t;
    if (w < a.R) {
        const int r = (int)w;
        float *x = a.Xq + (int64_t)r * (M + D_t);
        const float *sv = a.s_new + (int64_t)a.root_pos[r] * M;
        for (int k = lane; k < M; k += kWave)
            x[k] = sv[k];
        for (int d = lane; d < D_t; d += kWave)
            x[M + d] = time_enc(a.omega[d], a.beta[d], 0.0);
        return;
    }
    const int64_t sl = w - a.R;
    if (sl >= (int64_t)a.R * a.nb)
        return;
    const int r = (int)(sl / a.nb), j = (int)(sl % a.nb);
    const int Dkv = M + D_e + D_t;
    float *x = a.kap + sl * Dkv;
    if (j >= a.cnt[r]) {
        for (int k = lane; k < Dkv; k += kWave)
            x[k] = 0.f;
        return;
    }
    const float *su = a.s_new + (int64_t)a.nbr_pos[sl] * M;
    const float *f = a.efeat + (int64_t)a.eid[sl] * D_e;
    const double dt = a.root_ts[r] - a.nts[sl];
    for (int k = lane; k < M; k += kWave)
        x[k] = su[k];
    for (int k = lane; k < D_e; k += kWave)
        x[M + k] = f[k];
    for (int d = lane; d < D_t; d += kWave)
        x[M + D_e + d] = time_enc(a.omega[d], a.beta[d], dt);
}

// One wavefront per root: the scores of each head over the root's valid
// slots, their softmax (alpha [R x H x nb]) and a = sum_j alpha_j V_j into
// Xo[:, 0:M]; Xo[:, M:2M] = s'_v.  Lanes hold the output dims k = lane,
// lane + 64 (M <= 128).
struct CoreArgs {
    int R, nb, M, H;
    float scale;
    const int32_t *cnt, *root_pos;
    const float *Q, *KV, *s_new, *dXo;   // [R x M], [R nb x 2M], [cap x M], [R x 2M]
    float *alpha, *Xo;                   // [R x H x nb], [R x 2M]
    float *dKV, *dQ;                     // [R nb x 2M], [R x M]
};

__device__ __forceinline__ float wave_max(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}

__global__ __launch_bounds__(256) void k_att_core(CoreArgs a)
{
    const int r = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (r >= a.R)
        return;
    const int M = a.M, H = a.H, nb = a.nb, dh = M / H, cr = a.cnt[r];
    float q[2], acc[2] = {0.f, 0.f};
    int head[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int k = lane + 64 * u;
        q[u] = k < M ? a.Q[(int64_t)r * M + k] : 0.f;
        head[u] = k < M ? k / dh : -1;
    }
    for (int eta = 0; eta < H && cr > 0; ++eta) {
        float mine = -INFINITY;   // lane j < cr: the score of slot j
        for (int j = 0; j < cr; ++j) {
            const float *K = a.KV + ((int64_t)r * nb + j) * 2 * M;
            float p = 0.f;
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (head[u] == eta)
                    p += q[u] * K[lane + 64 * u];
            const float sc = wave_sum(p) * a.scale;
            if (lane == j)
                mine = sc;
        }
        const float mx = wave_max(mine);
        const float ex = lane < cr ? expf(mine - mx) : 0.f;
        const float al = ex / wave_sum(ex);
        if (lane < cr)
            a.alpha[((int64_t)r * H + eta) * nb + lane] = al;
        for (int j = 0; j < cr; ++j) {
            const float alj = __shfl(al, j, kWave);
            const float *V = a.KV + ((int64_t)r * nb + j) * 2 * M + M;
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (head[u] == eta)
                    acc[u] += alj * V[lane + 64 * u];
        }
    }
    const float *sv = a.s_new + (int64_t)a.root_pos[r] * M;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int k = lane + 64 * u;
        if (k < M) {
            a.Xo[(int64_t)r * 2 * M + k] = acc[u];
            a.Xo[(int64_t)r * 2 * M + M + k] = sv[k];
        }
    }
}

// Backward of the core, one wavefront per root: with da = dXo[:, 0:M],
// dalpha_j = da . V_j (per head), dscore_j = alpha_j (dalpha_j - sum alpha
// dalpha), dV_j = alpha_j da, dK_j = dscore_j q scale, dq = sum_j dscore_j K_j
// scale.  Slots past the count get zero rows.
__global__ __launch_bounds__(256) void k_att_core_bwd(CoreArgs a)
{
    const int r = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (r >= a.R)
        return;
    const int M = a.M, H = a.H, nb = a.nb, dh = M / H, cr = a.cnt[r];
    float q[2], da[2], dq[2] = {0.f, 0.f};
    int head[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int k = lane + 64 * u;
        q[u] = k < M ? a.Q[(int64_t)r * M + k] : 0.f;
        da[u] = k < M ? a.dXo[(int64_t)r * 2 * M + k] : 0.f;
        head[u] = k < M ? k / dh : -1;
    }
    for (int eta = 0; eta < H && cr > 0; ++eta) {
        const float *al = a.alpha + ((int64_t)r * H + eta) * nb;
        float sdot = 0.f;
        for (int j = 0; j < cr; ++j) {
            const float *V = a.KV + ((int64_t)r * nb + j) * 2 * M + M;
            float p = 0.f;
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (head[u] == eta)
                    p += da[u] * V[lane + 64 * u];
            sdot += al[j] * wave_sum(p);
        }
        for (int j = 0; j < cr; ++j) {
            const float *K = a.KV + ((int64_t)r * nb + j) * 2 * M;
            const float *V = K + M;
            float p = 0.f;
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (head[u] == eta)
                    p += da[u] * V[lane + 64 * u];
            const float dal = wave_sum(p);
            const float dsc = al[j] * (dal - sdot) * a.scale;
            float *dK = a.dKV + ((int64_t)r * nb + j) * 2 * M;
#pragma unroll
            for (int u = 0; u < 2; ++u)
                if (head[u] == eta) {
                    const int k = lane + 64 * u;
                    dK[k] = dsc * q[u];
                    dK[M + k] = al[j] * da[u];
                    dq[u] += dsc * K[k];
                }
        }
    }
    for (int j = cr; j < nb; ++j) {
        float *dK = a.dKV + ((int64_t)r * nb + j) * 2 * M;
        for (int k = lane; k < 2 * M; k += kWave)
            dK[k] = 0.f;
    }
    if (cr == 0)
        for (int j = 0; j < nb; ++j) {
            float *dK = a.dKV + ((int64_t)r * nb + j) * 2 * M;
            for (int k = lane; k < 2 * M; k += kWave)
                dK[k] = 0.f;
        }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int k = lane + 64 * u;
        if (k < M)
            a.dQ[(int64_t)r * M + k] = dq[u];
    }
}

// dst = src where gate > 0, else 0 (the ReLU of the output projection)
__global__ __launch_bounds__(256) void k_relu_mask(const float *__restrict__ src,
                                                   const float *__restrict__ gate,
                                                   float *__restrict__ dst, int64_t n)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t < n)
        dst[t] = gate[t] > 0.f ? src[t] : 0.f;
}

// ------------------------------------------- gradient of the new memories
// Keys (node << 32) | contributor: contributor r < R is root r (it reads s'
// of node root_pos[r]), R + sl is slot sl (node nbr_pos[sl]); empty slots get
// the largest key.
__global__ __launch_bounds__(256) void k_ds_keys(int R, int nb, const int32_t *__restrict__ root_pos,
                                                 const int32_t *__restrict__ nbr_pos,
                                                 const int32_t *__restrict__ cnt,
                                                 uint64_t *__restrict__ keys)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const int64_t S = (int64_t)R * nb;
    if (t >= R + S)
        return;
    uint64_t key;
    if (t < R) {
        key = ((uint64_t)(uint32_t)root_pos[t] << 32) | (uint64_t)t;
    } else {
        const int64_t sl = t - R;
        const int r = (int)(sl / nb), j = (int)(sl % nb);
        key = j < cnt[r] ? ((uint64_t)(uint32_t)nbr_pos[sl] << 32) | (uint64_t)t : ~(uint64_t)0;
    }
    keys[t] = key;
}

// Segment bounds of the sorted keys: seg[p] .. seg_end[p] hold node p's
// contributors, in contributor order.
__global__ __launch_bounds__(256) void k_ds_bounds(int64_t n, const uint64_t *__restrict__ keys,
                                                   int32_t cap, int32_t *__restrict__ seg,
                                                   int32_t *__restrict__ seg_end)
{
    const int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    const uint64_t k = keys[i];
    if (k == ~(uint64_t)0)
        return;
    const int32_t p = (int32_t)(k >> 32);
    if (p < 0 || p >= cap)
        return;
    if (i == 0 || (keys[i - 1] >> 32) != (k >> 32))
        seg[p] = (int32_t)i;
    if (i == n - 1 || (keys[i + 1] >> 32) != (k >> 32))
        seg_end[p] = (int32_t)(i + 1);
}

// The sum runs in fixed chunks of kDsChunk contributors so that nodes with
// many contributors (hubs) spread over many wavefronts.  k_ds_chunks counts
// each node's chunks and scans the counts (one workgroup: chunk_off[p] is the
// first chunk of node p, chunk_off[cap] the total); k_ds_partial sums one
// chunk per wavefront iteration (a grid-stride loop over the chunks); k_ds
// adds each node's chunk sums in order.  ds[p] is, in contributor order, the
// sum of dXq[r] + dXo[r][M:2M] over its roots and of dKm[sl] over its slots.
constexpr int kDsChunk = 64;
constexpr int kDsScanThreads = 1024;

__global__ __launch_bounds__(kDsScanThreads) void k_ds_chunks(const int32_t *__restrict__ n_nodes,
                                                              int32_t cap,
                                                              const int32_t *__restrict__ seg,
                                                              const int32_t *__restrict__ seg_end,
                                                              int32_t *__restrict__ chunk_off)
{
    __shared__ int32_t s_sum[kDsScanThreads];
    const int n = min(*n_nodes, cap), tid = threadIdx.x;
    // each thread takes a contiguous run of nodes
    const int per = (cap + kDsScanThreads - 1) / kDsScanThreads;
    const int p0 = tid * per, p1 = min(cap, p0 + per);
    auto chunks = [&](int p) {
        return p < n ? (max(seg_end[p] - seg[p], 0) + kDsChunk - 1) / kDsChunk : 0;
    };
    int32_t local = 0;
    for (int p = p0; p < p1; ++p)
        local += chunks(p);
    s_sum[tid] = local;
    __syncthreads();
    for (int o = 1; o < kDsScanThreads; o <<= 1) {   // inclusive scan (Hillis-Steele)
        const int32_t v = tid >= o ? s_sum[tid - o] : 0;
        __syncthreads();
        s_sum[tid] += v;
        __syncthreads();
    }
    int32_t run = s_sum[tid] - local;
    for (int p = p0; p < p1; ++p) {
        chunk_off[p] = run;
        run += chunks(p);
    }
    if (tid == kDsScanThreads - 1)
        chunk_off[cap] = s_sum[tid];
}

__global__ __launch_bounds__(256) void k_ds_partial(int32_t cap, int M, int R, int64_t n_items,
                                                    const uint64_t *__restrict__ keys,
                                                    const int32_t *__restrict__ seg,
                                                    const int32_t *__restrict__ seg_end,
                                                    const int32_t *__restrict__ chunk_off,
                                                    const float *__restrict__ dXq,
                                                    const float *__restrict__ dXo,
                                                    const float *__restrict__ dKm,
                                                    float *__restrict__ part)
{
    const int lane = threadIdx.x & 63;
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    const int32_t total = chunk_off[cap];
    for (int64_t t = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6; t < total; t += nw) {
        int lo = 0, hi = cap;   // the node p with chunk_off[p] <= t < chunk_off[p + 1]
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (chunk_off[mid] <= t)
                lo = mid;
            else
                hi = mid;
        }
        const int p = lo;
        const int64_t i0 = max((int64_t)seg[p], (int64_t)0) + (t - chunk_off[p]) * kDsChunk;
        const int64_t i1 = min(min((int64_t)seg_end[p], i0 + kDsChunk), n_items);
        float acc[2] = {0.f, 0.f};
        for (int64_t i = i0; i < i1; ++i) {
            const int64_t c = (int64_t)(keys[i] & 0xffffffffu);
            if (c >= n_items)
                continue;
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int k = lane + 64 * u;
                if (k >= M)
                    continue;
                acc[u] += c < R ? dXq[c * M + k] + dXo[c * 2 * M + M + k]
                                : dKm[(c - R) * M + k];
            }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int k = lane + 64 * u;
            if (k < M)
                part[t * M + k] = acc[u];
        }
    }
}

__global__ __launch_bounds__(256) void k_ds(const int32_t *__restrict__ n_nodes, int32_t cap,
                                            int M, const int32_t *__restrict__ chunk_off,
                                            const float *__restrict__ part, float *__restrict__ ds)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (p >= cap)
        return;
    const int n = min(*n_nodes, cap);
    float acc[2] = {0.f, 0.f};
    if (p < n)
        for (int32_t t = chunk_off[p]; t < chunk_off[p + 1]; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int k = lane + 64 * u;
                if (k < M)
                    acc[u] += part[(int64_t)t * M + k];
            }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int k = lane + 64 * u;
        if (k < M)
            ds[(int64_t)p * M + k] = acc[u];
    }
}

// ------------------------------------------------------------------- GRU
// Rows of the memory updater's inputs: X[p] = [mail || phi(mail_ts - mem_ts)]
// and Hm[p] = mem[p] for nodes with mail (p < n_nodes, ver >= 0), zero rows
// for the others (up to cap), one wavefront per row.
struct GruRowArgs {
    const int32_t *n_nodes;
    int cap, M, D_m, D_t;
    const float *mem, *mail;
    const double *mem_ts, *mail_ts, *omega, *beta;
    const int32_t *ver;
    float *X, *Hm;
};

__global__ __launch_bounds__(256) void k_gru_rows(GruRowArgs a)
{
    const int p = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (p >= a.cap)
        return;
    const int M = a.M, D_m = a.D_m, D_t = a.D_t, D_x = D_m + D_t;
    float *x = a.X + (int64_t)p * D_x, *hm = a.Hm + (int64_t)p * M;
    const bool on = p < min(*a.n_nodes, a.cap) && a.ver[p] >= 0;
    if (!on) {
        for (int k = lane; k < D_x; k += kWave)
            x[k] = 0.f;
        for (int k = lane; k < M; k += kWave)
            hm[k] = 0.f;
        return;
    }
    const float *ml = a.mail + (int64_t)p * D_m;
    for (int k = lane; k < D_m; k += kWave)
        x[k] = ml[k];
    const double dt = a.mail_ts[p] - a.mem_ts[p];
    for (int d = lane; d < D_t; d += kWave)
        x[D_m + d] = time_enc(a.omega[d], a.beta[d], dt);
    for (int k = lane; k < M; k += kWave)
        hm[k] = a.mem[(int64_t)p * M + k];
}

// One thread per (node, hidden unit): the gates again from Gx = X W_ih^t +
// b_ih and Gh = Hm W_hh^t + b_hh, then the gradients of the gate
// pre-activations: dGx = [da_r | da_z | da_n], dGh = [da_r | da_z | da_n r].
__global__ __launch_bounds__(256) void k_gru_bwd(const int32_t *__restrict__ n_nodes, int cap,
                                                 int M, const int32_t *__restrict__ ver,
                                                 const float *__restrict__ Gx,
                                                 const float *__restrict__ Gh,
                                                 const float *__restrict__ Hm,
                                                 const float *__restrict__ ds,
                                                 float *__restrict__ dGx, float *__restrict__ dGh)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= (int64_t)cap * M)
        return;
    const int p = (int)(t / M), j = (int)(t % M);
    const int64_t o = (int64_t)p * 3 * M;
    if (p >= min(*n_nodes, cap) || ver[p] < 0) {
        dGx[o + j] = dGx[o + M + j] = dGx[o + 2 * M + j] = 0.f;
        dGh[o + j] = dGh[o + M + j] = dGh[o + 2 * M + j] = 0.f;
        return;
    }
    const float r = sigmoidf(Gx[o + j] + Gh[o + j]);
    const float z = sigmoidf(Gx[o + M + j] + Gh[o + M + j]);
    const float hn = Gh[o + 2 * M + j];
    const float n = tanhf(Gx[o + 2 * M + j] + r * hn);
    const float d = ds[(int64_t)p * M + j];
    const float dn = d * (1.f - z), dz = d * (Hm[(int64_t)p * M + j] - n);
    const float dan = dn * (1.f - n * n);
    const float dar = dan * hn * r * (1.f - r), daz = dz * z * (1.f - z);
    dGx[o + j] = dar;
    dGx[o + M + j] = daz;
    dGx[o + 2 * M + j] = dan;
    dGh[o + j] = dar;
    dGh[o + M + j] = daz;
    dGh[o + 2 * M + j] = dan * r;
}

// ------------------------------------------------------------- optimizer
__global__ __launch_bounds__(256) void k_sgd(float *__restrict__ theta, const float *__restrict__ g,
                                             int64_t n, float lr)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t < n)
        theta[t] -= lr * g[t];
}

// Adam with bias correction: c1 = 1 - beta1^t, c2 = 1 - beta2^t
__global__ __launch_bounds__(256) void k_adam(float *__restrict__ theta,
                                              const float *__restrict__ g, float *__restrict__ m1,
                                              float *__restrict__ m2, int64_t n, float lr,
                                              float b1, float b2, float eps, float c1, float c2)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t >= n)
        return;
    const float gt = g[t];
    const float a = b1 * m1[t] + (1.f - b1) * gt;
    const float v = b2 * m2[t] + (1.f - b2) * gt * gt;
    m1[t] = a;
    m2[t] = v;
    theta[t] -= lr * (a / c1) / (sqrtf(v / c2) + eps);
}

__global__ __launch_bounds__(256) void k_fill_f32(float *__restrict__ p, int64_t n, float v)
{
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (t < n)
        p[t] = v;
}

constexpr int kNParams = 17;

}  // namespace

struct tgm_trainer {
    tgm_model_t model = nullptr;
    int32_t M = 0, D_e = 0, D_t = 0, H = 0, nb = 0, D_m = 0, D_x = 0, Dq = 0, Dkv = 0;
    int32_t max_roots = 0, max_b = 0, max_nodes = 0;
    int32_t opt = TGM_OPT_ADAM;
    float lr = 1e-4f, beta1 = 0.9f, beta2 = 0.999f, eps = 1e-8f;
    int64_t steps = 0;
    int64_t n_params = 0;
    int64_t off[kNParams + 1] = {};
    float *theta = nullptr, *grad = nullptr, *m1 = nullptr, *m2 = nullptr;
    // work space
    float *ones = nullptr, *part = nullptr;
    int64_t part_floats = 0;
    float *Zs = nullptr, *Zd = nullptr, *dZsrc = nullptr, *dZdst = nullptr, *act = nullptr;
    float *dsc = nullptr, *lossv = nullptr, *loss = nullptr;
    float *dh = nullptr, *Xq = nullptr, *Q = nullptr, *kap = nullptr, *KV = nullptr;
    float *alpha = nullptr, *Xo = nullptr, *O = nullptr, *dO = nullptr, *dXo = nullptr;
    float *dKV = nullptr, *dQ = nullptr, *dKm = nullptr, *dXq = nullptr, *ds = nullptr;
    float *X = nullptr, *Hm = nullptr, *Gx = nullptr, *Gh = nullptr, *dGx = nullptr,
          *dGh = nullptr;
    uint64_t *keys = nullptr, *keys_sorted = nullptr;
    int32_t *seg = nullptr, *seg_end = nullptr, *chunk_off = nullptr;
    float *ds_part = nullptr;   // [(R + S) / kDsChunk + max_nodes] x M chunk sums
    void *sort_tmp = nullptr;
    size_t sort_bytes = 0;
    float *p(int k) const { return theta + off[k]; }
    float *gr(int k) const { return grad + off[k]; }
};

namespace {

// C = op(A) op(B) (+ bias) (+ C): split-K when the output has few tiles and
// the reduction is long (the weight gradients), so the grid fills the GPU
tgm_status_t gemm(const tgm_trainer *tr, bool ta, bool tb, int m, int n, int k, const float *A,
                  int lda, const float *B, int ldb, float *C, int ldc, const float *bias,
                  bool accumulate, hipStream_t s)
{
    if (m <= 0 || n <= 0)
        return TGM_OK;
    GemmArgs g;
    g.m = m;
    g.n = n;
    g.k = k;
    g.A = A;
    g.lda = lda;
    g.B = B;
    g.ldb = ldb;
    g.C = C;
    g.ldc = ldc;
    g.bias = bias;
    g.accumulate = accumulate ? 1 : 0;
    g.part = tr->part;
    g.m_live = nullptr;
    const int64_t tiles = cdiv(m, kGT) * cdiv(n, kGT);
    int splits = 1;
    if (tiles < 512 && k > 4 * kGK * 16) {
        splits = (int)std::min<int64_t>(cdiv(k, 256), std::max<int64_t>(1, 1024 / tiles));
        splits = std::min(splits, kMaxSplits);
        while (splits > 1 && (int64_t)splits * m * n > tr->part_floats)
            --splits;
    }
    int kchunk = round_up((int32_t)cdiv(std::max(k, 1), splits), kGK);
    splits = std::max(1, (int)cdiv(std::max(k, 1), kchunk));
    g.splits = splits;
    g.kchunk = kchunk;
    const dim3 grid((unsigned)cdiv(n, kGT), (unsigned)cdiv(m, kGT), (unsigned)splits);
    if (!ta && !tb)
        TGM_LAUNCH((k_gemm<false, false>), grid, dim3(256), 0, s, g);
    else if (!ta && tb)
        TGM_LAUNCH((k_gemm<false, true>), grid, dim3(256), 0, s, g);
    else if (ta && !tb)
        TGM_LAUNCH((k_gemm<true, false>), grid, dim3(256), 0, s, g);
    else
        TGM_LAUNCH((k_gemm<true, true>), grid, dim3(256), 0, s, g);
    if (splits > 1)
        TGM_LAUNCH(k_gemm_reduce, dim3((unsigned)cdiv((int64_t)m * n, 256)), dim3(256), 0, s, g);
    return TGM_OK;
}

// column sums of X [rows x n] (leading dimension ldx): the bias gradients
tgm_status_t colsum(const tgm_trainer *tr, int rows, int n, const float *X, int ldx, float *out,
                    hipStream_t s)
{
    return gemm(tr, true, false, 1, n, rows, tr->ones, 1, X, ldx, out, n, nullptr, false, s);
}

}  // namespace

tgm_status_t tgm::gemm_f32(bool ta, bool tb, int m, int n, int k, const float *A, int lda,
                          const float *B, int ldb, float *C, int ldc, const float *bias,
                          bool accumulate, hipStream_t s, const int32_t *m_live)
{
    if (m <= 0 || n <= 0)
        return TGM_OK;
    GemmArgs g;
    g.m = m;
    g.n = n;
    g.k = k;
    g.A = A;
    g.lda = lda;
    g.B = B;
    g.ldb = ldb;
    g.C = C;
    g.ldc = ldc;
    g.bias = bias;
    g.accumulate = accumulate ? 1 : 0;
    g.part = nullptr;
    g.m_live = m_live;
    g.splits = 1;
    g.kchunk = round_up((int32_t)std::max(k, 1), kGK);
    const dim3 grid((unsigned)cdiv(n, kGT), (unsigned)cdiv(m, kGT), 1);
    if (!ta && !tb)
        TGM_LAUNCH((k_gemm<false, false>), grid, dim3(256), 0, s, g);
    else if (!ta && tb)
        TGM_LAUNCH((k_gemm<false, true>), grid, dim3(256), 0, s, g);
    else if (ta && !tb)
        TGM_LAUNCH((k_gemm<true, false>), grid, dim3(256), 0, s, g);
    else
        TGM_LAUNCH((k_gemm<true, true>), grid, dim3(256), 0, s, g);
    return TGM_OK;
}

// ======================================================================== API

extern "C" tgm_status_t tgm_trainer_destroy(tgm_trainer_t tr)
{
    if (!tr)
        return TGM_EINVAL;
    float *bufs[] = {tr->theta, tr->grad, tr->m1, tr->m2, tr->ones, tr->part, tr->Zs, tr->Zd,
                     tr->dZsrc, tr->dZdst, tr->act, tr->dsc, tr->lossv, tr->loss, tr->dh, tr->Xq,
                     tr->Q, tr->kap, tr->KV, tr->alpha, tr->Xo, tr->O, tr->dO, tr->dXo, tr->dKV,
                     tr->dQ, tr->dKm, tr->dXq, tr->ds, tr->X, tr->Hm, tr->Gx, tr->Gh, tr->dGx,
                     tr->dGh};
    for (float *b : bufs)
        (void)hipFree(b);
    (void)hipFree(tr->keys);
    (void)hipFree(tr->keys_sorted);
    (void)hipFree(tr->seg);
    (void)hipFree(tr->seg_end);
    (void)hipFree(tr->chunk_off);
    (void)hipFree(tr->ds_part);
    (void)hipFree(tr->sort_tmp);
    delete tr;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_trainer_create(tgm_model_t m, const tgm_weights *w,
                                           const tgm_predictor *pred, const tgm_optimizer *opt,
                                           void *stream, tgm_trainer_t *out)
{
    if (!out)
        return TGM_EINVAL;
    *out = nullptr;
    if (!m || !w || !pred || !opt || m->kind != TGM_MODEL_TGN)
        return TGM_EINVAL;
    if (!w->W_ih || !w->W_hh || !w->b_ih || !w->b_hh || !w->W_q || !w->b_q || !w->W_k ||
        !w->b_k || !w->W_v || !w->b_v || !w->W_o || !w->b_o || !pred->W_src || !pred->W_dst ||
        !pred->b_p || !pred->w_out)
        return TGM_EINVAL;
    if ((opt->kind != TGM_OPT_SGD && opt->kind != TGM_OPT_ADAM) || !(opt->lr >= 0.f) ||
        (opt->kind == TGM_OPT_ADAM &&
         (!(opt->beta1 >= 0.f && opt->beta1 < 1.f) || !(opt->beta2 >= 0.f && opt->beta2 < 1.f) ||
          !(opt->eps > 0.f))))
        return TGM_EINVAL;
    if (m->M > 128 || m->max_roots % 3 != 0)
        return TGM_EINVAL;
    tgm_trainer *tr = new tgm_trainer();
    tr->model = m;
    const int M = m->M, D_e = m->D_e, D_t = m->D_t, nb = m->nb;
    tr->M = M;
    tr->D_e = D_e;
    tr->D_t = D_t;
    tr->H = m->H;
    tr->nb = nb;
    tr->D_m = m->D_m;
    tr->D_x = m->D_x;
    tr->Dq = M + D_t;
    tr->Dkv = M + D_e + D_t;
    tr->max_roots = m->max_roots;
    tr->max_b = m->max_roots / 3;
    tr->max_nodes = m->max_nodes;
    tr->opt = opt->kind;
    tr->lr = opt->lr;
    tr->beta1 = opt->beta1;
    tr->beta2 = opt->beta2;
    tr->eps = opt->eps;
    const int64_t D_x = tr->D_x, Dq = tr->Dq, Dkv = tr->Dkv;
    const int64_t sizes[kNParams] = {3 * M * D_x, 3 * (int64_t)M * M, 3 * M, 3 * M, M * Dq, M,
                                     M * Dkv, M, M * Dkv, M, 2 * (int64_t)M * M, M,
                                     (int64_t)M * M, (int64_t)M * M, M, M, 1};
    for (int k = 0; k < kNParams; ++k)
        tr->off[k + 1] = tr->off[k] + sizes[k];
    tr->n_params = tr->off[kNParams];
    const int64_t R = tr->max_roots, B = tr->max_b, S = R * nb, C = tr->max_nodes;
    const int64_t n_items = R + S;
    // the largest weight-gradient output times the largest split count
    const int64_t mn = std::max<int64_t>({3 * M * D_x, 2 * (int64_t)M * Dkv, M * Dq,
                                          2 * (int64_t)M * M, 3 * (int64_t)M * M});
    tr->part_floats = (int64_t)kMaxSplits * mn;
    tgm_status_t st = TGM_OK;
    auto alloc = [&](auto **ptr, int64_t count) {
        if (st == TGM_OK &&
            dev_malloc(ptr, sizeof(**ptr) * (size_t)std::max<int64_t>(count, 1)) != hipSuccess)
            st = TGM_ENOMEM;
    };
    alloc(&tr->theta, tr->n_params);
    alloc(&tr->grad, tr->n_params);
    alloc(&tr->m1, tr->n_params);
    alloc(&tr->m2, tr->n_params);
    alloc(&tr->ones, std::max({S, C, R}));
    alloc(&tr->part, tr->part_floats);
    alloc(&tr->Zs, B * M);
    alloc(&tr->Zd, 2 * B * M);
    alloc(&tr->dZsrc, B * M);
    alloc(&tr->dZdst, 2 * B * M);
    alloc(&tr->act, 2 * B * M);
    alloc(&tr->dsc, 2 * B);
    alloc(&tr->lossv, B);
    alloc(&tr->loss, 1);
    alloc(&tr->dh, R * M);
    alloc(&tr->Xq, R * Dq);
    alloc(&tr->Q, R * M);
    alloc(&tr->kap, S * Dkv);
    alloc(&tr->KV, S * 2 * M);
    alloc(&tr->alpha, R * tr->H * nb);
    alloc(&tr->Xo, R * 2 * M);
    alloc(&tr->O, R * M);
    alloc(&tr->dO, R * M);
    alloc(&tr->dXo, R * 2 * M);
    alloc(&tr->dKV, S * 2 * M);
    alloc(&tr->dQ, R * M);
    alloc(&tr->dKm, S * M);
    alloc(&tr->dXq, R * M);
    alloc(&tr->ds, C * M);
    alloc(&tr->X, C * D_x);
    alloc(&tr->Hm, C * M);
    alloc(&tr->Gx, C * 3 * M);
    alloc(&tr->Gh, C * 3 * M);
    alloc(&tr->dGx, C * 3 * M);
    alloc(&tr->dGh, C * 3 * M);
    alloc(&tr->keys, n_items);
    alloc(&tr->keys_sorted, n_items);
    alloc(&tr->seg, C);
    alloc(&tr->seg_end, C);
    alloc(&tr->chunk_off, C + 1);
    alloc(&tr->ds_part, (n_items / kDsChunk + C + 1) * M);
    if (st == TGM_OK) {
        size_t bytes = 0;
        if (hipcub::DeviceRadixSort::SortKeys(nullptr, bytes, tr->keys, tr->keys_sorted,
                                              (int)n_items, 0, 64) != hipSuccess)
            st = TGM_EDEVICE;
        tr->sort_bytes = bytes;
        alloc((char **)&tr->sort_tmp, (int64_t)bytes);
    }
    if (st != TGM_OK) {
        tgm_trainer_destroy(tr);
        return st;
    }
    // the parameter vector: the model's weights and the predictor's
    hipStream_t s = as_stream(stream);
    const float *src[kNParams] = {w->W_ih, w->W_hh, w->b_ih, w->b_hh, w->W_q, w->b_q,
                                  w->W_k, w->b_k, w->W_v, w->b_v, w->W_o, w->b_o,
                                  pred->W_src, pred->W_dst, pred->b_p, pred->w_out, nullptr};
    for (int k = 0; k < kNParams && st == TGM_OK; ++k)
        if (src[k])
            st = upload(tr->p(k), src[k], sizeof(float) * (size_t)sizes[k]);
    if (st == TGM_OK)
        st = upload(tr->p(16), &pred->b_out, sizeof(float));
    if (st == TGM_OK &&
        (hipMemsetAsync(tr->m1, 0, sizeof(float) * tr->n_params, s) != hipSuccess ||
         hipMemsetAsync(tr->m2, 0, sizeof(float) * tr->n_params, s) != hipSuccess ||
         hipMemsetAsync(tr->grad, 0, sizeof(float) * tr->n_params, s) != hipSuccess ||
         hipMemsetAsync(tr->loss, 0, sizeof(float), s) != hipSuccess ||
         hipMemsetAsync(tr->seg, 0, sizeof(int32_t) * C, s) != hipSuccess ||
         hipMemsetAsync(tr->seg_end, 0, sizeof(int32_t) * C, s) != hipSuccess))
        st = TGM_EDEVICE;
    if (st == TGM_OK) {
        const int64_t n1 = std::max({S, C, R});
        hipLaunchKernelGGL(k_fill_f32, dim3((unsigned)cdiv(n1, 256)), dim3(256), 0, s, tr->ones,
                           n1, 1.f);
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess)
            st = TGM_EDEVICE;
    }
    if (st != TGM_OK) {
        tgm_trainer_destroy(tr);
        return st;
    }
    *out = tr;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_trainer_info(tgm_trainer_t tr, int64_t *n_params, int64_t *sizes,
                                         int64_t *steps)
{
    if (!tr)
        return TGM_EINVAL;
    if (n_params)
        *n_params = tr->n_params;
    if (sizes)
        for (int k = 0; k < kNParams; ++k)
            sizes[k] = tr->off[k + 1] - tr->off[k];
    if (steps)
        *steps = tr->steps;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_trainer_read(tgm_trainer_t tr, float *params, float *grad,
                                         float *loss, void *stream)
{
    if (!tr)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t bytes = sizeof(float) * (size_t)tr->n_params;
    if (params)
        TGM_HIP(hipMemcpyAsync(params, tr->theta, bytes, hipMemcpyDeviceToDevice, s));
    if (grad)
        TGM_HIP(hipMemcpyAsync(grad, tr->grad, bytes, hipMemcpyDeviceToDevice, s));
    if (loss)
        TGM_HIP(hipMemcpyAsync(loss, tr->loss, sizeof(float), hipMemcpyDeviceToDevice, s));
    return TGM_OK;
}

tgm_status_t tgm::train_step_launch(tgm_trainer_t tr, tgm_model_t m, tgm_graph_t g, int32_t b,
                                    const tgm_sample_buffers &sb, const tgm_fetch_buffers &fb,
                                    const float *mem_new, const float *h, int32_t cap,
                                    float *loss_out, hipStream_t s)
{
    if (!tr || !m || !g || tr->model != m || b < 0 || cap < 0 || !mem_new || !h)
        return TGM_EINVAL;
    if (b == 0)
        return TGM_OK;
    if (3 * b > tr->max_roots || cap > tr->max_nodes)
        return TGM_ESIZE;
    if (!sb.root_pos || !sb.root_ts || !sb.nbr_pos || !sb.eid || !sb.nts || !sb.cnt ||
        !sb.n_nodes || !fb.mem || !fb.mem_ts || !fb.mail || !fb.mail_ts || !fb.ver)
        return TGM_EINVAL;
    if (g->D_e != tr->D_e || (tr->D_e > 0 && !g->efeat))
        return TGM_EINVAL;
    const int M = tr->M, nb = tr->nb, R = 3 * b, Dq = tr->Dq, Dkv = tr->Dkv, D_x = tr->D_x;
    const int64_t S = (int64_t)R * nb;
    const float *W_ih = tr->p(0), *W_hh = tr->p(1), *b_ih = tr->p(2), *b_hh = tr->p(3);
    const float *W_q = tr->p(4), *b_q = tr->p(5), *W_k = tr->p(6), *b_k = tr->p(7);
    const float *W_v = tr->p(8), *b_v = tr->p(9), *W_o = tr->p(10), *b_o = tr->p(11);
    const float *W_src = tr->p(12), *W_dst = tr->p(13);

    // link predictor and loss
    TGM_TRY_STATUS(gemm(tr, false, true, b, M, M, h, M, W_src, M, tr->Zs, M, nullptr, false, s));
    TGM_TRY_STATUS(gemm(tr, false, true, 2 * b, M, M, h + (int64_t)b * M, M, W_dst, M, tr->Zd, M,
                        nullptr, false, s));
    PredArgs pa{b, M, tr->Zs, tr->Zd, tr->p(14), tr->p(15), tr->p(16), tr->dZsrc, tr->dZdst,
                tr->act, tr->dsc, tr->lossv};
    TGM_LAUNCH(k_pred, dim3((unsigned)cdiv((int64_t)b * kWave, 256)), dim3(256), 0, s, pa);
    TGM_LAUNCH(k_loss, dim3(1), dim3(256), 0, s, tr->lossv, b, tr->loss);
    if (loss_out)
        TGM_HIP(hipMemcpyAsync(loss_out, tr->loss, sizeof(float), hipMemcpyDeviceToDevice, s));
    // predictor gradients; the gradient of h
    TGM_TRY_STATUS(gemm(tr, true, false, 1, M, 2 * b, tr->dsc, 1, tr->act, M, tr->gr(15), M,
                        nullptr, false, s));
    TGM_TRY_STATUS(gemm(tr, true, false, 1, 1, 2 * b, tr->ones, 1, tr->dsc, 1, tr->gr(16), 1,
                        nullptr, false, s));
    TGM_TRY_STATUS(colsum(tr, b, M, tr->dZsrc, M, tr->gr(14), s));
    TGM_TRY_STATUS(gemm(tr, true, false, M, M, b, tr->dZsrc, M, h, M, tr->gr(12), M, nullptr,
                        false, s));
    TGM_TRY_STATUS(gemm(tr, true, false, M, M, 2 * b, tr->dZdst, M, h + (int64_t)b * M, M,
                        tr->gr(13), M, nullptr, false, s));
    TGM_TRY_STATUS(gemm(tr, false, false, b, M, M, tr->dZsrc, M, W_src, M, tr->dh, M, nullptr,
                        false, s));
    TGM_TRY_STATUS(gemm(tr, false, false, 2 * b, M, M, tr->dZdst, M, W_dst, M,
                        tr->dh + (int64_t)b * M, M, nullptr, false, s));

    // attention: its inputs and intermediate values again
    RowArgs ra{R, nb, M, tr->D_e, tr->D_t, sb.root_pos, sb.nbr_pos, sb.eid, sb.cnt, sb.root_ts,
               sb.nts, m->omega, m->beta, mem_new, g->efeat, tr->Xq, tr->kap};
    TGM_LAUNCH(k_att_rows, dim3((unsigned)cdiv((R + S) * kWave, 256)), dim3(256), 0, s, ra);
    TGM_TRY_STATUS(gemm(tr, false, true, R, M, Dq, tr->Xq, Dq, W_q, Dq, tr->Q, M, b_q, false, s));
    TGM_TRY_STATUS(gemm(tr, false, true, (int)S, M, Dkv, tr->kap, Dkv, W_k, Dkv, tr->KV, 2 * M,
                        b_k, false, s));
    TGM_TRY_STATUS(gemm(tr, false, true, (int)S, M, Dkv, tr->kap, Dkv, W_v, Dkv, tr->KV + M,
                        2 * M, b_v, false, s));
    CoreArgs ca{R, nb, M, tr->H, 1.f / sqrtf((float)(M / tr->H)), sb.cnt, sb.root_pos, tr->Q,
                tr->KV, mem_new, tr->dXo, tr->alpha, tr->Xo, tr->dKV, tr->dQ};
    TGM_LAUNCH(k_att_core, dim3((unsigned)cdiv((int64_t)R * kWave, 256)), dim3(256), 0, s, ca);
    TGM_TRY_STATUS(gemm(tr, false, true, R, M, 2 * M, tr->Xo, 2 * M, W_o, 2 * M, tr->O, M, b_o,
                        false, s));
    // attention backward
    TGM_LAUNCH(k_relu_mask, dim3((unsigned)cdiv((int64_t)R * M, 256)), dim3(256), 0, s, tr->dh,
               tr->O, tr->dO, (int64_t)R * M);
    TGM_TRY_STATUS(gemm(tr, true, false, M, 2 * M, R, tr->dO, M, tr->Xo, 2 * M, tr->gr(10), 2 * M,
                        nullptr, false, s));
    TGM_TRY_STATUS(colsum(tr, R, M, tr->dO, M, tr->gr(11), s));
    TGM_TRY_STATUS(gemm(tr, false, false, R, 2 * M, M, tr->dO, M, W_o, 2 * M, tr->dXo, 2 * M,
                        nullptr, false, s));
    TGM_LAUNCH(k_att_core_bwd, dim3((unsigned)cdiv((int64_t)R * kWave, 256)), dim3(256), 0, s,
               ca);
    TGM_TRY_STATUS(gemm(tr, true, false, M, Dkv, (int)S, tr->dKV, 2 * M, tr->kap, Dkv, tr->gr(6),
                        Dkv, nullptr, false, s));
    TGM_TRY_STATUS(gemm(tr, true, false, M, Dkv, (int)S, tr->dKV + M, 2 * M, tr->kap, Dkv,
                        tr->gr(8), Dkv, nullptr, false, s));
    TGM_TRY_STATUS(colsum(tr, (int)S, M, tr->dKV, 2 * M, tr->gr(7), s));
    TGM_TRY_STATUS(colsum(tr, (int)S, M, tr->dKV + M, 2 * M, tr->gr(9), s));
    TGM_TRY_STATUS(gemm(tr, true, false, M, Dq, R, tr->dQ, M, tr->Xq, Dq, tr->gr(4), Dq, nullptr,
                        false, s));
    TGM_TRY_STATUS(colsum(tr, R, M, tr->dQ, M, tr->gr(5), s));
    // gradients of the updated memories the attention read: slots, roots
    TGM_TRY_STATUS(gemm(tr, false, false, (int)S, M, M, tr->dKV, 2 * M, W_k, Dkv, tr->dKm, M,
                        nullptr, false, s));
    TGM_TRY_STATUS(gemm(tr, false, false, (int)S, M, M, tr->dKV + M, 2 * M, W_v, Dkv, tr->dKm, M,
                        nullptr, true, s));
    TGM_TRY_STATUS(gemm(tr, false, false, R, M, M, tr->dQ, M, W_q, Dq, tr->dXq, M, nullptr,
                        false, s));
    const int64_t n_items = R + S;
    TGM_LAUNCH(k_ds_keys, dim3((unsigned)cdiv(n_items, 256)), dim3(256), 0, s, R, nb,
               sb.root_pos, sb.nbr_pos, sb.cnt, tr->keys);
    size_t sort_bytes = tr->sort_bytes;
    TGM_HIP(hipcub::DeviceRadixSort::SortKeys(tr->sort_tmp, sort_bytes, tr->keys,
                                              tr->keys_sorted, (int)n_items, 0, 64, s));
    TGM_LAUNCH(k_ds_bounds, dim3((unsigned)cdiv(n_items, 256)), dim3(256), 0, s, n_items,
               tr->keys_sorted, cap, tr->seg, tr->seg_end);
    TGM_LAUNCH(k_ds_chunks, dim3(1), dim3(kDsScanThreads), 0, s, sb.n_nodes, cap, tr->seg,
               tr->seg_end, tr->chunk_off);
    TGM_LAUNCH(k_ds_partial, dim3(2048), dim3(256), 0, s, cap, M, R, n_items, tr->keys_sorted,
               tr->seg, tr->seg_end, tr->chunk_off, tr->dXq, tr->dXo, tr->dKm, tr->ds_part);
    TGM_LAUNCH(k_ds, dim3((unsigned)cdiv((int64_t)cap * kWave, 256)), dim3(256), 0, s,
               sb.n_nodes, cap, M, tr->chunk_off, tr->ds_part, tr->ds);

    // memory updater (GRU) backward
    GruRowArgs gra{sb.n_nodes, cap, M, tr->D_m, tr->D_t, fb.mem, fb.mail, fb.mem_ts, fb.mail_ts,
                   m->omega, m->beta, fb.ver, tr->X, tr->Hm};
    TGM_LAUNCH(k_gru_rows, dim3((unsigned)cdiv((int64_t)cap * kWave, 256)), dim3(256), 0, s,
               gra);
    TGM_TRY_STATUS(gemm(tr, false, true, cap, 3 * M, D_x, tr->X, D_x, W_ih, D_x, tr->Gx, 3 * M,
                        b_ih, false, s));
    TGM_TRY_STATUS(gemm(tr, false, true, cap, 3 * M, M, tr->Hm, M, W_hh, M, tr->Gh, 3 * M, b_hh,
                        false, s));
    TGM_LAUNCH(k_gru_bwd, dim3((unsigned)cdiv((int64_t)cap * M, 256)), dim3(256), 0, s,
               sb.n_nodes, cap, M, fb.ver, tr->Gx, tr->Gh, tr->Hm, tr->ds, tr->dGx, tr->dGh);
    TGM_TRY_STATUS(gemm(tr, true, false, 3 * M, D_x, cap, tr->dGx, 3 * M, tr->X, D_x, tr->gr(0),
                        D_x, nullptr, false, s));
    TGM_TRY_STATUS(gemm(tr, true, false, 3 * M, M, cap, tr->dGh, 3 * M, tr->Hm, M, tr->gr(1), M,
                        nullptr, false, s));
    TGM_TRY_STATUS(colsum(tr, cap, 3 * M, tr->dGx, 3 * M, tr->gr(2), s));
    TGM_TRY_STATUS(colsum(tr, cap, 3 * M, tr->dGh, 3 * M, tr->gr(3), s));

    // optimizer step, then the model's packed operands from the new weights
    tr->steps++;
    const int64_t n = tr->n_params;
    if (tr->opt == TGM_OPT_SGD) {
        TGM_LAUNCH(k_sgd, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, tr->theta, tr->grad, n,
                   tr->lr);
    } else {
        const double c1 = 1.0 - std::pow((double)tr->beta1, (double)tr->steps);
        const double c2 = 1.0 - std::pow((double)tr->beta2, (double)tr->steps);
        TGM_LAUNCH(k_adam, dim3((unsigned)cdiv(n, 256)), dim3(256), 0, s, tr->theta, tr->grad,
                   tr->m1, tr->m2, n, tr->lr, tr->beta1, tr->beta2, tr->eps, (float)c1,
                   (float)c2);
    }
    ModelParams mp{W_ih, W_hh, b_ih, b_hh, W_q, b_q, W_k, b_k, W_v, b_v, W_o, b_o};
    return model_repack(m, mp, s);
}

extern "C" tgm_status_t tgm_train_step(tgm_trainer_t tr, tgm_model_t m, tgm_graph_t g, int32_t b,
                                       const tgm_sample_buffers *sb, const tgm_fetch_buffers *fb,
                                       const float *mem_new, const float *h, int32_t cap,
                                       float *loss, void *stream)
{
    if (!sb || !fb)
        return TGM_EINVAL;
    return tgm::train_step_launch(tr, m, g, b, *sb, *fb, mem_new, h, cap, loss,
                                  as_stream(stream));
}

extern "C" tgm_status_t tgm_state_set_training(tgm_state_t st, tgm_trainer_t tr, float *loss_log,
                                               int64_t log_len)
{
    if (!st || (tr && loss_log && log_len < 1))
        return TGM_EINVAL;
    st->trainer = tr;
    st->loss_log = tr ? loss_log : nullptr;
    st->loss_log_len = tr && loss_log ? log_len : 0;
    return TGM_OK;
}
