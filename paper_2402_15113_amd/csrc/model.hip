// Memory update (GRU + latest-message reduce + staged write-back) and the
// attention embedding.  The dense contractions run on fp32 MFMA
// (v_mfma_f32_16x16x4_f32); everything else is vector code.
#include <cmath>

#include "common.h"

using namespace tgm;

namespace {

constexpr int kMaxWaves = 8;
constexpr int kAttMaxCB = 2;   // K|V column blocks per wave
constexpr int kAttMaxRB = 5;   // 16-row slot blocks per workgroup

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + expf(-x)); }

// ------------------------------------------------------------------ GRU
// One workgroup per 16 node-set rows, one wavefront per 16-wide block of
// hidden units (round-robin when there are more blocks than waves).  The
// rows' GRU inputs [mail || phi(mail_ts - mem_ts) | mem] are staged once in
// LDS; each wave accumulates the four gate pre-activations of its hidden
// block (r and z over [x | h]; n split into its x part and its h part, which
// the reset gate scales) and applies the gates in registers.
// Also resets the latest-message slots of its rows (consumed next by k_latest).
__global__ __launch_bounds__(512) void k_gru(
    const int32_t *__restrict__ n_nodes, const float *__restrict__ mem,
    const double *__restrict__ mem_ts, const float *__restrict__ mail,
    const double *__restrict__ mail_ts, const int32_t *__restrict__ ver,
    const f4 *__restrict__ bx, const f4 *__restrict__ bh, const float *__restrict__ bias,
    const double *__restrict__ omega, const double *__restrict__ beta, int M, int D_m, int D_t,
    int KXC, int KHC, int MB, float *__restrict__ mem_new, double *__restrict__ new_mem_ts,
    int32_t *__restrict__ win)
{
    extern __shared__ float lds[];
    __shared__ int s_has[16];
    const int n = *n_nodes;
    const int row0 = blockIdx.x * 16;
    if (row0 >= n)
        return;
    const int KX = KXC * 16, KH = KHC * 16;
    const int SA = KX + KH + 4;
    const int nw = blockDim.x >> 6;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    for (int rr = wave; rr < 16; rr += nw) {
        const int p = row0 + rr;
        float *a = lds + rr * SA;
        if (p < n) {
            const bool has = ver[p] >= 0;
            if (lane == 0) {
                s_has[rr] = has;
                win[p] = -1;
            }
            for (int k = lane; k < KH; k += kWave)
                a[KX + k] = k < M ? mem[(int64_t)p * M + k] : 0.f;
            if (has) {
                for (int k = lane; k < D_m; k += kWave)
                    a[k] = mail[(int64_t)p * D_m + k];
                const double dt = mail_ts[p] - mem_ts[p];
                for (int d = lane; d < D_t; d += kWave)
                    a[D_m + d] = time_enc(omega[d], beta[d], dt);
                for (int k = D_m + D_t + lane; k < KX; k += kWave)
                    a[k] = 0.f;
            } else {
                for (int k = lane; k < KX; k += kWave)
                    a[k] = 0.f;
            }
        } else {
            if (lane == 0)
                s_has[rr] = 0;
            for (int k = lane; k < KX + KH; k += kWave)
                a[k] = 0.f;
        }
    }
    __syncthreads();

    const float *arow = lds + (lane & 15) * SA + 4 * (lane >> 4);
    const int64_t gx = (int64_t)KXC * MB * kWave;   // stride between gates in bx
    const int64_t gh = (int64_t)KHC * MB * kWave;
    for (int hb = wave; hb < MB; hb += nw) {
        f4 ar = {0, 0, 0, 0}, az = ar, anx = ar, anh = ar;
        const f4 *px = bx + (int64_t)hb * kWave + lane;
        for (int kc = 0; kc < KXC; ++kc) {
            const f4 a = *reinterpret_cast<const f4 *>(arow + kc * 16);
            const f4 b0 = px[0], b1 = px[gx], b2 = px[2 * gx];
            px += (int64_t)MB * kWave;
            ar = mfma_k16(a, b0, ar);
            az = mfma_k16(a, b1, az);
            anx = mfma_k16(a, b2, anx);
        }
        const f4 *ph = bh + (int64_t)hb * kWave + lane;
        for (int kc = 0; kc < KHC; ++kc) {
            const f4 a = *reinterpret_cast<const f4 *>(arow + KX + kc * 16);
            const f4 b0 = ph[0], b1 = ph[gh], b2 = ph[2 * gh];
            ph += (int64_t)MB * kWave;
            ar = mfma_k16(a, b0, ar);
            az = mfma_k16(a, b1, az);
            anh = mfma_k16(a, b2, anh);
        }
        const int col = hb * 16 + (lane & 15);
        if (col < M) {
            const int MP = MB * 16;
            const float br = bias[col], bz = bias[MP + col], bin = bias[2 * MP + col],
                        bhn = bias[3 * MP + col];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int rr = 4 * (lane >> 4) + v;
                const int p = row0 + rr;
                if (p < n) {
                    const float h = lds[rr * SA + KX + col];
                    float o = h;
                    if (s_has[rr]) {
                        const float r = sigmoidf_(ar[v] + br);
                        const float z = sigmoidf_(az[v] + bz);
                        const float nn = tanhf(anx[v] + bin + r * (anh[v] + bhn));
                        o = (1.0f - z) * nn + z * h;
                    }
                    mem_new[(int64_t)p * M + col] = o;
                }
            }
        }
    }
    if (new_mem_ts && threadIdx.x < 16) {
        const int p = row0 + threadIdx.x;
        if (p < n)
            new_mem_ts[p] = s_has[threadIdx.x] ? mail_ts[p] : mem_ts[p];
    }
}

// Latest-message reduce.  Candidate c = 2 (e - first) + role is the message
// of event first + c/2 to its source (role 0) or destination (role 1).  The
// stream is sorted by (t, e), so the candidate order is the (t, e, role)
// order and the latest message of a node is its largest c: an integer max,
// exact and order-independent.  Candidates of one wavefront that hit the same
// node are first reduced with lane shuffles (the wave's candidates are
// consecutive, so a node's last lane in the wave holds its wave maximum); only
// that lane issues the atomic.
__global__ __launch_bounds__(256) void k_latest(int32_t n_cand, const int32_t *__restrict__ n_nodes,
                                                const int32_t *__restrict__ src_pos,
                                                const int32_t *__restrict__ dst_pos,
                                                int32_t *__restrict__ win)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    const int lane = threadIdx.x & 63;
    const int n = *n_nodes;
    int p = c < n_cand ? ((c & 1) ? dst_pos[c >> 1] : src_pos[c >> 1]) : -1;
    const bool live = p >= 0 && p < n;   // positions outside the node set are dropped
    if (!live)
        p = -1 - lane;
    // is there a later lane in this wave with the same position?
    bool later = false;
    for (int o = 1; o < kWave; ++o) {
        const int q = __shfl(p, (lane + o) & 63, kWave);
        later |= (lane + o < kWave) && q == p;
    }
    if (live && !later)
        atomicMax(&win[p], c);
}

// Stage the write set of one iteration: one wavefront per candidate; the
// winning candidate of its node writes the node's new memory, its message
// [s'_self || s'_other || efeat[e]] and the timestamps.
__global__ __launch_bounds__(256) void k_stage(
    int32_t n_cand, const int32_t *__restrict__ n_nodes, int64_t first, int M, int D_m, int D_e,
    const int32_t *__restrict__ src,
    const int32_t *__restrict__ dst, const double *__restrict__ t,
    const float *__restrict__ efeat, const int32_t *__restrict__ src_pos,
    const int32_t *__restrict__ dst_pos, const int32_t *__restrict__ win,
    const float *__restrict__ mem_new, const int32_t *__restrict__ ver,
    const double *__restrict__ mem_ts, const double *__restrict__ mail_ts,
    int32_t *__restrict__ r_flag, int32_t *__restrict__ r_node, float *__restrict__ r_mem,
    double *__restrict__ r_mem_ts, float *__restrict__ r_mail, double *__restrict__ r_mail_ts)
{
    const int c = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (c >= n_cand)
        return;
    const int k = c >> 1, role = c & 1;
    const int n = *n_nodes;
    const int p = role ? dst_pos[k] : src_pos[k];
    const int q = role ? src_pos[k] : dst_pos[k];
    if (p < 0 || p >= n || q < 0 || q >= n || win[p] != c) {
        if (lane == 0)
            r_flag[c] = 0;
        return;
    }
    const int64_t e = first + k;
    const float *sp = mem_new + (int64_t)p * M;
    float *ml = r_mail + (int64_t)c * D_m;
    wave_copy_row(r_mem + (int64_t)c * M, sp, M, lane);
    wave_copy_row(ml, sp, M, lane);
    wave_copy_row(ml + M, mem_new + (int64_t)q * M, M, lane);
    if (D_e > 0)
        wave_copy_row(ml + 2 * M, efeat + e * D_e, D_e, lane);
    if (lane == 0) {
        r_flag[c] = 1;
        r_node[c] = role ? dst[e] : src[e];
        r_mem_ts[c] = ver[p] >= 0 ? mail_ts[p] : mem_ts[p];
        r_mail_ts[c] = t[e];
    }
}

__global__ void k_winner_out(const int32_t *__restrict__ n_nodes, int32_t cap, int64_t first,
                             const int32_t *__restrict__ win, int64_t *__restrict__ winner)
{
    const int p = blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= cap || p >= *n_nodes)
        return;
    const int32_t c = win[p];
    winner[p] = c >= 0 ? 2 * first + c : -1;
}

// ------------------------------------------------------------------ embed
// Node projections P[p] = s'_p [W_q^s; W_k^s; W_v^s]^T: the memory part of the
// query, key and value projections depends only on the node, so it is
// computed once per node of the set instead of once per slot.
__global__ __launch_bounds__(512) void k_node_proj(const int32_t *__restrict__ n_nodes,
                                                   const float *__restrict__ mem_new, int M,
                                                   int PC, const f4 *__restrict__ pb, int PNB,
                                                   float *__restrict__ P)
{
    extern __shared__ float lds[];
    const int n = *n_nodes;
    const int row0 = blockIdx.x * 16;
    if (row0 >= n)
        return;
    const int K = PC * 16, SA = K + 4, ldP = PNB * 16;
    const int nw = blockDim.x >> 6;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (int rr = wave; rr < 16; rr += nw) {
        const int p = row0 + rr;
        for (int k = lane; k < K; k += kWave)
            lds[rr * SA + k] = (p < n && k < M) ? mem_new[(int64_t)p * M + k] : 0.f;
    }
    __syncthreads();
    const float *arow = lds + (lane & 15) * SA + 4 * (lane >> 4);
    for (int cb = wave; cb < PNB; cb += nw) {
        f4 acc = {0, 0, 0, 0};
        const f4 *pp = pb + (int64_t)cb * kWave + lane;
        for (int kc = 0; kc < PC; ++kc) {
            acc = mfma_k16(*reinterpret_cast<const f4 *>(arow + kc * 16), *pp, acc);
            pp += (int64_t)PNB * kWave;
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int p = row0 + 4 * (lane >> 4) + v;
            if (p < n)
                P[(int64_t)p * ldP + cb * 16 + (lane & 15)] = acc[v];
        }
    }
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
    const float *b_k, *b_v, *c_q;
    const f4 *out_b;
    int OC, ONB;
    const float *b_o;
    const float *mem_new;
    float *h;
};

// Attention embedding of RT roots per workgroup (their RT*nb slots fill RBa
// 16-row MFMA blocks):
//  1. stage each slot's [efeat[eid] || phi(t_root - t_slot)] row in LDS;
//  2. one MFMA GEMM gives the per-slot part of K and V for all heads;
//  3. add the node projections of the neighbour and the biases (K, V back to
//     LDS); q = P_q[root] + (W_q^t phi(0) + b_q);
//  4. one wavefront per (root, head): scores, softmax, weighted sum of V;
//  5. the output projection ReLU(W_o [a || s'_v] + b_o) as a second MFMA GEMM.
__global__ __launch_bounds__(512) void k_attn(AttnArgs g)
{
    extern __shared__ float lds[];
    const int r0 = blockIdx.x * g.RT;
    const int nroots = min(g.RT, g.R - r0);
    if (nroots <= 0)
        return;
    const int M = g.M, nb = g.nb, D_e = g.D_e, D_t = g.D_t;
    const int n = *g.n_nodes;   // positions and event ids are bounds-checked
    const int RA = g.RBa * 16;
    const int KF = g.KFC * 16, SA = KF + 4;
    const int SKV = g.KVNB * 16 + 4;
    const int ORB = (g.RT + 15) / 16;
    const int SAO = g.OC * 16 + 4;
    float *A = lds;                                   // [RA][SA], then K|V [RA][SKV]
    float *Q = lds + RA * (SA > SKV ? SA : SKV);      // [RT][M]
    float *AO = Q + g.RT * M;                         // [ORB*16][SAO]: [a || s'_v]
    const int nw = blockDim.x >> 6;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    // 1. slot rows
    for (int sr = wave; sr < RA; sr += nw) {
        float *row = A + sr * SA;
        const int r = sr / nb, j = sr - r * nb;
        const bool valid = r < nroots && j < g.cnt[r0 + r];
        if (valid) {
            const int64_t sl = (int64_t)(r0 + r) * nb + j;
            const int64_t e = g.eid[sl];
            if (D_e > 0 && e >= 0 && e < g.E)
                wave_copy_row(row, g.efeat + e * D_e, D_e, lane);
            else
                for (int k = lane; k < D_e; k += kWave)
                    row[k] = 0.f;
            const double dt = g.root_ts[r0 + r] - g.nts[sl];
            for (int d = lane; d < D_t; d += kWave)
                row[D_e + d] = time_enc(g.omega[d], g.beta[d], dt);
            for (int k = D_e + D_t + lane; k < KF; k += kWave)
                row[k] = 0.f;
        } else {
            for (int k = lane; k < KF; k += kWave)
                row[k] = 0.f;
        }
    }
    // query rows and the s'_v half of the output-projection input
    for (int r = wave; r < ORB * 16; r += nw) {
        float *ao = AO + r * SAO;
        const int pv = r < nroots ? g.root_pos[r0 + r] : -1;
        const bool ok = pv >= 0 && pv < n;
        const float *pq = g.P + (int64_t)(ok ? pv : 0) * g.ldP;
        const float *sv = g.mem_new + (int64_t)(ok ? pv : 0) * M;
        for (int k = lane; k < M; k += kWave) {
            if (r < g.RT)
                Q[r * M + k] = (ok ? pq[k] : 0.f) + g.c_q[k];
            ao[M + k] = ok ? sv[k] : 0.f;
            if (r >= nroots)
                ao[k] = 0.f;
        }
        for (int k = 2 * M + lane; k < g.OC * 16; k += kWave)
            ao[k] = 0.f;
    }
    __syncthreads();

    // 2. per-slot K|V GEMM; wave w owns column blocks w and w + nw (at most
    //    kMaxCB blocks per wave; all indices below are compile-time so the
    //    accumulators stay in registers)
    f4 acc[kAttMaxCB][kAttMaxRB];
    const float *arow = A + (lane & 15) * SA + 4 * (lane >> 4);
#pragma unroll
    for (int i = 0; i < kAttMaxCB; ++i) {
        const int cb = wave + i * nw;
#pragma unroll
        for (int rb = 0; rb < kAttMaxRB; ++rb)
            acc[i][rb] = f4{0, 0, 0, 0};
        if (cb < g.KVNB) {
            const f4 *pb = g.kv_b + (int64_t)cb * kWave + lane;
            for (int kc = 0; kc < g.KFC; ++kc) {
                const f4 b = *pb;
                pb += (int64_t)g.KVNB * kWave;
#pragma unroll
                for (int rb = 0; rb < kAttMaxRB; ++rb)
                    if (rb < g.RBa)
                        acc[i][rb] = mfma_k16(
                            *reinterpret_cast<const f4 *>(arow + rb * 16 * SA + kc * 16), b,
                            acc[i][rb]);
            }
        }
    }
    __syncthreads();   // every read of the slot rows is done

    // 3. K | V rows: per-slot part + node projection of the neighbour + bias.
    //    Column col < M is K, col in [M, 2M) is V; both sit at P[M + col].
    float *KV = A;
#pragma unroll
    for (int i = 0; i < kAttMaxCB; ++i) {
        const int cb = wave + i * nw;
        const int col = cb * 16 + (lane & 15);
        if (cb < g.KVNB && col < 2 * M) {
            const float bias = col < M ? g.b_k[col] : g.b_v[col - M];
#pragma unroll
            for (int rb = 0; rb < kAttMaxRB; ++rb) {
                if (rb < g.RBa) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int row = rb * 16 + 4 * (lane >> 4) + v;
                        const int r = row / nb, j = row - r * nb;
                        if (r < nroots && j < g.cnt[r0 + r]) {
                            const int np = g.nbr_pos[(int64_t)(r0 + r) * nb + j];
                            const float pk =
                                (np >= 0 && np < n) ? g.P[(int64_t)np * g.ldP + M + col] : 0.f;
                            KV[row * SKV + col] = acc[i][rb][v] + bias + pk;
                        }
                    }
                }
            }
        }
    }
    __syncthreads();

    // 4. per (root, head) attention; head width d_h <= 128
    const int d_h = M / g.H;
    const float scale = 1.0f / sqrtf((float)d_h);
    for (int task = wave; task < nroots * g.H; task += nw) {
        const int r = task / g.H, eta = task - r * g.H;
        const int c = g.cnt[r0 + r];
        const int o = eta * d_h;
        const float *qr = Q + r * M + o;
        float *ao = AO + r * SAO + o;
        // lane j keeps score j
        float my_s = -INFINITY;
        for (int j = 0; j < c; ++j) {
            const float *kr = KV + (r * nb + j) * SKV + o;
            float part = 0.f;
            if (lane < d_h)
                part = qr[lane] * kr[lane];
            if (lane + kWave < d_h)
                part += qr[lane + kWave] * kr[lane + kWave];
            const float sj = wave_sum(part) * scale;
            if (lane == j)
                my_s = sj;
        }
        float mx = my_s;
#pragma unroll
        for (int sh = 32; sh > 0; sh >>= 1)
            mx = fmaxf(mx, __shfl_xor(mx, sh, kWave));
        const float ex = lane < c ? expf(my_s - mx) : 0.f;
        const float den = wave_sum(ex);
        const float alpha = c > 0 ? ex / den : 0.f;
        float a0 = 0.f, a1 = 0.f;
        for (int j = 0; j < c; ++j) {
            const float al = __shfl(alpha, j, kWave);
            const float *vr = KV + (r * nb + j) * SKV + M + o;
            if (lane < d_h)
                a0 += al * vr[lane];
            if (lane + kWave < d_h)
                a1 += al * vr[lane + kWave];
        }
        if (lane < d_h)
            ao[lane] = a0;
        if (lane + kWave < d_h)
            ao[lane + kWave] = a1;
    }
    __syncthreads();

    // 5. h = ReLU(W_o [a || s'_v] + b_o)
    const float *orow = AO + (lane & 15) * SAO + 4 * (lane >> 4);
    for (int cb = wave; cb < g.ONB; cb += nw) {
        for (int orb = 0; orb < ORB; ++orb) {
            f4 ac = {0, 0, 0, 0};
            const f4 *pb = g.out_b + (int64_t)cb * kWave + lane;
            for (int kc = 0; kc < g.OC; ++kc) {
                ac = mfma_k16(*reinterpret_cast<const f4 *>(orow + orb * 16 * SAO + kc * 16), *pb,
                              ac);
                pb += (int64_t)g.ONB * kWave;
            }
            const int col = cb * 16 + (lane & 15);
            if (col < M) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int r = orb * 16 + 4 * (lane >> 4) + v;
                    if (r < nroots)
                        g.h[(int64_t)(r0 + r) * M + col] = fmaxf(ac[v] + g.b_o[col], 0.f);
                }
            }
        }
    }
}

// q bias folded at creation: c_q = W_q^t phi(0) + b_q with phi(0)_d = cos(beta_d).
__global__ void k_fold_q_bias(int M, int D_t, const float *__restrict__ W_q,
                              const float *__restrict__ b_q, const double *__restrict__ beta,
                              float *__restrict__ c_q)
{
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= M)
        return;
    double acc = b_q[k];
    for (int d = 0; d < D_t; ++d)
        acc += (double)W_q[(int64_t)k * (M + D_t) + M + d] * cos(beta[d]);
    c_q[k] = (float)acc;
}

int waves_for(int blocks) { return blocks < kMaxWaves ? (blocks < 1 ? 1 : blocks) : kMaxWaves; }

size_t gru_lds(const tgm_model *m) { return sizeof(float) * 16 * ((m->KXC + m->KHC) * 16 + 4); }
size_t proj_lds(const tgm_model *m) { return sizeof(float) * 16 * (m->PC * 16 + 4); }

int attn_roots(const tgm_model *m, int *RBa)
{
    // slots of RT roots fill at most 5 MFMA row blocks
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
    return sizeof(float) * ((size_t)RA * (SA > SKV ? SA : SKV) + (size_t)RT * m->M +
                            (size_t)ORB * 16 * (m->OC * 16 + 4));
}

}  // namespace

// ======================================================================== API

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
    hipFree(m->b_k);
    hipFree(m->b_v);
    hipFree(m->c_q);
    hipFree(m->out_b);
    hipFree(m->b_o);
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
    // wavefront slots (M <= 128) and a head is at most two lanes wide per lane
    if (M <= 0 || D_e < 0 || D_t < 0 || H <= 0 || M % H != 0 || nb < 1 || nb > 64 ||
        d->max_nodes <= 0 || d->max_roots < 0 || 2 * M > 16 * kMaxWaves * kAttMaxCB ||
        M / H > 2 * kWave)
        return TGM_EINVAL;
    if (!w->W_ih || !w->W_hh || !w->b_ih || !w->b_hh || (D_t > 0 && (!w->omega || !w->beta)) ||
        !w->W_q || !w->b_q || !w->W_k || !w->b_k || !w->W_v || !w->b_v || !w->W_o || !w->b_o)
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
            wkv[(size_t)n * KF + k] = w->W_k[(size_t)n * Dkv + M + k];
            wkv[(size_t)(M + n) * KF + k] = w->W_v[(size_t)n * Dkv + M + k];
        }
    auto kvb = pack_b(wkv.data(), 2 * M, KF, 0, KF, m->KFC, m->KVNB);
    auto ob = pack_b(w->W_o, M, 2 * M, 0, 2 * M, m->OC, m->ONB);

    float *wq_dev = nullptr;
    tgm_status_t st = TGM_OK;
    do {
        auto alloc = [&](void **p, size_t bytes) {
            return hipMalloc(p, bytes ? bytes : 16) == hipSuccess;
        };
        if (!alloc((void **)&m->gru_bx, bx.size() * 4) || !alloc((void **)&m->gru_bh, bh.size() * 4) ||
            !alloc((void **)&m->gru_bias, bias.size() * 4) ||
            !alloc((void **)&m->omega, sizeof(double) * D_t) ||
            !alloc((void **)&m->beta, sizeof(double) * D_t) ||
            !alloc((void **)&m->proj_b, pb.size() * 4) ||
            !alloc((void **)&m->P, sizeof(float) * (size_t)d->max_nodes * m->PNB * 16) ||
            !alloc((void **)&m->kv_b, kvb.size() * 4) || !alloc((void **)&m->b_k, 4 * M) ||
            !alloc((void **)&m->b_v, 4 * M) || !alloc((void **)&m->c_q, 4 * M) ||
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
        if ((st = upload(m->b_k, w->b_k, 4 * M)) != TGM_OK) break;
        if ((st = upload(m->b_v, w->b_v, 4 * M)) != TGM_OK) break;
        if ((st = upload(m->out_b, ob.data(), ob.size() * 4)) != TGM_OK) break;
        if ((st = upload(m->b_o, w->b_o, 4 * M)) != TGM_OK) break;
        if ((st = upload(wq_dev, w->W_q, sizeof(float) * (size_t)M * Dq)) != TGM_OK) break;
        float *bq_dev = m->c_q;   // b_q staged in c_q, folded in place
        if ((st = upload(bq_dev, w->b_q, 4 * M)) != TGM_OK) break;
        hipLaunchKernelGGL(k_fold_q_bias, dim3(cdiv(M, 64)), dim3(64), 0, s, M, D_t, wq_dev,
                           bq_dev, m->beta, m->c_q);
        if (hipGetLastError() != hipSuccess || hipStreamSynchronize(s) != hipSuccess) {
            st = TGM_EDEVICE;
            break;
        }
        // large LDS footprints need an explicit opt-in
        if (hipFuncSetAttribute((const void *)k_gru, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)gru_lds(m)) != hipSuccess ||
            hipFuncSetAttribute((const void *)k_node_proj,
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)proj_lds(m)) != hipSuccess ||
            hipFuncSetAttribute((const void *)k_attn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)attn_lds(m)) != hipSuccess) {
            st = TGM_EINVAL;   // dimensions beyond the LDS of one workgroup
            break;
        }
    } while (0);
    hipFree(wq_dev);
    if (st != TGM_OK) {
        tgm_model_destroy(m);
        return st;
    }
    *out = m;
    return TGM_OK;
}

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
    if (!st || !m || !g || !n_nodes || cap < 0 || b < 0 || first_event < 0 ||
        first_event + b > g->E)
        return TGM_EINVAL;
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
    hipStream_t s = as_stream(stream);
    if (cap > 0) {
        const int nw = waves_for(m->MB);
        TGM_LAUNCH(k_gru, dim3(cdiv(cap, 16)), dim3(64 * nw), gru_lds(m), s, n_nodes, mem,
                           mem_ts, mail, mail_ts, ver, m->gru_bx, m->gru_bh, m->gru_bias,
                           m->omega, m->beta, m->M, m->D_m, m->D_t, m->KXC, m->KHC, m->MB,
                           mem_new, new_mem_ts, st->win);
    }
    const int n_cand = 2 * b;
    const size_t base = (size_t)(iter % slots) * st->ring_rows();
    if (n_cand > 0) {
        TGM_LAUNCH(k_latest, dim3(cdiv(n_cand, 256)), dim3(256), 0, s, n_cand, n_nodes,
                           src_pos, dst_pos, st->win);
        TGM_LAUNCH(k_stage, dim3(cdiv(n_cand, 4)), dim3(256), 0, s, n_cand, n_nodes,
                           first_event,
                           m->M, m->D_m, m->D_e, g->src, g->dst, g->t, g->efeat, src_pos, dst_pos,
                           st->win, mem_new, ver, mem_ts, mail_ts, st->r_flag + base,
                           st->r_node + base, st->r_mem + base * st->M, st->r_mem_ts + base,
                           st->r_mail + base * st->D_m, st->r_mail_ts + base);
    }
    if (winner && cap > 0) {
        TGM_LAUNCH(k_winner_out, dim3(cdiv(cap, 256)), dim3(256), 0, s, n_nodes, cap,
                           first_event, st->win, winner);
    }
    tgm_state::Slot &sl = st->ring[iter % slots];
    sl.iter = iter;
    sl.b = b;
    sl.staged = true;
    st->staged_through = iter;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_embed(tgm_model_t m, tgm_graph_t g, int32_t R, int32_t nb,
                                  const int32_t *root_pos, const double *root_ts,
                                  const int32_t *nbr_pos, const int32_t *eid, const double *nts,
                                  const int32_t *cnt, const float *mem_new,
                                  const int32_t *n_nodes, int32_t cap, float *h, void *stream)
{
    if (!m || !g || R < 0 || nb != m->nb || !n_nodes || cap < 0 || g->D_e != m->D_e)
        return TGM_EINVAL;
    if (R > m->max_roots || cap > m->max_nodes)
        return TGM_ESIZE;
    if (R == 0)
        return TGM_OK;
    if (!root_pos || !root_ts || !nbr_pos || !eid || !nts || !cnt || !mem_new || !h || cap == 0)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    TGM_LAUNCH(k_node_proj, dim3(cdiv(cap, 16)), dim3(64 * waves_for(m->PNB)),
                       proj_lds(m), s, n_nodes, mem_new, m->M, m->PC, m->proj_b, m->PNB, m->P);
    AttnArgs a;
    a.R = R; a.nb = nb; a.RT = attn_roots(m, &a.RBa); a.M = m->M; a.H = m->H;
    a.E = g->E; a.n_nodes = n_nodes;
    a.D_e = m->D_e; a.D_t = m->D_t;
    a.root_pos = root_pos; a.nbr_pos = nbr_pos; a.eid = eid; a.cnt = cnt;
    a.root_ts = root_ts; a.nts = nts;
    a.P = m->P; a.ldP = m->PNB * 16;
    a.efeat = g->efeat; a.omega = m->omega; a.beta = m->beta;
    a.kv_b = m->kv_b; a.KFC = m->KFC; a.KVNB = m->KVNB;
    a.b_k = m->b_k; a.b_v = m->b_v; a.c_q = m->c_q;
    a.out_b = m->out_b; a.OC = m->OC; a.ONB = m->ONB; a.b_o = m->b_o;
    a.mem_new = mem_new; a.h = h;
    TGM_LAUNCH(k_attn, dim3(cdiv(R, a.RT)), dim3(64 * kMaxWaves), attn_lds(m), s, a);
    return TGM_OK;
}
