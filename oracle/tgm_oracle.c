/*
 * tgm_oracle.c -- plain fp64 CPU oracle for the per-batch memory-module stage
 * of memory-based temporal GNN training, as pipelined by MSPipe (Sheng, Su,
 * Huang, Wu; KDD'24, arXiv 2402.15113).
 *
 * TEST INFRASTRUCTURE.  This file is the yardstick the GPU library is checked
 * against; it is not part of the product.  Only the test-suite, the smoke check
 * and the CPU-baseline leg of the benchmark load it.  It shares no code, header,
 * table or helper with the HIP path.
 *
 * What it computes, step by step, for iteration i (batch of events
 * [iB, min(E,(i+1)B)) ):
 *   0. snapshot: the node state with the write sets of iterations <= i-1-s
 *      applied in order (Eq. 2 of Sec. 3.1 with the paper's k = s + 1;
 *      iterations before the first write set see the initial state, the
 *      warm-up rule of Appendix D, Algorithm 1);
 *   1. roots: source, destination and negative of every event, at its time;
 *   2. most-recent-nb temporal neighbours of each root, strictly earlier events
 *      only (Sec. 5 training settings; Appendix D.1);
 *   3. node set U = sorted unique(roots + sampled neighbours) and its state;
 *   3b. (optional, MSPipe-S, Sec. 3.3) staleness mitigation of the fetched
 *      memories of nodes whose last update lies further back than the
 *      p-quantile of the batch's gaps: a blend with the mean memory of the
 *      most similar (common neighbours) fresher nodes;
 *   4. memory update s' = GRU(mail || phi(mail_ts - mem_ts), mem) for nodes
 *      with mail (mem() of Eq. 1; Delta-t as defined under Eq. 1); for the
 *      JODIE model family an RNN cell takes the GRU's place;
 *   5. embedding h = emb(s'_v, s'_u | u in N(v)): one layer of multi-head
 *      scaled dot-product attention with a cosine time encoding (emb() of
 *      Eq. 1, "a single layer GAT"); for JODIE the time projection
 *      h = s'_v * (1 + w_t (t - ts'_v)) of the node's memory instead;
 *   6. messages m = msg(s'_v, s'_u, y_uv(t)) as identity concatenation (msg()
 *      of Eq. 1);
 *   7. latest-message reduce: one message per node, the one with the largest
 *      (t, e, role), role src = 0 < dst = 1;
 *   8. write set W_i of the positive endpoints, queued until iteration i+1+s.
 *
 * Everything floating is fp64; fp32 inputs (edge features, weights) are widened
 * exactly.  Parallel loops (OpenMP) run over independent nodes or roots only;
 * every dot product is summed in a fixed order, so results do not depend on the
 * thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_EEND (-2)

/* model families (Sec. 5 trains TGN, JODIE and APAN) */
#define ORC_TGN 0
#define ORC_JODIE 1
#define ORC_APAN 2

/* ------------------------------------------------------------------------- */
/* Time encoding: phi(dt)_d = cos(omega_d * dt + beta_d), the cosine functional
 * time encoding the paper's models inherit (TGAT, Xu et al. 2020), applied to
 * the time gaps Delta-t of Eq. 1.  omega and beta are inputs.                */
void orc_time_encode(int D_t, const double *omega, const double *beta,
                     double dt, double *out)
{
    for (int d = 0; d < D_t; ++d)
        out[d] = cos(omega[d] * dt + beta[d]);
}

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* ------------------------------------------------------------------------- */
/* Memory updater mem() of Eq. 1: the GRU cell (Cho et al. 2014).
 *   r = sig(W_ir x + b_ir + W_hr h + b_hr)
 *   z = sig(W_iz x + b_iz + W_hz h + b_hz)
 *   n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
 *   h' = (1 - z) * n + z * h
 * W_ih is [3M x D_x] and W_hh is [3M x M], row blocks in gate order r, z, n. */
void orc_gru_cell(int M, int D_x, const double *W_ih, const double *W_hh,
                  const double *b_ih, const double *b_hh,
                  const double *x, const double *h, double *out)
{
    for (int j = 0; j < M; ++j) {
        double ir = b_ih[j], iz = b_ih[M + j], in_ = b_ih[2 * M + j];
        double hr = b_hh[j], hz = b_hh[M + j], hn = b_hh[2 * M + j];
        const double *wr = W_ih + (size_t)j * D_x;
        const double *wz = W_ih + (size_t)(M + j) * D_x;
        const double *wn = W_ih + (size_t)(2 * M + j) * D_x;
        for (int k = 0; k < D_x; ++k) {
            ir += wr[k] * x[k];
            iz += wz[k] * x[k];
            in_ += wn[k] * x[k];
        }
        const double *ur = W_hh + (size_t)j * M;
        const double *uz = W_hh + (size_t)(M + j) * M;
        const double *un = W_hh + (size_t)(2 * M + j) * M;
        for (int k = 0; k < M; ++k) {
            hr += ur[k] * h[k];
            hz += uz[k] * h[k];
            hn += un[k] * h[k];
        }
        double r = sigmoid(ir + hr);
        double z = sigmoid(iz + hz);
        double n = tanh(in_ + r * hn);
        out[j] = (1.0 - z) * n + z * h[j];
    }
}

/* JODIE's memory updater: an RNN cell (Elman) on the same input as the GRU,
 *   h' = tanh(W_ih x + b_ih + W_hh h + b_hh),  W_ih [M x D_x], W_hh [M x M].
 * JODIE (Kumar et al. 2019) updates a node from its interactions with two
 * mutually recursive RNNs; the recursion runs through the message, which holds
 * the other endpoint's memory. */
void orc_rnn_cell(int M, int D_x, const double *W_ih, const double *W_hh,
                  const double *b_ih, const double *b_hh,
                  const double *x, const double *h, double *out)
{
    for (int j = 0; j < M; ++j) {
        double a = b_ih[j], u = b_hh[j];
        const double *w = W_ih + (size_t)j * D_x;
        for (int k = 0; k < D_x; ++k)
            a += w[k] * x[k];
        const double *v = W_hh + (size_t)j * M;
        for (int k = 0; k < M; ++k)
            u += v[k] * h[k];
        out[j] = tanh(a + u);
    }
}

/* JODIE's embedding, the time projection of a node's memory to the query
 * time tq: h = s * (1 + w_t * (tq - ts)), ts the memory's time. */
void orc_time_projection(int M, const double *w_t, const double *s, double ts, double tq,
                         double *out)
{
    const double d = tq - ts;
    for (int j = 0; j < M; ++j)
        out[j] = s[j] * (1.0 + w_t[j] * d);
}

/* y[rows] = W[rows x cols] * x[cols] + b[rows] */
static void matvec(int rows, int cols, const double *W, const double *b,
                   const double *x, double *y)
{
    for (int r = 0; r < rows; ++r) {
        double acc = b ? b[r] : 0.0;
        const double *w = W + (size_t)r * cols;
        for (int k = 0; k < cols; ++k)
            acc += w[k] * x[k];
        y[r] = acc;
    }
}

/* ------------------------------------------------------------------------- */
/* Embedding module emb() of Eq. 1 for one root v queried at time tq, from its
 * updated memory s_v and its cnt sampled neighbours u_j (memories s_u[j],
 * edge features f[j], event times nts[j]):
 *   q   = W_q [s_v || phi(0)] + b_q
 *   K_j = W_k [s_u_j || f_j || phi(tq - nts_j)] + b_k,  V_j likewise with W_v
 *   per head eta (width d_h = M / H):
 *     alpha_j = softmax_j( q_eta . K_eta,j / sqrt(d_h) ),  a_eta = sum_j alpha_j V_eta,j
 *   a = concat_eta a_eta  (a = 0 when cnt = 0)
 *   h = ReLU(W_o [a || s_v] + b_o)
 * Attention width d_a = M.                                                    */
typedef struct {
    int M, D_e, D_t, H;
    const double *omega, *beta;
    const double *W_q, *b_q, *W_k, *b_k, *W_v, *b_v, *W_o, *b_o;
} orc_attn_w;

static void embed_root(const orc_attn_w *w, const double *s_v, double tq,
                       int cnt, const double *const *s_u, const double *const *f,
                       const double *nts, double *h_out)
{
    const int M = w->M, D_e = w->D_e, D_t = w->D_t, H = w->H;
    const int d_a = M, d_h = M / H;
    const int D_q = M + D_t, D_kv = M + D_e + D_t;
    double *buf = (double *)malloc(sizeof(double) *
        (size_t)(D_q + d_a + D_kv + 2 * (size_t)(cnt > 0 ? cnt : 1) * d_a + cnt + d_a + d_a + M));
    double *xq = buf;                      /* [D_q] */
    double *q = xq + D_q;                  /* [d_a] */
    double *kap = q + d_a;                 /* [D_kv] */
    double *K = kap + D_kv;                /* [cnt x d_a] */
    double *V = K + (size_t)(cnt > 0 ? cnt : 1) * d_a;
    double *sc = V + (size_t)(cnt > 0 ? cnt : 1) * d_a;   /* [cnt] */
    double *a = sc + cnt;                  /* [d_a] */
    double *xo = a + d_a;                  /* [d_a + M] */

    memcpy(xq, s_v, sizeof(double) * M);
    orc_time_encode(D_t, w->omega, w->beta, 0.0, xq + M);
    matvec(d_a, D_q, w->W_q, w->b_q, xq, q);

    for (int j = 0; j < cnt; ++j) {
        memcpy(kap, s_u[j], sizeof(double) * M);
        for (int d = 0; d < D_e; ++d)
            kap[M + d] = f[j][d];
        orc_time_encode(D_t, w->omega, w->beta, tq - nts[j], kap + M + D_e);
        matvec(d_a, D_kv, w->W_k, w->b_k, kap, K + (size_t)j * d_a);
        matvec(d_a, D_kv, w->W_v, w->b_v, kap, V + (size_t)j * d_a);
    }

    const double scale = 1.0 / sqrt((double)d_h);
    for (int k = 0; k < d_a; ++k)
        a[k] = 0.0;
    for (int eta = 0; eta < H; ++eta) {
        const int o = eta * d_h;
        if (cnt == 0)
            break;
        double mx = -INFINITY;
        for (int j = 0; j < cnt; ++j) {
            double dot = 0.0;
            for (int k = 0; k < d_h; ++k)
                dot += q[o + k] * K[(size_t)j * d_a + o + k];
            sc[j] = dot * scale;
            if (sc[j] > mx)
                mx = sc[j];
        }
        /* softmax; the shift by the maximum leaves the value unchanged */
        double den = 0.0;
        for (int j = 0; j < cnt; ++j) {
            sc[j] = exp(sc[j] - mx);
            den += sc[j];
        }
        for (int j = 0; j < cnt; ++j) {
            const double al = sc[j] / den;
            for (int k = 0; k < d_h; ++k)
                a[o + k] += al * V[(size_t)j * d_a + o + k];
        }
    }

    memcpy(xo, a, sizeof(double) * d_a);
    memcpy(xo + d_a, s_v, sizeof(double) * M);
    matvec(M, d_a + M, w->W_o, w->b_o, xo, h_out);
    for (int k = 0; k < M; ++k)
        if (h_out[k] < 0.0)
            h_out[k] = 0.0;
    free(buf);
}

/* Exported form of embed_root for tests: s_u is [cnt x M], f is [cnt x D_e]. */
void orc_embed_one(int M, int D_e, int D_t, int H,
                   const double *omega, const double *beta,
                   const double *W_q, const double *b_q,
                   const double *W_k, const double *b_k,
                   const double *W_v, const double *b_v,
                   const double *W_o, const double *b_o,
                   const double *s_v, double tq, int cnt,
                   const double *s_u, const double *f, const double *nts,
                   double *h_out)
{
    orc_attn_w w = {M, D_e, D_t, H, omega, beta, W_q, b_q, W_k, b_k, W_v, b_v, W_o, b_o};
    const double **pu = (const double **)malloc(sizeof(void *) * (cnt > 0 ? cnt : 1));
    const double **pf = (const double **)malloc(sizeof(void *) * (cnt > 0 ? cnt : 1));
    for (int j = 0; j < cnt; ++j) {
        pu[j] = s_u + (size_t)j * M;
        pf[j] = f + (size_t)j * D_e;
    }
    embed_root(&w, s_v, tq, cnt, pu, pf, nts, h_out);
    free(pu);
    free(pf);
}

/* ------------------------------------------------------------------------- */
/* Temporal adjacency: for every node, the events that touch it, in event order.
 * Events are sorted by (t, e), so each list is sorted by (t, e) too.  A
 * self-loop is listed once.                                                   */
typedef struct {
    int N;
    int64_t E;
    int64_t *off;   /* [N+1] */
    int32_t *ev;    /* event ids */
} orc_adj;

static int build_adj(orc_adj *g, int N, int64_t E, const int32_t *src, const int32_t *dst)
{
    g->N = N;
    g->E = E;
    g->off = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
    if (!g->off)
        return ORC_EINVAL;
    for (int64_t e = 0; e < E; ++e) {
        g->off[src[e] + 1]++;
        if (dst[e] != src[e])
            g->off[dst[e] + 1]++;
    }
    for (int v = 0; v < N; ++v)
        g->off[v + 1] += g->off[v];
    g->ev = (int32_t *)malloc(sizeof(int32_t) * (size_t)(g->off[N] > 0 ? g->off[N] : 1));
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)N);
    if (!g->ev || !fill)
        return ORC_EINVAL;
    memcpy(fill, g->off, sizeof(int64_t) * (size_t)N);
    for (int64_t e = 0; e < E; ++e) {
        g->ev[fill[src[e]]++] = (int32_t)e;
        if (dst[e] != src[e])
            g->ev[fill[dst[e]]++] = (int32_t)e;
    }
    free(fill);
    return ORC_OK;
}

static void free_adj(orc_adj *g)
{
    free(g->off);
    free(g->ev);
    g->off = NULL;
    g->ev = NULL;
}

/* Most-recent-nb temporal neighbours of root v at query time tq: among the
 * events e' touching v with t[e'] < tq (strictly earlier), the nb largest by
 * (t[e'], e'), newest first.  The neighbour is the other endpoint (v itself for
 * a self-loop).  Unused slots hold nbr = eid = -1 and nts = 0.               */
static void sample_root(const orc_adj *g, const int32_t *src, const int32_t *dst,
                        const double *t, int v, double tq, int nb,
                        int32_t *nbr, int32_t *eid, double *nts, int32_t *cnt)
{
    int64_t lo = g->off[v], hi = g->off[v + 1];
    /* first list position whose event time is >= tq (binary search) */
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (t[g->ev[mid]] < tq)
            lo = mid + 1;
        else
            hi = mid;
    }
    int c = 0;
    for (int64_t k = lo - 1; k >= g->off[v] && c < nb; --k, ++c) {
        int32_t e = g->ev[k];
        nbr[c] = (src[e] == v) ? dst[e] : src[e];
        eid[c] = e;
        nts[c] = t[e];
    }
    *cnt = c;
    for (; c < nb; ++c) {
        nbr[c] = -1;
        eid[c] = -1;
        nts[c] = 0.0;
    }
}

/* Exported sampler over a stream (builds the adjacency on every call). */
int orc_sample(int N, int64_t E, const int32_t *src, const int32_t *dst, const double *t,
               int R, const int32_t *root, const double *root_ts, int nb,
               int32_t *nbr, int32_t *eid, double *nts, int32_t *cnt)
{
    orc_adj g;
    if (build_adj(&g, N, E, src, dst) != ORC_OK)
        return ORC_EINVAL;
    for (int r = 0; r < R; ++r)
        sample_root(&g, src, dst, t, root[r], root_ts[r], nb, nbr + (size_t)r * nb,
                    eid + (size_t)r * nb, nts + (size_t)r * nb, cnt + r);
    free_adj(&g);
    return ORC_OK;
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* ------------------------------------------------------------------------- */
/* Similarity-based staleness mitigation (MSPipe-S, Sec. 3.3).  Readings where
 * the text is silent:
 *   - the gap of a fetched node u is dt_u = T - mem_ts_u, T the time of the
 *     batch's first event (the time since u's memory was last updated);
 *   - gamma is the nearest-rank p-quantile of {dt_u : u in U}: the
 *     ceil(p |U|)-th smallest gap;
 *   - stale: dt_v > gamma; active: dt_u < gamma (then also fresher than any
 *     stale v);
 *   - the neighbours of a node are the distinct other endpoints of its nb
 *     most recent events before T (the sampler's temporal neighbourhood);
 *   - Omega(v) = the K active nodes with the most common neighbours (at least
 *     one), ties to the fresher memory, then the smaller id;
 *   - s_hat_v = lambda s_v + (1 - lambda) mean_{u in Omega(v)} s_u over the
 *     fetched (unmitigated) memories; v keeps s_v when Omega(v) is empty.   */

static int cmp_f64(const void *a, const void *b)
{
    double x = *(const double *)a, y = *(const double *)b;
    return (x > y) - (x < y);
}

/* nearest-rank p-quantile of n values (n >= 1) */
double orc_quantile_nearest_rank(int n, const double *x, double p)
{
    double *s = (double *)malloc(sizeof(double) * (size_t)n);
    memcpy(s, x, sizeof(double) * (size_t)n);
    qsort(s, (size_t)n, sizeof(double), cmp_f64);
    long rank = (long)ceil(p * (double)n);
    if (rank < 1)
        rank = 1;
    if (rank > n)
        rank = n;
    const double q = s[rank - 1];
    free(s);
    return q;
}

/* common elements of two sorted lists of distinct ids */
static int common_count(const int32_t *a, int na, const int32_t *b, int nb_)
{
    int i = 0, j = 0, c = 0;
    while (i < na && j < nb_) {
        if (a[i] < b[j])
            ++i;
        else if (a[i] > b[j])
            ++j;
        else {
            ++c; ++i; ++j;
        }
    }
    return c;
}

typedef struct {
    int sim;
    double mts;
    int32_t id, pos;
} orc_cand;

/* more common neighbours first, then the fresher memory, then the smaller id */
static int cmp_cand(const void *a, const void *b)
{
    const orc_cand *x = (const orc_cand *)a, *y = (const orc_cand *)b;
    if (x->sim != y->sim)
        return x->sim > y->sim ? -1 : 1;
    if (x->mts != y->mts)
        return x->mts > y->mts ? -1 : 1;
    return (x->id > y->id) - (x->id < y->id);
}

/* Mitigates the fetched rows fm [nU x M] of the nodes ids [nU] (with memory
 * times fmts) in place.  Returns gamma; writes the stale positions (ascending)
 * and their Omega positions when the pointers are given. */
static double mitigate(const orc_adj *g, const int32_t *src, const int32_t *dst,
                       const double *t, int nb, double T, int nU, const int32_t *ids,
                       double *fm, const double *fmts, int M, double p, double lambda, int K,
                       int32_t *stale_out, int32_t *omega_out, int *n_stale_out)
{
    double *dt = (double *)malloc(sizeof(double) * (size_t)nU);
    for (int k = 0; k < nU; ++k)
        dt[k] = T - fmts[k];
    const double gamma = orc_quantile_nearest_rank(nU, dt, p);
    /* neighbour sets: sorted distinct ids */
    const int nbc = nb > 0 ? nb : 1;
    int32_t *nset = (int32_t *)malloc(sizeof(int32_t) * (size_t)nU * nbc);
    int *ncnt = (int *)malloc(sizeof(int) * (size_t)nU);
    #pragma omp parallel for schedule(dynamic, 64)
    for (int k = 0; k < nU; ++k) {
        int32_t *nbr = nset + (size_t)k * nbc;
        int32_t *eid = (int32_t *)malloc(sizeof(int32_t) * nbc);
        double *nts = (double *)malloc(sizeof(double) * nbc);
        int32_t c = 0;
        sample_root(g, src, dst, t, ids[k], T, nb, nbr, eid, nts, &c);
        qsort(nbr, (size_t)c, sizeof(int32_t), cmp_i32);
        int d = 0;
        for (int j = 0; j < c; ++j)
            if (d == 0 || nbr[j] != nbr[d - 1])
                nbr[d++] = nbr[j];
        ncnt[k] = d;
        free(eid);
        free(nts);
    }
    int ns = 0;
    int32_t *stale = (int32_t *)malloc(sizeof(int32_t) * (size_t)nU);
    for (int k = 0; k < nU; ++k)
        if (dt[k] > gamma)
            stale[ns++] = k;
    double *out = (double *)malloc(sizeof(double) * ((size_t)ns * M + 1));
    int32_t *om = (int32_t *)malloc(sizeof(int32_t) * ((size_t)ns * (K > 0 ? K : 1) + 1));
    #pragma omp parallel for schedule(dynamic, 1)
    for (int q = 0; q < ns; ++q) {
        const int v = stale[q];
        orc_cand *cand = (orc_cand *)malloc(sizeof(orc_cand) * (size_t)nU);
        int nc = 0;
        for (int u = 0; u < nU; ++u) {
            if (!(dt[u] < gamma))
                continue;
            const int sim = common_count(nset + (size_t)v * nbc, ncnt[v],
                                         nset + (size_t)u * nbc, ncnt[u]);
            if (sim > 0) {
                cand[nc].sim = sim;
                cand[nc].mts = fmts[u];
                cand[nc].id = ids[u];
                cand[nc].pos = u;
                ++nc;
            }
        }
        qsort(cand, (size_t)nc, sizeof(orc_cand), cmp_cand);
        const int m = nc < K ? nc : K;
        for (int j = 0; j < K; ++j)
            om[(size_t)q * K + j] = j < m ? cand[j].pos : -1;
        for (int d = 0; d < M; ++d) {
            double x = fm[(size_t)v * M + d];
            if (m > 0) {
                double acc = 0.0;
                for (int j = 0; j < m; ++j)
                    acc += fm[(size_t)cand[j].pos * M + d];
                x = lambda * x + (1.0 - lambda) * (acc / m);
            }
            out[(size_t)q * M + d] = x;
        }
        free(cand);
    }
    /* stale rows are never sources (sources are active), so order is free */
    for (int q = 0; q < ns; ++q)
        memcpy(fm + (size_t)stale[q] * M, out + (size_t)q * M, sizeof(double) * M);
    if (stale_out)
        memcpy(stale_out, stale, sizeof(int32_t) * (size_t)ns);
    if (omega_out)
        memcpy(omega_out, om, sizeof(int32_t) * (size_t)ns * K);
    *n_stale_out = ns;
    free(dt); free(nset); free(ncnt); free(stale); free(out); free(om);
    return gamma;
}

/* ------------------------------------------------------------------------- */
/* The stateful driver.                                                        */
typedef struct {
    int64_t iter;
    int n;
    int32_t *node;
    double *mem, *mem_ts, *mail, *mail_ts;
    /* APAN: the mails the iteration delivers, in delivery order (node,
     * message [D_m], event time) */
    int n_del;
    int32_t *del_node;
    double *del_mail, *del_t;
} orc_wset;

typedef struct {
    int N;
    int64_t E;
    const int32_t *src, *dst, *neg;
    const double *t;
    const float *efeat;
    int D_e, M, D_t, H, nb, B, s;
    int D_m, D_x;
    /* fp64 weights */
    double *W_ih, *W_hh, *b_ih, *b_hh, *omega, *beta;
    double *W_q, *b_q, *W_k, *b_k, *W_v, *b_v, *W_o, *b_o;
    orc_adj adj;
    /* committed state */
    double *mem, *mem_ts, *mail, *mail_ts;
    int32_t *ver;
    /* queued write sets, oldest first */
    orc_wset *q;
    int nq, capq;
    int64_t next_iter;
    /* staleness mitigation (off unless orc_set_mitigation enables it) */
    int mit_on, mit_K;
    double mit_p, mit_lambda;
    /* model family and JODIE's projection vector */
    int kind;
    double *w_t;
    /* APAN: every node's mailbox, its K_mb latest mails oldest first (rows
     * [N x K_mb x D_m], times [N x K_mb], count [N]); whether each mail also
     * goes to the sampled neighbours of its node */
    int K_mb, propagate;
    double *mb, *mb_ts;
    int32_t *mb_cnt;
    /* training (off unless orc_set_training enables it): every trained
     * parameter in one vector theta (the weights above point into it), the
     * link predictor's weights, the gradient of the last step, the optimizer's
     * moments and step count */
    int train_on, opt;
    double lr, beta1, beta2, eps;
    int64_t n_params, opt_steps;
    double *theta, *grad, *m1, *m2;
    double *W_src, *W_dst, *b_p, *w_out, *b_out;
} orc_ctx;

typedef struct {
    int N;
    int64_t E;
    const int32_t *src, *dst, *neg;
    const double *t;
    const float *efeat;
    int D_e, M, D_t, H, nb, B, s;
    const float *W_ih, *W_hh, *b_ih, *b_hh;
    const double *omega, *beta;
    const float *W_q, *b_q, *W_k, *b_k, *W_v, *b_v, *W_o, *b_o;
    /* ORC_TGN (the fields above) or ORC_JODIE: W_ih [M x D_x], W_hh [M x M],
     * b_ih, b_hh [M], w_t [M]; the attention weights are not read */
    int kind;
    const float *w_t;
    /* ORC_APAN: mailbox size and propagation to neighbours; W_q [M x (M +
     * D_t)], b_q, W_k [M x (D_m + D_t)], b_k of the mailbox attention */
    int K_mb, propagate;
} orc_desc;

/* Per-iteration outputs; every pointer may be NULL.  Capacities: R = 3B roots,
 * U <= N nodes. */
typedef struct {
    int64_t iter;
    int32_t b, R, n_U, pad_;
    int32_t *root;
    double *root_ts;
    int32_t *nbr, *eid;
    double *nts;
    int32_t *cnt;
    int32_t *U, *root_pos, *nbr_pos;
    double *f_mem, *f_mem_ts, *f_mail, *f_mail_ts;
    int32_t *f_ver;
    double *s_new, *new_mem_ts;
    double *h;
    int64_t *winner;
    /* staleness mitigation: mitigated rows [n_U x M], stale positions
     * [n_stale], their Omega as positions [n_stale x K] (-1 padded), gamma */
    double *m_mem;
    int32_t *m_stale, *m_omega;
    double m_gamma;
    int32_t m_n_stale, m_pad;
    /* the exact memories of U [n_U x M]: the committed state with every write
     * set of iterations <= i-1 applied, i.e. what a fetch without staleness
     * would read at this point of the run (for the staleness error of Sec. 5.5
     * and App. E.2) */
    double *x_mem;
    /* training: the loss of the iteration, the gradient of every parameter
     * [n_params] and the parameters after the optimizer step [n_params], in
     * the order of orc_param_layout */
    double loss;
    double *grad, *params;
    /* the smallest |pre-activation| of the ReLUs the gradient passes (the
     * predictor's z and the attention's output projection): the margin by
     * which no branch of the backward is near its kink */
    double relu_margin;
    /* APAN: the fetched mailboxes, oldest mail first: rows [n_U x K_mb x D_m],
     * times [n_U x K_mb], counts [n_U] */
    double *f_mb, *f_mb_ts;
    int32_t *f_mb_cnt;
} orc_step_out;

static double *widen(const float *x, size_t n)
{
    double *y = (double *)malloc(sizeof(double) * (n ? n : 1));
    for (size_t i = 0; i < n; ++i)
        y[i] = (double)x[i];
    return y;
}

static double *copyd(const double *x, size_t n)
{
    double *y = (double *)malloc(sizeof(double) * (n ? n : 1));
    if (n)
        memcpy(y, x, sizeof(double) * n);
    return y;
}

void *orc_create(const orc_desc *d)
{
    if (!d || d->N <= 0 || d->E < 0 || d->M <= 0 || d->H <= 0 || d->M % d->H != 0 ||
        d->nb < 0 || d->B <= 0 || d->s < 0 || d->D_t < 0 || d->D_e < 0 ||
        (d->kind != ORC_TGN && d->kind != ORC_JODIE && d->kind != ORC_APAN) ||
        (d->kind == ORC_JODIE && !d->w_t) || (d->kind == ORC_APAN && d->K_mb < 1))
        return NULL;
    orc_ctx *c = (orc_ctx *)calloc(1, sizeof(orc_ctx));
    c->N = d->N; c->E = d->E;
    c->src = d->src; c->dst = d->dst; c->neg = d->neg; c->t = d->t; c->efeat = d->efeat;
    c->D_e = d->D_e; c->M = d->M; c->D_t = d->D_t; c->H = d->H; c->nb = d->nb;
    c->B = d->B; c->s = d->s;
    c->D_m = 2 * d->M + d->D_e;
    c->D_x = c->D_m + d->D_t;
    const int M = c->M, D_x = c->D_x, D_t = c->D_t, D_e = c->D_e;
    c->kind = d->kind;
    const int G = c->kind == ORC_JODIE ? 1 : 3;   /* gate row blocks of the updater */
    c->W_ih = widen(d->W_ih, (size_t)G * M * D_x);
    c->W_hh = widen(d->W_hh, (size_t)G * M * M);
    c->b_ih = widen(d->b_ih, (size_t)G * M);
    c->b_hh = widen(d->b_hh, (size_t)G * M);
    c->omega = copyd(d->omega, (size_t)D_t);
    c->beta = copyd(d->beta, (size_t)D_t);
    if (c->kind == ORC_TGN) {
        c->W_q = widen(d->W_q, (size_t)M * (M + D_t));
        c->b_q = widen(d->b_q, (size_t)M);
        c->W_k = widen(d->W_k, (size_t)M * (M + D_e + D_t));
        c->b_k = widen(d->b_k, (size_t)M);
        c->W_v = widen(d->W_v, (size_t)M * (M + D_e + D_t));
        c->b_v = widen(d->b_v, (size_t)M);
        c->W_o = widen(d->W_o, (size_t)M * (2 * M));
        c->b_o = widen(d->b_o, (size_t)M);
    } else if (c->kind == ORC_APAN) {
        c->W_q = widen(d->W_q, (size_t)M * (M + D_t));
        c->b_q = widen(d->b_q, (size_t)M);
        c->W_k = widen(d->W_k, (size_t)M * (c->D_m + D_t));
        c->b_k = widen(d->b_k, (size_t)M);
        c->K_mb = d->K_mb;
        c->propagate = d->propagate != 0;
        c->mb = (double *)calloc((size_t)c->N * d->K_mb * c->D_m + 1, sizeof(double));
        c->mb_ts = (double *)calloc((size_t)c->N * d->K_mb, sizeof(double));
        c->mb_cnt = (int32_t *)calloc((size_t)c->N, sizeof(int32_t));
    } else {
        c->w_t = widen(d->w_t, (size_t)M);
    }
    if (build_adj(&c->adj, c->N, c->E, c->src, c->dst) != ORC_OK)
        return NULL;
    c->mem = (double *)calloc((size_t)c->N * M, sizeof(double));
    c->mem_ts = (double *)calloc((size_t)c->N, sizeof(double));
    c->mail = (double *)calloc((size_t)c->N * c->D_m + 1, sizeof(double));
    c->mail_ts = (double *)calloc((size_t)c->N, sizeof(double));
    c->ver = (int32_t *)malloc(sizeof(int32_t) * (size_t)c->N);
    for (int v = 0; v < c->N; ++v)
        c->ver[v] = -1;
    c->capq = c->s + 2;
    c->q = (orc_wset *)calloc((size_t)c->capq, sizeof(orc_wset));
    return c;
}

static void free_wset(orc_wset *w)
{
    free(w->node); free(w->mem); free(w->mem_ts); free(w->mail); free(w->mail_ts);
    free(w->del_node); free(w->del_mail); free(w->del_t);
    memset(w, 0, sizeof(*w));
}

void orc_destroy(void *p)
{
    orc_ctx *c = (orc_ctx *)p;
    if (!c)
        return;
    if (c->train_on) {   /* the weights live in theta */
        free(c->theta); free(c->grad); free(c->m1); free(c->m2);
    } else {
        free(c->W_ih); free(c->W_hh); free(c->b_ih); free(c->b_hh);
        free(c->W_q); free(c->b_q); free(c->W_k); free(c->b_k); free(c->W_v); free(c->b_v);
        free(c->W_o); free(c->b_o);
    }
    free(c->omega); free(c->beta); free(c->w_t);
    free(c->mb); free(c->mb_ts); free(c->mb_cnt);
    free_adj(&c->adj);
    free(c->mem); free(c->mem_ts); free(c->mail); free(c->mail_ts); free(c->ver);
    for (int k = 0; k < c->nq; ++k)
        free_wset(&c->q[k]);
    free(c->q);
    free(c);
}

/* Apply the oldest queued write set to the committed state (last writer wins). */
static void apply_oldest(orc_ctx *c)
{
    orc_wset *w = &c->q[0];
    const int M = c->M, D_m = c->D_m;
    for (int k = 0; k < w->n; ++k) {
        const int v = w->node[k];
        memcpy(c->mem + (size_t)v * M, w->mem + (size_t)k * M, sizeof(double) * M);
        memcpy(c->mail + (size_t)v * D_m, w->mail + (size_t)k * D_m, sizeof(double) * D_m);
        c->mem_ts[v] = w->mem_ts[k];
        c->mail_ts[v] = w->mail_ts[k];
        c->ver[v] = (int32_t)w->iter;
    }
    /* APAN: each delivered mail joins its node's mailbox as the newest; a
     * full mailbox drops its oldest */
    const int K = c->K_mb;
    for (int k = 0; k < w->n_del; ++k) {
        const int v = w->del_node[k];
        double *rows = c->mb + (size_t)v * K * D_m, *ts = c->mb_ts + (size_t)v * K;
        if (c->mb_cnt[v] == K) {
            memmove(rows, rows + D_m, sizeof(double) * (size_t)(K - 1) * D_m);
            memmove(ts, ts + 1, sizeof(double) * (size_t)(K - 1));
            c->mb_cnt[v]--;
        }
        memcpy(rows + (size_t)c->mb_cnt[v] * D_m, w->del_mail + (size_t)k * D_m,
               sizeof(double) * D_m);
        ts[c->mb_cnt[v]] = w->del_t[k];
        c->mb_cnt[v]++;
    }
    free_wset(w);
    memmove(c->q, c->q + 1, sizeof(orc_wset) * (size_t)(c->nq - 1));
    c->nq--;
    memset(&c->q[c->nq], 0, sizeof(orc_wset));
}

/* Commit every queued write set (end of the run). */
void orc_flush(void *p)
{
    orc_ctx *c = (orc_ctx *)p;
    while (c->nq > 0)
        apply_oldest(c);
}

/* Replace the committed state and the iteration counter; drops the queue.
 * Reads at iterations i >= it then see this state plus the write sets of
 * iterations it .. i-1-s. */
void orc_set_state(void *p, int64_t it, const double *mem, const double *mem_ts,
                   const double *mail, const double *mail_ts, const int32_t *ver)
{
    orc_ctx *c = (orc_ctx *)p;
    while (c->nq > 0) {
        free_wset(&c->q[0]);
        memmove(c->q, c->q + 1, sizeof(orc_wset) * (size_t)(c->nq - 1));
        c->nq--;
    }
    memcpy(c->mem, mem, sizeof(double) * (size_t)c->N * c->M);
    memcpy(c->mem_ts, mem_ts, sizeof(double) * (size_t)c->N);
    memcpy(c->mail, mail, sizeof(double) * (size_t)c->N * c->D_m);
    memcpy(c->mail_ts, mail_ts, sizeof(double) * (size_t)c->N);
    memcpy(c->ver, ver, sizeof(int32_t) * (size_t)c->N);
    c->next_iter = it;
}

/* Queue a write set of iteration `it` behind the queued ones (after
 * orc_set_state: the pending updates of a saved state, which the snapshot of
 * iteration i applies once it <= i-1-s, Eq. 2).  Rows: node [n], mem [n x M],
 * mem_ts [n], mail [n x D_m], mail_ts [n]; iterations must grow.  Returns 0,
 * or -1 for an iteration not after the last queued one. */
int orc_push_wset(void *p, int64_t it, int n, const int32_t *node, const double *mem,
                  const double *mem_ts, const double *mail, const double *mail_ts)
{
    orc_ctx *c = (orc_ctx *)p;
    if (n < 0 || (c->nq > 0 && c->q[c->nq - 1].iter >= it))
        return -1;
    const int M = c->M, D_m = c->D_m;
    orc_wset W;
    memset(&W, 0, sizeof(W));
    W.iter = it;
    W.n = n;
    W.node = (int32_t *)malloc(sizeof(int32_t) * (n ? n : 1));
    W.mem = (double *)malloc(sizeof(double) * ((size_t)n * M + 1));
    W.mem_ts = (double *)malloc(sizeof(double) * (n ? n : 1));
    W.mail = (double *)malloc(sizeof(double) * ((size_t)n * D_m + 1));
    W.mail_ts = (double *)malloc(sizeof(double) * (n ? n : 1));
    if (n) {
        memcpy(W.node, node, sizeof(int32_t) * (size_t)n);
        memcpy(W.mem, mem, sizeof(double) * (size_t)n * M);
        memcpy(W.mem_ts, mem_ts, sizeof(double) * (size_t)n);
        if (D_m)
            memcpy(W.mail, mail, sizeof(double) * (size_t)n * D_m);
        memcpy(W.mail_ts, mail_ts, sizeof(double) * (size_t)n);
    }
    if (c->nq == c->capq) {
        c->capq *= 2;
        c->q = (orc_wset *)realloc(c->q, sizeof(orc_wset) * (size_t)c->capq);
    }
    c->q[c->nq++] = W;
    return 0;
}

void orc_get_state(void *p, double *mem, double *mem_ts, double *mail, double *mail_ts,
                   int32_t *ver)
{
    orc_ctx *c = (orc_ctx *)p;
    if (mem) memcpy(mem, c->mem, sizeof(double) * (size_t)c->N * c->M);
    if (mem_ts) memcpy(mem_ts, c->mem_ts, sizeof(double) * (size_t)c->N);
    if (mail) memcpy(mail, c->mail, sizeof(double) * (size_t)c->N * c->D_m);
    if (mail_ts) memcpy(mail_ts, c->mail_ts, sizeof(double) * (size_t)c->N);
    if (ver) memcpy(ver, c->ver, sizeof(int32_t) * (size_t)c->N);
}

int64_t orc_next_iter(void *p) { return ((orc_ctx *)p)->next_iter; }

/* APAN: the committed mailboxes, oldest mail first (rows [N x K_mb x D_m],
 * times [N x K_mb], counts [N]; any pointer may be NULL). */
void orc_get_mailbox(void *p, double *mb, double *mb_ts, int32_t *mb_cnt)
{
    orc_ctx *c = (orc_ctx *)p;
    if (c->kind != ORC_APAN)
        return;
    const size_t N = (size_t)c->N, K = (size_t)c->K_mb;
    if (mb) memcpy(mb, c->mb, sizeof(double) * N * K * c->D_m);
    if (mb_ts) memcpy(mb_ts, c->mb_ts, sizeof(double) * N * K);
    if (mb_cnt) memcpy(mb_cnt, c->mb_cnt, sizeof(int32_t) * N);
}

/* APAN: replace the committed mailboxes (the layouts of orc_get_mailbox,
 * oldest mail first; mails past a count are not read).  Returns 0, or -1
 * for a model without mailboxes or a count outside [0, K_mb] (nothing is
 * changed then). */
int orc_set_mailbox(void *p, const double *mb, const double *mb_ts, const int32_t *mb_cnt)
{
    orc_ctx *c = (orc_ctx *)p;
    if (c->kind != ORC_APAN)
        return -1;
    const size_t N = (size_t)c->N, K = (size_t)c->K_mb, D_m = (size_t)c->D_m;
    for (size_t v = 0; v < N; ++v)
        if (mb_cnt[v] < 0 || mb_cnt[v] > (int32_t)K)
            return -1;
    for (size_t v = 0; v < N; ++v) {
        c->mb_cnt[v] = mb_cnt[v];
        for (size_t j = 0; j < K; ++j) {
            const int used = (int32_t)j < mb_cnt[v];
            for (size_t k = 0; k < D_m; ++k)
                c->mb[(v * K + j) * D_m + k] = used ? mb[(v * K + j) * D_m + k] : 0.0;
            c->mb_ts[v * K + j] = used ? mb_ts[v * K + j] : 0.0;
        }
    }
    return 0;
}

/* Enables (on != 0) the staleness mitigation of step 3b with quantile p,
 * blend weight lambda and at most K similar nodes. */
int orc_set_mitigation(void *p, int on, double pq, double lambda, int K)
{
    orc_ctx *c = (orc_ctx *)p;
    if (on && (K < 1 || !(pq >= 0.0 && pq <= 1.0) || !(lambda >= 0.0 && lambda <= 1.0)))
        return ORC_EINVAL;
    c->mit_on = on != 0;
    c->mit_p = pq;
    c->mit_lambda = lambda;
    c->mit_K = K;
    return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Training (the step after the stage: loss, gradient, optimizer).
 *
 * The training samples of an iteration are its b positive pairs (src, dst)
 * and b negative pairs (src, neg) (Sec. 5, training settings: equal numbers of
 * positive and negative pairs, link prediction).  Link predictor, a two-layer
 * perceptron over the two endpoint embeddings (reading R28):
 *   z = W_src h_u + W_dst h_v + b_p,   score(u, v) = w_out . ReLU(z) + b_out
 * Loss, binary cross-entropy with the scores as logits (reading R29):
 *   L = (1/b) sum_e [ softplus(-score(src_e, dst_e)) + softplus(score(src_e, neg_e)) ]
 * The gradient flows through h into the attention's weights and the updated
 * memories s', and through s' into the memory updater's weights for the
 * nodes that hold mail.  The fetched memories and mails are inputs of the
 * iteration, and the time encoding's omega and beta are not trained (reading
 * R30).  The optimizer takes one step per iteration after the write set is
 * staged (reading R31): SGD, theta -= lr g (the update of the convergence
 * analysis of Sec. 4), or Adam with bias correction (the optimizer of the
 * training settings, with its learning rate).
 *
 * Parameter vector order (orc_param_sizes): W_ih [3M x D_x], W_hh [3M x M],
 * b_ih [3M], b_hh [3M], W_q [M x (M + D_t)], b_q [M], W_k [M x D_kv], b_k [M],
 * W_v [M x D_kv], b_v [M], W_o [M x 2M], b_o [M], W_src [M x M], W_dst [M x M],
 * b_p [M], w_out [M], b_out [1]; D_kv = M + D_e + D_t. */
#define ORC_NPT 17
#define ORC_SGD 0
#define ORC_ADAM 1

static void param_sizes(const orc_ctx *c, int64_t *sz)
{
    const int64_t M = c->M, D_x = c->D_x, D_q = c->M + c->D_t, D_kv = c->M + c->D_e + c->D_t;
    const int64_t v[ORC_NPT] = {3 * M * D_x, 3 * M * M, 3 * M, 3 * M, M * D_q, M, M * D_kv, M,
                                M * D_kv, M, M * 2 * M, M, M * M, M * M, M, M, 1};
    memcpy(sz, v, sizeof(v));
}

/* views[k] = the k-th parameter tensor inside a vector of the layout above */
static void param_views(const orc_ctx *c, double *base, double **views)
{
    int64_t sz[ORC_NPT];
    param_sizes(c, sz);
    for (int k = 0; k < ORC_NPT; ++k) {
        views[k] = base;
        base += sz[k];
    }
}

void orc_param_sizes(void *p, int64_t *sizes)
{
    param_sizes((const orc_ctx *)p, sizes);
}

static double softplus(double x) { return x > 0.0 ? x + log1p(exp(-x)) : log1p(exp(x)); }

/* Turns training on (TGN models): the predictor's weights (fp32, widened),
 * the optimizer (ORC_SGD or ORC_ADAM) and its constants.  Returns 0, or -1. */
int orc_set_training(void *p, int opt, double lr, double beta1, double beta2, double eps,
                     const float *W_src, const float *W_dst, const float *b_p,
                     const float *w_out, float b_out)
{
    orc_ctx *c = (orc_ctx *)p;
    if (c->kind != ORC_TGN || c->train_on || (opt != ORC_SGD && opt != ORC_ADAM) ||
        !(lr >= 0.0) || !W_src || !W_dst || !b_p || !w_out)
        return ORC_EINVAL;
    int64_t sz[ORC_NPT], n = 0;
    param_sizes(c, sz);
    for (int k = 0; k < ORC_NPT; ++k)
        n += sz[k];
    c->n_params = n;
    c->theta = (double *)malloc(sizeof(double) * (size_t)n);
    c->grad = (double *)calloc((size_t)n, sizeof(double));
    c->m1 = (double *)calloc((size_t)n, sizeof(double));
    c->m2 = (double *)calloc((size_t)n, sizeof(double));
    double *v[ORC_NPT];
    param_views(c, c->theta, v);
    double *old[12] = {c->W_ih, c->W_hh, c->b_ih, c->b_hh, c->W_q, c->b_q,
                       c->W_k, c->b_k, c->W_v, c->b_v, c->W_o, c->b_o};
    for (int k = 0; k < 12; ++k) {
        memcpy(v[k], old[k], sizeof(double) * (size_t)sz[k]);
        free(old[k]);
    }
    const int M = c->M;
    for (int64_t k = 0; k < (int64_t)M * M; ++k) {
        v[12][k] = W_src[k];
        v[13][k] = W_dst[k];
    }
    for (int k = 0; k < M; ++k) {
        v[14][k] = b_p[k];
        v[15][k] = w_out[k];
    }
    v[16][0] = b_out;
    c->W_ih = v[0]; c->W_hh = v[1]; c->b_ih = v[2]; c->b_hh = v[3];
    c->W_q = v[4]; c->b_q = v[5]; c->W_k = v[6]; c->b_k = v[7];
    c->W_v = v[8]; c->b_v = v[9]; c->W_o = v[10]; c->b_o = v[11];
    c->W_src = v[12]; c->W_dst = v[13]; c->b_p = v[14]; c->w_out = v[15]; c->b_out = v[16];
    c->train_on = 1;
    c->opt = opt;
    c->lr = lr;
    c->beta1 = beta1;
    c->beta2 = beta2;
    c->eps = eps;
    c->opt_steps = 0;
    return ORC_OK;
}

int64_t orc_param_count(void *p) { return ((orc_ctx *)p)->n_params; }

void orc_get_params(void *p, double *out)
{
    orc_ctx *c = (orc_ctx *)p;
    if (c->train_on)
        memcpy(out, c->theta, sizeof(double) * (size_t)c->n_params);
}

/* Loss and gradient of one iteration (into c->grad), from the iteration's
 * forward values: root and neighbour positions in the node set, the fetched
 * rows (fm: after the mitigation when it is on), the updated memories sn
 * [nU x M] and the embeddings h [R x M].  Intermediate values of the
 * attention and the memory updater are recomputed here from the same inputs.
 * Returns the loss. */
static double train_gradient(orc_ctx *c, int b, int R, int nU, const int32_t *root_pos,
                             const double *rts, const int32_t *nbr_pos, const int32_t *eid,
                             const double *nts, const int32_t *cnt, const double *fm,
                             const double *fmts, const double *fl, const double *flts,
                             const int32_t *fver, const double *sn, const double *h,
                             double *margin_out)
{
    double margin = INFINITY;
    const int M = c->M, D_e = c->D_e, D_t = c->D_t, H = c->H, nb = c->nb;
    const int D_x = c->D_x, D_m = c->D_m;
    const int D_q = M + D_t, D_kv = M + D_e + D_t, d_h = M / H;
    const int nbs = nb > 0 ? nb : 1;
    double *g[ORC_NPT];
    param_views(c, c->grad, g);
    memset(c->grad, 0, sizeof(double) * (size_t)c->n_params);
    double *gW_ih = g[0], *gW_hh = g[1], *gb_ih = g[2], *gb_hh = g[3];
    double *gW_q = g[4], *gb_q = g[5], *gW_k = g[6], *gb_k = g[7], *gW_v = g[8], *gb_v = g[9];
    double *gW_o = g[10], *gb_o = g[11], *gW_src = g[12], *gW_dst = g[13], *gb_p = g[14];
    double *gw_out = g[15], *gb_out = g[16];

    /* the link predictor and the loss, event by event */
    double *dh = (double *)calloc((size_t)R * M + 1, sizeof(double));
    double *zp = (double *)malloc(sizeof(double) * 4 * M);
    double *zn = zp + M, *dzp = zn + M, *dzn = dzp + M;
    double loss = 0.0;
    for (int e = 0; e < b; ++e) {
        const double *hs = h + (size_t)e * M, *hd = h + (size_t)(b + e) * M;
        const double *hn = h + (size_t)(2 * b + e) * M;
        double sp = c->b_out[0], sq = c->b_out[0];
        for (int i = 0; i < M; ++i) {
            double a = c->b_p[i], an = c->b_p[i];
            for (int k = 0; k < M; ++k) {
                a += c->W_src[(size_t)i * M + k] * hs[k] + c->W_dst[(size_t)i * M + k] * hd[k];
                an += c->W_src[(size_t)i * M + k] * hs[k] + c->W_dst[(size_t)i * M + k] * hn[k];
            }
            zp[i] = a;
            zn[i] = an;
            sp += c->w_out[i] * (a > 0.0 ? a : 0.0);
            sq += c->w_out[i] * (an > 0.0 ? an : 0.0);
        }
        for (int i = 0; i < M; ++i)
            margin = fmin(margin, fmin(fabs(zp[i]), fabs(zn[i])));
        loss += softplus(-sp) + softplus(sq);
        const double dsp = (sigmoid(sp) - 1.0) / b, dsq = sigmoid(sq) / b;
        gb_out[0] += dsp + dsq;
        for (int i = 0; i < M; ++i) {
            gw_out[i] += dsp * (zp[i] > 0.0 ? zp[i] : 0.0) + dsq * (zn[i] > 0.0 ? zn[i] : 0.0);
            dzp[i] = zp[i] > 0.0 ? dsp * c->w_out[i] : 0.0;
            dzn[i] = zn[i] > 0.0 ? dsq * c->w_out[i] : 0.0;
            gb_p[i] += dzp[i] + dzn[i];
            for (int k = 0; k < M; ++k) {
                gW_src[(size_t)i * M + k] += (dzp[i] + dzn[i]) * hs[k];
                gW_dst[(size_t)i * M + k] += dzp[i] * hd[k] + dzn[i] * hn[k];
            }
        }
        for (int k = 0; k < M; ++k) {
            double a = 0.0, ad = 0.0, an = 0.0;
            for (int i = 0; i < M; ++i) {
                a += c->W_src[(size_t)i * M + k] * (dzp[i] + dzn[i]);
                ad += c->W_dst[(size_t)i * M + k] * dzp[i];
                an += c->W_dst[(size_t)i * M + k] * dzn[i];
            }
            dh[(size_t)e * M + k] += a;
            dh[(size_t)(b + e) * M + k] += ad;
            dh[(size_t)(2 * b + e) * M + k] += an;
        }
    }
    free(zp);

    /* the attention, root by root: its forward values again, then the
     * gradients of its inputs and of the slot-level projections */
    const size_t RS = (size_t)R * nbs;
    double *kap = (double *)calloc(RS * D_kv + 1, sizeof(double));
    double *dK = (double *)calloc(RS * M + 1, sizeof(double));
    double *dV = (double *)calloc(RS * M + 1, sizeof(double));
    double *ds_slot = (double *)calloc(RS * M + 1, sizeof(double));
    double *xq = (double *)malloc(sizeof(double) * ((size_t)R * D_q + 1));
    double *dq = (double *)calloc((size_t)R * M + 1, sizeof(double));
    double *xo = (double *)malloc(sizeof(double) * ((size_t)R * 2 * M + 1));
    double *dzo = (double *)malloc(sizeof(double) * ((size_t)R * M + 1));
    double *ds_root = (double *)malloc(sizeof(double) * ((size_t)R * M + 1));
    const double scale = 1.0 / sqrt((double)d_h);
    double *omarg = (double *)malloc(sizeof(double) * (R > 0 ? R : 1));
    #pragma omp parallel for schedule(dynamic, 8)
    for (int r = 0; r < R; ++r) {
        const int cr = cnt[r];
        const double *sv = sn + (size_t)root_pos[r] * M;
        double *K = (double *)malloc(sizeof(double) * ((size_t)nbs * M * 2 + 4 * (size_t)M +
                                                       (size_t)H * nbs + nbs));
        double *V = K + (size_t)nbs * M;
        double *q = V + (size_t)nbs * M, *o = q + M, *dxo = o + M;   /* dxo: [2M] */
        double *al = dxo + 2 * M, *dal = al + (size_t)H * nbs;
        double *xqr = xq + (size_t)r * D_q, *xor_ = xo + (size_t)r * 2 * M;
        memcpy(xqr, sv, sizeof(double) * M);
        orc_time_encode(D_t, c->omega, c->beta, 0.0, xqr + M);
        matvec(M, D_q, c->W_q, c->b_q, xqr, q);
        for (int j = 0; j < cr; ++j) {
            const size_t sl = (size_t)r * nb + j;
            double *kp = kap + sl * D_kv;
            memcpy(kp, sn + (size_t)nbr_pos[sl] * M, sizeof(double) * M);
            for (int d = 0; d < D_e; ++d)
                kp[M + d] = (double)c->efeat[(size_t)eid[sl] * D_e + d];
            orc_time_encode(D_t, c->omega, c->beta, rts[r] - nts[sl], kp + M + D_e);
            matvec(M, D_kv, c->W_k, c->b_k, kp, K + (size_t)j * M);
            matvec(M, D_kv, c->W_v, c->b_v, kp, V + (size_t)j * M);
        }
        for (int k = 0; k < M; ++k)
            xor_[k] = 0.0;
        for (int eta = 0; eta < H && cr > 0; ++eta) {
            const int o0 = eta * d_h;
            double mx = -INFINITY, den = 0.0;
            for (int j = 0; j < cr; ++j) {
                double dot = 0.0;
                for (int k = 0; k < d_h; ++k)
                    dot += q[o0 + k] * K[(size_t)j * M + o0 + k];
                al[eta * nbs + j] = dot * scale;
                if (al[eta * nbs + j] > mx)
                    mx = al[eta * nbs + j];
            }
            for (int j = 0; j < cr; ++j) {
                al[eta * nbs + j] = exp(al[eta * nbs + j] - mx);
                den += al[eta * nbs + j];
            }
            for (int j = 0; j < cr; ++j) {
                al[eta * nbs + j] /= den;
                for (int k = 0; k < d_h; ++k)
                    xor_[o0 + k] += al[eta * nbs + j] * V[(size_t)j * M + o0 + k];
            }
        }
        memcpy(xor_ + M, sv, sizeof(double) * M);
        matvec(M, 2 * M, c->W_o, c->b_o, xor_, o);
        double *dzr = dzo + (size_t)r * M;
        omarg[r] = INFINITY;
        for (int i = 0; i < M; ++i) {
            dzr[i] = o[i] > 0.0 ? dh[(size_t)r * M + i] : 0.0;
            omarg[r] = fmin(omarg[r], fabs(o[i]));
        }
        for (int k = 0; k < 2 * M; ++k) {
            double a = 0.0;
            for (int i = 0; i < M; ++i)
                a += c->W_o[(size_t)i * 2 * M + k] * dzr[i];
            dxo[k] = a;
        }
        /* dxo[0, M): the gradient of the attention output a; [M, 2M): of s_v */
        double *dqr = dq + (size_t)r * M;
        for (int eta = 0; eta < H && cr > 0; ++eta) {
            const int o0 = eta * d_h;
            double sdot = 0.0;
            for (int j = 0; j < cr; ++j) {
                double a = 0.0;
                for (int k = 0; k < d_h; ++k)
                    a += dxo[o0 + k] * V[(size_t)j * M + o0 + k];
                dal[j] = a;
                sdot += al[eta * nbs + j] * a;
            }
            for (int j = 0; j < cr; ++j) {
                const double aj = al[eta * nbs + j];
                const double dsc = aj * (dal[j] - sdot);
                const size_t sl = (size_t)r * nb + j;
                for (int k = 0; k < d_h; ++k) {
                    dV[sl * M + o0 + k] = aj * dxo[o0 + k];
                    dK[sl * M + o0 + k] = dsc * q[o0 + k] * scale;
                    dqr[o0 + k] += dsc * K[(size_t)j * M + o0 + k] * scale;
                }
            }
        }
        double *dsr = ds_root + (size_t)r * M;
        for (int m = 0; m < M; ++m) {
            double a = dxo[M + m];
            for (int i = 0; i < M; ++i)
                a += c->W_q[(size_t)i * D_q + m] * dqr[i];
            dsr[m] = a;
        }
        for (int j = 0; j < cr; ++j) {
            const size_t sl = (size_t)r * nb + j;
            for (int m = 0; m < M; ++m) {
                double a = 0.0;
                for (int i = 0; i < M; ++i)
                    a += c->W_k[(size_t)i * D_kv + m] * dK[sl * M + i] +
                         c->W_v[(size_t)i * D_kv + m] * dV[sl * M + i];
                ds_slot[sl * M + m] = a;
            }
        }
        free(K);
    }
    for (int r = 0; r < R; ++r)
        margin = fmin(margin, omarg[r]);
    free(omarg);
    *margin_out = margin;
    /* the attention's weight gradients, one output row per thread */
    #pragma omp parallel for schedule(dynamic, 4)
    for (int i = 0; i < M; ++i) {
        for (int r = 0; r < R; ++r) {
            const double z = dzo[(size_t)r * M + i], d = dq[(size_t)r * M + i];
            gb_o[i] += z;
            gb_q[i] += d;
            for (int k = 0; k < 2 * M; ++k)
                gW_o[(size_t)i * 2 * M + k] += z * xo[(size_t)r * 2 * M + k];
            for (int k = 0; k < D_q; ++k)
                gW_q[(size_t)i * D_q + k] += d * xq[(size_t)r * D_q + k];
            for (int j = 0; j < cnt[r]; ++j) {
                const size_t sl = (size_t)r * nb + j;
                const double dk = dK[sl * M + i], dv = dV[sl * M + i];
                gb_k[i] += dk;
                gb_v[i] += dv;
                for (int k = 0; k < D_kv; ++k) {
                    gW_k[(size_t)i * D_kv + k] += dk * kap[sl * D_kv + k];
                    gW_v[(size_t)i * D_kv + k] += dv * kap[sl * D_kv + k];
                }
            }
        }
    }
    /* the gradient of every updated memory: its roots, then its slots */
    double *ds = (double *)calloc((size_t)nU * M + 1, sizeof(double));
    for (int r = 0; r < R; ++r)
        for (int m = 0; m < M; ++m)
            ds[(size_t)root_pos[r] * M + m] += ds_root[(size_t)r * M + m];
    for (int r = 0; r < R; ++r)
        for (int j = 0; j < cnt[r]; ++j) {
            const size_t sl = (size_t)r * nb + j;
            for (int m = 0; m < M; ++m)
                ds[(size_t)nbr_pos[sl] * M + m] += ds_slot[sl * M + m];
        }
    free(kap); free(dK); free(dV); free(ds_slot); free(xq); free(dq); free(xo); free(dzo);
    free(ds_root); free(dh);

    /* the memory updater (GRU), node by node for nodes with mail */
    double *X = (double *)calloc((size_t)nU * D_x + 1, sizeof(double));
    double *dGx = (double *)calloc((size_t)nU * 3 * M + 1, sizeof(double));
    double *dGh = (double *)calloc((size_t)nU * 3 * M + 1, sizeof(double));
    #pragma omp parallel for schedule(dynamic, 8)
    for (int k = 0; k < nU; ++k) {
        if (fver[k] < 0)
            continue;
        double *x = X + (size_t)k * D_x;
        const double *hm = fm + (size_t)k * M;
        memcpy(x, fl + (size_t)k * D_m, sizeof(double) * D_m);
        orc_time_encode(D_t, c->omega, c->beta, flts[k] - fmts[k], x + D_m);
        for (int j = 0; j < M; ++j) {
            double ir = c->b_ih[j], iz = c->b_ih[M + j], in_ = c->b_ih[2 * M + j];
            double hr = c->b_hh[j], hz = c->b_hh[M + j], hn = c->b_hh[2 * M + j];
            for (int q = 0; q < D_x; ++q) {
                ir += c->W_ih[(size_t)j * D_x + q] * x[q];
                iz += c->W_ih[(size_t)(M + j) * D_x + q] * x[q];
                in_ += c->W_ih[(size_t)(2 * M + j) * D_x + q] * x[q];
            }
            for (int q = 0; q < M; ++q) {
                hr += c->W_hh[(size_t)j * M + q] * hm[q];
                hz += c->W_hh[(size_t)(M + j) * M + q] * hm[q];
                hn += c->W_hh[(size_t)(2 * M + j) * M + q] * hm[q];
            }
            const double r = sigmoid(ir + hr), z = sigmoid(iz + hz), n = tanh(in_ + r * hn);
            const double d = ds[(size_t)k * M + j];
            const double dn = d * (1.0 - z), dz = d * (hm[j] - n);
            const double dan = dn * (1.0 - n * n);
            const double dar = dan * hn * r * (1.0 - r), daz = dz * z * (1.0 - z);
            double *gx = dGx + (size_t)k * 3 * M, *gh = dGh + (size_t)k * 3 * M;
            gx[j] = dar; gx[M + j] = daz; gx[2 * M + j] = dan;
            gh[j] = dar; gh[M + j] = daz; gh[2 * M + j] = dan * r;
        }
    }
    #pragma omp parallel for schedule(dynamic, 4)
    for (int i = 0; i < 3 * M; ++i) {
        for (int k = 0; k < nU; ++k) {
            if (fver[k] < 0)
                continue;
            const double gx = dGx[(size_t)k * 3 * M + i], gh = dGh[(size_t)k * 3 * M + i];
            gb_ih[i] += gx;
            gb_hh[i] += gh;
            for (int q = 0; q < D_x; ++q)
                gW_ih[(size_t)i * D_x + q] += gx * X[(size_t)k * D_x + q];
            for (int q = 0; q < M; ++q)
                gW_hh[(size_t)i * M + q] += gh * fm[(size_t)k * M + q];
        }
    }
    free(X); free(dGx); free(dGh); free(ds);
    return loss / b;
}

/* One optimizer step on theta with the gradient of the last iteration. */
static void optimizer_step(orc_ctx *c)
{
    c->opt_steps++;
    const int64_t n = c->n_params;
    if (c->opt == ORC_SGD) {
        for (int64_t k = 0; k < n; ++k)
            c->theta[k] -= c->lr * c->grad[k];
        return;
    }
    const double b1 = c->beta1, b2 = c->beta2;
    const double c1 = 1.0 - pow(b1, (double)c->opt_steps), c2 = 1.0 - pow(b2, (double)c->opt_steps);
    for (int64_t k = 0; k < n; ++k) {
        const double g = c->grad[k];
        c->m1[k] = b1 * c->m1[k] + (1.0 - b1) * g;
        c->m2[k] = b2 * c->m2[k] + (1.0 - b2) * g * g;
        const double mh = c->m1[k] / c1, vh = c->m2[k] / c2;
        c->theta[k] -= c->lr * mh / (sqrt(vh) + c->eps);
    }
}

/* One iteration of the stage.  Returns ORC_EEND when the stream is exhausted. */
int orc_step(void *p, orc_step_out *o)
{
    orc_ctx *c = (orc_ctx *)p;
    const int64_t i = c->next_iter;
    const int64_t lo = i * c->B;
    if (lo >= c->E)
        return ORC_EEND;
    const int64_t hi = (lo + c->B < c->E) ? lo + c->B : c->E;
    const int b = (int)(hi - lo);
    const int R = 3 * b, nb = c->nb, M = c->M, D_m = c->D_m, D_x = c->D_x;
    const int D_t = c->D_t, D_e = c->D_e, N = c->N;

    /* 0. snapshot: apply every queued write set of iteration <= i-1-s */
    while (c->nq > 0 && c->q[0].iter <= i - 1 - c->s)
        apply_oldest(c);

    /* 1. roots: sources, then destinations, then negatives, at the event time */
    int32_t *root = (int32_t *)malloc(sizeof(int32_t) * R);
    double *rts = (double *)malloc(sizeof(double) * R);
    for (int k = 0; k < b; ++k) {
        root[k] = c->src[lo + k];
        root[b + k] = c->dst[lo + k];
        root[2 * b + k] = c->neg[lo + k];
        rts[k] = rts[b + k] = rts[2 * b + k] = c->t[lo + k];
    }

    /* 2. temporal sampling */
    const size_t RS = (size_t)R * (nb > 0 ? nb : 1);
    int32_t *nbr = (int32_t *)malloc(sizeof(int32_t) * RS);
    int32_t *eid = (int32_t *)malloc(sizeof(int32_t) * RS);
    double *nts = (double *)malloc(sizeof(double) * RS);
    int32_t *cnt = (int32_t *)malloc(sizeof(int32_t) * R);
    for (int r = 0; r < R; ++r)
        sample_root(&c->adj, c->src, c->dst, c->t, root[r], rts[r], nb,
                    nbr + (size_t)r * nb, eid + (size_t)r * nb, nts + (size_t)r * nb, cnt + r);

    /* 3. node set: sorted unique ids of roots and valid neighbours */
    int32_t *ids = (int32_t *)malloc(sizeof(int32_t) * (R + RS));
    size_t nid = 0;
    for (int r = 0; r < R; ++r)
        ids[nid++] = root[r];
    for (size_t k = 0; k < (size_t)R * nb; ++k)
        if (nbr[k] >= 0)
            ids[nid++] = nbr[k];
    qsort(ids, nid, sizeof(int32_t), cmp_i32);
    int nU = 0;
    for (size_t k = 0; k < nid; ++k)
        if (nU == 0 || ids[k] != ids[nU - 1])
            ids[nU++] = ids[k];
    int32_t *pos = (int32_t *)malloc(sizeof(int32_t) * N);
    for (int v = 0; v < N; ++v)
        pos[v] = -1;
    for (int k = 0; k < nU; ++k)
        pos[ids[k]] = k;

    /* fetched rows from the snapshot */
    double *fm = (double *)malloc(sizeof(double) * (size_t)nU * M);
    double *fmts = (double *)malloc(sizeof(double) * nU);
    double *fl = (double *)malloc(sizeof(double) * ((size_t)nU * D_m + 1));
    double *flts = (double *)malloc(sizeof(double) * nU);
    int32_t *fver = (int32_t *)malloc(sizeof(int32_t) * nU);
    for (int k = 0; k < nU; ++k) {
        const int v = ids[k];
        memcpy(fm + (size_t)k * M, c->mem + (size_t)v * M, sizeof(double) * M);
        memcpy(fl + (size_t)k * D_m, c->mail + (size_t)v * D_m, sizeof(double) * D_m);
        fmts[k] = c->mem_ts[v];
        flts[k] = c->mail_ts[v];
        fver[k] = c->ver[v];
    }

    /* APAN: the fetched mailboxes */
    const int K = c->K_mb;
    double *fmb = NULL, *fmbt = NULL;
    int32_t *fmbc = NULL;
    if (c->kind == ORC_APAN) {
        fmb = (double *)malloc(sizeof(double) * ((size_t)nU * K * D_m + 1));
        fmbt = (double *)malloc(sizeof(double) * ((size_t)nU * K + 1));
        fmbc = (int32_t *)malloc(sizeof(int32_t) * (nU > 0 ? nU : 1));
        for (int k = 0; k < nU; ++k) {
            const int v = ids[k];
            memcpy(fmb + (size_t)k * K * D_m, c->mb + (size_t)v * K * D_m,
                   sizeof(double) * (size_t)K * D_m);
            memcpy(fmbt + (size_t)k * K, c->mb_ts + (size_t)v * K, sizeof(double) * K);
            fmbc[k] = c->mb_cnt[v];
        }
    }

    /* 3b. staleness mitigation of the fetched memories (when enabled); the
     * fetched rows are reported as read, the mitigated ones separately */
    double *fm_read = NULL, gamma = 0.0;
    int n_stale = 0;
    if (c->mit_on && nU > 0) {
        fm_read = (double *)malloc(sizeof(double) * (size_t)nU * M);
        memcpy(fm_read, fm, sizeof(double) * (size_t)nU * M);
        gamma = mitigate(&c->adj, c->src, c->dst, c->t, nb, c->t[lo], nU, ids, fm, fmts, M,
                         c->mit_p, c->mit_lambda, c->mit_K, o ? o->m_stale : NULL,
                         o ? o->m_omega : NULL, &n_stale);
    }

    /* 4. memory update of every node in U that holds mail */
    double *sn = (double *)malloc(sizeof(double) * (size_t)nU * M);
    double *nmts = (double *)malloc(sizeof(double) * nU);
    if (c->kind == ORC_APAN) {
        /* APAN's memory updater: the node's mailbox aggregated by attention
         * (query from its memory, keys from each mail with the encoding of
         * its age relative to the newest mail, the mails as values), then
         * the GRU on [aggregate || phi(newest mail time - memory time)] */
        const int D_mk = D_m + D_t;
        const double scale = 1.0 / sqrt((double)M);
        #pragma omp parallel for schedule(dynamic, 8)
        for (int k = 0; k < nU; ++k) {
            const int cntk = fmbc[k];
            const double *hm = fm + (size_t)k * M;
            if (cntk == 0) {
                memcpy(sn + (size_t)k * M, hm, sizeof(double) * M);
                nmts[k] = fmts[k];
                continue;
            }
            const double *rows = fmb + (size_t)k * K * D_m, *ts = fmbt + (size_t)k * K;
            const double tref = ts[cntk - 1];
            double *buf = (double *)malloc(sizeof(double) * ((size_t)M + D_t + M + D_mk + M +
                                                              K + D_x));
            double *xq = buf, *q = xq + M + D_t, *kap = q + M, *kk = kap + D_mk, *sc = kk + M;
            double *x = sc + K;
            memcpy(xq, hm, sizeof(double) * M);
            orc_time_encode(D_t, c->omega, c->beta, 0.0, xq + M);
            matvec(M, M + D_t, c->W_q, c->b_q, xq, q);
            double mx = -INFINITY;
            for (int j = 0; j < cntk; ++j) {
                memcpy(kap, rows + (size_t)j * D_m, sizeof(double) * D_m);
                orc_time_encode(D_t, c->omega, c->beta, tref - ts[j], kap + D_m);
                matvec(M, D_mk, c->W_k, c->b_k, kap, kk);
                double dot = 0.0;
                for (int i2 = 0; i2 < M; ++i2)
                    dot += q[i2] * kk[i2];
                sc[j] = dot * scale;
                if (sc[j] > mx)
                    mx = sc[j];
            }
            double den = 0.0;
            for (int j = 0; j < cntk; ++j) {
                sc[j] = exp(sc[j] - mx);
                den += sc[j];
            }
            for (int d = 0; d < D_m; ++d)
                x[d] = 0.0;
            for (int j = 0; j < cntk; ++j)
                for (int d = 0; d < D_m; ++d)
                    x[d] += (sc[j] / den) * rows[(size_t)j * D_m + d];
            orc_time_encode(D_t, c->omega, c->beta, tref - fmts[k], x + D_m);
            orc_gru_cell(M, D_x, c->W_ih, c->W_hh, c->b_ih, c->b_hh, x, hm, sn + (size_t)k * M);
            nmts[k] = tref;
            free(buf);
        }
    } else {
    #pragma omp parallel for schedule(dynamic, 8)
    for (int k = 0; k < nU; ++k) {
        if (fver[k] >= 0) {
            double *x = (double *)malloc(sizeof(double) * D_x);
            memcpy(x, fl + (size_t)k * D_m, sizeof(double) * D_m);
            orc_time_encode(D_t, c->omega, c->beta, flts[k] - fmts[k], x + D_m);
            if (c->kind == ORC_JODIE)
                orc_rnn_cell(M, D_x, c->W_ih, c->W_hh, c->b_ih, c->b_hh, x, fm + (size_t)k * M,
                             sn + (size_t)k * M);
            else
                orc_gru_cell(M, D_x, c->W_ih, c->W_hh, c->b_ih, c->b_hh, x, fm + (size_t)k * M,
                             sn + (size_t)k * M);
            nmts[k] = flts[k];
            free(x);
        } else {
            memcpy(sn + (size_t)k * M, fm + (size_t)k * M, sizeof(double) * M);
            nmts[k] = fmts[k];
        }
    }
    }

    /* 5. embeddings of every root */
    double *h = (double *)malloc(sizeof(double) * (size_t)R * M);
    orc_attn_w aw = {M, D_e, D_t, c->H, c->omega, c->beta, c->W_q, c->b_q, c->W_k, c->b_k,
                     c->W_v, c->b_v, c->W_o, c->b_o};
    #pragma omp parallel for schedule(dynamic, 8)
    for (int r = 0; r < R; ++r) {
        if (c->kind == ORC_APAN) {   /* APAN's embedding: the updated memory */
            memcpy(h + (size_t)r * M, sn + (size_t)pos[root[r]] * M, sizeof(double) * M);
            continue;
        }
        if (c->kind == ORC_JODIE) {
            const int pr = pos[root[r]];
            orc_time_projection(M, c->w_t, sn + (size_t)pr * M, nmts[pr], rts[r],
                                h + (size_t)r * M);
            continue;
        }
        const int cr = cnt[r];
        const double **pu = (const double **)malloc(sizeof(void *) * (nb > 0 ? nb : 1));
        const double **pf = (const double **)malloc(sizeof(void *) * (nb > 0 ? nb : 1));
        double *frow = (double *)malloc(sizeof(double) * ((size_t)(nb > 0 ? nb : 1) * D_e + 1));
        for (int j = 0; j < cr; ++j) {
            const size_t sl = (size_t)r * nb + j;
            pu[j] = sn + (size_t)pos[nbr[sl]] * M;
            for (int d = 0; d < D_e; ++d)
                frow[(size_t)j * D_e + d] = (double)c->efeat[(size_t)eid[sl] * D_e + d];
            pf[j] = frow + (size_t)j * D_e;
        }
        embed_root(&aw, sn + (size_t)pos[root[r]] * M, rts[r], cr, pu, pf,
                   nts + (size_t)r * nb, h + (size_t)r * M);
        free(pu); free(pf); free(frow);
    }

    /* 6-7. messages of the positive events and the latest-message reduce:
     * per endpoint node, the candidate (t, e, role) that is largest wins */
    int64_t *win = (int64_t *)malloc(sizeof(int64_t) * (nU > 0 ? nU : 1));
    for (int k = 0; k < nU; ++k)
        win[k] = -1;
    for (int64_t e = lo; e < hi; ++e) {
        for (int role = 0; role < 2; ++role) {
            const int w = role == 0 ? c->src[e] : c->dst[e];
            const int k = pos[w];
            const int64_t cand = 2 * e + role;
            if (win[k] < 0) {
                win[k] = cand;
            } else {
                const int64_t e0 = win[k] / 2;
                const int r0 = (int)(win[k] % 2);
                const int later = (c->t[e] > c->t[e0]) ||
                                  (c->t[e] == c->t[e0] && (e > e0 || (e == e0 && role > r0)));
                if (later)
                    win[k] = cand;
            }
        }
    }

    /* 8. write set of iteration i: updated memory and the winning message */
    orc_wset W;
    memset(&W, 0, sizeof(W));
    W.iter = i;
    int nw = 0;
    for (int k = 0; k < nU; ++k)
        nw += win[k] >= 0;
    W.n = nw;
    W.node = (int32_t *)malloc(sizeof(int32_t) * (nw ? nw : 1));
    W.mem = (double *)malloc(sizeof(double) * ((size_t)nw * M + 1));
    W.mem_ts = (double *)malloc(sizeof(double) * (nw ? nw : 1));
    W.mail = (double *)malloc(sizeof(double) * ((size_t)nw * D_m + 1));
    W.mail_ts = (double *)malloc(sizeof(double) * (nw ? nw : 1));
    int w_ = 0;
    for (int k = 0; k < nU; ++k) {
        if (win[k] < 0)
            continue;
        const int64_t e = win[k] / 2;
        const int role = (int)(win[k] % 2);
        const int other = role == 0 ? c->dst[e] : c->src[e];
        W.node[w_] = ids[k];
        memcpy(W.mem + (size_t)w_ * M, sn + (size_t)k * M, sizeof(double) * M);
        W.mem_ts[w_] = nmts[k];
        double *ml = W.mail + (size_t)w_ * D_m;
        memcpy(ml, sn + (size_t)k * M, sizeof(double) * M);
        memcpy(ml + M, sn + (size_t)pos[other] * M, sizeof(double) * M);
        for (int d = 0; d < D_e; ++d)
            ml[2 * M + d] = (double)c->efeat[(size_t)e * D_e + d];
        W.mail_ts[w_] = c->t[e];
        ++w_;
    }
    /* APAN: the mails of the batch, in (t, e, role) order, each to its node
     * and (with propagation) then to the node's sampled neighbours at the
     * event's time, in slot order */
    if (c->kind == ORC_APAN) {
        const int per = 1 + (c->propagate ? nb : 0);
        W.del_node = (int32_t *)malloc(sizeof(int32_t) * ((size_t)2 * b * per + 1));
        W.del_mail = (double *)malloc(sizeof(double) * ((size_t)2 * b * per * D_m + 1));
        W.del_t = (double *)malloc(sizeof(double) * ((size_t)2 * b * per + 1));
        int nd = 0;
        for (int64_t e = lo; e < hi; ++e)
            for (int role = 0; role < 2; ++role) {
                const int v = role == 0 ? c->src[e] : c->dst[e];
                const int other = role == 0 ? c->dst[e] : c->src[e];
                const int r = role * b + (int)(e - lo);   /* v's root in this batch */
                const int nrecv = 1 + (c->propagate ? cnt[r] : 0);
                for (int hop = 0; hop < nrecv; ++hop) {
                    const int w = hop == 0 ? v : nbr[(size_t)r * nb + hop - 1];
                    double *ml = W.del_mail + (size_t)nd * D_m;
                    memcpy(ml, sn + (size_t)pos[v] * M, sizeof(double) * M);
                    memcpy(ml + M, sn + (size_t)pos[other] * M, sizeof(double) * M);
                    for (int d = 0; d < D_e; ++d)
                        ml[2 * M + d] = (double)c->efeat[(size_t)e * D_e + d];
                    W.del_node[nd] = w;
                    W.del_t[nd] = c->t[e];
                    ++nd;
                }
            }
        W.n_del = nd;
    }
    if (c->nq == c->capq) {
        c->capq *= 2;
        c->q = (orc_wset *)realloc(c->q, sizeof(orc_wset) * (size_t)c->capq);
    }
    c->q[c->nq++] = W;

    /* 9. training (when enabled): loss and gradient of this iteration, then
     * the optimizer step (the next iteration runs with the new weights) */
    double loss = 0.0, margin = INFINITY;
    if (c->train_on) {
        int32_t *rp = (int32_t *)malloc(sizeof(int32_t) * R);
        int32_t *np_ = (int32_t *)malloc(sizeof(int32_t) * (RS ? RS : 1));
        for (int r = 0; r < R; ++r)
            rp[r] = pos[root[r]];
        for (size_t k = 0; k < (size_t)R * nb; ++k)
            np_[k] = nbr[k] >= 0 ? pos[nbr[k]] : -1;
        loss = train_gradient(c, b, R, nU, rp, rts, np_, eid, nts, cnt, fm, fmts, fl, flts,
                              fver, sn, h, &margin);
        optimizer_step(c);
        free(rp);
        free(np_);
    }

    /* outputs */
    if (o) {
        o->loss = loss;
        o->relu_margin = margin;
        if (fmb && o->f_mb)
            memcpy(o->f_mb, fmb, sizeof(double) * (size_t)nU * K * D_m);
        if (fmbt && o->f_mb_ts)
            memcpy(o->f_mb_ts, fmbt, sizeof(double) * (size_t)nU * K);
        if (fmbc && o->f_mb_cnt)
            memcpy(o->f_mb_cnt, fmbc, sizeof(int32_t) * (size_t)nU);
        if (c->train_on && o->grad)
            memcpy(o->grad, c->grad, sizeof(double) * (size_t)c->n_params);
        if (c->train_on && o->params)
            memcpy(o->params, c->theta, sizeof(double) * (size_t)c->n_params);
        o->iter = i; o->b = b; o->R = R; o->n_U = nU;
        if (o->root) memcpy(o->root, root, sizeof(int32_t) * R);
        if (o->root_ts) memcpy(o->root_ts, rts, sizeof(double) * R);
        if (o->nbr) memcpy(o->nbr, nbr, sizeof(int32_t) * (size_t)R * nb);
        if (o->eid) memcpy(o->eid, eid, sizeof(int32_t) * (size_t)R * nb);
        if (o->nts) memcpy(o->nts, nts, sizeof(double) * (size_t)R * nb);
        if (o->cnt) memcpy(o->cnt, cnt, sizeof(int32_t) * R);
        if (o->U) memcpy(o->U, ids, sizeof(int32_t) * nU);
        if (o->root_pos)
            for (int r = 0; r < R; ++r) o->root_pos[r] = pos[root[r]];
        if (o->nbr_pos)
            for (size_t k = 0; k < (size_t)R * nb; ++k)
                o->nbr_pos[k] = nbr[k] >= 0 ? pos[nbr[k]] : -1;
        if (o->f_mem) memcpy(o->f_mem, fm_read ? fm_read : fm, sizeof(double) * (size_t)nU * M);
        if (o->m_mem) memcpy(o->m_mem, fm, sizeof(double) * (size_t)nU * M);
        if (o->x_mem) {
            /* the committed rows, then the queued write sets of iterations
             * before i in order (a later write wins) */
            for (int k = 0; k < nU; ++k)
                memcpy(o->x_mem + (size_t)k * M, c->mem + (size_t)ids[k] * M,
                       sizeof(double) * M);
            for (int q = 0; q < c->nq && c->q[q].iter < i; ++q)   /* not W_i */
                for (int j = 0; j < c->q[q].n; ++j)
                    if (pos[c->q[q].node[j]] >= 0)
                        memcpy(o->x_mem + (size_t)pos[c->q[q].node[j]] * M,
                               c->q[q].mem + (size_t)j * M, sizeof(double) * M);
        }
        o->m_gamma = gamma;
        o->m_n_stale = n_stale;
        if (o->f_mem_ts) memcpy(o->f_mem_ts, fmts, sizeof(double) * nU);
        if (o->f_mail) memcpy(o->f_mail, fl, sizeof(double) * (size_t)nU * D_m);
        if (o->f_mail_ts) memcpy(o->f_mail_ts, flts, sizeof(double) * nU);
        if (o->f_ver) memcpy(o->f_ver, fver, sizeof(int32_t) * nU);
        if (o->s_new) memcpy(o->s_new, sn, sizeof(double) * (size_t)nU * M);
        if (o->new_mem_ts) memcpy(o->new_mem_ts, nmts, sizeof(double) * nU);
        if (o->h) memcpy(o->h, h, sizeof(double) * (size_t)R * M);
        if (o->winner) memcpy(o->winner, win, sizeof(int64_t) * nU);
    }

    free(root); free(rts); free(nbr); free(eid); free(nts); free(cnt); free(ids); free(pos);
    free(fm); free(fmts); free(fl); free(flts); free(fver); free(sn); free(nmts); free(h);
    free(fm_read);
    free(fmb); free(fmbt); free(fmbc);
    free(win);
    c->next_iter = i + 1;
    return ORC_OK;
}

/* Thread count of the OpenMP loops (over independent nodes and roots; every
 * sum has a fixed order, so results do not depend on it).  n < 1 leaves it
 * unchanged.  Returns the count the next loops will use. */
int orc_set_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}
