// Node memory / mailbox tables, the staleness-bounded write-back ring, and
// the versioned fetch.
#include <algorithm>

#include "common.h"

using namespace tgm;

namespace {

__global__ void k_state_init(int32_t N, int32_t M, int32_t D_m, float *__restrict__ mem,
                             double *__restrict__ mem_ts, float *__restrict__ mail,
                             double *__restrict__ mail_ts, int32_t *__restrict__ ver,
                             uint64_t *__restrict__ win)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (int64_t k = t0; k < (int64_t)N * M; k += stride)
        mem[k] = 0.f;
    for (int64_t k = t0; k < (int64_t)N * D_m; k += stride)
        mail[k] = 0.f;
    for (int64_t k = t0; k < N; k += stride) {
        mem_ts[k] = 0.0;
        mail_ts[k] = 0.0;
        ver[k] = -1;
        win[k] = 0;
    }
}

// Commit one staged write set: one wavefront per candidate slot; flagged
// slots (the latest message of their node) overwrite the node's rows.  Nodes
// are distinct within a write set, so slots never collide.
__global__ __launch_bounds__(256) void k_commit(
    int32_t n_cand, int64_t iter, int32_t M, int32_t D_m, const int32_t *__restrict__ flag,
    const int32_t *__restrict__ node, const float *__restrict__ r_mem,
    const double *__restrict__ r_mem_ts, const float *__restrict__ r_mail,
    const double *__restrict__ r_mail_ts, float *__restrict__ mem, double *__restrict__ mem_ts,
    float *__restrict__ mail, double *__restrict__ mail_ts, int32_t *__restrict__ ver)
{
    const int c = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6);
    const int lane = threadIdx.x & 63;
    if (c >= n_cand || !flag[c])
        return;
    const int32_t v = node[c];
    double mts = 0.0, lts = 0.0;
    if (lane == 0) {
        mts = r_mem_ts[c];
        lts = r_mail_ts[c];
    }
    wave_copy_2rows(mem + (int64_t)v * M, r_mem + (int64_t)c * M, M,
                    mail + (int64_t)v * D_m, r_mail + (int64_t)c * D_m, D_m, lane);
    if (lane == 0) {
        mem_ts[v] = mts;
        mail_ts[v] = lts;
        ver[v] = (int32_t)iter;
    }
}

// Gather the committed rows of the node set: one wavefront per kGatherNPW
// consecutive nodes.
__global__ __launch_bounds__(256) void k_gather_state(GatherPlan g)
{
    const int p0 = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6) * kGatherNPW;
    const int n = min(*g.n_nodes, g.cap);
    if (p0 >= n)
        return;
    gather_rows(g, p0, n, threadIdx.x & 63);
}

tgm_status_t commit_through(tgm_state *st, int64_t target, hipStream_t s)
{
    const int slots = st->s + 1;
    for (int64_t j = st->committed_through + 1; j <= target; ++j) {
        tgm_state::Slot &sl = st->ring[j % slots];
        if (!sl.staged || sl.iter != j)
            return TGM_EORDER;
        const int n_cand = 2 * sl.b;
        if (n_cand > 0) {
            const size_t base = (size_t)(j % slots) * st->ring_rows();
            TGM_LAUNCH(k_commit, dim3(cdiv(n_cand, 4)), dim3(256), 0, s, n_cand, j, st->M,
                               st->D_m, st->r_flag + base, st->r_node + base,
                               st->r_mem + base * st->M, st->r_mem_ts + base,
                               st->r_mail + base * st->D_m, st->r_mail_ts + base, st->mem,
                               st->mem_ts, st->mail, st->mail_ts, st->ver);
        }
        sl.staged = false;
        st->committed_through = j;
    }
    return TGM_OK;
}

}  // namespace

// ======================================================================== API

extern "C" tgm_status_t tgm_state_reset(tgm_state_t st, void *stream)
{
    if (!st)
        return TGM_EINVAL;
    hipLaunchKernelGGL(k_state_init, dim3(1024), dim3(256), 0, as_stream(stream), st->N, st->M,
                       st->D_m, st->mem, st->mem_ts, st->mail, st->mail_ts, st->ver, st->win);
    TGM_LAUNCHED();
    st->win_tag = 0;
    for (auto &sl : st->ring)
        sl = tgm_state::Slot();
    st->committed_through = -1;
    st->staged_through = -1;
    st->last_fetch = INT64_MIN;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_destroy(tgm_state_t st)
{
    if (!st)
        return TGM_EINVAL;
    hipFree(st->mem);
    hipFree(st->mem_ts);
    hipFree(st->mail);
    hipFree(st->mail_ts);
    hipFree(st->ver);
    hipFree(st->r_flag);
    hipFree(st->r_node);
    hipFree(st->r_mem);
    hipFree(st->r_mail);
    hipFree(st->r_mem_ts);
    hipFree(st->r_mail_ts);
    hipFree(st->win);
    hipFree(st->xwin);
    delete st;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_create(int32_t N, int32_t M, int32_t D_m, int32_t s,
                                         int32_t max_batch, void *stream, tgm_state_t *out)
{
    if (!out || N <= 0 || M <= 0 || D_m < 0 || s < 0 || max_batch <= 0)
        return TGM_EINVAL;
    *out = nullptr;
    tgm_state *st = new tgm_state();
    st->N = N;
    st->M = M;
    st->D_m = D_m;
    st->s = s;
    st->max_batch = max_batch;
    st->ring.resize(s + 1);
    const size_t rows = (size_t)(s + 1) * st->ring_rows();
    bool ok = hipMalloc(&st->mem, sizeof(float) * N * (size_t)M) == hipSuccess &&
              hipMalloc(&st->mem_ts, sizeof(double) * N) == hipSuccess &&
              hipMalloc(&st->mail, sizeof(float) * (N * (size_t)D_m + 1)) == hipSuccess &&
              hipMalloc(&st->mail_ts, sizeof(double) * N) == hipSuccess &&
              hipMalloc(&st->ver, sizeof(int32_t) * N) == hipSuccess &&
              hipMalloc(&st->r_flag, sizeof(int32_t) * rows) == hipSuccess &&
              hipMalloc(&st->r_node, sizeof(int32_t) * rows) == hipSuccess &&
              hipMalloc(&st->r_mem, sizeof(float) * rows * M) == hipSuccess &&
              hipMalloc(&st->r_mail, sizeof(float) * (rows * D_m + 1)) == hipSuccess &&
              hipMalloc(&st->r_mem_ts, sizeof(double) * rows) == hipSuccess &&
              hipMalloc(&st->r_mail_ts, sizeof(double) * rows) == hipSuccess &&
              hipMalloc(&st->win, sizeof(uint64_t) * N) == hipSuccess;
    if (!ok) {
        tgm_state_destroy(st);
        return TGM_ENOMEM;
    }
    tgm_status_t rc = tgm_state_reset(st, stream);
    if (rc != TGM_OK) {
        tgm_state_destroy(st);
        return rc;
    }
    *out = st;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_flush(tgm_state_t st, void *stream)
{
    if (!st)
        return TGM_EINVAL;
    return commit_through(st, st->staged_through, as_stream(stream));
}

extern "C" tgm_status_t tgm_state_read(tgm_state_t st, float *mem, double *mem_ts, float *mail,
                                       double *mail_ts, int32_t *ver, void *stream)
{
    if (!st)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t N = st->N;
    if (mem) TGM_HIP(hipMemcpyAsync(mem, st->mem, sizeof(float) * N * st->M, hipMemcpyDeviceToDevice, s));
    if (mem_ts) TGM_HIP(hipMemcpyAsync(mem_ts, st->mem_ts, sizeof(double) * N, hipMemcpyDeviceToDevice, s));
    if (mail && st->D_m) TGM_HIP(hipMemcpyAsync(mail, st->mail, sizeof(float) * N * st->D_m, hipMemcpyDeviceToDevice, s));
    if (mail_ts) TGM_HIP(hipMemcpyAsync(mail_ts, st->mail_ts, sizeof(double) * N, hipMemcpyDeviceToDevice, s));
    if (ver) TGM_HIP(hipMemcpyAsync(ver, st->ver, sizeof(int32_t) * N, hipMemcpyDeviceToDevice, s));
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_load(tgm_state_t st, int64_t iter, const float *mem,
                                       const double *mem_ts, const float *mail,
                                       const double *mail_ts, const int32_t *ver, void *stream)
{
    if (!st || iter < 0 || !mem || !mem_ts || (!mail && st->D_m) || !mail_ts || !ver)
        return TGM_EINVAL;
    hipStream_t s = as_stream(stream);
    const size_t N = st->N;
    TGM_HIP(hipMemcpyAsync(st->mem, mem, sizeof(float) * N * st->M, hipMemcpyDeviceToDevice, s));
    TGM_HIP(hipMemcpyAsync(st->mem_ts, mem_ts, sizeof(double) * N, hipMemcpyDeviceToDevice, s));
    if (st->D_m)
        TGM_HIP(hipMemcpyAsync(st->mail, mail, sizeof(float) * N * st->D_m, hipMemcpyDeviceToDevice, s));
    TGM_HIP(hipMemcpyAsync(st->mail_ts, mail_ts, sizeof(double) * N, hipMemcpyDeviceToDevice, s));
    TGM_HIP(hipMemcpyAsync(st->ver, ver, sizeof(int32_t) * N, hipMemcpyDeviceToDevice, s));
    for (auto &sl : st->ring)
        sl = tgm_state::Slot();
    st->committed_through = iter - 1;
    st->staged_through = iter - 1;
    st->last_fetch = INT64_MIN;
    return TGM_OK;
}

tgm_status_t tgm::fetch_plan(tgm_state_t st, int64_t iter, const int32_t *nodes,
                             const int32_t *n_nodes, int32_t cap, float *mem, double *mem_ts,
                             float *mail, double *mail_ts, int32_t *ver, hipStream_t s,
                             GatherPlan *plan)
{
    if (!st || iter < 0 || cap < 0 || !n_nodes)
        return TGM_EINVAL;
    if (cap > 0 && (!nodes || !mem || !mem_ts || (!mail && st->D_m) || !mail_ts || !ver))
        return TGM_EINVAL;
    if (cap > st->N)
        return TGM_ESIZE;
    if (iter < st->last_fetch)
        return TGM_EORDER;
    const int64_t target = iter - 1 - st->s;
    if (target > st->staged_through)
        return TGM_EORDER;
    tgm_status_t rc = commit_through(st, target, s);
    if (rc != TGM_OK)
        return rc;
    st->last_fetch = iter;
    GatherPlan p;
    p.nodes = nodes; p.n_nodes = n_nodes; p.cap = cap; p.M = st->M; p.D_m = st->D_m;
    p.mem = st->mem; p.mail = st->mail; p.mem_ts = st->mem_ts; p.mail_ts = st->mail_ts;
    p.ver = st->ver;
    p.o_mem = mem; p.o_mail = mail; p.o_mem_ts = mem_ts; p.o_mail_ts = mail_ts; p.o_ver = ver;
    *plan = p;
    return TGM_OK;
}

tgm_status_t tgm::launch_gather(const GatherPlan &plan, hipStream_t s)
{
    if (plan.cap == 0)
        return TGM_OK;
    TGM_LAUNCH(k_gather_state, dim3(cdiv(plan.cap, 4 * kGatherNPW)), dim3(256), 0, s, plan);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_fetch_memory(tgm_state_t st, int64_t iter, const int32_t *nodes,
                                         const int32_t *n_nodes, int32_t cap, float *mem,
                                         double *mem_ts, float *mail, double *mail_ts,
                                         int32_t *ver, void *stream)
{
    GatherPlan plan;
    const hipStream_t s = as_stream(stream);
    const tgm_status_t rc =
        fetch_plan(st, iter, nodes, n_nodes, cap, mem, mem_ts, mail, mail_ts, ver, s, &plan);
    return rc != TGM_OK ? rc : launch_gather(plan, s);
}
