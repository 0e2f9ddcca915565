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
    gather_rows<true>(g, p0, n, threadIdx.x & 63);
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
    for (hipEvent_t e : st->run_ev)
        if (e)
            hipEventDestroy(e);
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
    bool ok = dev_malloc(&st->mem, sizeof(float) * N * (size_t)M) == hipSuccess &&
              dev_malloc(&st->mem_ts, sizeof(double) * N) == hipSuccess &&
              dev_malloc(&st->mail, sizeof(float) * (N * (size_t)D_m + 1)) == hipSuccess &&
              dev_malloc(&st->mail_ts, sizeof(double) * N) == hipSuccess &&
              dev_malloc(&st->ver, sizeof(int32_t) * N) == hipSuccess &&
              dev_malloc(&st->r_flag, sizeof(int32_t) * rows) == hipSuccess &&
              dev_malloc(&st->r_node, sizeof(int32_t) * rows) == hipSuccess &&
              dev_malloc(&st->r_mem, sizeof(float) * rows * M) == hipSuccess &&
              dev_malloc(&st->r_mail, sizeof(float) * (rows * D_m + 1)) == hipSuccess &&
              dev_malloc(&st->r_mem_ts, sizeof(double) * rows) == hipSuccess &&
              dev_malloc(&st->r_mail_ts, sizeof(double) * rows) == hipSuccess &&
              dev_malloc(&st->win, sizeof(uint64_t) * N) == hipSuccess &&
              dev_malloc(&st->xwin, sizeof(uint64_t) * N * (size_t)TGM_MAX_SAMPLE_SETS) ==
                  hipSuccess;
    if (!ok) {
        tgm_state_destroy(st);
        return TGM_ENOMEM;
    }
    // the executor's latest-message key arrays: one per sample buffer set,
    // indexed by node-set position (< N); zero keys are older than every tag
    st->xwin_slots = TGM_MAX_SAMPLE_SETS;
    st->xwin_cap = N;
    st->xwin_tag = 0;
    for (hipEvent_t &e : st->run_ev)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
            tgm_state_destroy(st);
            return TGM_EDEVICE;
        }
    if (hipMemsetAsync(st->xwin, 0, sizeof(uint64_t) * N * (size_t)TGM_MAX_SAMPLE_SETS,
                       as_stream(stream)) != hipSuccess) {
        tgm_state_destroy(st);
        return TGM_EDEVICE;
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

// ============================================================== checkpoints
//
// A checkpoint is the whole versioned state: the committed tables, the ring
// of staged write sets (the s pending updates a fetch has not needed yet) and
// the protocol counters.  Layout (host bytes, every section 8-byte aligned):
//   int64 header[kCkptHeader]: magic, format, N, M, D_m, s, max_batch,
//         committed_through, staged_through, last_fetch, slots (= s + 1)
//   int64 slot[slots][3]: iteration, b, staged
//   mem [N x M] f32, mem_ts [N] f64, mail [N x D_m] f32, mail_ts [N] f64,
//   ver [N] i32, then the ring rows (slots x 2 max_batch rows): r_flag i32,
//   r_node i32, r_mem [x M] f32, r_mail [x D_m] f32, r_mem_ts f64,
//   r_mail_ts f64.
// The latest-message keys (win, xwin) are not part of it: they are scratch of
// one update call, filtered by a tag that only grows in the state they live in.

namespace {

constexpr int64_t kCkptMagic = 0x74676d2d636b7074LL;   // "tgm-ckpt"
constexpr int64_t kCkptFormat = 1;
constexpr int kCkptHeader = 11;

struct CkptSection {
    void *dev;
    size_t bytes;
};

size_t align8(size_t x) { return (x + 7) & ~(size_t)7; }

// the device arrays of a state in checkpoint order
std::vector<CkptSection> ckpt_sections(const tgm_state *st)
{
    const size_t N = st->N, M = st->M, Dm = st->D_m;
    const size_t rows = (size_t)(st->s + 1) * st->ring_rows();
    return {{st->mem, sizeof(float) * N * M},       {st->mem_ts, sizeof(double) * N},
            {st->mail, sizeof(float) * N * Dm},     {st->mail_ts, sizeof(double) * N},
            {st->ver, sizeof(int32_t) * N},         {st->r_flag, sizeof(int32_t) * rows},
            {st->r_node, sizeof(int32_t) * rows},   {st->r_mem, sizeof(float) * rows * M},
            {st->r_mail, sizeof(float) * rows * Dm}, {st->r_mem_ts, sizeof(double) * rows},
            {st->r_mail_ts, sizeof(double) * rows}};
}

size_t ckpt_meta_bytes(const tgm_state *st)
{
    return sizeof(int64_t) * (kCkptHeader + 3 * (size_t)(st->s + 1));
}

size_t ckpt_bytes(const tgm_state *st)
{
    size_t b = ckpt_meta_bytes(st);
    for (const CkptSection &c : ckpt_sections(st))
        b += align8(c.bytes);
    return b;
}

}  // namespace

extern "C" tgm_status_t tgm_state_checkpoint_bytes(tgm_state_t st, size_t *bytes)
{
    if (!st || !bytes)
        return TGM_EINVAL;
    *bytes = ckpt_bytes(st);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_save(tgm_state_t st, void *buf, size_t bytes, void *stream)
{
    if (!st || !buf)
        return TGM_EINVAL;
    if (bytes < ckpt_bytes(st))
        return TGM_ESIZE;
    hipStream_t s = as_stream(stream);
    char *p = static_cast<char *>(buf);
    int64_t *h = reinterpret_cast<int64_t *>(p);
    const int64_t head[kCkptHeader] = {kCkptMagic,          kCkptFormat,        st->N,
                                       st->M,               st->D_m,            st->s,
                                       st->max_batch,       st->committed_through,
                                       st->staged_through,  st->last_fetch,     st->s + 1};
    for (int k = 0; k < kCkptHeader; ++k)
        h[k] = head[k];
    for (int j = 0; j <= st->s; ++j) {
        h[kCkptHeader + 3 * j] = st->ring[j].iter;
        h[kCkptHeader + 3 * j + 1] = st->ring[j].b;
        h[kCkptHeader + 3 * j + 2] = st->ring[j].staged ? 1 : 0;
    }
    p += ckpt_meta_bytes(st);
    for (const CkptSection &c : ckpt_sections(st)) {
        if (c.bytes)
            TGM_HIP(hipMemcpyAsync(p, c.dev, c.bytes, hipMemcpyDeviceToHost, s));
        p += align8(c.bytes);
    }
    TGM_HIP(hipStreamSynchronize(s));
    return TGM_OK;
}

extern "C" tgm_status_t tgm_state_restore(tgm_state_t st, const void *buf, size_t bytes,
                                          void *stream)
{
    if (!st || !buf)
        return TGM_EINVAL;
    if (bytes < sizeof(int64_t) * kCkptHeader)
        return TGM_ESIZE;
    const int64_t *h = static_cast<const int64_t *>(buf);
    if (h[0] != kCkptMagic || h[1] != kCkptFormat || h[2] != st->N || h[3] != st->M ||
        h[4] != st->D_m || h[5] != st->s || h[6] != st->max_batch || h[10] != st->s + 1)
        return TGM_EINVAL;
    if (bytes < ckpt_bytes(st))
        return TGM_ESIZE;
    // the counters must describe a state the protocol can reach
    const int64_t committed = h[7], staged = h[8], last_fetch = h[9];
    if (committed < -1 || staged < committed || staged - committed > st->s + 1)
        return TGM_EINVAL;
    std::vector<tgm_state::Slot> ring(st->s + 1);
    for (int j = 0; j <= st->s; ++j) {
        const int64_t it = h[kCkptHeader + 3 * j], b = h[kCkptHeader + 3 * j + 1],
                      on = h[kCkptHeader + 3 * j + 2];
        if (b < 0 || b > st->max_batch || (on != 0 && on != 1))
            return TGM_EINVAL;
        ring[j].iter = it;
        ring[j].b = (int32_t)b;
        ring[j].staged = on == 1;
    }
    for (int64_t j = committed + 1; j <= staged; ++j) {
        const tgm_state::Slot &sl = ring[j % (st->s + 1)];
        if (!sl.staged || sl.iter != j)
            return TGM_EINVAL;
    }
    hipStream_t s = as_stream(stream);
    const char *p = static_cast<const char *>(buf) + ckpt_meta_bytes(st);
    for (const CkptSection &c : ckpt_sections(st)) {
        if (c.bytes)
            TGM_HIP(hipMemcpyAsync(c.dev, p, c.bytes, hipMemcpyHostToDevice, s));
        p += align8(c.bytes);
    }
    TGM_HIP(hipStreamSynchronize(s));
    st->ring = ring;
    st->committed_through = committed;
    st->staged_through = staged;
    st->last_fetch = last_fetch;
    return TGM_OK;
}
