// Pipelined executor of the stage.  The sample and node set of an iteration
// depend on the event stream only, so they run a chunk of iterations ahead on
// a second stream; the fetch, update and embedding run in iteration order on
// the main stream (each update commits the write set the next fetch needs).
// Cross-stream waits are host calls of several microseconds each, so the
// streams synchronise once per chunk, not once per iteration.
#include <hip/hip_runtime.h>

#include "common.h"

using namespace tgm;

namespace {

struct Events {
    hipEvent_t e[5] = {nullptr, nullptr, nullptr, nullptr, nullptr};
    ~Events()
    {
        for (hipEvent_t x : e)
            if (x)
                hipEventDestroy(x);
    }
    bool create()
    {
        for (hipEvent_t &x : e)
            if (hipEventCreateWithFlags(&x, hipEventDisableTiming) != hipSuccess)
                return false;
        return true;
    }
};

#define TGM_TRY(call)                      \
    do {                                   \
        const tgm_status_t st_ = (call);   \
        if (st_ != TGM_OK)                 \
            return st_;                    \
    } while (0)

}  // namespace

extern "C" tgm_status_t tgm_stage_run(tgm_graph_t g, tgm_state_t st, tgm_model_t m,
                                      int64_t i0, int64_t n, int32_t B, int32_t nb, int32_t cap,
                                      const tgm_sample_buffers *sb, int32_t nsb,
                                      const tgm_fetch_buffers *fb, float *mem_new,
                                      double *new_mem_ts, int64_t *winner, float *h,
                                      void *stream, void *prefetch_stream)
{
    if (!g || !st || !m || !sb || !fb || i0 < 0 || n < 0 || B < 1 || !mem_new || !h)
        return TGM_EINVAL;
    if (nsb < 2 || (nsb & 1))
        return TGM_EINVAL;
    if (n == 0)
        return TGM_OK;
    if ((i0 + n - 1) * (int64_t)B >= g->E)
        return TGM_EINVAL;   // past the last batch
    hipStream_t main = as_stream(stream), pre = as_stream(prefetch_stream);
    if (main == pre)
        return TGM_EINVAL;
    Events ev;   // 0-1: sampled chunk by parity, 2-3: computed chunk by parity, 4: start
    if (!ev.create())
        return TGM_EDEVICE;
    const int64_t K = nsb / 2;                 // iterations per chunk
    const int64_t nch = (n + K - 1) / K;
    auto sample_chunk = [&](int64_t c) -> tgm_status_t {
        for (int64_t k = c * K; k < std::min(n, (c + 1) * K); ++k) {
            const int64_t lo = (i0 + k) * B;
            const int32_t b = (int32_t)std::min<int64_t>(B, g->E - lo);
            const tgm_sample_buffers &s = sb[k % nsb];
            TGM_TRY(tgm_sample_nodes(g, lo, b, nb, s.root, s.root_ts, s.nbr, s.eid, s.nts, s.cnt,
                                     s.nodes, s.n_nodes, cap, s.root_pos, s.nbr_pos, pre));
        }
        TGM_HIP(hipEventRecord(ev.e[c & 1], pre));
        return TGM_OK;
    };
    // the prefetch stream starts after everything issued before on the main one
    TGM_HIP(hipEventRecord(ev.e[4], main));
    TGM_HIP(hipStreamWaitEvent(pre, ev.e[4], 0));
    TGM_TRY(sample_chunk(0));
    for (int64_t c = 0; c < nch; ++c) {
        if (c + 1 < nch) {
            if (c >= 1)   // chunk c-1, the last user of these sample sets, is computed
                TGM_HIP(hipStreamWaitEvent(pre, ev.e[2 + ((c - 1) & 1)], 0));
            TGM_TRY(sample_chunk(c + 1));
        }
        TGM_HIP(hipStreamWaitEvent(main, ev.e[c & 1], 0));
        for (int64_t k = c * K; k < std::min(n, (c + 1) * K); ++k) {
            const int64_t i = i0 + k, lo = i * B;
            const int32_t b = (int32_t)std::min<int64_t>(B, g->E - lo);
            const tgm_sample_buffers &s = sb[k % nsb];
            TGM_TRY(tgm_fetch_memory(st, i, s.nodes, s.n_nodes, cap, fb->mem, fb->mem_ts,
                                     fb->mail, fb->mail_ts, fb->ver, main));
            TGM_TRY(tgm_update_memory(st, m, g, i, s.nodes, s.n_nodes, cap, fb->mem, fb->mem_ts,
                                      fb->mail, fb->mail_ts, fb->ver, lo, b, s.root_pos,
                                      s.root_pos + b, mem_new, new_mem_ts, winner, main));
            TGM_TRY(tgm_embed(m, g, 3 * b, nb, s.root_pos, s.root_ts, s.nbr_pos, s.eid, s.nts,
                              s.cnt, mem_new, s.n_nodes, cap, h, main));
        }
        TGM_HIP(hipEventRecord(ev.e[2 + (c & 1)], main));
    }
    // the events may be destroyed now: the waits already enqueued keep the
    // state they captured
    return TGM_OK;
}
