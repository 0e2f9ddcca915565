// Pipelined executor of the stage.  The sample and node set of an iteration
// (and, with staleness mitigation on, the node set's neighbour sets) depend on
// the event stream only, so they run a chunk of iterations ahead on a second
// stream.  On the main stream each iteration is three launches: the
// GRU; the staging of its write set fused with the node projections; the
// attention fused with the gather of the next iteration's fetch (which needs
// only the staging's commits and runs on the CUs the attention leaves free).
// Cross-stream waits are host calls of several microseconds each, so the
// streams synchronise once per chunk, not once per iteration.
#include <hip/hip_runtime.h>


#include "common.h"

using namespace tgm;

extern "C" tgm_status_t tgm_stage_run(tgm_graph_t g, tgm_state_t st, tgm_model_t m,
                                      int64_t i0, int64_t n, int32_t B, int32_t nb, int32_t cap,
                                      const tgm_sample_buffers *sb, int32_t nsb,
                                      const tgm_fetch_buffers *fb, float *mem_new,
                                      double *new_mem_ts, int64_t *winner, float *h,
                                      float *h_trace, float *s_trace, void *stream,
                                      void *prefetch_stream)
{
    if (!g || !st || !m || !sb || !fb || i0 < 0 || n < 0 || B < 1 || !mem_new || !h)
        return TGM_EINVAL;
    if (nsb < 2 || (nsb & 1))
        return TGM_EINVAL;
    if (nsb > st->xwin_slots || (st->mit && mitigate_slots(st->mit) < 1 + nsb))
        return TGM_ESIZE;
    const bool train = st->trainer != nullptr;
    if (train && m->kind != TGM_MODEL_TGN)
        return TGM_EINVAL;
    if (n == 0)
        return TGM_OK;
    if ((i0 + n - 1) * (int64_t)B >= g->E)
        return TGM_EINVAL;   // past the last batch
    hipStream_t main = as_stream(stream), pre = as_stream(prefetch_stream);
    if (main == pre)
        return TGM_EINVAL;
    // events 0-1: sampled chunk by parity, 2-3: computed chunk by parity, 4: start
    hipEvent_t *const ev = st->run_ev;
    // Chunks of iterations: 1, 2, 4, ... then K = nsb / 2 each, so the main
    // stream waits only for the first iteration's sample before it starts,
    // and each chunk is sampled while the one before it is computed.  A chunk
    // and the next hold at most nsb iterations together, so the sample sets a
    // chunk fills were last read by chunks already computed.
    const int64_t K = nsb / 2;
    int64_t r = 0;   // ramp chunks: sizes 2^c < K
    while ((int64_t(1) << r) < K)
        ++r;
    auto chunk_lo = [&](int64_t c) {
        const int64_t lo = c <= r ? (int64_t(1) << c) - 1 : ((int64_t(1) << r) - 1) + (c - r) * K;
        return std::min(lo, n);
    };
    int64_t nch = 0;
    while (chunk_lo(nch) < n)
        ++nch;
    auto batch = [&](int64_t k, int64_t *lo) {   // the k-th iteration of the run
        *lo = (i0 + k) * B;
        return (int32_t)std::min<int64_t>(B, g->E - *lo);
    };
    // with mitigation on, the neighbour sets of each node set are built beside
    // the sample, into mitigator slot 1 + (k % nsb); the latest-message reduce
    // of each batch also runs beside its sample, into key array k % nsb (so
    // the update's GRU launch skips it)
    // Fetches in place: with neither mitigation (which blends fetched rows)
    // nor training (whose backward reads them), an iteration's fetch forms
    // only phi, and its GRU reads the node set's rows from the committed
    // tables, which hold the same snapshot until that iteration's staging
    // commits the next write set.  The last iteration's fetch still fills the
    // fetch buffers, which the caller reads after the run.
    const bool inplace_ok = !st->mit && !train && m->gru_w && new_mem_ts;
    auto inplace = [&](int64_t k) { return inplace_ok && k + 1 < n; };
    uint64_t *xwin[TGM_MAX_SAMPLE_SETS] = {};
    uint64_t xtag[TGM_MAX_SAMPLE_SETS] = {};
    auto sample_chunk = [&](int64_t c) -> tgm_status_t {
        for (int64_t k = chunk_lo(c); k < chunk_lo(c + 1); ++k) {
            int64_t lo = 0;
            const int32_t b = batch(k, &lo);
            const tgm_sample_buffers &s = sb[k % nsb];
            TGM_TRY_STATUS(tgm_sample_nodes(g, lo, b, nb, s.root, s.root_ts, s.nbr, s.eid, s.nts,
                                            s.cnt, s.nodes, s.n_nodes, cap, s.root_pos,
                                            s.nbr_pos, pre));
            if (st->mit)
                TGM_TRY_STATUS(mitigate_prep_launch(st->mit, g, lo, s.nodes, s.n_nodes, cap,
                                                    (int32_t)(1 + k % nsb), pre));
            TGM_TRY_STATUS(exec_latest_launch(st, (int32_t)(k % nsb), b, s.root_pos,
                                              s.root_pos + b, s.n_nodes, pre, &xwin[k % nsb],
                                              &xtag[k % nsb]));
        }
        TGM_HIP(hipEventRecord(ev[c & 1], pre));
        return TGM_OK;
    };
    // the prefetch stream starts after everything issued before on the main one
    TGM_HIP(hipEventRecord(ev[4], main));
    TGM_HIP(hipStreamWaitEvent(pre, ev[4], 0));
    TGM_TRY_STATUS(sample_chunk(0));
    TGM_HIP(hipStreamWaitEvent(main, ev[0], 0));
    {   // the first iteration's fetch on its own
        GatherPlan plan;
        TGM_TRY_STATUS(fetch_plan(st, i0, sb[0].nodes, sb[0].n_nodes, cap, fb->mem, fb->mem_ts,
                                  fb->mail, fb->mail_ts, fb->ver, main, &plan));
        phi_plan(m, &plan);
        if (inplace(0))
            plan.phi_only();
        TGM_TRY_STATUS(launch_gather(plan, main));
    }
    for (int64_t c = 0; c < nch; ++c) {
        if (c + 1 < nch) {
            if (c >= 1)   // chunk c-1, the last user of these sample sets, is computed
                TGM_HIP(hipStreamWaitEvent(pre, ev[2 + ((c - 1) & 1)], 0));
            TGM_TRY_STATUS(sample_chunk(c + 1));
        }
        const int64_t kend = chunk_lo(c + 1);
        for (int64_t k = chunk_lo(c); k < kend; ++k) {
            int64_t lo = 0;
            const int32_t b = batch(k, &lo);
            const bool more = k + 1 < n;
            // the next iteration's samples are the next chunk's: the wait goes
            // right before the launch that fetches for it (in training mode,
            // which fetches after the step, before the whole iteration)
            hipEvent_t next_ready = nullptr;
            if (more && k + 1 == kend) {
                if (train)
                    TGM_HIP(hipStreamWaitEvent(main, ev[(c + 1) & 1], 0));
                else
                    next_ready = ev[(c + 1) & 1];
            }
            // in training mode the next fetch waits for the training step,
            // which reads this iteration's fetch buffers
            const tgm_sample_buffers *next = more ? &sb[(k + 1) % nsb] : nullptr;
            TGM_TRY_STATUS(compute_iteration(st, m, g, i0 + k, sb[k % nsb], *fb, cap, lo, b, nb,
                                             mem_new, new_mem_ts, winner, h,
                                             train ? nullptr : next, (int32_t)(1 + k % nsb),
                                             xwin[k % nsb], xtag[k % nsb], main, inplace(k),
                                             inplace(k + 1), next_ready));
            if (train) {
                float *lo_ = st->loss_log ? st->loss_log + (i0 + k) % st->loss_log_len : nullptr;
                TGM_TRY_STATUS(train_step_launch(st->trainer, m, g, b, sb[k % nsb], *fb, mem_new,
                                                 h, cap, lo_, main));
                if (next) {
                    GatherPlan plan;
                    TGM_TRY_STATUS(fetch_plan(st, i0 + k + 1, next->nodes, next->n_nodes, cap,
                                              fb->mem, fb->mem_ts, fb->mail, fb->mail_ts,
                                              fb->ver, main, &plan));
                    phi_plan(m, &plan);
                    TGM_TRY_STATUS(launch_gather(plan, main));
                }
            }
            // per-iteration copies of the embeddings and new memories
            if (h_trace && b > 0)
                TGM_HIP(hipMemcpyAsync(h_trace + (size_t)k * 3 * B * m->M, h,
                                       sizeof(float) * 3 * (size_t)b * m->M,
                                       hipMemcpyDeviceToDevice, main));
            if (s_trace)
                TGM_HIP(hipMemcpyAsync(s_trace + (size_t)k * cap * m->M, mem_new,
                                       sizeof(float) * (size_t)cap * m->M,
                                       hipMemcpyDeviceToDevice, main));
        }
        TGM_HIP(hipEventRecord(ev[2 + (c & 1)], main));
    }
    // the events may be destroyed now: the waits already enqueued keep the
    // state they captured
    return TGM_OK;
}
