// Minimal-staleness bound of MSPipe (Sec. 3.2): the stage start/end times of
// Eq. 3 and Eq. 4 for given stage durations, and per iteration the smallest
// staleness k_i whose memory fetch, delayed until the update of iteration
// i - k_i is done (C1), still ends before the compute stage starts (C2), with
// 1 <= k_i < min(i, k_max) (C3).  Host code: O(n k_max) time, O(n) memory.
//
// Stages: 1 sample, 2 feature fetch, 3 memory fetch, 4 compute, 5 memory
// update.  Iterations are 1..n; before the first one every stage has ended at
// time 0.  An iteration with an empty k range is a warm-up iteration (k_i = 0,
// no wait).  When no k in the range meets C2, k_i is the largest in the range
// and the delayed fetch stalls the compute stage.
#include <algorithm>
#include <vector>

#include "common.h"

extern "C" tgm_status_t tgm_min_staleness(const double *tau, int64_t n, int32_t k_max,
                                          int32_t *k, double *fetch_start, double *stall,
                                          double *b, double *e)
{
    if (!tau || n < 0 || k_max < 1 || !k)
        return TGM_EINVAL;
    for (int j = 0; j < 5; ++j)
        if (!(tau[j] >= 0.0))   // also rejects NaN
            return TGM_EINVAL;
    // times of iterations 0..n, stage j at [i * 5 + j - 1]
    std::vector<double> B((size_t)(n + 1) * 5, 0.0), E((size_t)(n + 1) * 5, 0.0);
    auto at = [](std::vector<double> &v, int64_t i, int j) -> double & {
        return v[(size_t)i * 5 + (j - 1)];
    };
    for (int64_t i = 1; i <= n; ++i) {
        at(B, i, 1) = at(E, i - 1, 1);                                // Eq. 3, j = 1
        at(E, i, 1) = at(B, i, 1) + tau[0];
        at(B, i, 2) = std::max(at(E, i, 1), at(E, i - 1, 3));          // j = 2
        at(E, i, 2) = at(B, i, 2) + tau[1];
        for (int j = 3; j <= 5; ++j) {                                // j = 3..5
            at(B, i, j) = std::max(at(E, i, j - 1), at(E, i - 1, j));
            at(E, i, j) = at(B, i, j) + tau[j - 1];
        }
    }
    for (int64_t i = 1; i <= n; ++i) {
        const int64_t hi = std::min<int64_t>(i, k_max);   // k < hi
        int64_t ki = 0;
        double start = at(B, i, 3), st = 0.0;
        if (hi > 1) {
            ki = hi - 1;   // the most staleness allowed, if none is stall-free
            for (int64_t kk = 1; kk < hi; ++kk)
                if (at(E, i - kk, 5) <= at(B, i, 4) - tau[2]) {
                    ki = kk;
                    break;
                }
            start = std::max(at(B, i, 3), at(E, i - ki, 5));
            st = std::max(0.0, start + tau[2] - at(B, i, 4));
        }
        k[i - 1] = (int32_t)ki;
        if (fetch_start)
            fetch_start[i - 1] = start;
        if (stall)
            stall[i - 1] = st;
    }
    if (b)
        std::copy(B.begin() + 5, B.end(), b);
    if (e)
        std::copy(E.begin() + 5, E.end(), e);
    return TGM_OK;
}
