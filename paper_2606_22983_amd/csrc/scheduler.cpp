// Interaction-aware batch selection for one stage and one scheduling round
// (LiveServe §4, the scheduling procedure and its algorithm).  Host code; it
// produces the batches the decode and prefill kernels consume.
//
// Each ready request is put in an urgency class from its stage-aware playback
// buffer P (seconds of produced-but-unconsumed output):
//   U0  first audio produced and P <= P_safe: playback at risk; ordered by P
//       ascending (closest to underrun first);
//   U1  no first audio yet: on the audio TTFP path; ordered by ready age
//       descending (FCFS-style aging);
//   U2  first audio produced and P > P_safe: ordered by the utility
//       U = beta * U_kv - alpha * C_barge, descending, with
//       U_kv = K * R_occ (KV held times the stage's occupied/allocatable KV
//       ratio) and C_barge = max(0, P - P_safe) / P_safe.
// The three lists are joined U0, U1, U2 and scanned in that order; admission
// stops at the first request whose tokens or KV blocks exceed what is left of
// the round's budgets.
//
// Fail-closed inputs (§6): a round in which any request lacks a playback
// buffer (NaN) orders every request by ready age alone; a round without the
// KV occupancy (NaN), or a U2 request without its KV size (< 0), orders U2 by
// ready age instead of the utility.  Ties go to the smaller request index.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <numeric>
#include <vector>

#include "liveserve_kv.h"

namespace ls {
void set_last_error(const char *fmt, ...);
}

namespace {

ls_status sched_fail(ls_status st, const char *fmt, ...) {
    char buf[300];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    ls::set_last_error("%s", buf);
    return st;
}

}  // namespace

extern "C" ls_status ls_schedule_round(const ls_sched_stage *stage, int32_t n, const ls_sched_request *req,
                                       int32_t *order, int32_t *classes, double *utility,
                                       int32_t *num_admitted) {
    if (!stage || n < 0 || (n > 0 && (!req || !order)) || !num_admitted)
        return sched_fail(LS_EINVAL, "ls_schedule_round: bad argument");
    *num_admitted = 0;
    if (!(stage->p_safe_s > 0.0) || std::isnan(stage->alpha) || std::isnan(stage->beta) ||
        stage->token_budget < 0 || stage->kv_block_budget < 0)
        return sched_fail(LS_EINVAL, "ls_schedule_round: p_safe must be > 0, weights finite, budgets >= 0");
    for (int32_t i = 0; i < n; ++i)
        if (req[i].tokens_needed < 0 || req[i].kv_blocks_needed < 0 || std::isnan(req[i].ready_age_s))
            return sched_fail(LS_EINVAL, "ls_schedule_round: request %d has a negative demand or NaN age", i);

    bool buffers_known = true;
    for (int32_t i = 0; i < n; ++i) buffers_known = buffers_known && !std::isnan(req[i].playback_buffer_s);
    const double ps = stage->p_safe_s;
    std::vector<int32_t> cls((size_t)n);
    std::vector<double> u((size_t)n, 0.0);
    std::vector<char> by_age((size_t)n, 0);
    for (int32_t i = 0; i < n; ++i) {
        const double p = req[i].playback_buffer_s;
        if (!buffers_known) cls[(size_t)i] = 1;                  // one FCFS list by ready age
        else if (!req[i].first_audio_done) cls[(size_t)i] = 1;
        else cls[(size_t)i] = p <= ps ? 0 : 2;
        if (cls[(size_t)i] == 2) {
            if (std::isnan(stage->kv_occupancy) || req[i].kv_blocks_held < 0) {
                by_age[(size_t)i] = 1;
            } else {
                const double u_kv = (double)req[i].kv_blocks_held * stage->kv_occupancy;
                const double c_barge = std::max(0.0, p - ps) / ps;
                u[(size_t)i] = stage->beta * u_kv - stage->alpha * c_barge;
            }
        }
    }
    // U2 falls back to ready age as a whole when any of its members lacks the inputs.
    bool u2_by_age = false;
    for (int32_t i = 0; i < n; ++i) u2_by_age = u2_by_age || (cls[(size_t)i] == 2 && by_age[(size_t)i]);

    std::vector<int32_t> idx((size_t)n);
    std::iota(idx.begin(), idx.end(), 0);
    std::sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) {
        const int32_t ca = cls[(size_t)a], cb = cls[(size_t)b];
        if (ca != cb) return ca < cb;
        double ka, kb;            // smaller key first
        if (ca == 0) {
            ka = req[a].playback_buffer_s;
            kb = req[b].playback_buffer_s;
        } else if (ca == 1 || u2_by_age) {
            ka = -req[a].ready_age_s;
            kb = -req[b].ready_age_s;
        } else {
            ka = -u[(size_t)a];
            kb = -u[(size_t)b];
        }
        if (ka != kb) return ka < kb;
        return a < b;
    });
    int64_t tokens = stage->token_budget, blocks = stage->kv_block_budget;
    int32_t admitted = 0;
    for (int32_t k = 0; k < n; ++k) {
        const ls_sched_request &r = req[idx[(size_t)k]];
        if (r.tokens_needed > tokens || r.kv_blocks_needed > blocks) break;
        tokens -= r.tokens_needed;
        blocks -= r.kv_blocks_needed;
        ++admitted;
    }
    for (int32_t k = 0; k < n; ++k) {
        order[k] = idx[(size_t)k];
        if (classes) classes[k] = cls[(size_t)k];
        if (utility) utility[k] = u[(size_t)k];
    }
    *num_admitted = admitted;
    return LS_OK;
}
