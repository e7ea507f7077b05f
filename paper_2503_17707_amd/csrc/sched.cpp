// Epoch-based adapter switching (PipeBoost, Section 4.3.2), host side.
//
// With merged LoRA a device runs one adapter at a time, and changing adapters
// costs a restore and a merge of every layer's attention weights.  Requests
// are therefore queued per adapter: batches of the active adapter go first and
// the scheduler moves to another adapter only at epoch boundaries (after a
// fixed number of batches of the active one) or when the active queue runs
// dry.  The next adapter is the one whose oldest queued request has waited
// longest, so no queue starves.  Epoch length 0 is the eager baseline the
// paper compares against: requests are served in arrival order and a batch is
// a run of consecutive arrivals that share an adapter.
#include <stdint.h>

#include <deque>
#include <limits>
#include <vector>

#include "../../include/pipeboost.h"

__attribute__((visibility("hidden"))) int pb_fail_status(int code, const char* msg);  // model.cpp

struct pb_sched {
    struct Req {
        int64_t id;
        uint64_t seq;  // arrival order
    };
    int n_adapters = 0;
    int epoch = 0;
    std::vector<std::deque<Req>> q;  // index a + 1: adapter a (index 0 is the base model)
    uint64_t seq = 0;
    int active = -2;                 // adapter of the last batch (-2: none yet)
    int served = 0;                  // batches of the active adapter in this epoch
    int64_t switches = 0;
    int64_t pending = 0;
};

namespace {

// Queue index whose head arrived first, skipping `skip` (-1: skip none);
// -1 when every considered queue is empty.
int oldest_queue(const pb_sched* s, int skip) {
    int best = -1;
    uint64_t best_seq = std::numeric_limits<uint64_t>::max();
    for (int i = 0; i < (int)s->q.size(); ++i) {
        if (i == skip || s->q[i].empty()) continue;
        if (s->q[i].front().seq < best_seq) {
            best_seq = s->q[i].front().seq;
            best = i;
        }
    }
    return best;
}

}  // namespace

extern "C" {

int pb_sched_create(int32_t n_adapters, int32_t epoch_batches, pb_sched** out) {
    if (!out) return pb_fail_status(PB_EINVAL, "out is NULL");
    *out = nullptr;
    if (n_adapters < 0 || n_adapters > 1 << 20) return pb_fail_status(PB_EINVAL, "bad adapter count");
    if (epoch_batches < 0) return pb_fail_status(PB_EINVAL, "epoch_batches must be >= 0");
    pb_sched* s = new pb_sched;
    s->n_adapters = n_adapters;
    s->epoch = epoch_batches;
    s->q.resize((size_t)n_adapters + 1);
    *out = s;
    return PB_OK;
}

int pb_sched_destroy(pb_sched* s) {
    delete s;
    return PB_OK;
}

int pb_sched_submit(pb_sched* s, int64_t request_id, int32_t adapter) {
    if (!s) return pb_fail_status(PB_EINVAL, "scheduler is NULL");
    if (adapter < -1 || adapter >= s->n_adapters) return pb_fail_status(PB_EINVAL, "adapter outside [-1, n_adapters)");
    s->q[(size_t)adapter + 1].push_back({request_id, s->seq++});
    s->pending += 1;
    return PB_OK;
}

int pb_sched_next(pb_sched* s, int32_t max_batch, int64_t* ids, int32_t* n, int32_t* adapter, int32_t* switched) {
    if (!s || !ids || !n || !adapter || !switched) return pb_fail_status(PB_EINVAL, "NULL argument");
    if (max_batch < 1) return pb_fail_status(PB_EINVAL, "max_batch must be >= 1");
    *n = 0;
    if (s->pending == 0) return PB_OK;
    const int cur = s->active + 1;  // queue index of the active adapter (-1: none yet)
    int pick;
    int limit = max_batch;
    if (s->epoch == 0) {
        // eager: the oldest request decides, and the batch stops at the first
        // later arrival of another adapter
        pick = oldest_queue(s, -1);
        const int other = oldest_queue(s, pick);
        const uint64_t stop = other < 0 ? std::numeric_limits<uint64_t>::max() : s->q[other].front().seq;
        int run = 0;
        for (const auto& r : s->q[pick]) {
            if (r.seq > stop || run == max_batch) break;
            ++run;
        }
        limit = run;
    } else {
        const bool active_has_work = cur >= 0 && !s->q[cur].empty();
        if (active_has_work && s->served < s->epoch) {
            pick = cur;
        } else {
            pick = oldest_queue(s, cur);
            if (pick < 0) pick = cur;  // no other queue has work: stay
        }
    }
    const int a = pick - 1;
    *switched = a != s->active ? 1 : 0;
    if (a != s->active) {
        if (s->active != -2) s->switches += 1;
        s->active = a;
        s->served = 0;
    }
    auto& qq = s->q[pick];
    int k = 0;
    while (k < limit && !qq.empty()) {
        ids[k++] = qq.front().id;
        qq.pop_front();
    }
    s->pending -= k;
    s->served += 1;
    *n = k;
    *adapter = a;
    return PB_OK;
}

int pb_sched_stats(pb_sched* s, int64_t* pending, int64_t* switches, int32_t* active) {
    if (!s) return pb_fail_status(PB_EINVAL, "scheduler is NULL");
    if (pending) *pending = s->pending;
    if (switches) *switches = s->switches;
    if (active) *active = s->active;
    return PB_OK;
}

}  // extern "C"
