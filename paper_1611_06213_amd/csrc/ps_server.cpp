// Host side of the parameter server: the C ABI declared in include/ps.h.
//
// The host keeps the protocol state of the paper's server (Sec. 2.1, 4.1):
// the FIFO of pushed gradients with its fixed number of slots, the scalar
// timestamp, each learner's timestamp and last pull, and the staleness
// statistics. Device work is only ever enqueued on the server's stream:
// ps_push moves no data, ps_apply_pending launches one fused kernel per run
// of equal-dtype gradients, the pulls launch one fan-out.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "ps.h"
#include "ps_kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int fail_hip(hipError_t e, const char *what) {
    return fail(PS_EHIP, "%s: %s", what, hipGetErrorString(e));
}

struct PushDesc {
    int learner;
    int dtype;
    const void *grad;
    uint64_t learner_ts;   // timestamp of the weights the learner held at push
};

struct PullKey {
    const void *dst = nullptr;
    int dtype = -1;
    uint64_t ts = 0;
    bool valid = false;
};

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Vector level a buffer allows (see launch_apply): 2 if 16-byte aligned, 1 if
// a bf16 buffer is 8-byte aligned, else 0.
int level_of(const void *p, int dtype) {
    if (aligned(p, 16)) return 2;
    if (dtype == PS_BF16 && aligned(p, 8)) return 1;
    return 0;
}

}  // namespace

struct ps_server {
    size_t n = 0;
    float lr = 0.0f;
    float m = 0.0f;
    float *w = nullptr;
    float *v = nullptr;
    int device = 0;
    hipStream_t stream = nullptr;
    int depth = PS_MAX_QUEUE_DEPTH / 2;
    bool pull_skip = true;
    int fuse_max_r = 1;   // ps_apply_pull writes up to this many replicas in the apply pass
    gadei::Geometry geo;

    std::vector<PushDesc> queue;
    uint64_t ts = 0;
    std::vector<uint64_t> learner_ts;   // indexed by learner id, grown on demand
    std::vector<PullKey> last_pull;
    std::vector<int64_t> last_staleness;
    ps_stats stats{};
};

namespace {

int check(const ps_server *ps) {
    if (ps == nullptr) return fail(PS_EINVAL, "null server handle");
    return PS_OK;
}

int check_learner(int id) {
    if (id < 0 || id >= PS_MAX_LEARNERS)
        return fail(PS_EINVAL, "learner id %d outside [0, %d)", id, PS_MAX_LEARNERS);
    return PS_OK;
}

void grow(ps_server *ps, int id) {
    if (static_cast<size_t>(id) >= ps->learner_ts.size()) {
        ps->learner_ts.resize(id + 1, 0);
        ps->last_pull.resize(id + 1);
    }
}

int use_device(const ps_server *ps) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
    if (cur != ps->device) {
        e = hipSetDevice(ps->device);
        if (e != hipSuccess) return fail_hip(e, "hipSetDevice");
    }
    return PS_OK;
}

// Which of the n requested pulls must write, after the queue (if fused) has
// been applied and the timestamp is `ts_after`. A pull is skipped when the
// same learner last pulled into the same buffer, same dtype, at ts_after
// (Sec. 4.1); duplicates inside one call see the earlier entry's effect.
// Validates everything before the caller changes any state.
int plan_pulls(ps_server *ps, int n, const int *ids, void *const *dsts, int dtype,
               uint64_t ts_after, std::vector<int> &write) {
    if (n < 0 || n > PS_MAX_REPLICAS)
        return fail(PS_EINVAL, "pull count %d outside [0, %d]", n, PS_MAX_REPLICAS);
    if (n > 0 && (ids == nullptr || dsts == nullptr))
        return fail(PS_EINVAL, "null learner id or destination array");
    if (dtype != PS_F32 && dtype != PS_BF16) return fail(PS_EINVAL, "bad pull dtype %d", dtype);
    write.clear();
    std::vector<std::pair<int, const void *>> seen;   // (learner, dst) written in this call
    for (int i = 0; i < n; ++i) {
        if (int rc = check_learner(ids[i])) return rc;
        if (dsts[i] == nullptr) return fail(PS_EINVAL, "null destination %d", i);
        const int l = ids[i];
        bool current = false;
        if (ps->pull_skip) {
            for (auto &s : seen)
                if (s.first == l && s.second == dsts[i]) current = true;
            if (!current && static_cast<size_t>(l) < ps->last_pull.size()) {
                const PullKey &k = ps->last_pull[l];
                current = k.valid && k.dst == dsts[i] && k.dtype == dtype && k.ts == ts_after;
            }
        }
        if (current) continue;
        for (int j : write)
            if (dsts[j] == dsts[i])
                return fail(PS_EINVAL, "destination %d repeats destination %d", i, j);
        write.push_back(i);
        seen.emplace_back(l, dsts[i]);
    }
    return PS_OK;
}

void commit_pulls(ps_server *ps, int n, const int *ids, void *const *dsts, int dtype,
                  const std::vector<int> &write) {
    ps->stats.pulls += n;
    ps->stats.pulls_skipped += n - static_cast<int>(write.size());
    for (int i = 0; i < n; ++i) {
        grow(ps, ids[i]);
        ps->learner_ts[ids[i]] = ps->ts;
    }
    for (int i : write) {
        PullKey &k = ps->last_pull[ids[i]];
        k.dst = dsts[i];
        k.dtype = dtype;
        k.ts = ps->ts;
        k.valid = true;
    }
}

// Staleness of each queued gradient when applied (Sec. 2.1), then advance
// the timestamp and empty the queue.
void commit_apply(ps_server *ps) {
    ps->last_staleness.clear();
    for (const PushDesc &d : ps->queue) {
        const int64_t s = static_cast<int64_t>(ps->ts - d.learner_ts);
        ps->last_staleness.push_back(s);
        const uint64_t u = static_cast<uint64_t>(s);
        ps->stats.staleness_sum += u;
        ps->stats.staleness_max = std::max(ps->stats.staleness_max, u);
        ps->stats.staleness_hist[std::min<uint64_t>(u, PS_STALENESS_BINS - 1)] += 1;
        ps->ts += 1;
    }
    ps->stats.pushes_applied += ps->queue.size();
    ps->stats.applies += 1;
    ps->stats.timestamp = ps->ts;
    ps->queue.clear();
}

// Launch the queue as runs of equal gradient dtype, oldest first. The last
// run also writes the replicas listed in `write` when pull_dtype >= 0.
int launch_queue(ps_server *ps, int pull_dtype, void *const *dsts, const std::vector<int> &write) {
    gadei::ApplyArgs a;
    std::memset(&a, 0, sizeof a);
    a.w = ps->w;
    a.v = ps->v;
    a.n = ps->n;
    a.lr = ps->lr;
    a.m = ps->m;
    const size_t q = ps->queue.size();
    size_t start = 0;
    while (start < q) {
        const int gdt = ps->queue[start].dtype;
        size_t end = start;
        int level = 2;
        while (end < q && ps->queue[end].dtype == gdt) {
            a.g[end - start] = ps->queue[end].grad;
            level = std::min(level, level_of(ps->queue[end].grad, gdt));
            ++end;
        }
        a.k = static_cast<int>(end - start);
        a.r = 0;
        int pdt = -1;
        if (end == q && pull_dtype >= 0 && !write.empty()) {
            pdt = pull_dtype;
            a.r = static_cast<int>(write.size());
            for (size_t j = 0; j < write.size(); ++j) {
                a.dst[j] = dsts[write[j]];
                level = std::min(level, level_of(a.dst[j], pull_dtype));
            }
        }
        hipError_t e = gadei::launch_apply(a, gdt, pdt, level, ps->geo, ps->stream);
        if (e != hipSuccess) return fail_hip(e, "apply kernel launch");
        start = end;
    }
    return PS_OK;
}

int launch_pulls(ps_server *ps, void *const *dsts, int dtype, const std::vector<int> &write) {
    if (write.empty()) return PS_OK;
    gadei::PullArgs a;
    std::memset(&a, 0, sizeof a);
    a.w = ps->w;
    a.n = ps->n;
    a.r = static_cast<int>(write.size());
    int level = 2;
    for (size_t j = 0; j < write.size(); ++j) {
        a.dst[j] = dsts[write[j]];
        level = std::min(level, level_of(a.dst[j], dtype));
    }
    hipError_t e = gadei::launch_pull(a, dtype, level, ps->geo, ps->stream);
    if (e != hipSuccess) return fail_hip(e, "pull kernel launch");
    return PS_OK;
}

}  // namespace

extern "C" {

const char *ps_last_error(void) { return g_err.c_str(); }

ps_server *ps_create(size_t n_params, float lr, float momentum) {
    if (n_params == 0) {
        fail(PS_EINVAL, "n_params must be positive");
        return nullptr;
    }
    if (!std::isfinite(lr) || !std::isfinite(momentum)) {
        fail(PS_EINVAL, "lr and momentum must be finite");
        return nullptr;
    }
    ps_server *ps = new (std::nothrow) ps_server();
    if (ps == nullptr) {
        fail(PS_ENOMEM, "host allocation failed");
        return nullptr;
    }
    ps->n = n_params;
    ps->lr = lr;
    ps->m = momentum;
    hipError_t e = hipGetDevice(&ps->device);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&ps->w), n_params * sizeof(float));
    if (e == hipSuccess && momentum != 0.0f)
        e = hipMalloc(reinterpret_cast<void **>(&ps->v), n_params * sizeof(float));
    if (e == hipSuccess) e = hipMemset(ps->w, 0, n_params * sizeof(float));
    if (e == hipSuccess && ps->v) e = hipMemset(ps->v, 0, n_params * sizeof(float));
    if (e != hipSuccess) {
        fail(e == hipErrorOutOfMemory ? PS_ENOMEM : PS_EHIP, "ps_create: %s", hipGetErrorString(e));
        if (ps->w) (void)hipFree(ps->w);
        if (ps->v) (void)hipFree(ps->v);
        delete ps;
        return nullptr;
    }
    ps->queue.reserve(PS_MAX_QUEUE_DEPTH);
    ps->geo.occupancy_cap_lds = gadei::one_block_per_cu_lds();
    return ps;
}

void ps_destroy(ps_server *ps) {
    if (ps == nullptr) return;
    if (use_device(ps) == PS_OK) {
        (void)hipStreamSynchronize(ps->stream);
        if (ps->w) (void)hipFree(ps->w);
        if (ps->v) (void)hipFree(ps->v);
    }
    delete ps;
}

int ps_push_dtype(ps_server *ps, int learner_id, const void *grad, int dtype) {
    if (int rc = check(ps)) return rc;
    if (int rc = check_learner(learner_id)) return rc;
    if (grad == nullptr) return fail(PS_EINVAL, "null gradient");
    if (dtype != PS_F32 && dtype != PS_BF16) return fail(PS_EINVAL, "bad gradient dtype %d", dtype);
    if (static_cast<int>(ps->queue.size()) >= ps->depth) {
        ps->stats.pushes_rejected += 1;
        return fail(PS_EFULL, "queue full (%d pending)", ps->depth);
    }
    const uint64_t lts =
        static_cast<size_t>(learner_id) < ps->learner_ts.size() ? ps->learner_ts[learner_id] : 0;
    ps->queue.push_back(PushDesc{learner_id, dtype, grad, lts});
    ps->stats.pushes_accepted += 1;
    return PS_OK;
}

int ps_push(ps_server *ps, int learner_id, const void *grad) {
    return ps_push_dtype(ps, learner_id, grad, PS_F32);
}

int ps_apply_pending(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    if (ps->queue.empty()) return PS_OK;
    if (int rc = use_device(ps)) return rc;
    static const std::vector<int> none;
    if (int rc = launch_queue(ps, -1, nullptr, none)) return rc;
    commit_apply(ps);
    return PS_OK;
}

int ps_apply_sync(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    if (ps->queue.empty()) return PS_OK;
    const int gdt = ps->queue.front().dtype;
    for (const PushDesc &d : ps->queue)
        if (d.dtype != gdt) return fail(PS_EINVAL, "synchronous step needs one gradient dtype");
    if (int rc = use_device(ps)) return rc;
    gadei::ApplyArgs a;
    std::memset(&a, 0, sizeof a);
    a.w = ps->w;
    a.v = ps->v;
    a.n = ps->n;
    a.lr = ps->lr;
    a.m = ps->m;
    a.k = static_cast<int>(ps->queue.size());
    int level = 2;
    for (size_t j = 0; j < ps->queue.size(); ++j) {
        a.g[j] = ps->queue[j].grad;
        level = std::min(level, level_of(a.g[j], gdt));
    }
    hipError_t e = gadei::launch_sync(a, gdt, level, ps->geo, ps->stream);
    if (e != hipSuccess) return fail_hip(e, "synchronous step launch");
    // one update: every gradient is applied at the same timestamp
    ps->last_staleness.clear();
    for (const PushDesc &d : ps->queue) {
        const uint64_t u = ps->ts - d.learner_ts;
        ps->last_staleness.push_back(static_cast<int64_t>(u));
        ps->stats.staleness_sum += u;
        ps->stats.staleness_max = std::max(ps->stats.staleness_max, u);
        ps->stats.staleness_hist[std::min<uint64_t>(u, PS_STALENESS_BINS - 1)] += 1;
    }
    ps->ts += 1;
    ps->stats.pushes_applied += ps->queue.size();
    ps->stats.applies += 1;
    ps->stats.timestamp = ps->ts;
    ps->queue.clear();
    return PS_OK;
}

int ps_pull_many(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype) {
    if (int rc = check(ps)) return rc;
    std::vector<int> write;
    if (int rc = plan_pulls(ps, n, learner_ids, dsts, dst_dtype, ps->ts, write)) return rc;
    if (!write.empty()) {
        if (int rc = use_device(ps)) return rc;
        if (int rc = launch_pulls(ps, dsts, dst_dtype, write)) return rc;
    }
    commit_pulls(ps, n, learner_ids, dsts, dst_dtype, write);
    return PS_OK;
}

int ps_pull(ps_server *ps, int learner_id, void *dst) {
    return ps_pull_many(ps, 1, &learner_id, &dst, PS_F32);
}

int ps_apply_pull(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype) {
    if (int rc = check(ps)) return rc;
    if (ps->queue.empty()) return ps_pull_many(ps, n, learner_ids, dsts, dst_dtype);
    std::vector<int> write;
    const uint64_t ts_after = ps->ts + ps->queue.size();
    if (int rc = plan_pulls(ps, n, learner_ids, dsts, dst_dtype, ts_after, write)) return rc;
    if (int rc = use_device(ps)) return rc;
    if (static_cast<int>(write.size()) <= ps->fuse_max_r) {
        if (int rc = launch_queue(ps, dst_dtype, dsts, write)) return rc;
    } else {
        static const std::vector<int> none;
        if (int rc = launch_queue(ps, -1, nullptr, none)) return rc;
        if (int rc = launch_pulls(ps, dsts, dst_dtype, write)) return rc;
    }
    commit_apply(ps);
    commit_pulls(ps, n, learner_ids, dsts, dst_dtype, write);
    return PS_OK;
}

int ps_set_stream(ps_server *ps, void *hip_stream) {
    if (int rc = check(ps)) return rc;
    ps->stream = static_cast<hipStream_t>(hip_stream);
    return PS_OK;
}

int ps_set_queue_depth(ps_server *ps, int depth) {
    if (int rc = check(ps)) return rc;
    if (depth < 1 || depth > PS_MAX_QUEUE_DEPTH)
        return fail(PS_EINVAL, "queue depth %d outside [1, %d]", depth, PS_MAX_QUEUE_DEPTH);
    if (static_cast<size_t>(depth) < ps->queue.size())
        return fail(PS_ESTATE, "%zu gradients pending, more than depth %d", ps->queue.size(), depth);
    ps->depth = depth;
    return PS_OK;
}

int ps_set_pull_fusion(ps_server *ps, int max_replicas) {
    if (int rc = check(ps)) return rc;
    if (max_replicas < 0 || max_replicas > PS_MAX_REPLICAS)
        return fail(PS_EINVAL, "fusion limit %d outside [0, %d]", max_replicas, PS_MAX_REPLICAS);
    ps->fuse_max_r = max_replicas;
    return PS_OK;
}

int ps_set_pull_skip(ps_server *ps, int enabled) {
    if (int rc = check(ps)) return rc;
    ps->pull_skip = enabled != 0;
    return PS_OK;
}

int ps_set_weights(ps_server *ps, const float *src) {
    if (int rc = check(ps)) return rc;
    if (src == nullptr) return fail(PS_EINVAL, "null source");
    if (!ps->queue.empty()) return fail(PS_ESTATE, "gradients pending");
    if (int rc = use_device(ps)) return rc;
    hipError_t e = hipMemcpyAsync(ps->w, src, ps->n * sizeof(float), hipMemcpyDeviceToDevice,
                                  ps->stream);
    if (e != hipSuccess) return fail_hip(e, "weights copy");
    if (ps->v) {
        e = gadei::launch_zero(ps->v, ps->n, ps->stream);
        if (e != hipSuccess) return fail_hip(e, "velocity reset");
    }
    ps->ts = 0;
    ps->learner_ts.clear();
    ps->last_pull.clear();
    ps->last_staleness.clear();
    ps->stats = ps_stats{};
    return PS_OK;
}

const float *ps_weights(const ps_server *ps) { return ps ? ps->w : nullptr; }
const float *ps_velocity(const ps_server *ps) { return ps ? ps->v : nullptr; }
size_t ps_num_params(const ps_server *ps) { return ps ? ps->n : 0; }
uint64_t ps_timestamp(const ps_server *ps) { return ps ? ps->ts : 0; }

int ps_pending(const ps_server *ps) {
    if (int rc = check(ps)) return rc;
    return static_cast<int>(ps->queue.size());
}

int ps_last_staleness(const ps_server *ps, int64_t *out, int cap) {
    if (int rc = check(ps)) return rc;
    if (cap < 0 || (cap > 0 && out == nullptr)) return fail(PS_EINVAL, "bad output buffer");
    const int count = static_cast<int>(ps->last_staleness.size());
    for (int i = 0; i < count && i < cap; ++i) out[i] = ps->last_staleness[i];
    return count;
}

int ps_sync(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    if (int rc = use_device(ps)) return rc;
    hipError_t e = hipStreamSynchronize(ps->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    return PS_OK;
}

int ps_get_stats(const ps_server *ps, ps_stats *out) {
    if (int rc = check(ps)) return rc;
    if (out == nullptr) return fail(PS_EINVAL, "null stats output");
    *out = ps->stats;
    out->timestamp = ps->ts;
    return PS_OK;
}

}  // extern "C"
