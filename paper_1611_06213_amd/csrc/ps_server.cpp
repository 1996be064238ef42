// Host side of the parameter server: the C ABI declared in include/ps.h.
//
// The host keeps the protocol state of the paper's server (Sec. 2.1, 4.1):
// the queued gradients with their fixed number of slots, the scalar
// timestamp, each learner's timestamp and last pull, and the staleness
// statistics. Device work is only ever enqueued on the server's stream:
// ps_push moves no data, an apply launches one kernel per run of equal-dtype
// gradients, a pull launches one fan-out.
//
// Queue modes. FIFO: one queue of `depth` slots in push-call order. Round
// robin: every learner has its own queue of `slots` slots (the paper's lambda
// single-producer single-consumer queues) and the server visits learners in
// increasing id order, cyclically, starting after the learner it served
// last, taking one gradient per visit (Sec. 4.1). Either way an apply takes a
// "batch" of at most `depth` gradients, which the kernels fold in order.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdio>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <new>
#include <set>
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
    hipEvent_t ready;      // producer's event the apply waits for, or null
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
    hipStream_t pull_stream = nullptr;   // lock-free pulls when pull_lock_free
    bool pull_lock_free = false;
    int depth = PS_MAX_QUEUE_DEPTH / 2;
    bool pull_skip = true;
    int fuse_max_r = 1;   // ps_apply_pull writes up to this many replicas in the apply pass
    gadei::Geometry geo;

    int mode = PS_QUEUE_FIFO;
    std::vector<PushDesc> fifo;            // FIFO mode
    int slots = 1;                         // round-robin mode: slots per learner
    std::vector<std::deque<PushDesc>> rr;  // ... queue of each learner id
    std::set<int> waiting;                 // ... ids whose queue is not empty
    size_t rr_count = 0;
    int last_served = -1;

    uint64_t ts = 0;
    std::vector<uint64_t> learner_ts;   // indexed by learner id, grown on demand
    std::vector<PullKey> last_pull;
    std::vector<int64_t> last_staleness;
    std::vector<int> last_applied;
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

size_t pending(const ps_server *ps) {
    return ps->mode == PS_QUEUE_FIFO ? ps->fifo.size() : ps->rr_count;
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

// The gradients an apply takes, in the order it applies them, and how many
// each learner queue gives (round-robin mode). Nothing is removed while
// planning: consume() does that once the launch has succeeded.
struct Batch {
    std::vector<PushDesc> items;
    std::vector<std::pair<int, int>> taken;   // (learner, count), round robin
    int last_served = -1;
};

void plan_async(const ps_server *ps, Batch &b) {
    b.items.clear();
    b.taken.clear();
    b.last_served = ps->last_served;
    if (ps->mode == PS_QUEUE_FIFO) {
        b.items = ps->fifo;
        return;
    }
    std::vector<std::pair<int, size_t>> avail;   // (learner, queued), increasing id
    for (int l : ps->waiting) avail.emplace_back(l, ps->rr[l].size());
    std::vector<size_t> used(avail.size(), 0);
    size_t left = ps->rr_count;
    int cur = ps->last_served;
    while (static_cast<int>(b.items.size()) < ps->depth && left > 0) {
        // the next learner after `cur`, cyclically, whose queue still has one
        size_t pick = avail.size();
        for (size_t j = 0; j < avail.size(); ++j)
            if (avail[j].first > cur && used[j] < avail[j].second) {
                pick = j;
                break;
            }
        if (pick == avail.size())
            for (size_t j = 0; j < avail.size(); ++j)
                if (used[j] < avail[j].second) {
                    pick = j;
                    break;
                }
        const int l = avail[pick].first;
        b.items.push_back(ps->rr[l][used[pick]]);
        ++used[pick];
        --left;
        cur = l;
    }
    for (size_t j = 0; j < avail.size(); ++j)
        if (used[j]) b.taken.emplace_back(avail[j].first, static_cast<int>(used[j]));
    b.last_served = cur;
}

// Synchronous step: FIFO takes every pending gradient in push order; round
// robin the oldest gradient of every waiting learner, in increasing id.
void plan_sync(const ps_server *ps, Batch &b) {
    b.items.clear();
    b.taken.clear();
    b.last_served = ps->last_served;
    if (ps->mode == PS_QUEUE_FIFO) {
        b.items = ps->fifo;
        return;
    }
    for (int l : ps->waiting) {
        b.items.push_back(ps->rr[l].front());
        b.taken.emplace_back(l, 1);
    }
}

void consume(ps_server *ps, const Batch &b) {
    if (ps->mode == PS_QUEUE_FIFO) {
        ps->fifo.erase(ps->fifo.begin(), ps->fifo.begin() + b.items.size());
        return;
    }
    for (const auto &t : b.taken) {
        auto &q = ps->rr[t.first];
        for (int i = 0; i < t.second; ++i) q.pop_front();
        if (q.empty()) ps->waiting.erase(t.first);
    }
    ps->rr_count -= b.items.size();
    ps->last_served = b.last_served;
}

// Which of the n requested pulls must write, after the batch (if fused) has
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

// `ordered`: the replicas were written after every earlier apply, so they
// hold the weights at the current timestamp and a repeat can be skipped. A
// lock-free pull may have raced an apply: its replicas never count as
// current.
void commit_pulls(ps_server *ps, int n, const int *ids, void *const *dsts, int dtype,
                  const std::vector<int> &write, bool ordered) {
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
        k.valid = ordered;
    }
}

void record_staleness(ps_server *ps, const PushDesc &d, uint64_t at) {
    const uint64_t u = at - d.learner_ts;
    ps->last_staleness.push_back(static_cast<int64_t>(u));
    ps->last_applied.push_back(d.learner);
    ps->stats.staleness_sum += u;
    ps->stats.staleness_max = std::max(ps->stats.staleness_max, u);
    ps->stats.staleness_hist[std::min<uint64_t>(u, PS_STALENESS_BINS - 1)] += 1;
}

// Asynchronous apply done: staleness of each gradient when applied (Sec.
// 2.1), one timestamp step per gradient, and the batch leaves its queues.
void commit_async(ps_server *ps, const Batch &b) {
    ps->last_staleness.clear();
    ps->last_applied.clear();
    for (const PushDesc &d : b.items) {
        record_staleness(ps, d, ps->ts);
        ps->ts += 1;
    }
    ps->stats.pushes_applied += b.items.size();
    ps->stats.applies += 1;
    ps->stats.timestamp = ps->ts;
    consume(ps, b);
}

// Make the server's stream wait (on the device) for every producer event of
// the batch, each once.
int wait_ready(ps_server *ps, const std::vector<PushDesc> &items) {
    std::vector<hipEvent_t> seen;
    for (const PushDesc &d : items) {
        if (d.ready == nullptr || std::find(seen.begin(), seen.end(), d.ready) != seen.end())
            continue;
        seen.push_back(d.ready);
        hipError_t e = hipStreamWaitEvent(ps->stream, d.ready, 0);
        if (e != hipSuccess) return fail_hip(e, "waiting for a producer event");
    }
    return PS_OK;
}

// Host-side wait for lock-free pulls still reading w (before w is reset,
// saved, loaded or freed).
int drain_pulls(ps_server *ps) {
    if (!ps->pull_lock_free) return PS_OK;
    hipError_t e = hipStreamSynchronize(ps->pull_stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize (pull stream)");
    return PS_OK;
}

// Launch a batch as runs of equal gradient dtype, in order. The last run
// also writes the replicas listed in `write` when pull_dtype >= 0.
int launch_batch(ps_server *ps, const std::vector<PushDesc> &items, int pull_dtype,
                 void *const *dsts, const std::vector<int> &write) {
    if (int rc = wait_ready(ps, items)) return rc;
    gadei::ApplyArgs a;
    std::memset(&a, 0, sizeof a);
    a.w = ps->w;
    a.v = ps->v;
    a.n = ps->n;
    a.lr = ps->lr;
    a.m = ps->m;
    const size_t q = items.size();
    size_t start = 0;
    while (start < q) {
        const int gdt = items[start].dtype;
        size_t end = start;
        int level = 2;
        while (end < q && items[end].dtype == gdt) {
            a.g[end - start] = items[end].grad;
            level = std::min(level, level_of(items[end].grad, gdt));
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

// `ordered`: on the server's stream, after every earlier apply; otherwise on
// the lock-free pull stream when that mode is on.
int launch_pulls(ps_server *ps, void *const *dsts, int dtype, const std::vector<int> &write,
                 bool ordered) {
    if (write.empty()) return PS_OK;
    hipStream_t s = (!ordered && ps->pull_lock_free) ? ps->pull_stream : ps->stream;
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
    hipError_t e = gadei::launch_pull(a, dtype, level, ps->geo, s);
    if (e != hipSuccess) return fail_hip(e, "pull kernel launch");
    return PS_OK;
}

// An apply with nothing to apply launches nothing; the last-apply queries
// then report an empty apply.
void clear_last(ps_server *ps) {
    ps->last_staleness.clear();
    ps->last_applied.clear();
}

// ---------------------------------------------------------------- checkpoint
//
// File layout (little-endian, as the host writes it):
//   CkptHeader, then learner_ts[n_learner_ts] (uint64), then w[n] (fp32),
//   then v[n] (fp32) when the server has momentum.
// `checksum` is FNV-1a (64-bit) over every byte after the header.

struct CkptHeader {
    char magic[8];
    uint32_t version;
    uint32_t has_v;
    uint64_t n;
    float lr;
    float m;
    uint64_t ts;
    int64_t last_served;
    uint64_t n_learner_ts;
    uint64_t checksum;
};

constexpr char kMagic[8] = {'G', 'A', 'D', 'E', 'I', 'P', 'S', '1'};
constexpr size_t kChunk = size_t(16) << 20;   // floats per device<->host copy

struct Fnv {
    uint64_t h = 1469598103934665603ull;
    void add(const void *p, size_t bytes) {
        const unsigned char *c = static_cast<const unsigned char *>(p);
        for (size_t i = 0; i < bytes; ++i) {
            h ^= c[i];
            h *= 1099511628211ull;
        }
    }
};

int write_all(FILE *f, const void *p, size_t bytes, Fnv *fnv) {
    if (fnv) fnv->add(p, bytes);
    return std::fwrite(p, 1, bytes, f) == bytes ? PS_OK : fail(PS_EIO, "checkpoint write failed");
}

// Device array -> file, in chunks through a host buffer.
int save_array(FILE *f, const float *dev, size_t n, std::vector<float> &buf, Fnv &fnv) {
    for (size_t off = 0; off < n; off += kChunk) {
        const size_t cnt = std::min(kChunk, n - off);
        hipError_t e = hipMemcpy(buf.data(), dev + off, cnt * sizeof(float), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return fail_hip(e, "checkpoint read-back");
        if (int rc = write_all(f, buf.data(), cnt * sizeof(float), &fnv)) return rc;
    }
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
    ps->fifo.reserve(PS_MAX_QUEUE_DEPTH);
    ps->geo.occupancy_cap_lds = gadei::one_block_per_cu_lds();
    return ps;
}

void ps_destroy(ps_server *ps) {
    if (ps == nullptr) return;
    if (use_device(ps) == PS_OK) {
        (void)hipStreamSynchronize(ps->stream);
        if (ps->pull_lock_free) (void)hipStreamSynchronize(ps->pull_stream);
        if (ps->w) (void)hipFree(ps->w);
        if (ps->v) (void)hipFree(ps->v);
    }
    delete ps;
}

int ps_push_async(ps_server *ps, int learner_id, const void *grad, int dtype, void *ready_event);

int ps_push_dtype(ps_server *ps, int learner_id, const void *grad, int dtype) {
    return ps_push_async(ps, learner_id, grad, dtype, nullptr);
}

int ps_push_async(ps_server *ps, int learner_id, const void *grad, int dtype, void *ready_event) {
    if (int rc = check(ps)) return rc;
    if (int rc = check_learner(learner_id)) return rc;
    if (grad == nullptr) return fail(PS_EINVAL, "null gradient");
    if (dtype != PS_F32 && dtype != PS_BF16) return fail(PS_EINVAL, "bad gradient dtype %d", dtype);
    const uint64_t lts =
        static_cast<size_t>(learner_id) < ps->learner_ts.size() ? ps->learner_ts[learner_id] : 0;
    const PushDesc d{learner_id, dtype, grad, lts, static_cast<hipEvent_t>(ready_event)};
    if (ps->mode == PS_QUEUE_FIFO) {
        if (static_cast<int>(ps->fifo.size()) >= ps->depth) {
            ps->stats.pushes_rejected += 1;
            return fail(PS_EFULL, "queue full (%d pending)", ps->depth);
        }
        ps->fifo.push_back(d);
    } else {
        if (static_cast<size_t>(learner_id) >= ps->rr.size()) ps->rr.resize(learner_id + 1);
        auto &q = ps->rr[learner_id];
        if (static_cast<int>(q.size()) >= ps->slots) {
            ps->stats.pushes_rejected += 1;
            return fail(PS_EFULL, "learner %d queue full (%d slots)", learner_id, ps->slots);
        }
        q.push_back(d);
        ps->waiting.insert(learner_id);
        ps->rr_count += 1;
    }
    ps->stats.pushes_accepted += 1;
    return PS_OK;
}

int ps_push(ps_server *ps, int learner_id, const void *grad) {
    return ps_push_dtype(ps, learner_id, grad, PS_F32);
}

int ps_apply_pending(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    if (pending(ps) == 0) {
        clear_last(ps);
        return PS_OK;
    }
    if (int rc = use_device(ps)) return rc;
    Batch b;
    plan_async(ps, b);
    static const std::vector<int> none;
    if (int rc = launch_batch(ps, b.items, -1, nullptr, none)) return rc;
    commit_async(ps, b);
    return PS_OK;
}

int ps_apply_sync(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    if (pending(ps) == 0) {
        clear_last(ps);
        return PS_OK;
    }
    Batch b;
    plan_sync(ps, b);
    if (b.items.size() > PS_MAX_QUEUE_DEPTH)
        return fail(PS_ESTATE, "%zu learners waiting, more than one step can average (%d)",
                    b.items.size(), PS_MAX_QUEUE_DEPTH);
    const int gdt = b.items.front().dtype;
    for (const PushDesc &d : b.items)
        if (d.dtype != gdt) return fail(PS_EINVAL, "synchronous step needs one gradient dtype");
    if (int rc = use_device(ps)) return rc;
    if (int rc = wait_ready(ps, b.items)) return rc;
    gadei::ApplyArgs a;
    std::memset(&a, 0, sizeof a);
    a.w = ps->w;
    a.v = ps->v;
    a.n = ps->n;
    a.lr = ps->lr;
    a.m = ps->m;
    a.k = static_cast<int>(b.items.size());
    int level = 2;
    for (size_t j = 0; j < b.items.size(); ++j) {
        a.g[j] = b.items[j].grad;
        level = std::min(level, level_of(a.g[j], gdt));
    }
    hipError_t e = gadei::launch_sync(a, gdt, level, ps->geo, ps->stream);
    if (e != hipSuccess) return fail_hip(e, "synchronous step launch");
    // one update: every gradient is applied at the same timestamp
    ps->last_staleness.clear();
    ps->last_applied.clear();
    for (const PushDesc &d : b.items) record_staleness(ps, d, ps->ts);
    ps->ts += 1;
    ps->stats.pushes_applied += b.items.size();
    ps->stats.applies += 1;
    ps->stats.timestamp = ps->ts;
    consume(ps, b);
    return PS_OK;
}

int ps_pull_many(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype) {
    if (int rc = check(ps)) return rc;
    std::vector<int> write;
    if (int rc = plan_pulls(ps, n, learner_ids, dsts, dst_dtype, ps->ts, write)) return rc;
    if (!write.empty()) {
        if (int rc = use_device(ps)) return rc;
        if (int rc = launch_pulls(ps, dsts, dst_dtype, write, false)) return rc;
    }
    commit_pulls(ps, n, learner_ids, dsts, dst_dtype, write, !ps->pull_lock_free);
    return PS_OK;
}

int ps_pull(ps_server *ps, int learner_id, void *dst) {
    return ps_pull_many(ps, 1, &learner_id, &dst, PS_F32);
}

int ps_apply_pull(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype) {
    if (int rc = check(ps)) return rc;
    if (pending(ps) == 0) {
        const int rc = ps_pull_many(ps, n, learner_ids, dsts, dst_dtype);
        if (rc == PS_OK) clear_last(ps);
        return rc;
    }
    Batch b;
    plan_async(ps, b);
    std::vector<int> write;
    const uint64_t ts_after = ps->ts + b.items.size();
    if (int rc = plan_pulls(ps, n, learner_ids, dsts, dst_dtype, ts_after, write)) return rc;
    if (int rc = use_device(ps)) return rc;
    if (static_cast<int>(write.size()) <= ps->fuse_max_r) {
        if (int rc = launch_batch(ps, b.items, dst_dtype, dsts, write)) return rc;
    } else {
        static const std::vector<int> none;
        if (int rc = launch_batch(ps, b.items, -1, nullptr, none)) return rc;
        if (int rc = launch_pulls(ps, dsts, dst_dtype, write, true)) return rc;
    }
    commit_async(ps, b);
    commit_pulls(ps, n, learner_ids, dsts, dst_dtype, write, true);
    return PS_OK;
}

int ps_drop_learner(ps_server *ps, int learner_id) {
    if (int rc = check(ps)) return rc;
    if (int rc = check_learner(learner_id)) return rc;
    int dropped = 0;
    if (ps->mode == PS_QUEUE_FIFO) {
        auto keep = std::remove_if(ps->fifo.begin(), ps->fifo.end(),
                                   [&](const PushDesc &d) { return d.learner == learner_id; });
        dropped = static_cast<int>(ps->fifo.end() - keep);
        ps->fifo.erase(keep, ps->fifo.end());
    } else if (static_cast<size_t>(learner_id) < ps->rr.size()) {
        dropped = static_cast<int>(ps->rr[learner_id].size());
        ps->rr[learner_id].clear();
        ps->waiting.erase(learner_id);
        ps->rr_count -= dropped;
    }
    ps->stats.pushes_dropped += dropped;
    return dropped;
}

int ps_save(ps_server *ps, const char *path) {
    if (int rc = check(ps)) return rc;
    if (path == nullptr) return fail(PS_EINVAL, "null path");
    if (pending(ps) != 0) return fail(PS_ESTATE, "gradients pending");
    if (int rc = use_device(ps)) return rc;
    hipError_t e = hipStreamSynchronize(ps->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    FILE *f = std::fopen(path, "wb");
    if (f == nullptr) return fail(PS_EIO, "cannot open %s for writing", path);
    CkptHeader h;
    std::memset(&h, 0, sizeof h);
    std::memcpy(h.magic, kMagic, sizeof kMagic);
    h.version = 1;
    h.has_v = ps->v != nullptr;
    h.n = ps->n;
    h.lr = ps->lr;
    h.m = ps->m;
    h.ts = ps->ts;
    h.last_served = ps->last_served;
    h.n_learner_ts = ps->learner_ts.size();
    int rc = write_all(f, &h, sizeof h, nullptr);
    Fnv fnv;
    std::vector<float> buf;
    if (rc == PS_OK && h.n_learner_ts)
        rc = write_all(f, ps->learner_ts.data(), h.n_learner_ts * sizeof(uint64_t), &fnv);
    if (rc == PS_OK) {
        buf.resize(std::min(kChunk, ps->n));
        rc = save_array(f, ps->w, ps->n, buf, fnv);
    }
    if (rc == PS_OK && ps->v) rc = save_array(f, ps->v, ps->n, buf, fnv);
    if (rc == PS_OK) {
        h.checksum = fnv.h;
        if (std::fseek(f, 0, SEEK_SET) != 0) rc = fail(PS_EIO, "checkpoint seek failed");
        else rc = write_all(f, &h, sizeof h, nullptr);
    }
    if (std::fclose(f) != 0 && rc == PS_OK) rc = fail(PS_EIO, "checkpoint close failed");
    return rc;
}

int ps_load(ps_server *ps, const char *path) {
    if (int rc = check(ps)) return rc;
    if (path == nullptr) return fail(PS_EINVAL, "null path");
    if (pending(ps) != 0) return fail(PS_ESTATE, "gradients pending");
    FILE *f = std::fopen(path, "rb");
    if (f == nullptr) return fail(PS_EIO, "cannot open %s", path);
    CkptHeader h;
    int rc = PS_OK;
    if (std::fread(&h, 1, sizeof h, f) != sizeof h || std::memcmp(h.magic, kMagic, 8) != 0 ||
        h.version != 1)
        rc = fail(PS_EIO, "%s is not a parameter-server checkpoint", path);
    else if (h.n != ps->n || (h.has_v != 0) != (ps->v != nullptr))
        rc = fail(PS_EINVAL, "checkpoint holds %llu params%s; server has %zu%s",
                  static_cast<unsigned long long>(h.n), h.has_v ? " with momentum" : "", ps->n,
                  ps->v ? " with momentum" : "");
    else if (std::memcmp(&h.lr, &ps->lr, sizeof(float)) != 0 ||
             std::memcmp(&h.m, &ps->m, sizeof(float)) != 0)
        rc = fail(PS_EINVAL, "checkpoint lr/momentum differ from the server's");
    else if (h.n_learner_ts > static_cast<uint64_t>(PS_MAX_LEARNERS))
        rc = fail(PS_EIO, "corrupt checkpoint (learner table)");
    // read and verify everything before touching the server
    std::vector<uint64_t> lts;
    std::vector<float> w, v;
    Fnv fnv;
    if (rc == PS_OK) {
        lts.resize(h.n_learner_ts);
        w.resize(h.n);
        if (h.has_v) v.resize(h.n);
        const size_t lb = lts.size() * sizeof(uint64_t), wb = w.size() * sizeof(float);
        if (std::fread(lts.data(), 1, lb, f) != lb || std::fread(w.data(), 1, wb, f) != wb ||
            (h.has_v && std::fread(v.data(), 1, wb, f) != wb))
            rc = fail(PS_EIO, "checkpoint truncated");
        else {
            fnv.add(lts.data(), lb);
            fnv.add(w.data(), wb);
            if (h.has_v) fnv.add(v.data(), wb);
            if (fnv.h != h.checksum) rc = fail(PS_EIO, "checkpoint checksum mismatch");
        }
    }
    std::fclose(f);
    if (rc != PS_OK) return rc;
    if (int rc2 = use_device(ps)) return rc2;
    if (int rc2 = drain_pulls(ps)) return rc2;
    hipError_t e = hipStreamSynchronize(ps->stream);
    if (e == hipSuccess) e = hipMemcpy(ps->w, w.data(), h.n * sizeof(float), hipMemcpyHostToDevice);
    if (e == hipSuccess && ps->v)
        e = hipMemcpy(ps->v, v.data(), h.n * sizeof(float), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail_hip(e, "checkpoint upload");
    ps->ts = h.ts;
    ps->last_served = static_cast<int>(h.last_served);
    ps->learner_ts.assign(lts.begin(), lts.end());
    ps->last_pull.assign(lts.size(), PullKey{});
    clear_last(ps);
    ps->stats = ps_stats{};
    ps->stats.timestamp = ps->ts;
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
    if (ps->mode == PS_QUEUE_FIFO && static_cast<size_t>(depth) < ps->fifo.size())
        return fail(PS_ESTATE, "%zu gradients pending, more than depth %d", ps->fifo.size(), depth);
    ps->depth = depth;
    return PS_OK;
}

int ps_set_queue_mode(ps_server *ps, int mode, int slots_per_learner) {
    if (int rc = check(ps)) return rc;
    if (mode != PS_QUEUE_FIFO && mode != PS_QUEUE_ROUND_ROBIN)
        return fail(PS_EINVAL, "bad queue mode %d", mode);
    if (mode == PS_QUEUE_ROUND_ROBIN &&
        (slots_per_learner < 1 || slots_per_learner > PS_MAX_QUEUE_DEPTH))
        return fail(PS_EINVAL, "slots per learner %d outside [1, %d]", slots_per_learner,
                    PS_MAX_QUEUE_DEPTH);
    if (pending(ps) != 0) return fail(PS_ESTATE, "gradients pending");
    ps->mode = mode;
    if (mode == PS_QUEUE_ROUND_ROBIN) ps->slots = slots_per_learner;
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
    if (pending(ps) != 0) return fail(PS_ESTATE, "gradients pending");
    if (int rc = use_device(ps)) return rc;
    if (int rc = drain_pulls(ps)) return rc;
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
    ps->last_applied.clear();
    ps->last_served = -1;
    ps->stats = ps_stats{};
    return PS_OK;
}

const float *ps_weights(const ps_server *ps) { return ps ? ps->w : nullptr; }
const float *ps_velocity(const ps_server *ps) { return ps ? ps->v : nullptr; }
size_t ps_num_params(const ps_server *ps) { return ps ? ps->n : 0; }
uint64_t ps_timestamp(const ps_server *ps) { return ps ? ps->ts : 0; }

int ps_pending(const ps_server *ps) {
    if (int rc = check(ps)) return rc;
    return static_cast<int>(pending(ps));
}

int ps_last_staleness(const ps_server *ps, int64_t *out, int cap) {
    if (int rc = check(ps)) return rc;
    if (cap < 0 || (cap > 0 && out == nullptr)) return fail(PS_EINVAL, "bad output buffer");
    const int count = static_cast<int>(ps->last_staleness.size());
    for (int i = 0; i < count && i < cap; ++i) out[i] = ps->last_staleness[i];
    return count;
}

int ps_last_applied(const ps_server *ps, int *learner_ids, int cap) {
    if (int rc = check(ps)) return rc;
    if (cap < 0 || (cap > 0 && learner_ids == nullptr)) return fail(PS_EINVAL, "bad output buffer");
    const int count = static_cast<int>(ps->last_applied.size());
    for (int i = 0; i < count && i < cap; ++i) learner_ids[i] = ps->last_applied[i];
    return count;
}

int ps_sync(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    if (int rc = use_device(ps)) return rc;
    hipError_t e = hipStreamSynchronize(ps->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    return drain_pulls(ps);
}

int ps_record(ps_server *ps, void *event) {
    if (int rc = check(ps)) return rc;
    if (event == nullptr) return fail(PS_EINVAL, "null event");
    if (int rc = use_device(ps)) return rc;
    hipError_t e = hipEventRecord(static_cast<hipEvent_t>(event), ps->stream);
    if (e != hipSuccess) return fail_hip(e, "hipEventRecord");
    return PS_OK;
}

int ps_set_pull_stream(ps_server *ps, void *hip_stream) {
    if (int rc = check(ps)) return rc;
    if (int rc = use_device(ps)) return rc;
    if (int rc = drain_pulls(ps)) return rc;
    ps->pull_lock_free = hip_stream != nullptr;
    ps->pull_stream = static_cast<hipStream_t>(hip_stream);
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
