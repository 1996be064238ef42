// Host-side protocol state of the parameter server; see ps_protocol.h.
#include "ps_protocol.h"

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <string>

namespace gadei {

namespace {
thread_local std::string g_err;
}  // namespace

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

const char *last_error() { return g_err.c_str(); }

int check_learner(int id) {
    if (id < 0 || id >= PS_MAX_LEARNERS)
        return fail(PS_EINVAL, "learner id %d outside [0, %d)", id, PS_MAX_LEARNERS);
    return PS_OK;
}

Protocol::Protocol() { fifo_.reserve(PS_MAX_QUEUE_DEPTH); }

size_t Protocol::pending() const { return mode == PS_QUEUE_FIFO ? fifo_.size() : rr_count_; }

void Protocol::grow(int id) {
    if (static_cast<size_t>(id) >= learner_ts.size()) {
        learner_ts.resize(static_cast<size_t>(id) + 1, 0);
        last_pull.resize(static_cast<size_t>(id) + 1);
    }
}

int Protocol::push(int learner, int dtype, const void *grad, void *ready) {
    if (int rc = check_learner(learner)) return rc;
    if (grad == nullptr) return fail(PS_EINVAL, "null gradient");
    if (dtype != PS_F32 && dtype != PS_BF16) return fail(PS_EINVAL, "bad gradient dtype %d", dtype);
    if (retired(learner)) return fail(PS_ESTATE, "learner %d has retired", learner);
    const uint64_t lts =
        static_cast<size_t>(learner) < learner_ts.size() ? learner_ts[learner] : 0;
    const PushDesc d{learner, dtype, grad, lts, ready};
    if (mode == PS_QUEUE_FIFO) {
        if (static_cast<int>(fifo_.size()) >= depth) {
            stats.pushes_rejected += 1;
            return fail(PS_EFULL, "queue full (%d pending)", depth);
        }
        fifo_.push_back(d);
    } else {
        if (static_cast<size_t>(learner) >= rr_.size()) rr_.resize(static_cast<size_t>(learner) + 1);
        auto &q = rr_[learner];
        if (static_cast<int>(q.size()) >= slots) {
            stats.pushes_rejected += 1;
            return fail(PS_EFULL, "learner %d queue full (%d slots)", learner, slots);
        }
        q.push_back(d);
        waiting_.insert(learner);
        rr_count_ += 1;
    }
    stats.pushes_accepted += 1;
    return PS_OK;
}

void Protocol::plan_async(Batch &b) const {
    b.items.clear();
    b.taken.clear();
    b.last_served = last_served;
    if (mode == PS_QUEUE_FIFO) {
        b.items = fifo_;
        return;
    }
    std::vector<std::pair<int, size_t>> avail;   // (learner, queued), increasing id
    for (int l : waiting_) avail.emplace_back(l, rr_[l].size());
    std::vector<size_t> used(avail.size(), 0);
    size_t left = rr_count_;
    int cur = last_served;
    while (static_cast<int>(b.items.size()) < depth && left > 0) {
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
        b.items.push_back(rr_[l][used[pick]]);
        ++used[pick];
        --left;
        cur = l;
    }
    for (size_t j = 0; j < avail.size(); ++j)
        if (used[j]) b.taken.emplace_back(avail[j].first, static_cast<int>(used[j]));
    b.last_served = cur;
}

int Protocol::plan_sync(Batch &b) const {
    b.items.clear();
    b.taken.clear();
    b.last_served = last_served;
    if (mode == PS_QUEUE_FIFO) {
        b.items = fifo_;
    } else {
        for (int l : waiting_) {
            b.items.push_back(rr_[l].front());
            b.taken.emplace_back(l, 1);
        }
    }
    if (b.items.size() > PS_MAX_QUEUE_DEPTH)
        return fail(PS_ESTATE, "%zu learners waiting, more than one step can average (%d)",
                    b.items.size(), PS_MAX_QUEUE_DEPTH);
    for (const PushDesc &d : b.items)
        if (d.dtype != b.items.front().dtype)
            return fail(PS_EINVAL, "synchronous step needs one gradient dtype");
    return PS_OK;
}

void Protocol::consume(const Batch &b) {
    if (mode == PS_QUEUE_FIFO) {
        fifo_.erase(fifo_.begin(), fifo_.begin() + static_cast<ptrdiff_t>(b.items.size()));
        return;
    }
    for (const auto &t : b.taken) {
        auto &q = rr_[t.first];
        for (int i = 0; i < t.second; ++i) q.pop_front();
        if (q.empty()) waiting_.erase(t.first);
    }
    rr_count_ -= b.items.size();
    last_served = b.last_served;
}

void Protocol::record_staleness(const PushDesc &d, uint64_t at) {
    const uint64_t u = at - d.learner_ts;
    last_staleness.push_back(static_cast<int64_t>(u));
    last_applied.push_back(d.learner);
    stats.staleness_sum += u;
    stats.staleness_max = std::max(stats.staleness_max, u);
    stats.staleness_hist[std::min<uint64_t>(u, PS_STALENESS_BINS - 1)] += 1;
}

void Protocol::commit_async(const Batch &b) {
    clear_last();
    for (const PushDesc &d : b.items) {
        record_staleness(d, ts);
        ts += 1;
    }
    stats.pushes_applied += b.items.size();
    stats.applies += 1;
    stats.timestamp = ts;
    consume(b);
}

void Protocol::commit_sync(const Batch &b) {
    // one update: every gradient is applied at the same timestamp
    clear_last();
    for (const PushDesc &d : b.items) record_staleness(d, ts);
    ts += 1;
    stats.pushes_applied += b.items.size();
    stats.applies += 1;
    stats.timestamp = ts;
    consume(b);
}

void Protocol::clear_last() {
    last_staleness.clear();
    last_applied.clear();
}

int Protocol::plan_pulls(int n, const int *ids, void *const *dsts, int dtype, uint64_t ts_after,
                         std::vector<int> &write) const {
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
        if (retired(ids[i])) return fail(PS_ESTATE, "learner %d has retired", ids[i]);
        const int l = ids[i];
        bool current = false;
        if (pull_skip) {
            for (auto &s : seen)
                if (s.first == l && s.second == dsts[i]) current = true;
            if (!current && static_cast<size_t>(l) < last_pull.size()) {
                const PullKey &k = last_pull[l];
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

void Protocol::commit_pulls(int n, const int *ids, void *const *dsts, int dtype,
                            const std::vector<int> &write, bool ordered) {
    stats.pulls += static_cast<uint64_t>(n);
    stats.pulls_skipped += static_cast<uint64_t>(n) - write.size();
    for (int i = 0; i < n; ++i) {
        grow(ids[i]);
        learner_ts[ids[i]] = ts;
    }
    for (int i : write) {
        PullKey &k = last_pull[ids[i]];
        k.dst = dsts[i];
        k.dtype = dtype;
        k.ts = ts;
        k.valid = ordered;
    }
}

bool Protocol::references(const void *lo, const void *hi) const {
    const auto in = [&](const PushDesc &d) {
        const char *g = static_cast<const char *>(d.grad);
        return g >= static_cast<const char *>(lo) && g < static_cast<const char *>(hi);
    };
    for (const PushDesc &d : fifo_)
        if (in(d)) return true;
    for (const auto &q : rr_)
        for (const PushDesc &d : q)
            if (in(d)) return true;
    return false;
}

int Protocol::drop_learner(int learner) {
    if (int rc = check_learner(learner)) return rc;
    int dropped = 0;
    if (mode == PS_QUEUE_FIFO) {
        auto keep = std::remove_if(fifo_.begin(), fifo_.end(),
                                   [&](const PushDesc &d) { return d.learner == learner; });
        dropped = static_cast<int>(fifo_.end() - keep);
        fifo_.erase(keep, fifo_.end());
    } else if (static_cast<size_t>(learner) < rr_.size()) {
        dropped = static_cast<int>(rr_[learner].size());
        rr_[learner].clear();
        waiting_.erase(learner);
        rr_count_ -= static_cast<size_t>(dropped);
    }
    stats.pushes_dropped += static_cast<uint64_t>(dropped);
    return dropped;
}

int Protocol::retire_learner(int learner) {
    if (int rc = check_learner(learner)) return rc;
    retired_.insert(learner);
    return static_cast<int>(queued_of(learner).size());
}

bool Protocol::retired(int learner) const { return retired_.count(learner) != 0; }

std::vector<PushDesc> Protocol::queued_of(int learner) const {
    std::vector<PushDesc> out;
    if (mode == PS_QUEUE_FIFO) {
        for (const PushDesc &d : fifo_)
            if (d.learner == learner) out.push_back(d);
    } else if (learner >= 0 && static_cast<size_t>(learner) < rr_.size()) {
        out.assign(rr_[learner].begin(), rr_[learner].end());
    }
    return out;
}

int Protocol::set_depth(int new_depth) {
    if (new_depth < 1 || new_depth > PS_MAX_QUEUE_DEPTH)
        return fail(PS_EINVAL, "queue depth %d outside [1, %d]", new_depth, PS_MAX_QUEUE_DEPTH);
    if (mode == PS_QUEUE_FIFO && static_cast<size_t>(new_depth) < fifo_.size())
        return fail(PS_ESTATE, "%zu gradients pending, more than depth %d", fifo_.size(),
                    new_depth);
    depth = new_depth;
    return PS_OK;
}

int Protocol::set_mode(int new_mode, int slots_per_learner) {
    if (new_mode != PS_QUEUE_FIFO && new_mode != PS_QUEUE_ROUND_ROBIN)
        return fail(PS_EINVAL, "bad queue mode %d", new_mode);
    if (new_mode == PS_QUEUE_ROUND_ROBIN &&
        (slots_per_learner < 1 || slots_per_learner > PS_MAX_QUEUE_DEPTH))
        return fail(PS_EINVAL, "slots per learner %d outside [1, %d]", slots_per_learner,
                    PS_MAX_QUEUE_DEPTH);
    if (pending() != 0) return fail(PS_ESTATE, "gradients pending");
    mode = new_mode;
    if (new_mode == PS_QUEUE_ROUND_ROBIN) slots = slots_per_learner;
    return PS_OK;
}

void Protocol::reset() {
    retired_.clear();
    ts = 0;
    learner_ts.clear();
    last_pull.clear();
    clear_last();
    last_served = -1;
    stats = ps_stats{};
}

void Protocol::restore(uint64_t new_ts, int new_last_served, const std::vector<uint64_t> &lts) {
    retired_.clear();
    ts = new_ts;
    last_served = new_last_served;
    learner_ts = lts;
    last_pull.assign(lts.size(), PullKey{});
    clear_last();
    stats = ps_stats{};
    stats.timestamp = ts;
}

}  // namespace gadei
