// Host-side protocol state of the parameter server (Sec. 2.1, 4.1, 4.2):
// the gradient queues with their fixed number of slots, the scalar
// timestamp, each learner's timestamp and last pull, and the staleness
// statistics. Plain C++ without device calls: ps_server.cpp drives the
// kernels from it, and the same code builds and runs on the host alone.
//
// Queue modes. FIFO: one queue of `depth` slots in push-call order. Round
// robin: every learner has its own queue of `slots` slots (the paper's lambda
// single-producer single-consumer queues) and the server visits learners in
// increasing id order, cyclically, starting after the learner it served
// last, taking one gradient per visit (Sec. 4.1). Either way an apply takes a
// "batch" of at most `depth` gradients, which the kernels fold in order.
//
// Every operation that can fail validates first and changes nothing on
// failure; the plan_* / commit_* split lets the caller launch device work
// between the two and commit only what it launched.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <deque>
#include <set>
#include <utility>
#include <vector>

#include "ps.h"

namespace gadei {

// Record the message of a failed call (read back by ps_last_error, per
// thread) and return `code`.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
const char *last_error();

int check_learner(int id);

struct PushDesc {
    int learner;
    int dtype;             // PS_F32 | PS_BF16
    const void *grad;      // borrowed device buffer
    uint64_t learner_ts;   // timestamp of the weights the learner held at push
    void *ready;           // producer event (a hipEvent_t) the apply waits for, or null
};

struct PullKey {
    const void *dst = nullptr;
    int dtype = -1;
    uint64_t ts = 0;
    bool valid = false;
};

// The gradients an apply takes, in the order it applies them, and how many
// each learner queue gives (round-robin mode).
struct Batch {
    std::vector<PushDesc> items;
    std::vector<std::pair<int, int>> taken;   // (learner, count), round robin
    int last_served = -1;
};

struct Protocol {
    int mode = PS_QUEUE_FIFO;
    int depth = PS_MAX_QUEUE_DEPTH / 2;
    int slots = 1;                       // round robin: slots per learner
    bool pull_skip = true;
    int last_served = -1;                // round robin: last learner served
    uint64_t ts = 0;                     // applied gradients (Sec. 2.1)
    std::vector<uint64_t> learner_ts;    // indexed by learner id, grown on demand
    std::vector<PullKey> last_pull;
    std::vector<int64_t> last_staleness; // of the most recent apply, in order
    std::vector<int> last_applied;       // ... and the learners applied
    ps_stats stats{};

    Protocol();

    size_t pending() const;

    // Enqueue one gradient; PS_EFULL (nothing enqueued) on a full queue.
    int push(int learner, int dtype, const void *grad, void *ready);

    // Asynchronous apply: FIFO takes every pending gradient in push order;
    // round robin up to `depth` in service order. Nothing is removed.
    void plan_async(Batch &b) const;
    // Synchronous step: FIFO takes every pending gradient in push order;
    // round robin the oldest gradient of every waiting learner, increasing
    // id. PS_ESTATE if more than PS_MAX_QUEUE_DEPTH, PS_EINVAL if the
    // dtypes differ. The batch must not be empty.
    int plan_sync(Batch &b) const;
    // The batch was launched: staleness of each gradient when applied, the
    // timestamp (one step per gradient, or one for the whole synchronous
    // step), and the batch leaves its queues.
    void commit_async(const Batch &b);
    void commit_sync(const Batch &b);
    // An apply call with nothing to apply: the last-apply queries then
    // report an empty apply.
    void clear_last();

    // Which of the n requested pulls must write once the weights carry
    // timestamp `ts_after`. A pull is skipped when the same learner last
    // pulled into the same buffer, same dtype, at ts_after (Sec. 4.1);
    // duplicates inside one call see the earlier entry's effect. Two written
    // pulls may not share a buffer.
    int plan_pulls(int n, const int *ids, void *const *dsts, int dtype, uint64_t ts_after,
                   std::vector<int> &write) const;
    // `ordered`: the replicas were written after every earlier apply, so
    // they hold the weights at the current timestamp and a repeat can be
    // skipped. A lock-free pull may have raced an apply: its replicas never
    // count as current.
    void commit_pulls(int n, const int *ids, void *const *dsts, int dtype,
                      const std::vector<int> &write, bool ordered);

    // Whether a queued gradient starts in [lo, hi).
    bool references(const void *lo, const void *hi) const;

    // Discard a dead learner's queued gradients (Sec. 4.3); returns the count.
    int drop_learner(int learner);
    // A dead learner whose queued gradients stay queued and are applied in
    // their turn (the stateless server of Sec. 4.3; Theorem 2): later pushes
    // and pulls under its id are refused with PS_ESTATE until reset() or
    // restore(). Returns how many of its gradients are still queued.
    int retire_learner(int learner);
    bool retired(int learner) const;
    // The queued gradients of one learner, oldest first.
    std::vector<PushDesc> queued_of(int learner) const;
    int set_depth(int new_depth);
    int set_mode(int new_mode, int slots_per_learner);
    // New weights: timestamp 0, every learner at 0, history and stats cleared.
    void reset();
    // State restored from a checkpoint; pull history and stats start afresh.
    void restore(uint64_t new_ts, int new_last_served, const std::vector<uint64_t> &lts);

   private:
    std::vector<PushDesc> fifo_;             // FIFO mode
    std::vector<std::deque<PushDesc>> rr_;   // round robin: queue of each learner id
    std::set<int> waiting_;                  // ... ids whose queue is not empty
    size_t rr_count_ = 0;
    std::set<int> retired_;                  // learners retired (retire_learner)

    void grow(int id);
    void consume(const Batch &b);
    void record_staleness(const PushDesc &d, uint64_t at);
};

}  // namespace gadei
