// Drives the parameter server's host protocol (gadei::Protocol: queues,
// timestamps, pull skipping, staleness) from a command script on stdin, the
// way the C ABI drives it around its kernel launches, and prints one line per
// command. Built with the host sanitizers by tests/test_protocol.py, which
// runs the same script through the oracle's server and compares the lines.
//
// Commands (one per line):
//   push L DT ID          gradient ID of learner L, dtype DT
//   apply                 asynchronous apply (ps_apply_pending)
//   sync                  synchronous step (ps_apply_sync)
//   pull DT L1 D1 ...     ordered pulls of learners Li into buffers Di (ps_pull_many)
//   applypull DT L1 D1 .. ps_apply_pull
//   drop L | retire L | depth K | mode M S | skip 0|1 | state
//   fronts A1 A2 ...      front choice for streams at addresses Ai (0 = none)
//   rows B C              row layout of C rows of B bytes: head stride span
//   shape K M B [N]       launch shape of a K-gradient apply (M = 1: momentum; B = 1: bf16)
//                         over N coordinates (default 138,357,544)
//   sync_shape K M B      the same for a synchronous step over K learners
//   fuse R K [N]          1 if ps_apply_pull writes R replicas from the apply of K gradients
//                         over N coordinates (default 138,357,544)
#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "ps_layout.h"
#include "ps_protocol.h"

namespace {

const void *grad_ptr(long id) { return reinterpret_cast<const void *>((id + 1) * 64); }
void *dst_ptr(long d) { return reinterpret_cast<void *>((d + 1) * 4096); }

void print_applied(const gadei::Protocol &p) {
    std::printf(" ts=%llu", static_cast<unsigned long long>(p.ts));
    for (size_t i = 0; i < p.last_applied.size(); ++i)
        std::printf(" %d:%lld", p.last_applied[i], static_cast<long long>(p.last_staleness[i]));
}

void read_pulls(std::istringstream &in, int &dt, std::vector<int> &ids, std::vector<void *> &dsts) {
    in >> dt;
    long l, d;
    while (in >> l >> d) {
        ids.push_back(static_cast<int>(l));
        dsts.push_back(dst_ptr(d));
    }
}

void print_written(const std::vector<int> &write) {
    std::printf(" w=");
    for (size_t i = 0; i < write.size(); ++i) std::printf(i ? ",%d" : "%d", write[i]);
}

}  // namespace

int main() {
    gadei::Protocol p;
    std::string line;
    while (std::getline(std::cin, line)) {
        std::istringstream in(line);
        std::string cmd;
        if (!(in >> cmd)) continue;
        if (cmd == "push") {
            long l, dt, id;
            in >> l >> dt >> id;
            std::printf("push %d", p.push(static_cast<int>(l), static_cast<int>(dt), grad_ptr(id),
                                          nullptr));
        } else if (cmd == "apply") {
            if (p.pending() == 0) {
                p.clear_last();
            } else {
                gadei::Batch b;
                p.plan_async(b);
                p.commit_async(b);
            }
            std::printf("apply 0");
            print_applied(p);
        } else if (cmd == "sync") {
            int rc = 0;
            if (p.pending() == 0) {
                p.clear_last();
            } else {
                gadei::Batch b;
                rc = p.plan_sync(b);
                if (rc == 0) p.commit_sync(b);
            }
            std::printf("sync %d", rc);
            print_applied(p);
        } else if (cmd == "pull") {
            int dt = 0;
            std::vector<int> ids;
            std::vector<void *> dsts;
            read_pulls(in, dt, ids, dsts);
            std::vector<int> write;
            const int n = static_cast<int>(ids.size());
            int rc = p.plan_pulls(n, ids.data(), dsts.data(), dt, p.ts, write);
            if (rc == 0) p.commit_pulls(n, ids.data(), dsts.data(), dt, write, true);
            else write.clear();
            std::printf("pull %d", rc);
            print_written(write);
        } else if (cmd == "applypull") {
            int dt = 0;
            std::vector<int> ids;
            std::vector<void *> dsts;
            read_pulls(in, dt, ids, dsts);
            const int n = static_cast<int>(ids.size());
            std::vector<int> write;
            int rc;
            if (p.pending() == 0) {
                rc = p.plan_pulls(n, ids.data(), dsts.data(), dt, p.ts, write);
                if (rc == 0) {
                    p.commit_pulls(n, ids.data(), dsts.data(), dt, write, true);
                    p.clear_last();
                }
            } else {
                gadei::Batch b;
                p.plan_async(b);
                rc = p.plan_pulls(n, ids.data(), dsts.data(), dt, p.ts + b.items.size(), write);
                if (rc == 0) {
                    p.commit_async(b);
                    p.commit_pulls(n, ids.data(), dsts.data(), dt, write, true);
                }
            }
            if (rc != 0) write.clear();
            std::printf("applypull %d", rc);
            print_applied(p);
            print_written(write);
        } else if (cmd == "drop") {
            long l;
            in >> l;
            std::printf("drop %d", p.drop_learner(static_cast<int>(l)));
        } else if (cmd == "retire") {
            long l;
            in >> l;
            std::printf("retire %d", p.retire_learner(static_cast<int>(l)));
        } else if (cmd == "depth") {
            long k;
            in >> k;
            std::printf("depth %d", p.set_depth(static_cast<int>(k)));
        } else if (cmd == "mode") {
            long m, s;
            in >> m >> s;
            std::printf("mode %d", p.set_mode(static_cast<int>(m), static_cast<int>(s)));
        } else if (cmd == "skip") {
            long on;
            in >> on;
            p.pull_skip = on != 0;
            std::printf("skip");
        } else if (cmd == "fronts") {
            std::vector<const void *> ptrs;
            unsigned long long a;
            while (in >> a) ptrs.push_back(reinterpret_cast<const void *>(static_cast<uintptr_t>(a)));
            std::printf("fronts %d", gadei::fronts_log2_for(ptrs.data(), static_cast<int>(ptrs.size())));
        } else if (cmd == "rows") {
            unsigned long long bytes;
            long count;
            in >> bytes >> count;
            const gadei::RowLayout r = gadei::row_layout(bytes, static_cast<int>(count));
            std::printf("rows %zu %zu %zu %zu", r.head, r.stride, r.span,
                        gadei::velocity_offset(bytes));
        } else if (cmd == "fuse") {
            long r, k;
            size_t n = 138357544;
            in >> r >> k;
            if (!(in >> n)) n = 138357544;
            std::printf("fuse %d",
                        gadei::fuse_replicas(static_cast<int>(r), static_cast<int>(k), n) ? 1 : 0);
        } else if (cmd == "shape" || cmd == "sync_shape") {
            long k, m, b = 0;
            size_t n = 138357544;
            in >> k >> m >> b;
            if (!(in >> n)) n = 138357544;
            const gadei::ApplyShape sh =
                cmd == "shape" ? gadei::apply_shape(static_cast<int>(k), m != 0, b != 0, n)
                               : gadei::sync_shape(static_cast<int>(k), m != 0, b != 0);
            std::printf("%s %d %d %d", cmd.c_str(), sh.blocks_per_cu, sh.fronts_log2, sh.group);
        } else if (cmd == "state") {
            std::printf("state ts=%llu pending=%zu pulls=%llu skipped=%llu smax=%llu ssum=%llu hist=",
                        static_cast<unsigned long long>(p.ts), p.pending(),
                        static_cast<unsigned long long>(p.stats.pulls),
                        static_cast<unsigned long long>(p.stats.pulls_skipped),
                        static_cast<unsigned long long>(p.stats.staleness_max),
                        static_cast<unsigned long long>(p.stats.staleness_sum));
            for (int b = 0; b < PS_STALENESS_BINS; ++b)
                if (p.stats.staleness_hist[b])
                    std::printf("%d:%llu,", b, static_cast<unsigned long long>(p.stats.staleness_hist[b]));
        } else {
            std::fprintf(stderr, "unknown command: %s\n", cmd.c_str());
            return 2;
        }
        std::printf("\n");
    }
    return 0;
}
