// Host side of the parameter server: the C ABI declared in include/ps.h.
//
// The protocol state of the paper's server (Sec. 2.1, 4.1) -- queues,
// timestamps, pull history, staleness -- lives in gadei::Protocol
// (ps_protocol.h), which does no device work. This file owns the device side:
// w and v in HBM, the server's stream, and the kernel launches. ps_push moves
// no data, an apply launches one kernel per run of equal-dtype gradients, a
// pull launches one fan-out. Every call validates and plans on the host,
// launches, and only then commits the protocol state.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "ps.h"
#include "ps_kernels.h"
#include "ps_layout.h"
#include "ps_protocol.h"

using gadei::align_up;
using gadei::Batch;
using gadei::fail;
using gadei::kRowAlign;
using gadei::PushDesc;

namespace {

// One device allocation carved into staggered rows (ps_alloc_rows).
struct RowSet {
    void *base;          // what hipMalloc returned
    char *first;         // row 0
    char *end;           // one past the last row's data
};

}  // namespace

// One kernel launch of a call, with every argument it was given: the plan
// that a captured graph (ps_graph_create) replays. Zero-filled before use,
// so two records compare equal byte for byte exactly when the launches are
// the same.
struct LaunchRecord {
    int kind;   // 0 apply, 1 synchronous step, 2 pull fan-out
    int grad_dtype;
    int pull_dtype;
    int level;
    int blocks_per_cu;
    int group;
    gadei::ApplyArgs apply;
    gadei::PullArgs pull;
};

struct ps_server {
    size_t n = 0;
    float lr = 0.0f;
    float m = 0.0f;
    void *wv_base = nullptr;   // one allocation holding w and v
    float *w = nullptr;
    float *v = nullptr;
    std::vector<RowSet> row_sets;
    int device = 0;
    hipStream_t stream = nullptr;
    hipStream_t pull_stream = nullptr;   // lock-free pulls when pull_lock_free
    bool pull_lock_free = false;
    // recorded on pull_stream so that ps_apply_pull's replica writes follow
    // earlier lock-free pulls into the same buffers
    hipEvent_t pulls_done = nullptr;
    // ps_apply_pull writes up to this many replicas in the apply pass; -1:
    // chosen per call (fuse_replicas)
    int fuse_max_r = -1;
    // ps_set_launch_shape: -1 / 0 = the shape tables' choice
    int force_blocks_per_cu = -1;
    int force_group = 0;
    gadei::Geometry geo;
    gadei::Protocol proto;
    // ps_graph_create / ps_graph_launch: the launches of the calls in
    // progress are recorded here; with plan_only they are not made
    std::vector<LaunchRecord> *record = nullptr;
    bool plan_only = false;
    // Every call on the handle holds this lock, so several host threads (a
    // push thread per learner, as in Sec. 4.1) may share one server; device
    // work is enqueued in lock order. Recursive: some calls use others.
    mutable std::recursive_mutex mu;
};

#define PS_LOCK(ps) std::lock_guard<std::recursive_mutex> ps_lock_(ps->mu)

namespace {

int fail_hip(hipError_t e, const char *what) {
    return fail(PS_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Vector level a buffer allows (see launch_apply): 2 if 16-byte aligned, 1 if
// a bf16 buffer is 8-byte aligned, else 0.
int level_of(const void *p, int dtype) {
    if (aligned(p, 16)) return 2;
    if (dtype == PS_BF16 && aligned(p, 8)) return 1;
    return 0;
}

// Whether [p, p + bytes) shares a byte with w or v.
bool overlaps_state(const ps_server *ps, const void *p, size_t bytes) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = a + bytes;
    for (const float *x : {static_cast<const float *>(ps->w), static_cast<const float *>(ps->v)}) {
        if (x == nullptr) continue;
        const uintptr_t lo = reinterpret_cast<uintptr_t>(x), hi = lo + ps->n * sizeof(float);
        if (a < hi && lo < b) return true;
    }
    return false;
}

size_t elem_bytes(int dtype) { return dtype == PS_BF16 ? 2 : 4; }

// Replica buffers must not overlap w or v (a bf16 replica written over w
// would corrupt it). Called after plan_pulls has validated the arguments.
int check_dsts(const ps_server *ps, int n, void *const *dsts, int dtype) {
    for (int i = 0; i < n; ++i)
        if (overlaps_state(ps, dsts[i], ps->n * elem_bytes(dtype)))
            return fail(PS_EINVAL, "destination %d overlaps the server's w or v", i);
    return PS_OK;
}

int check(const ps_server *ps) {
    if (ps == nullptr) return fail(PS_EINVAL, "null server handle");
    return PS_OK;
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

// Make the server's stream wait (on the device) for every producer event of
// the batch, each once.
int wait_ready(ps_server *ps, const std::vector<PushDesc> &items) {
    std::vector<void *> seen;
    for (const PushDesc &d : items) {
        if (d.ready == nullptr || std::find(seen.begin(), seen.end(), d.ready) != seen.end())
            continue;
        seen.push_back(d.ready);
        hipError_t e = hipStreamWaitEvent(ps->stream, static_cast<hipEvent_t>(d.ready), 0);
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

// Fronts for an apply over a.g[0..k) of dtype gdt (-1: no shape table), w
// and v: the server's setting, or chosen from the buffers' offsets
// (fronts_log2_for), and for buffers at distinct offsets from the apply's
// shape (apply_shape).
int fronts_for(const ps_server *ps, const gadei::ApplyArgs &a, int gdt) {
    if (ps->geo.fronts_log2 >= 0) return ps->geo.fronts_log2;
    const void *p[PS_MAX_QUEUE_DEPTH + 2];
    int c = 0;
    for (int j = 0; j < a.k; ++j) p[c++] = a.g[j];
    p[c++] = a.w;
    p[c++] = a.v;   // null without momentum: not a stream
    const int f = gadei::fronts_log2_for(p, c);
    if (f == 0 && gdt >= 0)
        return gadei::apply_shape(a.k, a.v != nullptr, gdt == PS_BF16, a.n).fronts_log2;
    return f;
}

// The launch shape for a table entry, with the caller's overrides.
gadei::Shape shape_for(const ps_server *ps, const gadei::ApplyShape &t) {
    gadei::Shape shape;
    shape.blocks_per_cu = ps->force_blocks_per_cu >= 0 ? ps->force_blocks_per_cu : t.blocks_per_cu;
    shape.group = ps->force_group > 0 ? ps->force_group : t.group;
    return shape;
}

// The three kernel launches of the calls, through the recorder.
hipError_t run_apply(ps_server *ps, const gadei::ApplyArgs &a, int gdt, int pdt, int level,
                     const gadei::Shape &shape, bool sync) {
    if (ps->record) {
        LaunchRecord r;
        std::memset(&r, 0, sizeof r);
        r.kind = sync ? 1 : 0;
        r.grad_dtype = gdt;
        r.pull_dtype = pdt;
        r.level = level;
        r.blocks_per_cu = shape.blocks_per_cu;
        r.group = shape.group;
        r.apply = a;
        ps->record->push_back(r);
    }
    if (ps->plan_only) return hipSuccess;
    return sync ? gadei::launch_sync(a, gdt, level, shape, ps->geo, ps->stream)
                : gadei::launch_apply(a, gdt, pdt, level, shape, ps->geo, ps->stream);
}

hipError_t run_pull(ps_server *ps, const gadei::PullArgs &a, int dtype, int level, hipStream_t s) {
    if (ps->record) {
        LaunchRecord r;
        std::memset(&r, 0, sizeof r);
        r.kind = 2;
        r.pull_dtype = dtype;
        r.level = level;
        r.pull = a;
        ps->record->push_back(r);
    }
    if (ps->plan_only) return hipSuccess;
    return gadei::launch_pull(a, dtype, level, ps->geo, s);
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
        a.fronts_log2 = fronts_for(ps, a, gdt);
        const gadei::Shape shape =
            shape_for(ps, gadei::apply_shape(a.k, a.v != nullptr, gdt == PS_BF16, a.n));
        int pdt = -1;
        if (end == q && pull_dtype >= 0 && !write.empty()) {
            pdt = pull_dtype;
            a.r = static_cast<int>(write.size());
            for (size_t j = 0; j < write.size(); ++j) {
                a.dst[j] = dsts[write[j]];
                level = std::min(level, level_of(a.dst[j], pull_dtype));
            }
        }
        hipError_t e = run_apply(ps, a, gdt, pdt, level, shape, false);
        if (e != hipSuccess) return fail_hip(e, "apply kernel launch");
        start = end;
    }
    return PS_OK;
}

// Make the server's stream wait (on the device) for every lock-free pull
// enqueued so far. ps_apply_pull marks its replicas current; without this an
// earlier lock-free pull into the same buffer, still running on the pull
// stream, could land after the newer weights.
int order_after_pulls(ps_server *ps) {
    if (!ps->pull_lock_free) return PS_OK;
    hipError_t e = hipEventRecord(ps->pulls_done, ps->pull_stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(ps->stream, ps->pulls_done, 0);
    if (e != hipSuccess) return fail_hip(e, "ordering after lock-free pulls");
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
    hipError_t e = run_pull(ps, a, dtype, level, s);
    if (e != hipSuccess) return fail_hip(e, "pull kernel launch");
    return PS_OK;
}

// ---------------------------------------------------------------- checkpoint
//
// File layout (little-endian, as the host writes it):
//   CkptHeader, then learner_ts[n_learner_ts] (uint64), then w[n] (fp32),
//   then v[n] (fp32) when the server has momentum.
// `checksum` is FNV-1a (64-bit) over the header (with `checksum` itself
// zero) and then every byte after it.

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
    int32_t queue_mode;   // the queue configuration the run was made with:
    int32_t depth;        // a restart under another one would serve the
    int32_t slots;        // gradients in another order
    int32_t reserved;
    uint64_t checksum;
};

constexpr char kMagic[8] = {'G', 'A', 'D', 'E', 'I', 'P', 'S', '1'};
// 2: the checksum covers the header too; 3: the queue configuration is kept
constexpr uint32_t kVersion = 3;
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

// Row sets this process mapped with ps_import_rows: first row -> the base
// hipIpcOpenMemHandle returned and the handle it was opened from.
struct Import {
    void *base;
    hipIpcMemHandle_t handle;
};
std::mutex g_import_mu;
std::map<void *, Import> g_imports;

}  // namespace

// A captured script: its device work as one HIP graph, the launches it was
// captured from, and its own copy of the script (ids and buffer lists).
struct ps_graph {
    ps_server *server = nullptr;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    hipEvent_t done = nullptr;   // recorded after each replay
    std::vector<ps_op> ops;
    std::vector<std::vector<int>> ids;
    std::vector<std::vector<void *>> dsts;
    std::vector<LaunchRecord> plan;
};

namespace {

// What a script needs of the server to be captured or replayed: a stream
// other than the legacy null stream (which cannot be captured), ordered
// pulls only (lock-free pulls run on a second stream), and an empty queue
// (so that the script's applies take only its own pushes).
int graph_state(const ps_server *ps) {
    if (ps->stream == nullptr)
        return fail(PS_ESTATE, "graphs need a server stream other than the null stream");
    if (ps->pull_lock_free) return fail(PS_ESTATE, "graphs need ordered pulls");
    if (ps->proto.pending() != 0) return fail(PS_ESTATE, "gradients pending");
    return PS_OK;
}

// The script's calls made for real or, with plan_only, planned and
// committed on the host without launching; the launches land in *rec.
int run_recorded(ps_server *ps, const ps_graph &g, std::vector<LaunchRecord> &rec, bool plan_only) {
    ps->record = &rec;
    ps->plan_only = plan_only;
    int rc;
    try {
        rc = ps_run(ps, g.ops.data(), static_cast<int>(g.ops.size()), nullptr);
    } catch (...) {
        rc = fail(PS_ENOMEM, "host allocation failed");
    }
    ps->record = nullptr;
    ps->plan_only = false;
    return rc;
}

bool same_plan(const std::vector<LaunchRecord> &a, const std::vector<LaunchRecord> &b) {
    return a.size() == b.size() &&
           (a.empty() || std::memcmp(a.data(), b.data(), a.size() * sizeof(LaunchRecord)) == 0);
}

// Waits for the graph's last replay before freeing it.
void free_graph(ps_graph *g) {
    if (g->done) {
        (void)hipEventSynchronize(g->done);
        (void)hipEventDestroy(g->done);
    }
    if (g->exec) (void)hipGraphExecDestroy(g->exec);
    if (g->graph) (void)hipGraphDestroy(g->graph);
    delete g;
}

}  // namespace

extern "C" {

const char *ps_last_error(void) { return gadei::last_error(); }

int ps_import_rows(const void *handle, size_t offset, void **first_row) {
    if (handle == nullptr || first_row == nullptr) return fail(PS_EINVAL, "null argument");
    hipIpcMemHandle_t h;
    std::memcpy(&h, handle, sizeof h);
    std::lock_guard<std::mutex> lock(g_import_mu);
    for (const auto &kv : g_imports)
        if (std::memcmp(&kv.second.handle, &h, sizeof h) == 0)
            return fail(PS_EINVAL, "row set already imported in this process");
    void *base = nullptr;
    hipError_t e = hipIpcOpenMemHandle(&base, h, hipIpcMemLazyEnablePeerAccess);
    if (e != hipSuccess) return fail_hip(e, "hipIpcOpenMemHandle");
    // the offset must name a byte of the mapped allocation
    void *range_base = nullptr;
    size_t range_size = 0;
    e = hipMemGetAddressRange(&range_base, &range_size, base);
    if (e != hipSuccess || range_base != base || offset >= range_size) {
        (void)hipIpcCloseMemHandle(base);
        if (e != hipSuccess) return fail_hip(e, "hipMemGetAddressRange");
        return fail(PS_EINVAL, "offset %zu outside the %zu-byte allocation", offset, range_size);
    }
    void *first = static_cast<char *>(base) + offset;
    try {
        g_imports[first] = Import{base, h};
    } catch (...) {
        (void)hipIpcCloseMemHandle(base);
        return fail(PS_ENOMEM, "host allocation failed");
    }
    *first_row = first;
    return PS_OK;
}

int ps_release_rows(void *first_row) {
    void *base = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_import_mu);
        auto it = g_imports.find(first_row);
        if (it == g_imports.end()) return fail(PS_EINVAL, "not a row set imported here");
        base = it->second.base;
        g_imports.erase(it);
    }
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipIpcCloseMemHandle(base);
    if (e != hipSuccess) return fail_hip(e, "hipIpcCloseMemHandle");
    return PS_OK;
}

ps_server *ps_create(size_t n_params, float lr, float momentum) {
    if (n_params == 0 || n_params > (size_t(1) << 48)) {
        fail(PS_EINVAL, "n_params must be in [1, 2^48]");
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
    // w and v in one allocation, v one stagger after w's 2 MiB-rounded end
    const size_t bytes = n_params * sizeof(float);
    const size_t v_off = gadei::velocity_offset(bytes);
    hipError_t e = hipGetDevice(&ps->device);
    if (e == hipSuccess)
        e = hipMalloc(&ps->wv_base, (momentum != 0.0f ? v_off + bytes : bytes) + kRowAlign);
    if (e == hipSuccess) {
        char *w = align_up(ps->wv_base, kRowAlign);
        ps->w = reinterpret_cast<float *>(w);
        if (momentum != 0.0f) ps->v = reinterpret_cast<float *>(w + v_off);
        e = hipMemset(ps->w, 0, bytes);
    }
    if (e == hipSuccess && ps->v) e = hipMemset(ps->v, 0, bytes);
    if (e != hipSuccess) {
        fail(e == hipErrorOutOfMemory ? PS_ENOMEM : PS_EHIP, "ps_create: %s", hipGetErrorString(e));
        if (ps->wv_base) (void)hipFree(ps->wv_base);
        delete ps;
        return nullptr;
    }
    for (int b = 1; b <= 4; ++b) ps->geo.lds_for_blocks[b] = gadei::blocks_per_cu_lds(b);
    return ps;
}

void ps_destroy(ps_server *ps) {
    if (ps == nullptr) return;
    {
        PS_LOCK(ps);   // waits for a call still running on another thread
        if (use_device(ps) == PS_OK) {
            (void)hipStreamSynchronize(ps->stream);
            if (ps->pull_lock_free) (void)hipStreamSynchronize(ps->pull_stream);
            for (const RowSet &r : ps->row_sets) (void)hipFree(r.base);
            (void)hipFree(ps->wv_base);
            if (ps->pulls_done) (void)hipEventDestroy(ps->pulls_done);
        }
    }
    delete ps;
}

int ps_alloc_rows(ps_server *ps, int count, int dtype, void **rows) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (count < 1 || count > PS_MAX_ROWS)
        return fail(PS_EINVAL, "row count %d outside [1, %d]", count, PS_MAX_ROWS);
    if (dtype != PS_F32 && dtype != PS_BF16) return fail(PS_EINVAL, "bad row dtype %d", dtype);
    if (rows == nullptr) return fail(PS_EINVAL, "null rows output");
    if (int rc = use_device(ps)) return rc;
    const gadei::RowLayout lay = gadei::row_layout(ps->n * (dtype == PS_BF16 ? 2 : 4), count);
    void *base = nullptr;
    hipError_t e = hipMalloc(&base, lay.span + kRowAlign);
    if (e != hipSuccess)
        return fail(e == hipErrorOutOfMemory ? PS_ENOMEM : PS_EHIP, "ps_alloc_rows: %s",
                    hipGetErrorString(e));
    char *first = align_up(base, kRowAlign) + lay.head;
    try {
        ps->row_sets.push_back(RowSet{base, first, first - lay.head + lay.span});
    } catch (...) {
        (void)hipFree(base);
        return fail(PS_ENOMEM, "host allocation failed");
    }
    for (int i = 0; i < count; ++i) rows[i] = first + static_cast<size_t>(i) * lay.stride;
    return PS_OK;
}

int ps_free_rows(ps_server *ps, void *first_row) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    auto it = std::find_if(ps->row_sets.begin(), ps->row_sets.end(),
                           [&](const RowSet &r) { return r.first == first_row; });
    if (it == ps->row_sets.end()) return fail(PS_EINVAL, "not the first row of a row set");
    if (ps->proto.references(it->first, it->end))
        return fail(PS_ESTATE, "a pending gradient lies in these rows");
    if (int rc = use_device(ps)) return rc;
    if (int rc = drain_pulls(ps)) return rc;
    hipError_t e = hipStreamSynchronize(ps->stream);
    if (e == hipSuccess) e = hipFree(it->base);
    if (e != hipSuccess) return fail_hip(e, "ps_free_rows");
    ps->row_sets.erase(it);
    return PS_OK;
}

int ps_push_async(ps_server *ps, int learner_id, const void *grad, int dtype, void *ready_event) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (grad != nullptr && overlaps_state(ps, grad, ps->n * elem_bytes(dtype)))
        return fail(PS_EINVAL, "gradient buffer overlaps the server's w or v");
    return ps->proto.push(learner_id, dtype, grad, ready_event);
}

int ps_push_dtype(ps_server *ps, int learner_id, const void *grad, int dtype) {
    return ps_push_async(ps, learner_id, grad, dtype, nullptr);
}

int ps_push(ps_server *ps, int learner_id, const void *grad) {
    return ps_push_dtype(ps, learner_id, grad, PS_F32);
}

int ps_apply_pending(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (ps->proto.pending() == 0) {
        ps->proto.clear_last();
        return PS_OK;
    }
    if (int rc = use_device(ps)) return rc;
    Batch b;
    ps->proto.plan_async(b);
    static const std::vector<int> none;
    if (int rc = launch_batch(ps, b.items, -1, nullptr, none)) return rc;
    ps->proto.commit_async(b);
    return PS_OK;
}

int ps_apply_sync(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (ps->proto.pending() == 0) {
        ps->proto.clear_last();
        return PS_OK;
    }
    Batch b;
    if (int rc = ps->proto.plan_sync(b)) return rc;
    const int gdt = b.items.front().dtype;
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
    a.fronts_log2 = fronts_for(ps, a, -1);   // the phase rule only (no apply_shape)
    const gadei::Shape shape = shape_for(ps, gadei::sync_shape(a.k, a.v != nullptr, gdt == PS_BF16));
    hipError_t e = run_apply(ps, a, gdt, -1, level, shape, true);
    if (e != hipSuccess) return fail_hip(e, "synchronous step launch");
    ps->proto.commit_sync(b);
    return PS_OK;
}

int ps_pull_many(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    std::vector<int> write;
    if (int rc = ps->proto.plan_pulls(n, learner_ids, dsts, dst_dtype, ps->proto.ts, write))
        return rc;
    if (int rc = check_dsts(ps, n, dsts, dst_dtype)) return rc;
    if (!write.empty()) {
        if (int rc = use_device(ps)) return rc;
        if (int rc = launch_pulls(ps, dsts, dst_dtype, write, false)) return rc;
    }
    ps->proto.commit_pulls(n, learner_ids, dsts, dst_dtype, write, !ps->pull_lock_free);
    return PS_OK;
}

int ps_pull(ps_server *ps, int learner_id, void *dst) {
    return ps_pull_many(ps, 1, &learner_id, &dst, PS_F32);
}

int ps_apply_pull(ps_server *ps, int n, const int *learner_ids, void *const *dsts, int dst_dtype) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (ps->proto.pending() == 0) {
        const int rc = ps_pull_many(ps, n, learner_ids, dsts, dst_dtype);
        if (rc == PS_OK) ps->proto.clear_last();
        return rc;
    }
    Batch b;
    ps->proto.plan_async(b);
    std::vector<int> write;
    const uint64_t ts_after = ps->proto.ts + b.items.size();
    if (int rc = ps->proto.plan_pulls(n, learner_ids, dsts, dst_dtype, ts_after, write))
        return rc;
    if (int rc = check_dsts(ps, n, dsts, dst_dtype)) return rc;
    if (int rc = use_device(ps)) return rc;
    if (!write.empty())
        if (int rc = order_after_pulls(ps)) return rc;
    const int r = static_cast<int>(write.size());
    const bool fuse = ps->fuse_max_r >= 0 ? r <= ps->fuse_max_r
                                           : gadei::fuse_replicas(r, static_cast<int>(b.items.size()), ps->n);
    if (fuse) {
        if (int rc = launch_batch(ps, b.items, dst_dtype, dsts, write)) return rc;
    } else {
        static const std::vector<int> none;
        if (int rc = launch_batch(ps, b.items, -1, nullptr, none)) return rc;
        if (int rc = launch_pulls(ps, dsts, dst_dtype, write, true)) {
            ps->proto.commit_async(b);   // the apply is on the stream: its gradients are consumed
            return rc;
        }
    }
    ps->proto.commit_async(b);
    ps->proto.commit_pulls(n, learner_ids, dsts, dst_dtype, write, true);
    return PS_OK;
}

int ps_drop_learner(ps_server *ps, int learner_id) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    return ps->proto.drop_learner(learner_id);
}

int ps_retire_learner(ps_server *ps, int learner_id) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (int rc = gadei::check_learner(learner_id)) return rc;
    // its gradients stay queued, so they must live in memory the server
    // owns: a borrowed buffer may have gone with the learner
    for (const PushDesc &d : ps->proto.queued_of(learner_id)) {
        const char *g = static_cast<const char *>(d.grad);
        const size_t bytes = ps->n * elem_bytes(d.dtype);
        const bool owned = std::any_of(ps->row_sets.begin(), ps->row_sets.end(), [&](const RowSet &r) {
            return g >= r.first && g <= r.end && bytes <= static_cast<size_t>(r.end - g);
        });
        if (!owned)
            return fail(PS_ESTATE,
                        "learner %d has a queued gradient outside the server's rows; drop it "
                        "(ps_drop_learner) instead",
                        learner_id);
    }
    return ps->proto.retire_learner(learner_id);
}

static_assert(sizeof(hipIpcMemHandle_t) == PS_IPC_HANDLE_BYTES, "IPC handle size");

int ps_export_rows(ps_server *ps, void *first_row, void *handle, size_t *offset) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (handle == nullptr || offset == nullptr) return fail(PS_EINVAL, "null output");
    auto it = std::find_if(ps->row_sets.begin(), ps->row_sets.end(),
                           [&](const RowSet &r) { return r.first == first_row; });
    if (it == ps->row_sets.end()) return fail(PS_EINVAL, "not the first row of a row set");
    if (int rc = use_device(ps)) return rc;
    hipIpcMemHandle_t h;
    hipError_t e = hipIpcGetMemHandle(&h, it->base);
    if (e != hipSuccess) return fail_hip(e, "hipIpcGetMemHandle");
    std::memcpy(handle, &h, sizeof h);
    *offset = static_cast<size_t>(it->first - static_cast<char *>(it->base));
    return PS_OK;
}

int ps_save(ps_server *ps, const char *path) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (path == nullptr) return fail(PS_EINVAL, "null path");
    if (ps->proto.pending() != 0) return fail(PS_ESTATE, "gradients pending");
    if (int rc = use_device(ps)) return rc;
    if (int rc = drain_pulls(ps)) return rc;
    hipError_t e = hipStreamSynchronize(ps->stream);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    FILE *f = std::fopen(path, "wb");
    if (f == nullptr) return fail(PS_EIO, "cannot open %s for writing", path);
    const gadei::Protocol &pr = ps->proto;
    CkptHeader h;
    std::memset(&h, 0, sizeof h);
    std::memcpy(h.magic, kMagic, sizeof kMagic);
    h.version = kVersion;
    h.has_v = ps->v != nullptr;
    h.n = ps->n;
    h.lr = ps->lr;
    h.m = ps->m;
    h.ts = pr.ts;
    h.last_served = pr.last_served;
    h.n_learner_ts = pr.learner_ts.size();
    h.queue_mode = pr.mode;
    h.depth = pr.depth;
    h.slots = pr.mode == PS_QUEUE_ROUND_ROBIN ? pr.slots : 0;
    Fnv fnv;
    int rc = write_all(f, &h, sizeof h, &fnv);   // checksum still zero here
    std::vector<float> buf;
    if (rc == PS_OK && h.n_learner_ts)
        rc = write_all(f, pr.learner_ts.data(), h.n_learner_ts * sizeof(uint64_t), &fnv);
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
    PS_LOCK(ps);
    if (path == nullptr) return fail(PS_EINVAL, "null path");
    if (ps->proto.pending() != 0) return fail(PS_ESTATE, "gradients pending");
    FILE *f = std::fopen(path, "rb");
    if (f == nullptr) return fail(PS_EIO, "cannot open %s", path);
    CkptHeader h;
    int rc = PS_OK;
    if (std::fread(&h, 1, sizeof h, f) != sizeof h || std::memcmp(h.magic, kMagic, 8) != 0)
        rc = fail(PS_EIO, "%s is not a parameter-server checkpoint", path);
    else if (h.version != kVersion)
        rc = fail(PS_EIO, "checkpoint format version %u; this library reads %u", h.version,
                  kVersion);
    else if (h.n != ps->n || (h.has_v != 0) != (ps->v != nullptr))
        rc = fail(PS_EINVAL, "checkpoint holds %llu params%s; server has %zu%s",
                  static_cast<unsigned long long>(h.n), h.has_v ? " with momentum" : "", ps->n,
                  ps->v ? " with momentum" : "");
    else if (std::memcmp(&h.lr, &ps->lr, sizeof(float)) != 0 ||
             std::memcmp(&h.m, &ps->m, sizeof(float)) != 0)
        rc = fail(PS_EINVAL, "checkpoint lr/momentum differ from the server's");
    else if (h.queue_mode != ps->proto.mode || h.depth != ps->proto.depth ||
             h.slots != (ps->proto.mode == PS_QUEUE_ROUND_ROBIN ? ps->proto.slots : 0))
        rc = fail(PS_EINVAL,
                  "checkpoint queue configuration (mode %d, depth %d, slots %d) differs from "
                  "the server's (mode %d, depth %d, slots %d)",
                  h.queue_mode, h.depth, h.slots, ps->proto.mode, ps->proto.depth,
                  ps->proto.mode == PS_QUEUE_ROUND_ROBIN ? ps->proto.slots : 0);
    else if (h.n_learner_ts > static_cast<uint64_t>(PS_MAX_LEARNERS) || h.last_served < -1 ||
             h.last_served >= PS_MAX_LEARNERS)
        rc = fail(PS_EIO, "corrupt checkpoint (learner table)");
    // read and verify everything before touching the server
    std::vector<uint64_t> lts;
    std::vector<float> w, v;
    Fnv fnv;
    if (rc == PS_OK) {
        CkptHeader z = h;
        z.checksum = 0;
        fnv.add(&z, sizeof z);
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
    ps->proto.restore(h.ts, static_cast<int>(h.last_served), lts);
    return PS_OK;
}

int ps_set_stream(ps_server *ps, void *hip_stream) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    ps->stream = static_cast<hipStream_t>(hip_stream);
    return PS_OK;
}

int ps_set_queue_depth(ps_server *ps, int depth) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    return ps->proto.set_depth(depth);
}

int ps_set_queue_mode(ps_server *ps, int mode, int slots_per_learner) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    return ps->proto.set_mode(mode, slots_per_learner);
}

int ps_set_pull_fusion(ps_server *ps, int max_replicas) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (max_replicas < -1 || max_replicas > PS_MAX_REPLICAS)
        return fail(PS_EINVAL, "fusion limit %d outside [-1, %d]", max_replicas, PS_MAX_REPLICAS);
    ps->fuse_max_r = max_replicas;
    return PS_OK;
}

int ps_set_fronts(ps_server *ps, int fronts_log2) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (fronts_log2 < -1 || fronts_log2 > 3)
        return fail(PS_EINVAL, "fronts_log2 %d outside [-1, 3]", fronts_log2);
    ps->geo.fronts_log2 = fronts_log2;
    return PS_OK;
}

int ps_set_launch_shape(ps_server *ps, int blocks_per_cu, int group) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (blocks_per_cu < -1 || blocks_per_cu > 4)
        return fail(PS_EINVAL, "blocks_per_cu %d outside [-1, 4]", blocks_per_cu);
    if (group != 0 && group != 4 && group != 8 && group != 12 && group != 16 && group != 24 &&
        group != 32)
        return fail(PS_EINVAL, "group %d is not 0, 4, 8, 12, 16, 24 or 32", group);
    ps->force_blocks_per_cu = blocks_per_cu;
    ps->force_group = group;
    return PS_OK;
}

int ps_set_pull_skip(ps_server *ps, int enabled) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    ps->proto.pull_skip = enabled != 0;
    return PS_OK;
}

int ps_set_weights(ps_server *ps, const float *src) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (src == nullptr) return fail(PS_EINVAL, "null source");
    if (overlaps_state(ps, src, ps->n * sizeof(float)))
        return fail(PS_EINVAL, "source overlaps the server's w or v");
    if (ps->proto.pending() != 0) return fail(PS_ESTATE, "gradients pending");
    if (int rc = use_device(ps)) return rc;
    if (int rc = drain_pulls(ps)) return rc;
    hipError_t e = hipMemcpyAsync(ps->w, src, ps->n * sizeof(float), hipMemcpyDeviceToDevice,
                                  ps->stream);
    if (e != hipSuccess) return fail_hip(e, "weights copy");
    if (ps->v) {
        e = gadei::launch_zero(ps->v, ps->n, ps->stream);
        if (e != hipSuccess) return fail_hip(e, "velocity reset");
    }
    ps->proto.reset();
    return PS_OK;
}

const float *ps_weights(const ps_server *ps) { return ps ? ps->w : nullptr; }
const float *ps_velocity(const ps_server *ps) { return ps ? ps->v : nullptr; }
size_t ps_num_params(const ps_server *ps) { return ps ? ps->n : 0; }
uint64_t ps_timestamp(const ps_server *ps) {
    if (ps == nullptr) return 0;
    PS_LOCK(ps);
    return ps->proto.ts;
}

int ps_pending(const ps_server *ps) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    return static_cast<int>(ps->proto.pending());
}

int ps_last_staleness(const ps_server *ps, int64_t *out, int cap) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (cap < 0 || (cap > 0 && out == nullptr)) return fail(PS_EINVAL, "bad output buffer");
    const std::vector<int64_t> &s = ps->proto.last_staleness;
    const int count = static_cast<int>(s.size());
    for (int i = 0; i < count && i < cap; ++i) out[i] = s[i];
    return count;
}

int ps_last_applied(const ps_server *ps, int *learner_ids, int cap) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (cap < 0 || (cap > 0 && learner_ids == nullptr)) return fail(PS_EINVAL, "bad output buffer");
    const std::vector<int> &a = ps->proto.last_applied;
    const int count = static_cast<int>(a.size());
    for (int i = 0; i < count && i < cap; ++i) learner_ids[i] = a[i];
    return count;
}

int ps_run(ps_server *ps, const ps_op *ops, int count, int *done) {
    if (done) *done = 0;
    if (int rc = check(ps)) return rc;
    if (count < 0 || (count > 0 && ops == nullptr)) return fail(PS_EINVAL, "bad op script");
    PS_LOCK(ps);
    for (int i = 0; i < count; ++i) {
        const ps_op &o = ops[i];
        int rc;
        switch (o.kind) {
            case PS_OP_PUSH: rc = ps_push_dtype(ps, o.learner_id, o.grad, o.dtype); break;
            case PS_OP_APPLY: rc = ps_apply_pending(ps); break;
            case PS_OP_APPLY_SYNC: rc = ps_apply_sync(ps); break;
            case PS_OP_PULL: rc = ps_pull_many(ps, o.count, o.learner_ids, o.dsts, o.dtype); break;
            case PS_OP_APPLY_PULL: rc = ps_apply_pull(ps, o.count, o.learner_ids, o.dsts, o.dtype); break;
            default: rc = fail(PS_EINVAL, "op %d: unknown kind %d", i, o.kind);
        }
        if (rc != PS_OK) return rc;
        if (done) *done = i + 1;
    }
    return PS_OK;
}

int ps_graph_create(ps_server *ps, const ps_op *ops, int count, ps_graph **out) {
    if (out) *out = nullptr;
    if (int rc = check(ps)) return rc;
    if (out == nullptr || count < 1 || ops == nullptr) return fail(PS_EINVAL, "bad graph script");
    PS_LOCK(ps);
    if (int rc = graph_state(ps)) return rc;
    if (int rc = use_device(ps)) return rc;
    ps_graph *g = nullptr;
    try {
        g = new ps_graph;
        g->server = ps;
        g->ops.assign(ops, ops + count);
        g->ids.resize(count);
        g->dsts.resize(count);
        for (int i = 0; i < count; ++i) {
            ps_op &o = g->ops[i];
            if (o.kind == PS_OP_PULL || o.kind == PS_OP_APPLY_PULL) {
                if (o.count < 0 || o.count > PS_MAX_REPLICAS ||
                    (o.count > 0 && (o.learner_ids == nullptr || o.dsts == nullptr))) {
                    free_graph(g);
                    return fail(PS_EINVAL, "op %d: bad pull list", i);
                }
                g->ids[i].assign(o.learner_ids, o.learner_ids + o.count);
                g->dsts[i].assign(o.dsts, o.dsts + o.count);
                o.learner_ids = g->ids[i].data();
                o.dsts = g->dsts[i].data();
            }
        }
    } catch (...) {
        if (g) free_graph(g);
        return fail(PS_ENOMEM, "host allocation failed");
    }
    // Capture: the calls run as usual, their kernels go into the graph
    // instead of running, and the server's host state is put back, since
    // nothing has run yet.
    const gadei::Protocol saved = ps->proto;
    hipError_t e = hipStreamBeginCapture(ps->stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) {
        free_graph(g);
        return fail_hip(e, "hipStreamBeginCapture");
    }
    int rc = run_recorded(ps, *g, g->plan, false);
    e = hipStreamEndCapture(ps->stream, &g->graph);
    ps->proto = saved;
    if (rc == PS_OK && e != hipSuccess) rc = fail_hip(e, "hipStreamEndCapture");
    if (rc == PS_OK && g->plan.empty()) rc = fail(PS_EINVAL, "the script launches no kernel");
    if (rc == PS_OK) {
        e = hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0);
        if (e != hipSuccess) rc = fail_hip(e, "hipGraphInstantiate");
    }
    if (rc == PS_OK) {
        e = hipEventCreateWithFlags(&g->done, hipEventDisableTiming);
        if (e != hipSuccess) rc = fail_hip(e, "hipEventCreateWithFlags");
    }
    if (rc != PS_OK) {
        free_graph(g);
        return rc;
    }
    *out = g;
    return PS_OK;
}

int ps_graph_launch(ps_server *ps, ps_graph *g) {
    if (int rc = check(ps)) return rc;
    if (g == nullptr || g->server != ps) return fail(PS_EINVAL, "not a graph of this server");
    PS_LOCK(ps);
    if (int rc = graph_state(ps)) return rc;
    if (int rc = use_device(ps)) return rc;
    // The calls again, planned and committed on the host only: the replay
    // is valid if they would launch exactly the captured kernels.
    const gadei::Protocol saved = ps->proto;
    std::vector<LaunchRecord> now;
    int rc = run_recorded(ps, *g, now, true);
    if (rc == PS_OK && !same_plan(now, g->plan))
        rc = fail(PS_ESTATE, "the script would now launch other kernels than were captured");
    if (rc == PS_OK) {
        const hipError_t e = hipGraphLaunch(g->exec, ps->stream);
        if (e != hipSuccess)
            rc = fail_hip(e, "hipGraphLaunch");
        else   // the work is enqueued and committed; the event only serves destroy
            (void)hipEventRecord(g->done, ps->stream);
    }
    if (rc != PS_OK) ps->proto = saved;
    return rc;
}

void ps_graph_destroy(ps_graph *g) {
    if (g != nullptr) free_graph(g);
}

int ps_sync(ps_server *ps) {
    if (int rc = check(ps)) return rc;
    hipStream_t s, ps_s;
    bool lock_free;
    {
        // take the streams under the lock, wait without it so that pushes
        // from other threads are not held up by the wait
        PS_LOCK(ps);
        if (int rc = use_device(ps)) return rc;
        s = ps->stream;
        ps_s = ps->pull_stream;
        lock_free = ps->pull_lock_free;
    }
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
    if (lock_free) {
        e = hipStreamSynchronize(ps_s);
        if (e != hipSuccess) return fail_hip(e, "hipStreamSynchronize (pull stream)");
    }
    return PS_OK;
}

int ps_record(ps_server *ps, void *event) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (event == nullptr) return fail(PS_EINVAL, "null event");
    if (int rc = use_device(ps)) return rc;
    hipError_t e = hipEventRecord(static_cast<hipEvent_t>(event), ps->stream);
    if (e != hipSuccess) return fail_hip(e, "hipEventRecord");
    return PS_OK;
}

int ps_set_pull_stream(ps_server *ps, void *hip_stream) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (int rc = use_device(ps)) return rc;
    if (int rc = drain_pulls(ps)) return rc;
    if (hip_stream != nullptr && ps->pulls_done == nullptr) {
        hipError_t e = hipEventCreateWithFlags(&ps->pulls_done, hipEventDisableTiming);
        if (e != hipSuccess) {
            ps->pulls_done = nullptr;
            return fail_hip(e, "hipEventCreateWithFlags");
        }
    }
    ps->pull_lock_free = hip_stream != nullptr;
    ps->pull_stream = static_cast<hipStream_t>(hip_stream);
    return PS_OK;
}

int ps_get_stats(const ps_server *ps, ps_stats *out) {
    if (int rc = check(ps)) return rc;
    PS_LOCK(ps);
    if (out == nullptr) return fail(PS_EINVAL, "null stats output");
    *out = ps->proto.stats;
    out->timestamp = ps->proto.ts;
    return PS_OK;
}

}  // extern "C"
