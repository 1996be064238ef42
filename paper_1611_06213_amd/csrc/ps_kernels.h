// Internal interface between the host library (ps_server.cpp) and the HIP
// kernels (ps_kernels.hip). Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "ps.h"

namespace gadei {

// Kernel argument block of one fused apply (and optional pull fan-out).
// Passed by value, so the K gradient and R replica pointers travel in the
// kernel-argument segment and are read with scalar loads.
struct ApplyArgs {
    float *w;                 // n fp32 weights, updated in place
    float *v;                 // n fp32 velocities (momentum only)
    uint64_t n;
    float lr;
    float m;
    int k;                    // gradients to fold, 1..PS_MAX_QUEUE_DEPTH
    int r;                    // replicas to write after the update, 0..PS_MAX_REPLICAS
    int fronts_log2;          // blocks sweep 2^fronts_log2 evenly spaced fronts (front_block)
    const void *g[PS_MAX_QUEUE_DEPTH];   // oldest first
    void *dst[PS_MAX_REPLICAS];
};

struct PullArgs {
    const float *w;
    uint64_t n;
    int r;
    void *dst[PS_MAX_REPLICAS];
};

// Launch geometry: blocks are 256 threads; max_blocks caps the grid (the
// kernels then stride over the remaining chunks). 0 = one chunk per lane.
// The kernels may reserve LDS (they use none) so that only a few blocks fit
// per compute unit: lds_for_blocks[b] leaves room for exactly b blocks
// (b = 1..4; 0 = no such reservation on this device; chosen at server
// creation). Every apply and synchronous step is told its shape
// (apply_shape, sync_shape; ps_layout.h).
struct Geometry {
    int max_blocks = 0;
    int fronts_log2 = -1;   // -1: chosen per apply (fronts_log2_for, ps_layout.h)
    unsigned lds_for_blocks[5] = {0, 0, 0, 0, 0};
};

// How one apply launch runs: resident blocks per compute unit (1..4; 0 = as
// many as fit) and gradients per load group (4, 8, 12, 16, 24 or 32; others
// = 16; the synchronous step takes 4, 8, 12 or 16, others = 16).
struct Shape {
    int blocks_per_cu = 0;
    int group = 16;
};

// LDS bytes that leave room for exactly `blocks` (1..4) blocks per compute
// unit on the current device, or 0 if the device does not allow such a
// reservation.
unsigned blocks_per_cu_lds(int blocks);

// grad_dtype: PS_F32 | PS_BF16. pull_dtype: -1 (no replicas), PS_F32, PS_BF16.
// level: 2 = every buffer 16-byte aligned; 1 = fp32 buffers 16-byte and bf16
// buffers 8-byte aligned; 0 = anything else (scalar kernels).
// shape: residency and group size of the vector kernels (the scalar kernel
// for misaligned buffers ignores it).
hipError_t launch_apply(const ApplyArgs &a, int grad_dtype, int pull_dtype, int level,
                        const Shape &shape, const Geometry &geo, hipStream_t s);
hipError_t launch_pull(const PullArgs &a, int pull_dtype, int level, const Geometry &geo,
                       hipStream_t s);
// Synchronous step over a.k gradients of one dtype (no replicas).
hipError_t launch_sync(const ApplyArgs &a, int grad_dtype, int level, const Shape &shape,
                       const Geometry &geo, hipStream_t s);
hipError_t launch_zero(float *p, uint64_t n, hipStream_t s);

}  // namespace gadei
