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
struct Geometry {
    int max_blocks = 0;
};

// grad_dtype: PS_F32 | PS_BF16. pull_dtype: -1 (no replicas), PS_F32, PS_BF16.
// vec: every pointer meets the vector alignment (16 B fp32, 8 B bf16).
hipError_t launch_apply(const ApplyArgs &a, int grad_dtype, int pull_dtype, bool vec,
                        const Geometry &geo, hipStream_t s);
hipError_t launch_pull(const PullArgs &a, int pull_dtype, bool vec, const Geometry &geo,
                       hipStream_t s);
hipError_t launch_zero(float *p, uint64_t n, hipStream_t s);

}  // namespace gadei
