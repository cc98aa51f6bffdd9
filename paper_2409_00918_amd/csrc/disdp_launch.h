// Internal interface between the C-ABI front end (disdp_api.cpp) and the
// gfx950 kernels (disdp_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime_api.h>

namespace disdp {

constexpr int kMaxW = 64;

enum GradType { kGradF32 = 0, kGradBF16 = 1, kGradI32 = 2 };
enum AggMode { kAggFP32 = 0, kAggFixed = 1 };
enum Kind { kAggregateOnly = 0, kAggregateAdam = 1 };

// Per-step constants of the optimizer, evaluated once on the host.
struct StepScalars {
    float b1, omb1;   // beta1, 1 - beta1
    float b2, omb2;   // beta2, 1 - beta2
    float bc1, bc2;   // 1 - beta1^t, 1 - beta2^t
    float decay;      // 1 - lr * weight_decay
    float lr, eps, grad_scale;
};

// Everything a kernel needs, passed by value in the kernel-argument segment.
struct LaunchArgs {
    const void *g[kMaxW];  // W contribution pointers (device)
    float *p, *m, *v;      // in-place state (device), NULL in aggregate-only
    uint16_t *p16;         // bf16 parameter copy, may be NULL
    float *agg_f32;        // optional fp32 aggregate
    int32_t *agg_i32;      // optional int32 aggregate (fixed mode)
    int64_t n;             // elements from the pointers on
    int head;              // 0-255 elements just before the pointers, done one
                           // by one (the pointers advanced past them)
    int W, gdtype, mode, frac_bits;
    float qscale, dqscale; // 2^k and 2^-k (fixed mode)
    StepScalars s;
    const StepScalars *s_dev;  // when set, the step constants are read here
                               // when the kernel runs, and `s` is unused
};

// Enqueues the kernel for `a` on `stream`.  `vector_path` selects the
// 4-elements-per-lane kernels (every pointer, after the head, on a 4-byte
// boundary).
hipError_t launch(const LaunchArgs &a, Kind kind, bool vector_path,
                  hipStream_t stream);

// Several tensors of one optimizer step in one launch: virtual block b of
// the launch belongs to the last tensor j with tile_start[j] <= b, and is
// tile b - tile_start[j] of it (256 elements).  The struct travels in the
// kernel-argument segment and stays under 4 KiB.
constexpr int kMultiMaxTensors = 48;
constexpr int kMultiMaxPtrs = 320;
constexpr int kMultiTileGroups = 64;  // 4-element groups per virtual block
struct MultiArgs {
    int count;                                  // tensors in this launch (>= 1)
    int W, gdtype, mode, frac_bits;
    float qscale, dqscale;                      // 2^k and 2^-k (fixed mode)
    StepScalars s;
    const StepScalars *s_dev;                   // as in LaunchArgs
    int64_t tile_start[kMultiMaxTensors + 1];   // [count] = blocks in all
    int64_t n[kMultiMaxTensors];                // elements from the pointers on
    int head[kMultiMaxTensors];                 // 0-255 elements before them
    void *ptr[kMultiMaxPtrs];                   // tensor j at j * (W + 4): the W
                                                // contributions, p, m, v, bf16
                                                // copy (may be NULL)
};
static_assert(sizeof(MultiArgs) <= 4096, "kernel arguments above 4 KiB");
hipError_t launch_multi(const MultiArgs &a, hipStream_t stream);

// The float-to-int32 format conversion of one buffer.
struct QuantizeArgs {
    const void *g;     // n elements of gdtype (kGradF32 or kGradBF16)
    int32_t *out;      // n int32
    int64_t n;
    int head;          // as in LaunchArgs
    int gdtype;
    float qscale;      // 2^k
};
hipError_t launch_quantize(const QuantizeArgs &q, bool vector_path, hipStream_t stream);

}  // namespace disdp
