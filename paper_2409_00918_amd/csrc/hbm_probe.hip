// Measurement helper for the benchmark, not part of the libdisdp ABI: a
// plain device-to-device copy of known size, written the way the fused
// kernels stream memory (16-byte non-temporal loads and stores, one-wave
// blocks).  It gives the HBM bandwidth a simple copy reaches on the GPU at
// hand, and the known byte count against which rocprofv3's FETCH_SIZE /
// WRITE_SIZE counters are scaled.  Of the copies tried on MI355X (64- or
// 256-lane blocks, one or two 16-byte vectors per lane, occupancy caps of
// 8-24 waves per CU) this one was fastest: 6.70 TB/s against 6.45 with
// 256-lane blocks; every cap made it slower.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr int kBlock = 64;
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kBlock) void copy16(const f32x4 *__restrict__ src,
                                                 f32x4 *__restrict__ dst, int64_t n16)
{
    const int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    if (i < n16)
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

}  // namespace

// Copies `bytes` bytes (a multiple of 16, both pointers 16-byte aligned,
// regions not overlapping, bytes / 16 < 2^32: one lane per 16 bytes, and a
// dispatch counts its lanes in 32 bits) from src to dst on
// `stream`.  Returns 0, or -1 for bad arguments (nothing launched), or the
// HIP error code of the launch.
extern "C" int disdp_probe_copy(const void *src, void *dst, int64_t bytes, hipStream_t stream)
{
    if (!src || !dst || bytes <= 0 || (bytes & 15) ||
        (reinterpret_cast<uintptr_t>(src) & 15) || (reinterpret_cast<uintptr_t>(dst) & 15))
        return -1;
    const int64_t n16 = bytes / 16;
    const int64_t blocks = (n16 + kBlock - 1) / kBlock;
    if (blocks * kBlock > 0xffffffffLL)
        return -1;
    const uintptr_t s = reinterpret_cast<uintptr_t>(src), d = reinterpret_cast<uintptr_t>(dst);
    if (s < d + static_cast<uintptr_t>(bytes) && d < s + static_cast<uintptr_t>(bytes))
        return -1;
    const f32x4 *s16 = static_cast<const f32x4 *>(src);
    f32x4 *d16 = static_cast<f32x4 *>(dst);
    void *args[] = {&s16, &d16, const_cast<int64_t *>(&n16)};
    return static_cast<int>(hipLaunchKernel(reinterpret_cast<const void *>(&copy16),
                                            dim3(static_cast<unsigned>(blocks)), dim3(kBlock),
                                            args, 0, stream));
}
