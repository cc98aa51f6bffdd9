// gfx950 kernels of libdisdp: the W-way reduction of a shard's gradient
// contributions (the SmartSwitch's aggregation in DisDP, Sections III-A and
// III-C, in fp32 or in the integer format of Section III-B), optionally
// fused with the parameter server's mixed-precision Adam step and its bf16
// parameter copy (Section III-D, step 5).
//
// The path is a pure HBM stream: per element it reads W contributions and
// 12 bytes of state and writes 12 bytes of state and 2 bytes of copy, with
// a few dozen ALU operations in between.  No MFMA: there is no contraction.
// Design for CDNA4:
//   * one lane owns 4 consecutive elements, so every stream moves in 16-byte
//     (fp32) or 8-byte (bf16) vector accesses and each wave instruction
//     covers 1 KiB / 512 B of contiguous memory;
//   * a block owns a tile of one group per lane; all loads of a lane (W
//     contributions and p, m, v) are issued before any arithmetic, so each
//     lane keeps W + 3 vector loads in flight;
//   * one tile per block over a grid that covers the shard, so every byte is
//     read once and written once;
//   * data are touched once, so loads and stores carry the non-temporal hint;
//   * no atomics, no cross-lane traffic: each element's reduction is one
//     lane's serial chain in worker order, which makes results independent
//     of grid size and identical to an element-wise evaluation.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <cstring>

#include "disdp_launch.h"

// One rounding per written operation: never contract a*b+c into an FMA.
#pragma clang fp contract(off)

// Launch shapes.  The default ("solo") shape -- one-wave (64-lane) blocks
// each owning one tile of 64 four-element groups, non-temporal loads and
// stores, tiles in natural order -- was the best or tied-best in
// interleaved A/B runs on MI355X over the 7B/8, 13B/16 and 175B/64 shards;
// the alternatives measured were within 2% or slower (persistent grids, more
// groups per lane, 128- to 1024-lane blocks, wave-contiguous groups,
// XCD-chunked tile orders, hints on one side only).  One-wave blocks beat
// 256-lane blocks at the same resident waves by 2-6%: a retiring wave frees
// its slot at once instead of waiting for the slowest wave of its block.
// The "shared" shape (four-wave blocks, one occupancy cap per mode) is for
// a GPU whose compute kernels run on other streams at the same time: a
// retiring four-wave block leaves a hole a compute workgroup can take, so
// the chip is shared more evenly (see launch_shape below).
#define DISDP_LAUNCH_BOUNDS __launch_bounds__(256)
#define DISDP_WAVE_LAUNCH_BOUNDS __launch_bounds__(64)

namespace disdp {
namespace {

constexpr int kWave = 64;
constexpr int kMaxBlock = 256;   // lanes per block of the shared shape
// lanes per block of the many-tensor and quantize kernels (one wave)
constexpr int kWaveBlock = kWave;

// Vector types of the 4-element groups, declared only 4-byte aligned: a
// group of an array that starts off its natural vector boundary (arrays with
// unrelated misalignments) is one 16- or 8-byte access at a 4-byte-aligned
// address, which the global memory instructions take as they are (for
// naturally aligned groups the machine code is the same).
typedef float f32x4 __attribute__((ext_vector_type(4), aligned(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2), aligned(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4), aligned(4)));

// Non-temporal group loads and stores (every byte is touched once).
// Overloads, not a template: deducing the vector type would drop the
// typedef's 4-byte alignment.
#define DISDP_NT_ACCESS(T)                                                              \
    __device__ __forceinline__ T ld_nt(const T *p) { return __builtin_nontemporal_load(p); } \
    __device__ __forceinline__ void st_nt(T *p, T v) { __builtin_nontemporal_store(v, p); }
DISDP_NT_ACCESS(f32x4)
DISDP_NT_ACCESS(u32x2)
DISDP_NT_ACCESS(i32x4)
#undef DISDP_NT_ACCESS

// ---- element operations ---------------------------------------------------

// bf16 bits -> fp32: the bf16 pattern is the upper half of the fp32 one.
__device__ __forceinline__ float widen_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float widen_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even; NaN -> quiet NaN with its sign.
__device__ __forceinline__ uint32_t to_bf16(float x)
{
    const uint32_t u = __float_as_uint(x);
    const uint32_t rounded = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    const uint32_t qnan = ((u >> 16) & 0x8000u) | 0x7fc0u;
    return (u & 0x7fffffffu) > 0x7f800000u ? qnan : rounded;
}

// Contribution -> int32 at scale 2^k: exact scaling, rint (ties to even),
// saturation, NaN -> 0 (the integer switch format, Section III-B), in three
// instructions and no branches.
__device__ __forceinline__ int32_t quantize(float x, float scale)
{
    const float r = __builtin_rintf(x * scale);
    // The hardware conversion already has the format's saturation: a float
    // at or above 2^31 (+inf included) gives INT32_MAX, one below -2^31
    // (-inf included) INT32_MIN, NaN 0, anything else its (integral) value.
    // A C++ cast leaves those cases undefined, hence the instruction itself.
    int32_t q;
    asm("v_cvt_i32_f32 %0, %1" : "=v"(q) : "v"(r));
    return q;
}

__device__ __forceinline__ int32_t saturate32(int64_t s)
{
    const int64_t hi = s > INT32_MAX ? int64_t(INT32_MAX) : s;
    return static_cast<int32_t>(hi < INT32_MIN ? int64_t(INT32_MIN) : hi);
}

// The step constants of a launch: by value in the arguments, or read from
// memory when the kernel runs (one uniform load per wave, scalar cache).
template <class A>
__device__ __forceinline__ StepScalars step_scalars_of(const A &a)
{
    return a.s_dev ? *a.s_dev : a.s;
}

// One AdamW step on one element (decoupled decay, bias-corrected moments,
// eps outside the square root).  `/` and sqrtf are the correctly rounded
// IEEE operations on this target.
__device__ __forceinline__ void adamw(const StepScalars &s, float agg, float &p, float &m,
                                      float &v)
{
    const float g = agg * s.grad_scale;
    const float mi = s.b1 * m + s.omb1 * g;
    const float vi = s.b2 * v + s.omb2 * (g * g);
    const float mh = mi / s.bc1;
    const float vh = vi / s.bc2;
    const float d = sqrtf(vh) + s.eps;
    p = p * s.decay - s.lr * (mh / d);
    m = mi;
    v = vi;
}

// ---- loading contributions -----------------------------------------------

// What one element of a contribution holds once loaded: a float (fp32 or
// widened bf16), or an int32 already in the switch's integer format.
template <int GT>
struct Contrib {
    using type = float;
};
template <>
struct Contrib<kGradI32> {
    using type = int32_t;
};

// Four consecutive elements of contribution `base` at group index `grp`.
template <int GT>
__device__ __forceinline__ void load_group(const void *base, int64_t grp,
                                           typename Contrib<GT>::type (&x)[4])
{
    if constexpr (GT == kGradI32) {
        const i32x4 v = ld_nt(reinterpret_cast<const i32x4 *>(base) + grp);
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else if constexpr (GT == kGradF32) {
        const f32x4 v = ld_nt(reinterpret_cast<const f32x4 *>(base) + grp);
        x[0] = v.x;
        x[1] = v.y;
        x[2] = v.z;
        x[3] = v.w;
    } else {
        const u32x2 h = ld_nt(reinterpret_cast<const u32x2 *>(base) + grp);
        x[0] = widen_lo(h.x);
        x[1] = widen_hi(h.x);
        x[2] = widen_lo(h.y);
        x[3] = widen_hi(h.y);
    }
}

template <int GT>
__device__ __forceinline__ typename Contrib<GT>::type load_one(const void *base, int64_t i)
{
    if constexpr (GT == kGradI32)
        return reinterpret_cast<const int32_t *>(base)[i];
    else if constexpr (GT == kGradF32)
        return reinterpret_cast<const float *>(base)[i];
    else
        return widen_lo(reinterpret_cast<const uint16_t *>(base)[i]);
}

// ---- the reduction of one element over its W contributions ----------------

// Accumulator of one element: fp32 running sum, or exact 64-bit integer sum.
template <int MODE>
struct Acc {
    float f;
    int64_t s;
    __device__ __forceinline__ void first(float x, float qscale)
    {
        if constexpr (MODE == kAggFP32)
            f = x;
        else
            s = quantize(x, qscale);
    }
    __device__ __forceinline__ void next(float x, float qscale)
    {
        if constexpr (MODE == kAggFP32)
            f = f + x;
        else
            s += quantize(x, qscale);
    }
    // contributions already in the integer format (fixed mode only)
    __device__ __forceinline__ void first(int32_t q, float)
    {
        static_assert(MODE == kAggFixed, "int32 contributions are summed as integers");
        s = q;
    }
    __device__ __forceinline__ void next(int32_t q, float)
    {
        static_assert(MODE == kAggFixed, "int32 contributions are summed as integers");
        s += q;
    }
    // (fp32 aggregate, int32 aggregate)
    __device__ __forceinline__ float result(float dqscale, int32_t &ai) const
    {
        if constexpr (MODE == kAggFP32) {
            ai = 0;
            return f;
        } else {
            ai = saturate32(s);
            return static_cast<float>(ai) * dqscale;
        }
    }
};

// ---- writing one group's results -----------------------------------------

template <int MODE, bool ADAM, class A>
__device__ __forceinline__ void finish_group(const A &a, int64_t grp, const float (&agg)[4],
                                             const int32_t (&ai)[4], f32x4 P, f32x4 M, f32x4 V)
{
    if (a.agg_f32)
        st_nt(reinterpret_cast<f32x4 *>(a.agg_f32) + grp, f32x4{agg[0], agg[1], agg[2], agg[3]});
    if constexpr (MODE == kAggFixed) {
        if (a.agg_i32)
            st_nt(reinterpret_cast<i32x4 *>(a.agg_i32) + grp, i32x4{ai[0], ai[1], ai[2], ai[3]});
    }
    if constexpr (ADAM) {
        float p[4] = {P.x, P.y, P.z, P.w};
        float m[4] = {M.x, M.y, M.z, M.w};
        float v[4] = {V.x, V.y, V.z, V.w};
        const StepScalars sc = step_scalars_of(a);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            adamw(sc, agg[e], p[e], m[e], v[e]);
        st_nt(reinterpret_cast<f32x4 *>(a.p) + grp, f32x4{p[0], p[1], p[2], p[3]});
        st_nt(reinterpret_cast<f32x4 *>(a.m) + grp, f32x4{m[0], m[1], m[2], m[3]});
        st_nt(reinterpret_cast<f32x4 *>(a.v) + grp, f32x4{v[0], v[1], v[2], v[3]});
        if (a.p16)
            st_nt(reinterpret_cast<u32x2 *>(a.p16) + grp,
                  u32x2{to_bf16(p[0]) | (to_bf16(p[1]) << 16),
                        to_bf16(p[2]) | (to_bf16(p[3]) << 16)});
    }
}

// ---- one group per lane, W known at compile time --------------------------

// Group `grp`: every load first, then the arithmetic, then the stores.
template <int W, int GT, int MODE, bool ADAM, class A>
__device__ __forceinline__ void process_group(const A &a, int64_t grp)
{
    typename Contrib<GT>::type c[W][4];
    f32x4 P{}, M{}, V{};
#pragma unroll
    for (int w = 0; w < W; ++w)
        load_group<GT>(a.g[w], grp, c[w]);
    if constexpr (ADAM) {
        P = ld_nt(reinterpret_cast<const f32x4 *>(a.p) + grp);
        M = ld_nt(reinterpret_cast<const f32x4 *>(a.m) + grp);
        V = ld_nt(reinterpret_cast<const f32x4 *>(a.v) + grp);
    }
    float agg[4];
    int32_t ai[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        Acc<MODE> acc;
        acc.first(c[0][e], a.qscale);
#pragma unroll
        for (int w = 1; w < W; ++w)
            acc.next(c[w][e], a.qscale);
        agg[e] = acc.result(a.dqscale, ai[e]);
    }
    finish_group<MODE, ADAM>(a, grp, agg, ai, P, M, V);
}

// ---- one group per lane, W known only at run time (W <= 64) ---------------

// K contributions w0 .. w0+K-1 into the accumulators: all K loads issued,
// then the additions in worker order.  No branch separates the loads, so
// none waits for the one before (a conditional load per contribution made
// the compiler wait after each).  `first`: w0 is contribution 0.
template <int K, int GT, int MODE, class A>
__device__ __forceinline__ void accumulate_piece(const A &a, int64_t grp, int w0,
                                                 bool first, Acc<MODE> (&acc)[4])
{
    typename Contrib<GT>::type c[K][4];
#pragma unroll
    for (int j = 0; j < K; ++j)
        load_group<GT>(a.g[w0 + j], grp, c[j]);
#pragma unroll
    for (int j = 0; j < K; ++j) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (j == 0 && first)
                acc[e].first(c[j][e], a.qscale);
            else
                acc[e].next(c[j][e], a.qscale);
        }
    }
}

// Contributions in chunks of 128 bytes per lane (8 fp32 or int32, 16 bf16),
// then the remaining W mod chunk in pieces of 8, 4, 2 and 1.
template <int GT, int MODE, bool ADAM, class A>
__device__ __forceinline__ void process_group_rt(const A &a, int64_t grp)
{
    constexpr int kChunk = GT == kGradBF16 ? 16 : 8;
    f32x4 P{}, M{}, V{};
    if constexpr (ADAM) {
        P = ld_nt(reinterpret_cast<const f32x4 *>(a.p) + grp);
        M = ld_nt(reinterpret_cast<const f32x4 *>(a.m) + grp);
        V = ld_nt(reinterpret_cast<const f32x4 *>(a.v) + grp);
    }
    Acc<MODE> acc[4];
    int w0 = 0;
    for (; w0 + kChunk <= a.W; w0 += kChunk)
        accumulate_piece<kChunk, GT, MODE>(a, grp, w0, w0 == 0, acc);
    const int rest = a.W - w0;
    if constexpr (kChunk > 8) {
        if (rest & 8) {
            accumulate_piece<8, GT, MODE>(a, grp, w0, w0 == 0, acc);
            w0 += 8;
        }
    }
    if (rest & 4) {
        accumulate_piece<4, GT, MODE>(a, grp, w0, w0 == 0, acc);
        w0 += 4;
    }
    if (rest & 2) {
        accumulate_piece<2, GT, MODE>(a, grp, w0, w0 == 0, acc);
        w0 += 2;
    }
    if (rest & 1)
        accumulate_piece<1, GT, MODE>(a, grp, w0, w0 == 0, acc);
    float agg[4];
    int32_t ai[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        agg[e] = acc[e].result(a.dqscale, ai[e]);
    finish_group<MODE, ADAM>(a, grp, agg, ai, P, M, V);
}

// ---- one element -----------------------------------------------------------

template <int GT, int MODE, bool ADAM, class A>
__device__ __forceinline__ void process_element(const A &a, int64_t i)
{
    Acc<MODE> acc;
    acc.first(load_one<GT>(a.g[0], i), a.qscale);
    for (int w = 1; w < a.W; ++w)
        acc.next(load_one<GT>(a.g[w], i), a.qscale);
    int32_t ai;
    const float agg = acc.result(a.dqscale, ai);
    if (a.agg_f32)
        a.agg_f32[i] = agg;
    if constexpr (MODE == kAggFixed) {
        if (a.agg_i32)
            a.agg_i32[i] = ai;
    }
    if constexpr (ADAM) {
        float p = a.p[i], m = a.m[i], v = a.v[i];
        adamw(step_scalars_of(a), agg, p, m, v);
        a.p[i] = p;
        a.m[i] = m;
        a.v[i] = v;
        if (a.p16)
            a.p16[i] = static_cast<uint16_t>(to_bf16(p));
    }
}

// ---- kernels -----------------------------------------------------------------

// Vector kernel.  W > 0: compile-time worker count; W == 0: run-time worker
// count.  One 4-element group per lane, grid-stride over the groups [0,
// n/4) (one pass when the grid covers the shard; a grid clamped to what one
// dispatch counts walks on); the last n % 4 elements and the a.head
// elements before the (advanced) pointers go to lanes of block 0.  Every
// pointer is on a 4-byte boundary; the front end chose the head.  Block
// size is the launch's (64 or 256 lanes).
template <int W, int GT, int MODE, bool ADAM>
__global__ DISDP_LAUNCH_BOUNDS void vector_kernel(LaunchArgs a)
{
    const int64_t n_groups = a.n >> 2;
    const int lanes = blockDim.x;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * lanes;
    for (int64_t grp = static_cast<int64_t>(blockIdx.x) * lanes + threadIdx.x; grp < n_groups;
         grp += stride) {
        if constexpr (W > 0)
            process_group<W, GT, MODE, ADAM>(a, grp);
        else
            process_group_rt<GT, MODE, ADAM>(a, grp);
    }
    if (blockIdx.x == 0 && threadIdx.x < (a.n & 3))
        process_element<GT, MODE, ADAM>(a, (n_groups << 2) + threadIdx.x);
    // the elements before the advanced pointers
    if (blockIdx.x == 0)
        for (int j = threadIdx.x; j < a.head; j += lanes)
            process_element<GT, MODE, ADAM>(a, static_cast<int64_t>(j) - a.head);
}

// Element-wise kernel, for an array not aligned to its element size or bf16
// arrays that no head puts on 4-byte boundaries together.
template <int GT, int MODE, bool ADAM>
__global__ DISDP_LAUNCH_BOUNDS void element_kernel(LaunchArgs a)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < a.n;
         i += stride)
        process_element<GT, MODE, ADAM>(a, i);
}

// ---- several tensors in one launch ------------------------------------------

// Tensor j of a multi-tensor launch, with the members the group helpers
// read from LaunchArgs (the contribution pointers stay in the argument
// segment).
struct TensorView {
    const void *const *g;
    float *p, *m, *v;
    uint16_t *p16;
    float *agg_f32;
    int32_t *agg_i32;
    float qscale, dqscale;
    StepScalars s;
    const StepScalars *s_dev;
    int W;
};

// Fused aggregation + AdamW over the tensors of `ma`, one 256-element tile
// per virtual block, grid-stride over the virtual blocks.  Per tensor as in
// vector_kernel: whole groups one per lane, the last n % 4 elements by the
// tensor's last tile, its head elements by its first tile.
template <int W, int GT, int MODE>
__global__ DISDP_WAVE_LAUNCH_BOUNDS void multi_kernel(MultiArgs ma)
{
    const int64_t total = ma.tile_start[ma.count];
    const int per_tensor = ma.W + 4;
    for (int64_t vb = blockIdx.x; vb < total; vb += gridDim.x) {
        int lo = 0, hi = ma.count - 1;   // the last j with tile_start[j] <= vb
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (ma.tile_start[mid] <= vb)
                lo = mid;
            else
                hi = mid - 1;
        }
        const int j = lo;
        void *const *tp = ma.ptr + j * per_tensor;
        TensorView t;
        t.g = const_cast<const void *const *>(tp);
        t.p = static_cast<float *>(tp[ma.W]);
        t.m = static_cast<float *>(tp[ma.W + 1]);
        t.v = static_cast<float *>(tp[ma.W + 2]);
        t.p16 = static_cast<uint16_t *>(tp[ma.W + 3]);
        t.agg_f32 = nullptr;
        t.agg_i32 = nullptr;
        t.qscale = ma.qscale;
        t.dqscale = ma.dqscale;
        t.s = ma.s;
        t.s_dev = ma.s_dev;
        t.W = ma.W;
        const int64_t n = ma.n[j];
        const int64_t n_groups = n >> 2;
        const int64_t tile = vb - ma.tile_start[j];
        for (int l = threadIdx.x; l < kMultiTileGroups; l += kWaveBlock) {
            const int64_t grp = tile * kMultiTileGroups + l;
            if (grp < n_groups) {
                if constexpr (W > 0)
                    process_group<W, GT, MODE, true>(t, grp);
                else
                    process_group_rt<GT, MODE, true>(t, grp);
            }
        }
        if (vb == ma.tile_start[j + 1] - 1 && threadIdx.x < (n & 3))
            process_element<GT, MODE, true>(t, (n_groups << 2) + threadIdx.x);
        if (tile == 0)
            for (int e = threadIdx.x; e < ma.head[j]; e += kWaveBlock)
                process_element<GT, MODE, true>(t, static_cast<int64_t>(e) - ma.head[j]);
    }
}

// ---- the format conversion as a producer ------------------------------------

// out = quantize(g) over 4-element groups (one group per lane, grid-stride
// over kWaveBlock-lane blocks), the last n % 4 and the head elements by
// block 0.
template <int GT>
__global__ DISDP_WAVE_LAUNCH_BOUNDS void quantize_vector_kernel(QuantizeArgs q)
{
    const int64_t n_groups = q.n >> 2;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kWaveBlock;
    for (int64_t grp = static_cast<int64_t>(blockIdx.x) * kWaveBlock + threadIdx.x; grp < n_groups;
         grp += stride) {
        float x[4];
        load_group<GT>(q.g, grp, x);
        st_nt(reinterpret_cast<i32x4 *>(q.out) + grp,
              i32x4{quantize(x[0], q.qscale), quantize(x[1], q.qscale),
                    quantize(x[2], q.qscale), quantize(x[3], q.qscale)});
    }
    if (blockIdx.x == 0 && threadIdx.x < (q.n & 3)) {
        const int64_t i = (n_groups << 2) + threadIdx.x;
        q.out[i] = quantize(load_one<GT>(q.g, i), q.qscale);
    }
    if (blockIdx.x == 0)
        for (int j = threadIdx.x; j < q.head; j += kWaveBlock) {
            const int64_t i = static_cast<int64_t>(j) - q.head;
            q.out[i] = quantize(load_one<GT>(q.g, i), q.qscale);
        }
}

template <int GT>
__global__ DISDP_WAVE_LAUNCH_BOUNDS void quantize_element_kernel(QuantizeArgs q)
{
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kWaveBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kWaveBlock + threadIdx.x; i < q.n; i += stride)
        q.out[i] = quantize(load_one<GT>(q.g, i), q.qscale);
}

// ---- host side: grid sizing and dispatch --------------------------------------

// Resident waves per CU for a fixed-point kernel converting float
// contributions, by the bytes of loads a lane keeps in flight, as in fp32
// mode; a lane converting bf16 contributions (twice the conversions per
// byte) holds its loads for a smaller share of the time and wants more
// waves.  Interleaved A/B of the fused call at n = 4e8 over caps of 6-14
// (TB/s at the chosen cap, the next best in brackets): fp32 W = 1, 2
// (64, 80 B) 14: 6.48, 6.49 (12: 6.28, 6.41); W = 4 (112 B) 12: 6.61;
// W = 8 (176 B) 8: 6.59 (10: 6.49); W = 12, 24 (240, 432 B) 6: 6.44, 6.04
// (8: 6.24, 6.01); bf16 W = 4 (80 B) 14: 6.43 (12: 6.28); W = 8 (112 B)
// 12: 6.38 (14: 6.34); W = 16, 32 (176, 304 B) 10: 6.19, 6.00 (8: 6.16,
// 5.93).  Int32 contributions need no conversion and take the fp32-mode
// caps.
constexpr int fixed_mode_waves(int lane_bytes, bool bf16)
{
    return lane_bytes <= 80 ? 14 : lane_bytes <= 112 ? 12 : bf16 ? 10 : lane_bytes <= 176 ? 8 : 6;
}

// Resident waves per CU in fp32 mode (and for int32 contributions), by the
// bytes of loads a lane keeps in flight: fewer bytes per wave need more
// waves to keep enough requests in flight, more bytes fewer.  Interleaved
// A/B of the fused call at n = 4e8 over caps of 6-16: 12 waves for lanes up
// to 112 B (fp32 W <= 4, bf16 W <= 8, the optimizer step alone), 8 up to
// 176 B (fp32 W = 5-8, bf16 W = 12, 16), 6 beyond (fp32 W = 12, 16).
constexpr int fp32_mode_waves(int lane_bytes)
{
    return lane_bytes <= 112 ? 12 : lane_bytes <= 176 ? 8 : 6;
}

// The same for the run-time worker-count kernel, from the actual W: whole
// chunks keep 128 B per lane in flight (8 waves suffice), a remainder adds
// round trips with fewer bytes (10), and W below one chunk is all such
// pieces (14).  Measured for fp32 W = 9, 24, 64 and bf16 W = 13, 32, 64.
// Converting bf16 in fixed mode wants two more waves.  Fixed mode at
// n = 4e8 over caps of 6-14 (TB/s at the chosen cap, the next best in
// brackets): fp32 W = 9, 13 10: 6.55, 6.47 (12: 6.51; 8: 6.44); bf16
// W = 17, 40 12: 6.35, 6.17 (14: 6.24, 6.06); W = 32 10: 6.05 (12: 5.97).
// Four-byte contributions (fp32 or int32) over two or more chunks keep
// more round trips in flight per wave and want fewer waves: interleaved
// at n = 2e8 over caps of 5-12, fp32 mode W = 17-32 6 waves (+0.4% to
// +2.9% against 8-10), W = 40-64 5 waves (+3.0% to +4.8%); fixed mode
// converting fp32, W = 17 7 waves (+1.6%), W = 20-64 6 waves (+0.2% to
// +2.0%).  bf16 contributions were within about 1% of the best at the
// rules above.
int runtime_w_waves(int W, int gt, int mode)
{
    const bool bf16 = gt == kGradBF16;
    const int chunk = bf16 ? 16 : 8;
    if (mode == kAggFixed && gt != kGradI32) {
        if (!bf16 && W >= 2 * chunk)
            return W < 20 ? 7 : 6;
        return (W % chunk ? 10 : 8) + (bf16 ? 2 : 0);
    }
    if (!bf16 && W >= 2 * chunk)
        return W <= 32 ? 6 : 5;
    return W < chunk ? 14 : W % chunk ? 10 : 8;
}

// The launch shape of the vector kernels for one call.
//   solo   (default): one-wave blocks, occupancy caps from the tables above
//          -- the fastest shape when the kernel has the GPU to itself.
//   shared (DISDP_LAUNCH_SHAPE=shared in the environment): four-wave blocks
//          capped at 12 waves per CU, 20 for fixed-point kernels that
//          convert float contributions.  Next to a bf16 GEMM loop on
//          another stream of the same (unmasked) GPU, the solo shape's
//          stream of one-wave blocks refills every slot a retiring block
//          frees and the GEMM slows about 10x while the fused call slows
//          1.1x; a retiring four-wave block leaves a hole of four wave slots
//          that a GEMM workgroup can take, and the two slow each other about
//          evenly (measured 1.7x and 2.0x), at 3-5% below the solo shape's
//          rate when alone.
// The variable is read on every call, so a process can switch between
// calls; any other value means solo.
struct Shape {
    int lanes;        // lanes per block
    bool shared;
};

Shape launch_shape()
{
    const char *s = std::getenv("DISDP_LAUNCH_SHAPE");
    if (s && std::strcmp(s, "shared") == 0)
        return Shape{kMaxBlock, true};
    return Shape{kWave, false};
}

constexpr int kSharedWaves = 12;
constexpr int kSharedWavesConverting = 20;

// Dynamic LDS bytes a vector-kernel block reserves so that at most
// `blocks_per_cu` blocks fit on a CU (0 = no cap), cached per device.
int occupancy_lds_bytes(int blocks_per_cu)
{
    constexpr int kMaxCap = 64;
    if (blocks_per_cu <= 0 || blocks_per_cu > kMaxCap)
        return 0;
    static std::atomic<int> cached[64][kMaxCap + 1];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 0;
    int b = cached[dev][blocks_per_cu].load(std::memory_order_relaxed);
    if (b == 0) {
        int per_cu = 0, per_block = 0;
        if (hipDeviceGetAttribute(&per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
                                  dev) != hipSuccess ||
            hipDeviceGetAttribute(&per_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
                hipSuccess ||
            per_cu <= 0) {
            b = -1;  // unknown: launch without a cap
        } else {
            b = (per_cu / blocks_per_cu) & ~1023;
            if (b > per_block)
                b = per_block;
            if (b <= 0)
                b = -1;
        }
        cached[dev][blocks_per_cu].store(b, std::memory_order_relaxed);
    }
    return b > 0 ? b : 0;
}

int cu_count()
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 256;
    int c = cached[dev].load(std::memory_order_relaxed);
    if (c <= 0) {
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            c <= 0)
            c = 256;
        cached[dev].store(c, std::memory_order_relaxed);
    }
    return c;
}

// CUs `stream` may run on: the number of bits of its CU mask among the
// device's CUs (hipExtStreamCreateWithCUMask), or all of them when the
// runtime cannot say.  An error the query records is cleared only when no
// error was pending before it, so a caller's own pending error survives.
int stream_cus(hipStream_t stream)
{
    const int total = cu_count();
    constexpr int kMaxWords = 32;  // masks of up to 1024 CUs
    const int words = (total + 31) / 32;
    uint32_t mask[kMaxWords] = {};
    if (words > kMaxWords)
        return total;
    const hipError_t pending = hipPeekAtLastError();
    if (hipExtStreamGetCUMask(stream, words, mask) != hipSuccess) {
        if (pending == hipSuccess)
            (void)hipGetLastError();
        return total;
    }
    int c = 0;
    for (int i = 0; i < total; ++i)
        c += (mask[i / 32] >> (i % 32)) & 1u;
    return c > 0 ? c : total;
}

// Resident-block cap per CU for a launch of `lanes`-lane blocks on
// `stream`: `base_waves` is the cap in waves for the whole chip.  What
// streams best is a number of resident waves chip-wide, so on a stream
// restricted to fewer CUs each CU takes proportionally more, up to
// kMaxScaledWaves (the register limit of the W = 8 kernels).  Measured on
// the 7B/8 shard with 32 / 64 / 128 CUs: 20 waves per CU streamed 41% / 35%
// / 19% faster than the full-chip cap of the time (12 waves per CU, in
// 4-wave blocks).
constexpr int kMaxScaledWaves = 20;
int blocks_per_cu_cap(int base_waves, int lanes, hipStream_t stream)
{
    if (base_waves <= 0)
        return 0;
    const int total = cu_count();
    const int mine = stream_cus(stream);
    int waves = base_waves;
    if (mine < total) {
        const int scaled = (base_waves * total + mine - 1) / mine;
        waves = scaled < kMaxScaledWaves ? scaled
                                         : (base_waves > kMaxScaledWaves ? base_waves : kMaxScaledWaves);
    }
    const int blocks = waves / (lanes / kWave);
    return blocks > 0 ? blocks : 1;
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// A dispatch counts its work-items in 32 bits per dimension, so a grid of
// `block`-lane blocks holds at most (2^32 - 1) / block of them.  Every
// kernel here walks its work grid-stride, so a clamped grid still covers a
// shard of any accepted size.
constexpr int64_t kMaxGridLanes = 0xffffffffLL;
int64_t clamp_grid(int64_t blocks, int block)
{
    const int64_t max_blocks = kMaxGridLanes / block;
    return blocks < 1 ? 1 : blocks > max_blocks ? max_blocks : blocks;
}

// `blocks` blocks of `lanes` lanes (clamped), `lds_bytes` of dynamic LDS
// reserved per block (an occupancy cap).
hipError_t launch_kernel(const void *fn, int64_t blocks, int lanes, const LaunchArgs &a,
                         hipStream_t stream, int lds_bytes = 0)
{
    blocks = clamp_grid(blocks, lanes);
    void *args[] = {const_cast<LaunchArgs *>(&a)};
    return hipLaunchKernel(fn, dim3(static_cast<unsigned>(blocks)), dim3(lanes), args,
                           static_cast<size_t>(lds_bytes), stream);
}

template <int W, int GT, int MODE, bool ADAM>
hipError_t launch_vector(const LaunchArgs &a, Shape shape, hipStream_t stream)
{
    const int64_t blocks = ceil_div(a.n >> 2, shape.lanes);
    // bytes of loads one lane keeps in flight: 4 elements of each
    // contribution, plus p, m and v with the optimizer (run-time W: many)
    constexpr int kGradBytes = GT == kGradBF16 ? 2 : 4;
    constexpr int kLaneBytes = W > 0 ? 4 * (W * kGradBytes + (ADAM ? 12 : 0)) : 1 << 30;
    constexpr bool kConverts = MODE == kAggFixed && GT != kGradI32;
    int base;
    if (shape.shared)
        base = kConverts ? kSharedWavesConverting : kSharedWaves;
    else
        base = W == 0      ? runtime_w_waves(a.W, GT, MODE)
               : kConverts ? fixed_mode_waves(kLaneBytes, GT == kGradBF16)
                           : fp32_mode_waves(kLaneBytes);
    return launch_kernel(reinterpret_cast<const void *>(&vector_kernel<W, GT, MODE, ADAM>), blocks,
                         shape.lanes, a, stream,
                         occupancy_lds_bytes(blocks_per_cu_cap(base, shape.lanes, stream)));
}

// The element kernel walks the shard grid-stride with 32 waves per CU (its
// registers allow that many resident).
constexpr int kElementWavesPerCu = 32;

template <int GT, int MODE, bool ADAM>
hipError_t dispatch_w(const LaunchArgs &a, bool vec, Shape shape, hipStream_t stream)
{
    if (!vec) {
        const int64_t cap = static_cast<int64_t>(cu_count()) * kElementWavesPerCu /
                            (shape.lanes / kWave);
        const int64_t need = ceil_div(a.n, shape.lanes);
        return launch_kernel(reinterpret_cast<const void *>(&element_kernel<GT, MODE, ADAM>),
                             need < cap ? need : cap, shape.lanes, a, stream);
    }
    switch (a.W) {
    case 1: return launch_vector<1, GT, MODE, ADAM>(a, shape, stream);
    case 2: return launch_vector<2, GT, MODE, ADAM>(a, shape, stream);
    case 3: return launch_vector<3, GT, MODE, ADAM>(a, shape, stream);
    case 4: return launch_vector<4, GT, MODE, ADAM>(a, shape, stream);
    case 5: return launch_vector<5, GT, MODE, ADAM>(a, shape, stream);
    case 6: return launch_vector<6, GT, MODE, ADAM>(a, shape, stream);
    case 7: return launch_vector<7, GT, MODE, ADAM>(a, shape, stream);
    case 8: return launch_vector<8, GT, MODE, ADAM>(a, shape, stream);
    case 12: return launch_vector<12, GT, MODE, ADAM>(a, shape, stream);
    case 16: return launch_vector<16, GT, MODE, ADAM>(a, shape, stream);
    default: return launch_vector<0, GT, MODE, ADAM>(a, shape, stream);
    }
}

template <bool ADAM>
hipError_t dispatch(const LaunchArgs &a, bool vec, Shape shape, hipStream_t stream)
{
    if (a.gdtype == kGradI32)  // the front end admits int32 only in fixed mode
        return dispatch_w<kGradI32, kAggFixed, ADAM>(a, vec, shape, stream);
    if (a.gdtype == kGradF32)
        return a.mode == kAggFP32 ? dispatch_w<kGradF32, kAggFP32, ADAM>(a, vec, shape, stream)
                                  : dispatch_w<kGradF32, kAggFixed, ADAM>(a, vec, shape, stream);
    return a.mode == kAggFP32 ? dispatch_w<kGradBF16, kAggFP32, ADAM>(a, vec, shape, stream)
                              : dispatch_w<kGradBF16, kAggFixed, ADAM>(a, vec, shape, stream);
}

}  // namespace

hipError_t launch(const LaunchArgs &a, Kind kind, bool vector_path, hipStream_t stream)
{
    const Shape shape = launch_shape();
    return kind == kAggregateAdam ? dispatch<true>(a, vector_path, shape, stream)
                                  : dispatch<false>(a, vector_path, shape, stream);
}

namespace {

// The many-tensor kernel always runs one-wave blocks: its virtual block is
// one 64-group tile.
template <int W, int GT, int MODE>
hipError_t launch_multi_w(const MultiArgs &a, hipStream_t stream)
{
    constexpr int kGradBytes = GT == kGradBF16 ? 2 : 4;
    constexpr int kLaneBytes = W > 0 ? 4 * (W * kGradBytes + 12) : 1 << 30;
    constexpr bool kConverts = MODE == kAggFixed && GT != kGradI32;
    const int base = W == 0    ? runtime_w_waves(a.W, GT, MODE)
                     : kConverts ? fixed_mode_waves(kLaneBytes, GT == kGradBF16)
                                 : fp32_mode_waves(kLaneBytes);
    const int lds = occupancy_lds_bytes(blocks_per_cu_cap(base, kWaveBlock, stream));
    const int64_t blocks = clamp_grid(a.tile_start[a.count], kWaveBlock);
    void *args[] = {const_cast<MultiArgs *>(&a)};
    return hipLaunchKernel(reinterpret_cast<const void *>(&multi_kernel<W, GT, MODE>),
                           dim3(static_cast<unsigned>(blocks)), dim3(kWaveBlock), args,
                           static_cast<size_t>(lds), stream);
}

template <int GT, int MODE>
hipError_t launch_multi_gm(const MultiArgs &a, hipStream_t stream)
{
    switch (a.W) {
    case 1: return launch_multi_w<1, GT, MODE>(a, stream);
    case 2: return launch_multi_w<2, GT, MODE>(a, stream);
    case 3: return launch_multi_w<3, GT, MODE>(a, stream);
    case 4: return launch_multi_w<4, GT, MODE>(a, stream);
    case 5: return launch_multi_w<5, GT, MODE>(a, stream);
    case 6: return launch_multi_w<6, GT, MODE>(a, stream);
    case 7: return launch_multi_w<7, GT, MODE>(a, stream);
    case 8: return launch_multi_w<8, GT, MODE>(a, stream);
    case 12: return launch_multi_w<12, GT, MODE>(a, stream);
    case 16: return launch_multi_w<16, GT, MODE>(a, stream);
    default: return launch_multi_w<0, GT, MODE>(a, stream);
    }
}

}  // namespace

hipError_t launch_multi(const MultiArgs &a, hipStream_t stream)
{
    if (a.gdtype == kGradI32)  // the front end admits int32 only in fixed mode
        return launch_multi_gm<kGradI32, kAggFixed>(a, stream);
    if (a.gdtype == kGradF32)
        return a.mode == kAggFP32 ? launch_multi_gm<kGradF32, kAggFP32>(a, stream)
                                  : launch_multi_gm<kGradF32, kAggFixed>(a, stream);
    return a.mode == kAggFP32 ? launch_multi_gm<kGradBF16, kAggFP32>(a, stream)
                              : launch_multi_gm<kGradBF16, kAggFixed>(a, stream);
}

hipError_t launch_quantize(const QuantizeArgs &q, bool vector_path, hipStream_t stream)
{
    const void *fn;
    int64_t blocks;
    if (vector_path) {
        fn = q.gdtype == kGradBF16 ? reinterpret_cast<const void *>(&quantize_vector_kernel<kGradBF16>)
                                   : reinterpret_cast<const void *>(&quantize_vector_kernel<kGradF32>);
        blocks = ceil_div(q.n >> 2, kWaveBlock);
    } else {
        fn = q.gdtype == kGradBF16 ? reinterpret_cast<const void *>(&quantize_element_kernel<kGradBF16>)
                                   : reinterpret_cast<const void *>(&quantize_element_kernel<kGradF32>);
        blocks = ceil_div(q.n, kWaveBlock);
    }
    blocks = clamp_grid(blocks, kWaveBlock);
    void *args[] = {const_cast<QuantizeArgs *>(&q)};
    return hipLaunchKernel(fn, dim3(static_cast<unsigned>(blocks)), dim3(kWaveBlock), args, 0,
                           stream);
}

}  // namespace disdp
