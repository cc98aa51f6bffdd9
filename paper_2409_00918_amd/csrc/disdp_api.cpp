// C-ABI front end of libdisdp: argument checks (host only, before any HIP
// call), the per-step optimizer constants, and the choice between the
// vector and element-wise kernels.  The ABI itself is documented in
// include/disdp.h.
#include "disdp.h"

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <cstring>
#include <iterator>
#include <map>
#include <vector>

#include "disdp_launch.h"

// disdp_step_scalars_t is the public image of the kernels' StepScalars.
static_assert(sizeof(disdp_step_scalars_t) == sizeof(disdp::StepScalars),
              "step scalars layout");
static_assert(offsetof(disdp_step_scalars_t, bias_correction1) ==
                      offsetof(disdp::StepScalars, bc1) &&
                  offsetof(disdp_step_scalars_t, decay) == offsetof(disdp::StepScalars, decay) &&
                  offsetof(disdp_step_scalars_t, grad_scale) ==
                      offsetof(disdp::StepScalars, grad_scale),
              "step scalars layout");

namespace {

using disdp::LaunchArgs;

struct Span {
    uintptr_t lo, hi;  // [lo, hi)
};

Span span_of(const void *p, int64_t n, int elem_bytes)
{
    uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Span{lo, lo + static_cast<uintptr_t>(n) * static_cast<uintptr_t>(elem_bytes)};
}

bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

int grad_bytes(int gdtype) { return gdtype == DISDP_DT_BF16 ? 2 : 4; }

// Largest n accepted: keeps every byte count far below 2^63.
constexpr int64_t kMaxN = int64_t(1) << 56;

disdp_status_t check_counts(int W, int gdtype, int64_t n, int mode, int frac_bits)
{
    if (n < 0 || n > kMaxN || W < 1 || W > disdp::kMaxW)
        return DISDP_ERR_INVALID_ARG;
    if (gdtype != DISDP_DT_F32 && gdtype != DISDP_DT_BF16 && gdtype != DISDP_DT_I32)
        return DISDP_ERR_UNSUPPORTED;
    if (mode != DISDP_AGG_FP32 && mode != DISDP_AGG_FIXED)
        return DISDP_ERR_UNSUPPORTED;
    if (gdtype == DISDP_DT_I32 && mode != DISDP_AGG_FIXED)
        return DISDP_ERR_UNSUPPORTED;  // integer contributions are summed as integers
    if (mode == DISDP_AGG_FIXED && (frac_bits < 0 || frac_bits > 30))
        return DISDP_ERR_INVALID_ARG;
    return DISDP_OK;
}

disdp_status_t check_hparams(const disdp_adamw_hparams_t *hp)
{
    if (!hp)
        return DISDP_ERR_INVALID_ARG;
    if (hp->step < 1)
        return DISDP_ERR_INVALID_ARG;
    // written so that NaN fails every test
    if (!(hp->beta1 >= 0.0f && hp->beta1 < 1.0f) ||
        !(hp->beta2 >= 0.0f && hp->beta2 < 1.0f))
        return DISDP_ERR_INVALID_ARG;
    if (!(hp->eps >= 0.0f) || !std::isfinite(hp->eps) || !std::isfinite(hp->lr) ||
        !std::isfinite(hp->weight_decay) || !std::isfinite(hp->grad_scale))
        return DISDP_ERR_INVALID_ARG;
    return DISDP_OK;
}

// The step constants: 1 - beta^t and 1 - lr*wd in double, rounded once.
disdp::StepScalars step_scalars(const disdp_adamw_hparams_t *hp)
{
    disdp::StepScalars s;
    s.b1 = hp->beta1;
    s.omb1 = 1.0f - hp->beta1;
    s.b2 = hp->beta2;
    s.omb2 = 1.0f - hp->beta2;
    const double t = static_cast<double>(hp->step);
    s.bc1 = static_cast<float>(1.0 - std::pow(static_cast<double>(hp->beta1), t));
    s.bc2 = static_cast<float>(1.0 - std::pow(static_cast<double>(hp->beta2), t));
    s.decay = static_cast<float>(1.0 - static_cast<double>(hp->lr) *
                                           static_cast<double>(hp->weight_decay));
    s.lr = hp->lr;
    s.eps = hp->eps;
    s.grad_scale = hp->grad_scale;
    return s;
}

// True when the GPU can dereference `p` at that very address: device or
// managed memory, or pinned host memory mapped for the device at the same
// address (hipHostMalloc).  Pageable host memory and unknown addresses are
// refused here, so they never reach a kernel.
// `device_memory` (when given) says whether it is device or managed memory.
bool gpu_addressable(const void *p, bool *device_memory = nullptr)
{
    if (device_memory)
        *device_memory = false;
    hipPointerAttribute_t at;
    const hipError_t pending = hipPeekAtLastError();
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        // clear the error this query recorded, unless the caller already had
        // one pending: that one must stay reported
        if (pending == hipSuccess)
            (void)hipGetLastError();
        return false;
    }
    switch (at.type) {
    case hipMemoryTypeDevice:
    case hipMemoryTypeManaged:
    case hipMemoryTypeUnified:
        if (device_memory)
            *device_memory = true;
        return true;
    case hipMemoryTypeHost:
        return at.devicePointer == p;
    default:
        return false;
    }
}

// gpu_addressable over the many pointers of one call: the device (or
// managed) allocations already confirmed in this call are remembered, and a
// pointer inside one of them needs no further query of the runtime.  Arrays
// carved out of a few large allocations cost one query per allocation.
class AddressableSet {
  public:
    bool check(const void *p)
    {
        const uintptr_t a = reinterpret_cast<uintptr_t>(p);
        if (a - last_lo_ < last_size_)
            return true;
        auto it = known_.upper_bound(a);  // first allocation starting above a
        if (it != known_.begin() && a - std::prev(it)->first < std::prev(it)->second) {
            last_lo_ = std::prev(it)->first;
            last_size_ = std::prev(it)->second;
            return true;
        }
        bool device_memory = false;
        if (!gpu_addressable(p, &device_memory))
            return false;
        if (device_memory) {
            hipDeviceptr_t base = nullptr;
            size_t size = 0;
            const hipError_t pending = hipPeekAtLastError();
            if (hipMemGetAddressRange(&base, &size, const_cast<void *>(p)) == hipSuccess &&
                a - reinterpret_cast<uintptr_t>(base) < size) {
                last_lo_ = reinterpret_cast<uintptr_t>(base);
                last_size_ = size;
                known_[last_lo_] = size;
            } else if (pending == hipSuccess) {
                (void)hipGetLastError();  // as in gpu_addressable
            }
        }
        return true;
    }

  private:
    std::map<uintptr_t, size_t> known_;  // allocation start -> size
    uintptr_t last_lo_ = 0;
    size_t last_size_ = 0;
};

// A vector kernel's tile is 256 elements (a one-wave block of 64 lanes x 4
// elements): 1 KiB of every 4-byte array.  Tiles that start on a 1 KiB
// boundary stream about 5% faster on MI355X than tiles straddling two
// (measured with every array offset by 64, 128 or 192 elements against 0,
// 256 or 512), so the head reaches a 256-element boundary when it can.
constexpr int kTileElems = 256;

// Elements to do one by one before the vector kernels can take arrays
// `p[0..np)` of element sizes `esz` that share a phase: the distance to the
// next common 256-, 64- or 4-element boundary (the coarsest they share),
// -1 when they share none or an array is not aligned to its own element
// size.  Never more than n.
int common_head(const void *const *p, const int *esz, int np, int64_t n)
{
    if (np == 0)
        return 0;
    int ph = -1;
    bool same256 = true, same64 = true, same4 = true;
    for (int i = 0; i < np; ++i) {
        const uintptr_t u = reinterpret_cast<uintptr_t>(p[i]);
        if (u % esz[i])
            return -1;
        const int e = static_cast<int>((u / esz[i]) % kTileElems);
        if (ph < 0)
            ph = e;
        same256 = same256 && e == ph;
        same64 = same64 && (e & 63) == (ph & 63);
        same4 = same4 && (e & 3) == (ph & 3);
    }
    int64_t head;
    if (same256)
        head = (kTileElems - ph) % kTileElems;
    else if (same64)
        head = (64 - (ph & 63)) & 63;
    else if (same4)
        head = (4 - (ph & 3)) & 3;
    else
        return -1;
    return static_cast<int>(head < n ? head : n);
}

// Elements to do one by one before the vector kernels can take arrays that
// share no phase (common_head found none): the reference array `p[ref]` (the
// first output) is brought to a 256-element boundary, or to one element past
// it when that puts every 2-byte array on a 4-byte boundary, and every other
// array is then accessed at whatever 4-byte-aligned address it has (a group
// access needs 4-byte alignment only).  -1 when no head does that (2-byte
// arrays at both odd and even element offsets) or an array is not aligned
// to its element size.  Never more than n.
int shifted_head(const void *const *p, const int *esz, int np, int ref, int64_t n)
{
    for (int i = 0; i < np; ++i)
        if (reinterpret_cast<uintptr_t>(p[i]) % esz[i])
            return -1;
    const uintptr_t r = reinterpret_cast<uintptr_t>(p[ref]) / esz[ref];
    int head = static_cast<int>((kTileElems - r % kTileElems) % kTileElems);
    for (int attempt = 0; attempt < 2; ++attempt, head = (head + 1) % kTileElems) {
        bool ok = true;
        for (int i = 0; i < np && ok; ++i)
            ok = (reinterpret_cast<uintptr_t>(p[i]) +
                  static_cast<uintptr_t>(head) * static_cast<uintptr_t>(esz[i])) % 4 == 0;
        if (ok)
            return static_cast<int>(head < n ? head : n);
    }
    return -1;
}

// The head of a launch over arrays p[0..np), the first output at p[ref]:
// the common phase when the arrays share one, else the shifted head, else
// -1 (the element-wise kernel).
int vector_head(const void *const *p, const int *esz, int np, int ref, int64_t n)
{
    const int head = common_head(p, esz, np, n);
    return head >= 0 || ref >= np ? head : shifted_head(p, esz, np, ref, n);
}

// Shared body of the aggregation and optimizer entry points.  `adam`
// selects the optimizer; for disdp_adam_step the single contribution is the
// fp32 aggregate itself (an aggregate of one fp32 contribution is that
// contribution, unrounded).  With `scalars_in_memory` the step constants
// are not derived from `hp` but read by the kernel from `s_dev`.
disdp_status_t run(const void *const *grads, int W, int gdtype, int64_t n,
                   int mode, int frac_bits, float *param, float *m, float *v,
                   uint16_t *p16, float *agg_f32, int32_t *agg_i32,
                   const disdp_adamw_hparams_t *hp, bool adam,
                   bool agg_f32_required, hipStream_t stream,
                   bool scalars_in_memory = false, const disdp::StepScalars *s_dev = nullptr)
{
    disdp_status_t st = check_counts(W, gdtype, n, mode, frac_bits);
    if (st != DISDP_OK)
        return st;
    if (adam && !scalars_in_memory && (st = check_hparams(hp)) != DISDP_OK)
        return st;
    if (mode == DISDP_AGG_FP32 && agg_i32)
        return DISDP_ERR_INVALID_ARG;  // an int32 aggregate exists only in fixed mode
    if (n == 0)
        return DISDP_OK;

    // NULL pointers
    if (!grads)
        return DISDP_ERR_INVALID_ARG;
    for (int w = 0; w < W; ++w)
        if (!grads[w])
            return DISDP_ERR_INVALID_ARG;
    if (adam && (!param || !m || !v))
        return DISDP_ERR_INVALID_ARG;
    if (scalars_in_memory && (!s_dev || (reinterpret_cast<uintptr_t>(s_dev) & 3)))
        return DISDP_ERR_INVALID_ARG;
    if (!adam) {
        if (agg_f32_required && !agg_f32)
            return DISDP_ERR_INVALID_ARG;
        if (!agg_f32 && !agg_i32)
            return DISDP_ERR_INVALID_ARG;
    }

    // Overlap: every output against every other buffer.
    const int gb = grad_bytes(gdtype);
    Span outs[6];
    int nout = 0;
    if (param) outs[nout++] = span_of(param, n, 4);
    if (m) outs[nout++] = span_of(m, n, 4);
    if (v) outs[nout++] = span_of(v, n, 4);
    if (p16) outs[nout++] = span_of(p16, n, 2);
    if (agg_f32) outs[nout++] = span_of(agg_f32, n, 4);
    if (agg_i32) outs[nout++] = span_of(agg_i32, n, 4);
    for (int i = 0; i < nout; ++i) {
        for (int j = i + 1; j < nout; ++j)
            if (overlaps(outs[i], outs[j]))
                return DISDP_ERR_ALIAS;
        for (int w = 0; w < W; ++w)
            if (overlaps(outs[i], span_of(grads[w], n, gb)))
                return DISDP_ERR_ALIAS;
        if (s_dev && overlaps(outs[i], span_of(s_dev, 1, sizeof(disdp::StepScalars))))
            return DISDP_ERR_ALIAS;
    }

    // Every array must be addressable by the GPU as given (first HIP call).
    for (int w = 0; w < W; ++w)
        if (!gpu_addressable(grads[w]))
            return DISDP_ERR_INVALID_ARG;
    for (const void *p : {static_cast<const void *>(param), static_cast<const void *>(m),
                          static_cast<const void *>(v), static_cast<const void *>(p16),
                          static_cast<const void *>(agg_f32), static_cast<const void *>(agg_i32),
                          static_cast<const void *>(s_dev)})
        if (p && !gpu_addressable(p))
            return DISDP_ERR_INVALID_ARG;

    LaunchArgs a;
    std::memset(&a, 0, sizeof a);
    for (int w = 0; w < W; ++w)
        a.g[w] = grads[w];
    a.p = param;
    a.m = m;
    a.v = v;
    a.p16 = p16;
    a.agg_f32 = agg_f32;
    a.agg_i32 = agg_i32;
    a.n = n;
    a.W = W;
    a.gdtype = gdtype;
    a.mode = mode;
    a.frac_bits = (mode == DISDP_AGG_FIXED) ? frac_bits : 0;
    a.qscale = std::ldexp(1.0f, a.frac_bits);
    a.dqscale = std::ldexp(1.0f, -a.frac_bits);
    if (adam && !s_dev)
        a.s = step_scalars(hp);
    a.s_dev = s_dev;

    // Vector kernels move 4 elements per lane: 16-byte groups of 4-byte
    // arrays, 8-byte groups of 2-byte arrays.  Arrays that all start the same
    // number of elements past such a boundary (a sub-range of aligned arrays)
    // take the vector kernel too: their first elements are done one by one
    // and the pointers advanced.  When the arrays agree modulo 256 (or 64)
    // elements the pointers are advanced to such a boundary, which starts
    // every tile on a 1 KiB boundary (or at least every wave's stores on
    // whole cache lines), as for aligned arrays.  Arrays with unrelated
    // offsets put the first output on a tile boundary and the others
    // wherever they fall on 4-byte boundaries.
    const void *ptrs[disdp::kMaxW + 6];
    int sizes[disdp::kMaxW + 6];
    int np = 0;
    for (int w = 0; w < W; ++w) {
        ptrs[np] = grads[w];
        sizes[np++] = gb;
    }
    const void *outs_p[] = {param, m, v, p16, agg_f32, agg_i32};
    const int outs_sz[] = {4, 4, 4, 2, 4, 4};
    for (int k = 0; k < 6; ++k)
        if (outs_p[k]) {
            ptrs[np] = outs_p[k];
            sizes[np++] = outs_sz[k];
        }
    const int head = vector_head(ptrs, sizes, np, /*ref=*/W, n);
    const bool vec = head >= 0;
    if (head > 0) {
        a.head = head;
        a.n = n - head;
        for (int w = 0; w < W; ++w)
            a.g[w] = static_cast<const char *>(grads[w]) + static_cast<int64_t>(head) * gb;
        a.p = param ? param + head : nullptr;
        a.m = m ? m + head : nullptr;
        a.v = v ? v + head : nullptr;
        a.p16 = p16 ? p16 + head : nullptr;
        a.agg_f32 = agg_f32 ? agg_f32 + head : nullptr;
        a.agg_i32 = agg_i32 ? agg_i32 + head : nullptr;
    }

    hipError_t e = disdp::launch(a, adam ? disdp::kAggregateAdam : disdp::kAggregateOnly,
                                 vec, stream);
    return e == hipSuccess ? DISDP_OK : DISDP_ERR_HIP;
}

// Largest tensor count of disdp_aggregate_adam_multi.
constexpr int kMaxTensors = 65536;

// A byte interval [lo, hi) and whether the call writes it.
struct Tagged {
    uintptr_t lo, hi;
    bool out;
};

// True when some written interval overlaps any other interval (written or
// read); read intervals may overlap one another.  One sort and one sweep:
// for a pair that overlaps, the later-starting interval starts before the
// end of the earlier one, which the sweep keeps as the largest end so far.
bool written_overlap(std::vector<Tagged> &spans)
{
    const auto by_start = [](const Tagged &a, const Tagged &b) { return a.lo < b.lo; };
    if (!std::is_sorted(spans.begin(), spans.end(), by_start))
        std::sort(spans.begin(), spans.end(), by_start);
    uintptr_t max_end = 0, max_out_end = 0;
    for (const Tagged &t : spans) {
        if (t.lo < max_out_end || (t.out && t.lo < max_end))
            return true;
        max_end = std::max(max_end, t.hi);
        if (t.out)
            max_out_end = std::max(max_out_end, t.hi);
    }
    return false;
}

}  // namespace

extern "C" {

disdp_status_t disdp_aggregate(const void *const *grads, int W, disdp_dtype_t gdtype,
                               int64_t n, disdp_agg_mode_t mode, int frac_bits,
                               float *agg_out_f32, int32_t *agg_out_i32,
                               hipStream_t stream)
{
    return run(grads, W, gdtype, n, mode, frac_bits, nullptr, nullptr, nullptr,
               nullptr, agg_out_f32, agg_out_i32, nullptr, /*adam=*/false,
               /*agg_f32_required=*/mode == DISDP_AGG_FP32, stream);
}

disdp_status_t disdp_adam_step(const float *grad, float *param, float *m, float *v,
                               uint16_t *param_bf16_out, int64_t n,
                               const disdp_adamw_hparams_t *hp, hipStream_t stream)
{
    const void *grads[1] = {grad};
    return run(grads, 1, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, param, m, v,
               param_bf16_out, nullptr, nullptr, hp, /*adam=*/true,
               /*agg_f32_required=*/false, stream);
}

disdp_status_t disdp_aggregate_adam(const void *const *grads, int W,
                                    disdp_dtype_t gdtype, int64_t n,
                                    disdp_agg_mode_t mode, int frac_bits,
                                    float *param, float *m, float *v,
                                    uint16_t *param_bf16_out, float *agg_out_f32,
                                    int32_t *agg_out_i32,
                                    const disdp_adamw_hparams_t *hp,
                                    hipStream_t stream)
{
    return run(grads, W, gdtype, n, mode, frac_bits, param, m, v, param_bf16_out,
               agg_out_f32, agg_out_i32, hp, /*adam=*/true,
               /*agg_f32_required=*/false, stream);
}

disdp_status_t disdp_step_scalars(const disdp_adamw_hparams_t *hp, disdp_step_scalars_t *out)
{
    if (!out)
        return DISDP_ERR_INVALID_ARG;
    const disdp_status_t st = check_hparams(hp);
    if (st != DISDP_OK)
        return st;
    const disdp::StepScalars sc = step_scalars(hp);
    std::memcpy(out, &sc, sizeof sc);
    return DISDP_OK;
}

disdp_status_t disdp_aggregate_adam_dev(const void *const *grads, int W,
                                        disdp_dtype_t gdtype, int64_t n,
                                        disdp_agg_mode_t mode, int frac_bits,
                                        float *param, float *m, float *v,
                                        uint16_t *param_bf16_out, float *agg_out_f32,
                                        int32_t *agg_out_i32,
                                        const disdp_step_scalars_t *scalars,
                                        hipStream_t stream)
{
    return run(grads, W, gdtype, n, mode, frac_bits, param, m, v, param_bf16_out,
               agg_out_f32, agg_out_i32, nullptr, /*adam=*/true,
               /*agg_f32_required=*/false, stream, /*scalars_in_memory=*/true,
               reinterpret_cast<const disdp::StepScalars *>(scalars));
}

disdp_status_t disdp_aggregate_adam_multi(const void *const *grads, int W,
                                          disdp_dtype_t gdtype, int T, const int64_t *n,
                                          disdp_agg_mode_t mode, int frac_bits,
                                          float *const *param, float *const *m,
                                          float *const *v, uint16_t *const *param_bf16_out,
                                          const disdp_adamw_hparams_t *hp,
                                          const disdp_step_scalars_t *scalars, hipStream_t stream)
{
    if (T < 0 || T > kMaxTensors)
        return DISDP_ERR_INVALID_ARG;
    disdp_status_t st = check_counts(W, gdtype, 0, mode, frac_bits);
    if (st != DISDP_OK)
        return st;
    if ((hp != nullptr) == (scalars != nullptr))
        return DISDP_ERR_INVALID_ARG;      // exactly one source of the constants
    if (hp && (st = check_hparams(hp)) != DISDP_OK)
        return st;
    if (scalars && (reinterpret_cast<uintptr_t>(scalars) & 3))
        return DISDP_ERR_INVALID_ARG;
    if (T > 0 && !n)
        return DISDP_ERR_INVALID_ARG;
    bool any = false;
    for (int j = 0; j < T; ++j) {
        if (n[j] < 0 || n[j] > kMaxN)
            return DISDP_ERR_INVALID_ARG;
        any = any || n[j] > 0;
    }
    if (!any)
        return DISDP_OK;

    // NULL pointers, then overlap over every tensor's buffers at once
    if (!grads || !param || !m || !v)
        return DISDP_ERR_INVALID_ARG;
    const int gb = grad_bytes(gdtype);
    for (int j = 0; j < T; ++j) {
        if (n[j] == 0)
            continue;
        for (int w = 0; w < W; ++w)
            if (!grads[static_cast<int64_t>(j) * W + w])
                return DISDP_ERR_INVALID_ARG;
        if (!param[j] || !m[j] || !v[j])
            return DISDP_ERR_INVALID_ARG;
    }
    // Array by array: when every array holds its tensors in address order
    // (sub-ranges of flat shard arrays) the list arrives sorted.
    std::vector<Tagged> spans;
    spans.reserve(static_cast<size_t>(T) * (W + 4) + 1);
    auto add = [&](auto arr, int64_t stride, int esz, bool out) {
        for (int j = 0; j < T; ++j) {
            const void *p = arr[static_cast<int64_t>(j) * stride];
            if (n[j] > 0 && p) {
                const Span sp = span_of(p, n[j], esz);
                spans.push_back({sp.lo, sp.hi, out});
            }
        }
    };
    for (int w = 0; w < W; ++w)
        add(grads + w, W, gb, false);
    add(param, 1, 4, true);
    add(m, 1, 4, true);
    add(v, 1, 4, true);
    if (param_bf16_out)
        add(param_bf16_out, 1, 2, true);
    if (scalars) {
        const Span sp = span_of(scalars, 1, sizeof(disdp_step_scalars_t));
        spans.push_back({sp.lo, sp.hi, false});
    }
    if (written_overlap(spans))
        return DISDP_ERR_ALIAS;
    AddressableSet addressable;
    if (scalars && !addressable.check(scalars))
        return DISDP_ERR_INVALID_ARG;
    for (int j = 0; j < T; ++j) {
        if (n[j] == 0)
            continue;
        for (int w = 0; w < W; ++w)
            if (!addressable.check(grads[static_cast<int64_t>(j) * W + w]))
                return DISDP_ERR_INVALID_ARG;
        if (!addressable.check(param[j]) || !addressable.check(m[j]) ||
            !addressable.check(v[j]) ||
            (param_bf16_out && param_bf16_out[j] && !addressable.check(param_bf16_out[j])))
            return DISDP_ERR_INVALID_ARG;
    }

    // Batches of tensors per launch; a tensor the vector kernels cannot
    // take goes through the single-tensor path (the element kernel).
    disdp::MultiArgs ma;
    std::memset(&ma, 0, sizeof ma);
    ma.W = W;
    ma.gdtype = gdtype;
    ma.mode = mode;
    ma.frac_bits = (mode == DISDP_AGG_FIXED) ? frac_bits : 0;
    ma.qscale = std::ldexp(1.0f, ma.frac_bits);
    ma.dqscale = std::ldexp(1.0f, -ma.frac_bits);
    const disdp::StepScalars *s_dev = reinterpret_cast<const disdp::StepScalars *>(scalars);
    if (hp)
        ma.s = step_scalars(hp);
    ma.s_dev = s_dev;
    const int per_tensor = W + 4;
    const int cap = std::min(disdp::kMultiMaxTensors, disdp::kMultiMaxPtrs / per_tensor);
    auto flush = [&]() -> bool {
        if (ma.count == 0)
            return true;
        const hipError_t e = disdp::launch_multi(ma, stream);
        ma.count = 0;
        return e == hipSuccess;
    };
    for (int j = 0; j < T; ++j) {
        if (n[j] == 0)
            continue;
        const void *const *gj = grads + static_cast<int64_t>(j) * W;
        uint16_t *p16 = param_bf16_out ? param_bf16_out[j] : nullptr;
        const void *ptrs[disdp::kMaxW + 4];
        int sizes[disdp::kMaxW + 4];
        int np = 0;
        for (int w = 0; w < W; ++w) {
            ptrs[np] = gj[w];
            sizes[np++] = gb;
        }
        const void *state[] = {param[j], m[j], v[j]};
        for (const void *sp : state) {
            ptrs[np] = sp;
            sizes[np++] = 4;
        }
        if (p16) {
            ptrs[np] = p16;
            sizes[np++] = 2;
        }
        const int head = vector_head(ptrs, sizes, np, /*ref=*/W, n[j]);
        if (head < 0) {
            st = run(gj, W, gdtype, n[j], mode, frac_bits, param[j], m[j], v[j], p16, nullptr,
                     nullptr, hp, /*adam=*/true, /*agg_f32_required=*/false, stream,
                     /*scalars_in_memory=*/s_dev != nullptr, s_dev);
            if (st != DISDP_OK)
                return st;
            continue;
        }
        if (ma.count == cap && !flush())
            return DISDP_ERR_HIP;
        const int c = ma.count;
        void **slot = ma.ptr + c * per_tensor;
        for (int w = 0; w < W; ++w)
            slot[w] = const_cast<char *>(static_cast<const char *>(gj[w])) +
                      static_cast<int64_t>(head) * gb;
        slot[W] = param[j] + head;
        slot[W + 1] = m[j] + head;
        slot[W + 2] = v[j] + head;
        slot[W + 3] = p16 ? p16 + head : nullptr;
        ma.n[c] = n[j] - head;
        ma.head[c] = head;
        const int64_t groups = ma.n[c] >> 2;
        const int64_t tiles =
            std::max<int64_t>(1, (groups + disdp::kMultiTileGroups - 1) / disdp::kMultiTileGroups);
        ma.tile_start[c + 1] = ma.tile_start[c] + tiles;
        ma.count = c + 1;
    }
    return flush() ? DISDP_OK : DISDP_ERR_HIP;
}

disdp_status_t disdp_quantize(const void *grad, disdp_dtype_t gdtype, int64_t n,
                              int frac_bits, int32_t *out, hipStream_t stream)
{
    if (n < 0 || n > kMaxN)
        return DISDP_ERR_INVALID_ARG;
    if (gdtype != DISDP_DT_F32 && gdtype != DISDP_DT_BF16)
        return DISDP_ERR_UNSUPPORTED;
    if (frac_bits < 0 || frac_bits > 30)
        return DISDP_ERR_INVALID_ARG;
    if (n == 0)
        return DISDP_OK;
    if (!grad || !out)
        return DISDP_ERR_INVALID_ARG;
    if (overlaps(span_of(out, n, 4), span_of(grad, n, grad_bytes(gdtype))))
        return DISDP_ERR_ALIAS;
    if (!gpu_addressable(grad) || !gpu_addressable(out))
        return DISDP_ERR_INVALID_ARG;
    disdp::QuantizeArgs q;
    q.g = grad;
    q.out = out;
    q.n = n;
    q.head = 0;
    q.gdtype = gdtype;
    q.qscale = std::ldexp(1.0f, frac_bits);
    // as in run(): a misalignment is peeled off one element at a time
    const int gb = grad_bytes(gdtype);
    const void *ptrs[2] = {grad, out};
    const int sizes[2] = {gb, 4};
    const int head = vector_head(ptrs, sizes, 2, /*ref=*/1, n);
    const bool vec = head >= 0;
    if (head > 0) {
        q.head = head;
        q.n = n - head;
        q.g = static_cast<const char *>(grad) + static_cast<int64_t>(head) * gb;
        q.out = out + head;
    }
    return disdp::launch_quantize(q, vec, stream) == hipSuccess ? DISDP_OK : DISDP_ERR_HIP;
}

disdp_status_t disdp_shard_layout(int64_t n, int W, disdp_dtype_t gdtype, unsigned flags,
                                  int64_t *offsets, int64_t *total_bytes)
{
    if (n < 0 || n > kMaxN || W < 1 || W > disdp::kMaxW || !offsets || !total_bytes)
        return DISDP_ERR_INVALID_ARG;
    if (gdtype != DISDP_DT_F32 && gdtype != DISDP_DT_BF16 && gdtype != DISDP_DT_I32)
        return DISDP_ERR_UNSUPPORTED;
    constexpr int64_t kPage = int64_t(1) << 21;
    auto pages = [](int64_t bytes) { return (bytes + kPage - 1) / kPage * kPage; };
    // element size of each array in placement order; 0 = not requested
    int esz[disdp::kMaxW + 6];
    for (int w = 0; w < W; ++w)
        esz[w] = grad_bytes(gdtype);
    esz[W + 0] = 4;  // param
    esz[W + 1] = 4;  // m
    esz[W + 2] = 4;  // v
    esz[W + 3] = (flags & DISDP_LAYOUT_BF16_COPY) ? 2 : 0;
    esz[W + 4] = (flags & DISDP_LAYOUT_AGG_F32) ? 4 : 0;
    esz[W + 5] = (flags & DISDP_LAYOUT_AGG_I32) ? 4 : 0;
    // Every array starts on a 32 MiB boundary (16 pages of 2 MiB), the next
    // one at the first boundary at least 17 pages past the end of the
    // previous one -- measured on MI355X over arrays of 128 to 5216 pages,
    // the placement whose slowest case streamed fastest (see the header).
    if (n == 0) {  // nothing to place: every requested array at offset 0
        for (int i = 0; i < W + 6; ++i)
            offsets[i] = esz[i] ? 0 : -1;
        *total_bytes = 0;
        return DISDP_OK;
    }
    constexpr int64_t kAlign = 16 * kPage;
    constexpr int64_t kGap = 17 * kPage;
    int64_t at = 0;          // start of the next array, kAlign aligned
    int64_t end = -1;        // end of the previous array, -1 before the first
    // Every step adds at most kGap + kAlign plus the array: checked against
    // the int64 range before it is taken (n <= 2^56 and W <= 64 can exceed it).
    constexpr int64_t kMaxTotal = INT64_MAX;
    for (int i = 0; i < W + 6; ++i) {
        const int esize = esz[i];
        if (esize == 0) {
            offsets[i] = -1;
            continue;
        }
        const int64_t span = pages(n * esize);
        if ((end < 0 ? at : end) > kMaxTotal - kGap - kAlign - span)
            return DISDP_ERR_INVALID_ARG;
        if (end >= 0)
            at = (end + kGap + kAlign - 1) / kAlign * kAlign;
        offsets[i] = at;
        end = at + span;
    }
    at = end < 0 ? 0 : end;
    *total_bytes = at;
    return DISDP_OK;
}

const char *disdp_status_string(disdp_status_t status)
{
    switch (status) {
    case DISDP_OK: return "ok";
    case DISDP_ERR_INVALID_ARG: return "invalid argument";
    case DISDP_ERR_UNSUPPORTED: return "unsupported dtype or mode";
    case DISDP_ERR_ALIAS: return "output overlaps another buffer";
    case DISDP_ERR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

}  // extern "C"
