// Host-side fuzz of the C-ABI front end (paper_2409_00918_amd/csrc/disdp_api.cpp)
// built with g++ under AddressSanitizer and UndefinedBehaviorSanitizer,
// without a GPU: the two HIP runtime calls the front end makes and the two
// kernel-launch entry points are replaced by the stubs below, which record
// what would have been launched.
//
//   * disdp_shard_layout over random n (up to 2^56), W, dtypes and flags:
//     status, and every placement invariant of a successful layout;
//   * each entry point with exactly one argument error injected into an
//     otherwise valid call: the documented status, and no launch (valid
//     fused calls: the step constants passed by value, or by address only);
//   * disdp_aggregate_adam_multi over random tensor lists: batch packing,
//     per-tensor heads and pointers, the single-tensor fallback, injected
//     errors;
//   * valid calls whose arrays share, or do not share, a misalignment: the
//     vector/element choice, the head of elements done one by one and the
//     advanced pointers (on a common boundary, or every array on a 4-byte
//     boundary with the first output on a 64-element one).
//
// Prints "api_fuzz: ok" and exits 0; any failed check prints the case and
// exits 1; a sanitizer finding aborts.
#include <cinttypes>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <set>
#include <vector>

#include "disdp.h"
#include "disdp_launch.h"

// ---- stubs for what the front end calls below it ---------------------------
namespace {
int g_launches = 0;
int g_queries = 0;
bool g_addressable = true;
disdp::LaunchArgs g_args;
bool g_vec = false;
disdp::QuantizeArgs g_qargs;
std::vector<disdp::LaunchArgs> g_singles;  // every single-tensor launch
std::vector<bool> g_single_vec;
std::vector<disdp::MultiArgs> g_multis;    // every multi-tensor launch
}  // namespace

namespace disdp {
hipError_t launch(const LaunchArgs &a, Kind, bool vector_path, hipStream_t)
{
    ++g_launches;
    g_args = a;
    g_vec = vector_path;
    g_singles.push_back(a);
    g_single_vec.push_back(vector_path);
    return hipSuccess;
}
hipError_t launch_multi(const MultiArgs &a, hipStream_t)
{
    ++g_launches;
    g_multis.push_back(a);
    return hipSuccess;
}
hipError_t launch_quantize(const QuantizeArgs &q, bool vector_path, hipStream_t)
{
    ++g_launches;
    g_qargs = q;
    g_vec = vector_path;
    return hipSuccess;
}
}  // namespace disdp

// Device memory is modelled as 64 GiB allocations aligned to their size,
// except one 1 TiB region that the GPU cannot address.
constexpr uintptr_t kAllocBytes = uintptr_t(1) << 36;
constexpr uintptr_t kBadLo = uintptr_t(1) << 50, kBadHi = kBadLo + (uintptr_t(1) << 40);
bool unaddressable(const void *p)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    return !g_addressable || (a >= kBadLo && a < kBadHi);
}

extern "C" hipError_t hipPointerGetAttributes(hipPointerAttribute_t *at, const void *p)
{
    ++g_queries;
    std::memset(at, 0, sizeof *at);
    if (unaddressable(p))
        return hipErrorInvalidValue;
    at->type = hipMemoryTypeDevice;
    at->devicePointer = const_cast<void *>(p);
    return hipSuccess;
}

extern "C" hipError_t hipMemGetAddressRange(hipDeviceptr_t *base, size_t *size, hipDeviceptr_t p)
{
    if (unaddressable(p))
        return hipErrorInvalidValue;
    *base = reinterpret_cast<hipDeviceptr_t>(reinterpret_cast<uintptr_t>(p) & ~(kAllocBytes - 1));
    *size = kAllocBytes;
    return hipSuccess;
}

extern "C" hipError_t hipGetLastError(void) { return hipSuccess; }
extern "C" hipError_t hipPeekAtLastError(void) { return hipSuccess; }

// ---- helpers ------------------------------------------------------------------
namespace {

uint64_t rng_state = 0x9E3779B97F4A7C15ull;
uint64_t next()
{
    uint64_t x = (rng_state += 0x9E3779B97F4A7C15ull);
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}
int64_t below(int64_t k) { return static_cast<int64_t>(next() % static_cast<uint64_t>(k)); }

int failures = 0;
#define CHECK(cond, ...)                                                   \
    do {                                                                   \
        if (!(cond)) {                                                     \
            std::printf("FAIL %s:%d: %s: ", __FILE__, __LINE__, #cond);    \
            std::printf(__VA_ARGS__);                                      \
            std::printf("\n");                                             \
            if (++failures > 20)                                           \
                std::exit(1);                                              \
        }                                                                  \
    } while (0)

constexpr int64_t kPage = int64_t(1) << 21;

// ---- disdp_shard_layout --------------------------------------------------------
void fuzz_layout(int iters)
{
    for (int it = 0; it < iters; ++it) {
        int64_t n;
        switch (below(6)) {
        case 0: n = below(5); break;
        case 1: n = below(1 << 20); break;
        case 2: n = below(int64_t(1) << 40); break;
        case 3: n = int64_t(1) << 56; break;
        case 4: n = below((int64_t(1) << 56) + 1); break;
        default: n = -below(1000) - 1; break;
        }
        const int W = static_cast<int>(below(67));  // 0 and 65, 66 invalid
        const int gdt = static_cast<int>(below(4));  // 3 invalid
        const unsigned flags = static_cast<unsigned>(below(8));
        int64_t off[disdp::kMaxW + 6];
        int64_t total = -7;
        const disdp_status_t st =
            disdp_shard_layout(n, W, static_cast<disdp_dtype_t>(gdt), flags, off, &total);
        const bool bad_count = n < 0 || n > (int64_t(1) << 56) || W < 1 || W > 64;
        if (bad_count) {
            CHECK(st == DISDP_ERR_INVALID_ARG, "n=%" PRId64 " W=%d st=%d", n, W, st);
            continue;
        }
        if (gdt == 3) {
            CHECK(st == DISDP_ERR_UNSUPPORTED, "gdt=3 st=%d", st);
            continue;
        }
        // element sizes in placement order; 0 = not requested
        int esz[disdp::kMaxW + 6];
        for (int w = 0; w < W; ++w)
            esz[w] = gdt == 1 ? 2 : 4;
        esz[W] = esz[W + 1] = esz[W + 2] = 4;
        esz[W + 3] = (flags & 1) ? 2 : 0;
        esz[W + 4] = (flags & 2) ? 4 : 0;
        esz[W + 5] = (flags & 4) ? 4 : 0;
        // a lower bound of the total in 128-bit arithmetic
        __int128 need = 0;
        for (int i = 0; i < W + 6; ++i)
            if (esz[i])
                need += (static_cast<__int128>(n) * esz[i] + kPage - 1) / kPage * kPage;
        if (st != DISDP_OK) {
            CHECK(st == DISDP_ERR_INVALID_ARG && need > (static_cast<__int128>(INT64_MAX) / 2),
                  "refused a layout of %.3g bytes: st=%d", static_cast<double>(need), st);
            continue;
        }
        CHECK(need <= INT64_MAX, "accepted an int64-overflowing layout");
        if (n == 0) {
            CHECK(total == 0, "n = 0: total %" PRId64, total);
            for (int i = 0; i < W + 6; ++i)
                CHECK(off[i] == (esz[i] ? 0 : -1), "n = 0: array %d at %" PRId64, i, off[i]);
            continue;
        }
        const int64_t kAlign = 16 * kPage, kGap = 17 * kPage;
        int64_t prev_end = -1;
        for (int i = 0; i < W + 6; ++i) {
            if (!esz[i]) {
                CHECK(off[i] == -1, "array %d not requested but placed", i);
                continue;
            }
            CHECK(off[i] >= 0 && off[i] % kAlign == 0, "array %d offset %" PRId64, i, off[i]);
            if (prev_end < 0)
                CHECK(off[i] == 0, "first array at %" PRId64, off[i]);
            else
                CHECK(off[i] >= prev_end + kGap && off[i] - kAlign < prev_end + kGap,
                      "array %d not at the first boundary 17 pages past the previous end", i);
            const int64_t end = off[i] + (n * esz[i] + kPage - 1) / kPage * kPage;
            CHECK(end <= total, "array %d ends past the total", i);
            prev_end = end;
        }
        CHECK(total == prev_end, "total %" PRId64 " != last end %" PRId64, total, prev_end);
    }
}

// ---- one error injected into a valid call ---------------------------------------
struct Call {
    int entry;  // 0 aggregate, 1 adam_step, 2 aggregate_adam, 3 quantize,
                // 4 aggregate_adam_dev
    int W, gdt, mode, k;
    int64_t n;
    const void *g[disdp::kMaxW];
    const void *const *grads;
    float *p, *m, *v, *af;
    uint16_t *p16;
    int32_t *ai;
    disdp_adamw_hparams_t hp;
    bool hp_null;
    const disdp_step_scalars_t *s;  // aggregate_adam_dev
};

bool fused(int entry) { return entry == 2 || entry == 4; }

// Fake, never dereferenced, well separated addresses: array i at base + i * 2^40.
char *fake(int i) { return reinterpret_cast<char *>((uintptr_t(1) << 44) + (uintptr_t(i) << 40)); }

Call valid_call(int entry)
{
    Call c{};
    c.entry = entry;
    c.W = entry == 1 || entry == 3 ? 1 : 1 + static_cast<int>(below(64));
    c.mode = entry == 1 ? DISDP_AGG_FP32 : static_cast<int>(below(2));
    c.gdt = entry == 1 ? DISDP_DT_F32
            : (c.mode == DISDP_AGG_FIXED && entry != 3) ? static_cast<int>(below(3))
                                                        : static_cast<int>(below(2));
    c.k = static_cast<int>(below(31));
    c.n = 1 + below(1 << 30);
    for (int w = 0; w < c.W; ++w)
        c.g[w] = fake(w);
    c.grads = c.g;
    c.p = reinterpret_cast<float *>(fake(70));
    c.m = reinterpret_cast<float *>(fake(71));
    c.v = reinterpret_cast<float *>(fake(72));
    c.p16 = below(2) ? reinterpret_cast<uint16_t *>(fake(73)) : nullptr;
    c.af = reinterpret_cast<float *>(fake(74));
    c.ai = c.mode == DISDP_AGG_FIXED ? reinterpret_cast<int32_t *>(fake(75)) : nullptr;
    if (fused(entry) && below(2)) {
        c.af = nullptr;
        c.ai = nullptr;
    }
    c.hp = {1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 1 + below(100000), 1.0f};
    c.s = reinterpret_cast<const disdp_step_scalars_t *>(fake(76) + 4 * below(1000));
    return c;
}

disdp_status_t issue(const Call &c)
{
    const disdp_adamw_hparams_t *hp = c.hp_null ? nullptr : &c.hp;
    switch (c.entry) {
    case 0:
        return disdp_aggregate(c.grads, c.W, static_cast<disdp_dtype_t>(c.gdt), c.n,
                               static_cast<disdp_agg_mode_t>(c.mode), c.k, c.af, c.ai, nullptr);
    case 1:
        return disdp_adam_step(c.grads ? static_cast<const float *>(c.grads[0]) : nullptr, c.p,
                               c.m, c.v, c.p16, c.n, hp, nullptr);
    case 2:
        return disdp_aggregate_adam(c.grads, c.W, static_cast<disdp_dtype_t>(c.gdt), c.n,
                                    static_cast<disdp_agg_mode_t>(c.mode), c.k, c.p, c.m, c.v,
                                    c.p16, c.af, c.ai, hp, nullptr);
    case 4:
        return disdp_aggregate_adam_dev(c.grads, c.W, static_cast<disdp_dtype_t>(c.gdt), c.n,
                                        static_cast<disdp_agg_mode_t>(c.mode), c.k, c.p, c.m,
                                        c.v, c.p16, c.af, c.ai, c.s, nullptr);
    default:
        return disdp_quantize(c.grads ? c.grads[0] : nullptr,
                              static_cast<disdp_dtype_t>(c.gdt), c.n, c.k,
                              c.ai ? c.ai : reinterpret_cast<int32_t *>(fake(75)), nullptr);
    }
}

void fuzz_errors(int iters)
{
    for (int it = 0; it < iters; ++it) {
        const int entry = static_cast<int>(below(5));
        Call c = valid_call(entry);
        if (entry == 0 && c.mode == DISDP_AGG_FP32 && !c.af)
            c.af = reinterpret_cast<float *>(fake(74));
        if (entry == 0 && c.mode == DISDP_AGG_FIXED && !c.af && !c.ai)
            c.ai = reinterpret_cast<int32_t *>(fake(75));
        disdp_status_t want = DISDP_OK;
        const int kind = static_cast<int>(below(14));
        switch (kind) {
        case 0:  // n out of range
            c.n = below(2) ? -1 - below(100) : (int64_t(1) << 56) + 1 + below(100);
            want = DISDP_ERR_INVALID_ARG;
            break;
        case 1:  // W out of range (the two single-buffer calls have none)
            if (entry == 0 || fused(entry)) {
                c.W = below(2) ? 0 : 65 + static_cast<int>(below(100));
                want = DISDP_ERR_INVALID_ARG;
            }
            break;
        case 2:  // unknown dtype or mode
            if (entry != 1) {
                if (below(2) || entry == 3)
                    c.gdt = 3 + static_cast<int>(below(5));
                else
                    c.mode = 2 + static_cast<int>(below(5));
                want = DISDP_ERR_UNSUPPORTED;
            }
            break;
        case 3:  // bad frac_bits in fixed mode (quantize: always checked)
            if ((entry != 1 && c.mode == DISDP_AGG_FIXED) || entry == 3) {
                c.k = below(2) ? -1 - static_cast<int>(below(10)) : 31 + static_cast<int>(below(10));
                want = DISDP_ERR_INVALID_ARG;
            }
            break;
        case 4:  // bad hyperparameters (aggregate_adam_dev reads none)
            if (entry == 1 || entry == 2) {
                switch (below(7)) {
                case 0: c.hp.step = -below(5); break;
                case 1: c.hp.beta1 = 1.0f; break;
                case 2: c.hp.beta2 = NAN; break;
                case 3: c.hp.eps = -1e-8f; break;
                case 4: c.hp.lr = INFINITY; break;
                case 5: c.hp.grad_scale = NAN; break;
                default: c.hp_null = true; break;
                }
                want = DISDP_ERR_INVALID_ARG;
            }
            break;
        case 5:  // NULL contribution array or pointer
            if (below(2) && entry != 1 && entry != 3)
                c.grads = nullptr;
            else
                c.g[below(c.W)] = nullptr;
            want = DISDP_ERR_INVALID_ARG;
            break;
        case 6:  // NULL state
            if (entry == 1 || fused(entry)) {
                c.m = nullptr;
                want = DISDP_ERR_INVALID_ARG;
            }
            break;
        case 7:  // an output overlapping a contribution somewhere inside it
            if (entry == 0 && c.af) {
                c.af = reinterpret_cast<float *>(const_cast<char *>(
                    static_cast<const char *>(c.g[below(c.W)]) +
                    (c.gdt == DISDP_DT_BF16 ? 2 : 4) * below(c.n)));
                want = DISDP_ERR_ALIAS;
            } else if (entry == 1 || fused(entry)) {
                c.v = reinterpret_cast<float *>(const_cast<char *>(
                    static_cast<const char *>(c.g[below(c.W)]) + 2 * below(c.n)));
                want = DISDP_ERR_ALIAS;
            } else if (entry == 3) {
                c.ai = reinterpret_cast<int32_t *>(const_cast<char *>(
                    static_cast<const char *>(c.g[0]) + 2 * below(c.n)));
                want = DISDP_ERR_ALIAS;
            }
            break;
        case 8:  // two outputs overlapping
            if (entry == 1 || fused(entry)) {
                c.p = c.m + below(c.n);
                want = DISDP_ERR_ALIAS;
            }
            break;
        case 9:  // an int32 aggregate in fp32 mode
            if ((entry == 0 || fused(entry)) && c.mode == DISDP_AGG_FP32) {
                c.ai = reinterpret_cast<int32_t *>(fake(75));
                want = DISDP_ERR_INVALID_ARG;
            }
            break;
        case 10:  // memory the GPU cannot address
            g_addressable = false;
            want = DISDP_ERR_INVALID_ARG;
            break;
        case 12:  // step scalars missing or not 4-byte aligned
            if (entry == 4) {
                c.s = below(2) ? nullptr
                               : reinterpret_cast<const disdp_step_scalars_t *>(
                                     reinterpret_cast<const char *>(c.s) + 1 + below(3));
                want = DISDP_ERR_INVALID_ARG;
            }
            break;
        case 13:  // step scalars overlapping an output (the first or last bytes of one)
            if (entry == 4) {
                const int64_t nb = 4 * c.n;
                const int64_t at = below(2) ? 4 * below(c.n < 10 ? c.n : 10)
                                            : nb - 4 * (1 + below(c.n < 10 ? c.n : 10));
                float *out = below(2) ? c.p : c.v;
                c.s = reinterpret_cast<const disdp_step_scalars_t *>(
                    reinterpret_cast<const char *>(out) + at);
                want = DISDP_ERR_ALIAS;
            }
            break;
        default:  // empty shard: accepted, nothing launched
            c.n = 0;
            c.grads = below(2) ? nullptr : c.grads;
            want = DISDP_OK;
            break;
        }
        const int launches = g_launches;
        const disdp_status_t st = issue(c);
        g_addressable = true;
        CHECK(st == want, "entry %d kind %d: status %d, want %d (W=%d gdt=%d mode=%d n=%" PRId64
              ")", entry, kind, st, want, c.W, c.gdt, c.mode, c.n);
        const bool launched = g_launches != launches;
        CHECK(launched == (want == DISDP_OK && c.n > 0),
              "entry %d kind %d: launched=%d", entry, kind, launched);
        if (launched && fused(entry)) {
            // the constants travel by value, or only their address does
            const disdp::StepScalars zero{};
            if (entry == 4)
                CHECK(g_args.s_dev == reinterpret_cast<const disdp::StepScalars *>(c.s) &&
                          std::memcmp(&g_args.s, &zero, sizeof zero) == 0,
                      "aggregate_adam_dev: scalars not passed by address only");
            else
                CHECK(!g_args.s_dev && g_args.s.b1 == c.hp.beta1 && g_args.s.lr == c.hp.lr,
                      "aggregate_adam: scalars not passed by value");
        }
        CHECK(std::strlen(disdp_status_string(st)) > 0, "empty status string");
    }
    for (int s = -5; s < 10; ++s)
        CHECK(disdp_status_string(static_cast<disdp_status_t>(s)) != nullptr, "status %d", s);
}

// ---- valid calls: which kernel, head and advanced pointers ------------------------
void fuzz_alignment(int iters)
{
    for (int it = 0; it < iters; ++it) {
        const int W = 1 + static_cast<int>(below(16));
        const int gdt = static_cast<int>(below(2));
        const int gb = gdt == 1 ? 2 : 4;
        const int64_t n = 1 + (below(2) ? below(130) : below(1 << 24));
        // every array on a 1 KiB boundary plus a shared phase, then optionally
        // disturbed: a different phase mod 64 but the same mod 4, a different
        // phase mod 4, or an address not a multiple of the element size
        const int phase = static_cast<int>(below(64));
        const int disturb = static_cast<int>(below(5));
        const int victim = static_cast<int>(below(W + 4));
        int extra = 0;
        if (disturb == 1)
            extra = 4 * (1 + static_cast<int>(below(15)));
        else if (disturb == 2)
            extra = 1 + static_cast<int>(below(3));
        else if (disturb == 4)
            extra = 64 * (1 + static_cast<int>(below(3)));
        const void *g[disdp::kMaxW];
        for (int w = 0; w < W; ++w)
            g[w] = fake(w) + int64_t(gb) * (phase + (victim == w ? extra : 0)) +
                   (disturb == 3 && victim == w ? 1 : 0);
        auto arr = [&](int idx, int esz) {
            return fake(70 + idx) + int64_t(esz) * (phase + (victim == W + idx ? extra : 0)) +
                   (disturb == 3 && victim == W + idx ? 1 : 0);
        };
        float *p = reinterpret_cast<float *>(arr(0, 4));
        float *m = reinterpret_cast<float *>(arr(1, 4));
        float *v = reinterpret_cast<float *>(arr(2, 4));
        uint16_t *p16 = reinterpret_cast<uint16_t *>(arr(3, 2));
        const disdp_adamw_hparams_t hp = {1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 3, 1.0f};
        const disdp_status_t st = disdp_aggregate_adam(g, W, static_cast<disdp_dtype_t>(gdt), n,
                                                       DISDP_AGG_FP32, 0, p, m, v, p16, nullptr,
                                                       nullptr, &hp, nullptr);
        CHECK(st == DISDP_OK, "status %d", st);
        const disdp::LaunchArgs &a = g_args;
        // disturb 0: one shared phase mod 256 -> head to the 256-element
        // boundary; 4: same phase mod 64 only -> head to the 64-element one;
        // 1: same phase mod 4 only -> head to the 4-element one;
        // 2: no shared phase -> head taking p to a 256-element boundary, or
        // one element past it, such that every 2-byte array lands on a 4-byte
        // boundary (the fake bases are multiples of 4), else element kernel;
        // 3: an element not aligned to its size -> element kernel
        auto ph = [&](int idx) { return phase + (victim == idx ? extra : 0); };
        bool want_vec = disturb <= 1 || disturb == 4;
        int64_t want_head = disturb == 0   ? (256 - phase) % 256
                            : disturb == 4 ? (64 - phase) & 63
                            : disturb == 1 ? (4 - (phase & 3)) & 3
                                           : 0;
        if (disturb == 2) {
            const int h0 = (256 - ph(W) % 256) % 256;
            for (int h : {h0, (h0 + 1) % 256}) {
                bool ok = (ph(W + 3) + h) % 2 == 0;           // the bf16 copy
                for (int w = 0; w < W && gb == 2; ++w)
                    ok = ok && (ph(w) + h) % 2 == 0;          // bf16 contributions
                if (ok) {
                    want_vec = true;
                    want_head = h;
                    break;
                }
            }
        }
        if (want_head > n)
            want_head = n;
        CHECK(g_vec == want_vec, "vec %d want %d (disturb %d phase %d)", g_vec, want_vec, disturb,
              phase);
        CHECK(a.head == want_head, "head %d want %d (disturb %d phase %d n %" PRId64 ")", a.head,
              static_cast<int>(want_head), disturb, phase, n);
        CHECK(a.head + a.n == n, "head %d + n %" PRId64 " != %" PRId64, a.head, a.n, n);
        CHECK(a.p == p + a.head && a.m == m + a.head && a.v == v + a.head &&
                  a.p16 == p16 + a.head,
              "state pointers not advanced by the head");
        for (int w = 0; w < W; ++w)
            CHECK(a.g[w] == static_cast<const char *>(g[w]) + int64_t(a.head) * gb,
                  "contribution %d not advanced by the head", w);
        if (g_vec && a.n > 0 && disturb == 2) {
            const uintptr_t pe = reinterpret_cast<uintptr_t>(a.p) / 4 % 256;
            CHECK(pe == 0 || pe == 1, "p at element %d past a 256-element boundary",
                  static_cast<int>(pe));
            const void *all[] = {a.p, a.m, a.v, a.p16};
            for (const void *q : all)
                CHECK(reinterpret_cast<uintptr_t>(q) % 4 == 0, "state not on a 4-byte boundary");
            for (int w = 0; w < W; ++w)
                CHECK(reinterpret_cast<uintptr_t>(a.g[w]) % 4 == 0,
                      "contribution %d not on a 4-byte boundary", w);
        } else if (g_vec && a.n > 0) {
            const int gran = disturb == 0 ? 256 : disturb == 4 ? 64 : 4;
            for (int w = 0; w < W; ++w)
                CHECK((reinterpret_cast<uintptr_t>(a.g[w]) / gb) % gran == 0,
                      "contribution %d not on a %d-element boundary", w, gran);
            CHECK((reinterpret_cast<uintptr_t>(a.p) / 4) % gran == 0 &&
                      (reinterpret_cast<uintptr_t>(a.p16) / 2) % gran == 0,
                  "state not on a %d-element boundary", gran);
        }
    }
}

// ---- many tensors in one call ------------------------------------------------
// Random tensor lists (sizes, worker counts, per-tensor phases, some tensors
// empty, some with an element-misaligned array): every non-empty tensor must
// be launched exactly once, either in one batch slot -- with its head, its
// pointers advanced by the head onto 4-byte boundaries, its tile range
// ceil((n - head) / 4 / 64) (at least 1) -- or, when no head fits, on its own
// through the element kernel; batches within their capacity.  Then one
// error per call: an output overlapping a buffer of another tensor, a NULL
// pointer, a bad count.
char *addr(int64_t slot) { return reinterpret_cast<char *>((uintptr_t(1) << 46) + (uintptr_t(slot) << 34)); }

void fuzz_multi(int iters)
{
    for (int it = 0; it < iters; ++it) {
        const int W = below(4) ? 1 + static_cast<int>(below(16)) : 1 + static_cast<int>(below(64));
        const int mode = static_cast<int>(below(2));
        const int gdt = mode == DISDP_AGG_FIXED ? static_cast<int>(below(3)) : static_cast<int>(below(2));
        const int gb = gdt == DISDP_DT_BF16 ? 2 : 4;
        const int T = static_cast<int>(below(120));
        std::vector<int64_t> n(T);
        std::vector<const void *> g(static_cast<size_t>(T) * W);
        std::vector<float *> p(T), m(T), v(T);
        std::vector<uint16_t *> p16(T);
        std::vector<bool> odd(T, false);
        const bool copies = below(4) != 0;
        int64_t slot = 0;
        for (int j = 0; j < T; ++j) {
            n[j] = below(5) == 0 ? 0 : below(3) == 0 ? below(300) : below(1 << 20);
            const int64_t phase = below(3) ? below(512) : 0;
            const bool unrelated = below(4) == 0;
            odd[j] = below(16) == 0;
            for (int w = 0; w < W; ++w)
                g[static_cast<size_t>(j) * W + w] =
                    addr(slot++) + gb * (unrelated ? below(512) : phase) + (odd[j] && w == 0 ? 1 : 0);
            p[j] = reinterpret_cast<float *>(addr(slot++) + 4 * phase);
            m[j] = reinterpret_cast<float *>(addr(slot++) + 4 * (unrelated ? below(512) : phase));
            v[j] = reinterpret_cast<float *>(addr(slot++) + 4 * phase);
            p16[j] = copies && below(8) ? reinterpret_cast<uint16_t *>(addr(slot++) + 2 * phase)
                                        : nullptr;
        }
        const disdp_adamw_hparams_t hp = {1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 1 + below(1000), 1.0f};
        // the step's constants by value, or in (fake) device memory
        const bool dev = below(2) != 0;
        const disdp_step_scalars_t *sc =
            dev ? reinterpret_cast<const disdp_step_scalars_t *>(addr(slot++) + 4 * below(64))
                : nullptr;
        g_singles.clear();
        g_single_vec.clear();
        g_multis.clear();
        // one runtime query per allocation touched, however many arrays it holds
        std::set<uintptr_t> allocs;
        for (int j = 0; j < T; ++j) {
            if (n[j] == 0)
                continue;
            for (int w = 0; w < W; ++w)
                allocs.insert(reinterpret_cast<uintptr_t>(g[static_cast<size_t>(j) * W + w]) /
                              kAllocBytes);
            for (const void *q : {static_cast<const void *>(p[j]), static_cast<const void *>(m[j]),
                                  static_cast<const void *>(v[j]),
                                  static_cast<const void *>(copies ? p16[j] : nullptr)})
                if (q)
                    allocs.insert(reinterpret_cast<uintptr_t>(q) / kAllocBytes);
        }
        if (sc && !allocs.empty())
            allocs.insert(reinterpret_cast<uintptr_t>(sc) / kAllocBytes);
        const int queries = g_queries;
        const disdp_status_t st = disdp_aggregate_adam_multi(
            g.data(), W, static_cast<disdp_dtype_t>(gdt), T, n.data(),
            static_cast<disdp_agg_mode_t>(mode), 24, p.data(), m.data(), v.data(),
            copies ? p16.data() : nullptr, dev ? nullptr : &hp, sc, nullptr);
        CHECK(st == DISDP_OK, "multi: status %d (T=%d W=%d)", st, T, W);
        if (st != DISDP_OK)
            continue;
        // plus the single-tensor path's own checks of every array it is given
        int single_queries = 0;
        for (const disdp::LaunchArgs &a : g_singles)
            single_queries += W + 3 + (a.p16 ? 1 : 0) + (a.s_dev ? 1 : 0);
        CHECK(g_queries - queries <= static_cast<int>(allocs.size()) + single_queries,
              "multi: %d pointer queries for %zu allocations and %zu single launches",
              g_queries - queries, allocs.size(), g_singles.size());
        const int per = W + 4;
        const int cap = std::min(disdp::kMultiMaxTensors, disdp::kMultiMaxPtrs / per);
        std::vector<int> seen(T, 0);
        for (const disdp::MultiArgs &ma : g_multis) {
            CHECK(ma.count >= 1 && ma.count <= cap, "batch of %d tensors (cap %d)", ma.count, cap);
            CHECK(ma.W == W && ma.tile_start[0] == 0, "batch header");
            CHECK(dev ? (ma.s_dev == reinterpret_cast<const disdp::StepScalars *>(sc) && ma.s.b1 == 0.0f)
                      : (!ma.s_dev && ma.s.b1 == hp.beta1),
                  "batch step constants");
            for (int c = 0; c < ma.count; ++c) {
                const char *pp = static_cast<const char *>(ma.ptr[c * per + W]);
                const int h = ma.head[c];
                int j = -1;
                for (int k = 0; k < T; ++k)
                    if (n[k] > 0 && reinterpret_cast<const char *>(p[k]) + int64_t(h) * 4 == pp)
                        j = k;
                CHECK(j >= 0, "batch slot %d matches no tensor", c);
                if (j < 0)
                    continue;
                ++seen[j];
                CHECK(h >= 0 && h <= 255 && h <= n[j] && ma.n[c] + h == n[j],
                      "tensor %d: head %d n %lld of %lld", j, h, (long long)ma.n[c], (long long)n[j]);
                const int64_t tiles = std::max<int64_t>(1, ((ma.n[c] >> 2) + 63) / 64);
                CHECK(ma.tile_start[c + 1] - ma.tile_start[c] == tiles, "tensor %d: tiles", j);
                for (int w = 0; w < W; ++w) {
                    const char *q = static_cast<const char *>(ma.ptr[c * per + w]);
                    CHECK(q == static_cast<const char *>(g[static_cast<size_t>(j) * W + w]) + int64_t(h) * gb,
                          "tensor %d contribution %d not advanced by the head", j, w);
                    CHECK(ma.n[c] == 0 || reinterpret_cast<uintptr_t>(q) % 4 == 0,
                          "tensor %d contribution %d off a 4-byte boundary", j, w);
                }
                CHECK(ma.ptr[c * per + W + 1] == m[j] + h && ma.ptr[c * per + W + 2] == v[j] + h,
                      "tensor %d state not advanced", j);
                CHECK((p16[j] && copies) ? ma.ptr[c * per + W + 3] == p16[j] + h
                                         : ma.ptr[c * per + W + 3] == nullptr,
                      "tensor %d copy pointer", j);
            }
        }
        for (size_t i = 0; i < g_singles.size(); ++i) {
            const disdp::LaunchArgs &a = g_singles[i];
            int j = -1;
            for (int k = 0; k < T; ++k)
                if (n[k] > 0 && a.p == p[k] && a.n == n[k])
                    j = k;
            CHECK(j >= 0 && !g_single_vec[i], "single launch matches no tensor or is not elementwise");
            CHECK(a.s_dev == reinterpret_cast<const disdp::StepScalars *>(sc),
                  "single launch step constants");
            if (j >= 0)
                ++seen[j];
        }
        for (int j = 0; j < T; ++j)
            CHECK(seen[j] == (n[j] > 0 ? 1 : 0), "tensor %d launched %d times (n %lld)", j, seen[j],
                  (long long)n[j]);

        // one injected error
        int j0 = -1;
        for (int k = 0; k < T; ++k)
            if (n[k] > 8)
                j0 = k;
        if (j0 < 0)
            continue;
        const int kind = static_cast<int>(below(7));
        disdp_status_t want = DISDP_OK;
        std::vector<float *> p2 = p, m2 = m;
        std::vector<const void *> g2 = g;
        std::vector<int64_t> n2 = n;
        int T2 = T;
        if (kind == 0) {       // tensor j0's m inside another tensor's contribution
            int k1 = -1;
            for (int k = 0; k < T; ++k)
                if (k != j0 && n[k] > 0)
                    k1 = k;
            if (k1 < 0)
                continue;
            m2[j0] = reinterpret_cast<float *>(const_cast<char *>(
                static_cast<const char *>(g[static_cast<size_t>(k1) * W]) + gb * below(n[k1])));
            want = DISDP_ERR_ALIAS;
        } else if (kind == 1) {  // two tensors sharing a weight array
            int k1 = -1;
            for (int k = 0; k < T; ++k)
                if (k != j0 && n[k] > 0)
                    k1 = k;
            if (k1 < 0)
                continue;
            p2[j0] = p[k1];
            want = DISDP_ERR_ALIAS;
        } else if (kind == 2) {  // a NULL contribution
            g2[static_cast<size_t>(j0) * W + below(W)] = nullptr;
            want = DISDP_ERR_INVALID_ARG;
        } else if (kind == 3) {  // a negative count, or too many tensors
            if (below(2))
                n2[j0] = -1 - below(5);
            else
                T2 = 65537;
            want = DISDP_ERR_INVALID_ARG;
        } else if (kind == 4) {  // step constants: both sources, none, or misaligned
            want = DISDP_ERR_INVALID_ARG;
        } else if (kind == 5) {  // device step constants inside an output
            want = DISDP_ERR_ALIAS;
        } else {                 // one array of tensor j0 in memory the GPU cannot address
            char *bad = reinterpret_cast<char *>(kBadLo) + 4096 * below(1 << 20);
            const int which = static_cast<int>(below(W + 2));
            if (which < W)
                g2[static_cast<size_t>(j0) * W + which] = bad;
            else if (which == W)
                p2[j0] = reinterpret_cast<float *>(bad);
            else
                m2[j0] = reinterpret_cast<float *>(bad);
            want = DISDP_ERR_INVALID_ARG;
        }
        const disdp_adamw_hparams_t *hp2 = dev ? nullptr : &hp;
        const disdp_step_scalars_t *sc2 = sc;
        if (kind == 4) {
            const int how = static_cast<int>(below(3));
            const disdp_step_scalars_t *some =
                reinterpret_cast<const disdp_step_scalars_t *>(addr(slot++));
            hp2 = how == 0 ? &hp : nullptr;
            sc2 = how == 0 ? some
                  : how == 1 ? nullptr
                             : reinterpret_cast<const disdp_step_scalars_t *>(
                                   reinterpret_cast<const char *>(some) + 1 + below(3));
        } else if (kind == 5) {
            hp2 = nullptr;
            sc2 = reinterpret_cast<const disdp_step_scalars_t *>(
                reinterpret_cast<const char *>(v[j0]) + 4 * below(n[j0]));
        }
        const int before = g_launches;
        const disdp_status_t st2 = disdp_aggregate_adam_multi(
            g2.data(), W, static_cast<disdp_dtype_t>(gdt), T2, n2.data(),
            static_cast<disdp_agg_mode_t>(mode), 24, p2.data(), m2.data(), v.data(),
            copies ? p16.data() : nullptr, hp2, sc2, nullptr);
        CHECK(st2 == want, "multi error kind %d: status %d want %d", kind, st2, want);
        CHECK(g_launches == before, "multi error kind %d launched", kind);
    }
}

}  // namespace

int main()
{
    fuzz_layout(200000);
    fuzz_errors(200000);
    fuzz_alignment(100000);
    fuzz_multi(3000);
    if (failures) {
        std::printf("api_fuzz: %d failures\n", failures);
        return 1;
    }
    std::printf("api_fuzz: ok\n");
    return 0;
}
