// Standalone C++ user of libdisdp: the C ABI of include/disdp.h driven with
// the system HIP runtime and no PyTorch, its results compared bit for bit
// with the CPU oracle (liboracle.so, loaded with dlopen: the oracle is test
// infrastructure and is only ever linked by tests).
//
//   abi_driver <path to liboracle.so>
//
// Cases: the fused call over several steps (device and pinned host state),
// one HIP graph replayed across optimizer steps, the conversion feeding
// int32 contributions, a planned shard, virtual-memory-API memory, and the
// error paths.  Prints one line per case and "abi_driver: all ok" at the
// end; exits 1 on
// the first mismatch, 2 on a HIP or setup error.  Inputs are a splitmix64
// counter hash of (seed, index) mapped to [-1, 1) and scaled, with a sparse
// x100 outlier tail: the same host bytes go to the oracle and to the GPU.
#include <dlfcn.h>
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "disdp.h"

namespace {

// ---- oracle entry points (oracle/disdp_oracle.c) ---------------------------
using fused_fn = void (*)(const void *const *, int, int, int64_t, int, int, float *, float *,
                          float *, uint16_t *, float *, int32_t *, float, float, float, float,
                          float, int64_t, float);
using quant_fn = void (*)(const void *, int, int64_t, int, int32_t *);
fused_fn oracle_fused = nullptr;
quant_fn oracle_quantize_array = nullptr;

#define HIP_OK(expr)                                                                     \
    do {                                                                                 \
        hipError_t e_ = (expr);                                                          \
        if (e_ != hipSuccess) {                                                          \
            std::fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #expr,            \
                         hipGetErrorString(e_));                                         \
            std::exit(2);                                                                \
        }                                                                                \
    } while (0)

uint64_t mix(uint64_t x)
{
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

// Value i of stream `seed`: uniform in [-sigma, sigma), x100 on ~1% of i.
float draw(uint64_t seed, int64_t i, float sigma)
{
    const uint64_t h = mix(seed * 0x100000001B3ull + static_cast<uint64_t>(i));
    float u = static_cast<float>(static_cast<int32_t>(h >> 40) - (1 << 23)) / 8388608.0f;
    float x = u * sigma;
    if ((h & 0xff) < 3)
        x *= 100.0f;
    return x;
}

uint16_t bf16_bits(float x)  // round to nearest even (inputs are finite)
{
    uint32_t u;
    std::memcpy(&u, &x, 4);
    return static_cast<uint16_t>((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

int failures = 0;

bool same(const void *a, const void *b, size_t bytes, const char *what, const char *label)
{
    if (std::memcmp(a, b, bytes) == 0)
        return true;
    std::printf("MISMATCH %s: %s\n", label, what);
    ++failures;
    return false;
}

void expect(disdp_status_t got, disdp_status_t want, const char *label)
{
    if (got != want) {
        std::printf("MISMATCH %s: status %d (%s), expected %d\n", label, got,
                    disdp_status_string(got), want);
        ++failures;
    }
}

// W contribution buffers on the host: fp32 values, or their bf16 bits.
struct HostGrads {
    int W, gdtype;
    int64_t n;
    std::vector<std::vector<float>> f;
    std::vector<std::vector<uint16_t>> h;
    HostGrads(int W_, int gdtype_, int64_t n_, uint64_t seed, float sigma)
        : W(W_), gdtype(gdtype_), n(n_)
    {
        for (int w = 0; w < W; ++w) {
            std::vector<float> x(n);
            for (int64_t i = 0; i < n; ++i)
                x[i] = draw(seed * 131 + w, i, sigma);
            if (gdtype == DISDP_DT_BF16) {
                std::vector<uint16_t> b(n);
                for (int64_t i = 0; i < n; ++i)
                    b[i] = bf16_bits(x[i]);
                h.push_back(b);
            } else {
                f.push_back(x);
            }
        }
    }
    const void *ptr(int w) const
    {
        return gdtype == DISDP_DT_BF16 ? static_cast<const void *>(h[w].data())
                                       : static_cast<const void *>(f[w].data());
    }
    size_t bytes() const { return static_cast<size_t>(n) * (gdtype == DISDP_DT_BF16 ? 2 : 4); }
};

struct Hp {
    float lr = 1e-4f, b1 = 0.9f, b2 = 0.95f, eps = 1e-8f, wd = 0.1f;
};

disdp_adamw_hparams_t hparams(const Hp &h, int64_t t)
{
    disdp_adamw_hparams_t p;
    p.lr = h.lr;
    p.beta1 = h.b1;
    p.beta2 = h.b2;
    p.eps = h.eps;
    p.weight_decay = h.wd;
    p.step = t;
    p.grad_scale = 1.0f;
    return p;
}

// One fused case: `steps` steps with fresh contributions, state in device
// memory (or in mapped pinned host memory when host_state), on a created
// stream; every output compared with the oracle after every step.
void fused_case(const char *label, int W, int gdtype, int64_t n, int mode, int k, int steps,
                bool host_state, bool want_agg)
{
    hipStream_t s;
    HIP_OK(hipStreamCreate(&s));
    std::vector<float> p(n), m(n), v(n);
    for (int64_t i = 0; i < n; ++i) {
        p[i] = draw(7001, i, 0.02f);
        m[i] = draw(7002, i, 1e-4f);
        const float r = draw(7003, i, 1e-4f);
        v[i] = r * r;
    }
    const size_t gb = static_cast<size_t>(n) * (gdtype == DISDP_DT_BF16 ? 2 : 4);
    std::vector<void *> dg(W);
    for (int w = 0; w < W; ++w)
        HIP_OK(hipMalloc(&dg[w], gb));
    float *dp, *dm, *dv, *daf = nullptr;
    uint16_t *d16;
    int32_t *dai = nullptr;
    const size_t fb = static_cast<size_t>(n) * 4;
    if (host_state) {
        HIP_OK(hipHostMalloc(reinterpret_cast<void **>(&dp), fb, hipHostMallocDefault));
        HIP_OK(hipHostMalloc(reinterpret_cast<void **>(&dm), fb, hipHostMallocDefault));
        HIP_OK(hipHostMalloc(reinterpret_cast<void **>(&dv), fb, hipHostMallocDefault));
        HIP_OK(hipHostMalloc(reinterpret_cast<void **>(&d16), n * 2, hipHostMallocDefault));
    } else {
        HIP_OK(hipMalloc(&dp, fb));
        HIP_OK(hipMalloc(&dm, fb));
        HIP_OK(hipMalloc(&dv, fb));
        HIP_OK(hipMalloc(&d16, n * 2));
    }
    if (want_agg) {
        HIP_OK(hipMalloc(&daf, fb));
        if (mode == DISDP_AGG_FIXED)
            HIP_OK(hipMalloc(&dai, fb));
    }
    HIP_OK(hipMemcpy(dp, p.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dm, m.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dv, v.data(), fb, hipMemcpyDefault));

    std::vector<uint16_t> want16(n), got16(n);
    std::vector<float> gp(n), gm(n), gv(n), waf(n), gaf(n);
    std::vector<int32_t> wai(n), gai(n);
    Hp h;
    bool ok = true;
    for (int t = 1; t <= steps && ok; ++t) {
        HostGrads g(W, gdtype, n, 1000 + t, 1e-4f);
        std::vector<const void *> hp_ptrs(W);
        for (int w = 0; w < W; ++w) {
            HIP_OK(hipMemcpy(dg[w], g.ptr(w), gb, hipMemcpyDefault));
            hp_ptrs[w] = g.ptr(w);
        }
        const disdp_adamw_hparams_t hp = hparams(h, t);
        expect(disdp_aggregate_adam(dg.data(), W, static_cast<disdp_dtype_t>(gdtype), n,
                                    static_cast<disdp_agg_mode_t>(mode), k, dp, dm, dv, d16,
                                    daf, dai, &hp, s),
               DISDP_OK, label);
        HIP_OK(hipStreamSynchronize(s));
        oracle_fused(hp_ptrs.data(), W, gdtype, n, mode, k, p.data(), m.data(), v.data(),
                     want16.data(), want_agg ? waf.data() : nullptr,
                     (want_agg && mode == DISDP_AGG_FIXED) ? wai.data() : nullptr, h.lr, h.b1,
                     h.b2, h.eps, h.wd, t, 1.0f);
        HIP_OK(hipMemcpy(gp.data(), dp, fb, hipMemcpyDefault));
        HIP_OK(hipMemcpy(gm.data(), dm, fb, hipMemcpyDefault));
        HIP_OK(hipMemcpy(gv.data(), dv, fb, hipMemcpyDefault));
        HIP_OK(hipMemcpy(got16.data(), d16, n * 2, hipMemcpyDefault));
        ok = same(gp.data(), p.data(), fb, "p", label) && ok;
        ok = same(gm.data(), m.data(), fb, "m", label) && ok;
        ok = same(gv.data(), v.data(), fb, "v", label) && ok;
        ok = same(got16.data(), want16.data(), n * 2, "p16", label) && ok;
        if (want_agg) {
            HIP_OK(hipMemcpy(gaf.data(), daf, fb, hipMemcpyDefault));
            ok = same(gaf.data(), waf.data(), fb, "agg_f32", label) && ok;
            if (mode == DISDP_AGG_FIXED) {
                HIP_OK(hipMemcpy(gai.data(), dai, fb, hipMemcpyDefault));
                ok = same(gai.data(), wai.data(), fb, "agg_i32", label) && ok;
            }
        }
    }
    std::printf("%s %s: W=%d n=%lld steps=%d\n", ok ? "ok" : "FAIL", label, W,
                static_cast<long long>(n), steps);
    for (int w = 0; w < W; ++w)
        HIP_OK(hipFree(dg[w]));
    if (host_state) {
        HIP_OK(hipHostFree(dp));
        HIP_OK(hipHostFree(dm));
        HIP_OK(hipHostFree(dv));
        HIP_OK(hipHostFree(d16));
    } else {
        HIP_OK(hipFree(dp));
        HIP_OK(hipFree(dm));
        HIP_OK(hipFree(dv));
        HIP_OK(hipFree(d16));
    }
    if (daf)
        HIP_OK(hipFree(daf));
    if (dai)
        HIP_OK(hipFree(dai));
    HIP_OK(hipStreamDestroy(s));
}

// One HIP graph for every optimizer step: a copy node refreshes the step's
// constants (disdp_step_scalars, written into pinned host memory before each
// replay) in device memory, then disdp_aggregate_adam_dev reads them.  Fresh
// contributions are copied in eagerly between replays; every step is
// compared with the oracle.
void graph_case(const char *label, int W, int gdtype, int64_t n, int mode, int k, int steps)
{
    hipStream_t s;
    HIP_OK(hipStreamCreate(&s));
    std::vector<float> p(n), m(n), v(n);
    for (int64_t i = 0; i < n; ++i) {
        p[i] = draw(7101, i, 0.02f);
        m[i] = draw(7102, i, 1e-4f);
        const float r = draw(7103, i, 1e-4f);
        v[i] = r * r;
    }
    const size_t gb = static_cast<size_t>(n) * (gdtype == DISDP_DT_BF16 ? 2 : 4);
    const size_t fb = static_cast<size_t>(n) * 4;
    std::vector<void *> dg(W);
    for (int w = 0; w < W; ++w)
        HIP_OK(hipMalloc(&dg[w], gb));
    float *dp, *dm, *dv;
    uint16_t *d16;
    disdp_step_scalars_t *dsc, *hsc;
    HIP_OK(hipMalloc(&dp, fb));
    HIP_OK(hipMalloc(&dm, fb));
    HIP_OK(hipMalloc(&dv, fb));
    HIP_OK(hipMalloc(&d16, n * 2));
    HIP_OK(hipMalloc(&dsc, sizeof *dsc));
    HIP_OK(hipHostMalloc(reinterpret_cast<void **>(&hsc), sizeof *hsc, hipHostMallocDefault));
    HIP_OK(hipMemcpy(dp, p.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dm, m.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dv, v.data(), fb, hipMemcpyDefault));

    hipGraph_t graph;
    hipGraphExec_t exec;
    HIP_OK(hipStreamBeginCapture(s, hipStreamCaptureModeGlobal));
    HIP_OK(hipMemcpyAsync(dsc, hsc, sizeof *dsc, hipMemcpyHostToDevice, s));
    const disdp_status_t cst =
        disdp_aggregate_adam_dev(dg.data(), W, static_cast<disdp_dtype_t>(gdtype), n,
                                 static_cast<disdp_agg_mode_t>(mode), k, dp, dm, dv, d16,
                                 nullptr, nullptr, dsc, s);
    HIP_OK(hipStreamEndCapture(s, &graph));
    expect(cst, DISDP_OK, label);
    HIP_OK(hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0));

    std::vector<uint16_t> want16(n), got16(n);
    std::vector<float> gp(n), gm(n), gv(n);
    Hp h;
    bool ok = cst == DISDP_OK;
    for (int t = 1; t <= steps && ok; ++t) {
        HostGrads g(W, gdtype, n, 2000 + t, 1e-4f);
        std::vector<const void *> hp_ptrs(W);
        for (int w = 0; w < W; ++w) {
            HIP_OK(hipMemcpy(dg[w], g.ptr(w), gb, hipMemcpyDefault));
            hp_ptrs[w] = g.ptr(w);
        }
        const disdp_adamw_hparams_t hp = hparams(h, t);
        expect(disdp_step_scalars(&hp, hsc), DISDP_OK, label);
        HIP_OK(hipGraphLaunch(exec, s));
        HIP_OK(hipStreamSynchronize(s));
        oracle_fused(hp_ptrs.data(), W, gdtype, n, mode, k, p.data(), m.data(), v.data(),
                     want16.data(), nullptr, nullptr, h.lr, h.b1, h.b2, h.eps, h.wd, t, 1.0f);
        HIP_OK(hipMemcpy(gp.data(), dp, fb, hipMemcpyDefault));
        HIP_OK(hipMemcpy(gm.data(), dm, fb, hipMemcpyDefault));
        HIP_OK(hipMemcpy(gv.data(), dv, fb, hipMemcpyDefault));
        HIP_OK(hipMemcpy(got16.data(), d16, n * 2, hipMemcpyDefault));
        ok = same(gp.data(), p.data(), fb, "p", label) && ok;
        ok = same(gm.data(), m.data(), fb, "m", label) && ok;
        ok = same(gv.data(), v.data(), fb, "v", label) && ok;
        ok = same(got16.data(), want16.data(), n * 2, "p16", label) && ok;
    }
    std::printf("%s %s: W=%d n=%lld replays=%d\n", ok ? "ok" : "FAIL", label, W,
                static_cast<long long>(n), steps);
    HIP_OK(hipGraphExecDestroy(exec));
    HIP_OK(hipGraphDestroy(graph));
    for (int w = 0; w < W; ++w)
        HIP_OK(hipFree(dg[w]));
    HIP_OK(hipFree(dp));
    HIP_OK(hipFree(dm));
    HIP_OK(hipFree(dv));
    HIP_OK(hipFree(d16));
    HIP_OK(hipFree(dsc));
    HIP_OK(hipHostFree(hsc));
    HIP_OK(hipStreamDestroy(s));
}

// Many tensors in separate buffers through one disdp_aggregate_adam_multi
// call (sizes from empty to a few tiles plus ragged tails, one tensor at an
// odd element offset), every tensor compared with the oracle.
void multi_case(int W, int gdtype, int mode, int k)
{
    const char *label = "multi-tensor call";
    hipStream_t s;
    HIP_OK(hipStreamCreate(&s));
    const int64_t sizes[] = {0, 1, 3, 4, 257, 1000, 4099, 65541, 7, 300007, 2, 256};
    const int T = static_cast<int>(sizeof sizes / sizeof sizes[0]);
    const size_t eb = gdtype == DISDP_DT_BF16 ? 2 : 4;
    std::vector<void *> allocs;
    std::vector<const void *> g(static_cast<size_t>(T) * W);
    std::vector<float *> dp(T), dm(T), dv(T);
    std::vector<uint16_t *> d16(T);
    std::vector<std::vector<float>> p(T), m(T), v(T);
    std::vector<HostGrads> hg;
    for (int j = 0; j < T; ++j) {
        const int64_t n = sizes[j];
        const int off = j == 5 ? 3 : 0;   // tensor 5 starts 3 elements into its buffers
        hg.emplace_back(W, gdtype, n, 3000 + j, 1e-4f);
        for (int w = 0; w < W; ++w) {
            void *b;
            HIP_OK(hipMalloc(&b, (n + off + 1) * eb));
            allocs.push_back(b);
            char *q = static_cast<char *>(b) + off * eb;
            HIP_OK(hipMemcpy(q, hg[j].ptr(w), n * eb, hipMemcpyDefault));
            g[static_cast<size_t>(j) * W + w] = q;
        }
        p[j].resize(n);
        m[j].resize(n);
        v[j].resize(n);
        for (int64_t i = 0; i < n; ++i) {
            p[j][i] = draw(7201 + j, i, 0.02f);
            m[j][i] = draw(7301 + j, i, 1e-4f);
            const float r = draw(7401 + j, i, 1e-4f);
            v[j][i] = r * r;
        }
        float **outs[] = {&dp[j], &dm[j], &dv[j]};
        std::vector<float> *src[] = {&p[j], &m[j], &v[j]};
        for (int a = 0; a < 3; ++a) {
            void *b;
            HIP_OK(hipMalloc(&b, (n + off + 1) * 4));
            allocs.push_back(b);
            *outs[a] = static_cast<float *>(b) + off;
            HIP_OK(hipMemcpy(*outs[a], src[a]->data(), n * 4, hipMemcpyDefault));
        }
        void *b;
        HIP_OK(hipMalloc(&b, (n + off + 1) * 2));
        allocs.push_back(b);
        d16[j] = static_cast<uint16_t *>(b) + off;
    }
    Hp h;
    const disdp_adamw_hparams_t hp = hparams(h, 4);
    expect(disdp_aggregate_adam_multi(g.data(), W, static_cast<disdp_dtype_t>(gdtype), T, sizes,
                                      static_cast<disdp_agg_mode_t>(mode), k, dp.data(),
                                      dm.data(), dv.data(), d16.data(), &hp, nullptr, s),
           DISDP_OK, label);
    HIP_OK(hipStreamSynchronize(s));
    bool ok = true;
    for (int j = 0; j < T && ok; ++j) {
        const int64_t n = sizes[j];
        if (n == 0)
            continue;
        std::vector<const void *> hp_ptrs(W);
        for (int w = 0; w < W; ++w)
            hp_ptrs[w] = hg[j].ptr(w);
        std::vector<uint16_t> want16(n), got16(n);
        std::vector<float> gp(n), gm(n), gv(n);
        oracle_fused(hp_ptrs.data(), W, gdtype, n, mode, k, p[j].data(), m[j].data(),
                     v[j].data(), want16.data(), nullptr, nullptr, h.lr, h.b1, h.b2, h.eps, h.wd,
                     4, 1.0f);
        HIP_OK(hipMemcpy(gp.data(), dp[j], n * 4, hipMemcpyDefault));
        HIP_OK(hipMemcpy(gm.data(), dm[j], n * 4, hipMemcpyDefault));
        HIP_OK(hipMemcpy(gv.data(), dv[j], n * 4, hipMemcpyDefault));
        HIP_OK(hipMemcpy(got16.data(), d16[j], n * 2, hipMemcpyDefault));
        ok = same(gp.data(), p[j].data(), n * 4, "p", label) && ok;
        ok = same(gm.data(), m[j].data(), n * 4, "m", label) && ok;
        ok = same(gv.data(), v[j].data(), n * 4, "v", label) && ok;
        ok = same(got16.data(), want16.data(), n * 2, "p16", label) && ok;
    }
    std::printf("%s %s: T=%d W=%d gdtype=%d mode=%d\n", ok ? "ok" : "FAIL", label, T, W, gdtype,
                mode);
    for (void *b : allocs)
        HIP_OK(hipFree(b));
    HIP_OK(hipStreamDestroy(s));
}

// The worker-side conversion, then the aggregation of int32 contributions,
// against the oracle's conversion and fixed-point aggregation of the floats.
void quantize_case(int W, int64_t n, int k)
{
    const char *label = "quantize+int32 contributions";
    HostGrads g(W, DISDP_DT_F32, n, 4242, 1e-4f);
    const size_t b = static_cast<size_t>(n) * 4;
    std::vector<void *> df(W), dq(W);
    std::vector<const void *> hf(W);
    std::vector<int32_t> want(n), got(n);
    bool ok = true;
    for (int w = 0; w < W; ++w) {
        HIP_OK(hipMalloc(&df[w], b));
        HIP_OK(hipMalloc(&dq[w], b));
        HIP_OK(hipMemcpy(df[w], g.ptr(w), b, hipMemcpyDefault));
        hf[w] = g.ptr(w);
        expect(disdp_quantize(df[w], DISDP_DT_F32, n, k, static_cast<int32_t *>(dq[w]), 0),
               DISDP_OK, label);
        HIP_OK(hipDeviceSynchronize());
        oracle_quantize_array(g.ptr(w), DISDP_DT_F32, n, k, want.data());
        HIP_OK(hipMemcpy(got.data(), dq[w], b, hipMemcpyDefault));
        ok = same(got.data(), want.data(), b, "quantized contribution", label) && ok;
    }
    int32_t *dai;
    HIP_OK(hipMalloc(&dai, b));
    expect(disdp_aggregate(dq.data(), W, DISDP_DT_I32, n, DISDP_AGG_FIXED, k, nullptr, dai, 0),
           DISDP_OK, label);
    HIP_OK(hipDeviceSynchronize());
    std::vector<float> p(n, 0.0f), m(n, 0.0f), v(n, 0.0f);
    std::vector<uint16_t> p16(n);
    oracle_fused(hf.data(), W, DISDP_DT_F32, n, DISDP_AGG_FIXED, k, p.data(), m.data(), v.data(),
                 p16.data(), nullptr, want.data(), 1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 1, 1.0f);
    HIP_OK(hipMemcpy(got.data(), dai, b, hipMemcpyDefault));
    ok = same(got.data(), want.data(), b, "int32 aggregate", label) && ok;
    std::printf("%s %s: W=%d n=%lld k=%d\n", ok ? "ok" : "FAIL", label, W,
                static_cast<long long>(n), k);
    for (int w = 0; w < W; ++w) {
        HIP_OK(hipFree(df[w]));
        HIP_OK(hipFree(dq[w]));
    }
    HIP_OK(hipFree(dai));
}

// The placement planner with one hipMalloc slab: offsets inside the slab,
// then a fused step on the views against the oracle.
void layout_case(int W, int64_t n)
{
    const char *label = "shard layout slab";
    std::vector<int64_t> off(W + 6);
    int64_t total = 0;
    expect(disdp_shard_layout(n, W, DISDP_DT_F32, DISDP_LAYOUT_BF16_COPY, off.data(), &total),
           DISDP_OK, label);
    char *slab;
    HIP_OK(hipMalloc(&slab, total));
    HostGrads g(W, DISDP_DT_F32, n, 5151, 1e-3f);
    std::vector<const void *> dg(W), hg(W);
    const size_t fb = static_cast<size_t>(n) * 4;
    for (int w = 0; w < W; ++w) {
        dg[w] = slab + off[w];
        hg[w] = g.ptr(w);
        HIP_OK(hipMemcpy(slab + off[w], g.ptr(w), fb, hipMemcpyDefault));
    }
    std::vector<float> p(n), m(n, 0.0f), v(n, 0.0f), got(n);
    std::vector<uint16_t> p16(n), g16(n);
    for (int64_t i = 0; i < n; ++i)
        p[i] = draw(6001, i, 0.02f);
    float *dp = reinterpret_cast<float *>(slab + off[W]);
    float *dm = reinterpret_cast<float *>(slab + off[W + 1]);
    float *dv = reinterpret_cast<float *>(slab + off[W + 2]);
    uint16_t *d16 = reinterpret_cast<uint16_t *>(slab + off[W + 3]);
    HIP_OK(hipMemcpy(dp, p.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dm, m.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dv, v.data(), fb, hipMemcpyDefault));
    Hp h;
    const disdp_adamw_hparams_t hp = hparams(h, 1);
    expect(disdp_aggregate_adam(dg.data(), W, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, dp, dm, dv,
                                d16, nullptr, nullptr, &hp, 0),
           DISDP_OK, label);
    HIP_OK(hipDeviceSynchronize());
    oracle_fused(hg.data(), W, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, p.data(), m.data(), v.data(),
                 p16.data(), nullptr, nullptr, h.lr, h.b1, h.b2, h.eps, h.wd, 1, 1.0f);
    bool ok = true;
    HIP_OK(hipMemcpy(got.data(), dp, fb, hipMemcpyDefault));
    ok = same(got.data(), p.data(), fb, "p", label) && ok;
    HIP_OK(hipMemcpy(got.data(), dv, fb, hipMemcpyDefault));
    ok = same(got.data(), v.data(), fb, "v", label) && ok;
    HIP_OK(hipMemcpy(g16.data(), d16, n * 2, hipMemcpyDefault));
    ok = same(g16.data(), p16.data(), n * 2, "p16", label) && ok;
    std::printf("%s %s: W=%d n=%lld total=%lld bytes\n", ok ? "ok" : "FAIL", label, W,
                static_cast<long long>(n), static_cast<long long>(total));
    HIP_OK(hipFree(slab));
}

// Memory from the virtual-memory API (one physical allocation mapped at a
// reserved range, as VMM-based allocators hand it out): accepted by the
// pointer checks and computed like any device memory.
void vmm_case(int W, int64_t n)
{
    const char *label = "virtual-memory-API allocation";
    hipMemAllocationProp prop = {};
    prop.type = hipMemAllocationTypePinned;
    prop.location.type = hipMemLocationTypeDevice;
    HIP_OK(hipGetDevice(&prop.location.id));
    size_t gran = 0;
    HIP_OK(hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityMinimum));
    std::vector<int64_t> off(W + 6);
    int64_t total = 0;
    expect(disdp_shard_layout(n, W, DISDP_DT_F32, DISDP_LAYOUT_BF16_COPY, off.data(), &total),
           DISDP_OK, label);
    const size_t size = (static_cast<size_t>(total) + gran - 1) / gran * gran;
    hipMemGenericAllocationHandle_t h;
    HIP_OK(hipMemCreate(&h, size, &prop, 0));
    void *va = nullptr;
    HIP_OK(hipMemAddressReserve(&va, size, 0, nullptr, 0));
    HIP_OK(hipMemMap(va, size, 0, h, 0));
    hipMemAccessDesc acc = {};
    acc.location = prop.location;
    acc.flags = hipMemAccessFlagsProtReadWrite;
    HIP_OK(hipMemSetAccess(va, size, &acc, 1));
    char *slab = static_cast<char *>(va);
    HostGrads g(W, DISDP_DT_F32, n, 6262, 1e-3f);
    std::vector<const void *> dg(W), hg(W);
    const size_t fb = static_cast<size_t>(n) * 4;
    for (int w = 0; w < W; ++w) {
        dg[w] = slab + off[w];
        hg[w] = g.ptr(w);
        HIP_OK(hipMemcpy(slab + off[w], g.ptr(w), fb, hipMemcpyDefault));
    }
    std::vector<float> p(n), m(n, 0.0f), v(n, 0.0f), got(n);
    std::vector<uint16_t> p16(n), g16(n);
    for (int64_t i = 0; i < n; ++i)
        p[i] = draw(6002, i, 0.02f);
    float *dp = reinterpret_cast<float *>(slab + off[W]);
    float *dm = reinterpret_cast<float *>(slab + off[W + 1]);
    float *dv = reinterpret_cast<float *>(slab + off[W + 2]);
    uint16_t *d16 = reinterpret_cast<uint16_t *>(slab + off[W + 3]);
    HIP_OK(hipMemcpy(dp, p.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dm, m.data(), fb, hipMemcpyDefault));
    HIP_OK(hipMemcpy(dv, v.data(), fb, hipMemcpyDefault));
    Hp hh;
    const disdp_adamw_hparams_t hp = hparams(hh, 2);
    expect(disdp_aggregate_adam(dg.data(), W, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, dp, dm, dv,
                                d16, nullptr, nullptr, &hp, 0),
           DISDP_OK, label);
    HIP_OK(hipDeviceSynchronize());
    oracle_fused(hg.data(), W, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, p.data(), m.data(), v.data(),
                 p16.data(), nullptr, nullptr, hh.lr, hh.b1, hh.b2, hh.eps, hh.wd, 2, 1.0f);
    bool ok = true;
    HIP_OK(hipMemcpy(got.data(), dp, fb, hipMemcpyDefault));
    ok = same(got.data(), p.data(), fb, "p", label) && ok;
    HIP_OK(hipMemcpy(got.data(), dm, fb, hipMemcpyDefault));
    ok = same(got.data(), m.data(), fb, "m", label) && ok;
    HIP_OK(hipMemcpy(g16.data(), d16, n * 2, hipMemcpyDefault));
    ok = same(g16.data(), p16.data(), n * 2, "p16", label) && ok;
    std::printf("%s %s: W=%d n=%lld mapped %zu bytes\n", ok ? "ok" : "FAIL", label, W,
                static_cast<long long>(n), size);
    HIP_OK(hipMemUnmap(va, size));
    HIP_OK(hipMemAddressFree(va, size));
    HIP_OK(hipMemRelease(h));
}

// Argument errors a C caller can make; none of them launches anything.
void error_case()
{
    const char *label = "argument errors";
    const int64_t n = 4096;
    float *a, *b;
    HIP_OK(hipMalloc(&a, n * 4));
    HIP_OK(hipMalloc(&b, n * 4));
    std::vector<float> pageable(n, 0.0f);
    const void *g1[1] = {a};
    const void *gp[1] = {pageable.data()};
    disdp_adamw_hparams_t hp = hparams(Hp(), 1);
    // an output that is also an input
    expect(disdp_aggregate(g1, 1, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, a, nullptr, 0),
           DISDP_ERR_ALIAS, label);
    // pageable host memory is refused before any launch
    expect(disdp_aggregate(gp, 1, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, b, nullptr, 0),
           DISDP_ERR_INVALID_ARG, label);
    // an int32 aggregate in fp32 mode; int32 contributions in fp32 mode
    expect(disdp_aggregate(g1, 1, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, b,
                           reinterpret_cast<int32_t *>(b), 0),
           DISDP_ERR_INVALID_ARG, label);
    expect(disdp_aggregate(g1, 1, DISDP_DT_I32, n, DISDP_AGG_FP32, 0, b, nullptr, 0),
           DISDP_ERR_UNSUPPORTED, label);
    // beta1 = 1 and step 0
    hp.beta1 = 1.0f;
    expect(disdp_adam_step(a, b, b, b, nullptr, n, &hp, 0), DISDP_ERR_INVALID_ARG, label);
    hp = hparams(Hp(), 0);
    float *c;
    HIP_OK(hipMalloc(&c, n * 4 * 3));
    expect(disdp_adam_step(a, c, c + n, c + 2 * n, nullptr, n, &hp, 0), DISDP_ERR_INVALID_ARG,
           label);
    // n == 0 needs no pointers
    hp = hparams(Hp(), 1);
    expect(disdp_aggregate_adam(nullptr, 1, DISDP_DT_F32, 0, DISDP_AGG_FP32, 0, nullptr, nullptr,
                                nullptr, nullptr, nullptr, nullptr, &hp, 0),
           DISDP_OK, label);
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipGetLastError());  // the refused pointer query left no sticky error
    // An error the caller has not read yet survives a call whose pointer
    // query fails: make one on the host (an out-of-range device index; no
    // device work), let the library refuse pageable memory, and the error
    // is still reported, then cleared by reading it.
    int count = 0;
    HIP_OK(hipGetDeviceCount(&count));
    if (hipSetDevice(count + 7) == hipSuccess) {
        std::printf("FAIL %s: device %d accepted\n", label, count + 7);
        ++failures;
    }
    expect(disdp_aggregate(gp, 1, DISDP_DT_F32, n, DISDP_AGG_FP32, 0, b, nullptr, 0),
           DISDP_ERR_INVALID_ARG, label);
    if (hipGetLastError() == hipSuccess) {
        std::printf("FAIL %s: a pending error was cleared by the library\n", label);
        ++failures;
    }
    HIP_OK(hipGetLastError());  // read once: gone
    std::printf("%s %s\n", failures ? "FAIL" : "ok", label);
    HIP_OK(hipFree(a));
    HIP_OK(hipFree(b));
    HIP_OK(hipFree(c));
}

}  // namespace

int main(int argc, char **argv)
{
    if (argc != 2) {
        std::fprintf(stderr, "usage: %s <liboracle.so>\n", argv[0]);
        return 2;
    }
    void *o = dlopen(argv[1], RTLD_NOW | RTLD_LOCAL);
    if (!o) {
        std::fprintf(stderr, "dlopen %s: %s\n", argv[1], dlerror());
        return 2;
    }
    oracle_fused = reinterpret_cast<fused_fn>(dlsym(o, "oracle_fused"));
    oracle_quantize_array = reinterpret_cast<quant_fn>(dlsym(o, "oracle_quantize_array"));
    if (!oracle_fused || !oracle_quantize_array) {
        std::fprintf(stderr, "oracle symbols missing\n");
        return 2;
    }
    int dev = 0;
    HIP_OK(hipGetDevice(&dev));
    std::printf("abi_driver: device %d\n", dev);
    std::fflush(stdout);
    fused_case("fp32 W=8 device state", 8, DISDP_DT_F32, 1000003, DISDP_AGG_FP32, 0, 3, false,
               true);
    std::fflush(stdout);
    fused_case("fixed bf16 W=5 device state", 5, DISDP_DT_BF16, 777777, DISDP_AGG_FIXED, 24, 2,
               false, true);
    std::fflush(stdout);
    fused_case("fp32 W=3 pinned host state", 3, DISDP_DT_F32, 300007, DISDP_AGG_FP32, 0, 2, true,
               false);
    std::fflush(stdout);
    // the launch shape for a GPU shared with compute kernels, chosen through
    // the environment on each call: same results, checked against the oracle
    setenv("DISDP_LAUNCH_SHAPE", "shared", 1);
    fused_case("shared shape fp32 W=8 device state", 8, DISDP_DT_F32, 1000003, DISDP_AGG_FP32,
               0, 2, false, true);
    std::fflush(stdout);
    fused_case("shared shape fixed W=24 device state", 24, DISDP_DT_F32, 300007,
               DISDP_AGG_FIXED, 24, 2, false, true);
    std::fflush(stdout);
    unsetenv("DISDP_LAUNCH_SHAPE");
    graph_case("graph replay fp32 W=6", 6, DISDP_DT_F32, 500009, DISDP_AGG_FP32, 0, 4);
    std::fflush(stdout);
    graph_case("graph replay fixed bf16 W=13", 13, DISDP_DT_BF16, 200003, DISDP_AGG_FIXED, 24, 3);
    std::fflush(stdout);
    multi_case(4, DISDP_DT_F32, DISDP_AGG_FP32, 0);
    std::fflush(stdout);
    multi_case(9, DISDP_DT_BF16, DISDP_AGG_FIXED, 24);
    std::fflush(stdout);
    quantize_case(6, 500009, 24);
    std::fflush(stdout);
    layout_case(4, 1 << 20);
    std::fflush(stdout);
    vmm_case(3, 3 << 19);
    std::fflush(stdout);
    error_case();
    if (failures) {
        std::printf("abi_driver: %d mismatches\n", failures);
        return 1;
    }
    std::printf("abi_driver: all ok\n");
    return 0;
}
