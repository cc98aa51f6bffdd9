/*
 * disdp_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU statement of what the parameter-server
 * hot path of DisDP computes for one model shard (arXiv 2409.00918):
 *
 *   1. the W-way aggregation of the workers' gradient contributions that the
 *      SmartSwitch performs in the network (Section III-A "Overall
 *      Architecture"; Section III-C "Packet Transport Procedure"), either as a
 *      float sum or in the integer format the SmartNIC format-conversion unit
 *      produces for the switch (Section III-B "Format Conversion Unit");
 *   2. the mixed-precision Adam step the parameter server runs on the
 *      aggregated gradient: 2-byte gradient + 12-byte model states in,
 *      12-byte model states + 2-byte parameter copy out (Section III-D,
 *      "Backward Stage", step 5, and Table III).
 *
 * Only tests/, the smoke entry point and the CPU-baseline leg of the
 * benchmark may load this file's library.  It shares no code, header, table
 * or constant with the HIP path, and nothing in the product links it.
 *
 * Arithmetic: IEEE-754 binary32, one rounding per written operation, round to
 * nearest even, no contraction into fused multiply-add (build with
 * -ffp-contract=off, never -ffast-math), denormals kept.  The paper fixes the
 * state precision (12 bytes = fp32 master weight, m and v) but gives no
 * formula, so the operation order below is the reading this oracle commits
 * to; each choice is listed at the point where it is made.
 *
 * Parity status: every function here is pinned by tests that do not re-type
 * its formula (exact rational arithmetic, closed forms, invariants and a
 * library optimizer); none is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* ---- gradient element types ------------------------------------------- */
enum { ORACLE_DT_F32 = 0, ORACLE_DT_BF16 = 1, ORACLE_DT_I32 = 2 };
enum { ORACLE_AGG_FP32 = 0, ORACLE_AGG_FIXED = 1 };

/* bf16 -> fp32: a bf16 value is the top half of the fp32 with the same
 * sign, exponent and leading 7 mantissa bits, so widening is exact. */
float oracle_bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* fp32 -> bf16 with IEEE round-to-nearest-even on the 16 discarded bits
 * (the 2-byte parameter copy of Section III-D, step 5).  Ties go to the
 * even bf16 significand; values past the largest finite bf16 round to
 * infinity as IEEE prescribes.  NaN keeps its sign and becomes the quiet NaN
 * with payload 0x40 (a reading: the paper never meets NaN). */
uint16_t oracle_bf16_rne(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)(((u >> 16) & 0x8000u) | 0x7fc0u);
    uint32_t lsb = (u >> 16) & 1u;           /* last kept bit: breaks ties to even */
    return (uint16_t)((u + 0x7fffu + lsb) >> 16);
}

static float load_grad(const void *buf, int gdtype, int64_t i)
{
    if (gdtype == ORACLE_DT_BF16)
        return oracle_bf16_to_f32(((const uint16_t *)buf)[i]);
    return ((const float *)buf)[i];
}

/* ---- W-way aggregation, float mode ------------------------------------- */
/* The switch sums the W partial gradients of one element.  Reading: a sum
 * (not a mean), accumulated in fp32 in worker order 0, 1, ..., W-1, with one
 * rounding per addition. */
void oracle_aggregate_f32(const void *const *g, int W, int gdtype, int64_t n,
                          float *agg)
{
    for (int64_t i = 0; i < n; ++i) {
        float acc = load_grad(g[0], gdtype, i);
        for (int w = 1; w < W; ++w)
            acc = acc + load_grad(g[w], gdtype, i);
        agg[i] = acc;
    }
}

/* ---- W-way aggregation, fixed-point mode -------------------------------- */
/* Float-to-integer format conversion for an integer-only switch (Section
 * III-B, following SwitchML): scale by 2^k, round to the nearest integer
 * (ties to even), saturate to int32.  Readings: scaling by a power of two is
 * exact in fp32 unless it overflows, and an overflow to +-inf saturates like
 * any other out-of-range value; NaN contributes 0. */
int32_t oracle_quantize(float x, int k)
{
    float y = x * ldexpf(1.0f, k);
    if (y != y)
        return 0;
    float r = nearbyintf(y);                 /* default rounding: nearest even */
    if (r >= 2147483648.0f)
        return INT32_MAX;
    if (r < -2147483648.0f)
        return INT32_MIN;
    return (int32_t)r;
}

/* The format conversion over a whole buffer, as a worker's NIC would apply
 * it before pushing (Section III-B): out[i] = quantize(g[i], k). */
void oracle_quantize_array(const void *g, int gdtype, int64_t n, int k,
                           int32_t *out)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = oracle_quantize(load_grad(g, gdtype, i), k);
}

/* The integer a contribution brings to the switch: float contributions are
 * converted here; int32 contributions arrive already converted. */
static int32_t contribution_q(const void *buf, int gdtype, int64_t i, int k)
{
    if (gdtype == ORACLE_DT_I32)
        return ((const int32_t *)buf)[i];
    return oracle_quantize(load_grad(buf, gdtype, i), k);
}

/* Integer sum over the W workers (in a 64-bit accumulator, so the sum is
 * exact and independent of the order in which contributions arrive), then
 * one saturation to int32, then the conversion back to float: int32 -> fp32
 * rounds to nearest even, and the multiplication by 2^-k is exact. */
void oracle_aggregate_fixed(const void *const *g, int W, int gdtype, int64_t n,
                            int k, int32_t *agg_i32, float *agg_f32)
{
    for (int64_t i = 0; i < n; ++i) {
        int64_t s = 0;
        for (int w = 0; w < W; ++w)
            s += (int64_t)contribution_q(g[w], gdtype, i, k);
        int32_t a;
        if (s > (int64_t)INT32_MAX)
            a = INT32_MAX;
        else if (s < (int64_t)INT32_MIN)
            a = INT32_MIN;
        else
            a = (int32_t)s;
        if (agg_i32)
            agg_i32[i] = a;
        if (agg_f32)
            agg_f32[i] = (float)a * ldexpf(1.0f, -k);
    }
}

/* ---- per-step scalars --------------------------------------------------- */
/* The step-dependent constants of Adam with decoupled weight decay, taken
 * from the fp32 hyperparameters the caller passes:
 *   out[0] = beta1              out[1] = 1 - beta1   (fp32 subtraction)
 *   out[2] = beta2              out[3] = 1 - beta2   (fp32 subtraction)
 *   out[4] = 1 - beta1^t        out[5] = 1 - beta2^t (double, rounded once)
 *   out[6] = 1 - lr * wd        (double, rounded once)
 * The bias corrections use the fp32 betas, so at t = 1 out[4] equals out[1]
 * exactly. */
void oracle_scalars(float lr, float beta1, float beta2, float wd, int64_t t,
                    float out[7])
{
    out[0] = beta1;
    out[1] = 1.0f - beta1;
    out[2] = beta2;
    out[3] = 1.0f - beta2;
    out[4] = (float)(1.0 - pow((double)beta1, (double)t));
    out[5] = (float)(1.0 - pow((double)beta2, (double)t));
    out[6] = (float)(1.0 - (double)lr * (double)wd);
}

/* ---- Adam with decoupled weight decay on the aggregated gradient -------- */
/* One optimizer step on one element (Section III-D, step 5):
 *   g  = agg * grad_scale
 *   m  = beta1 m + (1 - beta1) g
 *   v  = beta2 v + (1 - beta2) g^2
 *   m^ = m / (1 - beta1^t),   v^ = v / (1 - beta2^t)
 *   p  = p (1 - lr wd) - lr m^ / (sqrt(v^) + eps)
 *   p16 = bf16(p)
 * Readings: eps outside the square root; decay applied to the pre-update
 * parameter as a factor; each product and quotient rounded on its own.
 * s[] holds the scalars of oracle_scalars for this step. */
static void adamw_element(const float s[7], float lr, float eps,
                          float grad_scale, float agg, float *p, float *m,
                          float *v, uint16_t *p16)
{
    const float b1 = s[0], omb1 = s[1], b2 = s[2], omb2 = s[3];
    const float bc1 = s[4], bc2 = s[5], decay = s[6];
    float g = agg * grad_scale;
    float mi = b1 * *m + omb1 * g;
    float gg = g * g;
    float vi = b2 * *v + omb2 * gg;
    float mh = mi / bc1;
    float vh = vi / bc2;
    float d = sqrtf(vh) + eps;
    float upd = mh / d;
    float pi = *p * decay - lr * upd;
    *m = mi;
    *v = vi;
    *p = pi;
    if (p16)
        *p16 = oracle_bf16_rne(pi);
}

/* The optimizer step over a shard of n elements whose gradient has already
 * been aggregated.  p, m and v are updated in place; p16 may be NULL. */
void oracle_adamw(const float *agg, float *p, float *m, float *v, uint16_t *p16,
                  int64_t n, float lr, float beta1, float beta2, float eps,
                  float wd, int64_t t, float grad_scale)
{
    float s[7];
    oracle_scalars(lr, beta1, beta2, wd, t, s);
    for (int64_t i = 0; i < n; ++i)
        adamw_element(s, lr, eps, grad_scale, agg[i], p + i, m + i, v + i,
                      p16 ? p16 + i : 0);
}

/* ---- the whole path: aggregation then the optimizer step ---------------- */
/* Composition of the two steps above, element by element: what the
 * parameter server does with each element of the shard once the switch has
 * aggregated it.  agg_f32 / agg_i32 receive the aggregate when non-NULL
 * (agg_i32 only in fixed-point mode). */
void oracle_fused(const void *const *g, int W, int gdtype, int64_t n, int mode,
                  int k, float *p, float *m, float *v, uint16_t *p16,
                  float *agg_f32, int32_t *agg_i32, float lr, float beta1,
                  float beta2, float eps, float wd, int64_t t, float grad_scale)
{
    float s[7];
    oracle_scalars(lr, beta1, beta2, wd, t, s);
    const void *gi[64];
    for (int64_t i = 0; i < n; ++i) {
        for (int w = 0; w < W; ++w)
            gi[w] = (gdtype == ORACLE_DT_BF16)
                        ? (const void *)((const uint16_t *)g[w] + i)
                        : (const void *)((const float *)g[w] + i);  /* f32, i32: 4 bytes */
        float a;
        if (mode == ORACLE_AGG_FIXED) {
            int32_t ai;
            oracle_aggregate_fixed(gi, W, gdtype, 1, k, &ai, &a);
            if (agg_i32)
                agg_i32[i] = ai;
        } else {
            oracle_aggregate_f32(gi, W, gdtype, 1, &a);
        }
        if (agg_f32)
            agg_f32[i] = a;
        adamw_element(s, lr, eps, grad_scale, a, p + i, m + i, v + i,
                      p16 ? p16 + i : 0);
    }
}

/* Non-zero when the x86 SSE control word flushes or treats denormals as
 * zero; the oracle's results assume it does neither. */
unsigned oracle_mxcsr_ftz_daz(void)
{
#if defined(__x86_64__)
    unsigned csr;
    __asm__ volatile("stmxcsr %0" : "=m"(csr));
    return csr & ((1u << 15) | (1u << 6));
#else
    return 0;
#endif
}
