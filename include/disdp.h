/*
 * disdp.h -- C ABI of the parameter-server hot path of DisDP
 * (arXiv 2409.00918) on one MI355X (gfx950).
 *
 * In DisDP each worker pushes its partial gradient of a model layer, the
 * SmartSwitch sums the W contributions in the network, and a parameter
 * server pulls the aggregate, runs a mixed-precision Adam step on its
 * 12-byte model states and serves the 2-byte parameter copy back
 * (Section III-A "Overall Architecture"; Section III-D "Backward Stage",
 * steps 3, 5 and 1-2; Table III).  This library performs that reduction and
 * that optimizer step on one GPU, for one shard of N elements whose W
 * contributions already sit in device memory:
 *
 *   disdp_aggregate      -- the W-way reduction alone (the switch's job),
 *   disdp_adam_step      -- the optimizer step alone (step 5),
 *   disdp_aggregate_adam -- both in one pass over memory, with the bf16
 *                           parameter copy fused into the store;
 *   disdp_quantize       -- the worker-side conversion of a gradient into the
 *                           integer format the fixed-point mode sums;
 *   disdp_shard_layout   -- where to place a shard's arrays in one
 *                           allocation for the fastest streaming;
 *   disdp_step_scalars, disdp_aggregate_adam_dev
 *                        -- the fused call with the step's constants in
 *                           device memory, for one HIP graph replayed
 *                           across optimizer steps;
 *   disdp_aggregate_adam_multi
 *                        -- the fused call over many tensors in separate
 *                           buffers, a batch of tensors per launch.
 *
 * The calls follow the shape of the paper's asynchronous push/pull API
 * (Table II: a buffer pointer and a length; completion awaited through a
 * handle): a HIP stream plays the role of the handle.
 *
 * Common conventions
 * ------------------
 * Ownership   The caller owns every buffer.  The library allocates nothing,
 *             keeps no state between calls, never synchronises and is
 *             re-entrant.  `grads` is a HOST array of W pointers, read before
 *             the call returns.
 * Memory      Every array pointer must be one the GPU can dereference at that
 *             address: device (or managed) memory, or pinned host memory
 *             mapped for the device (hipHostMalloc), whose device address is
 *             its host address.  Host-resident arrays are streamed by the
 *             kernels over the host link -- e.g. the 12-byte states of a
 *             shard too large for HBM, kept in host DRAM as the paper's
 *             parameter server keeps them (Section III-D, steps 4 and 6).
 * Layout      Every array is flat and contiguous with N elements
 *             (0 <= N <= 2^56, else DISDP_ERR_INVALID_ARG); index i
 *             is the same parameter in every array.  fp32 arrays hold IEEE
 *             binary32; bf16 arrays hold raw bf16 bit patterns (uint16_t);
 *             the int32 aggregate is two's complement.
 * Asynchrony  Work is enqueued on `stream` (0 = the null stream) and the
 *             call returns at once; completion is the caller's
 *             hipStreamSynchronize or an event.  A call enqueues kernel
 *             launches only (no allocation, memset, copy or wait), so it
 *             may be captured in a HIP graph; the hyperparameters, step t
 *             included, are kernel arguments and are fixed at capture
 *             (disdp_aggregate_adam_dev reads them from device memory when
 *             its kernel runs instead).
 * Alignment   Any alignment is accepted; results never depend on it.  The
 *             vector kernels run when every array starts the same number of
 *             elements past a 4-element boundary (16 bytes for 4-byte
 *             arrays, 8 for bf16), e.g. any sub-range of aligned arrays: the
 *             first few elements (up to 255, reaching a common 256- or
 *             64-element boundary when the arrays agree that far) are done
 *             one by one.
 *             Arrays with unrelated offsets take them too when every array
 *             is aligned to its element size and the bf16 arrays can reach
 *             4-byte boundaries together: the first output is brought to a
 *             256-element boundary (or one element past it) and the others
 *             are read and written at 4-byte-aligned addresses.  Otherwise
 *             (an array not aligned to its element size, or bf16 arrays at
 *             both odd and even element offsets) an element-wise kernel
 *             runs.
 * Errors      Arguments are checked on the host in this order: counts and
 *             enumerations, hyperparameters, then (only when n > 0) NULL
 *             pointers, overlap, and -- the first HIP call -- that every
 *             array is GPU-addressable (hipPointerGetAttributes; pageable or
 *             unknown memory gives DISDP_ERR_INVALID_ARG).  A failed check
 *             returns its code and enqueues nothing.  n == 0 returns
 *             DISDP_OK with no launch (NULL pointers are then allowed).
 *             Outputs must not overlap one another nor any input; p, m and
 *             v are updated in place (each is its own input).  Contributions
 *             may overlap each other (the same buffer may be passed twice).
 *             A launch failure returns DISDP_ERR_HIP.  A runtime query
 *             the library makes (pointer attributes, the stream's CU mask)
 *             that fails leaves no error behind when none was pending
 *             before the call; when the caller already had one pending, the
 *             error state is left set (the runtime keeps a single last
 *             error, which the failed query may have replaced), so
 *             hipGetLastError still reports an error.
 * Numerics    IEEE binary32, round to nearest even, one rounding per
 *             operation, no fused multiply-add, denormals kept; results are
 *             a deterministic function of the inputs (no atomics, no
 *             dependence on grid size).
 * Sharing     The kernels are memory-bound and by default launch one-wave
 *             blocks, the fastest shape when they have the GPU to
 *             themselves.  On a GPU whose compute kernels run at the same
 *             time on other streams, that shape refills every slot a
 *             retiring block frees: measured next to a bf16 GEMM loop on the
 *             7B/8 shard, the GEMM slowed about 10x and the fused call 1.1x.
 *             Two knobs trade this, neither changing any result:
 *               - DISDP_LAUNCH_SHAPE=shared in the environment (read on every
 *                 call) selects four-wave blocks with one occupancy cap per
 *                 mode, which share an unmasked chip more evenly (about 2x
 *                 each) at a few percent below the default rate alone;
 *               - a CU-masked stream (hipExtStreamCreateWithCUMask) confines
 *                 the kernels to its CUs; the library reads the mask and
 *                 raises its per-CU occupancy cap to match.
 *             The many-tensor call and disdp_quantize always launch
 *             one-wave blocks.
 * Known issue (memory from hipExtMallocWithFlags with
 *             hipDeviceMallocContiguous; not allocated by this library):
 *             on MI355X, after such a block was released with hipFree and
 *             the same address range was handed out again by another
 *             allocator, kernels read stale or zero values from memory that
 *             had just been written by a synchronised copy.  The cause was
 *             not found.  Callers that allocate shard memory that way should
 *             keep those blocks for the life of the process (the Python
 *             binding pools them) rather than freeing them.
 */
#ifndef DISDP_H
#define DISDP_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DISDP_OK = 0,
    DISDP_ERR_INVALID_ARG = 1, /* bad count, range, hyperparameter or NULL */
    DISDP_ERR_UNSUPPORTED = 2, /* unknown dtype or aggregation mode        */
    DISDP_ERR_ALIAS = 3,       /* an output overlaps another buffer        */
    DISDP_ERR_HIP = 4          /* the HIP runtime refused the launch       */
} disdp_status_t;

/* Element type of the W gradient contributions.  Workers produce fp16/bf16
 * or fp32 gradients (Section III-B "Format Conversion Unit"); bf16 is
 * widened to fp32 exactly before any arithmetic.  DISDP_DT_I32 marks
 * contributions already converted to the switch's integer format at scale
 * 2^frac_bits (the output of disdp_quantize); they are summed as they are,
 * so they are accepted in DISDP_AGG_FIXED mode only. */
typedef enum { DISDP_DT_F32 = 0, DISDP_DT_BF16 = 1, DISDP_DT_I32 = 2 } disdp_dtype_t;

/* How the W contributions are summed.
 *  DISDP_AGG_FP32   acc = g_0[i]; acc = acc + g_w[i] for w = 1 .. W-1, in
 *                   fp32, always in this worker order.
 *  DISDP_AGG_FIXED  the integer format an integer-only switch sums
 *                   (Section III-B, following SwitchML): each contribution
 *                   becomes q_w = sat32(round_half_even(g_w[i] * 2^k))
 *                   (NaN -> 0, +-inf and out-of-range values saturate);
 *                   S = sum of q_w in 64-bit integers (exact, so independent
 *                   of the order contributions arrive in); A = sat32(S);
 *                   the float aggregate is (float)A * 2^-k. */
typedef enum { DISDP_AGG_FP32 = 0, DISDP_AGG_FIXED = 1 } disdp_agg_mode_t;

/* Adam with decoupled weight decay (Section III-D, step 5: 17 flops per
 * element on the aggregated gradient and the fp32 master weight, m and v).
 * With g = agg * grad_scale and t = step:
 *   m = beta1 m + (1 - beta1) g
 *   v = beta2 v + (1 - beta2) g^2
 *   p = p (1 - lr weight_decay) - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)
 * 1 - beta^t and 1 - lr weight_decay are evaluated in double on the host
 * and rounded once to fp32; 1 - beta is an fp32 subtraction.
 * Valid ranges: step >= 1; 0 <= beta1, beta2 < 1; eps >= 0; all values
 * finite.  eps == 0 is accepted: then a zero gradient with v == 0 gives
 * 0/0 = NaN, as IEEE arithmetic does. */
typedef struct {
    float lr;
    float beta1;
    float beta2;
    float eps;
    float weight_decay;
    int64_t step;      /* t >= 1; the caller counts steps */
    float grad_scale;  /* applied to the aggregate; 1.0f = plain sum */
} disdp_adamw_hparams_t;

/* W-way reduction of one shard (the SmartSwitch's aggregation, Section
 * III-A and III-C "Packet Transport Procedure").
 *   grads       host array of W device pointers, each to n elements of
 *               `gdtype`; 1 <= W <= 64.  DISDP_DT_I32 only in fixed mode.
 *   mode        DISDP_AGG_FP32 or DISDP_AGG_FIXED; frac_bits = k in [0, 30]
 *               (checked in fixed mode only).
 *   agg_out_f32 fp32 aggregate (n elements).  Required in FP32 mode.
 *   agg_out_i32 int32 aggregate A (n elements); fixed mode only, must be
 *               NULL in FP32 mode.  In fixed mode at least one of the two
 *               outputs must be non-NULL.
 * Returns DISDP_OK or an error code (see the conventions above). */
disdp_status_t disdp_aggregate(const void *const *grads, int W,
                               disdp_dtype_t gdtype, int64_t n,
                               disdp_agg_mode_t mode, int frac_bits,
                               float *agg_out_f32, int32_t *agg_out_i32,
                               hipStream_t stream);

/* The optimizer step alone on an already aggregated fp32 gradient
 * (Section III-D, step 5: reads a gradient and 12 bytes of state, writes
 * 12 bytes of state and a 2-byte parameter copy).
 *   grad            fp32 aggregate (n elements), read only.
 *   param, m, v     fp32 master weight and moments, updated in place.
 *   param_bf16_out  bf16 copy of the updated weight, round to nearest even
 *                   (NaN keeps its sign, becomes 0x7FC0 | sign); NULL = skip.
 *   hp              host pointer, read before the call returns. */
disdp_status_t disdp_adam_step(const float *grad, float *param, float *m,
                               float *v, uint16_t *param_bf16_out, int64_t n,
                               const disdp_adamw_hparams_t *hp,
                               hipStream_t stream);

/* Aggregation and optimizer step fused into one pass: each element's W
 * contributions, p, m and v are read once and p, m, v and the bf16 copy
 * written once.  Equal, bit for bit, to disdp_aggregate followed by
 * disdp_adam_step on its fp32 aggregate.
 *   agg_out_f32 / agg_out_i32   optional copies of the aggregate (NULL = not
 *               written; agg_out_i32 only in fixed mode).
 * Other arguments as in disdp_aggregate and disdp_adam_step. */
disdp_status_t disdp_aggregate_adam(const void *const *grads, int W,
                                    disdp_dtype_t gdtype, int64_t n,
                                    disdp_agg_mode_t mode, int frac_bits,
                                    float *param, float *m, float *v,
                                    uint16_t *param_bf16_out,
                                    float *agg_out_f32, int32_t *agg_out_i32,
                                    const disdp_adamw_hparams_t *hp,
                                    hipStream_t stream);

/* The per-step constants of the optimizer, as the calls above derive them
 * from disdp_adamw_hparams_t on the host: beta1, 1 - beta1, beta2, 1 - beta2,
 * the bias corrections 1 - beta1^t and 1 - beta2^t (double, rounded once),
 * 1 - lr weight_decay (double, rounded once), lr, eps and grad_scale. */
typedef struct {
    float beta1, one_minus_beta1;
    float beta2, one_minus_beta2;
    float bias_correction1, bias_correction2;
    float decay;
    float lr, eps, grad_scale;
} disdp_step_scalars_t;

/* Fills `out` with the constants of step hp->step, exactly as
 * disdp_aggregate_adam computes them.  Pure host computation, no HIP call.
 * Returns DISDP_ERR_INVALID_ARG for NULL pointers or invalid
 * hyperparameters (the ranges of disdp_adamw_hparams_t). */
disdp_status_t disdp_step_scalars(const disdp_adamw_hparams_t *hp, disdp_step_scalars_t *out);

/* disdp_aggregate_adam with the step constants read from memory when the
 * kernel runs instead of when the call is made: `scalars` points to a
 * disdp_step_scalars_t in device memory (or pinned host memory mapped for
 * the device), 4-byte aligned, filled by disdp_step_scalars; it must not
 * overlap an output (DISDP_ERR_ALIAS).  For HIP graphs: a captured
 * graph whose copy node refreshes `scalars` from a host buffer that the
 * caller rewrites before each replay serves every optimizer step with one
 * capture, and gives the same bits as disdp_aggregate_adam with that step's
 * hyperparameters.  The contents of `scalars` are not checked (the pointer
 * is); every other argument as in disdp_aggregate_adam. */
disdp_status_t disdp_aggregate_adam_dev(const void *const *grads, int W,
                                        disdp_dtype_t gdtype, int64_t n,
                                        disdp_agg_mode_t mode, int frac_bits,
                                        float *param, float *m, float *v,
                                        uint16_t *param_bf16_out,
                                        float *agg_out_f32, int32_t *agg_out_i32,
                                        const disdp_step_scalars_t *scalars,
                                        hipStream_t stream);

/* disdp_aggregate_adam over T tensors of one optimizer step (Section III-D,
 * step 5, applied tensor by tensor): for a shard whose tensors live in
 * separate buffers, one launch serves a batch of tensors instead of one
 * launch each (up to 48 tensors and 320 pointers per launch).  Equal, bit
 * for bit, to T disdp_aggregate_adam calls with the same hyperparameters.
 *   T               number of tensors, 0 <= T <= 65536.
 *   n               host array of T element counts (each 0 .. 2^56).
 *   grads           host array of T*W device pointers: contribution w of
 *                   tensor j is grads[j*W + w].
 *   param, m, v     host arrays of T device pointers (fp32, updated in
 *                   place).
 *   param_bf16_out  host array of T device pointers (an entry may be NULL),
 *                   or NULL: no bf16 copies.
 *   hp              one step for every tensor, as in disdp_aggregate_adam;
 *                   or NULL with `scalars` given.
 *   scalars         NULL, or the step's constants in device memory as for
 *                   disdp_aggregate_adam_dev (4-byte aligned, not
 *                   overlapping an output), read when the kernels run: one
 *                   captured HIP graph then serves every step.  Exactly one
 *                   of hp and scalars is non-NULL.
 * Every array is read before the call returns.  Tensors with n == 0 are
 * skipped (their pointers may be NULL).  Checks as for disdp_aggregate_adam,
 * over all tensors together: no output of any tensor may overlap any other
 * buffer of any tensor (DISDP_ERR_ALIAS; contributions may overlap one
 * another).  Alignment as for the other calls, per tensor.  The runtime is
 * asked about each device allocation the pointers fall in once per call, so
 * tensors carved out of a few large allocations are checked in a few
 * queries.  The checks use host memory proportional to T * (W + 4); a
 * launch failure after earlier batches were enqueued returns
 * DISDP_ERR_HIP. */
disdp_status_t disdp_aggregate_adam_multi(const void *const *grads, int W,
                                          disdp_dtype_t gdtype, int T, const int64_t *n,
                                          disdp_agg_mode_t mode, int frac_bits,
                                          float *const *param, float *const *m,
                                          float *const *v, uint16_t *const *param_bf16_out,
                                          const disdp_adamw_hparams_t *hp,
                                          const disdp_step_scalars_t *scalars,
                                          hipStream_t stream);

/* The float-to-integer format conversion a worker's NIC applies before
 * pushing its gradient to an integer-only switch (Section III-B "Format
 * Conversion Unit", following SwitchML): for every i,
 *   out[i] = sat32(round_half_even(grad[i] * 2^frac_bits)),
 * NaN -> 0, +-inf and out-of-range values saturate -- the same conversion
 * DISDP_AGG_FIXED applies inside the aggregation, so W buffers converted here
 * and aggregated as DISDP_DT_I32 give the same bits as aggregating the W
 * float buffers in fixed mode.
 *   grad        n elements of `gdtype` (DISDP_DT_F32 or DISDP_DT_BF16).
 *   frac_bits   k in [0, 30].
 *   out         n int32 (device), must not overlap grad.
 * Errors as for the other calls (DISDP_ERR_UNSUPPORTED for DISDP_DT_I32
 * input). */
disdp_status_t disdp_quantize(const void *grad, disdp_dtype_t gdtype, int64_t n,
                              int frac_bits, int32_t *out, hipStream_t stream);

/* Optional arrays a shard layout reserves room for (bit flags). */
enum {
    DISDP_LAYOUT_BF16_COPY = 1, /* the bf16 parameter copy            */
    DISDP_LAYOUT_AGG_F32 = 2,   /* an fp32 aggregate                  */
    DISDP_LAYOUT_AGG_I32 = 4    /* an int32 aggregate (fixed mode)    */
};

/* Where to place the arrays of one shard -- the W contributions and the
 * parameter server's 12-byte state and 2-byte copy (Section III-D, step 5)
 * -- inside ONE device allocation so that the fused kernel streams them at
 * its best and most repeatable rate.  The kernel walks every array in
 * lockstep, and on MI355X how the arrays' starts sit relative to each other
 * changes the streaming rate by up to 6%.  The arrays follow one another in
 * the order below, each starting on a 32 MiB boundary, the next one at the
 * first boundary at least 17 pages of 2 MiB past the end of the previous
 * one: over shards of 2^26 to 2.7e9 elements this placement's slowest case
 * streamed fastest of those measured.  Independent allocations land at
 * arbitrary relative offsets and run slower and less repeatably.  The cost
 * is at most 66 MiB of padding per array.
 * Pure computation: no HIP call, nothing allocated.
 *   n, W, gdtype  the shard (1 <= W <= 64; gdtype F32, BF16 or I32).
 *   flags         DISDP_LAYOUT_* arrays to include besides contributions and
 *                 p, m, v.
 *   offsets       caller array of W + 6 int64: byte offsets of
 *                 contributions 0..W-1, then param, m, v, param_bf16,
 *                 agg_f32, agg_i32 (-1 for arrays not requested).
 *   total_bytes   bytes to allocate (0 when n == 0; every requested array
 *                 is then at offset 0).  Offsets are multiples of 32 MiB, so
 *                 every array keeps the allocation's alignment (the vector
 *                 kernels need 16 bytes; hipMalloc gives more).  Only the
 *                 relative placement matters: moving a whole layout by
 *                 whole pages streamed at the same rate.
 * Returns DISDP_OK, or DISDP_ERR_INVALID_ARG / DISDP_ERR_UNSUPPORTED for a
 * bad n, W, NULL output or unknown dtype, and DISDP_ERR_INVALID_ARG when the
 * total would not fit in int64 (possible near the largest n with large W);
 * the outputs may then be partly written. */
disdp_status_t disdp_shard_layout(int64_t n, int W, disdp_dtype_t gdtype, unsigned flags,
                                  int64_t *offsets, int64_t *total_bytes);

/* A static, NUL-terminated English name for a status code (never NULL;
 * unknown codes give "unknown status"). */
const char *disdp_status_string(disdp_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* DISDP_H */
