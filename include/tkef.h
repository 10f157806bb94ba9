/*
 * tkef: exact top-k gradient sparsification with error feedback, and the
 * sparse aggregate + merged multi-tensor SGD update, for AMD MI355X (gfx950).
 *
 * C ABI. Every pointer argument documented as "device" must point to device
 * memory of the current HIP device; "host" pointers are read during the call
 * only. The caller owns every buffer. The library allocates no device memory:
 * all scratch space lives in a caller-provided workspace ("ws"), whose size is
 * reported by the *_info / *_workspace queries. All GPU work of a call is
 * enqueued on the caller's stream and is asynchronous with respect to the
 * host, except where a function says it synchronizes.
 *
 * Return codes: TKEF_OK (0) or a negative TKEF_E* code. A call that returns
 * an error has enqueued no GPU work, except TKEF_EHIP, which reports a HIP
 * runtime failure (launch or copy) after work may have been enqueued.
 * Problems that only the GPU can see (a NaN in the data, an unsorted or
 * out-of-range index list) set bits in an optional caller-owned device status
 * word (uint32, zeroed by the caller, bits OR-ed in by the library).
 *
 * Thread safety: plans are not shared between threads without external
 * locking; distinct plans may be used concurrently. Calls that share a
 * workspace must be ordered on one stream.
 *
 * HIP graphs: the *_execute calls of a bound plan only launch kernels, with
 * the same arguments on every call, and leave the workspace's zeroed scratch
 * as they found it, so they can be captured into a graph and replayed (the
 * buffers bound at bind must stay in place); so can tkef_sparsify1_static.
 * Binds, the other one-shot calls and tkef_sparsify_approx_result
 * synchronize and are not capturable.
 */
#ifndef TKEF_H
#define TKEF_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TKEF_VERSION 10200 /* major * 10000 + minor * 100 + patch */

/* return codes */
#define TKEF_OK 0
#define TKEF_EINVAL (-1)     /* null pointer, bad mode, bad count, aliasing */
#define TKEF_ERANGE (-2)     /* size >= 2^31, k outside [1, d], rho outside (0, 1] */
#define TKEF_EWORKSPACE (-3) /* workspace missing, too small or not 256-B aligned */
#define TKEF_EHIP (-4)       /* HIP runtime error */
#define TKEF_ESTATE (-5)     /* plan not bound, or bound to another workspace */
#define TKEF_ENOMEM (-6)     /* host allocation failed */

/* value formats of the (idx, val) lists */
#define TKEF_VAL_F32 0 /* binary32 (default) */
#define TKEF_VAL_F16 1 /* binary16, converted from binary32 with round-to-nearest-even
                          (overflow to infinity, subnormals kept); Sec. 5.3 sends FP16
                          elements */

/* selection modes */
#define TKEF_GLOBAL 0     /* one selection over the concatenated tensor list */
#define TKEF_PER_TENSOR 1 /* one selection per tensor, k_t from rho per tensor */
#define TKEF_APPROX 2     /* one selection over the concatenated list with MSTopK (Alg. 1) */

/* device status bits */
#define TKEF_STATUS_NAN 1u         /* sparsify saw a NaN in g + r */
#define TKEF_STATUS_UNSORTED 2u    /* an update index list is not ascending */
#define TKEF_STATUS_INDEX_RANGE 4u /* an update index lies outside [0, d) */
#define TKEF_STATUS_TIMEOUT 8u     /* a bounded wait between workgroups gave up: results invalid
                                       (the workgroups that gave up wrote no output) */
#define TKEF_STATUS_NONFINITE 16u  /* MSTopK saw an infinity or NaN in g + r (it then takes
                                       the first k positions) */

int tkef_version(void);
const char *tkef_strerror(int code);

/*
 * k = ceil(rho * d) evaluated in double precision, clamped to [1, d]; the
 * paper writes k = rho * d for a density 0 < rho < 1 (Sec. 3.2, sparse
 * format) without a rounding rule. Returns 0 for d == 0 and a negative code
 * for rho outside (0, 1] or d < 0.
 */
int64_t tkef_k_from_rho(int64_t d, double rho);

/* ========================================================================
 * Sparsify (Sec. 3.1, TopK operator; Alg. 1 output format; error feedback)
 *
 * For a list of T float32 gradient tensors g_t and residual tensors r_t
 * (same sizes), with global position i = offset_t + j in the concatenation:
 *   x_i = g_i + r_i                       (one binary32 add, round-to-nearest)
 *   S   = the k positions first in the order (|x| descending, i ascending)
 *   idx = S in ascending order (int32), val_j = x[idx_j] (bitwise, sign kept)
 *   r_i = x_i for i not in S, +0.0f for i in S     (residuals updated in place)
 * TKEF_GLOBAL selects once over all positions (k from rho over the total
 * size, or an explicit k). TKEF_PER_TENSOR selects k_t = tkef_k_from_rho(n_t,
 * rho) within each tensor; outputs are concatenated in tensor order and still
 * carry global positions. Magnitudes compare as IEEE values: -0 equals +0,
 * infinities rank above every finite value. A NaN in x sets
 * TKEF_STATUS_NAN; the selection is then unspecified (but every output is
 * still written within bounds).
 * ====================================================================== */

typedef struct tkef_sparsify_plan_s *tkef_sparsify_plan;

/* Host only. numels: host array of T sizes (each >= 0, total in [1, 2^31-1]).
 * k > 0 gives an explicit k (TKEF_GLOBAL only, k <= total); k == 0 takes k
 * from rho. The list takes ceil(numel_t / 8192) tiles per tensor, at most
 * 2^18 in all (TKEF_ERANGE otherwise); one tensor of 2^31 - 1 elements takes
 * exactly 2^18. */
int tkef_sparsify_plan_create(const int64_t *numels, int32_t ntensors, int32_t mode,
                              double rho, int64_t k, tkef_sparsify_plan *plan_out);
int tkef_sparsify_plan_destroy(tkef_sparsify_plan plan);

/* Host only. workspace_bytes: device workspace the plan needs; k_total: number
 * of (idx, val) pairs an execution writes; d_total: total positions;
 * ngroups: 1 (global) or T (per tensor); nlaunch: kernels per execution. */
int tkef_sparsify_plan_info(tkef_sparsify_plan plan, size_t *workspace_bytes,
                            int64_t *k_total, int64_t *d_total, int32_t *ngroups,
                            int32_t *nlaunch);

/* Host only: k of each selection group (ngroups entries). */
int tkef_sparsify_plan_group_k(tkef_sparsify_plan plan, int64_t *k_out, int32_t n);

/* Binds device tensors to the plan and writes the plan's descriptor tables
 * into ws (device, >= workspace_bytes, 256-B aligned). grads[t], residuals[t]:
 * host arrays of device pointers (non-null when numel > 0; g and r must not
 * overlap). Copies host -> device on `stream` and synchronizes that stream.
 * The ws then belongs to the plan until the next bind. */
int tkef_sparsify_plan_bind(tkef_sparsify_plan plan, const float *const *grads,
                            float *const *residuals, void *ws, size_t ws_bytes,
                            hipStream_t stream);

/* Runs one sparsify on the bound tensors: reads g, updates r in place, writes
 * k_total pairs to idx_out (device int32) and val_out (device float32, or
 * binary16 after tkef_sparsify_plan_set_value_format(plan, TKEF_VAL_F16)). ws
 * must be the bound workspace. status: optional device word. Asynchronous. */
int tkef_sparsify_execute(tkef_sparsify_plan plan, void *ws, size_t ws_bytes,
                          int32_t *idx_out, void *val_out, uint32_t *status,
                          hipStream_t stream);

/* Value format of val_out: TKEF_VAL_F32 (default) or TKEF_VAL_F16 (the wire
 * format of Sec. 5.3). With binary16 values the residual still keeps the
 * binary32 x where not selected and +0 where selected: the rounding of the
 * sent value is not fed back. Host only; TKEF_EINVAL for another format. */
int tkef_sparsify_plan_set_value_format(tkef_sparsify_plan plan, int32_t format);

/* MSTopK parameters of a TKEF_APPROX plan (Alg. 1). n_search: rounds of the
 * threshold bisection, 1..48 (the paper runs 30, which is the default; the
 * kernel count, 3 + ceil(max(0, n_search - 6) / 12), is reported by *_info
 * after this call). window_word: the 64-bit value the band offset is drawn from for the
 * next executions: offset = window_word mod (band - (k - k1) + 1), so a
 * caller wanting the paper's random offset passes a fresh random word per
 * execution. Host only; TKEF_EINVAL for another mode or n_search outside
 * 1..48.
 *
 * What a TKEF_APPROX execution computes (readings of Alg. 1): x = g + r as
 * above; a = |x|; mean = (the exact sum of a, rounded once to double) / d in
 * double; u = max a; round i of N takes ratio = l + (r - l) / 2 and
 * thres = mean + ratio * (u - mean) in double and counts n = #{a >= thres}
 * (a widened exactly); n <= k sets r = ratio and, if n > k1, (k1, thres1) =
 * (n, thres); otherwise l = ratio and, if n < k2, (k2, thres2) = (n, thres);
 * start l = 0, r = 1, k1 = 0, thres1 = +inf, k2 = d, thres2 = 0. The result
 * is {a >= thres1} plus the band members {thres2 <= a < thres1} of rank
 * offset .. offset + k - k1 - 1 in position order; idx ascending, val = x at
 * idx, r = x with the selected positions set to +0. Exactly k pairs. */
int tkef_sparsify_plan_set_approx(tkef_sparsify_plan plan, int32_t n_search,
                                  uint64_t window_word);

/* Host; synchronizes `stream`. Reads back the search result of the last
 * TKEF_APPROX execution on the bound ws: out[0] = the mean, out[1] = u (as
 * doubles); cnt[0] = k1, cnt[1] = k2 (the recorded counts), cnt[2] = the
 * window offset, cnt[3] = k - k1 (taken from the band), cnt[4] = the key
 * (binary32 bits with the sign cleared) of the smallest binary32 >= thres1
 * (2^31 when thres1 was never set), cnt[5] = the same for thres2. Either
 * array may be NULL. TKEF_EINVAL for another mode; TKEF_ESTATE if ws is not
 * the bound workspace. */
int tkef_sparsify_approx_result(tkef_sparsify_plan plan, void *ws, double *out,
                                int64_t *cnt, hipStream_t stream);

/* Optional timing hook: with n_events >= nlaunch + 1, each execution records
 * events[0] at the start of its first kernel and events[i + 1] at the end of
 * kernel i (HIP events created by the caller; the kernel dispatches record
 * them, so no extra commands run between the kernels). Pass NULL to switch it
 * off. Names of the kernels in launch order are available from
 * tkef_sparsify_plan_launch_name. */
int tkef_sparsify_plan_set_events(tkef_sparsify_plan plan, hipEvent_t *events,
                                  int32_t n_events);
const char *tkef_sparsify_plan_launch_name(tkef_sparsify_plan plan, int32_t i);

/* One-shot calls (the call shape sparsify(grad, residual, rho) -> idx, val):
 * create + bind + execute + destroy; each synchronizes `stream` once (during
 * bind). tkef_sparsify_workspace reports the workspace of a call with the
 * same numels, mode, rho and k, and its number of pairs (k_total). */
int tkef_sparsify_workspace(const int64_t *numels, int32_t ntensors, int32_t mode,
                            double rho, int64_t k, size_t *workspace_bytes,
                            int64_t *k_total);

/* Sparsify of a tensor list (the operation above; mode TKEF_GLOBAL,
 * TKEF_PER_TENSOR or TKEF_APPROX with N = 30 and window word 0). k > 0:
 * explicit k (not TKEF_PER_TENSOR); k == 0: k from rho. val_format: TKEF_VAL_F32
 * or TKEF_VAL_F16. idx_out / val_out (device) receive k_total pairs, grouped
 * by selection group in tensor order. counts_out: optional host array that
 * receives the k of each selection group (1 entry, or T for
 * TKEF_PER_TENSOR), written before any GPU work. */
int tkef_sparsify(const float *const *grads, float *const *residuals,
                  const int64_t *numels, int32_t ntensors, int32_t mode, double rho,
                  int64_t k, int32_t val_format, int32_t *idx_out, void *val_out,
                  int64_t *counts_out, void *ws, size_t ws_bytes, uint32_t *status,
                  hipStream_t stream);

/* One flat tensor with an explicit k: Alg. 1's interface (x, k) -> (values,
 * indices), Sec. 3.1, with the exact selection and error feedback above. g, r:
 * device, d elements each (1 <= d <= 2^31 - 1, not overlapping); 1 <= k <= d
 * (TKEF_ERANGE otherwise). idx_out (int32) and val_out (binary32): device, k
 * entries. ws: at least what tkef_sparsify_workspace(&d, 1, TKEF_GLOBAL, 0.0,
 * k, ...) reports. status: optional device word. Synchronizes `stream` once. */
int tkef_sparsify1(const float *g, float *r, int64_t d, int64_t k, int32_t *idx_out,
                   float *val_out, void *ws, size_t ws_bytes, uint32_t *status,
                   hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * tkef_sparsify1 without a workspace argument. Its scratch is a fixed array of
 * TKEF_STATIC_SCRATCH_BYTES in the library's device memory, one per GPU, held
 * until the process ends; the first call on a device looks up that device's
 * copy. Limits: 1 <= d <= TKEF_STATIC_MAX_D and 1 <= k <= min(d,
 * TKEF_STATIC_MAX_K) (TKEF_ERANGE otherwise). The call allocates nothing and
 * does not synchronize: four kernels on `stream` (a set-up kernel, then the
 * three of the exact selection). Results are those of tkef_sparsify1. All
 * calls on one GPU use that GPU's one array, which keeps the last call's
 * contents (each call clears what must start at zero): calls that overlap in
 * time on one GPU (other streams, other host threads) race and give wrong
 * results. */
#define TKEF_STATIC_MAX_D (1LL << 26)
#define TKEF_STATIC_MAX_K (1LL << 17)
#define TKEF_STATIC_SCRATCH_BYTES ((size_t)36 << 20)
int tkef_sparsify1_static(const float *g, float *r, int64_t d, int64_t k, int32_t *idx_out,
                          float *val_out, uint32_t *status, hipStream_t stream);

/* ========================================================================
 * Sparse aggregate + merged multi-tensor SGD update
 * (Alg. 2, accumulation of the gathered lists; Eq. (1) update)
 *
 * P workers' sparse gradients in the gathered layout that an All-Gather of
 * fixed-size lists produces: worker p's entries are idx[p*stride + j],
 * val[p*stride + j] for j < nnz_p (nnz_p = nnz[p] if an nnz array is given,
 * else stride). Indices are global positions in the concatenation of the T
 * parameter tensors; each worker's list must be ascending (repeats allowed and
 * summed). With G = sum over workers of their values at each position:
 *   mu == 0 and wd == 0:  w_i -= lr * G_i at every position some list names
 *                         (all other parameters are left untouched)
 *   otherwise, at every position:
 *       D = G_i + wd * w_i;  if mu != 0: b_i = mu * b_i + D, U = b_i; else U = D
 *       w_i -= lr * U
 * Each step is a binary32 operation with round-to-nearest (no fused
 * multiply-add). G is accumulated in binary32; where three or more workers
 * name one position, the order of its additions is unspecified, unless the
 * plan is set deterministic (tkef_update_plan_set_deterministic: worker
 * order, then list order).
 * ====================================================================== */

typedef struct tkef_update_plan_s *tkef_update_plan;

/* Host only. numels: T parameter sizes (total in [1, 2^31-1]); P workers
 * (1 <= P <= 65535); stride: entries reserved per worker in the gathered
 * arrays (0 <= stride <= 2^31-1). */
int tkef_update_plan_create(const int64_t *numels, int32_t ntensors, int32_t P,
                            int64_t stride, tkef_update_plan *plan_out);
int tkef_update_plan_destroy(tkef_update_plan plan);
int tkef_update_plan_info(tkef_update_plan plan, size_t *workspace_bytes,
                          int64_t *d_total, int32_t *nlaunch);

/* Binds parameter tensors (host array of T device pointers) and optional
 * momentum buffers (host array of T device pointers, or NULL) and writes the
 * descriptor tables into ws. Copies host -> device and synchronizes `stream`. */
int tkef_update_plan_bind(tkef_update_plan plan, float *const *params,
                          float *const *momentum, void *ws, size_t ws_bytes,
                          hipStream_t stream);

/* Applies one aggregate + update. idx (device int32) and val (device float32,
 * or binary16 after tkef_update_plan_set_value_format(plan, TKEF_VAL_F16);
 * binary16 values are widened exactly and summed in binary32) hold P * stride
 * entries; nnz: optional device int32 array of P counts (each clamped to
 * [0, stride]). mu != 0 needs momentum buffers at bind. lr, mu, wd must be
 * finite. Asynchronous. */
int tkef_update_execute(tkef_update_plan plan, const int32_t *idx, const void *val,
                        const int32_t *nnz, float lr, float mu, float wd, void *ws,
                        size_t ws_bytes, uint32_t *status, hipStream_t stream);

/* Aggregation only (Alg. 2, which returns the accumulated g~ = sum over the
 * m gathered lists, each added at its indices into a zeroed vector): writes
 * G_i into the bound tensors at every position (0 where no list names it);
 * their previous contents are not read. Same lists, value formats and
 * summation as tkef_update_execute; momentum buffers are not used.
 * Asynchronous. */
int tkef_aggregate_execute(tkef_update_plan plan, const int32_t *idx, const void *val,
                           const int32_t *nnz, void *ws, size_t ws_bytes, uint32_t *status,
                           hipStream_t stream);

/* Value format of the val arrays execute / aggregate read: TKEF_VAL_F32
 * (default) or TKEF_VAL_F16. Host only. */
int tkef_update_plan_set_value_format(tkef_update_plan plan, int32_t format);

/* Order of summation (Alg. 2 adds the gathered lists into g~ worker by
 * worker, Sec. 3.2). on = 1: every position's entries are added in that
 * order (workers p = 0..P-1, then list order within a worker), starting
 * from +0, one binary32 add at a time, so G, and with it every execute,
 * aggregate and LARS result of the plan, is bitwise reproducible and equals
 * that sequential sum. on = 0 (default): the entries of a position are
 * added in whatever order the device runs them (results within the
 * documented tolerance of the sequential sum, exact with two or fewer
 * entries per position). The ordered sum costs LDS and time (a counting
 * sort of each chunk of entries per update tile). Host only;
 * TKEF_EINVAL for other values. */
int tkef_update_plan_set_deterministic(tkef_update_plan plan, int32_t on);

/* Optional timing hook, as tkef_sparsify_plan_set_events. */
int tkef_update_plan_set_events(tkef_update_plan plan, hipEvent_t *events,
                                int32_t n_events);
const char *tkef_update_plan_launch_name(tkef_update_plan plan, int32_t i);

/* One-shot convenience: create + bind + execute + destroy (synchronizes
 * `stream` once, during bind). */
int tkef_update_workspace(const int64_t *numels, int32_t ntensors, int32_t P,
                          int64_t stride, size_t *workspace_bytes);
int tkef_sparse_aggregate_update(float *const *params, float *const *momentum,
                                 const int64_t *numels, int32_t ntensors,
                                 const int32_t *idx, const void *val, int32_t P,
                                 int64_t stride, const int32_t *nnz, float lr,
                                 float mu, float wd, void *ws, size_t ws_bytes,
                                 uint32_t *status, hipStream_t stream);
/* One-shot aggregation into the T tensors outs (create + bind + aggregate +
 * destroy; synchronizes `stream` once, during bind). val_format as above. */
int tkef_sparse_aggregate(float *const *outs, const int64_t *numels, int32_t ntensors,
                          const int32_t *idx, const void *val, int32_t val_format, int32_t P,
                          int64_t stride, const int32_t *nnz, void *ws, size_t ws_bytes,
                          uint32_t *status, hipStream_t stream);

/* Aggregate + update over P separate worker lists (the lists that Alg. 2
 * gathers from the nodes, each added at its indices, Sec. 3.2; then the
 * update of Eq. (1) above): the call shape sparse_aggregate_update(params,
 * {idx, val} x P, lr). idx[p], val[p]: host array of P device pointers, worker
 * p's nnz[p] global positions (int32, ascending, repeats summed) and binary32
 * values; nnz: host array of P counts (>= 0; a list with nnz[p] == 0 may have
 * null pointers). params / momentum / numels / lr / mu / wd as in
 * tkef_sparse_aggregate_update (momentum may be NULL iff mu == 0; mu == wd
 * == 0 takes the sparse plain step). ws: at least tkef_aggregate_workspace();
 * the host arrays are staged into it (a table of 32 bytes per worker).
 * Synchronizes `stream` once; the library allocates nothing. */
int tkef_aggregate_workspace(const int64_t *numels, int32_t ntensors, int32_t P,
                             size_t *workspace_bytes);
int tkef_aggregate_update(float *const *params, float *const *momentum,
                          const int64_t *numels, int32_t ntensors,
                          const int32_t *const *idx, const float *const *val,
                          const int64_t *nnz, int32_t P, float lr, float mu, float wd,
                          void *ws, size_t ws_bytes, uint32_t *status, hipStream_t stream);

/* ========================================================================
 * LARS (Eq. lars: the layer-wise rate rate_l = gamma * eta * ||w_l|| /
 * (||g_l|| + eps * ||w_l||), eps being the weight decay; the step is the one
 * of the LARS method the paper cites)
 *
 * A layer is one tensor of the update plan's list. Norms are Euclidean, summed
 * in double (in a fixed order: the same inputs give the same rates on every
 * run); gamma, eta and eps enter the rate in double, and eps (the weight
 * decay) must be >= 0. The rate is the equation's value wherever its
 * denominator is positive: 0 for ||w_l|| = 0 < ||g_l||, gamma * eta / eps for
 * ||g_l|| = 0 < ||w_l||. A zero denominator (g_l = 0 and eps * w_l = 0, where
 * the equation is undefined) gives rate 0; D below is then zero, so the step
 * does not depend on it. The step, in binary32 with the rate and eps each
 * rounded to binary32 once, for every position:
 *   D = g + eps * w;  U = rate * D;
 *   with momentum (mu != 0, momentum bound):  b = mu * b + U;  w = w - b
 *   without:                                  w = w - U
 * ====================================================================== */

/* Fused sparse aggregate + LARS step: g is the sum of the P workers' lists
 * (the layout and value format of tkef_update_execute). Four kernels: seg,
 * lars_norm (the tile sums and the partial norms), lars_rates, lars_step
 * (names from tkef_lars_launch_name(0, i); the timing hook of
 * tkef_update_plan_set_events takes 5 events). rate_out: optional device
 * array of ntensors doubles receiving the rates. mu != 0 needs momentum
 * buffers bound. TKEF_ERANGE for non-finite gamma, eta, eps or mu, or eps < 0. */
int tkef_lars_update_execute(tkef_update_plan plan, const int32_t *idx, const void *val,
                             const int32_t *nnz, double gamma, double eta, double eps,
                             float mu, double *rate_out, void *ws, size_t ws_bytes,
                             uint32_t *status, hipStream_t stream);

/* Dense gradients for tkef_lars_rates_execute: grads[t] (host array of device
 * pointers, non-null where numel > 0), same sizes as the bound parameters.
 * Host; copies a pointer table into ws and synchronizes `stream`. ws must be
 * the bound workspace (TKEF_ESTATE otherwise); a later bind forgets them. */
int tkef_update_plan_bind_grads(tkef_update_plan plan, const float *const *grads, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/* The layer-wise rates from the bound parameters and dense gradients (the
 * computation the paper distributes over GPUs layer by layer, Sec. 4.2: one
 * GPU's share is a plan over its layers). rate_out: device array of
 * ntensors doubles. Two kernels (tkef_lars_launch_name(1, i)). */
int tkef_lars_rates_execute(tkef_update_plan plan, double gamma, double eta, double eps,
                            double *rate_out, void *ws, size_t ws_bytes, hipStream_t stream);

/* Kernel names of the LARS executions: dense = 0 for tkef_lars_update_execute
 * (i = 0..3), 1 for tkef_lars_rates_execute (i = 0..1); NULL otherwise. */
const char *tkef_lars_launch_name(int32_t dense, int32_t i);

#ifdef __cplusplus
}
#endif

#endif /* TKEF_H */
