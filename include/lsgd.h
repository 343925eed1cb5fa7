/*
 * lsgd.h - C ABI of liblsgd.so: the Layered SGD gradient aggregation and
 * momentum-SGD update on one AMD Instinct MI355X (gfx950).
 *
 * Method: K. Yu, T. Flynn, S. Yoo, N. D'Imperio, "Layered SGD: A Decentralized
 * and Synchronous SGD Algorithm for Scalable Deep Neural Network Training",
 * arXiv 1906.05936. N = G*W workers each hold a gradient of the flat parameter
 * vector w (Sec. 3, Alg. 2: Δw^i of worker i). The workers are partitioned into G
 * equal subgroups (the inputs Alg. 3 declares: worker index i, node index j of G nodes;
 * Sec. 3: equal-cardinality partition). Per element, with PW the fixed pairwise
 * sum described below:
 *
 *   group mean   m_j  = PW(g_{members[j][0]}, ..., g_{members[j][W-1]}) / W
 *                       (Alg. 3: Reduce to the communicator and divide; Sec. 4.1 item 1)
 *   global mean  gbar = PW(m_0, ..., m_{G-1}) / G
 *                       (Alg. 3: Allreduce over communicators; Sec. 4.1 item 2)
 *   update       d = gbar + weight_decay*w;  v = momentum_coef*v + d;  w = w - lr*v
 *                       (Alg. 3 update step, the epsilon-step of Alg. 1/2, with the
 *                        momentum and weight decay of Sec. 5.3)
 *   copy-out     replica_r = w   (or w rounded to bfloat16, nearest-even)
 *                       (Alg. 3: Broadcast to the workers from the communicator)
 *
 * PW(x[0..k)) = x[0] if k == 1, else PW(x[0..h)) + PW(x[h..k)) with h the largest
 * power of two below k. Members of a group are taken in ascending worker id and
 * groups in ascending group id. All arithmetic is binary32, each operation
 * rounded to nearest-even, no fused multiply-add, subnormals kept; bf16
 * gradients widen to binary32 exactly. Results are therefore deterministic and
 * independent of launch shape. With W and G powers of two the two-level mean
 * equals the flat mean over all N workers bit for bit (Sec. 4.2: Algorithms 2
 * and 3 reach the same parameters).
 *
 * Conventions shared by every call:
 *  - Memory. Every buffer argument is caller-owned device memory on the current
 *    HIP device. Pointer ARRAYS (grads, replicas, group_means) are host arrays of
 *    device pointers, read during the call only. The library keeps no pointer
 *    after a call returns, except inside a plan.
 *  - Streams. `stream` is a hipStream_t (NULL = the null stream). Calls validate,
 *    enqueue on `stream` and return without synchronizing; outputs are ready when
 *    the stream reaches that point.
 *  - Validation happens before anything is enqueued. On any error nothing is
 *    launched and no output is touched. n == 0 is a no-op that returns LSGD_OK
 *    after the counts, dtypes and membership are validated (pointers may then
 *    be NULL).
 *  - Alignment. Every buffer must be 16-byte aligned (LSGD_ERR_ALIGN). For
 *    bandwidth, give all buffers of a call the same offset modulo 2 MB (as
 *    separate large allocations have): buffers packed back to back at
 *    arbitrary offsets measured up to 13% slower on MI355X.
 *  - Aliasing. Written buffers may not overlap each other or any read buffer
 *    (LSGD_ERR_ALIAS). Read buffers may overlap each other (several workers may
 *    pass the same gradient buffer).
 *  - Non-finite values are not checked; NaN and Inf propagate.
 *  - Thread safety. Calls on distinct streams and buffers may run concurrently.
 *    lsgd_last_error() is per thread.
 */
#ifndef LSGD_H
#define LSGD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define LSGD_API __attribute__((visibility("default")))
#else
#define LSGD_API
#endif

typedef enum lsgd_status {
    LSGD_OK = 0,
    LSGD_ERR_NULL = 1,   /* a required pointer (or pointer-array entry) is NULL        */
    LSGD_ERR_SIZE = 2,   /* n < 0, or a count < 1 (< 0 for replicas) or above its max  */
    LSGD_ERR_GROUPS = 3, /* group id out of [0,G), G does not divide N, unequal groups */
    LSGD_ERR_ALIGN = 4,  /* a buffer is not 16-byte aligned                            */
    LSGD_ERR_DTYPE = 5,  /* dtype is not one of lsgd_dtype                             */
    LSGD_ERR_HIP = 6,    /* the HIP runtime reported an error; see lsgd_last_error()   */
    LSGD_ERR_ALIAS = 7,  /* a written buffer overlaps another buffer of the call       */
    LSGD_ERR_UNSUPPORTED = 8 /* an option value or combination this call does not take */
} lsgd_status;

typedef enum lsgd_dtype {
    LSGD_F32 = 0,  /* IEEE binary32                                        */
    LSGD_BF16 = 1  /* bfloat16: the upper 16 bits of a binary32, as uint16 */
} lsgd_dtype;

/* Planless calls carry their pointer tables in the kernel arguments, so every
 * call accepts at most this many workers (hence groups) and replicas; plans
 * keep the same limits. */
#define LSGD_MAX_WORKERS 128
#define LSGD_MAX_REPLICAS 128

/* Static, never-NULL text for a status. */
LSGD_API const char* lsgd_status_string(lsgd_status status);

/* Detail of the last failing call made by this thread ("" if none). The
 * string stays valid until the next failing call on this thread. */
LSGD_API const char* lsgd_last_error(void);

/*
 * Launch shape of the planless kernels, process-wide (a tuning knob; results
 * of the steps are bit-identical for every shape, because each element is
 * computed by one lane from its own inputs in a fixed order). Plans launch one
 * workgroup per bucket: xcd_chunk applies at each lsgd_step_plan, units_per_lane
 * at lsgd_plan_create, blocks_per_cu only to their copy-out pass. The one
 * result that can depend on a shape is a LARS trust ratio
 * (lsgd_lars_step_plan): its norms are summed piece by piece, and a plan's
 * piece size is fixed by units_per_lane when the plan is created, so plans
 * created with different units_per_lane may give ratios (and hence LARS
 * steps) that differ in the last bit; for one plan, LARS results do not
 * depend on the shape.
 *   xcd_chunk       0 = workgroups in hardware order; C > 0 = each of the eight
 *                   XCDs runs C consecutive logical workgroups per turn (the grid
 *                   is padded to a multiple of 8*C; not applied to grids smaller
 *                   than 8*C); LSGD_XCD_CHUNK_AUTO (-1) = the C that gives each
 *                   XCD 512 KB of every buffer per turn. Range [-1, 65536].
 *   blocks_per_cu   0 = the grid covers the work; B > 0 = at most B workgroups per
 *                   compute unit, grid-stride. Range [0, 4096].
 *   units_per_lane  P: a workgroup walks P consecutive passes of its lane tiles
 *                   (256 lanes, each a tile of one or two 16-byte units) of
 *                   every buffer; plans created while P is set cut tensors into
 *                   pieces of P passes. Range [1, 256].
 * Defaults: xcd_chunk LSGD_XCD_CHUNK_AUTO, blocks_per_cu 0, units_per_lane 1.
 * Takes effect for
 * launches made after the call returns. Errors: LSGD_ERR_SIZE (out of range),
 * LSGD_ERR_NULL (get).
 */
#define LSGD_XCD_CHUNK_AUTO (-1)
LSGD_API lsgd_status lsgd_set_launch_shape(int32_t xcd_chunk, int32_t blocks_per_cu,
                                           int32_t units_per_lane);
LSGD_API lsgd_status lsgd_get_launch_shape(int32_t* xcd_chunk, int32_t* blocks_per_cu,
                                           int32_t* units_per_lane);

/* Where the steps (lsgd_step, lsgd_step_ex, lsgd_step_plan*, lsgd_sgd_step)
 * write their replicas (the copy-out, Alg. 3 broadcast step): inside the step
 * kernel, or in a copy-out pass of their own launched right after it on the
 * same stream, which reads the new parameters once more (4 bytes per element,
 * mostly from cache) and writes the replicas one window of the vector at a
 * time. Results are identical either way. LSGD_COPY_OUT_AUTO (the default)
 * takes the separate pass where it measured faster: for the fused steps when
 * the replica bytes R*s_r per element are at least 32 (for at most 16
 * workers with parameters and momentum within 288 MB, whose step kernels
 * access them through the caches: 64 for power-of-two groups in a
 * power-of-two count, 48 for every other group layout) or the gradient bytes
 * N*s_g at least 256;
 * for lsgd_sgd_step and the LARS update when R*s_r >= 16 (parameters and
 * momentum within 288 MB; beyond, binary32 replicas and R >= 4).
 * Process-wide, for launches after the call returns. Errors: LSGD_ERR_SIZE
 * (unknown mode). A tuning and measurement knob. */
#define LSGD_COPY_OUT_AUTO (-1)
#define LSGD_COPY_OUT_FUSED 0
#define LSGD_COPY_OUT_SEPARATE 1
LSGD_API lsgd_status lsgd_set_copy_out_mode(int32_t mode);
LSGD_API int32_t lsgd_get_copy_out_mode(void);

/* Where the fused steps (lsgd_step, lsgd_step_ex, lsgd_step_plan*) take the
 * separate copy-out form: the step kernel still writes the first `replicas`
 * replicas itself (fewer if the step has fewer) and the copy-out pass writes
 * the rest. -1 (the default) is the automatic choice: 16 bytes of replicas per
 * element (4 binary32 or 8 bfloat16 replicas) for steps with at most 16
 * workers whose parameters and momentum fit in 288 MB, none otherwise (the
 * step kernel's mostly-read stream mix takes a few write streams at little
 * cost; measured fastest). Results are identical for every value.
 * Process-wide, for launches after the call returns. Errors: LSGD_ERR_SIZE
 * (outside [-1, LSGD_MAX_REPLICAS]). A tuning and measurement knob. */
LSGD_API lsgd_status lsgd_set_step_replicas(int32_t replicas);
LSGD_API int32_t lsgd_get_step_replicas(void);

/*
 * The local layer alone (Alg. 3, Reduce to the communicator and divide):
 *   group_means[j][i] = PW over the W members of group j of grads[w][i], / W.
 * grads          [n_workers] device pointers, each n elements of dtype gdt.
 * group_of_worker[n_workers] host int32, the group of each worker, in [0, n_groups).
 * group_means    [n_groups] device pointers, each n binary32 elements (written).
 * 1 <= n_workers <= LSGD_MAX_WORKERS; n_groups divides n_workers and every group
 * has exactly n_workers/n_groups members.
 */
LSGD_API lsgd_status lsgd_group_mean(const void* const* grads, lsgd_dtype gdt,
                                     int32_t n_workers, const int32_t* group_of_worker,
                                     int32_t n_groups, int64_t n,
                                     float* const* group_means, void* stream);

/*
 * The global layer alone (Alg. 3, Allreduce over communicators), as a mean:
 *   grad_mean[i] = PW(group_means[0][i], ..., group_means[n_groups-1][i]) / n_groups.
 * group_means [n_groups] device pointers to n binary32 each; grad_mean n binary32
 * (written). 1 <= n_groups <= LSGD_MAX_WORKERS.
 */
LSGD_API lsgd_status lsgd_global_mean(const float* const* group_means, int32_t n_groups,
                                      int64_t n, float* grad_mean, void* stream);

/*
 * The update and copy-out alone (Alg. 3 update step and Broadcast; momentum and
 * weight decay of Sec. 5.3), in place on params and momentum (n binary32 each):
 *   d = grad_mean + weight_decay*params; momentum = momentum_coef*momentum + d;
 *   params = params - lr*momentum; replicas[r] = params (dtype rdt).
 * replicas: host array of n_replicas device pointers (may be NULL when
 * n_replicas == 0), each n elements of dtype rdt. 0 <= n_replicas <= LSGD_MAX_REPLICAS.
 * A fresh momentum buffer is zero-filled by the caller.
 */
LSGD_API lsgd_status lsgd_sgd_step(float* params, float* momentum, const float* grad_mean,
                                   int64_t n, float lr, float momentum_coef,
                                   float weight_decay, void* const* replicas,
                                   int32_t n_replicas, lsgd_dtype rdt, void* stream);

/*
 * The copy-out alone (Alg. 3 Broadcast of the updated parameters to the
 * workers; e.g. after restoring params):
 *   replicas[r][i] = params[i] (binary32) or params[i] rounded to bfloat16,
 *   nearest-even (rdt LSGD_BF16), for r < n_replicas.
 * params: n binary32 (read). replicas: host array of n_replicas device
 * pointers (may be NULL when n_replicas == 0), each n elements of dtype rdt,
 * written. 0 <= n_replicas <= LSGD_MAX_REPLICAS. Always the copy-out pass of
 * lsgd_set_copy_out_mode's separate form (replica-major over windows of
 * params), whatever the mode. n == 0 or n_replicas == 0 is a no-op. Errors:
 * LSGD_ERR_NULL, LSGD_ERR_SIZE, LSGD_ERR_DTYPE, LSGD_ERR_ALIGN (a buffer not
 * 16-byte aligned), LSGD_ERR_ALIAS (a replica overlapping params or another
 * replica), LSGD_ERR_HIP.
 */
LSGD_API lsgd_status lsgd_copy_out(const float* params, int64_t n, void* const* replicas,
                                   int32_t n_replicas, lsgd_dtype rdt, void* stream);

/*
 * One fused Layered SGD step: group means, global mean, update and copy-out.
 * The step kernel reads every gradient, parameter and momentum element once
 * and writes parameters and momentum once; the group means and the mean
 * gradient stay in registers. The replicas are written either by that kernel
 * or, where lsgd_set_copy_out_mode's rule takes the separate form (the
 * default with up to 16 workers at 64 or more replica bytes per element for
 * power-of-two groups in a power-of-two count, 48 for every other group
 * layout), by a copy-out
 * pass launched right after it, which reads the new parameters once more
 * (the step kernel then still writes the first lsgd_set_step_replicas
 * replicas). Vectors longer than 2^26 elements are processed range by range
 * (about 2^24 elements each, edges on multiples of 2^20 elements: the step
 * kernel, then its copy-out pass) unless the step kernel writes every
 * replica itself. Compile-time kernels (the pairwise trees unrolled) serve
 * power-of-two group counts with groups of 1 to 16 workers (a power of two,
 * or 3, 5, 6, 7 or 12), 32 to 128 workers in up to 4 groups, 32 to 128
 * groups of up to 4 workers, and 3, 5, 6, 7 or 12 groups of 1 to 8, 12, 16
 * or 32 workers (N at most 128);
 * every other grouping takes a runtime-layout kernel. Arguments as for the
 * three calls above. The results are bit-identical to lsgd_group_mean, then
 * lsgd_global_mean, then lsgd_sgd_step, in every form.
 */
LSGD_API lsgd_status lsgd_step(float* params, float* momentum, const void* const* grads,
                               lsgd_dtype gdt, int32_t n_workers,
                               const int32_t* group_of_worker, int32_t n_groups, int64_t n,
                               float lr, float momentum_coef, float weight_decay,
                               void* const* replicas, int32_t n_replicas, lsgd_dtype rdt,
                               void* stream);

/*
 * Variants of the fused step: the paper-literal form of the local layer, the
 * broadcast of the mean gradient, and a learning rate held in device memory.
 *
 * reduction
 *   LSGD_REDUCE_MEAN_OF_MEANS  as lsgd_step: equal subgroups, mean of each
 *                              group's W members, then mean of the G means.
 *   LSGD_REDUCE_LITERAL        Alg. 3 as printed: each communicator divides its
 *                              members' pairwise sum by N (all workers), the
 *                              allreduce over communicators sums (PW, ascending
 *                              group id) without a further division. Any
 *                              partition into non-empty groups (LSGD_ERR_GROUPS
 *                              for an empty group); the exact value is the flat
 *                              mean of Alg. 2 for every partition, and for equal
 *                              power-of-two groups the bits equal lsgd_step's.
 * broadcast_grad
 *   nonzero: every worker's gradient buffer receives the mean gradient in
 *   place (Alg. 3 Broadcast of the gathered gradient, Sec. 4.1 item 3: what the
 *   allreduce-and-divide of Alg. 2 leaves in each worker). binary32 gradients
 *   only (LSGD_ERR_DTYPE); the gradient buffers are then written buffers and may
 *   not overlap each other or any other buffer (LSGD_ERR_ALIAS).
 * lr_device
 *   non-NULL: the learning rate is read from this device address (4-byte
 *   aligned, LSGD_ERR_ALIGN) when the kernel runs, and the lr argument is
 *   ignored; with lsgd_lr_schedule_step in the same stream a captured HIP graph
 *   of whole steps follows the schedule on every replay.
 * A zero-initialised struct (or options == NULL) is lsgd_step.
 */
typedef enum lsgd_reduction {
    LSGD_REDUCE_MEAN_OF_MEANS = 0,
    LSGD_REDUCE_LITERAL = 1
} lsgd_reduction;

typedef struct lsgd_step_options {
    int32_t reduction;       /* lsgd_reduction                                  */
    int32_t broadcast_grad;  /* nonzero: write the mean gradient into every grad */
    const float* lr_device;  /* NULL: use the lr argument                       */
} lsgd_step_options;

LSGD_API lsgd_status lsgd_step_ex(float* params, float* momentum, void* const* grads,
                                  lsgd_dtype gdt, int32_t n_workers,
                                  const int32_t* group_of_worker, int32_t n_groups, int64_t n,
                                  float lr, float momentum_coef, float weight_decay,
                                  void* const* replicas, int32_t n_replicas, lsgd_dtype rdt,
                                  const lsgd_step_options* options, void* stream);

/*
 * Learning-rate schedule of Sec. 5.3: linear scaling (the target rate is
 * base_lr * global_batch / base_batch: 0.1 at 256, 6.4 at 16,384 in the paper),
 * a linear warmup from base_lr to the target over warmup_iters iterations
 * (0 = none), and a multiplication by decay_factor every decay_iters
 * iterations counted from the start (0 = never; 0.1 every 30 epochs in the
 * paper). Evaluated in binary64 and rounded to binary32 once:
 *   lr(t) = (t < warmup_iters ? base_lr + (target - base_lr) * (t / warmup_iters)
 *                             : target) * decay_factor^(t / decay_iters)
 * with the power taken as a running product of decay_factor terms.
 */
typedef struct lsgd_lr_schedule {
    double base_lr;
    double base_batch;
    double global_batch;
    int64_t warmup_iters;
    int64_t decay_iters;
    double decay_factor;
} lsgd_lr_schedule;

/* The schedule's rate for iteration t, on the host (same operations and bits as
 * the device step). Returns NaN for a NULL schedule, base_batch <= 0, or
 * negative t, warmup_iters or decay_iters. */
LSGD_API float lsgd_lr_at(const lsgd_lr_schedule* schedule, int64_t t);

/* Device-side schedule step, stream-ordered: lr_out[0] = lr(iteration[0]), then
 * iteration[0] += 1. iteration: device int64 (8-byte aligned), lr_out: device
 * float (4-byte aligned). The schedule struct is copied at the call. Errors:
 * LSGD_ERR_NULL, LSGD_ERR_ALIGN, LSGD_ERR_SIZE (invalid schedule fields). */
LSGD_API lsgd_status lsgd_lr_schedule_step(const lsgd_lr_schedule* schedule, int64_t* iteration,
                                           float* lr_out, void* stream);

/*
 * Multi-tensor plan: the fused step over a model's list of parameter tensors
 * (e.g. the 161 tensors of ResNet-50, the model of Sec. 5.3) in ONE kernel
 * launch. The plan copies a chunk table and a pointer table to device memory
 * once; lsgd_step_plan then launches one kernel. Tensors are cut into pieces
 * of 2048 elements (4096 for binary32 gradients with more than 16 workers in
 * a grouping with a compile-time kernel, as listed for lsgd_step, except 32
 * or more groups and 16 groups of 3 or 4; times the launch shape's
 * units_per_lane at creation);
 * small tensors are bucketed so that one workgroup covers several of them.
 *   numel     [n_tensors] host int64, elements of each tensor (>= 0).
 *   params, momentum [n_tensors] device pointers (binary32).
 *   grads     [n_workers * n_tensors] device pointers, worker-major:
 *             grads[w * n_tensors + t] is worker w's gradient of tensor t.
 *   replicas  [n_replicas * n_tensors] device pointers, replica-major, or NULL
 *             when n_replicas == 0.
 * The plan holds the pointers: the tensors must stay allocated, unmoved, while
 * the plan is used. Counts: n_tensors >= 1, 1 <= n_workers <= LSGD_MAX_WORKERS,
 * 0 <= n_replicas <= LSGD_MAX_REPLICAS. group_of_worker may be any partition
 * into n_groups non-empty groups (LSGD_ERR_GROUPS otherwise); the default
 * mean-of-means step and the LARS step need equal group sizes and return
 * LSGD_ERR_GROUPS on a plan whose groups differ, which takes the paper-literal
 * reduction (lsgd_step_plan_ex). The plan is bound to the device current at
 * creation.
 * lsgd_plan_create allocates device memory (LSGD_ERR_HIP if that fails) and
 * synchronizes the null stream once; lsgd_step_plan allocates nothing.
 */
typedef struct lsgd_plan lsgd_plan;

LSGD_API lsgd_status lsgd_plan_create(lsgd_plan** out, int32_t n_tensors, const int64_t* numel,
                                      float* const* params, float* const* momentum,
                                      const void* const* grads, lsgd_dtype gdt,
                                      int32_t n_workers, const int32_t* group_of_worker,
                                      int32_t n_groups, void* const* replicas,
                                      int32_t n_replicas, lsgd_dtype rdt);

LSGD_API lsgd_status lsgd_step_plan(const lsgd_plan* plan, float lr, float momentum_coef,
                                    float weight_decay, void* stream);

/* lsgd_step_plan with options, as lsgd_step_ex: the paper-literal reduction
 * (any partition), the gradient broadcast (binary32 gradients only, else
 * LSGD_ERR_DTYPE; every worker's gradient tensors are then written, so none
 * may overlap another buffer of the plan: LSGD_ERR_ALIAS) and lr_device.
 * Errors as lsgd_step_plan, plus LSGD_ERR_UNSUPPORTED (unknown reduction),
 * LSGD_ERR_GROUPS (mean of means on unequal groups), LSGD_ERR_ALIGN. */
LSGD_API lsgd_status lsgd_step_plan_ex(const lsgd_plan* plan, float lr, float momentum_coef,
                                       float weight_decay, const lsgd_step_options* options,
                                       void* stream);

/* The copy-out alone over a plan (Alg. 3 Broadcast; lsgd_copy_out for every
 * tensor): each replica tensor = its params tensor (binary32, or bfloat16
 * nearest-even), in one launch of the plan's copy-out pass. No-op for a plan
 * without replicas. Errors: LSGD_ERR_NULL (plan NULL), LSGD_ERR_HIP (wrong
 * device, launch failure). */
LSGD_API lsgd_status lsgd_plan_copy_out(const lsgd_plan* plan, void* stream);

/* ---- LARS on a plan: one trust ratio per tensor -------------------------
 *
 * The paper names layer-wise adaptive rate scaling (LARS) as compatible with
 * LSGD (Sec. 2) and as future work (Sec. 6) without defining it; the step
 * follows You, Gitman and Ginsburg, "Large Batch Training of Convolutional
 * Networks" (arXiv 1708.03888, eq. 6 and Alg. 1). Per tensor t of the plan,
 * with gbar the aggregated gradient of lsgd_step (mean of the G subgroup
 * means, same pairwise order) and p the parameters before the step:
 *   trust_t = trust_coef * ||p|| / (||gbar|| + weight_decay * ||p||),
 *             1 when ||p|| or ||gbar|| is zero;
 *   d = trust_t * (gbar + weight_decay * p);  m = momentum_coef * m + d;
 *   p = p - lr * m;  replicas = p (binary32 or nearest-even bfloat16).
 * Norms: sums of squares, square roots and the ratio in binary64, rounded
 * once to binary32 (the sums run in a fixed blocked order, so a trust ratio
 * can differ from a sequential binary64 evaluation only by the last bit in
 * rare cases). The elementwise operations are binary32, each rounded, no
 * fused multiply-add. lr sits outside the momentum (the heavy-ball form of
 * lsgd_step); with a constant lr this is the LARS paper's update.
 *
 * The step runs three kernels on `stream`: the mean gradient plus per-chunk
 * binary64 partial norms, the per-tensor trust ratios, then the update and
 * copy-out (the copy-out as a fourth kernel where lsgd_set_copy_out_mode's
 * rule for lsgd_sgd_step picks the separate pass). The workspace is caller-owned device memory of at least
 * lsgd_lars_workspace_size bytes, 256-byte aligned, that must not overlap any
 * buffer of the plan or trust_out; it holds the mean gradient (4 bytes per
 * element), the partial norms and the trust ratios, and its contents are not
 * needed between calls. Calls sharing a workspace must be ordered on one
 * stream. trust_out (optional, device, n_tensors floats, 4-byte aligned)
 * receives the trust ratios. lr_device (optional, device, 4-byte aligned):
 * when non-NULL the update reads the global rate there when it runs and `lr`
 * is ignored, as in lsgd_step_ex (so a captured graph can follow
 * lsgd_lr_schedule_step). Errors: LSGD_ERR_NULL (plan or workspace NULL),
 * LSGD_ERR_SIZE (workspace too small), LSGD_ERR_ALIGN, LSGD_ERR_ALIAS,
 * LSGD_ERR_HIP (wrong device or launch failure); nothing is launched on an
 * argument error. */
LSGD_API lsgd_status lsgd_lars_workspace_size(const lsgd_plan* plan, size_t* bytes);

LSGD_API lsgd_status lsgd_lars_step_plan(const lsgd_plan* plan, float lr, float momentum_coef,
                                         float weight_decay, float trust_coef, void* workspace,
                                         size_t workspace_bytes, float* trust_out,
                                         const float* lr_device, void* stream);

/*
 * lsgd_lars_step_plan without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc. The scratch that lsgd_lars_step_plan keeps in the
 * caller's workspace (the mean gradient, the partial norms and the trust
 * ratios) lives instead in an array owned by the library, of
 * LSGD_NOALLOC_SCRATCH_BYTES (128 MiB) on each device, which each device the
 * call runs on holds until the process ends. The call makes no allocation
 * (no hipMalloc, no host heap), launches the same kernels and gives the same
 * results, bit for bit. Plans whose lsgd_lars_workspace_size exceeds
 * LSGD_NOALLOC_SCRATCH_BYTES (about 33 million elements; ResNet-50's 25.6
 * million fit) are rejected with LSGD_ERR_SIZE and nothing is launched. Every
 * call on one device uses that device's one array and leaves its contents
 * there; no call needs them (every byte a call reads is written earlier in
 * the same call), but calls whose kernels may overlap on one device (other
 * streams, other host threads) race on it: order them on one stream. The
 * first call on a device looks the array up there (hipGetSymbolAddress; a
 * failure is LSGD_ERR_HIP). Other arguments and errors as
 * lsgd_lars_step_plan; trust_out and lr_device may not overlap the plan's
 * written buffers (LSGD_ERR_ALIAS).
 */
#define LSGD_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
LSGD_API lsgd_status lsgd_lars_step_plan_noalloc(const lsgd_plan* plan, float lr, float momentum_coef,
                                                 float weight_decay, float trust_coef, float* trust_out,
                                                 const float* lr_device, void* stream);

/* Tensors excluded from the layer-wise rates: exclude[t] != 0 gives tensor t
 * trust 1 in every later lsgd_lars_step_plan (so its update is the plain
 * step of lsgd_step_plan); NULL clears every exclusion. Implementations
 * commonly exclude biases and batch-normalisation parameters; the paper names
 * no exclusions, and a new plan excludes nothing. exclude is a host array of
 * n_tensors bytes. Copies to device memory synchronously: call it between
 * steps, not inside a captured graph. Errors: LSGD_ERR_NULL (plan),
 * LSGD_ERR_HIP (wrong device or copy failure). */
LSGD_API lsgd_status lsgd_plan_set_lars_exclude(lsgd_plan* plan, const uint8_t* exclude);

/* Frees the plan's device tables. NULL-safe. The caller synchronizes every
 * stream that ran lsgd_step_plan or lsgd_lars_step_plan with this plan first. */
LSGD_API void lsgd_plan_destroy(lsgd_plan* plan);

#ifdef __cplusplus
}
#endif

#endif /* LSGD_H */
