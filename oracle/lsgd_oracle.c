/*
 * CPU oracle for the Layered SGD gradient aggregation and parameter update.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this code. It shares no source, header,
 * table or helper with the GPU library, and the GPU library never calls it.
 *
 * Source: K. Yu, T. Flynn, S. Yoo, N. D'Imperio, "Layered SGD: A Decentralized
 * and Synchronous SGD Algorithm for Scalable Deep Neural Network Training",
 * arXiv 1906.05936.
 *
 * What is computed, per parameter element, with N = G*W workers:
 *   1. subgroup means   m_j  = PW(g_{members[j][0..W)}) / W       (Alg. 3, reduce
 *                             step at the communicator; Sec. 4.1 flow item 1)
 *   2. global mean      gbar = PW(m_0 .. m_{G-1}) / G              (Alg. 3, allreduce
 *                             step among communicators; Sec. 4.1 flow item 2)
 *   3. update           d = gbar + wd*p;  mom = mu*mom + d;  p = p - lr*mom
 *                             (Alg. 3 update step, in the epsilon-step form of
 *                             Alg. 1/2; momentum and weight decay from Sec. 5.3)
 *   4. copy-out         replica_r = p  (or its bfloat16 rounding)
 *                             (Alg. 3, broadcast step from the communicator to its workers)
 *   LARS (optional)     step 3 with d scaled by a per-tensor trust ratio (Sec. 2 and
 *                             Sec. 6 name LARS; its definition follows the LARS paper,
 *                             see oracle_lars_trust)
 * PW is the pairwise sum: PW(x[0..k)) = x[0] if k == 1, else
 * PW(x[0..h)) + PW(x[h..k)) with h the largest power of two below k. Members of a
 * group are taken in ascending worker id, groups in ascending group id. Equal
 * group sizes are required (Sec. 3: the minibatch partition has equal
 * cardinality, so every worker gradient carries equal weight).
 *
 * The paper fixes neither the summation order nor the momentum formula; the
 * readings taken here (pairwise order, divide by W then by G, heavy-ball
 * momentum with coupled L2 weight decay, momentum buffer starting at +0) are
 * the ones listed in the design notes of this repository.
 *
 * Built twice from oracle_real.inc: REAL=float (the parity oracle: every
 * operation rounded to nearest-even in binary32, no fused multiply-add, no
 * reassociation, subnormals kept; compile with -ffp-contract=off and without
 * -ffast-math) and REAL=double (only used to pin the binary32 build against
 * closed forms and error bounds).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Status codes of the oracle (its own; the GPU library has its own set). */
enum { ORACLE_OK = 0, ORACLE_ERR_NULL = 1, ORACLE_ERR_SIZE = 2, ORACLE_ERR_GROUPS = 3,
       ORACLE_ERR_DTYPE = 5 };

/* Gradient / replica element types. */
enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

/*
 * Subgroup indexing (the inputs Alg. 3 declares: worker index i of N, node index j of G;
 * Sec. 3: equal-cardinality partition; Sec. 5.1: four workers per node).
 * group_of_worker[i] in [0, G) names worker i's group. On success members holds
 * G rows of W = N/G worker ids, each row in ascending worker id.
 * Errors: NULL pointer, N < 1 or G < 1, an id out of range, G not dividing N,
 * or any group with a member count other than W.
 */
int oracle_members(int32_t n_workers, const int32_t* group_of_worker, int32_t n_groups,
                   int32_t* members)
{
    if (!group_of_worker || !members) return ORACLE_ERR_NULL;
    if (n_workers < 1 || n_groups < 1) return ORACLE_ERR_SIZE;
    if (n_workers % n_groups != 0) return ORACLE_ERR_GROUPS;
    int32_t W = n_workers / n_groups;
    for (int32_t i = 0; i < n_workers; ++i)
        if (group_of_worker[i] < 0 || group_of_worker[i] >= n_groups) return ORACLE_ERR_GROUPS;
    for (int32_t j = 0; j < n_groups; ++j) {
        int32_t count = 0;
        for (int32_t i = 0; i < n_workers; ++i) {
            if (group_of_worker[i] == j) {
                if (count == W) return ORACLE_ERR_GROUPS;
                members[(int64_t)j * W + count] = i;
                ++count;
            }
        }
        if (count != W) return ORACLE_ERR_GROUPS;
    }
    return ORACLE_OK;
}

/* bfloat16 bits -> binary32: the bf16 value is the top half of a binary32. */
float oracle_bf16_to_f32(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return f;
}

/*
 * binary32 -> bfloat16, round to nearest, ties to even, written from the
 * definition: keep the upper 16 bits, then compare the dropped lower 16 bits of
 * the magnitude with half a bf16 unit (0x8000). Above half rounds the magnitude
 * up (a carry into the exponent is the correct next binade, or infinity); exactly
 * half rounds up only when the kept bits are odd. NaN maps to a quiet NaN of the
 * same sign.
 */
uint16_t oracle_f32_to_bf16(float f)
{
    uint32_t b;
    memcpy(&b, &f, sizeof b);
    if ((b & 0x7f800000u) == 0x7f800000u && (b & 0x007fffffu) != 0u)
        return (uint16_t)((b >> 16) | 0x0040u);
    uint32_t kept = b >> 16;
    uint32_t dropped = b & 0xffffu;
    if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1u;
    return (uint16_t)kept;
}

/*
 * Subgroup indexing for the paper-literal reduction, which admits any
 * partition: every group needs at least one member. members holds the N
 * worker ids grouped by group id (ascending inside each group) and
 * group_start[j] .. group_start[j+1] delimits group j (G+1 entries).
 */
int oracle_partition(int32_t n_workers, const int32_t* group_of_worker, int32_t n_groups,
                     int32_t* members, int32_t* group_start)
{
    if (!group_of_worker || !members || !group_start) return ORACLE_ERR_NULL;
    if (n_workers < 1 || n_groups < 1) return ORACLE_ERR_SIZE;
    for (int32_t i = 0; i < n_workers; ++i)
        if (group_of_worker[i] < 0 || group_of_worker[i] >= n_groups) return ORACLE_ERR_GROUPS;
    int32_t at = 0;
    for (int32_t j = 0; j < n_groups; ++j) {
        group_start[j] = at;
        for (int32_t i = 0; i < n_workers; ++i)
            if (group_of_worker[i] == j) members[at++] = i;
        if (at == group_start[j]) return ORACLE_ERR_GROUPS;   /* empty group */
    }
    group_start[n_groups] = at;
    return ORACLE_OK;
}

/*
 * Learning-rate schedule of Sec. 5.3: the linear scaling rule (the rate grows
 * with the global minibatch: base_lr at base_batch, so the target is
 * base_lr * global_batch / base_batch), a warmup that raises the rate from
 * base_lr to the target linearly at every iteration over warmup_iters
 * iterations, and a decay by decay_factor every decay_iters iterations
 * (every 30 epochs in the paper). Computed in binary64, rounded to binary32
 * once at the end; the decay power is a product of decay_factor terms.
 */
float oracle_lr_at(int64_t t, double base_lr, double base_batch, double global_batch,
                   int64_t warmup_iters, int64_t decay_iters, double decay_factor)
{
    double target = base_lr * (global_batch / base_batch);
    double lr = target;
    if (warmup_iters > 0 && t < warmup_iters)
        lr = base_lr + (target - base_lr) * ((double)t / (double)warmup_iters);
    if (decay_iters > 0) {
        int64_t k = t / decay_iters;
        double f = 1.0;
        for (int64_t i = 0; i < k; ++i) f = f * decay_factor;
        lr = lr * f;
    }
    return (float)lr;
}

#define REAL float
#define SFX(name) name##_f32
#include "oracle_real.inc"
#undef REAL
#undef SFX

#define REAL double
#define SFX(name) name##_f64
#include "oracle_real.inc"
#undef REAL
#undef SFX

/* Array forms of the two bf16 conversions above, for the test harness. */
void oracle_f32_to_bf16_array(const float* x, uint16_t* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_f32_to_bf16(x[i]);
}

void oracle_bf16_to_f32_array(const uint16_t* x, float* out, int64_t n)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16_to_f32(x[i]);
}
