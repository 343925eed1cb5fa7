// The learning-rate schedule shared by host and device code (lsgd_lr_at,
// lsgd_lr_schedule_step). Included by lsgd_flat.hip only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsgd {

// Learning-rate schedule (linear scaling, warmup, step decay), evaluated in
// binary64 and rounded to binary32 once. Shared by the host function and the
// device step so that both give the same bits.
struct Schedule {
    double base_lr, base_batch, global_batch;
    int64_t warmup_iters, decay_iters;
    double decay_factor;
};

__host__ __device__ inline float schedule_lr(const Schedule& c, int64_t t) {
    const double target = c.base_lr * (c.global_batch / c.base_batch);
    double lr = target;
    if (c.warmup_iters > 0 && t < c.warmup_iters)
        lr = c.base_lr + (target - c.base_lr) * (static_cast<double>(t) / static_cast<double>(c.warmup_iters));
    if (c.decay_iters > 0) {
        const int64_t k = t / c.decay_iters;
        double f = 1.0;
        for (int64_t i = 0; i < k; ++i) f = f * c.decay_factor;
        lr = lr * f;
    }
    return static_cast<float>(lr);
}

// One lane reads the iteration, writes its rate and advances the counter.
static __global__ __launch_bounds__(64) void schedule_step_kernel(Schedule c, int64_t* iteration,
                                                                  float* lr_out) {
    if (threadIdx.x == 0) {
        const int64_t t = *iteration;
        *lr_out = schedule_lr(c, t);
        *iteration = t + 1;
    }
}

}  // namespace lsgd
