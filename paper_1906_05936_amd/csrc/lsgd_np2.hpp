// Compile-time (W, G) kernels for group counts G = 3, 5, 6, 7 and 12 (groups
// of 1 to 8, 12, 16 or 32 workers, N = W*G <= 128): the same kernels as for
// power-of-two counts (the group tree unrolled or streamed through the
// pairwise accumulator, the division by G a true division), instantiated in
// translation units of their own so that they compile in parallel with the
// others. Each picker returns a null kernel for a grouping it does not cover.
#pragma once

#include "lsgd_host.hpp"
#include "lsgd_kernels.hpp"

namespace lsgd {

struct PlanArgs;
struct LarsArgs;

struct Np2FlatPick {
    void (*kernel)(StepArgs);
    int tile;
};
Np2FlatPick pick_flat_np2(int W, int G, bool cached, bool bf16);

struct Np2PlanPick {
    void (*kernel)(PlanArgs);
    int tile;
};
Np2PlanPick pick_plan_np2(int W, int G, bool cached, bool bf16);

using Np2LarsKernel = void (*)(LarsArgs);
Np2LarsKernel pick_lars_np2(int W, int G, bool bf16);

}  // namespace lsgd
