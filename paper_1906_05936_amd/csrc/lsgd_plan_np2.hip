// Compile-time plan step and LARS norm kernels for group counts 3, 5, 6, 7
// and 12.
#include "lsgd_host.hpp"
#include "lsgd_np2.hpp"
#include "lsgd_plan_kernels.hpp"

namespace lsgd {
namespace {

using PlanKernel = void (*)(PlanArgs);

template <typename GT, int W, int G>
PlanKernel np2_plan(bool cached) {
    constexpr int U = tile_units<GT>(W * G, G);
    if constexpr (cached_state_for(W * G))
        if (cached) return plan_step_kernel<GT, W, G, U, 1>();
    return plan_step_kernel<GT, W, G, U, 0>();
}

template <typename GT, int G>
PlanKernel np2_plan_w(int W, bool cached) {
    switch (W) {
        case 1: return np2_plan<GT, 1, G>(cached);
        case 2: return np2_plan<GT, 2, G>(cached);
        case 3: return np2_plan<GT, 3, G>(cached);
        case 4: return np2_plan<GT, 4, G>(cached);
        case 5: return np2_plan<GT, 5, G>(cached);
        case 6: return np2_plan<GT, 6, G>(cached);
        case 7: return np2_plan<GT, 7, G>(cached);
        case 8: return np2_plan<GT, 8, G>(cached);
        case 12:
            if constexpr (12 * G <= kMaxWorkers) return np2_plan<GT, 12, G>(cached);
            else return nullptr;
        case 16:
            if constexpr (16 * G <= kMaxWorkers) return np2_plan<GT, 16, G>(cached);
            else return nullptr;
        case 32:
            if constexpr (32 * G <= kMaxWorkers) return np2_plan<GT, 32, G>(cached);
            else return nullptr;
    }
    return nullptr;
}

template <typename GT, int W, int G>
Np2LarsKernel np2_lars() {
    return lars_kernel_for<GT, W, G>();
}

template <typename GT, int G>
Np2LarsKernel np2_lars_w(int W) {
    switch (W) {
        case 1: return np2_lars<GT, 1, G>();
        case 2: return np2_lars<GT, 2, G>();
        case 3: return np2_lars<GT, 3, G>();
        case 4: return np2_lars<GT, 4, G>();
        case 5: return np2_lars<GT, 5, G>();
        case 6: return np2_lars<GT, 6, G>();
        case 7: return np2_lars<GT, 7, G>();
        case 8: return np2_lars<GT, 8, G>();
        case 12:
            if constexpr (12 * G <= kMaxWorkers) return np2_lars<GT, 12, G>();
            else return nullptr;
        case 16:
            if constexpr (16 * G <= kMaxWorkers) return np2_lars<GT, 16, G>();
            else return nullptr;
        case 32:
            if constexpr (32 * G <= kMaxWorkers) return np2_lars<GT, 32, G>();
            else return nullptr;
    }
    return nullptr;
}

template <typename GT>
PlanKernel np2_plan_g(int W, int G, bool cached) {
    switch (G) {
        case 3: return np2_plan_w<GT, 3>(W, cached);
        case 5: return np2_plan_w<GT, 5>(W, cached);
        case 6: return np2_plan_w<GT, 6>(W, cached);
        case 7: return np2_plan_w<GT, 7>(W, cached);
        case 12: return np2_plan_w<GT, 12>(W, cached);
    }
    return nullptr;
}

template <typename GT>
Np2LarsKernel np2_lars_g(int W, int G) {
    switch (G) {
        case 3: return np2_lars_w<GT, 3>(W);
        case 5: return np2_lars_w<GT, 5>(W);
        case 6: return np2_lars_w<GT, 6>(W);
        case 7: return np2_lars_w<GT, 7>(W);
        case 12: return np2_lars_w<GT, 12>(W);
    }
    return nullptr;
}

}  // namespace

Np2PlanPick pick_plan_np2(int W, int G, bool cached, bool bf16) {
    const PlanKernel k = bf16 ? np2_plan_g<uint16_t>(W, G, cached) : np2_plan_g<float>(W, G, cached);
    if (!k) return Np2PlanPick{nullptr, 1};
    return Np2PlanPick{k, bf16 ? tile_units<uint16_t>(W * G, G) : tile_units<float>(W * G, G)};
}

Np2LarsKernel pick_lars_np2(int W, int G, bool bf16) {
    return bf16 ? np2_lars_g<uint16_t>(W, G) : np2_lars_g<float>(W, G);
}

}  // namespace lsgd
