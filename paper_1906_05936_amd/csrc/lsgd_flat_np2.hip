// Compile-time flat step kernels for group counts 3, 5, 6, 7 and 12.
#include "lsgd_host.hpp"
#include "lsgd_kernels.hpp"
#include "lsgd_np2.hpp"

namespace lsgd {
namespace {

using FlatKernel = void (*)(StepArgs);

template <typename GT, int W, int G>
FlatKernel np2_flat(bool cached) {
    constexpr int U = tile_units<GT>(W * G, G);
    if constexpr (cached_state_for(W * G))
        if (cached) return flat_step_kernel<GT, W, G, U, 1>();
    return flat_step_kernel<GT, W, G, U, 0>();
}

template <typename GT, int G>
FlatKernel np2_flat_w(int W, bool cached) {
    switch (W) {
        case 1: return np2_flat<GT, 1, G>(cached);
        case 2: return np2_flat<GT, 2, G>(cached);
        case 3: return np2_flat<GT, 3, G>(cached);
        case 4: return np2_flat<GT, 4, G>(cached);
        case 5: return np2_flat<GT, 5, G>(cached);
        case 6: return np2_flat<GT, 6, G>(cached);
        case 7: return np2_flat<GT, 7, G>(cached);
        case 8: return np2_flat<GT, 8, G>(cached);
        case 12:
            if constexpr (12 * G <= kMaxWorkers) return np2_flat<GT, 12, G>(cached);
            else return nullptr;
        case 16:
            if constexpr (16 * G <= kMaxWorkers) return np2_flat<GT, 16, G>(cached);
            else return nullptr;
        case 32:
            if constexpr (32 * G <= kMaxWorkers) return np2_flat<GT, 32, G>(cached);
            else return nullptr;
    }
    return nullptr;
}

template <typename GT>
FlatKernel np2_flat_g(int W, int G, bool cached) {
    switch (G) {
        case 3: return np2_flat_w<GT, 3>(W, cached);
        case 5: return np2_flat_w<GT, 5>(W, cached);
        case 6: return np2_flat_w<GT, 6>(W, cached);
        case 7: return np2_flat_w<GT, 7>(W, cached);
        case 12: return np2_flat_w<GT, 12>(W, cached);
    }
    return nullptr;
}

}  // namespace

Np2FlatPick pick_flat_np2(int W, int G, bool cached, bool bf16) {
    const FlatKernel k = bf16 ? np2_flat_g<uint16_t>(W, G, cached) : np2_flat_g<float>(W, G, cached);
    if (!k) return Np2FlatPick{nullptr, 1};
    return Np2FlatPick{k, bf16 ? tile_units<uint16_t>(W * G, G) : tile_units<float>(W * G, G)};
}

}  // namespace lsgd
