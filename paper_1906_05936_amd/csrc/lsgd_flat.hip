// Planless entry points of liblsgd: lsgd_group_mean, lsgd_global_mean,
// lsgd_sgd_step and the fused lsgd_step over one flat parameter vector.
#include <string.h>

#include <algorithm>

#include "lsgd_host.hpp"
#include "lsgd_kernels.hpp"
#include "lsgd_np2.hpp"
#include "lsgd_schedule.hpp"

namespace lsgd {
namespace {

using FlatKernel = void (*)(StepArgs);

// A kernel and the number of units per lane tile it processes.
struct FlatPick {
    FlatKernel kernel;
    int tile;
};

// Compile-time (W, G) kernels for power-of-two group counts G with N = W*G
// <= 128: groups of up to 16 workers (W a power of two, or 3, 5, 6, 7 or 12), or
// 32 to 128 workers in up to 4 groups, or 32 to 128 groups of up to 4
// workers; every other grouping takes the segmented runtime-layout kernel.
// Both give the same bits.
// The compile-time kernel for (W, G), with parameters and momentum through
// the caches when `cached` (instantiated only where cached_state_for holds).
template <typename GT, int W, int G>
FlatKernel flat_ct(bool cached) {
    constexpr int U = tile_units<GT>(W * G, G);
    if constexpr (cached_state_for(W * G))
        if (cached) return flat_step_kernel<GT, W, G, U, 1>();
    return flat_step_kernel<GT, W, G, U, 0>();
}

template <typename GT, int W>
FlatKernel pick_flat_g(int G, bool cached) {
    switch (G) {
        case 1: return flat_ct<GT, W, 1>(cached);
        case 2: return flat_ct<GT, W, 2>(cached);
        case 4: return flat_ct<GT, W, 4>(cached);
        case 8: return flat_ct<GT, W, 8>(cached);
        case 16:
            if constexpr (W * 16 <= kMaxWorkers) return flat_ct<GT, W, 16>(cached);
            else return nullptr;
        case 32:
            if constexpr (W <= 4) return flat_ct<GT, W, 32>(cached);
            else return nullptr;
        case 64:
            if constexpr (W <= 2) return flat_ct<GT, W, 64>(cached);
            else return nullptr;
        case 128:
            if constexpr (W == 1) return flat_ct<GT, W, 128>(cached);
            else return nullptr;
    }
    return nullptr;
}

// Groups of 32 to 128 workers, in up to 4 groups.
template <typename GT, int W>
FlatKernel pick_flat_big_w(int G, bool cached) {
    switch (G) {
        case 1: return flat_ct<GT, W, 1>(cached);
        case 2:
            if constexpr (W * 2 <= kMaxWorkers) return flat_ct<GT, W, 2>(cached);
            else return nullptr;
        case 4:
            if constexpr (W * 4 <= kMaxWorkers) return flat_ct<GT, W, 4>(cached);
            else return nullptr;
    }
    return nullptr;
}

template <typename GT>
FlatPick pick_flat(int W, int G, bool cached) {
    FlatKernel k = nullptr;
    switch (W) {
        case 1: k = pick_flat_g<GT, 1>(G, cached); break;
        case 2: k = pick_flat_g<GT, 2>(G, cached); break;
        case 3: k = pick_flat_g<GT, 3>(G, cached); break;
        case 4: k = pick_flat_g<GT, 4>(G, cached); break;
        case 5: k = pick_flat_g<GT, 5>(G, cached); break;
        case 6: k = pick_flat_g<GT, 6>(G, cached); break;
        case 7: k = pick_flat_g<GT, 7>(G, cached); break;
        case 8: k = pick_flat_g<GT, 8>(G, cached); break;
        case 12: k = pick_flat_g<GT, 12>(G, cached); break;
        case 16: k = pick_flat_g<GT, 16>(G, cached); break;
        case 32: k = pick_flat_big_w<GT, 32>(G, cached); break;
        case 64: k = pick_flat_big_w<GT, 64>(G, cached); break;
        case 128: k = pick_flat_big_w<GT, 128>(G, cached); break;
    }
    if (k) return FlatPick{k, tile_units<GT>(W * G, G)};
    return FlatPick{nullptr, 1};
}

// Runtime group layouts: accumulator levels for the largest count.
// (the cached forms exist for counts up to 31, the only ones they can have)
template <typename GT>
FlatPick pick_flat_seg(int max_count, bool cached) {
    constexpr int U = SegTileUnits<GT>::U;
    switch (seg_levels(max_count)) {
        case 3: return FlatPick{cached ? step_flat_seg<GT, 3, U, 1> : step_flat_seg<GT, 3, U, 0>, U};
        case 4: return FlatPick{cached ? step_flat_seg<GT, 4, U, 1> : step_flat_seg<GT, 4, U, 0>, U};
        case 5: return FlatPick{cached ? step_flat_seg<GT, 5, U, 1> : step_flat_seg<GT, 5, U, 0>, U};
    }
    return FlatPick{step_flat_seg<GT, 8, U, 0>, U};
}

using MeanKernel = void (*)(MeanArgs);

struct MeanPick {
    MeanKernel kernel;
    int tile;
};

// Group means: compile-time W for powers of two up to 16, else runtime W.
template <typename GT>
MeanPick pick_group_mean(int W) {
    constexpr int U = sizeof(GT) == 4 ? 2 : 1;   // W gradients per tile: the unrolled form up to 16
    switch (W) {
        case 1: return MeanPick{group_mean_kernel_ct<GT, 1, U>, U};
        case 2: return MeanPick{group_mean_kernel_ct<GT, 2, U>, U};
        case 4: return MeanPick{group_mean_kernel_ct<GT, 4, U>, U};
        case 8: return MeanPick{group_mean_kernel_ct<GT, 8, U>, U};
        case 16: return MeanPick{group_mean_kernel_ct<GT, 16, U>, U};
    }
    switch (seg_levels(W)) {
        case 3: return MeanPick{group_mean_kernel<GT, 3>, 1};
        case 4: return MeanPick{group_mean_kernel<GT, 4>, 1};
        case 5: return MeanPick{group_mean_kernel<GT, 5>, 1};
    }
    return MeanPick{group_mean_kernel<GT, 8>, 1};
}

// Global mean: compile-time G for powers of two up to 128, else runtime G.
MeanPick pick_global_mean(int G) {
    switch (G) {
        case 1: return MeanPick{global_mean_kernel_ct<1, 2>, 2};
        case 2: return MeanPick{global_mean_kernel_ct<2, 2>, 2};
        case 4: return MeanPick{global_mean_kernel_ct<4, 2>, 2};
        case 8: return MeanPick{global_mean_kernel_ct<8, 2>, 2};
        case 16: return MeanPick{global_mean_kernel_ct<16, 2>, 2};
        case 32: return MeanPick{global_mean_kernel_ct<32, 2>, 2};
        case 64: return MeanPick{global_mean_kernel_ct<64, 2>, 2};
        case 128: return MeanPick{global_mean_kernel_ct<128, 2>, 2};
    }
    switch (seg_levels(G)) {
        case 3: return MeanPick{global_mean_kernel<3>, 1};
        case 4: return MeanPick{global_mean_kernel<4>, 1};
        case 5: return MeanPick{global_mean_kernel<5>, 1};
    }
    return MeanPick{global_mean_kernel<8>, 1};
}

size_t dtype_size(lsgd_dtype d) { return d == LSGD_BF16 ? 2 : 4; }

// Units per lane (U) and replicas per workgroup (RK) of the copy-out pass:
// either way a lane loads 32 bytes of p and stores 32 bytes. Measured over
// U, RK in {1, 2, 4} at R = 4..128: binary32 U = 2, RK = 1 fastest (+2-4%
// over the next), bfloat16 U = 1, RK = 2 (one replica per workgroup: -5 to
// -13%).
constexpr int kCopyUF32 = 2, kCopyRKF32 = 1;
constexpr int kCopyUBF16 = 1, kCopyRKBF16 = 2;

template <int VEC, int U, int RK>
lsgd_status launch_copy_out_rmajor(StepArgs& a, hipStream_t stream) {
    const int64_t units = (a.n + VEC - 1) / VEC;
    const int64_t span = static_cast<int64_t>(kBlock) * U;   // units per workgroup
    const int64_t need = (units + span - 1) / span;
    const int64_t win = copy_window_blocks(4 * VEC * span, need);
    const int64_t blocks = (need + win - 1) / win * ((a.n_replicas + RK - 1) / RK) * win;
    a.win_blocks = static_cast<int32_t>(win);
    a.copy_blocks = blocks;
    // one workgroup per logical block: grid-stride forms (2048-8192 workgroups) measured 10-25% slower
    const int64_t grid = std::min<int64_t>(blocks, stride_grid_cap());
    hipLaunchKernelGGL((copy_out_rmajor_kernel<VEC, U, RK>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0,
                       stream, a);
    return check_launch("lsgd_step (copy-out)");
}

// The copy-out pass of a flat step: p (already updated on `stream`) to the
// replicas in a.replicas[0 .. a.n_replicas).
lsgd_status launch_copy_out(StepArgs& a, void* stream) {
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (a.rdt == static_cast<int32_t>(LSGD_BF16)) return launch_copy_out_rmajor<8, kCopyUBF16, kCopyRKBF16>(a, s);
    return launch_copy_out_rmajor<4, kCopyUF32, kCopyRKF32>(a, s);
}

// Long vectors are processed range by range, unless one pass writes the
// replicas too: the step kernel over one range of elements (then, with the
// copy-out as a pass of its own, its copy passes over that range), then the
// next range. The copy-out pass then reads the new
// parameters of a range soon after the step kernel wrote them (a range of
// kRangeElems holds 64 MB of parameters, which the 256 MB Infinity Cache
// still holds) instead of after the whole vector, and the step kernel alone
// runs faster over ranges than over the whole vector in one launch. Measured
// on the 3.5e8-element 8x8 bfloat16 step, same process: with no replicas,
// ranges of 2^23, 2^24 and 2^26 elements +3.1%, +3.3% and +2.6% against one
// launch; with 64 replicas and the copy-out pass, +1.5%, +1.9% and +1.8%
// against ranges of 2^25 whose edges were not 2 MB apart (such ranges were no
// faster than one launch without replicas). On the 2.6e7-element 4x4 step two
// ranges lost 0.6%, so vectors up to kRangeSplitMin stay whole.
// Results are the same bits (every element is computed on its own).
constexpr int64_t kRangeElems = int64_t{1} << 24;
constexpr int64_t kRangeSplitMin = int64_t{1} << 26;
// Range edges fall on multiples of kRangeAlign elements: 2 MB or more in every
// buffer, so buffers that start at the same offset modulo 2 MB (as separate
// large allocations do) keep doing so within every range.
constexpr int64_t kRangeAlign = int64_t{1} << 20;

int64_t split_ranges(int64_t n) { return n > kRangeSplitMin ? (n + kRangeElems - 1) / kRangeElems : 1; }

// Start of range i of K over n elements (range K ends at n). With K > 1 the
// vector is longer than 4 * kRangeElems, so every range holds at least
// kRangeElems / 2 elements.
int64_t range_edge(int64_t n, int64_t K, int64_t i) { return i >= K ? n : (n / K * i) / kRangeAlign * kRangeAlign; }

// The arguments of a step restricted to elements [lo, hi): every per-element
// pointer advanced by lo elements (R replica pointers of rsz bytes).
StepArgs offset_args(const StepArgs& a, int64_t lo, int64_t hi, size_t gsz, size_t rsz, int32_t R) {
    StepArgs b = a;
    b.p = a.p + lo;
    b.m = a.m + lo;
    if (a.gbar) b.gbar = a.gbar + lo;
    b.n = hi - lo;
    for (int32_t k = 0; k < a.n_workers; ++k)
        b.grads[k] = static_cast<const char*>(a.grads[k]) + static_cast<size_t>(lo) * gsz;
    for (int32_t r = 0; r < R; ++r) b.replicas[r] = static_cast<char*>(a.replicas[r]) + static_cast<size_t>(lo) * rsz;
    return b;
}

// Name of gradient ranges in the aliasing check (compared by address).
const char* const kGradRange = "grad";

bool valid_dtype(lsgd_dtype d) { return d == LSGD_F32 || d == LSGD_BF16; }

Range range_of(const void* p, int64_t n, size_t esize, bool written, const char* what) {
    uintptr_t b = reinterpret_cast<uintptr_t>(p);
    return Range{b, b + static_cast<uintptr_t>(n) * esize, written, what};
}

// Checks the replica list: count, dtype, non-NULL, alignment; appends ranges.
lsgd_status check_replicas(void* const* replicas, int32_t n_replicas, lsgd_dtype rdt, int64_t n,
                           bool check_ptrs, std::vector<Range>& ranges) {
    if (n_replicas < 0 || n_replicas > kMaxReplicas)
        return fail(LSGD_ERR_SIZE, "n_replicas=%d outside [0, %d]", n_replicas, kMaxReplicas);
    if (!valid_dtype(rdt)) return fail(LSGD_ERR_DTYPE, "replica dtype %d", static_cast<int>(rdt));
    if (!check_ptrs) return LSGD_OK;
    if (n_replicas > 0 && !replicas) return fail(LSGD_ERR_NULL, "replicas is NULL with n_replicas=%d", n_replicas);
    for (int32_t r = 0; r < n_replicas; ++r) {
        if (!replicas[r]) return fail(LSGD_ERR_NULL, "replicas[%d] is NULL", r);
        if (!aligned16(replicas[r])) return fail(LSGD_ERR_ALIGN, "replicas[%d] is not 16-byte aligned", r);
        ranges.push_back(range_of(replicas[r], n, dtype_size(rdt), true, "replica"));
    }
    return LSGD_OK;
}

lsgd_status check_update_buffers(float* params, float* momentum, int64_t n, std::vector<Range>& ranges) {
    if (!params) return fail(LSGD_ERR_NULL, "params is NULL");
    if (!momentum) return fail(LSGD_ERR_NULL, "momentum is NULL");
    if (!aligned16(params)) return fail(LSGD_ERR_ALIGN, "params is not 16-byte aligned");
    if (!aligned16(momentum)) return fail(LSGD_ERR_ALIGN, "momentum is not 16-byte aligned");
    ranges.push_back(range_of(params, n, 4, true, "params"));
    ranges.push_back(range_of(momentum, n, 4, true, "momentum"));
    return LSGD_OK;
}

// Gradient pointers in member order with their ranges.
lsgd_status check_grads(const void* const* grads, lsgd_dtype gdt, const std::vector<int32_t>& order,
                        int64_t n, bool check_ptrs, const void** out, std::vector<Range>& ranges) {
    if (!valid_dtype(gdt)) return fail(LSGD_ERR_DTYPE, "gradient dtype %d", static_cast<int>(gdt));
    if (!check_ptrs) return LSGD_OK;
    if (!grads) return fail(LSGD_ERR_NULL, "grads is NULL");
    for (size_t k = 0; k < order.size(); ++k) {
        const void* g = grads[order[k]];
        if (!g) return fail(LSGD_ERR_NULL, "grads[%d] is NULL", order[k]);
        if (!aligned16(g)) return fail(LSGD_ERR_ALIGN, "grads[%d] is not 16-byte aligned", order[k]);
        out[k] = g;
        ranges.push_back(range_of(g, n, dtype_size(gdt), false, kGradRange));
    }
    return LSGD_OK;
}

}  // namespace
}  // namespace lsgd

using namespace lsgd;

extern "C" {

LSGD_API lsgd_status lsgd_step_ex(float* params, float* momentum, void* const* grads,
                                  lsgd_dtype gdt, int32_t n_workers, const int32_t* group_of_worker,
                                  int32_t n_groups, int64_t n, float lr, float momentum_coef,
                                  float weight_decay, void* const* replicas, int32_t n_replicas,
                                  lsgd_dtype rdt, const lsgd_step_options* options, void* stream) {
    const lsgd_step_options none = {LSGD_REDUCE_MEAN_OF_MEANS, 0, nullptr};
    const lsgd_step_options& o = options ? *options : none;
    if (o.reduction != LSGD_REDUCE_MEAN_OF_MEANS && o.reduction != LSGD_REDUCE_LITERAL)
        return fail(LSGD_ERR_UNSUPPORTED, "reduction %d", o.reduction);
    const bool literal = o.reduction == LSGD_REDUCE_LITERAL;
    const bool bcast = o.broadcast_grad != 0;
    if (n < 0) return fail(LSGD_ERR_SIZE, "n=%lld < 0", static_cast<long long>(n));
    std::vector<int32_t> order, gstart;
    lsgd_status st = literal ? partition_order(n_workers, group_of_worker, n_groups, order, gstart)
                             : member_order(n_workers, group_of_worker, n_groups, order);
    if (st != LSGD_OK) return st;
    if (bcast && gdt != LSGD_F32)
        return fail(LSGD_ERR_DTYPE, "broadcast_grad needs binary32 gradients, got dtype %d", static_cast<int>(gdt));
    const bool live = n > 0;
    StepArgs a;
    memset(&a, 0, sizeof a);
    std::vector<Range> ranges;
    if ((st = check_grads(grads, gdt, order, n, live, a.grads, ranges)) != LSGD_OK) return st;
    if ((st = check_replicas(replicas, n_replicas, rdt, n, live, ranges)) != LSGD_OK) return st;
    if (!live) return LSGD_OK;
    if ((st = check_update_buffers(params, momentum, n, ranges)) != LSGD_OK) return st;
    if (bcast)   // the gradient buffers are written too
        for (Range& r : ranges)
            if (r.what == kGradRange) r.written = true;
    if (o.lr_device) {
        if ((reinterpret_cast<uintptr_t>(o.lr_device) & 3u) != 0)
            return fail(LSGD_ERR_ALIGN, "lr_device is not 4-byte aligned");
        ranges.push_back(range_of(o.lr_device, 1, 4, false, "lr_device"));
    }
    if ((st = check_overlap(ranges)) != LSGD_OK) return st;

    // equal group sizes: the literal reduction then runs in the compile-time
    // kernels too (W = 0 marks unequal groups)
    int32_t W = n_workers / n_groups;
    if (literal)
        for (int32_t j = 0; j < n_groups; ++j)
            if (gstart[j + 1] - gstart[j] != gstart[1] - gstart[0]) W = 0;
    const bool cached = use_cached_state(n_workers, n);
    // a compile-time kernel for (W, G): power-of-two group counts, then 3, 5,
    // 6, 7 and 12 (lsgd_np2.hpp)
    auto pick_ct = [&](int32_t w, int32_t g) {
        FlatPick p = gdt == LSGD_BF16 ? pick_flat<uint16_t>(w, g, cached) : pick_flat<float>(w, g, cached);
        if (!p.kernel && np2_group_count(g)) {
            const Np2FlatPick q = pick_flat_np2(w, g, cached, gdt == LSGD_BF16);
            p = FlatPick{q.kernel, q.tile};
        }
        return p;
    };
    int32_t G = n_groups;
    FlatPick k{nullptr, 1};
    if (W > 0) k = pick_ct(W, G);
    if (!k.kernel && one_group_form(W, G, literal)) {
        W = n_workers;
        G = 1;
        k = pick_ct(W, G);
    }
    a.p = params;
    a.m = momentum;
    a.n = n;
    a.h = Hyper{lr, momentum_coef, weight_decay};
    a.n_workers = n_workers;
    a.n_groups = G;
    a.W = W;
    a.n_replicas = n_replicas;
    a.rdt = static_cast<int32_t>(rdt);
    a.lr_ptr = o.lr_device;
    a.literal = literal ? 1 : 0;
    for (int32_t r = 0; r < n_replicas; ++r) a.replicas[r] = replicas[r];

    const int64_t vec = gdt == LSGD_BF16 ? Unit<uint16_t>::VEC : Unit<float>::VEC;
    const bool segmented = !k.kernel;
    const bool pow2_grouping = !segmented && (W & (W - 1)) == 0 && (G & (G - 1)) == 0;
    if (segmented) {
        // runtime layout: group j is members [start[j], start[j+1]) of the member order
        int32_t max_count = G;
        for (int32_t j = 0; j <= G; ++j) {
            const int32_t b = literal ? gstart[j] : j * W;
            a.group_start[j] = static_cast<uint8_t>(b);
            if (j > 0) max_count = std::max(max_count, b - static_cast<int32_t>(a.group_start[j - 1]));
        }
        k = gdt == LSGD_BF16 ? pick_flat_seg<uint16_t>(max_count, cached) : pick_flat_seg<float>(max_count, cached);
    }
    // Copies per element besides parameters and momentum: the replicas, and
    // with the broadcast the mean gradient to the other N - 1 members. Split
    // off, the step kernel writes the mean gradient to the first member only
    // and copy passes of their own write the rest (range by range: split_ranges).
    const int32_t bcast_copies = bcast ? n_workers - 1 : 0;
    const bool split = separate_copy_out_bytes(
        n_workers, dtype_size(gdt), static_cast<int64_t>(n_replicas) * dtype_size(rdt) + 4 * bcast_copies, n,
        !pow2_grouping);
    a.bcast_grad = bcast ? (split ? 1 : n_workers) : 0;
    // split: the step kernel writes the first k replicas, the copy-out pass the rest
    const int32_t k_step = split ? replicas_in_step(n_workers, n_replicas, dtype_size(rdt), n) : n_replicas;
    a.n_replicas = k_step;
    const char* what = literal ? "lsgd_step_ex" : "lsgd_step";
    // a fused pass that writes replicas or broadcast copies stays one launch
    // (ranges measured 0.8% slower there: 3.5e8-element 8x8 bfloat16 step, 64 replicas)
    const int64_t K = split || (n_replicas == 0 && !bcast) ? split_ranges(n) : 1;
    for (int64_t i = 0; i < K; ++i) {
        const int64_t lo = range_edge(n, K, i), hi = range_edge(n, K, i + 1);
        StepArgs ra = K == 1 ? a : offset_args(a, lo, hi, dtype_size(gdt), dtype_size(rdt), n_replicas);
        const LaunchShape ls = launch_shape((ra.n + vec - 1) / vec, k.tile);
        ra.xcd_chunk = ls.xcd_chunk;
        ra.upl = ls.upl;
        hipLaunchKernelGGL(k.kernel, dim3(ls.blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream), ra);
        if ((st = check_launch(what)) != LSGD_OK) return st;
        if (!split) continue;
        if (n_replicas > k_step) {
            for (int32_t r = k_step; r < n_replicas; ++r) ra.replicas[r - k_step] = ra.replicas[r];
            ra.n_replicas = n_replicas - k_step;
            if ((st = launch_copy_out(ra, stream)) != LSGD_OK) return st;
        }
        if (bcast_copies > 0) {
            StepArgs b;
            memset(&b, 0, sizeof b);
            b.p = static_cast<float*>(const_cast<void*>(ra.grads[0]));   // read only by the copy pass
            b.n = ra.n;
            b.n_replicas = bcast_copies;
            b.rdt = static_cast<int32_t>(LSGD_F32);
            for (int32_t k2 = 0; k2 < bcast_copies; ++k2) b.replicas[k2] = const_cast<void*>(ra.grads[k2 + 1]);
            if ((st = launch_copy_out(b, stream)) != LSGD_OK) return st;
        }
    }
    return LSGD_OK;
}

LSGD_API lsgd_status lsgd_step(float* params, float* momentum, const void* const* grads,
                               lsgd_dtype gdt, int32_t n_workers, const int32_t* group_of_worker,
                               int32_t n_groups, int64_t n, float lr, float momentum_coef,
                               float weight_decay, void* const* replicas, int32_t n_replicas,
                               lsgd_dtype rdt, void* stream) {
    // Without options no gradient buffer is written, so dropping const is safe.
    return lsgd_step_ex(params, momentum, const_cast<void* const*>(grads), gdt, n_workers,
                        group_of_worker, n_groups, n, lr, momentum_coef, weight_decay, replicas,
                        n_replicas, rdt, nullptr, stream);
}

LSGD_API lsgd_status lsgd_group_mean(const void* const* grads, lsgd_dtype gdt, int32_t n_workers,
                                     const int32_t* group_of_worker, int32_t n_groups, int64_t n,
                                     float* const* group_means, void* stream) {
    if (n < 0) return fail(LSGD_ERR_SIZE, "n=%lld < 0", static_cast<long long>(n));
    std::vector<int32_t> order;
    lsgd_status st = member_order(n_workers, group_of_worker, n_groups, order);
    if (st != LSGD_OK) return st;
    const bool live = n > 0;
    MeanArgs a;
    memset(&a, 0, sizeof a);
    std::vector<Range> ranges;
    if ((st = check_grads(grads, gdt, order, n, live, a.in, ranges)) != LSGD_OK) return st;
    if (!live) return LSGD_OK;
    if (!group_means) return fail(LSGD_ERR_NULL, "group_means is NULL");
    for (int32_t j = 0; j < n_groups; ++j) {
        if (!group_means[j]) return fail(LSGD_ERR_NULL, "group_means[%d] is NULL", j);
        if (!aligned16(group_means[j])) return fail(LSGD_ERR_ALIGN, "group_means[%d] is not 16-byte aligned", j);
        ranges.push_back(range_of(group_means[j], n, 4, true, "group_mean"));
        a.out[j] = group_means[j];
    }
    if ((st = check_overlap(ranges)) != LSGD_OK) return st;
    a.n = n;
    a.n_workers = n_workers;
    a.n_groups = n_groups;
    a.W = n_workers / n_groups;
    const int64_t vec = gdt == LSGD_BF16 ? Unit<uint16_t>::VEC : Unit<float>::VEC;
    const MeanPick k = gdt == LSGD_BF16 ? pick_group_mean<uint16_t>(a.W) : pick_group_mean<float>(a.W);
    const LaunchShape ls = launch_shape((n + vec - 1) / vec, k.tile);
    a.xcd_chunk = ls.xcd_chunk;
    a.upl = ls.upl;
    hipLaunchKernelGGL(k.kernel, dim3(ls.blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream), a);
    return check_launch("lsgd_group_mean");
}

LSGD_API lsgd_status lsgd_global_mean(const float* const* group_means, int32_t n_groups, int64_t n,
                                      float* grad_mean, void* stream) {
    if (n < 0) return fail(LSGD_ERR_SIZE, "n=%lld < 0", static_cast<long long>(n));
    if (n_groups < 1 || n_groups > kMaxWorkers)
        return fail(LSGD_ERR_SIZE, "n_groups=%d outside [1, %d]", n_groups, kMaxWorkers);
    if (n == 0) return LSGD_OK;
    if (!group_means) return fail(LSGD_ERR_NULL, "group_means is NULL");
    if (!grad_mean) return fail(LSGD_ERR_NULL, "grad_mean is NULL");
    if (!aligned16(grad_mean)) return fail(LSGD_ERR_ALIGN, "grad_mean is not 16-byte aligned");
    MeanArgs a;
    memset(&a, 0, sizeof a);
    std::vector<Range> ranges;
    for (int32_t j = 0; j < n_groups; ++j) {
        if (!group_means[j]) return fail(LSGD_ERR_NULL, "group_means[%d] is NULL", j);
        if (!aligned16(group_means[j])) return fail(LSGD_ERR_ALIGN, "group_means[%d] is not 16-byte aligned", j);
        ranges.push_back(range_of(group_means[j], n, 4, false, "group_mean"));
        a.in[j] = group_means[j];
    }
    ranges.push_back(range_of(grad_mean, n, 4, true, "grad_mean"));
    lsgd_status st = check_overlap(ranges);
    if (st != LSGD_OK) return st;
    a.out[0] = grad_mean;
    a.n = n;
    a.n_groups = n_groups;
    const MeanPick k = pick_global_mean(n_groups);
    const LaunchShape ls = launch_shape((n + 3) / 4, k.tile);
    a.xcd_chunk = ls.xcd_chunk;
    a.upl = ls.upl;
    hipLaunchKernelGGL(k.kernel, dim3(ls.blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream), a);
    return check_launch("lsgd_global_mean");
}

LSGD_API lsgd_status lsgd_sgd_step(float* params, float* momentum, const float* grad_mean, int64_t n,
                                   float lr, float momentum_coef, float weight_decay,
                                   void* const* replicas, int32_t n_replicas, lsgd_dtype rdt,
                                   void* stream) {
    if (n < 0) return fail(LSGD_ERR_SIZE, "n=%lld < 0", static_cast<long long>(n));
    const bool live = n > 0;
    std::vector<Range> ranges;
    lsgd_status st = check_replicas(replicas, n_replicas, rdt, n, live, ranges);
    if (st != LSGD_OK) return st;
    if (!live) return LSGD_OK;
    if ((st = check_update_buffers(params, momentum, n, ranges)) != LSGD_OK) return st;
    if (!grad_mean) return fail(LSGD_ERR_NULL, "grad_mean is NULL");
    if (!aligned16(grad_mean)) return fail(LSGD_ERR_ALIGN, "grad_mean is not 16-byte aligned");
    ranges.push_back(range_of(grad_mean, n, 4, false, "grad_mean"));
    if ((st = check_overlap(ranges)) != LSGD_OK) return st;
    StepArgs a;
    memset(&a, 0, sizeof a);
    a.p = params;
    a.m = momentum;
    a.gbar = grad_mean;
    a.n = n;
    a.h = Hyper{lr, momentum_coef, weight_decay};
    a.n_replicas = n_replicas;
    a.rdt = static_cast<int32_t>(rdt);
    for (int32_t r = 0; r < n_replicas; ++r) a.replicas[r] = replicas[r];
    constexpr int kSgdTile = 2;
    const bool split = separate_copy_out_update(n_replicas, dtype_size(rdt), use_cached_state(1, n));
    if (split) a.n_replicas = 0;
    const FlatKernel sk = use_cached_state(1, n) ? sgd_kernel<kSgdTile, 1> : sgd_kernel<kSgdTile, 0>;
    const int64_t K = split || n_replicas == 0 ? split_ranges(n) : 1;   // range by range, as lsgd_step
    for (int64_t i = 0; i < K; ++i) {
        const int64_t lo = range_edge(n, K, i), hi = range_edge(n, K, i + 1);
        StepArgs ra = K == 1 ? a : offset_args(a, lo, hi, 4, dtype_size(rdt), n_replicas);
        const LaunchShape ls = launch_shape((ra.n + 3) / 4, kSgdTile);
        ra.xcd_chunk = ls.xcd_chunk;
        ra.upl = ls.upl;
        hipLaunchKernelGGL(sk, dim3(ls.blocks), dim3(kBlock), 0, static_cast<hipStream_t>(stream), ra);
        if ((st = check_launch("lsgd_sgd_step")) != LSGD_OK) return st;
        if (!split) continue;
        ra.n_replicas = n_replicas;
        if ((st = launch_copy_out(ra, stream)) != LSGD_OK) return st;
    }
    return LSGD_OK;
}

LSGD_API lsgd_status lsgd_copy_out(const float* params, int64_t n, void* const* replicas, int32_t n_replicas,
                                   lsgd_dtype rdt, void* stream) {
    if (n < 0) return fail(LSGD_ERR_SIZE, "n=%lld < 0", static_cast<long long>(n));
    const bool live = n > 0 && n_replicas > 0;
    std::vector<Range> ranges;
    lsgd_status st = check_replicas(replicas, n_replicas, rdt, n, live, ranges);
    if (st != LSGD_OK || !live) return st;
    if (!params) return fail(LSGD_ERR_NULL, "params is NULL");
    if (!aligned16(params)) return fail(LSGD_ERR_ALIGN, "params is not 16-byte aligned");
    ranges.push_back(range_of(params, n, 4, false, "params"));
    if ((st = check_overlap(ranges)) != LSGD_OK) return st;
    StepArgs a;
    memset(&a, 0, sizeof a);
    a.p = const_cast<float*>(params);   // read only by the copy-out kernel
    a.n = n;
    a.n_replicas = n_replicas;
    a.rdt = static_cast<int32_t>(rdt);
    for (int32_t r = 0; r < n_replicas; ++r) a.replicas[r] = replicas[r];
    return launch_copy_out(a, stream);
}

namespace {
bool schedule_valid(const lsgd_lr_schedule* c) {
    return c && c->base_batch > 0 && c->warmup_iters >= 0 && c->decay_iters >= 0;
}
lsgd::Schedule to_schedule(const lsgd_lr_schedule& c) {
    return lsgd::Schedule{c.base_lr, c.base_batch, c.global_batch, c.warmup_iters, c.decay_iters,
                          c.decay_factor};
}
}  // namespace

LSGD_API float lsgd_lr_at(const lsgd_lr_schedule* schedule, int64_t t) {
    if (!schedule_valid(schedule) || t < 0) return __builtin_nanf("");
    return schedule_lr(to_schedule(*schedule), t);
}

LSGD_API lsgd_status lsgd_lr_schedule_step(const lsgd_lr_schedule* schedule, int64_t* iteration,
                                           float* lr_out, void* stream) {
    if (!schedule || !iteration || !lr_out) return fail(LSGD_ERR_NULL, "schedule, iteration or lr_out is NULL");
    if (!schedule_valid(schedule))
        return fail(LSGD_ERR_SIZE, "schedule needs base_batch > 0 and non-negative iteration counts");
    if ((reinterpret_cast<uintptr_t>(iteration) & 7u) != 0 || (reinterpret_cast<uintptr_t>(lr_out) & 3u) != 0)
        return fail(LSGD_ERR_ALIGN, "iteration must be 8-byte and lr_out 4-byte aligned");
    std::vector<Range> ranges{range_of(iteration, 1, 8, true, "iteration"), range_of(lr_out, 1, 4, true, "lr_out")};
    lsgd_status st = check_overlap(ranges);
    if (st != LSGD_OK) return st;
    hipLaunchKernelGGL(schedule_step_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream),
                       to_schedule(*schedule), iteration, lr_out);
    return check_launch("lsgd_lr_schedule_step");
}

}  // extern "C"
