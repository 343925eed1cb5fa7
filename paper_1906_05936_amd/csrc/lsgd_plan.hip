// Multi-tensor plans of liblsgd: the fused step over a list of parameter
// tensors (a model's per-layer tensors) in one kernel launch.
//
// lsgd_plan_create cuts every tensor into pieces of P workgroup tile passes
// (256 lanes x the kernel's lane tile: 2048 elements for binary32 and bf16
// gradients alike, times P = the launch shape's passes per workgroup at plan
// creation, 1 by default), starting on unit boundaries, then packs consecutive
// pieces into buckets of at most one piece: a large tensor yields one bucket per piece
// (so it is walked exactly like the flat kernel walks a vector), while runs of
// small tensors (ResNet-50's 64..1024-element batch-norm and bias vectors)
// share a bucket. One workgroup runs one bucket; buckets are taken in the
// XCD-chunked order of the launch shape.
#include <string.h>

#include <algorithm>

#include "lsgd_host.hpp"
#include "lsgd_np2.hpp"
#include "lsgd_plan_kernels.hpp"

struct lsgd_plan {
    int device;
    int32_t n_tensors, n_workers, n_groups, W, n_replicas;
    lsgd_dtype gdt, rdt;
    int32_t n_buckets, n_chunks, stride;
    int64_t piece;  // elements per piece and per bucket
    int64_t total_elems;  // elements of all tensors
    lsgd::PlanChunk* d_chunks;
    int32_t* d_bucket_begin;
    lsgd::CopyDesc* d_copy_desc;
    void** d_ptrs;
    // LARS: per-tensor scratch offsets and chunk ranges, and every buffer's
    // byte range (for the workspace aliasing check)
    int64_t gbar_floats;
    int64_t* d_gbar_off;
    int32_t* d_tensor_chunks;
    uint8_t* d_lars_exclude;   // [n_tensors], zero until lsgd_plan_set_lars_exclude
    std::vector<lsgd::Range>* ranges;
    // the partition: groups of equal size W (W = 0 otherwise), group j is
    // members [group_start[j], group_start[j+1]) of the member order
    int32_t max_group;
    int32_t group_start[lsgd::kMaxWorkers + 1];
};

namespace lsgd {
namespace {

using PlanKernel = void (*)(PlanArgs);
using LarsKernel = void (*)(LarsArgs);

// LARS scratch: each tensor's slice of the mean-gradient scratch starts on a
// 64-float (256-byte) boundary.
constexpr int64_t kGbarAlign = 64;

// A kernel, the units per lane tile it processes, and whether it is the
// segmented (runtime-layout) form.
struct PlanPick {
    PlanKernel kernel;
    int tile;
    bool segmented;
};

// Elements per piece and per bucket: one tile pass of the plan's kernel.
template <typename GT>
constexpr int64_t piece_elems(int tile) { return static_cast<int64_t>(kBlock) * Unit<GT>::VEC * tile; }
static_assert(piece_elems<float>(1) % 8 == 0 && piece_elems<uint16_t>(1) % 8 == 0,
              "pieces must start on unit boundaries");

// The segmented plan kernel for groups and group counts up to max_count
// (the cached form exists for counts up to 31, the only ones it can have).
template <typename GT>
PlanKernel plan_seg(int max_count, bool cached) {
    switch (seg_levels(max_count)) {
        case 3: return cached ? step_plan_seg<GT, 3, 1> : step_plan_seg<GT, 3, 0>;
        case 4: return cached ? step_plan_seg<GT, 4, 1> : step_plan_seg<GT, 4, 0>;
        case 5: return cached ? step_plan_seg<GT, 5, 1> : step_plan_seg<GT, 5, 0>;
    }
    return step_plan_seg<GT, 8, 0>;
}

template <typename GT, int W, int G>
PlanKernel plan_ct(bool cached) {
    constexpr int U = tile_units<GT>(W * G, G);
    if constexpr (cached_state_for(W * G))
        if (cached) return plan_step_kernel<GT, W, G, U, 1>();
    return plan_step_kernel<GT, W, G, U, 0>();
}

template <typename GT, int W>
PlanKernel pick_plan_g(int G, bool cached) {
    switch (G) {
        case 1: return plan_ct<GT, W, 1>(cached);
        case 2: return plan_ct<GT, W, 2>(cached);
        case 4: return plan_ct<GT, W, 4>(cached);
        case 8: return plan_ct<GT, W, 8>(cached);
        case 16:
            if constexpr (W * 16 <= kMaxWorkers) return plan_ct<GT, W, 16>(cached);
            else return nullptr;
        case 32:
            if constexpr (W <= 4) return plan_ct<GT, W, 32>(cached);
            else return nullptr;
        case 64:
            if constexpr (W <= 2) return plan_ct<GT, W, 64>(cached);
            else return nullptr;
        case 128:
            if constexpr (W == 1) return plan_ct<GT, W, 128>(cached);
            else return nullptr;
    }
    return nullptr;
}

// Groups of 32 to 128 workers, in up to 4 groups.
template <typename GT, int W>
PlanKernel pick_plan_big_w(int G, bool cached) {
    switch (G) {
        case 1: return plan_ct<GT, W, 1>(cached);
        case 2:
            if constexpr (W * 2 <= kMaxWorkers) return plan_ct<GT, W, 2>(cached);
            else return nullptr;
        case 4:
            if constexpr (W * 4 <= kMaxWorkers) return plan_ct<GT, W, 4>(cached);
            else return nullptr;
    }
    return nullptr;
}

// The plan kernel for (W, G): compile-time for the power-of-two groupings of
// pick_flat (lsgd_flat.hip), with parameters and momentum through the caches
// when `cached`; else segmented.
template <typename GT>
PlanPick pick_plan(int W, int G, bool cached = false) {
    PlanKernel k = nullptr;
    switch (W) {
        case 1: k = pick_plan_g<GT, 1>(G, cached); break;
        case 2: k = pick_plan_g<GT, 2>(G, cached); break;
        case 3: k = pick_plan_g<GT, 3>(G, cached); break;
        case 4: k = pick_plan_g<GT, 4>(G, cached); break;
        case 5: k = pick_plan_g<GT, 5>(G, cached); break;
        case 6: k = pick_plan_g<GT, 6>(G, cached); break;
        case 7: k = pick_plan_g<GT, 7>(G, cached); break;
        case 8: k = pick_plan_g<GT, 8>(G, cached); break;
        case 12: k = pick_plan_g<GT, 12>(G, cached); break;
        case 16: k = pick_plan_g<GT, 16>(G, cached); break;
        case 32: k = pick_plan_big_w<GT, 32>(G, cached); break;
        case 64: k = pick_plan_big_w<GT, 64>(G, cached); break;
        case 128: k = pick_plan_big_w<GT, 128>(G, cached); break;
    }
    if (k) return PlanPick{k, tile_units<GT>(W * G, G), false};
    if (np2_group_count(G)) {   // group counts 3, 5, 6, 7 and 12 (lsgd_np2.hpp)
        const Np2PlanPick q = pick_plan_np2(W, G, cached, sizeof(GT) == 2);
        if (q.kernel) return PlanPick{q.kernel, q.tile, false};
    }
    return PlanPick{plan_seg<GT>(W > G ? W : G, cached), SegTileUnits<GT>::U, true};
}

lsgd_status check_device(const lsgd_plan* plan) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev != plan->device)
        return fail(LSGD_ERR_HIP, "plan was created on device %d, current device is %d", plan->device, dev);
    return LSGD_OK;
}

// Kernel arguments of a plan step and the launch shape over its buckets.
PlanArgs plan_args(const lsgd_plan* plan, Hyper h, const float* lr_device, LaunchShape& ls) {
    PlanArgs a;
    memset(&a, 0, sizeof a);
    a.chunks = plan->d_chunks;
    a.bucket_begin = plan->d_bucket_begin;
    a.copy_desc = plan->d_copy_desc;
    a.ptrs = plan->d_ptrs;
    a.stride = plan->stride;
    a.n_workers = plan->n_workers;
    a.cached_state = use_cached_state(plan->n_workers, plan->total_elems) ? 1 : 0;   // read by the LARS update
    a.n_groups = plan->n_groups;
    a.W = plan->W;
    a.n_replicas = plan->n_replicas;
    a.rdt = static_cast<int32_t>(plan->rdt);
    a.h = h;
    a.lr_ptr = lr_device;
    a.n_buckets = plan->n_buckets;
    a.copy_src = 0;                              // the copy-out: p to the replicas
    a.copy_dst = 2 + plan->n_workers;
    for (int32_t j = 0; j <= plan->n_groups; ++j) a.group_start[j] = static_cast<uint8_t>(plan->group_start[j]);
    const int64_t block_bytes = (plan->gdt == LSGD_BF16 ? 2 : 4) * plan->piece;
    ls = pad_for_xcd_chunk(plan->n_buckets, block_bytes);
    a.xcd_chunk = ls.xcd_chunk;
    return a;
}

// Replicas per workgroup of the plan's copy-out pass (as for flat steps: a
// lane loads 32 bytes of p and stores 32 bytes per tile).
constexpr int kPlanCopyRKF32 = 1, kPlanCopyRKBF16 = 2;

// The copy-out pass of a plan step: one workgroup per bucket and replica
// group; a lane tile covers a 2048-element piece (the usual piece size).
template <int VEC, int RK>
lsgd_status launch_plan_copy_out(const lsgd_plan* plan, PlanArgs& a, hipStream_t s) {
    constexpr int U = 2048 / (VEC * kBlock);
    static_assert(U >= 1, "at least one unit per lane");
    const int64_t win = copy_window_blocks(4 * plan->piece, plan->n_buckets);
    const int64_t blocks = (plan->n_buckets + win - 1) / win * ((a.n_replicas + RK - 1) / RK) * win;
    a.win_blocks = static_cast<int32_t>(win);
    a.copy_blocks = blocks;
    const int64_t grid = std::min<int64_t>(blocks, stride_grid_cap());   // the kernel strides over the rest
    hipLaunchKernelGGL((copy_out_plan_rmajor<VEC, U, RK>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, s, a);
    return check_launch("lsgd_step_plan (copy-out)");
}

// LARS pass-1 kernels: compile-time (W, G) as for the step, else segmented.
template <typename GT, int W>
LarsKernel pick_lars_g(int G) {
    switch (G) {
        case 1: return lars_kernel_for<GT, W, 1>();
        case 2: return lars_kernel_for<GT, W, 2>();
        case 4: return lars_kernel_for<GT, W, 4>();
        case 8: return lars_kernel_for<GT, W, 8>();
        case 16:
            if constexpr (W * 16 <= kMaxWorkers) return lars_kernel_for<GT, W, 16>();
            else return nullptr;
        case 32:
            if constexpr (W <= 4) return lars_kernel_for<GT, W, 32>();
            else return nullptr;
        case 64:
            if constexpr (W <= 2) return lars_kernel_for<GT, W, 64>();
            else return nullptr;
        case 128:
            if constexpr (W == 1) return lars_kernel_for<GT, W, 128>();
            else return nullptr;
    }
    return nullptr;
}

template <typename GT, int W>
LarsKernel pick_lars_big_w(int G) {
    switch (G) {
        case 1: return lars_kernel_for<GT, W, 1>();
        case 2:
            if constexpr (W * 2 <= kMaxWorkers) return lars_kernel_for<GT, W, 2>();
            else return nullptr;
        case 4:
            if constexpr (W * 4 <= kMaxWorkers) return lars_kernel_for<GT, W, 4>();
            else return nullptr;
    }
    return nullptr;
}

template <typename GT>
LarsKernel pick_lars(int W, int G) {
    LarsKernel k = nullptr;
    switch (W) {
        case 1: k = pick_lars_g<GT, 1>(G); break;
        case 2: k = pick_lars_g<GT, 2>(G); break;
        case 3: k = pick_lars_g<GT, 3>(G); break;
        case 4: k = pick_lars_g<GT, 4>(G); break;
        case 5: k = pick_lars_g<GT, 5>(G); break;
        case 6: k = pick_lars_g<GT, 6>(G); break;
        case 7: k = pick_lars_g<GT, 7>(G); break;
        case 8: k = pick_lars_g<GT, 8>(G); break;
        case 12: k = pick_lars_g<GT, 12>(G); break;
        case 16: k = pick_lars_g<GT, 16>(G); break;
        case 32: k = pick_lars_big_w<GT, 32>(G); break;
        case 64: k = pick_lars_big_w<GT, 64>(G); break;
        case 128: k = pick_lars_big_w<GT, 128>(G); break;
    }
    if (k) return k;
    if (np2_group_count(G))
        if (const Np2LarsKernel q = pick_lars_np2(W, G, sizeof(GT) == 2)) return q;
    switch (seg_levels(W > G ? W : G)) {
        case 3: return lars_norms_seg<GT, 3>;
        case 4: return lars_norms_seg<GT, 4>;
        case 5: return lars_norms_seg<GT, 5>;
    }
    return lars_norms_seg<GT, 8>;
}

// LARS workspace layout: [gbar scratch | per-chunk partials | trust ratios],
// each part starting on a 256-byte boundary.
struct LarsLayout {
    size_t gbar, partials, trust, total;
};

size_t round256(size_t x) { return (x + 255) / 256 * 256; }

LarsLayout lars_layout(const lsgd_plan* plan) {
    LarsLayout l;
    l.gbar = 0;
    l.partials = round256(static_cast<size_t>(plan->gbar_floats) * sizeof(float));
    l.trust = l.partials + round256(static_cast<size_t>(plan->n_chunks) * 2 * sizeof(double));
    l.total = l.trust + round256(static_cast<size_t>(plan->n_tensors) * sizeof(float));
    return l;
}

void free_plan(lsgd_plan* p) {
    if (!p) return;
    if (p->d_chunks) (void)hipFree(p->d_chunks);
    if (p->d_bucket_begin) (void)hipFree(p->d_bucket_begin);
    if (p->d_copy_desc) (void)hipFree(p->d_copy_desc);
    if (p->d_ptrs) (void)hipFree(p->d_ptrs);
    if (p->d_gbar_off) (void)hipFree(p->d_gbar_off);
    if (p->d_tensor_chunks) (void)hipFree(p->d_tensor_chunks);
    if (p->d_lars_exclude) (void)hipFree(p->d_lars_exclude);
    delete p->ranges;
    delete p;
}

}  // namespace

// The LARS step of a plan with its scratch at `workspace`. A caller-owned
// workspace is checked for size, alignment and overlap with every buffer of
// the call; a library-owned one (`library_workspace`, the per-device array of
// lsgd_lars_step_plan_noalloc) cannot overlap caller memory, and then the
// call also allocates nothing on the host: trust_out and lr_device are
// checked against the plan's ranges one by one.
lsgd_status lars_step(const lsgd_plan* plan, float lr, float momentum_coef, float weight_decay, float trust_coef,
                      void* workspace, size_t workspace_bytes, bool library_workspace, float* trust_out,
                      const float* lr_device, void* stream) {
    if (!plan) return fail(LSGD_ERR_NULL, "plan is NULL");
    if (!workspace) return fail(LSGD_ERR_NULL, "workspace is NULL");
    const LarsLayout l = lars_layout(plan);
    if (workspace_bytes < l.total)
        return fail(LSGD_ERR_SIZE, "workspace_bytes=%zu < %zu (lsgd_lars_workspace_size)", workspace_bytes, l.total);
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return fail(LSGD_ERR_ALIGN, "workspace is not 256-byte aligned");
    if (trust_out && (reinterpret_cast<uintptr_t>(trust_out) & 3u) != 0)
        return fail(LSGD_ERR_ALIGN, "trust_out is not 4-byte aligned");
    if (lr_device && (reinterpret_cast<uintptr_t>(lr_device) & 3u) != 0)
        return fail(LSGD_ERR_ALIGN, "lr_device is not 4-byte aligned");
    const uintptr_t tb = reinterpret_cast<uintptr_t>(trust_out);
    const uintptr_t te = tb + static_cast<uintptr_t>(plan->n_tensors) * sizeof(float);
    const uintptr_t lb = reinterpret_cast<uintptr_t>(lr_device);
    const uintptr_t le = lb + sizeof(float);
    lsgd_status st = LSGD_OK;
    if (library_workspace) {
        auto overlaps = [](uintptr_t b0, uintptr_t e0, uintptr_t b1, uintptr_t e1) { return b0 < e1 && b1 < e0; };
        if (trust_out && lr_device && overlaps(tb, te, lb, le))
            return fail(LSGD_ERR_ALIAS, "written buffer trust_out overlaps lr_device");
        for (const Range& r : *plan->ranges) {
            if (trust_out && overlaps(tb, te, r.begin, r.end))
                return fail(LSGD_ERR_ALIAS, "written buffer trust_out overlaps %s", r.what);
            if (lr_device && r.written && overlaps(lb, le, r.begin, r.end))
                return fail(LSGD_ERR_ALIAS, "buffer lr_device overlaps written buffer %s", r.what);
        }
    } else {
        std::vector<Range> ranges(*plan->ranges);
        const uintptr_t wb = reinterpret_cast<uintptr_t>(workspace);
        ranges.push_back(Range{wb, wb + l.total, true, "workspace"});
        if (trust_out) ranges.push_back(Range{tb, te, true, "trust_out"});
        if (lr_device) ranges.push_back(Range{lb, le, false, "lr_device"});
        if ((st = check_overlap(ranges)) != LSGD_OK) return st;
    }
    if (plan->W == 0) return fail(LSGD_ERR_GROUPS, "the LARS step needs equal group sizes; this plan's differ");
    if ((st = check_device(plan)) != LSGD_OK) return st;

    LarsArgs la;
    memset(&la, 0, sizeof la);
    LaunchShape ls;
    la.pa = plan_args(plan, Hyper{lr, momentum_coef, weight_decay}, lr_device, ls);
    la.gbar_off = plan->d_gbar_off;
    la.tensor_chunks = plan->d_tensor_chunks;
    char* ws = static_cast<char*>(workspace);
    la.gbar = reinterpret_cast<float*>(ws + l.gbar);
    la.partials = reinterpret_cast<double*>(ws + l.partials);
    la.trust = reinterpret_cast<float*>(ws + l.trust);
    la.trust_out = trust_out;
    la.exclude = plan->d_lars_exclude;
    la.n_tensors = plan->n_tensors;
    la.trust_coef = trust_coef;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (plan->n_buckets > 0) {
        int32_t W = plan->W, G = plan->n_groups;
        if (one_group_form(W, G, false)) {
            W = plan->n_workers;
            G = 1;
            la.pa.W = W;
            la.pa.n_groups = 1;
            la.pa.group_start[0] = 0;
            la.pa.group_start[1] = static_cast<uint8_t>(W);
        }
        const LarsKernel k1 = plan->gdt == LSGD_BF16 ? pick_lars<uint16_t>(W, G) : pick_lars<float>(W, G);
        hipLaunchKernelGGL(k1, dim3(ls.blocks), dim3(kBlock), 0, s, la);
        if ((st = check_launch("lsgd_lars_step_plan (norms)")) != LSGD_OK) return st;
    }
    hipLaunchKernelGGL(lars_trust_kernel, dim3(plan->n_tensors), dim3(kBlock), 0, s, la);
    if ((st = check_launch("lsgd_lars_step_plan (trust)")) != LSGD_OK) return st;
    if (plan->n_buckets == 0) return LSGD_OK;
    // the update reads and writes as lsgd_sgd_step does: the same copy-out rule
    const bool split = separate_copy_out_update(plan->n_replicas, plan->rdt == LSGD_BF16 ? 2 : 4,
                                                use_cached_state(plan->n_workers, plan->total_elems));
    if (split) la.pa.n_replicas = 0;
    hipLaunchKernelGGL(lars_update_kernel<2>, dim3(ls.blocks), dim3(kBlock), 0, s, la);
    if ((st = check_launch("lsgd_lars_step_plan (update)")) != LSGD_OK || !split) return st;
    la.pa.n_replicas = plan->n_replicas;
    return plan->rdt == LSGD_BF16 ? launch_plan_copy_out<8, kPlanCopyRKBF16>(plan, la.pa, s)
                                  : launch_plan_copy_out<4, kPlanCopyRKF32>(plan, la.pa, s);
}

}  // namespace lsgd

using namespace lsgd;

extern "C" {

LSGD_API lsgd_status lsgd_plan_create(lsgd_plan** out, int32_t n_tensors, const int64_t* numel,
                                      float* const* params, float* const* momentum,
                                      const void* const* grads, lsgd_dtype gdt, int32_t n_workers,
                                      const int32_t* group_of_worker, int32_t n_groups,
                                      void* const* replicas, int32_t n_replicas, lsgd_dtype rdt) {
    if (!out) return fail(LSGD_ERR_NULL, "out is NULL");
    *out = nullptr;
    if (n_tensors < 1) return fail(LSGD_ERR_SIZE, "n_tensors=%d < 1", n_tensors);
    if (!numel) return fail(LSGD_ERR_NULL, "numel is NULL");
    std::vector<int32_t> order, gstart;
    lsgd_status st = partition_order(n_workers, group_of_worker, n_groups, order, gstart);
    if (st != LSGD_OK) return st;
    // equal group sizes (the mean-of-means step needs them) give W > 0
    int32_t max_group = 0;
    bool equal = true;
    for (int32_t j = 0; j < n_groups; ++j) {
        const int32_t c = gstart[j + 1] - gstart[j];
        max_group = std::max(max_group, c);
        equal = equal && c == gstart[1] - gstart[0];
    }
    if (gdt != LSGD_F32 && gdt != LSGD_BF16) return fail(LSGD_ERR_DTYPE, "gradient dtype %d", (int)gdt);
    if (rdt != LSGD_F32 && rdt != LSGD_BF16) return fail(LSGD_ERR_DTYPE, "replica dtype %d", (int)rdt);
    if (n_replicas < 0 || n_replicas > kMaxReplicas)
        return fail(LSGD_ERR_SIZE, "n_replicas=%d outside [0, %d]", n_replicas, kMaxReplicas);
    if (!params || !momentum || !grads) return fail(LSGD_ERR_NULL, "params, momentum or grads is NULL");
    if (n_replicas > 0 && !replicas) return fail(LSGD_ERR_NULL, "replicas is NULL with n_replicas=%d", n_replicas);

    const size_t gsz = gdt == LSGD_BF16 ? 2 : 4, rsz = rdt == LSGD_BF16 ? 2 : 4;
    const int32_t stride = 2 + n_workers + n_replicas;
    std::vector<void*> table(static_cast<size_t>(n_tensors) * stride, nullptr);
    std::vector<Range> ranges;
    std::vector<PlanChunk> chunks;
    std::vector<int32_t> bucket_begin;
    // one tile pass of the kernel, times the launch shape's passes per workgroup
    const int32_t W = equal ? n_workers / n_groups : 0;
    const int tile = gdt == LSGD_BF16 ? pick_plan<uint16_t>(W, n_groups).tile : pick_plan<float>(W, n_groups).tile;
    const int64_t kPiece = (gdt == LSGD_BF16 ? piece_elems<uint16_t>(tile) : piece_elems<float>(tile)) *
                           launch_passes_per_block();
    int64_t bucket_fill = kPiece;  // forces a new bucket at the first piece
    std::vector<int64_t> gbar_off(n_tensors, 0);
    std::vector<int32_t> tensor_chunks(n_tensors + 1, 0);
    int64_t gbar_floats = 0;
    for (int32_t t = 0; t < n_tensors; ++t) {
        const int64_t ne = numel[t];
        if (ne < 0) return fail(LSGD_ERR_SIZE, "numel[%d]=%lld < 0", t, static_cast<long long>(ne));
        tensor_chunks[t] = static_cast<int32_t>(std::min<size_t>(chunks.size(), 0x7fffffff));
        gbar_off[t] = gbar_floats;
        gbar_floats += (ne + kGbarAlign - 1) / kGbarAlign * kGbarAlign;
        if (ne == 0) continue;
        void** row = &table[static_cast<size_t>(t) * stride];
        auto add = [&](void* p, size_t esz, bool written, const char* what, int idx) -> lsgd_status {
            if (!p) return fail(LSGD_ERR_NULL, "%s[%d] of tensor %d is NULL", what, idx, t);
            if (!aligned16(p)) return fail(LSGD_ERR_ALIGN, "%s[%d] of tensor %d is not 16-byte aligned", what, idx, t);
            const uintptr_t b = reinterpret_cast<uintptr_t>(p);
            ranges.push_back(Range{b, b + static_cast<uintptr_t>(ne) * esz, written, what});
            return LSGD_OK;
        };
        if ((st = add(params[t], 4, true, "params", t)) != LSGD_OK) return st;
        if ((st = add(momentum[t], 4, true, "momentum", t)) != LSGD_OK) return st;
        row[0] = params[t];
        row[1] = momentum[t];
        for (int32_t k = 0; k < n_workers; ++k) {
            const int32_t w = order[k];
            void* g = const_cast<void*>(grads[static_cast<size_t>(w) * n_tensors + t]);
            if ((st = add(g, gsz, false, "grads", w)) != LSGD_OK) return st;
            row[2 + k] = g;
        }
        for (int32_t r = 0; r < n_replicas; ++r) {
            void* rp = replicas[static_cast<size_t>(r) * n_tensors + t];
            if ((st = add(rp, rsz, true, "replicas", r)) != LSGD_OK) return st;
            row[2 + n_workers + r] = rp;
        }
        for (int64_t s0 = 0; s0 < ne; s0 += kPiece) {
            const int64_t len = std::min(kPiece, ne - s0);
            if (bucket_fill + len > kPiece) {
                bucket_begin.push_back(static_cast<int32_t>(chunks.size()));
                bucket_fill = 0;
            }
            // every piece but a tensor's last has len == kPiece (a multiple of the unit)
            chunks.push_back(PlanChunk{t, 0, s0, len});
            bucket_fill += len;
        }
    }
    if ((st = check_overlap(ranges)) != LSGD_OK) return st;
    if (chunks.size() > 0x7fffffff) return fail(LSGD_ERR_SIZE, "too many pieces");
    // one workgroup per bucket (and per tensor in the LARS trust kernel), in one launch
    if (static_cast<int64_t>(bucket_begin.size()) > kMaxGridBlocks || n_tensors > kMaxGridBlocks)
        return fail(LSGD_ERR_SIZE, "more than %lld buckets or tensors", static_cast<long long>(kMaxGridBlocks));
    bucket_begin.push_back(static_cast<int32_t>(chunks.size()));
    tensor_chunks[n_tensors] = static_cast<int32_t>(chunks.size());

    lsgd_plan* p = new lsgd_plan;
    memset(p, 0, sizeof *p);
    if (hipGetDevice(&p->device) != hipSuccess) {
        delete p;
        return fail(LSGD_ERR_HIP, "hipGetDevice failed");
    }
    p->n_tensors = n_tensors;
    p->n_workers = n_workers;
    p->n_groups = n_groups;
    p->W = W;
    p->max_group = max_group;
    for (int32_t j = 0; j <= n_groups; ++j) p->group_start[j] = gstart[j];
    p->n_replicas = n_replicas;
    p->gdt = gdt;
    p->rdt = rdt;
    p->n_chunks = static_cast<int32_t>(chunks.size());
    p->n_buckets = static_cast<int32_t>(bucket_begin.size()) - 1;
    p->stride = stride;
    p->piece = kPiece;
    for (int32_t t = 0; t < n_tensors; ++t) p->total_elems += numel[t];
    p->gbar_floats = gbar_floats;
    p->ranges = new std::vector<Range>(ranges);
    hipError_t e = hipSuccess;
    const size_t chunk_bytes = std::max<size_t>(1, chunks.size()) * sizeof(PlanChunk);
    const size_t bucket_bytes = bucket_begin.size() * sizeof(int32_t);
    const size_t table_bytes = table.size() * sizeof(void*);
    if (e == hipSuccess) e = hipMalloc(&p->d_chunks, chunk_bytes);
    if (e == hipSuccess) e = hipMalloc(&p->d_bucket_begin, bucket_bytes);
    if (e == hipSuccess) e = hipMalloc(&p->d_ptrs, table_bytes);
    if (e == hipSuccess && !chunks.empty())
        e = hipMemcpy(p->d_chunks, chunks.data(), chunks.size() * sizeof(PlanChunk), hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(p->d_bucket_begin, bucket_begin.data(), bucket_bytes, hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(p->d_ptrs, table.data(), table_bytes, hipMemcpyHostToDevice);
    std::vector<CopyDesc> desc(static_cast<size_t>(std::max(p->n_buckets, 1)));
    for (int32_t b = 0; b < p->n_buckets; ++b) {
        const PlanChunk& ch = chunks[static_cast<size_t>(bucket_begin[b])];
        desc[b] = CopyDesc{static_cast<const float*>(table[static_cast<size_t>(ch.tensor) * stride]), ch.tensor,
                           bucket_begin[b + 1] - bucket_begin[b], ch.start, ch.len};
    }
    if (e == hipSuccess) e = hipMalloc(&p->d_copy_desc, desc.size() * sizeof(CopyDesc));
    if (e == hipSuccess)
        e = hipMemcpy(p->d_copy_desc, desc.data(), desc.size() * sizeof(CopyDesc), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMalloc(&p->d_gbar_off, gbar_off.size() * sizeof(int64_t));
    if (e == hipSuccess) e = hipMalloc(&p->d_lars_exclude, static_cast<size_t>(n_tensors));
    if (e == hipSuccess) {
        const std::vector<uint8_t> none(static_cast<size_t>(n_tensors), 0);
        e = hipMemcpy(p->d_lars_exclude, none.data(), none.size(), hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipMalloc(&p->d_tensor_chunks, tensor_chunks.size() * sizeof(int32_t));
    if (e == hipSuccess)
        e = hipMemcpy(p->d_gbar_off, gbar_off.data(), gbar_off.size() * sizeof(int64_t), hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(p->d_tensor_chunks, tensor_chunks.data(), tensor_chunks.size() * sizeof(int32_t),
                      hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        free_plan(p);
        return fail(LSGD_ERR_HIP, "lsgd_plan_create: %s", hipGetErrorString(e));
    }
    *out = p;
    return LSGD_OK;
}

LSGD_API lsgd_status lsgd_step_plan_ex(const lsgd_plan* plan, float lr, float momentum_coef,
                                       float weight_decay, const lsgd_step_options* options,
                                       void* stream) {
    if (!plan) return fail(LSGD_ERR_NULL, "plan is NULL");
    const lsgd_step_options none = {LSGD_REDUCE_MEAN_OF_MEANS, 0, nullptr};
    const lsgd_step_options& o = options ? *options : none;
    if (o.reduction != LSGD_REDUCE_MEAN_OF_MEANS && o.reduction != LSGD_REDUCE_LITERAL)
        return fail(LSGD_ERR_UNSUPPORTED, "reduction %d", o.reduction);
    const bool literal = o.reduction == LSGD_REDUCE_LITERAL;
    const bool bcast = o.broadcast_grad != 0;
    const float* lr_device = o.lr_device;
    if (!literal && plan->W == 0)
        return fail(LSGD_ERR_GROUPS, "the mean-of-means step needs equal group sizes; this plan's differ");
    if (bcast && plan->gdt != LSGD_F32)
        return fail(LSGD_ERR_DTYPE, "broadcast_grad needs binary32 gradients");
    if (lr_device && (reinterpret_cast<uintptr_t>(lr_device) & 3u) != 0)
        return fail(LSGD_ERR_ALIGN, "lr_device is not 4-byte aligned");
    if (bcast || lr_device) {
        std::vector<Range> ranges(*plan->ranges);
        if (bcast)   // the gradient buffers are written too
            for (Range& r : ranges)
                if (strcmp(r.what, "grads") == 0) r.written = true;
        if (lr_device) {
            const uintptr_t lb = reinterpret_cast<uintptr_t>(lr_device);
            ranges.push_back(Range{lb, lb + sizeof(float), false, "lr_device"});
        }
        lsgd_status st = check_overlap(ranges);
        if (st != LSGD_OK) return st;
    }
    if (plan->n_buckets == 0) return LSGD_OK;
    lsgd_status st = check_device(plan);
    if (st != LSGD_OK) return st;
    LaunchShape ls;
    PlanArgs a = plan_args(plan, Hyper{lr, momentum_coef, weight_decay}, lr_device, ls);
    a.literal = literal ? 1 : 0;
    const bool cached = use_cached_state(plan->n_workers, plan->total_elems);
    // equal groups (W > 0): the compile-time kernels for powers of two, for
    // either reduction; the segmented kernel otherwise
    PlanKernel k = nullptr;
    bool segmented = true;
    int32_t W = plan->W, G = plan->n_groups;
    if (one_group_form(W, G, literal)) {
        W = plan->n_workers;
        G = 1;
        a.W = W;
        a.n_groups = 1;
        a.group_start[0] = 0;
        a.group_start[1] = static_cast<uint8_t>(W);
    }
    if (W > 0) {
        const PlanPick pk = plan->gdt == LSGD_BF16 ? pick_plan<uint16_t>(W, G, cached)
                                                   : pick_plan<float>(W, G, cached);
        k = pk.kernel;
        segmented = pk.segmented;
    } else {
        const int32_t max_count = std::max(plan->max_group, plan->n_groups);
        k = plan->gdt == LSGD_BF16 ? plan_seg<uint16_t>(max_count, cached) : plan_seg<float>(max_count, cached);
    }
    // as for flat steps: the replicas and the broadcast's copies of the mean
    // gradient to the other N - 1 members go to copy passes of their own
    // where the rule takes the separate form
    const int32_t bcast_copies = bcast ? plan->n_workers - 1 : 0;
    const bool split = separate_copy_out_bytes(
        plan->n_workers, plan->gdt == LSGD_BF16 ? 2 : 4,
        static_cast<int64_t>(plan->n_replicas) * (plan->rdt == LSGD_BF16 ? 2 : 4) + 4 * bcast_copies,
        plan->total_elems, segmented || (W & (W - 1)) != 0 || (G & (G - 1)) != 0);
    a.bcast_grad = bcast ? (split ? 1 : plan->n_workers) : 0;
    // split: the step kernel writes the first k replicas, the copy-out pass the rest
    const int32_t k_step = split ? replicas_in_step(plan->n_workers, plan->n_replicas, plan->rdt == LSGD_BF16 ? 2 : 4,
                                                    plan->total_elems)
                                 : plan->n_replicas;
    a.n_replicas = k_step;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k, dim3(ls.blocks), dim3(kBlock), 0, s, a);
    if ((st = check_launch("lsgd_step_plan")) != LSGD_OK || !split) return st;
    if (plan->n_replicas > k_step) {
        a.copy_dst = 2 + plan->n_workers + k_step;
        a.n_replicas = plan->n_replicas - k_step;
        st = plan->rdt == LSGD_BF16 ? launch_plan_copy_out<8, kPlanCopyRKBF16>(plan, a, s)
                                    : launch_plan_copy_out<4, kPlanCopyRKF32>(plan, a, s);
        if (st != LSGD_OK) return st;
    }
    if (bcast_copies > 0) {   // the first member's gradient (slot 2) to the others (slots 3 ..)
        a.copy_src = 2;
        a.copy_dst = 3;
        a.n_replicas = bcast_copies;
        a.rdt = static_cast<int32_t>(LSGD_F32);
        return launch_plan_copy_out<4, kPlanCopyRKF32>(plan, a, s);
    }
    return LSGD_OK;
}

LSGD_API lsgd_status lsgd_plan_copy_out(const lsgd_plan* plan, void* stream) {
    if (!plan) return fail(LSGD_ERR_NULL, "plan is NULL");
    if (plan->n_buckets == 0 || plan->n_replicas == 0) return LSGD_OK;
    lsgd_status st = check_device(plan);
    if (st != LSGD_OK) return st;
    LaunchShape ls;
    PlanArgs a = plan_args(plan, Hyper{0.f, 0.f, 0.f}, nullptr, ls);
    const hipStream_t s = static_cast<hipStream_t>(stream);
    return plan->rdt == LSGD_BF16 ? launch_plan_copy_out<8, kPlanCopyRKBF16>(plan, a, s)
                                  : launch_plan_copy_out<4, kPlanCopyRKF32>(plan, a, s);
}

LSGD_API lsgd_status lsgd_step_plan(const lsgd_plan* plan, float lr, float momentum_coef,
                                    float weight_decay, void* stream) {
    return lsgd_step_plan_ex(plan, lr, momentum_coef, weight_decay, nullptr, stream);
}

LSGD_API lsgd_status lsgd_lars_workspace_size(const lsgd_plan* plan, size_t* bytes) {
    if (!plan) return fail(LSGD_ERR_NULL, "plan is NULL");
    if (!bytes) return fail(LSGD_ERR_NULL, "bytes is NULL");
    *bytes = lars_layout(plan).total;
    return LSGD_OK;
}

LSGD_API lsgd_status lsgd_lars_step_plan(const lsgd_plan* plan, float lr, float momentum_coef,
                                         float weight_decay, float trust_coef, void* workspace,
                                         size_t workspace_bytes, float* trust_out,
                                         const float* lr_device, void* stream) {
    return lsgd::lars_step(plan, lr, momentum_coef, weight_decay, trust_coef, workspace, workspace_bytes, false,
                           trust_out, lr_device, stream);
}

LSGD_API lsgd_status lsgd_plan_set_lars_exclude(lsgd_plan* plan, const uint8_t* exclude) {
    if (!plan) return fail(LSGD_ERR_NULL, "plan is NULL");
    std::vector<uint8_t> flags(static_cast<size_t>(plan->n_tensors), 0);
    if (exclude)
        for (int32_t t = 0; t < plan->n_tensors; ++t) flags[t] = exclude[t] ? 1 : 0;
    lsgd_status st = check_device(plan);
    if (st != LSGD_OK) return st;
    const hipError_t e = hipMemcpy(plan->d_lars_exclude, flags.data(), flags.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(LSGD_ERR_HIP, "lsgd_plan_set_lars_exclude: %s", hipGetErrorString(e));
    return LSGD_OK;
}

LSGD_API void lsgd_plan_destroy(lsgd_plan* plan) { free_plan(plan); }

}  // extern "C"
