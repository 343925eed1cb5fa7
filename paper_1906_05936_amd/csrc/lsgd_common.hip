// Host helpers of liblsgd: error reporting, membership validation, aliasing
// checks and launch sizing.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <atomic>
#include <mutex>

#include "lsgd_host.hpp"
#include "lsgd_kernels.hpp"

namespace lsgd {

namespace {
thread_local std::string t_last_error;

constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];

// Process-wide launch shape (lsgd_set_launch_shape). Results never depend on it.
std::atomic<int32_t> g_xcd_chunk{kDefaultXcdChunk};
std::atomic<int32_t> g_blocks_per_cu{kDefaultBlocksPerCu};
std::atomic<int32_t> g_units_per_lane{kDefaultUnitsPerLane};
std::atomic<int32_t> g_copy_out_mode{LSGD_COPY_OUT_AUTO};
std::atomic<int32_t> g_step_replicas{-1};   // lsgd_set_step_replicas (-1: automatic)
}  // namespace

lsgd_status fail(lsgd_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_last_error = buf;
    return st;
}

lsgd_status check_launch(const char* what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(LSGD_ERR_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
    return LSGD_OK;
}

lsgd_status member_order(int32_t n_workers, const int32_t* group_of_worker, int32_t n_groups,
                         std::vector<int32_t>& order) {
    if (n_workers < 1 || n_workers > kMaxWorkers)
        return fail(LSGD_ERR_SIZE, "n_workers=%d outside [1, %d]", n_workers, kMaxWorkers);
    if (n_groups < 1) return fail(LSGD_ERR_SIZE, "n_groups=%d < 1", n_groups);
    if (!group_of_worker) return fail(LSGD_ERR_NULL, "group_of_worker is NULL");
    if (n_workers % n_groups != 0)
        return fail(LSGD_ERR_GROUPS, "n_groups=%d does not divide n_workers=%d", n_groups, n_workers);
    const int32_t W = n_workers / n_groups;
    std::vector<int32_t> fill(n_groups, 0);
    order.assign(n_workers, -1);
    for (int32_t i = 0; i < n_workers; ++i) {
        const int32_t j = group_of_worker[i];
        if (j < 0 || j >= n_groups)
            return fail(LSGD_ERR_GROUPS, "group_of_worker[%d]=%d outside [0, %d)", i, j, n_groups);
        if (fill[j] == W)
            return fail(LSGD_ERR_GROUPS, "group %d has more than W=%d members", j, W);
        order[static_cast<size_t>(j) * W + fill[j]++] = i;  // i ascends, so rows ascend
    }
    for (int32_t j = 0; j < n_groups; ++j)
        if (fill[j] != W) return fail(LSGD_ERR_GROUPS, "group %d has %d members, expected %d", j, fill[j], W);
    return LSGD_OK;
}

lsgd_status partition_order(int32_t n_workers, const int32_t* group_of_worker, int32_t n_groups,
                            std::vector<int32_t>& order, std::vector<int32_t>& group_start) {
    if (n_workers < 1 || n_workers > kMaxWorkers)
        return fail(LSGD_ERR_SIZE, "n_workers=%d outside [1, %d]", n_workers, kMaxWorkers);
    if (n_groups < 1) return fail(LSGD_ERR_SIZE, "n_groups=%d < 1", n_groups);
    if (!group_of_worker) return fail(LSGD_ERR_NULL, "group_of_worker is NULL");
    if (n_groups > n_workers)
        return fail(LSGD_ERR_GROUPS, "n_groups=%d > n_workers=%d leaves a group empty", n_groups, n_workers);
    std::vector<int32_t> count(n_groups, 0);
    for (int32_t i = 0; i < n_workers; ++i) {
        const int32_t j = group_of_worker[i];
        if (j < 0 || j >= n_groups)
            return fail(LSGD_ERR_GROUPS, "group_of_worker[%d]=%d outside [0, %d)", i, j, n_groups);
        ++count[j];
    }
    group_start.assign(n_groups + 1, 0);
    for (int32_t j = 0; j < n_groups; ++j) {
        if (count[j] == 0) return fail(LSGD_ERR_GROUPS, "group %d is empty", j);
        group_start[j + 1] = group_start[j] + count[j];
    }
    order.assign(n_workers, -1);
    std::vector<int32_t> fill(group_start.begin(), group_start.end() - 1);
    for (int32_t i = 0; i < n_workers; ++i) order[fill[group_of_worker[i]]++] = i;
    return LSGD_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

lsgd_status check_overlap(std::vector<Range>& ranges) {
    ranges.erase(std::remove_if(ranges.begin(), ranges.end(),
                                [](const Range& r) { return r.end <= r.begin; }),
                 ranges.end());
    std::sort(ranges.begin(), ranges.end(),
              [](const Range& a, const Range& b) { return a.begin < b.begin; });
    uintptr_t max_end_any = 0, max_end_written = 0;
    const char* last_any = "";
    const char* last_written = "";
    for (const Range& r : ranges) {
        if (r.written && r.begin < max_end_any)
            return fail(LSGD_ERR_ALIAS, "written buffer %s overlaps %s", r.what, last_any);
        if (!r.written && r.begin < max_end_written)
            return fail(LSGD_ERR_ALIAS, "buffer %s overlaps written buffer %s", r.what, last_written);
        if (r.end > max_end_any) { max_end_any = r.end; last_any = r.what; }
        if (r.written && r.end > max_end_written) { max_end_written = r.end; last_written = r.what; }
    }
    return LSGD_OK;
}

int device_cus() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int c = g_cus[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0)
        c = 256;
    g_cus[dev].store(c, std::memory_order_relaxed);
    return c;
}

// `blocks` logical workgroups padded to a multiple of 8 * xcd_chunk (the chunk
// is dropped for grids smaller than one full turn of the eight XCDs). The
// automatic chunk gives each XCD kAutoChunkBytes of every buffer per turn:
// a workgroup covers `block_bytes` of each buffer.
LaunchShape pad_for_xcd_chunk(int64_t blocks, int64_t block_bytes) {
    LaunchShape ls;
    int64_t need = blocks < 1 ? 1 : blocks;
    int64_t chunk = g_xcd_chunk.load(std::memory_order_relaxed);
    if (chunk == kXcdChunkAuto) chunk = std::max<int64_t>(1, kAutoChunkBytes / block_bytes);
    const int64_t group = 8 * std::max<int64_t>(chunk, 1);
    if (chunk > 0 && need >= group && (need + group - 1) / group * group <= kMaxGridBlocks) {
        need = (need + group - 1) / group * group;
    } else {
        chunk = 0;
    }
    // The kernels grid-stride, so a capped grid still covers the work (the
    // renumbering is off in that case, so it stays a bijection).
    if (need > kMaxGridBlocks) need = kMaxGridBlocks;
    ls.blocks = static_cast<unsigned>(need);
    ls.xcd_chunk = static_cast<uint32_t>(chunk);
    ls.upl = 1;
    return ls;
}

int32_t launch_passes_per_block() { return g_units_per_lane.load(std::memory_order_relaxed); }

// Automatic rule, from same-process measurements of the fused pass against
// step-then-copy-out (the replica-major pass) at N = 4..128 gradients and
// R = 1..128 replicas, flat steps and plans, binary32 and bfloat16. With
// nontemporal parameter and momentum accesses the separate pass won once the
// replicas take 32 bytes per element or more (R = 16 with 16 gradients:
// +7-9%; R = 64: +18-20%) or the gradients 256 bytes (128 binary32
// gradients, R = 2: +6%, R = 128: +20%), and was within 3% either way below
// that. When parameters and momentum go through the caches
// (use_cached_state) the fused pass gains more, and the crossing moves to 64
// bytes: at 32 the fused pass won by 2-4% (4x4 R = 8, 2x2 R = 8, 4x4
// bfloat16 R = 16), at 64 the separate one by 3-12% (4x4 R = 16, 2x2 R = 16,
// the ResNet-50 plan), at 256 by 28%. Groupings other than power-of-two
// groups in a power-of-two count cross earlier there: with the segmented
// kernels the separate pass won by 5-8% at 56 and 60 replica bytes (2x7,
// 3x5, 5x3 binary32) and lost by 3-8% at 24 and 36 (2x3, 3x2, 1x9); with
// their compile-time kernels the fused form lost 4% at 3x5 and 11% at 3x5
// with bfloat16 gradients (60 bytes) and 13% at 12x1 bfloat16 (48 bytes).
// Their crossing is 48 bytes (`other_layout`).
bool separate_copy_out_bytes(int32_t n_workers, size_t gsz, int64_t copy_bytes, int64_t n, bool other_layout) {
    if (copy_bytes <= 0) return false;
    const int32_t mode = g_copy_out_mode.load(std::memory_order_relaxed);
    if (mode == LSGD_COPY_OUT_FUSED) return false;
    if (mode == LSGD_COPY_OUT_SEPARATE) return true;
    const int64_t grad_bytes = static_cast<int64_t>(n_workers) * static_cast<int64_t>(gsz);
    const int64_t crossing = !use_cached_state(n_workers, n) ? 32 : other_layout ? 48 : 64;
    return copy_bytes >= crossing || grad_bytes >= 256;
}

// With the separate copy-out the step kernel still writes the first k replicas
// itself: its stream mix is mostly reads, and a few write streams added to it
// cost less time than the copy-out pass saves by writing them. Measured on the
// ResNet-50-sized 4x4 binary32 step with 16 replicas, same process (k
// replicas in the step kernel, 16 - k in the pass): k = 0 6479 GB/s, 1 6508,
// 2 6489, 3 6641, 4 6690, 5 6706, 6 6647, 8 6553, 10 6476, 12 6381, 16 (the
// fused step) 6337; the 161-tensor plan k = 0 6285, 4 6402; 32 replicas k = 0
// 6621, 4 6775; 64 replicas k = 0 6746, 4 6840; 2x2 with 16 replicas even;
// with 128 binary32 gradients or 64 bfloat16 ones (nontemporal parameter and
// momentum accesses) every k > 0 lost (128: k = 2 -1.4%, 4 -2.2%; 64 bfloat16:
// k = 4 -2%, 16 -3.8%). The rule: 16 bytes of replicas per element in the
// step kernel where parameters and momentum go through the caches, none
// otherwise.
int32_t replicas_in_step(int32_t n_workers, int32_t n_replicas, size_t rsz, int64_t n) {
    const int32_t forced = g_step_replicas.load(std::memory_order_relaxed);
    if (forced >= 0) return std::min(forced, n_replicas);
    if (!use_cached_state(n_workers, n)) return 0;
    return std::min<int32_t>(n_replicas, static_cast<int32_t>(16 / rsz));
}

// 8 MB of p per window: 1 MB in each of the eight XCD L2 caches (4 MB each),
// re-read there for every replica. Windows of 4-20 MB measured alike; from
// 24 MB the window no longer stays in L2 and the pass slows by a third.
constexpr int64_t kCopyWindowBytes = 8 << 20;

int64_t copy_window_blocks(int64_t block_p_bytes, int64_t blocks) {
    const int64_t target = std::max<int64_t>(8, kCopyWindowBytes / block_p_bytes / 8 * 8);
    const int64_t windows = std::max<int64_t>(1, (blocks + target - 1) / target);
    return ((blocks + windows - 1) / windows + 7) / 8 * 8;   // equal windows, the last one barely padded
}

// The same choice for lsgd_sgd_step (reads 12 bytes per element, writes 8 plus
// the replicas) and the LARS update. Measured with nontemporal parameter and
// momentum accesses: with binary32 replicas the separate pass won from R = 4
// (+2%; R = 8: +4%, R = 16: +15%, R = 64: +10%) and lost below (R = 1: -11%);
// with bfloat16 replicas the fused pass won or tied at every R up to 64. With
// them through the caches (`cached`): the separate pass won from 16 replica
// bytes per element (binary32 R = 4: +3%, R = 16: +4%; bfloat16 R = 8: +4%,
// R = 16: +14%, R = 64: +11%) and lost below (bfloat16 R = 4: -9%).
bool separate_copy_out_update(int32_t n_replicas, size_t rsz, bool cached) {
    if (n_replicas <= 0) return false;
    const int32_t mode = g_copy_out_mode.load(std::memory_order_relaxed);
    if (mode == LSGD_COPY_OUT_FUSED) return false;
    if (mode == LSGD_COPY_OUT_SEPARATE) return true;
    if (cached) return static_cast<int64_t>(n_replicas) * static_cast<int64_t>(rsz) >= 16;
    return rsz == 4 && n_replicas >= 4;
}

int64_t stride_grid_cap() {
    const int32_t bpc = g_blocks_per_cu.load(std::memory_order_relaxed);
    if (bpc <= 0) return kMaxGridBlocks;
    const int64_t cap = static_cast<int64_t>(device_cus()) * bpc / 8 * 8;
    return std::min<int64_t>(kMaxGridBlocks, std::max<int64_t>(8, cap));
}

LaunchShape launch_shape(int64_t units, int tile) {
    const int64_t upl = g_units_per_lane.load(std::memory_order_relaxed);
    const int64_t span = static_cast<int64_t>(kBlock) * upl * (tile < 1 ? 1 : tile);
    int64_t need = (units + span - 1) / span;
    const int32_t bpc = g_blocks_per_cu.load(std::memory_order_relaxed);
    if (bpc > 0) {
        const int64_t cap = static_cast<int64_t>(device_cus()) * bpc;
        if (need > cap) need = cap;
    }
    LaunchShape ls = pad_for_xcd_chunk(need, static_cast<int64_t>(kBlock) * 16 * (tile < 1 ? 1 : tile) * upl);
    ls.upl = static_cast<uint32_t>(upl);
    return ls;
}

}  // namespace lsgd

extern "C" {

LSGD_API const char* lsgd_status_string(lsgd_status status) {
    switch (status) {
        case LSGD_OK: return "LSGD_OK";
        case LSGD_ERR_NULL: return "LSGD_ERR_NULL: a required pointer is NULL";
        case LSGD_ERR_SIZE: return "LSGD_ERR_SIZE: a size or count is out of range";
        case LSGD_ERR_GROUPS: return "LSGD_ERR_GROUPS: invalid subgroup membership";
        case LSGD_ERR_ALIGN: return "LSGD_ERR_ALIGN: a buffer is not 16-byte aligned";
        case LSGD_ERR_DTYPE: return "LSGD_ERR_DTYPE: unsupported dtype";
        case LSGD_ERR_HIP: return "LSGD_ERR_HIP: the HIP runtime reported an error";
        case LSGD_ERR_ALIAS: return "LSGD_ERR_ALIAS: a written buffer overlaps another buffer";
        case LSGD_ERR_UNSUPPORTED: return "LSGD_ERR_UNSUPPORTED: option not supported by this call";
    }
    return "unknown lsgd_status";
}

LSGD_API const char* lsgd_last_error(void) { return lsgd::t_last_error.c_str(); }

LSGD_API lsgd_status lsgd_set_launch_shape(int32_t xcd_chunk, int32_t blocks_per_cu,
                                           int32_t units_per_lane) {
    if (xcd_chunk < lsgd::kXcdChunkAuto || xcd_chunk > 65536)
        return lsgd::fail(LSGD_ERR_SIZE, "xcd_chunk=%d outside [-1, 65536]", xcd_chunk);
    if (blocks_per_cu < 0 || blocks_per_cu > 4096)
        return lsgd::fail(LSGD_ERR_SIZE, "blocks_per_cu=%d outside [0, 4096]", blocks_per_cu);
    if (units_per_lane < 1 || units_per_lane > 256)
        return lsgd::fail(LSGD_ERR_SIZE, "units_per_lane=%d outside [1, 256]", units_per_lane);
    lsgd::g_xcd_chunk.store(xcd_chunk, std::memory_order_relaxed);
    lsgd::g_blocks_per_cu.store(blocks_per_cu, std::memory_order_relaxed);
    lsgd::g_units_per_lane.store(units_per_lane, std::memory_order_relaxed);
    return LSGD_OK;
}

LSGD_API lsgd_status lsgd_set_copy_out_mode(int32_t mode) {
    if (mode != LSGD_COPY_OUT_AUTO && mode != LSGD_COPY_OUT_FUSED && mode != LSGD_COPY_OUT_SEPARATE)
        return lsgd::fail(LSGD_ERR_SIZE, "copy-out mode %d", mode);
    lsgd::g_copy_out_mode.store(mode, std::memory_order_relaxed);
    return LSGD_OK;
}

LSGD_API int32_t lsgd_get_copy_out_mode(void) { return lsgd::g_copy_out_mode.load(std::memory_order_relaxed); }

LSGD_API lsgd_status lsgd_set_step_replicas(int32_t replicas) {
    if (replicas < -1 || replicas > LSGD_MAX_REPLICAS)
        return lsgd::fail(LSGD_ERR_SIZE, "step replicas %d outside [-1, %d]", replicas, LSGD_MAX_REPLICAS);
    lsgd::g_step_replicas.store(replicas, std::memory_order_relaxed);
    return LSGD_OK;
}

LSGD_API int32_t lsgd_get_step_replicas(void) { return lsgd::g_step_replicas.load(std::memory_order_relaxed); }

LSGD_API lsgd_status lsgd_get_launch_shape(int32_t* xcd_chunk, int32_t* blocks_per_cu,
                                           int32_t* units_per_lane) {
    if (!xcd_chunk || !blocks_per_cu || !units_per_lane)
        return lsgd::fail(LSGD_ERR_NULL, "output pointer is NULL");
    *xcd_chunk = lsgd::g_xcd_chunk.load(std::memory_order_relaxed);
    *blocks_per_cu = lsgd::g_blocks_per_cu.load(std::memory_order_relaxed);
    *units_per_lane = lsgd::g_units_per_lane.load(std::memory_order_relaxed);
    return LSGD_OK;
}

}  // extern "C"
