// Host-side helpers shared by the translation units of liblsgd: error text,
// argument validation, the membership-to-member-order map and launch sizing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "lsgd.h"

namespace lsgd {

// Records the detail of a failing call for lsgd_last_error() and returns `st`.
lsgd_status fail(lsgd_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// hipGetLastError() after a launch, mapped to LSGD_ERR_HIP with its text.
lsgd_status check_launch(const char* what);

// Subgroup indexing: validates the worker->group map (every id in [0, G), G | N,
// every group of exactly W = N/G members) and returns the member order, G rows
// of W worker ids, each row ascending. Returns LSGD_OK or LSGD_ERR_GROUPS/SIZE.
lsgd_status member_order(int32_t n_workers, const int32_t* group_of_worker, int32_t n_groups,
                         std::vector<int32_t>& order);

// Any partition into non-empty groups (the paper-literal reduction): member
// order grouped by group id, ascending worker id inside a group, and the
// G + 1 group offsets into it. LSGD_ERR_GROUPS for an id out of range or an
// empty group.
lsgd_status partition_order(int32_t n_workers, const int32_t* group_of_worker, int32_t n_groups,
                            std::vector<int32_t>& order, std::vector<int32_t>& group_start);

bool aligned16(const void* p);

// A byte range [begin, end) of one buffer argument; `written` for outputs.
struct Range {
    uintptr_t begin, end;
    bool written;
    const char* what;
};

// LSGD_ERR_ALIAS if a written range overlaps any other range (empty ranges
// never overlap). Sort-and-sweep, O(k log k).
lsgd_status check_overlap(std::vector<Range>& ranges);

// Default launch shape of the planless kernels: automatic XCD chunk (each XCD
// walks kAutoChunkBytes of every buffer per turn), one-shot grids, one pass per
// workgroup. Changed process-wide by lsgd_set_launch_shape.
constexpr int32_t kXcdChunkAuto = -1;
constexpr int64_t kAutoChunkBytes = 512 * 1024;
constexpr int32_t kDefaultXcdChunk = kXcdChunkAuto;
constexpr int32_t kDefaultBlocksPerCu = 0;
constexpr int32_t kDefaultUnitsPerLane = 1;

struct LaunchShape {
    unsigned blocks;     // grid size (padded to a multiple of 8 * xcd_chunk)
    uint32_t xcd_chunk;  // 0 when the grid is too small to renumber
    uint32_t upl;        // consecutive passes of kBlock units per logical block
};

// Grid for `units` 16-byte units processed in lane tiles of `tile` units:
// ceil(units / (kBlock * tile * upl)) workgroups, capped at compute units *
// blocks-per-CU when that is set (the kernels then grid-stride), then padded
// for the XCD chunking.
LaunchShape launch_shape(int64_t units, int tile = 1);

// The launch shape's passes per workgroup (units_per_lane).
int32_t launch_passes_per_block();

// Whether a step with N gradients of gsz bytes, n elements and `copy_bytes`
// bytes per element of copies (replicas, and the gradient broadcast's copies
// of the mean gradient to the other members) writes them in copy passes of
// their own (lsgd_set_copy_out_mode); `other_layout`: the step's grouping is
// not power-of-two groups in a power-of-two count.
bool separate_copy_out_bytes(int32_t n_workers, size_t gsz, int64_t copy_bytes, int64_t n, bool other_layout);
// One worker per group, in a group count with no compile-time kernel (not a
// power of two, nor 3, 5, 6, 7 or 12), under the mean of means: the result equals that of one group
// of all N workers in the same member order (the same pairwise sum over the
// same sequence of values, then one division by N = G; the group means are
// the members themselves), which the segmented kernels compute with one
// accumulator instead of finishing a group at every member. The steps take
// that form (W = N, G = 1). Measured on the ResNet-50 size, same process:
// 12x1 binary32 62% -> 82% of 8 TB/s (R = N) and 51% -> 80% (R = 0), 6x1
// 79% -> 88%, 12x1 bfloat16 50% -> 76% and 34% -> 66%.
// Group counts other than powers of two that have compile-time kernels too
// (lsgd_np2.hpp).
inline bool np2_group_count(int G) { return G == 3 || G == 5 || G == 6 || G == 7 || G == 12; }

inline bool one_group_form(int32_t W, int32_t G, bool literal) {
    return !literal && W == 1 && G > 1 && (G & (G - 1)) != 0 && !np2_group_count(G);
}
// With the separate copy-out: how many of the n_replicas replicas (rsz bytes
// each) the step kernel still writes itself; the copy-out pass writes the
// rest (lsgd_set_step_replicas).
int32_t replicas_in_step(int32_t n_workers, int32_t n_replicas, size_t rsz, int64_t n);
// The same for lsgd_sgd_step and the LARS update; `cached`: their parameter
// and momentum accesses go through the caches.
bool separate_copy_out_update(int32_t n_replicas, size_t rsz, bool cached);

// Largest grid of a grid-stride kernel whose XCD assignment must not change
// between strides: kMaxGridBlocks, or the blocks_per_cu cap of
// lsgd_set_launch_shape rounded down to a multiple of 8.
int64_t stride_grid_cap();

// Workgroups per window of the replica-major copy-out pass over `blocks`
// workgroups that each read `block_p_bytes` of p: about 8 MB of p per window,
// windows of equal size, a multiple of 8 workgroups (so that each XCD reads
// the same part of the window for every replica).
int64_t copy_window_blocks(int64_t block_p_bytes, int64_t blocks);

// Grid of exactly `blocks` logical workgroups, each covering `block_bytes` of
// every buffer, padded for the XCD chunking (kernels skip logical blocks
// >= `blocks`).
LaunchShape pad_for_xcd_chunk(int64_t blocks, int64_t block_bytes);

// Compute units of the current device (cached per device).
int device_cus();

inline bool is_pow2_le16(int x) { return x == 1 || x == 2 || x == 4 || x == 8 || x == 16; }

// lsgd_lars_step_plan with its scratch at `workspace` (workspace_bytes long);
// `library_workspace`: the scratch is the library's own per-device array
// (lsgd_lars_step_plan_noalloc), which no caller buffer can overlap, and the
// call then makes no host allocation either.
lsgd_status lars_step(const lsgd_plan* plan, float lr, float momentum_coef, float weight_decay, float trust_coef,
                      void* workspace, size_t workspace_bytes, bool library_workspace, float* trust_out,
                      const float* lr_device, void* stream);

}  // namespace lsgd
