// Measurement utility of liblsgd: lsgd_stream_copy (declared in lsgd_bench.h).
#include "lsgd_bench.h"
#include "lsgd_host.hpp"
#include "lsgd_kernels.hpp"

namespace lsgd {
namespace {

// Plain streaming copy: one 16-byte unit per lane, in the kernels' XCD-chunked
// block order.
__global__ __launch_bounds__(kBlock) void stream_copy_kernel(u32x4* __restrict__ dst, const u32x4* __restrict__ src,
                                                            int64_t units, uint32_t chunk) {
    for_units(units, chunk, 1, [&](int64_t u) {
        __builtin_nontemporal_store(__builtin_nontemporal_load(src + u), dst + u);
    });
}

}  // namespace
}  // namespace lsgd

using namespace lsgd;

extern "C" {

LSGD_API lsgd_status lsgd_stream_copy(void* dst, const void* src, int64_t bytes, void* stream) {
    if (bytes < 0 || bytes % 16 != 0)
        return fail(LSGD_ERR_SIZE, "bytes=%lld is not a non-negative multiple of 16",
                    static_cast<long long>(bytes));
    if (bytes == 0) return LSGD_OK;
    if (!dst || !src) return fail(LSGD_ERR_NULL, "dst or src is NULL");
    if (!aligned16(dst) || !aligned16(src)) return fail(LSGD_ERR_ALIGN, "dst or src is not 16-byte aligned");
    std::vector<Range> ranges{Range{reinterpret_cast<uintptr_t>(dst), reinterpret_cast<uintptr_t>(dst) + bytes, true, "dst"},
                              Range{reinterpret_cast<uintptr_t>(src), reinterpret_cast<uintptr_t>(src) + bytes, false, "src"}};
    lsgd_status st = check_overlap(ranges);
    if (st != LSGD_OK) return st;
    const int64_t units = bytes / 16;
    const LaunchShape ls = launch_shape(units);
    hipLaunchKernelGGL(stream_copy_kernel, dim3(ls.blocks), dim3(kBlock), 0,
                       static_cast<hipStream_t>(stream), static_cast<u32x4*>(dst),
                       static_cast<const u32x4*>(src), units, ls.xcd_chunk);
    return check_launch("lsgd_stream_copy");
}

}  // extern "C"
