// Device code of liblsgd's multi-tensor plans: the fused step over a list of
// tensors in one launch (chunk and bucket tables built by lsgd_plan_create),
// its copy-out pass, and the LARS step. Included by lsgd_plan.hip only.
#pragma once

#include "lsgd_kernels.hpp"

#pragma clang fp contract(off)

namespace lsgd {

// ------------------------------------------------------------- multi-tensor plan

// One piece of one tensor: elements [start, start+len). Pieces start at
// multiples of the unit size; only a tensor's last piece can end ragged.
struct PlanChunk {
    int32_t tensor;
    int32_t pad_;
    int64_t start;
    int64_t len;
};

// Per bucket, for the copy-out pass: its first piece (tensor, element range,
// the tensor's params) and the bucket's piece count, so that a workgroup
// finds its params address in one table read instead of three dependent ones.
struct CopyDesc {
    const float* p;
    int32_t tensor;
    int32_t n_chunks;
    int64_t start;
    int64_t len;
};

// Per tensor the device pointer table holds `stride` entries:
// [p, m, grads in member order (N), replicas (R)].
struct PlanArgs {
    const PlanChunk* chunks;
    const int32_t* bucket_begin;  // [n_buckets + 1]: workgroup b runs chunks [begin[b], begin[b+1])
    const CopyDesc* copy_desc;    // [n_buckets]
    void* const* ptrs;
    int32_t stride, n_workers, n_groups, W;
    int32_t n_replicas, rdt;
    int32_t n_buckets;
    uint32_t xcd_chunk;
    const float* lr_ptr;
    Hyper h;
    int32_t literal;       // paper-literal reduction (else mean of means)
    int32_t bcast_grad;    // write the mean gradient into the first bcast_grad (binary32) member buffers
    int32_t win_blocks;    // replica-major copy-out: buckets per window (a multiple of 8)
    int64_t copy_blocks;   // replica-major copy-out: logical workgroups (the grid strides over them)
    int32_t cached_state;  // LARS update: store parameters and momentum through the caches
    int32_t copy_src;      // copy-out pass: table slot of its source (0: p; 2: the first member's gradient)
    int32_t copy_dst;      // copy-out pass: table slot of its first destination (n_replicas of them)
    uint8_t group_start[kMaxWorkers + 4];  // runtime-layout kernel: group j is members [start[j], start[j+1])
};

// CACHED as for FlatSrcT (-1: PlanArgs::cached_state decides).
template <int CACHED>
struct PlanSrcT {
    void* const* t;  // this tensor's row of the pointer table
    const PlanArgs& a;
    Hyper h;
    __device__ const void* grad(int k) const { return read_table(&t[2 + k]); }
    __device__ float* p() const { return static_cast<float*>(read_table(&t[0])); }
    __device__ float* m() const { return static_cast<float*>(read_table(&t[1])); }
    __device__ void* replica(int r) const { return read_table(&t[2 + a.n_workers + r]); }
    __device__ int n_replicas() const { return a.n_replicas; }
    __device__ int rdt() const { return a.rdt; }
    __device__ Hyper hyper() const { return h; }
    __device__ int bcast_grad() const { return a.bcast_grad; }
    __device__ int n_workers() const { return a.n_workers; }
    __device__ int literal() const { return a.literal; }
    __device__ int cached_state() const { return CACHED < 0 ? a.cached_state : CACHED; }
};
using PlanSrc = PlanSrcT<-1>;

// One workgroup per bucket (in XCD-chunked order); a bucket is a run of chunks
// (one large piece, or several small tensors). Chunk and pointer-table reads
// are uniform per workgroup. chunk(s, ch, c) processes chunk c.
template <int CACHED = -1, typename ChunkFn>
__device__ __forceinline__ void for_plan_chunks(const PlanArgs& a, const ChunkFn& chunk) {
    const uint32_t b = logical_block(blockIdx.x, a.xcd_chunk);
    if (b >= static_cast<uint32_t>(a.n_buckets)) return;   // padding of the chunked grid
    const Hyper h = resolve_hyper(a.h, a.lr_ptr);
    const int32_t c_end = read_table(&a.bucket_begin[b + 1]);
    for (int32_t c = read_table(&a.bucket_begin[b]); c < c_end; ++c) {
        const PlanChunk* cp = &a.chunks[c];
        const PlanChunk ch{read_table(&cp->tensor), 0, read_table(&cp->start), read_table(&cp->len)};
        const PlanSrcT<CACHED> s{a.ptrs + static_cast<int64_t>(ch.tensor) * a.stride, a, h};
        chunk(s, ch, c);
    }
}

// Compile-time (W, G): tiles of U units kBlock apart, then the units of a
// partial last tile, then the ragged end (thread 0).
template <typename GT, int W, int G, int U, int CACHED>
__device__ __forceinline__ void step_plan_body(const PlanArgs& a) {
    constexpr int VEC = Unit<GT>::VEC;
    for_plan_chunks<CACHED>(a, [&](const auto& s, const PlanChunk& ch, int32_t) {
        const int64_t full = ch.len / VEC;
        for (int64_t t0 = threadIdx.x; t0 < full; t0 += static_cast<int64_t>(kBlock) * U) {
            if (t0 + static_cast<int64_t>(U - 1) * kBlock < full) {
                int64_t e0[U];
#pragma unroll
                for (int q = 0; q < U; ++q) e0[q] = ch.start + (t0 + static_cast<int64_t>(q) * kBlock) * VEC;
                fused_tile_ct<GT, W, G, U, false>(s, e0, VEC);
            } else {
                for (int64_t u = t0; u < full; u += kBlock)
                    fused_unit_ct<GT, W, G, false>(s, ch.start + u * VEC, VEC);
            }
        }
        const int rem = static_cast<int>(ch.len - full * VEC);
        if (rem != 0 && threadIdx.x == 0) fused_unit_ct<GT, W, G, true>(s, ch.start + full * VEC, rem);
    });
}

template <typename GT, int W, int G, int U, int CACHED>
__global__ __launch_bounds__(kBlock) void step_plan_kernel(PlanArgs a) {
    step_plan_body<GT, W, G, U, CACHED>(a);
}

// The same kernel with at most CAP waves per SIMD (see step_flat_ct_cap).
template <typename GT, int W, int G, int U, int CACHED, int CAP>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(1, CAP))) void step_plan_kernel_cap(PlanArgs a) {
    step_plan_body<GT, W, G, U, CACHED>(a);
}

// Wave caps of the compile-time plan step kernel, measured as for the flat
// one: the 161 ResNet-50 tensors, R = N, every grouping of the flat sweep
// with caps 2 and 3 against the uncapped kernel; a grouping is listed where
// a cap gains at least one point of the 8 TB/s peak.
constexpr WaveCapEntry kPlanWaveCapF32[] = {
    {1, 4, 2}, {2, 2, 2}, {2, 12, 2}, {4, 1, 2}, {5, 1, 2}, {16, 2, 2}, {1, 2, 3}, {1, 3, 3},
    {1, 5, 3}, {1, 6, 3}, {2, 1, 3}, {2, 3, 3}, {3, 1, 3}, {3, 16, 3}, {6, 16, 3}, {8, 6, 3},
    {12, 3, 3}, {12, 4, 3}, {12, 5, 3},
};
constexpr WaveCapEntry kPlanWaveCapBF16[] = {
    {1, 2, 2}, {1, 4, 2}, {1, 8, 2}, {2, 1, 2}, {2, 2, 2}, {2, 3, 2}, {2, 5, 2}, {2, 64, 2},
    {3, 1, 2}, {3, 2, 2}, {3, 3, 2}, {3, 6, 2}, {3, 8, 2}, {3, 12, 2}, {3, 16, 2}, {3, 32, 2},
    {4, 1, 2}, {4, 2, 2}, {4, 32, 2}, {5, 1, 2}, {5, 2, 2}, {5, 6, 2}, {5, 8, 2}, {5, 12, 2},
    {5, 16, 2}, {6, 1, 2}, {6, 8, 2}, {6, 12, 2}, {8, 1, 2}, {8, 16, 2}, {12, 5, 2}, {12, 6, 2},
    {12, 8, 2}, {2, 4, 3}, {2, 8, 3}, {4, 3, 3},
};
// The LARS norms kernel (pass 1), same measurement of the whole LARS step; its
// run-to-run spread reached three points, so an entry gains at least three.
constexpr WaveCapEntry kLarsWaveCapBF16[] = {
    {1, 16, 2}, {2, 8, 2}, {2, 32, 2}, {3, 6, 2}, {3, 8, 2}, {3, 12, 2}, {3, 16, 2}, {3, 32, 2},
    {4, 4, 2}, {4, 16, 2}, {5, 6, 2}, {5, 12, 2}, {8, 2, 2}, {8, 8, 2}, {16, 1, 2}, {16, 8, 2},
    {5, 2, 3}, {5, 4, 3}, {5, 8, 3}, {5, 16, 3}, {6, 2, 3}, {6, 4, 3}, {6, 6, 3}, {12, 1, 3},
    {12, 3, 3}, {12, 4, 3},
};
template <size_t K>
constexpr int wave_cap_in(const WaveCapEntry (&t)[K], int W, int G) {
    for (size_t i = 0; i < K; ++i)
        if (t[i].W == W && t[i].G == G) return t[i].cap;
    return 0;
}

template <typename GT, int W, int G, int U, int CACHED>
constexpr auto plan_step_kernel() {
    constexpr int cap = sizeof(GT) == 2 ? wave_cap_in(kPlanWaveCapBF16, W, G) : wave_cap_in(kPlanWaveCapF32, W, G);
    if constexpr (cap != 0) return step_plan_kernel_cap<GT, W, G, U, CACHED, cap>;
    else return step_plan_kernel<GT, W, G, U, CACHED>;
}

// Runtime group layouts (non-power-of-two or large counts, and the
// paper-literal reduction over any partition): one unit per lane.
template <typename GT, int LV, int CACHED>
__global__ __launch_bounds__(kBlock) void step_plan_seg(PlanArgs a) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int U = SegTileUnits<GT>::U;
    const bool literal = a.literal != 0;
    auto gs = [&](int j) { return static_cast<int>(a.group_start[j]); };
    for_plan_chunks<CACHED>(a, [&](const PlanSrcT<CACHED>& s, const PlanChunk& ch, int32_t) {
        const int64_t full = ch.len / VEC;
        for (int64_t t0 = threadIdx.x; t0 < full; t0 += static_cast<int64_t>(kBlock) * U) {
            if (t0 + static_cast<int64_t>(U - 1) * kBlock < full) {
                int64_t e0[U];
#pragma unroll
                for (int q = 0; q < U; ++q) e0[q] = ch.start + (t0 + static_cast<int64_t>(q) * kBlock) * VEC;
                fused_tile_seg<GT, LV, U, false>(s, a.n_workers, a.n_groups, gs, literal, e0, VEC);
            } else {
                for (int64_t u = t0; u < full; u += kBlock)
                    fused_unit_seg<GT, LV, false>(s, a.n_workers, a.n_groups, gs, literal, ch.start + u * VEC, VEC);
            }
        }
        const int rem = static_cast<int>(ch.len - full * VEC);
        if (rem != 0 && threadIdx.x == 0)
            fused_unit_seg<GT, LV, true>(s, a.n_workers, a.n_groups, gs, literal, ch.start + full * VEC, rem);
    });
}

// Replica-major copy-out pass over a plan's buckets (the layout of
// copy_out_rmajor_kernel with buckets in place of fixed-size blocks): workgroup
// b copies bucket w*win_blocks + s to replica group q (RK consecutive
// replicas), b = (w*ceil(R/RK) + q)*win_blocks + s; a lane loads U units of
// the source, then stores them to each destination of the group. The source
// is table slot copy_src of each tensor (p for the copy-out of the replicas;
// the first member's gradient for the copy pass of the gradient broadcast),
// the R destinations slots copy_dst .. copy_dst + R - 1.
// One piece [start, start+len) of a tensor to the nr replicas in dst.
template <int VEC, int U, int RK>
__device__ __forceinline__ void copy_out_piece(const float* p, void* const (&dst)[RK], int nr, int rdt,
                                               int64_t start, int64_t len) {
    const int64_t full = len / VEC;
    for (int64_t t0 = threadIdx.x; t0 < full; t0 += static_cast<int64_t>(kBlock) * U) {
        float x[U][VEC];
#pragma unroll
        for (int i = 0; i < U; ++i) {
            const int64_t u = t0 + static_cast<int64_t>(i) * kBlock;
            if (u < full) load_f32_cached<VEC, false>(p, start + u * VEC, VEC, x[i]);
        }
#pragma unroll
        for (int k = 0; k < RK; ++k) {
            if (k >= nr) break;
#pragma unroll
            for (int i = 0; i < U; ++i) {
                const int64_t u = t0 + static_cast<int64_t>(i) * kBlock;
                if (u < full) store_replica<VEC, false>(dst[k], rdt, start + u * VEC, VEC, x[i]);
            }
        }
    }
    const int rem = static_cast<int>(len - full * VEC);
    if (rem != 0 && threadIdx.x == 0) {
        float x[VEC];
        load_f32_cached<VEC, true>(p, start + full * VEC, rem, x);
        for (int k = 0; k < nr; ++k) store_replica<VEC, true>(dst[k], rdt, start + full * VEC, rem, x);
    }
}

template <int VEC, int U, int RK>
__device__ __forceinline__ void copy_out_plan_block(const PlanArgs& a, int64_t b) {
    const int n_rg = (a.n_replicas + RK - 1) / RK;
    const int64_t per_win = static_cast<int64_t>(a.win_blocks) * n_rg;
    const int64_t w = b / per_win;
    const int64_t rb = b - w * per_win;
    const int q = static_cast<int>(rb / a.win_blocks);
    const int64_t bucket = w * a.win_blocks + (rb - static_cast<int64_t>(q) * a.win_blocks);
    if (bucket >= a.n_buckets) return;   // padding of the last window
    const int r0 = q * RK;
    const int nr = min(RK, a.n_replicas - r0);
    const CopyDesc* d = &a.copy_desc[bucket];
    if (read_table(&d->n_chunks) == 1) {   // one piece: its params address comes with it
        void* const* t = a.ptrs + static_cast<int64_t>(read_table(&d->tensor)) * a.stride;
        void* dst[RK];
#pragma unroll
        for (int k = 0; k < RK; ++k) dst[k] = k < nr ? read_table(&t[a.copy_dst + r0 + k]) : nullptr;
        const float* p = a.copy_src == 0 ? read_table(&d->p) : static_cast<const float*>(read_table(&t[a.copy_src]));
        const int64_t start = read_table(&d->start), len = read_table(&d->len);
        const int64_t full = len / VEC;
        const int rem = static_cast<int>(len - full * VEC);
        if (full + (rem != 0 ? 1 : 0) <= static_cast<int64_t>(kBlock) * U) {
            // the piece is one lane tile: loads, then stores, as in the flat
            // pass (measured 4% faster than the loop of copy_out_piece)
            float x[U][VEC];
#pragma unroll
            for (int t = 0; t < U; ++t) {
                const int64_t u = threadIdx.x + static_cast<int64_t>(t) * kBlock;
                if (u < full) load_f32_cached<VEC, false>(p, start + u * VEC, VEC, x[t]);
                else if (u == full && rem != 0) load_f32_cached<VEC, true>(p, start + u * VEC, rem, x[t]);
            }
#pragma unroll
            for (int k = 0; k < RK; ++k) {
                if (k >= nr) break;
#pragma unroll
                for (int t = 0; t < U; ++t) {
                    const int64_t u = threadIdx.x + static_cast<int64_t>(t) * kBlock;
                    if (u < full) store_replica<VEC, false>(dst[k], a.rdt, start + u * VEC, VEC, x[t]);
                    else if (u == full && rem != 0) store_replica<VEC, true>(dst[k], a.rdt, start + u * VEC, rem, x[t]);
                }
            }
            return;
        }
        copy_out_piece<VEC, U, RK>(p, dst, nr, a.rdt, start, len);
        return;
    }
    const int32_t c_end = read_table(&a.bucket_begin[bucket + 1]);
    for (int32_t c = read_table(&a.bucket_begin[bucket]); c < c_end; ++c) {
        const PlanChunk* cp = &a.chunks[c];
        void* const* t = a.ptrs + static_cast<int64_t>(read_table(&cp->tensor)) * a.stride;
        void* dst[RK];
#pragma unroll
        for (int k = 0; k < RK; ++k) dst[k] = k < nr ? read_table(&t[a.copy_dst + r0 + k]) : nullptr;
        copy_out_piece<VEC, U, RK>(static_cast<const float*>(read_table(&t[a.copy_src])), dst, nr, a.rdt,
                                   read_table(&cp->start), read_table(&cp->len));
    }
}

template <int VEC, int U, int RK>
__global__ __launch_bounds__(kBlock) void copy_out_plan_rmajor(PlanArgs a) {
    for (int64_t b = blockIdx.x; b < a.copy_blocks; b += gridDim.x) copy_out_plan_block<VEC, U, RK>(a, b);
}

}  // namespace lsgd

namespace lsgd {

// ------------------------------------------------------------- LARS on a plan
//
// Layer-wise trust ratios (LARS, which the paper names in Sec. 2 and Sec. 6;
// definition of You, Gitman and Ginsburg, eq. 6 and Alg. 1) need each tensor's
// ||p|| and ||gbar|| before any of its elements is updated, so a step takes
// three launches over the plan:
//   1. lars_norms_*: the mean gradient of every element (the same pairwise
//      aggregation as the fused step), stored to a scratch slice per tensor,
//      and per-chunk binary64 sums of p^2 and gbar^2 (one workgroup-level
//      reduction per chunk, fixed order);
//   2. lars_trust_kernel: one workgroup per tensor sums its chunks' partials
//      (fixed order) and forms trust = eta*||p|| / (||gbar|| + wd*||p||) in
//      binary64, rounded once to binary32; 1 when a norm is zero or the
//      tensor is excluded from the layer-wise rates;
//   3. lars_update_kernel: d = trust*(gbar + wd*p), the heavy-ball update and
//      the copy-out, reading gbar back from the scratch.

struct LarsArgs {
    PlanArgs pa;                   // the plan's tables and counts
    const int64_t* gbar_off;       // [n_tensors]: tensor t's slice of `gbar` starts here (floats)
    const int32_t* tensor_chunks;  // [n_tensors + 1]: tensor t owns chunks [tc[t], tc[t+1])
    float* gbar;                   // scratch: aggregated gradient, one slice per tensor
    double* partials;              // [n_chunks][2]: sums of p^2 and gbar^2 over a chunk
    float* trust;                  // [n_tensors]
    float* trust_out;              // optional copy of the trust ratios
    const uint8_t* exclude;        // [n_tensors]: nonzero = the tensor takes trust 1
    int32_t n_tensors;
    float trust_coef;
};

// Workgroup sums of two doubles per lane, valid in thread 0. Within a wave an
// xor butterfly: partners add the same two values, and addition is
// commutative, so every lane holds the same bits after each round; then the
// four wave sums in a fixed order. Every thread of the block calls it.
__device__ __forceinline__ void block_sum2(double& a, double& b, double (*lds)[2]) {
    static_assert(kBlock == 256, "four waves per workgroup");
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        a += __shfl_xor(a, off, 64);
        b += __shfl_xor(b, off, 64);
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        lds[wave][0] = a;
        lds[wave][1] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        a = (lds[0][0] + lds[1][0]) + (lds[2][0] + lds[3][0]);
        b = (lds[0][1] + lds[1][1]) + (lds[2][1] + lds[3][1]);
    }
    __syncthreads();
}

// Mean gradient of a tile stored to the scratch slice, squares accumulated.
template <int T>
__device__ __forceinline__ void lars_accumulate(const float (&p)[T], const float (&g)[T], int cnt_total,
                                                double& sp, double& sg) {
#pragma unroll
    for (int v = 0; v < T; ++v) {
        if (v < cnt_total) {
            sp += static_cast<double>(p[v]) * static_cast<double>(p[v]);
            sg += static_cast<double>(g[v]) * static_cast<double>(g[v]);
        }
    }
}

template <typename GT, int U, bool TAIL>
__device__ __forceinline__ void lars_tile_out(const PlanSrc& s, float* gb, const int64_t (&e)[U], int cnt,
                                              const float (&gbar)[U * Unit<GT>::VEC], double& sp, double& sg) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    float p[T];
#pragma unroll
    for (int q = 0; q < U; ++q) {
        store_f32_cached<VEC, TAIL>(gb, e[q], cnt, slice<VEC, T>(gbar, q));
        load_f32_cached<VEC, TAIL>(s.p(), e[q], cnt, slice<VEC, T>(p, q));
    }
    // zero-filled tail elements add nothing, but skip them anyway
    lars_accumulate<T>(p, gbar, TAIL ? cnt : T, sp, sg);
}

// Pass 1, compile-time (W, G).
template <typename GT, int W, int G, int U>
__device__ __forceinline__ void lars_norms_body(const LarsArgs& la, double (&lds)[kBlock / 64][2]) {
    constexpr int VEC = Unit<GT>::VEC;
    for_plan_chunks(la.pa, [&](const PlanSrc& s, const PlanChunk& ch, int32_t c) {
        float* gb = la.gbar + read_table(&la.gbar_off[ch.tensor]);
        double sp = 0.0, sg = 0.0;
        const int64_t full = ch.len / VEC;
        for (int64_t t0 = threadIdx.x; t0 < full; t0 += static_cast<int64_t>(kBlock) * U) {
            if (t0 + static_cast<int64_t>(U - 1) * kBlock < full) {
                int64_t e0[U];
#pragma unroll
                for (int q = 0; q < U; ++q) e0[q] = ch.start + (t0 + static_cast<int64_t>(q) * kBlock) * VEC;
                float gbar[U * VEC];
                mean_tile_ct<GT, W, G, U, false>(s, e0, VEC, gbar);
                lars_tile_out<GT, U, false>(s, gb, e0, VEC, gbar, sp, sg);
            } else {
                for (int64_t u = t0; u < full; u += kBlock) {
                    const int64_t e[1] = {ch.start + u * VEC};
                    float gbar[VEC];
                    mean_tile_ct<GT, W, G, 1, false>(s, e, VEC, gbar);
                    lars_tile_out<GT, 1, false>(s, gb, e, VEC, gbar, sp, sg);
                }
            }
        }
        const int rem = static_cast<int>(ch.len - full * VEC);
        if (rem != 0 && threadIdx.x == 0) {
            const int64_t e[1] = {ch.start + full * VEC};
            float gbar[VEC];
            mean_tile_ct<GT, W, G, 1, true>(s, e, rem, gbar);
            lars_tile_out<GT, 1, true>(s, gb, e, rem, gbar, sp, sg);
        }
        block_sum2(sp, sg, lds);
        if (threadIdx.x == 0) {
            la.partials[2 * static_cast<int64_t>(c)] = sp;
            la.partials[2 * static_cast<int64_t>(c) + 1] = sg;
        }
    });
}

template <typename GT, int W, int G, int U>
__global__ __launch_bounds__(kBlock) void lars_norms_kernel(LarsArgs la) {
    __shared__ double lds[kBlock / 64][2];
    lars_norms_body<GT, W, G, U>(la, lds);
}

template <typename GT, int W, int G, int U, int CAP>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(1, CAP))) void lars_norms_kernel_cap(LarsArgs la) {
    __shared__ double lds[kBlock / 64][2];
    lars_norms_body<GT, W, G, U>(la, lds);
}

// The LARS norms kernel for (W, G), capped where kLarsWaveCapBF16 lists it.
template <typename GT, int W, int G>
constexpr auto lars_kernel_for() {
    constexpr int U = tile_units<GT>(W * G, G);
    constexpr int cap = sizeof(GT) == 2 ? wave_cap_in(kLarsWaveCapBF16, W, G) : 0;
    if constexpr (cap != 0) return lars_norms_kernel_cap<GT, W, G, U, cap>;
    else return lars_norms_kernel<GT, W, G, U>;
}

// Pass 1, runtime W and G (equal groups): one unit per lane.
template <typename GT, int LV>
__global__ __launch_bounds__(kBlock) void lars_norms_seg(LarsArgs la) {
    constexpr int VEC = Unit<GT>::VEC;
    __shared__ double lds[kBlock / 64][2];
    const int W = la.pa.W;
    auto gs = [&](int j) { return j * W; };
    for_plan_chunks(la.pa, [&](const PlanSrc& s, const PlanChunk& ch, int32_t c) {
        float* gb = la.gbar + read_table(&la.gbar_off[ch.tensor]);
        double sp = 0.0, sg = 0.0;
        const int64_t full = ch.len / VEC;
        for (int64_t u = threadIdx.x; u < full; u += kBlock) {
            const int64_t e[1] = {ch.start + u * VEC};
            float gbar[VEC];
            mean_unit_seg<GT, LV, false>(s, la.pa.n_workers, la.pa.n_groups, gs, false, e[0], VEC, gbar);
            lars_tile_out<GT, 1, false>(s, gb, e, VEC, gbar, sp, sg);
        }
        const int rem = static_cast<int>(ch.len - full * VEC);
        if (rem != 0 && threadIdx.x == 0) {
            const int64_t e[1] = {ch.start + full * VEC};
            float gbar[VEC];
            mean_unit_seg<GT, LV, true>(s, la.pa.n_workers, la.pa.n_groups, gs, false, e[0], rem, gbar);
            lars_tile_out<GT, 1, true>(s, gb, e, rem, gbar, sp, sg);
        }
        block_sum2(sp, sg, lds);
        if (threadIdx.x == 0) {
            la.partials[2 * static_cast<int64_t>(c)] = sp;
            la.partials[2 * static_cast<int64_t>(c) + 1] = sg;
        }
    });
}

// Pass 2: one workgroup per tensor.
static __global__ __launch_bounds__(kBlock) void lars_trust_kernel(LarsArgs la) {
    __shared__ double lds[kBlock / 64][2];
    const int32_t t = static_cast<int32_t>(blockIdx.x);
    if (t >= la.n_tensors) return;
    const int32_t c0 = la.tensor_chunks[t], c1 = la.tensor_chunks[t + 1];
    double sp = 0.0, sg = 0.0;
    for (int32_t c = c0 + static_cast<int32_t>(threadIdx.x); c < c1; c += kBlock) {
        sp += la.partials[2 * static_cast<int64_t>(c)];
        sg += la.partials[2 * static_cast<int64_t>(c) + 1];
    }
    block_sum2(sp, sg, lds);
    if (threadIdx.x == 0) {
        const double wn = sqrt(sp), gn = sqrt(sg);
        const double wd = static_cast<double>(la.pa.h.wd);
        const float tr = (wn == 0.0 || gn == 0.0 || la.exclude[t] != 0)
                             ? 1.0f
                             : static_cast<float>((static_cast<double>(la.trust_coef) * wn) / (gn + wd * wn));
        la.trust[t] = tr;
        if (la.trust_out) la.trust_out[t] = tr;
    }
}

// Pass 3: trust-scaled update of U binary32 units per lane.
template <int VEC>
__device__ __forceinline__ void lars_update(const Hyper& h, float trust, const float (&gbar)[VEC],
                                            float (&p)[VEC], float (&m)[VEC]) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        const float decayed = gbar[v] + h.wd * p[v];
        const float d = trust * decayed;
        m[v] = h.mu * m[v] + d;
        p[v] = p[v] - h.lr * m[v];
    }
}

template <int U, bool TAIL>
__device__ __forceinline__ void lars_update_tile(const PlanSrc& s, const float* gb, float trust,
                                                 const int64_t (&e0)[U], int cnt) {
    constexpr int T = U * 4;
    float g[T], p[T], m[T];
#pragma unroll
    for (int q = 0; q < U; ++q) load_f32_cached<4, TAIL>(gb, e0[q], cnt, slice<4, T>(g, q));
#pragma unroll
    for (int q = 0; q < U; ++q) load_f32_cached<4, TAIL>(s.p(), e0[q], cnt, slice<4, T>(p, q));
#pragma unroll
    for (int q = 0; q < U; ++q) load_f32<4, TAIL>(s.m(), e0[q], cnt, slice<4, T>(m, q));
    lars_update<T>(s.hyper(), trust, g, p, m);
    store_state<4, U, TAIL>(s, e0, cnt, p, m);
}

template <int U>
__global__ __launch_bounds__(kBlock) void lars_update_kernel(LarsArgs la) {
    for_plan_chunks(la.pa, [&](const PlanSrc& s, const PlanChunk& ch, int32_t) {
        const float* gb = la.gbar + read_table(&la.gbar_off[ch.tensor]);
        const float trust = read_table(&la.trust[ch.tensor]);
        const int64_t full = ch.len / 4;
        for (int64_t t0 = threadIdx.x; t0 < full; t0 += static_cast<int64_t>(kBlock) * U) {
            if (t0 + static_cast<int64_t>(U - 1) * kBlock < full) {
                int64_t e0[U];
#pragma unroll
                for (int q = 0; q < U; ++q) e0[q] = ch.start + (t0 + static_cast<int64_t>(q) * kBlock) * 4;
                lars_update_tile<U, false>(s, gb, trust, e0, 4);
            } else {
                for (int64_t u = t0; u < full; u += kBlock) {
                    const int64_t e[1] = {ch.start + u * 4};
                    lars_update_tile<1, false>(s, gb, trust, e, 4);
                }
            }
        }
        const int rem = static_cast<int>(ch.len - full * 4);
        if (rem != 0 && threadIdx.x == 0) {
            const int64_t e[1] = {ch.start + full * 4};
            lars_update_tile<1, true>(s, gb, trust, e, rem);
        }
    });
}

}  // namespace lsgd
