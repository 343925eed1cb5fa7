// Device code of liblsgd: the Layered SGD aggregation and update for gfx950.
//
// Every step is elementwise along the parameter vector, so the kernels stream
// HBM: each lane owns one 16-byte "unit" of the gradient layout (4 binary32 or
// 8 bfloat16 elements), loads all N worker units of it with 128-bit nontemporal
// loads, reduces them in registers in the fixed pairwise order, applies the
// update and writes parameters, momentum and replicas with 128-bit stores.
// No element is touched by two lanes, so there are no atomics, no LDS and no
// cross-lane reductions: a lane's result depends only on its own inputs.
//
// Rounding contract (matches the header): binary32, one rounding per written
// operation, no contraction into fused multiply-add.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#pragma clang fp contract(off)

namespace lsgd {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kMaxWorkers = 128;   // == LSGD_MAX_WORKERS
constexpr int kMaxReplicas = 128;  // == LSGD_MAX_REPLICAS
constexpr int kBlock = 256;        // threads per workgroup (4 wave64)
// A dispatch holds at most 2^32 - 1 work-items; grids stay at or below this
// many workgroups (a multiple of 8, the XCD count).
constexpr int64_t kMaxGridBlocks = (0xffffffffLL / kBlock) / 8 * 8;

enum : int { kF32 = 0, kBF16 = 1 };

// Elements per 16-byte gradient unit. bf16 is carried as its uint16 bits.
template <typename GT> struct Unit;
template <> struct Unit<float> { static constexpr int VEC = 4; };
template <> struct Unit<uint16_t> { static constexpr int VEC = 8; };

// Largest power of two strictly below k (k >= 2): the split point of the
// pairwise sum PW(x[0..k)) = PW(x[0..h)) + PW(x[h..k)).
__host__ __device__ constexpr int pw_split(int k) {
    int h = 1;
    while (h * 2 < k) h *= 2;
    return h;
}

// Workgroups are dispatched to the eight XCDs round-robin by block index (block
// b runs on XCD b % 8). With xcd_chunk = C > 0 the kernels renumber blocks so
// that each XCD runs C consecutive logical blocks per turn: the chip-wide set of
// active addresses stays one contiguous window per buffer, while each XCD walks
// C * 4 KB runs of every buffer, which keeps fewer distinct pages live in that
// XCD's address-translation caches. The host pads the grid to a multiple of
// 8*C so that the renumbering is a bijection on [0, gridDim.x).
__device__ __forceinline__ uint32_t logical_block(uint32_t b, uint32_t chunk) {
    if (chunk == 0) return b;
    const uint32_t x = b & 7u, i = b >> 3;
    return ((i / chunk) * 8u + x) * chunk + (i % chunk);
}

// Runs body(u) for every unit u in [0, units). A logical block owns `upl`
// consecutive passes of kBlock units (one unit per lane per pass), so each
// workgroup walks upl * 4 KB of every buffer in address order; logical blocks
// are taken in XCD-chunked order, grid-stride when the grid is smaller than
// the work.
template <typename Body>
__device__ __forceinline__ void for_units(int64_t units, uint32_t chunk, uint32_t upl,
                                          const Body& body) {
    const int64_t span = static_cast<int64_t>(kBlock) * upl;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * span;
    for (int64_t base = static_cast<int64_t>(logical_block(blockIdx.x, chunk)) * span; base < units;
         base += stride) {
        for (uint32_t q = 0; q < upl; ++q) {
            const int64_t u = base + static_cast<int64_t>(q) * kBlock + threadIdx.x;
            if (u < units) body(u);
        }
    }
}

// Tiled variant of for_units: a lane's tile is U units kBlock apart (so every
// wave instruction still covers 1 KB of one buffer), and a kernel visits each
// buffer once per tile for all U units (stream-major), which keeps consecutive
// instructions of a wave on the same pages and DRAM rows. tile(e0) gets the U
// element offsets of a tile whose units are all complete; unit(u) handles the
// units of the last, partial tile one by one (u < units_all).
template <int U, int VEC, typename TileFn, typename UnitFn>
__device__ __forceinline__ void for_tiles(int64_t units_full, int64_t units_all, uint32_t chunk,
                                          uint32_t upl, const TileFn& tile, const UnitFn& unit) {
    const int64_t tspan = static_cast<int64_t>(kBlock) * U;
    const int64_t span = tspan * upl;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * span;
    for (int64_t base = static_cast<int64_t>(logical_block(blockIdx.x, chunk)) * span; base < units_all;
         base += stride) {
        for (uint32_t pass = 0; pass < upl; ++pass) {
            const int64_t t0 = base + static_cast<int64_t>(pass) * tspan + threadIdx.x;
            if (t0 + static_cast<int64_t>(U - 1) * kBlock < units_full) {
                int64_t e0[U];
#pragma unroll
                for (int q = 0; q < U; ++q) e0[q] = (t0 + static_cast<int64_t>(q) * kBlock) * VEC;
                tile(e0);
            } else {
#pragma unroll
                for (int q = 0; q < U; ++q) {
                    const int64_t u = t0 + static_cast<int64_t>(q) * kBlock;
                    if (u < units_all) unit(u);
                }
            }
        }
    }
}

// The q-th VEC-float slice of a tile array.
template <int VEC, int T>
__device__ __forceinline__ float (&slice(float (&x)[T], int q))[VEC] {
    return *reinterpret_cast<float(*)[VEC]>(&x[q * VEC]);
}
template <int VEC, int T>
__device__ __forceinline__ const float (&slice(const float (&x)[T], int q))[VEC] {
    return *reinterpret_cast<const float(*)[VEC]>(&x[q * VEC]);
}

// ---------------------------------------------------------------- loads/stores

// Address-space views. Every buffer the kernels read or write is device
// global memory: accessing it through a global-space pointer gives the
// global_load / global_store forms, also for pointers the kernel itself read
// from a table (for those the compiler would otherwise use the generic flat
// forms). Tables that no kernel writes (the plans' chunk and pointer tables)
// are read through the constant space, so that they become scalar loads
// instead of vector loads the compiler must order after every store.
#define LSGD_GLOBAL __attribute__((address_space(1)))
#define LSGD_CONST __attribute__((address_space(4)))

template <typename T>
__device__ __forceinline__ const LSGD_GLOBAL T* gload_ptr(const void* p) {
    return (const LSGD_GLOBAL T*)(p);
}
template <typename T>
__device__ __forceinline__ LSGD_GLOBAL T* gstore_ptr(void* p) {
    return (LSGD_GLOBAL T*)(p);
}
template <typename T>
__device__ __forceinline__ T read_table(const T* p) {
    return *(const LSGD_CONST T*)(p);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// binary32 -> bfloat16 bits, nearest-even via the carry of a 0x7fff(+1 if odd)
// bias; NaN is returned as a quiet NaN of the same sign.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// One gradient unit of a worker, widened to binary32. TAIL units (the ragged end
// of a tensor, cnt < VEC) read element by element and zero-fill the rest.
template <typename GT, bool TAIL>
__device__ __forceinline__ void load_grad(const void* g, int64_t e0, int cnt,
                                          float (&x)[Unit<GT>::VEC]) {
    constexpr int VEC = Unit<GT>::VEC;
    const GT* p = static_cast<const GT*>(g) + e0;
    if constexpr (TAIL) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            if constexpr (sizeof(GT) == 4) x[v] = v < cnt ? gload_ptr<float>(p)[v] : 0.f;
            else x[v] = v < cnt ? bf16_bits_to_f32(gload_ptr<uint16_t>(p)[v]) : 0.f;
        }
    } else if constexpr (sizeof(GT) == 4) {
        f32x4 t = __builtin_nontemporal_load(gload_ptr<f32x4>(p));
        x[0] = t.x; x[1] = t.y; x[2] = t.z; x[3] = t.w;
    } else {
        u32x4 t = __builtin_nontemporal_load(gload_ptr<u32x4>(p));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            x[2 * q] = __uint_as_float(t[q] << 16);
            x[2 * q + 1] = __uint_as_float(t[q] & 0xffff0000u);
        }
    }
}

// VEC binary32 values at p + e0 (VEC is 4 or 8: one or two 128-bit accesses).
template <int VEC, bool TAIL>
__device__ __forceinline__ void load_f32(const float* p, int64_t e0, int cnt, float (&x)[VEC]) {
    if constexpr (TAIL) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) x[v] = v < cnt ? gload_ptr<float>(p + e0)[v] : 0.f;
    } else {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            f32x4 t = __builtin_nontemporal_load(gload_ptr<f32x4>(p + e0) + q);
            x[4 * q] = t.x; x[4 * q + 1] = t.y; x[4 * q + 2] = t.z; x[4 * q + 3] = t.w;
        }
    }
}

template <int VEC, bool TAIL>
__device__ __forceinline__ void store_f32(float* p, int64_t e0, int cnt, const float (&x)[VEC]) {
    if constexpr (TAIL) {
#pragma unroll
        for (int v = 0; v < VEC; ++v)
            if (v < cnt) gstore_ptr<float>(p + e0)[v] = x[v];
    } else {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            f32x4 t = {x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]};
            __builtin_nontemporal_store(t, gstore_ptr<f32x4>(p + e0) + q);
        }
    }
}

// Plain (cache-allocating) variants, for data that is read again soon: the
// LARS mean-gradient scratch (written by one kernel, read by the next).
template <int VEC, bool TAIL>
__device__ __forceinline__ void load_f32_cached(const float* p, int64_t e0, int cnt, float (&x)[VEC]) {
    if constexpr (TAIL) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) x[v] = v < cnt ? gload_ptr<float>(p + e0)[v] : 0.f;
    } else {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q) {
            const f32x4 t = *(gload_ptr<f32x4>(p + e0) + q);
            x[4 * q] = t.x; x[4 * q + 1] = t.y; x[4 * q + 2] = t.z; x[4 * q + 3] = t.w;
        }
    }
}

template <int VEC, bool TAIL>
__device__ __forceinline__ void store_f32_cached(float* p, int64_t e0, int cnt, const float (&x)[VEC]) {
    if constexpr (TAIL) {
#pragma unroll
        for (int v = 0; v < VEC; ++v)
            if (v < cnt) gstore_ptr<float>(p + e0)[v] = x[v];
    } else {
#pragma unroll
        for (int q = 0; q < VEC / 4; ++q)
            *(gstore_ptr<f32x4>(p + e0) + q) = f32x4{x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]};
    }
}

// A replica unit: binary32 copy, or nearest-even bfloat16 (VEC*2 bytes: 8 or 16).
template <int VEC, bool TAIL>
__device__ __forceinline__ void store_replica(void* r, int rdt, int64_t e0, int cnt,
                                              const float (&x)[VEC]) {
    if (rdt == kF32) {
        store_f32<VEC, TAIL>(static_cast<float*>(r), e0, cnt, x);
        return;
    }
    uint16_t* h = static_cast<uint16_t*>(r) + e0;
    if constexpr (TAIL) {
#pragma unroll
        for (int v = 0; v < VEC; ++v)
            if (v < cnt) gstore_ptr<uint16_t>(h)[v] = static_cast<uint16_t>(f32_to_bf16_bits(x[v]));
    } else if constexpr (VEC == 4) {
        u32x2 t = {f32_to_bf16_bits(x[0]) | (f32_to_bf16_bits(x[1]) << 16),
                   f32_to_bf16_bits(x[2]) | (f32_to_bf16_bits(x[3]) << 16)};
        __builtin_nontemporal_store(t, gstore_ptr<u32x2>(h));
    } else {
        u32x4 t;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            t[q] = f32_to_bf16_bits(x[2 * q]) | (f32_to_bf16_bits(x[2 * q + 1]) << 16);
        __builtin_nontemporal_store(t, gstore_ptr<u32x4>(h));
    }
}

// One 16-byte gradient unit as raw bits (4 binary32 or 8 bfloat16 values), so
// that a batch of loads in flight costs four registers each whatever the
// dtype. TAIL units read cnt elements and leave the rest zero.
template <typename GT, bool TAIL>
__device__ __forceinline__ u32x4 load_raw(const void* g, int64_t e0, int cnt) {
    const GT* p = static_cast<const GT*>(g) + e0;
    if constexpr (!TAIL) {
        return __builtin_nontemporal_load(gload_ptr<u32x4>(p));
    } else {
        constexpr int VEC = Unit<GT>::VEC;
        uint32_t h[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            if constexpr (sizeof(GT) == 4) h[v] = v < cnt ? gload_ptr<uint32_t>(p)[v] : 0u;
            else h[v] = v < cnt ? static_cast<uint32_t>(gload_ptr<uint16_t>(p)[v]) : 0u;
        }
        if constexpr (sizeof(GT) == 4) return u32x4{h[0], h[1], h[2], h[3]};
        else return u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
    }
}

// Raw unit bits -> binary32 values (bfloat16 widening is exact).
template <typename GT>
__device__ __forceinline__ void widen(const u32x4& r, float (&x)[Unit<GT>::VEC]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if constexpr (sizeof(GT) == 4) {
            x[q] = __uint_as_float(r[q]);
        } else {
            x[2 * q] = __uint_as_float(r[q] << 16);
            x[2 * q + 1] = __uint_as_float(r[q] & 0xffff0000u);
        }
    }
}

// ------------------------------------------------------------- pairwise sums

// Compile-time pairwise tree over leaves LO .. LO+CNT-1: leaf(k, x) produces the
// k-th term; the tree is PW with the largest-power-of-two split.
template <int LO, int CNT, int VEC, typename Leaf>
__device__ __forceinline__ void pw_tree(const Leaf& leaf, float (&out)[VEC]) {
    if constexpr (CNT == 1) {
        leaf(LO, out);
    } else {
        constexpr int H = pw_split(CNT);
        float a[VEC], b[VEC];
        pw_tree<LO, H, VEC>(leaf, a);
        pw_tree<LO + H, CNT - H, VEC>(leaf, b);
#pragma unroll
        for (int v = 0; v < VEC; ++v) out[v] = a[v] + b[v];
    }
}

// Runtime-count pairwise accumulator (a binary counter of partial sums). After
// k pushes, slot[l] holds the sum of an aligned block of 2^l terms for every set
// bit l of k; the largest block holds the earliest terms. result() folds the
// blocks from the smallest up, each time adding the earlier (larger) block on
// the left: exactly PW(x[0..k)) with the largest-power-of-two split.
// Every slot is updated by a select, never by a conditional store, so that the
// compiler cannot merge the per-level stores into one variable-index store
// (which would move the slots to scratch memory). `levels` (uniform, <= LEVELS)
// bounds the levels a push visits: pushes beyond 2^levels - 1 terms are not
// supported.
template <int VEC, int LEVELS>
struct PwAcc {
    float slot[LEVELS][VEC];
    uint32_t count = 0;

    __device__ __forceinline__ void push(float (&x)[VEC], int levels = LEVELS) {
        bool carrying = true;
#pragma unroll
        for (int l = 0; l < LEVELS; ++l) {
            if (l < levels) {
                const bool full = (count >> l) & 1u;
                const bool merge = carrying && full;
                const bool park = carrying && !full;
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const float merged = slot[l][v] + x[v];
                    slot[l][v] = park ? x[v] : slot[l][v];
                    x[v] = merge ? merged : x[v];
                }
                carrying = merge;
            }
        }
        ++count;
    }

    __device__ __forceinline__ void result(float (&out)[VEC], int levels = LEVELS) const {
        bool have = false;
#pragma unroll
        for (int l = 0; l < LEVELS; ++l) {
            if (l < levels && ((count >> l) & 1u)) {
#pragma unroll
                for (int v = 0; v < VEC; ++v) out[v] = have ? slot[l][v] + out[v] : slot[l][v];
                have = true;
            }
        }
    }
};

__host__ __device__ constexpr int ilog2(int x) { return x <= 1 ? 0 : 1 + ilog2(x / 2); }

// Largest divisor of k that is <= b (k, b >= 1); for a power of two k, the
// largest power of two <= b.
__host__ __device__ constexpr int largest_divisor_le(int k, int b) {
    return b <= 1 ? 1 : (k % b == 0 ? b : largest_divisor_le(k, b - 1));
}

// Levels a PwAcc needs for `cnt` pushes (uniform runtime value).
__device__ __forceinline__ int acc_levels(int cnt) { return 32 - __builtin_clz(static_cast<unsigned>(cnt)); }

// Member gradient loads a lane holds in one register batch of the segmented
// sum: 8 for binary32 gradients, 4 for bfloat16. Halving the bfloat16 batch
// cut its kernels from 186-256 VGPRs to 154-234 (3 waves per SIMD instead of
// 2 for counts up to 7) and their code by half; measured on the ResNet-50
// size, same process: 2x3 +9% (R = N) / +14% (R = 0), 6x4 +6% / +10%, 3x32
// +19% / +85%, 12x1 and 5x16 within 1%. The instruction cache was not the
// limit (0.01% misses with either batch, as for the compile-time kernels).
// For binary32 the same change was mixed (12x1 +8%, 2x3 +1%, 12x8 -1% / -2%,
// 3x32 -2%), so it keeps 8.
template <typename GT>
constexpr int seg_batch() { return sizeof(GT) == 2 ? 4 : 8; }

// Pairwise sums of consecutive runs of the N member-ordered gradients of one
// lane tile (U units, stream-major), for group layouts known only at run time:
// group j holds members [gs(j), gs(j+1)), j < G, and done(j, sum) receives PW
// over them for every element of the tile. Loads run ahead of the additions
// in two alternating register batches of seg_batch loads (seg_batch / U
// members) that ignore group boundaries, so a lane keeps between one and two
// batches of 128-bit loads in flight whatever the group sizes. Each group is
// folded through a binary-counter accumulator (LV levels: sizes below 2^LV).
// N, G and gs are uniform, so every branch here is uniform.
template <typename GT, int LV, int U, bool TAIL, typename Ptr, typename Start, typename Done>
__device__ __forceinline__ void pw_segments(int N, int G, const Ptr& ptr, const Start& gs, const int64_t (&e0)[U],
                                            int cnt, const Done& done) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    constexpr int B = seg_batch<GT>() / U;
    static_assert(B >= 1 && B * U == seg_batch<GT>(), "the batch holds whole members");
    u32x4 xa[B][U], xb[B][U];
    PwAcc<T, LV> acc;
    int j = 0;
    int gend = gs(1);
    int lv = acc_levels(gend - gs(0));
    auto fetch = [&](int k0, u32x4 (&x)[B][U]) {
#pragma unroll
        for (int q = 0; q < B; ++q) {
            if (k0 + q < N) {
                const void* g = ptr(k0 + q);
#pragma unroll
                for (int u = 0; u < U; ++u) x[q][u] = load_raw<GT, TAIL>(g, e0[u], cnt);
            }
        }
    };
    auto consume = [&](int k0, const u32x4 (&x)[B][U]) {
#pragma unroll
        for (int q = 0; q < B; ++q) {
            if (k0 + q < N) {
                float v[T];
#pragma unroll
                for (int u = 0; u < U; ++u) widen<GT>(x[q][u], slice<VEC, T>(v, u));
                acc.push(v, lv);
                if (k0 + q + 1 == gend) {
                    float sum[T];
                    acc.result(sum, lv);
                    acc.count = 0;
                    done(j, sum);
                    if (++j < G) {
                        const int gbeg = gend;
                        gend = gs(j + 1);
                        lv = acc_levels(gend - gbeg);
                    }
                }
            }
        }
    };
    fetch(0, xa);
#pragma unroll 1
    for (int k0 = 0; k0 < N; k0 += 2 * B) {
        if (k0 + B < N) fetch(k0 + B, xb);
        consume(k0, xa);
        if (k0 + 2 * B < N) fetch(k0 + 2 * B, xa);
        if (k0 + B < N) consume(k0 + B, xb);
    }
}

// Accumulator levels for runtime counts up to `max_count` (host side): the
// segmented kernels are built for 3, 4, 5 and 8 levels (counts up to 7, 15,
// 31 and 255). Every level holds a tile of partial sums in registers, so the
// smallest sufficient form runs more waves per SIMD (binary32 step kernel:
// 200 VGPRs at 5 levels, 168 at 3). Measured on the ResNet-50 size against
// 5 levels for everything up to 31, same process: unequal groups 2, 3, 5, 6
// +6.9% (R = 16), 6x4 +6.9%, 2x3 +5.8%, 4x6 +3.3% with 3 levels; 12x8 +2.1%
// and 4x10 +1.2% with 4; without replicas +3.5% to +20%; one loss, 3x5 with
// its 15 replicas written by the step kernel, -2.5%.
__host__ __device__ constexpr int seg_levels(int max_count) {
    return max_count <= 7 ? 3 : max_count <= 15 ? 4 : max_count <= 31 ? 5 : 8;
}

// ------------------------------------------------------------- the update

struct Hyper {
    float lr, mu, wd;
};

// Alg. 3 update with heavy-ball momentum and L2 weight decay, each operation
// rounded separately: d = gbar + wd*p; m = mu*m + d; p = p - lr*m.
template <int VEC>
__device__ __forceinline__ void sgd_update(const Hyper& h, const float (&gbar)[VEC],
                                           float (&p)[VEC], float (&m)[VEC]) {
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        float d = gbar[v] + h.wd * p[v];
        m[v] = h.mu * m[v] + d;
        p[v] = p[v] - h.lr * m[v];
    }
}

// ------------------------------------------------------------- pointer sources

// Kernel arguments of the planless calls. Pointer tables travel by value
// (kernarg segment, read with scalar loads). grads[] is in member order:
// entry j*W + k is the k-th member (ascending worker id) of group j.
struct StepArgs {
    float* p;
    float* m;
    const float* gbar;  // lsgd_sgd_step only
    int64_t n;
    Hyper h;
    int32_t n_workers, n_groups, W;
    int32_t n_replicas, rdt;
    uint32_t xcd_chunk, upl;
    const float* lr_ptr;   // non-null: the learning rate is read here when the kernel runs
    int32_t bcast_grad;    // write the mean gradient into the first bcast_grad (binary32) member buffers
    int32_t literal;       // paper-literal reduction (else mean of means)
    int32_t win_blocks;    // replica-major copy-out: workgroups per window and replica group (a multiple of 8)
    int64_t copy_blocks;   // replica-major copy-out: logical workgroups (the grid strides over them)
    uint8_t group_start[kMaxWorkers + 4];  // runtime-layout kernel: group j is members [start[j], start[j+1])
    const void* grads[kMaxWorkers];
    void* replicas[kMaxReplicas];
};

// The hyperparameters a kernel uses: lr from device memory when given.
__device__ __forceinline__ Hyper resolve_hyper(const Hyper& h, const float* lr_ptr) {
    Hyper r = h;
    if (lr_ptr) r.lr = *lr_ptr;
    return r;
}

// Group-mean outputs of lsgd_group_mean / inputs of lsgd_global_mean.
struct MeanArgs {
    int64_t n;
    int32_t n_workers, n_groups, W;
    uint32_t xcd_chunk, upl;
    const void* in[kMaxWorkers];
    float* out[kMaxWorkers];
};

// ------------------------------------------------------------- per-unit bodies


// Units per lane tile in the flat runtime-layout (segmented) kernel
// (measured: two binary32 units per lane, stream-major, +2-5% over one on
// 3x5, 4x6, 2x64 and 32x4 groupings, -1% on the literal 4x4 step; bf16 stays
// at one unit for registers).
template <typename GT> struct SegTileUnits;
template <> struct SegTileUnits<float> { static constexpr int U = 2; };
template <> struct SegTileUnits<uint16_t> { static constexpr int U = 1; };

// Widened gradient values one lane may hold at once: up to kUnrollFloats the
// whole two-level tree is unrolled with every load issued up front (32 fp32
// units = a 4x4 grouping with two-unit tiles); above it groups stream through
// in batches of about kStreamFloats, which bounds registers for the 32- to
// 128-worker groupings. Batches of 128 floats beat 64 by 2% on 8x8 bfloat16
// (177 VGPRs, two waves per SIMD) and tied elsewhere; 32 tied.
constexpr int kUnrollFloats = 128;
constexpr int kStreamFloats = 128;

// Units per lane tile in the compile-time fused kernels for N = W*G
// gradients. Binary32: two units (visited stream-major; measured +6-8% over
// one) while the whole tree fits the unrolled form (N <= 16), four once the
// groups stream through the accumulator (N >= 32: +3-8% over two at 8x4,
// 4x8, 8x8, 16x4, 2x16 and 16x8, in same-process A/Bs; at N <= 16 three or
// four units lose 1-3%, since they leave the unrolled form). bfloat16 tiles
// stay at one unit: two units measured -1% at 4x4, +0.6% / -0.2% on the
// 3.5e8-element 8x8 workload (step kernel alone / whole step), +1.6% at 8x8
// and +4% at 16x8 on 2.6e7 elements.
// With 32 or more groups the pairwise accumulator over groups holds
// log2(G) + 1 partial sums of the tile, and four-unit tiles spilled to
// scratch (2.3 KB per lane at 4x32 and 2x32): those kernels take two units.
// So do 16 groups of 4 (and of 3), whose four-unit kernels spilled 2.3 KB
// per lane; with two (158 VGPRs, no scratch) the ResNet-50-sized 16x4 step
// ran 49% faster with 64 replicas, 87% without, the plan step 5% and the
// LARS step 11% faster.
template <typename GT>
constexpr int tile_units(int n_workers, int n_groups = 1) {
    return sizeof(GT) == 4 ? (n_workers * 2 * Unit<GT>::VEC <= kUnrollFloats || n_groups >= 32 ||
                                      (n_groups == 16 && (n_workers == 48 || n_workers == 64))
                                  ? 2
                                  : 4)
                           : 1;
}

// Pairwise sum of K leaves (compile-time K) of T floats each: unrolled while
// K * LW floats (LW = floats a leaf loads) stay within kUnrollFloats, so that
// every load is issued up front; otherwise streamed in batches of about
// kStreamFloats through a compile-time-sized pairwise accumulator. Both give
// PW over the K leaves in order.
template <int K, int T, int LW, typename Leaf>
__device__ __forceinline__ void pw_leaves(const Leaf& leaf, float (&out)[T]) {
    if constexpr (K * LW <= kUnrollFloats) {
        pw_tree<0, K, T>(leaf, out);
    } else {
        // batches of a divisor of K leaves (a power of two where K is one), so
        // that they cover the K leaves exactly: a batch of kStreamFloats / LW
        // leaves that does not divide K would call leaf() past K
        constexpr int B0 = kStreamFloats / LW;
        constexpr int B = largest_divisor_le(K, B0 < 1 ? 1 : (B0 > K ? K : B0));
        static_assert(K % B == 0, "leaf batches cover the K leaves exactly");
        PwAcc<T, ilog2(K) + 1> acc;
#pragma unroll 1
        for (int j0 = 0; j0 < K; j0 += B) {
            float x[B][T];
#pragma unroll
            for (int q = 0; q < B; ++q) leaf(j0 + q, x[q]);
#pragma unroll
            for (int q = 0; q < B; ++q) acc.push(x[q]);
        }
        acc.result(out);
    }
}

// Optional broadcast of the mean gradient into the (binary32) gradient
// buffers of the first s.bcast_grad() members: all N when the step kernel
// writes the whole broadcast, only the first member when a copy pass of its
// own then copies that buffer to the others.
template <typename GT, int U, bool TAIL, typename Src>
__device__ __forceinline__ void broadcast_mean(const Src& s, const int64_t (&e0)[U], int cnt,
                                               float (&gbar)[U * Unit<GT>::VEC]) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    if constexpr (sizeof(GT) == 4) {
        const int nw = s.bcast_grad();
        if (nw > 0) {
            for (int k = 0; k < nw; ++k) {
                float* g = static_cast<float*>(const_cast<void*>(s.grad(k)));
#pragma unroll
                for (int q = 0; q < U; ++q) store_f32<VEC, TAIL>(g, e0[q], cnt, slice<VEC, T>(gbar, q));
            }
        }
    }
}

// Parameters and momentum loaded, through the caches where they will be
// stored through them (s.cached_state(); see store_state), else
// nontemporally.
template <int VEC, int U, bool TAIL, typename Src>
__device__ __forceinline__ void load_state(const Src& s, const int64_t (&e0)[U], int cnt,
                                           float (&p)[U * VEC], float (&m)[U * VEC]) {
    constexpr int T = U * VEC;
    if (s.cached_state()) {
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32_cached<VEC, TAIL>(s.p(), e0[q], cnt, slice<VEC, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32_cached<VEC, TAIL>(s.m(), e0[q], cnt, slice<VEC, T>(m, q));
    } else {
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32<VEC, TAIL>(s.p(), e0[q], cnt, slice<VEC, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32<VEC, TAIL>(s.m(), e0[q], cnt, slice<VEC, T>(m, q));
    }
}

// Parameters and momentum of the compile-time fused kernels and of the
// update kernel go through the caches (write-back) when there are at most 16
// gradient buffers and parameters plus momentum fit the Infinity Cache
// (kCachedStateBytes), nontemporally otherwise. Measured in the same process
// with the Infinity Cache flushed before every step (so that no step reads
// what the previous one left there), cached loads and stores against
// nontemporal ones: 4x4 +4% at n = 1.2e7, +7% at 2.6e7, +5% at 3e7, +3% at
// 3.5e7, +0.6% at 4e7, -1% at 5e7, -4% at 1e8 and 2e8; 2x2 +12-14% up to
// 3.5e7, even at 2e8; the update alone +8% at 2.6e7, -4% at 3.5e8. With 32
// and more buffers cached stores lost 1-5% at every size. The kernels are
// instantiated both ways where the first condition holds and the host picks
// one at launch (a runtime branch between the forms inside one kernel cost
// the 64- and 128-buffer kernels 2-3%).
constexpr int64_t kCachedStateBytes = int64_t{288} << 20;
__host__ __device__ constexpr bool cached_state_for(int n_workers) { return n_workers <= 16; }
// The whole rule, for n elements of parameters (and of momentum).
__host__ __device__ constexpr bool use_cached_state(int n_workers, int64_t n) {
    return cached_state_for(n_workers) && n <= kCachedStateBytes / 8;
}

// Parameters, momentum and replicas stored. Parameters and momentum go
// through the caches (write-back) when s.cached_state() is set, else with
// nontemporal stores.
template <int VEC, int U, bool TAIL, typename Src>
__device__ __forceinline__ void store_state(const Src& s, const int64_t (&e0)[U], int cnt,
                                            const float (&p)[U * VEC], const float (&m)[U * VEC]) {
    constexpr int T = U * VEC;
    if (s.cached_state()) {
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32_cached<VEC, TAIL>(s.p(), e0[q], cnt, slice<VEC, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32_cached<VEC, TAIL>(s.m(), e0[q], cnt, slice<VEC, T>(m, q));
    } else {
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32<VEC, TAIL>(s.p(), e0[q], cnt, slice<VEC, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32<VEC, TAIL>(s.m(), e0[q], cnt, slice<VEC, T>(m, q));
    }
    const int R = s.n_replicas();
    const int rdt = s.rdt();
    for (int r = 0; r < R; ++r) {
        void* rp = s.replica(r);
#pragma unroll
        for (int q = 0; q < U; ++q) store_replica<VEC, TAIL>(rp, rdt, e0[q], cnt, slice<VEC, T>(p, q));
    }
}

// The update on loaded state, then parameters, momentum and replicas stored.
template <int VEC, int U, bool TAIL, typename Src>
__device__ __forceinline__ void update_and_store(const Src& s, const int64_t (&e0)[U], int cnt,
                                                 const float (&gbar)[U * VEC], float (&p)[U * VEC],
                                                 float (&m)[U * VEC]) {
    sgd_update<U * VEC>(s.hyper(), gbar, p, m);
    store_state<VEC, U, TAIL>(s, e0, cnt, p, m);
}

// Everything after the mean gradient, for a tile of U units: optional
// broadcast, the update, and the copy-out.
template <typename GT, int U, bool TAIL, typename Src>
__device__ __forceinline__ void finish_tile(const Src& s, const int64_t (&e0)[U], int cnt,
                                            float (&gbar)[U * Unit<GT>::VEC]) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    broadcast_mean<GT, U, TAIL>(s, e0, cnt, gbar);
    float p[T], m[T];
    load_state<VEC, U, TAIL>(s, e0, cnt, p, m);
    update_and_store<VEC, U, TAIL>(s, e0, cnt, gbar, p, m);
}

// Fused step on one tile of U units, compile-time W and G (powers of two).
// Every array holds T = U*VEC floats: the tree is the same PW for each of them.
// Small N*T: the whole two-level tree is unrolled and every load issued up
// front. Large: groups are streamed GU at a time and folded into a pairwise
// accumulator over groups, which yields the same PW order. TAIL (the ragged
// end of a tensor, cnt < VEC elements) only with U = 1.
// Mean of means: each group's sum / W, then the sum over groups / G. With
// s.literal() (uniform) the paper-literal form: each group's sum / N = W*G,
// summed over the groups with no further division. Every divisor is a power
// of two, so each division is a multiplication by the exact reciprocal (the
// same rounding of the same exact quotient).
template <typename GT, int W, int G, int U, bool TAIL, typename Src>
__device__ __forceinline__ void mean_tile_ct(const Src& s, const int64_t (&e0)[U], int cnt,
                                             float (&gbar)[U * Unit<GT>::VEC]) {
    static_assert(!TAIL || U == 1, "ragged units are processed one at a time");
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    const bool lit = s.literal() != 0;
    // Divisions by powers of two are the exact multiplications by 1/W, 1/N or
    // 1/G; the others (W = 3, 5, 6 or 7; G = 3, 5, 6, 7 or 12; N of either)
    // are divisions. The mean of means divides each group's sum by W and the
    // total by G; the literal reduction each group's sum by N, the total by 1.
    constexpr bool kPow2W = (W & (W - 1)) == 0;
    constexpr bool kPow2G = (G & (G - 1)) == 0;
    const float group_div = lit ? static_cast<float>(W * G) : static_cast<float>(W);
    const float group_scale = 1.0f / group_div;
    const float total_scale = lit ? 1.0f : 1.0f / static_cast<float>(G);
    auto group_leaf = [&](int j, float (&gm)[T]) {
        auto member_leaf = [&](int k, float (&x)[T]) {
            const void* g = s.grad(j * W + k);
#pragma unroll
            for (int q = 0; q < U; ++q) load_grad<GT, TAIL>(g, e0[q], cnt, slice<VEC, T>(x, q));
        };
        float sum[T];
        if constexpr (W <= 16) pw_tree<0, W, T>(member_leaf, sum);
        else pw_leaves<W, T, T>(member_leaf, sum);   // larger groups: members streamed through an accumulator
        if constexpr (kPow2W && kPow2G) {
#pragma unroll
            for (int v = 0; v < T; ++v) gm[v] = sum[v] * group_scale;
        } else if constexpr (!kPow2W) {
#pragma unroll
            for (int v = 0; v < T; ++v) gm[v] = sum[v] / group_div;
        } else if (lit) {   // W a power of two, N not
#pragma unroll
            for (int v = 0; v < T; ++v) gm[v] = sum[v] / group_div;
        } else {
#pragma unroll
            for (int v = 0; v < T; ++v) gm[v] = sum[v] * group_scale;
        }
    };
    float tot[T];
    pw_leaves<G, T, W * T>(group_leaf, tot);
    if constexpr (kPow2G) {
#pragma unroll
        for (int v = 0; v < T; ++v) gbar[v] = tot[v] * total_scale;
    } else if (lit) {
#pragma unroll
        for (int v = 0; v < T; ++v) gbar[v] = tot[v];
    } else {
#pragma unroll
        for (int v = 0; v < T; ++v) gbar[v] = tot[v] / static_cast<float>(G);
    }
}

template <typename GT, int W, int G, int U, bool TAIL, typename Src>
__device__ __forceinline__ void fused_tile_ct(const Src& s, const int64_t (&e0)[U], int cnt) {
    float gbar[U * Unit<GT>::VEC];
    mean_tile_ct<GT, W, G, U, TAIL>(s, e0, cnt, gbar);
    finish_tile<GT, U, TAIL>(s, e0, cnt, gbar);
}

template <typename GT, int W, int G, bool TAIL, typename Src>
__device__ __forceinline__ void fused_unit_ct(const Src& s, int64_t e0, int cnt) {
    const int64_t e[1] = {e0};
    fused_tile_ct<GT, W, G, 1, TAIL>(s, e, cnt);
}

// The mean gradient of a lane tile (U units) for group layouts known only at
// run time. Group j is members [gs(j), gs(j+1)) of the member-ordered
// gradients. Mean of means (literal = false, equal groups of W): each group's
// PW sum / W, PW over the G results, / G. Paper-literal (any partition): each
// group's PW sum / N, PW over the G results, no further division.
template <typename GT, int LV, int U, bool TAIL, typename Src, typename Start>
__device__ __forceinline__ void mean_tile_seg(const Src& s, int N, int G, const Start& gs, bool literal,
                                              const int64_t (&e0)[U], int cnt,
                                              float (&gbar)[U * Unit<GT>::VEC]) {
    constexpr int T = U * Unit<GT>::VEC;
    const float dg = static_cast<float>(literal ? N : gs(1) - gs(0));
    PwAcc<T, LV> groups;
    const int glevels = acc_levels(G);
    pw_segments<GT, LV, U, TAIL>(N, G, [&](int k) { return s.grad(k); }, gs, e0, cnt,
                                 [&](int, float (&sum)[T]) {
#pragma unroll
                                     for (int v = 0; v < T; ++v) sum[v] = sum[v] / dg;
                                     groups.push(sum, glevels);
                                 });
    groups.result(gbar, glevels);
    if (!literal) {
        const float gf = static_cast<float>(G);
#pragma unroll
        for (int v = 0; v < T; ++v) gbar[v] = gbar[v] / gf;
    }
}

template <typename GT, int LV, bool TAIL, typename Src, typename Start>
__device__ __forceinline__ void mean_unit_seg(const Src& s, int N, int G, const Start& gs, bool literal,
                                              int64_t e0, int cnt, float (&gbar)[Unit<GT>::VEC]) {
    const int64_t e[1] = {e0};
    mean_tile_seg<GT, LV, 1, TAIL>(s, N, G, gs, literal, e, cnt, gbar);
}

// Fused step on a lane tile for runtime group layouts. Parameters and
// momentum are loaded first so that their latency overlaps the gradient
// stream.
template <typename GT, int LV, int U, bool TAIL, typename Src, typename Start>
__device__ __forceinline__ void fused_tile_seg(const Src& s, int N, int G, const Start& gs, bool literal,
                                               const int64_t (&e0)[U], int cnt) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    float p[T], m[T];
    load_state<VEC, U, TAIL>(s, e0, cnt, p, m);
    float gbar[T];
    mean_tile_seg<GT, LV, U, TAIL>(s, N, G, gs, literal, e0, cnt, gbar);
    broadcast_mean<GT, U, TAIL>(s, e0, cnt, gbar);
    update_and_store<VEC, U, TAIL>(s, e0, cnt, gbar, p, m);
}

template <typename GT, int LV, bool TAIL, typename Src, typename Start>
__device__ __forceinline__ void fused_unit_seg(const Src& s, int N, int G, const Start& gs, bool literal,
                                               int64_t e0, int cnt) {
    const int64_t e[1] = {e0};
    fused_tile_seg<GT, LV, 1, TAIL>(s, N, G, gs, literal, e, cnt);
}

// Pointer source for the planless fused step: everything from StepArgs.
// CACHED: store parameters and momentum through the caches (1) or
// nontemporally (0).
template <int CACHED>
struct FlatSrcT {
    const StepArgs& a;
    Hyper h;
    __device__ const void* grad(int k) const { return a.grads[k]; }
    __device__ float* p() const { return a.p; }
    __device__ float* m() const { return a.m; }
    __device__ void* replica(int r) const { return a.replicas[r]; }
    __device__ int n_replicas() const { return a.n_replicas; }
    __device__ int rdt() const { return a.rdt; }
    __device__ Hyper hyper() const { return h; }
    __device__ int bcast_grad() const { return a.bcast_grad; }
    __device__ int n_workers() const { return a.n_workers; }
    __device__ int literal() const { return a.literal; }
    __device__ int cached_state() const { return CACHED; }
};

// ------------------------------------------------------------- flat kernels

// Lane tiles over the units of a flat vector (for_tiles). The unit index space
// is [0, full] with unit `full` the ragged tail (n % VEC elements, present
// only when that is nonzero): the lane whose partial tile holds it runs it
// through the TAIL form of the unit body.
template <typename GT, int W, int G, int U, int CACHED>
__device__ __forceinline__ void step_flat_ct_body(const StepArgs& a) {
    constexpr int VEC = Unit<GT>::VEC;
    const FlatSrcT<CACHED> s{a, resolve_hyper(a.h, a.lr_ptr)};
    const int64_t full = a.n / VEC;
    const int rem = static_cast<int>(a.n - full * VEC);
    for_tiles<U, VEC>(
        full, full + (rem != 0), a.xcd_chunk, a.upl,
        [&](const int64_t (&e0)[U]) { fused_tile_ct<GT, W, G, U, false>(s, e0, VEC); },
        [&](int64_t u) {
            if (u < full) fused_unit_ct<GT, W, G, false>(s, u * VEC, VEC);
            else fused_unit_ct<GT, W, G, true>(s, u * VEC, rem);
        });
}

template <typename GT, int W, int G, int U, int CACHED>
__global__ __launch_bounds__(kBlock) void step_flat_ct(StepArgs a) {
    step_flat_ct_body<GT, W, G, U, CACHED>(a);
}

// The same kernel with at most CAP waves per SIMD. Left to itself, the
// compiler schedules for the highest occupancy the registers allow, and
// for some groupings it gets there by holding fewer loads in flight: the
// bfloat16 kernels for groups of 3 in 8 or more groups sink each gradient
// load to its use and wait for it (one 16-byte load in flight per wave), and
// the small binary32 groupings run four or more waves with short load
// batches. Under a cap of 2 or 3 the scheduler keeps a batch of loads in
// flight instead.
template <typename GT, int W, int G, int U, int CACHED, int CAP>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(1, CAP))) void step_flat_ct_cap(StepArgs a) {
    step_flat_ct_body<GT, W, G, U, CACHED>(a);
}

// The wave cap of the compile-time flat step kernel for G groups of W
// workers, 0 for none: measured, each grouping against the uncapped kernel
// at the ResNet-50 size (25.6M elements, same process, replicas R = N and
// R = 0). A grouping is listed where a cap gains at least one point of the
// 8 TB/s peak on the mean of the two and loses at most one in either.
struct WaveCapEntry {
    short W, G, cap;
};
constexpr WaveCapEntry kWaveCapF32[] = {
    {1, 8, 2},  {1, 16, 2}, {1, 128, 2}, {2, 4, 2},  {2, 8, 2},  {2, 12, 2}, {3, 3, 2},  {3, 4, 2},
    {3, 5, 2},  {4, 2, 2},  {4, 4, 2},   {4, 6, 2},  {5, 2, 2},  {5, 3, 2},  {6, 2, 2},  {8, 1, 2},
    {12, 1, 2}, {12, 5, 2}, {16, 1, 2},  {16, 2, 2}, {16, 4, 2}, {16, 8, 2}, {1, 2, 3},  {1, 3, 3},
    {1, 4, 3},  {1, 5, 3},  {1, 6, 3},   {2, 1, 3},  {2, 2, 3},  {3, 1, 3},  {3, 2, 3},  {3, 8, 3},
    {3, 12, 3}, {3, 16, 3}, {4, 1, 3},   {4, 3, 3},  {5, 1, 3},  {6, 1, 3},  {8, 6, 3},  {12, 3, 3},
};
constexpr WaveCapEntry kWaveCapBF16[] = {
    {1, 2, 2}, {1, 4, 2},  {2, 1, 2},  {2, 2, 2}, {3, 1, 2}, {3, 8, 2}, {3, 12, 2},
    {3, 16, 2}, {3, 32, 2}, {4, 1, 2}, {5, 16, 2}, {8, 1, 2}, {8, 6, 2}, {8, 12, 2},
    {1, 8, 3}, {1, 16, 3}, {2, 4, 3}, {4, 2, 3}, {5, 1, 3}, {6, 1, 3},
};
template <typename GT>
constexpr int flat_wave_cap(int W, int G) {
    constexpr bool kBF16 = sizeof(GT) == 2;
    const WaveCapEntry* t = kBF16 ? kWaveCapBF16 : kWaveCapF32;
    const int n = kBF16 ? sizeof(kWaveCapBF16) / sizeof(WaveCapEntry) : sizeof(kWaveCapF32) / sizeof(WaveCapEntry);
    for (int i = 0; i < n; ++i)
        if (t[i].W == W && t[i].G == G) return t[i].cap;
    return 0;
}

// The flat step kernel for (W, G): capped where the table says so.
template <typename GT, int W, int G, int U, int CACHED>
constexpr auto flat_step_kernel() {
    constexpr int cap = flat_wave_cap<GT>(W, G);
    if constexpr (cap != 0) return step_flat_ct_cap<GT, W, G, U, CACHED, cap>;
    else return step_flat_ct<GT, W, G, U, CACHED>;
}

// Runtime group layouts (non-power-of-two or large counts, and the
// paper-literal reduction): group j is members [group_start[j],
// group_start[j+1]) of the member-ordered pointer table.
template <typename GT, int LV, int U, int CACHED>
__global__ __launch_bounds__(kBlock) void step_flat_seg(StepArgs a) {
    constexpr int VEC = Unit<GT>::VEC;
    const FlatSrcT<CACHED> s{a, resolve_hyper(a.h, a.lr_ptr)};
    const int64_t full = a.n / VEC;
    const int rem = static_cast<int>(a.n - full * VEC);
    const bool literal = a.literal != 0;
    auto gs = [&](int j) { return static_cast<int>(a.group_start[j]); };
    for_tiles<U, VEC>(
        full, full + (rem != 0), a.xcd_chunk, a.upl,
        [&](const int64_t (&e0)[U]) { fused_tile_seg<GT, LV, U, false>(s, a.n_workers, a.n_groups, gs, literal, e0, VEC); },
        [&](int64_t u) {
            if (u < full) fused_unit_seg<GT, LV, false>(s, a.n_workers, a.n_groups, gs, literal, u * VEC, VEC);
            else fused_unit_seg<GT, LV, true>(s, a.n_workers, a.n_groups, gs, literal, u * VEC, rem);
        });
}

// lsgd_group_mean, compile-time W (a power of two): every group's mean of its
// W members for one tile of U units, stored stream-major.
template <typename GT, int W, int U, bool TAIL>
__device__ __forceinline__ void group_mean_tile(const MeanArgs& a, const int64_t (&e0)[U], int cnt) {
    constexpr int VEC = Unit<GT>::VEC;
    constexpr int T = U * VEC;
    for (int j = 0; j < a.n_groups; ++j) {
        float sum[T];
        pw_leaves<W, T, T>([&](int k, float (&x)[T]) {
            const void* g = a.in[j * W + k];
#pragma unroll
            for (int q = 0; q < U; ++q) load_grad<GT, TAIL>(g, e0[q], cnt, slice<VEC, T>(x, q));
        }, sum);
#pragma unroll
        for (int v = 0; v < T; ++v) sum[v] = sum[v] / static_cast<float>(W);
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32<VEC, TAIL>(a.out[j], e0[q], cnt, slice<VEC, T>(sum, q));
    }
}

template <typename GT, int W, int U>
__global__ __launch_bounds__(kBlock) void group_mean_kernel_ct(MeanArgs a) {
    constexpr int VEC = Unit<GT>::VEC;
    const int64_t full = a.n / VEC;
    const int rem = static_cast<int>(a.n - full * VEC);
    for_tiles<U, VEC>(
        full, full + (rem != 0), a.xcd_chunk, a.upl,
        [&](const int64_t (&e0)[U]) { group_mean_tile<GT, W, U, false>(a, e0, VEC); },
        [&](int64_t u) {
            const int64_t e[1] = {u * VEC};
            if (u < full) group_mean_tile<GT, W, 1, false>(a, e, VEC);
            else group_mean_tile<GT, W, 1, true>(a, e, rem);
        });
}

// lsgd_group_mean, runtime W (any equal-size grouping), one unit.
template <typename GT, int LV, bool TAIL>
__device__ __forceinline__ void group_mean_unit(const MeanArgs& a, int64_t e0, int cnt) {
    constexpr int VEC = Unit<GT>::VEC;
    const int W = a.W;
    const float wf = static_cast<float>(W);
    const int64_t e[1] = {e0};
    pw_segments<GT, LV, 1, TAIL>(a.n_workers, a.n_groups, [&](int k) { return a.in[k]; },
                                 [&](int j) { return j * W; }, e, cnt, [&](int j, float (&sum)[VEC]) {
#pragma unroll
                                  for (int v = 0; v < VEC; ++v) sum[v] = sum[v] / wf;
                                  store_f32<VEC, TAIL>(a.out[j], e0, cnt, sum);
                              });
}

template <typename GT, int LV>
__global__ __launch_bounds__(kBlock) void group_mean_kernel(MeanArgs a) {
    constexpr int VEC = Unit<GT>::VEC;
    const int64_t full = a.n / VEC;
    const int rem = static_cast<int>(a.n - full * VEC);
    for_units(full + (rem != 0), a.xcd_chunk, a.upl, [&](int64_t u) {
        if (u < full) group_mean_unit<GT, LV, false>(a, u * VEC, VEC);
        else group_mean_unit<GT, LV, true>(a, u * VEC, rem);
    });
}

// lsgd_global_mean, compile-time G (a power of two): PW over the G group
// means, / G, for one tile of U 4-element units.
template <int G, int U, bool TAIL>
__device__ __forceinline__ void global_mean_tile(const MeanArgs& a, const int64_t (&e0)[U], int cnt) {
    constexpr int T = U * 4;
    float s[T];
    pw_leaves<G, T, T>([&](int j, float (&x)[T]) {
        const float* in = static_cast<const float*>(a.in[j]);
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32<4, TAIL>(in, e0[q], cnt, slice<4, T>(x, q));
    }, s);
#pragma unroll
    for (int v = 0; v < T; ++v) s[v] = s[v] / static_cast<float>(G);
#pragma unroll
    for (int q = 0; q < U; ++q) store_f32<4, TAIL>(a.out[0], e0[q], cnt, slice<4, T>(s, q));
}

template <int G, int U>
__global__ __launch_bounds__(kBlock) void global_mean_kernel_ct(MeanArgs a) {
    const int64_t full = a.n / 4;
    const int rem = static_cast<int>(a.n - full * 4);
    for_tiles<U, 4>(
        full, full + (rem != 0), a.xcd_chunk, a.upl,
        [&](const int64_t (&e0)[U]) { global_mean_tile<G, U, false>(a, e0, 4); },
        [&](int64_t u) {
            const int64_t e[1] = {u * 4};
            if (u < full) global_mean_tile<G, 1, false>(a, e, 4);
            else global_mean_tile<G, 1, true>(a, e, rem);
        });
}

// lsgd_global_mean, runtime G, one unit: the G means form one run.
template <int LV, bool TAIL>
__device__ __forceinline__ void global_mean_unit(const MeanArgs& a, int64_t e0, int cnt) {
    const int G = a.n_groups;
    const float gf = static_cast<float>(G);
    const int64_t e[1] = {e0};
    pw_segments<float, LV, 1, TAIL>(G, 1, [&](int j) { return a.in[j]; }, [&](int j) { return j * G; },
                                    e, cnt, [&](int, float (&sum)[4]) {
#pragma unroll
                                     for (int v = 0; v < 4; ++v) sum[v] = sum[v] / gf;
                                     store_f32<4, TAIL>(a.out[0], e0, cnt, sum);
                                 });
}

template <int LV>
__global__ __launch_bounds__(kBlock) void global_mean_kernel(MeanArgs a) {
    const int64_t full = a.n / 4;
    const int rem = static_cast<int>(a.n - full * 4);
    for_units(full + (rem != 0), a.xcd_chunk, a.upl, [&](int64_t u) {
        if (u < full) global_mean_unit<LV, false>(a, u * 4, 4);
        else global_mean_unit<LV, true>(a, u * 4, rem);
    });
}

// lsgd_sgd_step: update and copy-out from a precomputed mean gradient, one
// tile of U 4-element units, stream-major.
template <int U, bool TAIL, int CACHED>
__device__ __forceinline__ void sgd_tile(const StepArgs& a, const Hyper& h, const int64_t (&e0)[U],
                                         int cnt) {
    constexpr int T = U * 4;
    float g[T], p[T], m[T];
#pragma unroll
    for (int q = 0; q < U; ++q) load_f32<4, TAIL>(a.gbar, e0[q], cnt, slice<4, T>(g, q));
    if constexpr (CACHED != 0) {
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32_cached<4, TAIL>(a.p, e0[q], cnt, slice<4, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32_cached<4, TAIL>(a.m, e0[q], cnt, slice<4, T>(m, q));
    } else {
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32<4, TAIL>(a.p, e0[q], cnt, slice<4, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) load_f32<4, TAIL>(a.m, e0[q], cnt, slice<4, T>(m, q));
    }
    sgd_update<T>(h, g, p, m);
    if constexpr (CACHED != 0) {
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32_cached<4, TAIL>(a.p, e0[q], cnt, slice<4, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32_cached<4, TAIL>(a.m, e0[q], cnt, slice<4, T>(m, q));
    } else {
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32<4, TAIL>(a.p, e0[q], cnt, slice<4, T>(p, q));
#pragma unroll
        for (int q = 0; q < U; ++q) store_f32<4, TAIL>(a.m, e0[q], cnt, slice<4, T>(m, q));
    }
    for (int r = 0; r < a.n_replicas; ++r) {
        void* rp = a.replicas[r];
#pragma unroll
        for (int q = 0; q < U; ++q) store_replica<4, TAIL>(rp, a.rdt, e0[q], cnt, slice<4, T>(p, q));
    }
}

template <int U, int CACHED>
__global__ __launch_bounds__(kBlock) void sgd_kernel(StepArgs a) {
    const Hyper h = resolve_hyper(a.h, a.lr_ptr);
    const int64_t full = a.n / 4;
    const int rem = static_cast<int>(a.n - full * 4);
    for_tiles<U, 4>(
        full, full + (rem != 0), a.xcd_chunk, a.upl,
        [&](const int64_t (&e0)[U]) { sgd_tile<U, false, CACHED>(a, h, e0, 4); },
        [&](int64_t u) {
            const int64_t e[1] = {u * 4};
            if (u < full) sgd_tile<1, false, CACHED>(a, h, e, 4);
            else sgd_tile<1, true, CACHED>(a, h, e, rem);
        });
}

// ------------------------------------------------------------- copy-out pass
//
// With several replicas the copy-out runs as a pass of its own after the step
// kernel (which then writes no replica). It runs replica-major over windows of
// the parameter vector: workgroup b writes block s of window w to replica
// group q (RK consecutive replicas), b = (w*ceil(R/RK) + q)*win_blocks + s, so
// at any time the chip writes a few replica streams instead of all R. With
// win_blocks a multiple of 8 each XCD (workgroups go to XCD b % 8) reads the
// same eighth of the window for every replica group: after the first group the
// window comes from that XCD's L2 (p is read with cache-allocating loads; a
// window is 8 MB, 1 MB per XCD). A lane loads U units of p and stores them to
// each of its group's replicas: several loads in flight and several stores per
// load keep the pass at the write bandwidth (one unit and one replica per lane
// left the bfloat16 pass at about half of it). Binary32 replicas take
// 4-element units, bfloat16 replicas 8-element units, so every store is 16
// bytes. Grids above kMaxGridBlocks stride over the logical workgroups.
template <int VEC, int U, int RK>
__device__ __forceinline__ void copy_out_rmajor_block(const StepArgs& a, int64_t b) {
    const int64_t full = a.n / VEC;
    const int rem = static_cast<int>(a.n - full * VEC);
    const int n_rg = (a.n_replicas + RK - 1) / RK;
    const int64_t per_win = static_cast<int64_t>(a.win_blocks) * n_rg;
    const int64_t w = b / per_win;
    const int64_t rb = b - w * per_win;
    const int q = static_cast<int>(rb / a.win_blocks);
    const int64_t sblk = rb - static_cast<int64_t>(q) * a.win_blocks;
    const int64_t u0 = (w * a.win_blocks + sblk) * kBlock * U + threadIdx.x;
    const int r0 = q * RK;
    float x[U][VEC];
#pragma unroll
    for (int t = 0; t < U; ++t) {
        const int64_t u = u0 + static_cast<int64_t>(t) * kBlock;
        if (u < full) load_f32_cached<VEC, false>(a.p, u * VEC, VEC, x[t]);
        else if (u == full && rem != 0) load_f32_cached<VEC, true>(a.p, u * VEC, rem, x[t]);
    }
#pragma unroll
    for (int k = 0; k < RK; ++k) {
        if (r0 + k >= a.n_replicas) break;
        void* dst = a.replicas[r0 + k];
#pragma unroll
        for (int t = 0; t < U; ++t) {
            const int64_t u = u0 + static_cast<int64_t>(t) * kBlock;
            if (u < full) store_replica<VEC, false>(dst, a.rdt, u * VEC, VEC, x[t]);
            else if (u == full && rem != 0) store_replica<VEC, true>(dst, a.rdt, u * VEC, rem, x[t]);
        }
    }
}

// The grid (a multiple of 8 workgroups, or all of them) strides over the
// logical workgroups, so each keeps its XCD.
template <int VEC, int U, int RK>
__global__ __launch_bounds__(kBlock) void copy_out_rmajor_kernel(StepArgs a) {
    for (int64_t b = blockIdx.x; b < a.copy_blocks; b += gridDim.x) copy_out_rmajor_block<VEC, U, RK>(a, b);
}

}  // namespace lsgd
