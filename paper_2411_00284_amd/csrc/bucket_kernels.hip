// gfx950 kernels and C-ABI entry points of the bucketed FSDP copy path.
//
// All four kernels are HBM-bound streams (no contraction, so no MFMA): one
// launch covers every parameter of a bucket.  The work of a launch is cut
// into tiles that never cross a parameter (and, for the W-way copies, never
// cross one rank's segment of a parameter), so that a tile is a plain
// contiguous copy, cast or reduction with 16-byte vector accesses.  Tiles are
// numbered parameter by parameter; the first tile of every parameter is kept
// in one register per lane of a wavefront, and a ballot over it finds the
// parameter of any tile in O(1).  The per-parameter table travels in the
// kernel arguments, read through the scalar cache.
//
// Numerics (SimpleFSDP sections 3.2.1 and 4):
//   * fp32 -> bf16 is IEEE round-half-to-even on the 16 dropped bits; NaN
//     gives (bits >> 16) | 0x0040;
//   * bf16 -> fp32 is exact (append 16 zero bits);
//   * the average is an fp32 sum over source ranks in order 0..W-1, starting
//     from the rank-0 value, then one IEEE division by W.  The library is
//     built without fast-math or fp contraction and with fp32 subnormals
//     enabled, so every add and the division are correctly rounded.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "plan_impl.h"

namespace fsdp {
namespace {

#ifndef FSDP_REDUCE_BATCH
#define FSDP_REDUCE_BATCH 4
#endif
#ifndef FSDP_BLOCKS_PER_CU
#define FSDP_BLOCKS_PER_CU 4096
#endif
#ifndef FSDP_NT_LOAD
#define FSDP_NT_LOAD 1
#endif
#ifndef FSDP_NT_STORE
#define FSDP_NT_STORE 1
#endif

constexpr int PMAX = FSDP_MAX_PARAMS;
constexpr int kReduceBatch = FSDP_REDUCE_BATCH;   // source ranks loaded before they are added
constexpr int kBlocksPerCU = FSDP_BLOCKS_PER_CU;  // workgroups per CU in the grid-stride launch
constexpr int kPackGridSlack = 4;                  // max workgroups per tile of work for the 2-D pack grid

// ------------------------------------------------------------------ device helpers

__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t bf16x2_bits(float lo, float hi) {
    return bf16_bits(lo) | (bf16_bits(hi) << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Parameter owning tile t: the last p with tile_start[p] <= t.  Every lane of
// the wave holds tile_start[lane] (INT_MAX past the last parameter).
__device__ __forceinline__ int param_of_tile(int my_start, int t) {
    const uint64_t m = __ballot(my_start <= t);
    return __builtin_amdgcn_readfirstlane(__popcll(m) - 1);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// 16-byte accesses; streamed data may bypass cache retention (non-temporal).
__device__ __forceinline__ uint4 ld16(const uint16_t* p) {
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
#if FSDP_NT_LOAD
    const u32x4 v = __builtin_nontemporal_load(q);
#else
    const u32x4 v = *q;
#endif
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st16(uint16_t* p, uint4 v) {
    u32x4* q = reinterpret_cast<u32x4*>(p);
    const u32x4 w = {v.x, v.y, v.z, v.w};
#if FSDP_NT_STORE
    __builtin_nontemporal_store(w, q);
#else
    *q = w;
#endif
}
__device__ __forceinline__ float4 ldf16(const float* p) {
    const f32x4* q = reinterpret_cast<const f32x4*>(p);
#if FSDP_NT_LOAD
    const f32x4 v = __builtin_nontemporal_load(q);
#else
    const f32x4 v = *q;
#endif
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void stf16(float* p, float4 v) {
    f32x4* q = reinterpret_cast<f32x4*>(p);
    const f32x4 w = {v.x, v.y, v.z, v.w};
#if FSDP_NT_STORE
    __builtin_nontemporal_store(w, q);
#else
    *q = w;
#endif
}

// ------------------------------------------------------------------ ag_pack

struct PackArgs {
    const float* src[PMAX];
    int64_t off[PMAX + 1];       // off[P] = S
    int64_t valid[PMAX];         // n_{p,rank} * inner_p
    int32_t tile_start[PMAX];
    uint64_t vec_mask;           // bit p: src 16-byte aligned and off_p % 8 == 0
    uint16_t* dst;
    int32_t nparams;
    int32_t ntiles;
};

__device__ __forceinline__ uint4 cast8(const float* __restrict__ s) {
    const float4 a = ldf16(s);
    const float4 b = ldf16(s + 4);
    return make_uint4(bf16x2_bits(a.x, a.y), bf16x2_bits(a.z, a.w),
                      bf16x2_bits(b.x, b.y), bf16x2_bits(b.z, b.w));
}

// Tile lt of parameter p: cast-and-pack its part of [off_p, off_{p+1}).
__device__ __forceinline__ void pack_tile(const PackArgs& a, int p, int lt) {
    const int64_t off = a.off[p];
    const int64_t region = a.off[p + 1] - off;
    const int64_t valid = a.valid[p];
    const float* __restrict__ src = a.src[p];
    uint16_t* __restrict__ dst = a.dst + off;
    const int64_t lo = int64_t(lt) * kPackTile;
    const int64_t hi = min(lo + kPackTile, region);
    if (lo >= hi) return;
    const bool vec = (a.vec_mask >> p) & 1;
    if (vec && hi - lo == kPackTile && lo + kPackTile <= valid) {
        uint4 v[kPackSteps];
#pragma unroll
        for (int u = 0; u < kPackSteps; ++u)
            v[u] = cast8(src + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec);
#pragma unroll
        for (int u = 0; u < kPackSteps; ++u)
            st16(dst + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec, v[u]);
        return;
    }
    for (int u = 0; u < kPackSteps; ++u) {
        const int64_t g = lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec;
        if (g >= hi) break;
        if (vec && g + kVec <= hi && (g + kVec <= valid || g >= valid)) {
            st16(dst + g, g < valid ? cast8(src + g) : make_uint4(0, 0, 0, 0));
            continue;
        }
        for (int e = 0; e < kVec; ++e) {
            const int64_t k = g + e;
            if (k < hi) dst[k] = k < valid ? uint16_t(bf16_bits(src[k])) : uint16_t(0);
        }
    }
}

// Tiles numbered across the bucket; the parameter of a tile comes from the
// wave-ballot lookup.
__global__ void __launch_bounds__(kCopyBlock) ag_pack_kernel(const PackArgs a) {
    const int lane = threadIdx.x & 63;
    const int my_start = lane < a.nparams ? a.tile_start[lane] : INT_MAX;
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const int p = param_of_tile(my_start, t);
        pack_tile(a, p, t - a.tile_start[p]);
    }
}

// Grid (x, P): blockIdx.y is the parameter, so a workgroup's first memory
// access is its data rather than the tile table.  Used when the parameters'
// tile counts are similar enough that few workgroups find no tile.
__global__ void __launch_bounds__(kCopyBlock) ag_pack_grid_kernel(const PackArgs a) {
    const int p = blockIdx.y;
    const int nt = int((a.off[p + 1] - a.off[p] + kPackTile - 1) / kPackTile);
    for (int lt = blockIdx.x; lt < nt; lt += gridDim.x) pack_tile(a, p, lt);
}

// ------------------------------------------------------------------ ag_unpack

struct UnpackArgs {
    uint16_t* dst[PMAX];
    int64_t off[PMAX];
    int64_t seg[PMAX];           // L_p
    int64_t elems[PMAX];         // N_p * inner_p
    int32_t tiles_per_seg[PMAX]; // ceil(L_p / tile)
    int32_t tile_start[PMAX];
    uint64_t dst_aligned;        // bit p: dst[p] 16-byte aligned
    const uint16_t* src;         // gathered, rank-major [W][S]
    int64_t chunk;               // S
    int32_t nparams;
    int32_t ntiles;
};

// Copy elements [lo, hi) of one segment; `vec` when both ends are 16-byte aligned at 0.
__device__ __forceinline__ void copy_range(const uint16_t* __restrict__ s, uint16_t* __restrict__ d,
                                           int64_t lo, int64_t hi, bool vec) {
    if (vec && hi - lo == kCopyTile) {
        uint4 v[kCopySteps];
#pragma unroll
        for (int u = 0; u < kCopySteps; ++u) v[u] = ld16(s + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec);
#pragma unroll
        for (int u = 0; u < kCopySteps; ++u) st16(d + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec, v[u]);
        return;
    }
    for (int u = 0; u < kCopySteps; ++u) {
        const int64_t g = lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec;
        if (g >= hi) break;
        if (vec && g + kVec <= hi) {
            st16(d + g, ld16(s + g));
            continue;
        }
        for (int e = 0; e < kVec; ++e)
            if (g + e < hi) d[g + e] = s[g + e];
    }
}

__global__ void __launch_bounds__(kCopyBlock) ag_unpack_kernel(const UnpackArgs a) {
    const int lane = threadIdx.x & 63;
    const int my_start = lane < a.nparams ? a.tile_start[lane] : INT_MAX;
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const int p = param_of_tile(my_start, t);
        const int lt = t - a.tile_start[p];
        const int tps = a.tiles_per_seg[p];
        const int i = lt / tps;                          // source rank
        const int64_t st = lt - int64_t(i) * tps;
        const int64_t L = a.seg[p];
        const int64_t rest = a.elems[p] - int64_t(i) * L;
        const int64_t v = rest < L ? (rest > 0 ? rest : 0) : L;
        const int64_t lo = st * kCopyTile;
        const int64_t hi = min(lo + kCopyTile, v);
        if (lo >= hi) continue;
        const int64_t soff = int64_t(i) * a.chunk + a.off[p];
        const int64_t doff = int64_t(i) * L;
        const bool vec = ((a.dst_aligned >> p) & 1) && ((soff | doff) & (kVec - 1)) == 0;
        copy_range(a.src + soff, a.dst[p] + doff, lo, hi, vec);
    }
}

// ------------------------------------------------------------------ rs_pack

struct RsPackArgs {
    const uint16_t* src[PMAX];   // full bf16 gradients
    int64_t off[PMAX + 1];       // off[P] = S
    int64_t seg[PMAX];
    int64_t elems[PMAX];
    int32_t tiles_per_seg[PMAX]; // ceil((off_{p+1} - off_p) / tile)
    int32_t tile_start[PMAX];
    uint64_t src_aligned;        // bit p: src[p] 16-byte aligned
    uint16_t* dst;               // send buffer, destination-major [W][S]
    int64_t chunk;
    int32_t nparams;
    int32_t ntiles;
};

__global__ void __launch_bounds__(kCopyBlock) rs_pack_kernel(const RsPackArgs a) {
    const int lane = threadIdx.x & 63;
    const int my_start = lane < a.nparams ? a.tile_start[lane] : INT_MAX;
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const int p = param_of_tile(my_start, t);
        const int lt = t - a.tile_start[p];
        const int tps = a.tiles_per_seg[p];
        const int j = lt / tps;                          // destination rank
        const int64_t st = lt - int64_t(j) * tps;
        const int64_t region = a.off[p + 1] - a.off[p];
        const int64_t L = a.seg[p];
        const int64_t rest = a.elems[p] - int64_t(j) * L;
        const int64_t v = rest < L ? (rest > 0 ? rest : 0) : L;
        const int64_t lo = st * kCopyTile;
        const int64_t hi = min(lo + kCopyTile, region);
        const int64_t doff = int64_t(j) * a.chunk + a.off[p];
        const int64_t soff = int64_t(j) * L;
        const uint16_t* __restrict__ s = a.src[p] + soff;
        uint16_t* __restrict__ d = a.dst + doff;
        const bool vec = ((a.src_aligned >> p) & 1) && ((soff | doff) & (kVec - 1)) == 0;
        if (vec && hi - lo == kCopyTile && (hi <= v || lo >= v)) {
            if (hi <= v) {
                copy_range(s, d, lo, hi, true);
            } else {
#pragma unroll
                for (int u = 0; u < kCopySteps; ++u)
                    st16(d + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec, make_uint4(0, 0, 0, 0));
            }
            continue;
        }
        for (int u = 0; u < kCopySteps; ++u) {
            const int64_t g = lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec;
            if (g >= hi) break;
            if (vec && g + kVec <= hi && (g + kVec <= v || g >= v)) {
                st16(d + g, g < v ? ld16(s + g) : make_uint4(0, 0, 0, 0));
                continue;
            }
            for (int e = 0; e < kVec; ++e) {
                const int64_t k = g + e;
                if (k < hi) d[k] = k < v ? s[k] : uint16_t(0);
            }
        }
    }
}

// ------------------------------------------------------------------ rs_reduce

struct ReduceArgs {
    float* dst[PMAX];
    int64_t off[PMAX];
    int64_t valid[PMAX];         // n_{p,rank} * inner_p
    int32_t tile_start[PMAX];
    uint64_t dst_aligned;        // bit p: dst[p] 16-byte aligned
    const uint16_t* src;         // recv, source-major [W][S]
    int64_t chunk;
    int32_t world;
    int32_t nparams;
    int32_t ntiles;
};

__device__ __forceinline__ void add8(float (&acc)[8], uint4 x) {
    acc[0] += bf16_lo(x.x); acc[1] += bf16_hi(x.x);
    acc[2] += bf16_lo(x.y); acc[3] += bf16_hi(x.y);
    acc[4] += bf16_lo(x.z); acc[5] += bf16_hi(x.z);
    acc[6] += bf16_lo(x.w); acc[7] += bf16_hi(x.w);
}

__device__ __forceinline__ void init8(float (&acc)[8], uint4 x) {
    acc[0] = bf16_lo(x.x); acc[1] = bf16_hi(x.x);
    acc[2] = bf16_lo(x.y); acc[3] = bf16_hi(x.y);
    acc[4] = bf16_lo(x.z); acc[5] = bf16_hi(x.z);
    acc[6] = bf16_lo(x.w); acc[7] = bf16_hi(x.w);
}

__device__ __forceinline__ void store_avg8(float* d, const float (&acc)[8], float wf) {
    stf16(d, make_float4(acc[0] / wf, acc[1] / wf, acc[2] / wf, acc[3] / wf));
    stf16(d + 4, make_float4(acc[4] / wf, acc[5] / wf, acc[6] / wf, acc[7] / wf));
}

// Loads of sources i0 .. i0+kReduceBatch-1 (those below W unless kFull) of a
// full tile; all are issued before any of them is used.
template <bool kFull>
__device__ __forceinline__ void load_sources(uint4 (&x)[kReduceBatch][kReduceSteps], const uint16_t* tile,
                                             int i0, int W, int64_t S, uint32_t t) {
    constexpr uint32_t kStride = uint32_t(kReduceBlock) * kVec;
#pragma unroll
    for (int b = 0; b < kReduceBatch; ++b) {
        if (kFull || i0 + b < W) {
            const uint16_t* src = tile + int64_t(i0 + b) * S;
#pragma unroll
            for (int u = 0; u < kReduceSteps; ++u) x[b][u] = ld16(src + t + u * kStride);
        }
    }
}

// A full tile: kReduceSteps groups of 8 outputs per thread, spaced kReduceBlock*kVec
// apart.  `tile` is the wave-uniform start of the tile in rank 0's chunk.  The
// W sources of every output are added in rank order 0..W-1, starting from
// source 0; the loads of kReduceBatch sources are issued ahead of their adds.
__device__ __forceinline__ void reduce_tile_vec(const uint16_t* __restrict__ tile, float* __restrict__ dtile,
                                                int W, int64_t S, float wf) {
    constexpr uint32_t kStride = uint32_t(kReduceBlock) * kVec;
    const uint32_t t = threadIdx.x * kVec;
    float acc[kReduceSteps][8];
    uint4 x[kReduceBatch][kReduceSteps];
    if (W >= kReduceBatch) load_sources<true>(x, tile, 0, W, S, t);
    else load_sources<false>(x, tile, 0, W, S, t);
#pragma unroll
    for (int u = 0; u < kReduceSteps; ++u) init8(acc[u], x[0][u]);
#pragma unroll
    for (int b = 1; b < kReduceBatch; ++b)
        if (b < W) {
#pragma unroll
            for (int u = 0; u < kReduceSteps; ++u) add8(acc[u], x[b][u]);
        }
    int i = kReduceBatch;
    for (; i + kReduceBatch <= W; i += kReduceBatch) {
        load_sources<true>(x, tile, i, W, S, t);
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b)
#pragma unroll
            for (int u = 0; u < kReduceSteps; ++u) add8(acc[u], x[b][u]);
    }
    if (i < W) {
        load_sources<false>(x, tile, i, W, S, t);
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b)
            if (i + b < W) {
#pragma unroll
                for (int u = 0; u < kReduceSteps; ++u) add8(acc[u], x[b][u]);
            }
    }
#pragma unroll
    for (int u = 0; u < kReduceSteps; ++u) store_avg8(dtile + t + u * kStride, acc[u], wf);
}

__global__ void __launch_bounds__(kReduceBlock) rs_reduce_kernel(const ReduceArgs a) {
    const int lane = threadIdx.x & 63;
    const int my_start = lane < a.nparams ? a.tile_start[lane] : INT_MAX;
    const int W = a.world;
    const float wf = float(W);
    const int64_t S = a.chunk;
    for (int t = blockIdx.x; t < a.ntiles; t += gridDim.x) {
        const int p = param_of_tile(my_start, t);
        const int64_t v = a.valid[p];
        const int64_t lo = int64_t(t - a.tile_start[p]) * kReduceTile;
        const uint16_t* __restrict__ s0 = a.src + a.off[p];
        float* __restrict__ d0 = a.dst[p];
        const bool vec = ((a.dst_aligned >> p) & 1) && ((a.off[p] | S) & (kVec - 1)) == 0;
        if (vec && lo + kReduceTile <= v) {
            reduce_tile_vec(s0 + lo, d0 + lo, W, S, wf);
            continue;
        }
        for (int u = 0; u < kReduceSteps; ++u) {
            const int64_t g = lo + (int64_t(u) * kReduceBlock + threadIdx.x) * kVec;
            if (g >= v) break;
            const uint16_t* __restrict__ s = s0 + g;
            float* __restrict__ d = d0 + g;
            if (vec && g + kVec <= v) {
                float acc[8];
                init8(acc, ld16(s));
                for (int i = 1; i < W; ++i) add8(acc, ld16(s + int64_t(i) * S));
                store_avg8(d, acc, wf);
                continue;
            }
            for (int e = 0; e < kVec; ++e) {
                if (g + e >= v) break;
                float acc = bf16_lo(s[e]);
                for (int i = 1; i < W; ++i) acc += bf16_lo(s[int64_t(i) * S + e]);
                d[e] = acc / wf;
            }
        }
    }
}

// ------------------------------------------------------------------ host side

int cu_count(fsdp_status* st) {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        *st = fail(FSDP_ERR_HIP, "hipGetDevice failed");
        return 0;
    }
    if (dev >= 0 && dev < 64) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
        *st = fail(FSDP_ERR_HIP, "hipDeviceGetAttribute(multiProcessorCount) failed");
        return 0;
    }
    if (dev >= 0 && dev < 64) cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

struct Span {
    uintptr_t lo, hi;   // [lo, hi) bytes
    int id;             // -1: the bucket buffer, else the parameter index
};

bool overlaps(const Span& x, const Span& y) { return x.lo < y.hi && y.lo < x.hi; }

// Outputs must be pairwise disjoint and disjoint from every input.
fsdp_status check_overlap(std::vector<Span> outs, const std::vector<Span>& ins) {
    std::sort(outs.begin(), outs.end(), [](const Span& a, const Span& b) { return a.lo < b.lo; });
    for (size_t k = 1; k < outs.size(); ++k)
        if (outs[k].lo < outs[k - 1].hi) return fail(FSDP_ERR_OVERLAP, "two outputs overlap");
    for (const Span& in : ins) {
        // first output ending after in.lo
        auto it = std::upper_bound(outs.begin(), outs.end(), in.lo,
                                   [](uintptr_t v, const Span& s) { return v < s.hi; });
        if (it != outs.end() && overlaps(*it, in)) return fail(FSDP_ERR_OVERLAP, "an output overlaps an input");
    }
    return FSDP_OK;
}

fsdp_status check_bucket_ptr(const void* ptr, int64_t elems, const char* name) {
    if (elems > 0 && ptr == nullptr) return fail(FSDP_ERR_INVALID, std::string(name) + " is NULL");
    if ((reinterpret_cast<uintptr_t>(ptr) & 15) != 0)
        return fail(FSDP_ERR_ALIGN, std::string(name) + " is not 16-byte aligned");
    return FSDP_OK;
}

fsdp_status check_param_ptr(const void* ptr, int64_t elems, int elem_bytes, int p, const char* what) {
    if (elems > 0 && ptr == nullptr)
        return fail(FSDP_ERR_INVALID, std::string(what) + "[" + std::to_string(p) + "] is NULL");
    if ((reinterpret_cast<uintptr_t>(ptr) & uintptr_t(elem_bytes - 1)) != 0)
        return fail(FSDP_ERR_ALIGN, std::string(what) + "[" + std::to_string(p) + "] is not element-aligned");
    return FSDP_OK;
}

const Plan* get_plan(const fsdp_plan* h, fsdp_status* st) {
    const Plan* pl = plan_of(h);
    if (!pl) *st = fail(FSDP_ERR_INVALID, "unknown plan handle");
    return pl;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// One launch of `kernel` over `ntiles` work tiles (grid-stride beyond
// kBlocksPerCU workgroups per CU).  A 2-D launch passes grid.y and the tile
// count of its x dimension.
template <typename Args>
fsdp_status launch(void (*kernel)(const Args), const Args& args, int ntiles, int block, hipStream_t stream,
                   dim3 grid2 = dim3(0, 1), int xtiles = 0) {
    if (ntiles == 0) return FSDP_OK;
    fsdp_status st = FSDP_OK;
    const int cus = cu_count(&st);
    if (st != FSDP_OK) return st;
    const dim3 grid = grid2.y > 1 || xtiles > 0
                          ? dim3(std::min(xtiles, cus * kBlocksPerCU), grid2.y)
                          : dim3(std::min(ntiles, cus * kBlocksPerCU));
    void* kargs[] = {const_cast<Args*>(&args)};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, dim3(block),
                                         kargs, 0, stream);
    if (e != hipSuccess) return fail(FSDP_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e));
    return FSDP_OK;
}

int32_t tiles(int64_t n, int64_t tile) { return int32_t((n + tile - 1) / tile); }

}  // namespace
}  // namespace fsdp

using namespace fsdp;

extern "C" fsdp_status fsdp_ag_pack(const fsdp_plan* h, int32_t rank, const float* const* shards,
                                    uint16_t* send_chunk, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (rank < 0 || rank >= pl->world) return fail(FSDP_ERR_INVALID, "rank out of range");
    if (shards == nullptr) return fail(FSDP_ERR_INVALID, "shards is NULL");
    if ((st = check_bucket_ptr(send_chunk, pl->chunk, "send_chunk")) != FSDP_OK) return st;
    PackArgs a{};
    std::vector<Span> ins;
    int32_t nt = 0, max_tiles = 0;
    for (int p = 0; p < pl->nparams; ++p) {
        const int64_t v = pl->local_elems(p, rank);
        if ((st = check_param_ptr(shards[p], v, 4, p, "shards")) != FSDP_OK) return st;
        a.src[p] = shards[p];
        a.off[p] = pl->off[p];
        a.valid[p] = v;
        a.tile_start[p] = nt;
        nt += tiles(pl->off[p + 1] - pl->off[p], kPackTile);
        max_tiles = std::max(max_tiles, tiles(pl->off[p + 1] - pl->off[p], kPackTile));
        if (aligned16(shards[p]) && (pl->off[p] & (kVec - 1)) == 0) a.vec_mask |= uint64_t(1) << p;
        if (v > 0) ins.push_back({uintptr_t(shards[p]), uintptr_t(shards[p] + v), p});
    }
    a.off[pl->nparams] = pl->chunk;
    a.dst = send_chunk;
    a.nparams = pl->nparams;
    a.ntiles = nt;
    if (pl->chunk > 0 &&
        (st = check_overlap({{uintptr_t(send_chunk), uintptr_t(send_chunk + pl->chunk), -1}}, ins)) != FSDP_OK)
        return st;
    // the 2-D grid launches P * max_tiles workgroups for nt tiles of work
    if (int64_t(pl->nparams) * max_tiles <= kPackGridSlack * int64_t(nt))
        return launch(ag_pack_grid_kernel, a, nt, kCopyBlock, stream, dim3(0, pl->nparams), max_tiles);
    return launch(ag_pack_kernel, a, nt, kCopyBlock, stream);
}

extern "C" fsdp_status fsdp_ag_unpack(const fsdp_plan* h, const uint16_t* gathered, uint16_t* const* params,
                                      hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (params == nullptr) return fail(FSDP_ERR_INVALID, "params is NULL");
    const int64_t total = int64_t(pl->world) * pl->chunk;
    if ((st = check_bucket_ptr(gathered, total, "gathered")) != FSDP_OK) return st;
    UnpackArgs a{};
    std::vector<Span> outs;
    int32_t nt = 0;
    for (int p = 0; p < pl->nparams; ++p) {
        const int64_t e = pl->elems[p];
        if ((st = check_param_ptr(params[p], e, 2, p, "params")) != FSDP_OK) return st;
        a.dst[p] = params[p];
        a.off[p] = pl->off[p];
        a.seg[p] = pl->seg[p];
        a.elems[p] = e;
        a.tiles_per_seg[p] = tiles(pl->seg[p], kCopyTile);
        a.tile_start[p] = nt;
        nt += pl->world * a.tiles_per_seg[p];
        if (aligned16(params[p])) a.dst_aligned |= uint64_t(1) << p;
        if (e > 0) outs.push_back({uintptr_t(params[p]), uintptr_t(params[p] + e), p});
    }
    a.src = gathered;
    a.chunk = pl->chunk;
    a.nparams = pl->nparams;
    a.ntiles = nt;
    std::vector<Span> ins;
    if (total > 0) ins.push_back({uintptr_t(gathered), uintptr_t(gathered + total), -1});
    if ((st = check_overlap(outs, ins)) != FSDP_OK) return st;
    return launch(ag_unpack_kernel, a, nt, kCopyBlock, stream);
}

extern "C" fsdp_status fsdp_rs_pack(const fsdp_plan* h, const uint16_t* const* grads, uint16_t* send_buf,
                                    hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (grads == nullptr) return fail(FSDP_ERR_INVALID, "grads is NULL");
    const int64_t total = int64_t(pl->world) * pl->chunk;
    if ((st = check_bucket_ptr(send_buf, total, "send_buf")) != FSDP_OK) return st;
    RsPackArgs a{};
    std::vector<Span> ins;
    int32_t nt = 0;
    for (int p = 0; p < pl->nparams; ++p) {
        const int64_t e = pl->elems[p];
        if ((st = check_param_ptr(grads[p], e, 2, p, "grads")) != FSDP_OK) return st;
        a.src[p] = grads[p];
        a.off[p] = pl->off[p];
        a.seg[p] = pl->seg[p];
        a.elems[p] = e;
        a.tiles_per_seg[p] = tiles(pl->off[p + 1] - pl->off[p], kCopyTile);
        a.tile_start[p] = nt;
        nt += pl->world * a.tiles_per_seg[p];
        if (aligned16(grads[p])) a.src_aligned |= uint64_t(1) << p;
        if (e > 0) ins.push_back({uintptr_t(grads[p]), uintptr_t(grads[p] + e), p});
    }
    a.off[pl->nparams] = pl->chunk;
    a.dst = send_buf;
    a.chunk = pl->chunk;
    a.nparams = pl->nparams;
    a.ntiles = nt;
    if (total > 0 &&
        (st = check_overlap({{uintptr_t(send_buf), uintptr_t(send_buf + total), -1}}, ins)) != FSDP_OK)
        return st;
    return launch(rs_pack_kernel, a, nt, kCopyBlock, stream);
}

extern "C" fsdp_status fsdp_rs_reduce(const fsdp_plan* h, int32_t rank, const uint16_t* recv,
                                      float* const* grad_shards, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (rank < 0 || rank >= pl->world) return fail(FSDP_ERR_INVALID, "rank out of range");
    if (grad_shards == nullptr) return fail(FSDP_ERR_INVALID, "grad_shards is NULL");
    const int64_t total = int64_t(pl->world) * pl->chunk;
    if ((st = check_bucket_ptr(recv, total, "recv")) != FSDP_OK) return st;
    ReduceArgs a{};
    std::vector<Span> outs;
    int32_t nt = 0;
    for (int p = 0; p < pl->nparams; ++p) {
        const int64_t v = pl->local_elems(p, rank);
        if ((st = check_param_ptr(grad_shards[p], v, 4, p, "grad_shards")) != FSDP_OK) return st;
        a.dst[p] = grad_shards[p];
        a.off[p] = pl->off[p];
        a.valid[p] = v;
        a.tile_start[p] = nt;
        nt += tiles(v, kReduceTile);
        if (aligned16(grad_shards[p])) a.dst_aligned |= uint64_t(1) << p;
        if (v > 0) outs.push_back({uintptr_t(grad_shards[p]), uintptr_t(grad_shards[p] + v), p});
    }
    a.src = recv;
    a.chunk = pl->chunk;
    a.world = pl->world;
    a.nparams = pl->nparams;
    a.ntiles = nt;
    std::vector<Span> ins;
    if (total > 0) ins.push_back({uintptr_t(recv), uintptr_t(recv + total), -1});
    if ((st = check_overlap(outs, ins)) != FSDP_OK) return st;
    return launch(rs_reduce_kernel, a, nt, kReduceBlock, stream);
}
