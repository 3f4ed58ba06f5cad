// gfx950 kernels and C-ABI entry points of the bucketed FSDP copy path.
//
// All kernels are HBM-bound streams (no contraction, so no MFMA): one launch
// covers every parameter of a bucket.  The work of a launch is cut into tiles
// that never cross a parameter (and, for the W-way copies, never cross one
// rank's segment of a parameter), so that a tile is a plain contiguous copy,
// cast or reduction with 16-byte vector accesses.  Tiles are numbered
// parameter by parameter; the first tile of every parameter is kept in one
// register per lane of a wavefront, and a ballot over it finds the parameter
// of any tile in O(1).  The per-parameter table travels in the kernel
// arguments: the pack and the reduce hold all of it in lanes (lane p holds
// parameter p's entries), the copies read the looked-up parameter's entries
// through the scalar cache.  Tile counts fit in 31 bits (the planner checks);
// grid-stride loops count in 64 bits so that the last step cannot overflow.
//
// A bucket buffer of W chunks is addressed either as one allocation (chunk i
// at base + i*stride) or through a table of W chunk pointers, so the same
// kernels can pull from or push to chunks that live in separate buffers (for
// an exchange fused with the copy: the chunks of the peers).
//
// Numerics (SimpleFSDP sections 3.2.1 and 4):
//   * fp32 -> bf16 is IEEE round-half-to-even on the 16 dropped bits (the
//     hardware conversion); NaN gives (bits >> 16) | 0x0040;
//   * bf16 -> fp32 is exact (append 16 zero bits); fp32 copies are bit copies;
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
#include <type_traits>

#include "plan_impl.h"

namespace fsdp {
namespace {

#ifndef FSDP_REDUCE_BATCH
#define FSDP_REDUCE_BATCH 4
#endif
#ifndef FSDP_BLOCKS_PER_CU
#define FSDP_BLOCKS_PER_CU 16384
#endif
#ifndef FSDP_XCD_RUN
#define FSDP_XCD_RUN 256
#endif
#ifndef FSDP_ANY_NEIGHBOUR
#define FSDP_ANY_NEIGHBOUR 1
#endif
#ifndef FSDP_NT_LOAD
#define FSDP_NT_LOAD 1
#endif
#ifndef FSDP_NT_STORE
#define FSDP_NT_STORE 1
#endif

constexpr int PMAX = FSDP_MAX_PARAMS;
constexpr int kMaxChunks = FSDP_MAX_CHUNKS;
// One parameter per lane of a wave64: the ballot lookup and the lane-held
// tables need every parameter's entry in one wavefront.
static_assert(PMAX <= 64, "the tile lookup holds one parameter per lane of a 64-wide wavefront");
static_assert(kCopyBlock % 64 == 0 && kPackBlock % 64 == 0 && kPackBigBlock % 64 == 0 && kReduceBlock % 128 == 0,
              "workgroups are whole wavefronts (the reduce's half-size tile included)");
constexpr int kReduceBatch = FSDP_REDUCE_BATCH;   // source ranks loaded before they are added
constexpr int kBlocksPerCU = FSDP_BLOCKS_PER_CU;  // workgroups per CU in the grid-stride launch
constexpr int kXcds = 8;                          // accelerator dies; workgroup b runs on die b % 8
constexpr int kXcdRun = FSDP_XCD_RUN;             // consecutive copy tiles dealt to one die
static_assert(kXcdRun >= 1, "a die takes at least one tile at a time");

// ------------------------------------------------------------------ device helpers

// fp32 -> bf16 with gfx950's packed conversion (v_cvt_pk_bf16_f32): IEEE
// round-half-to-even on the 16 dropped bits under the default rounding mode,
// subnormals kept, overflow to infinity; a NaN keeps its sign and top payload
// bits and gets the quiet bit, (bits >> 16) | 0x0040.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16x2_bits(float lo, float hi) {
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ uint32_t bf16_bits(float f) { return bf16x2_bits(f, 0.f) & 0xffffu; }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// IEEE binary16: the conversion instruction rounds to nearest even under the
// default mode, keeps subnormals and overflows to infinity; the way back is
// exact.
__device__ __forceinline__ uint32_t f16_bits(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(f));
}
__device__ __forceinline__ float f16_lo(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xffffu)));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
}

// Element formats a kernel reads or writes on a bucket wire.
constexpr int kF32 = 0;    // fp32, copied bit for bit
constexpr int kBF16 = 1;   // bf16
constexpr int kF16 = 2;    // IEEE binary16

// The exact fp32 value of the low / high 16-bit element of a word.
template <int kFrom>
__device__ __forceinline__ float widen_lo(uint32_t w) { return kFrom == kF16 ? f16_lo(w) : bf16_lo(w); }
template <int kFrom>
__device__ __forceinline__ float widen_hi(uint32_t w) { return kFrom == kF16 ? f16_hi(w) : bf16_hi(w); }

#ifndef FSDP_LDS_TABLE
#define FSDP_LDS_TABLE 0
#endif

#if FSDP_LDS_TABLE
// A measured alternative to reading the tile table from the kernel arguments:
// the first wave stages entries 0..63 (INT_MAX from n on) in LDS, and after a
// barrier every lane reads its entry there.
__device__ __forceinline__ int staged_entry(const int32_t* table, int n) {
    __shared__ int staged[64];
    if (threadIdx.x < 64) staged[threadIdx.x] = int(threadIdx.x) < n ? table[threadIdx.x] : INT_MAX;
    __syncthreads();
    return staged[threadIdx.x & 63];
}
#endif

// Parameter owning tile t: the last p with tile_start[p] <= t.  Every lane of
// the wave holds tile_start[lane] (INT_MAX past the last parameter).
__device__ __forceinline__ int param_of_tile(int my_start, int t) {
    const uint64_t m = __ballot(my_start <= t);
    return __builtin_amdgcn_readfirstlane(__popcll(m) - 1);
}

__device__ __forceinline__ bool is_aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// 16-byte accesses; streamed data bypasses cache retention (non-temporal).
__device__ __forceinline__ uint4 ld16(const void* p) {
    const u32x4* q = reinterpret_cast<const u32x4*>(p);
#if FSDP_NT_LOAD
    const u32x4 v = __builtin_nontemporal_load(q);
#else
    const u32x4 v = *q;
#endif
    return make_uint4(v.x, v.y, v.z, v.w);
}
// One 16-byte-aligned block.
__device__ __forceinline__ u32x4 ld_block(const u32x4* q) {
#if FSDP_NT_LOAD
    return __builtin_nontemporal_load(q);
#else
    return *q;
#endif
}

// Bytes [r, r + 16) of the 32 bytes v0 followed by v1 (0 < r < 16), joined
// with byte funnel shifts.
__device__ __forceinline__ uint4 join16(const u32x4& v0, const u32x4& v1, uint32_t r) {
    uint32_t w0, w1, w2, w3, w4;                      // the five words from word r / 4 on
    switch (r >> 2) {
        case 0: w0 = v0.x; w1 = v0.y; w2 = v0.z; w3 = v0.w; w4 = v1.x; break;
        case 1: w0 = v0.y; w1 = v0.z; w2 = v0.w; w3 = v1.x; w4 = v1.y; break;
        case 2: w0 = v0.z; w1 = v0.w; w2 = v1.x; w3 = v1.y; w4 = v1.z; break;
        default: w0 = v0.w; w1 = v1.x; w2 = v1.y; w3 = v1.z; w4 = v1.w; break;
    }
    const uint32_t b = r & 3u;                         // bytes into word r / 4
    return make_uint4(__builtin_amdgcn_alignbyte(w1, w0, b), __builtin_amdgcn_alignbyte(w2, w1, b),
                      __builtin_amdgcn_alignbyte(w3, w2, b), __builtin_amdgcn_alignbyte(w4, w3, b));
}

// 16 bytes from an address that is only 2-byte aligned (a segment of a dense
// bucket, A < 8): the aligned 16-byte block holding p, and when p is not
// 16-byte aligned the next one too, joined with byte funnel shifts.  Each of
// the two blocks holds at least one byte of [p, p + 16) and lies inside one
// 16-byte-aligned block, so it never reaches a page that [p, p + 16) does not.
__device__ __forceinline__ uint4 ld16_any(const void* p) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(p);
    const uint32_t r = uint32_t(a) & 15u;
    const u32x4* q = reinterpret_cast<const u32x4*>(a - r);
    const u32x4 v0 = ld_block(q);
    if (r == 0) return make_uint4(v0.x, v0.y, v0.z, v0.w);
    return join16(v0, ld_block(q + 1), r);
}

// Stores are non-temporal unless kNt is false: a chunk that other workgroups
// read back at once (the first half of a wide push) is stored through the cache.
template <bool kNt = bool(FSDP_NT_STORE)>
__device__ __forceinline__ void st16(void* p, uint4 v) {
    u32x4* q = reinterpret_cast<u32x4*>(p);
    const u32x4 w = {v.x, v.y, v.z, v.w};
    if constexpr (kNt) __builtin_nontemporal_store(w, q);
    else *q = w;
}
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint2 ld8(const void* p) {
    const u32x2* q = reinterpret_cast<const u32x2*>(p);
#if FSDP_NT_LOAD
    const u32x2 v = __builtin_nontemporal_load(q);
#else
    const u32x2 v = *q;
#endif
    return make_uint2(v.x, v.y);
}
template <bool kNt = bool(FSDP_NT_STORE)>
__device__ __forceinline__ void st8(void* p, uint2 v) {
    u32x2* q = reinterpret_cast<u32x2*>(p);
    const u32x2 w = {v.x, v.y};
    if constexpr (kNt) __builtin_nontemporal_store(w, q);
    else *q = w;
}
__device__ __forceinline__ float4 ld16f(const float* p) {
    const f32x4* q = reinterpret_cast<const f32x4*>(p);
#if FSDP_NT_LOAD
    const f32x4 v = __builtin_nontemporal_load(q);
#else
    const f32x4 v = *q;
#endif
    return make_float4(v.x, v.y, v.z, v.w);
}
template <bool kNt = bool(FSDP_NT_STORE)>
__device__ __forceinline__ void st16f(float* p, float4 v) {
    f32x4* q = reinterpret_cast<f32x4*>(p);
    const f32x4 w = {v.x, v.y, v.z, v.w};
    if constexpr (kNt) __builtin_nontemporal_store(w, q);
    else *q = w;
}

// ------------------------------------------------------------------ bucket chunk addressing

// One allocation holding W chunks, chunk i at base + i*stride bytes.
struct ContigChunks {
    char* base;
    int64_t stride;
    __device__ __forceinline__ char* at(int i) const { return base + int64_t(i) * stride; }
    __device__ __forceinline__ bool aligned() const { return ((uintptr_t(base) | uintptr_t(stride)) & 15) == 0; }
};

// Contiguous chunks seen as a typed tile pointer plus a stride in elements:
// chunk i of the tile at tile + i*stride.
template <typename T>
struct StridedTile {
    const T* tile;
    int64_t stride;
    __device__ __forceinline__ const T* at(int i) const { return tile + int64_t(i) * stride; }
};

// W chunks anywhere (up to kMaxChunks), chunk i at ptr[i]; the host checks
// that every chunk is 16-byte aligned.
struct TableChunks {
    char* ptr[kMaxChunks];
    __device__ __forceinline__ char* at(int i) const { return ptr[i]; }
    __device__ __forceinline__ bool aligned() const { return true; }
};

// ------------------------------------------------------------------ segment copy

// The block of the next lane (lane l gets lane l + 1's value; lane 63's
// result is not used): a DPP wave shift, run where every lane is active.
constexpr int kDppWaveShl1 = 0x130;   // DPP control: each lane reads lane + 1 of the wave
constexpr int kDppAllRows = 0xf;      // row and bank masks: every row and bank of the wave
__device__ __forceinline__ uint32_t next_lane(uint32_t v) {
    return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), kDppWaveShl1, kDppAllRows, kDppAllRows, false));
}
__device__ __forceinline__ u32x4 next_lane(const u32x4& v) {
    return u32x4{next_lane(v.x), next_lane(v.y), next_lane(v.z), next_lane(v.w)};
}

// d[k] = k < v ? s[k] : 0 for k in [lo, hi): one tile of kSteps steps of
// kCopyBlock threads x 8 elements, in 2-byte units (bf16, or the halves of
// fp32 words for a plain copy).  `vec`: s and d are 16-byte aligned at 0.
//
// When s + lo or d + lo is not 16-byte aligned (a dense bucket, A < 8), the
// 16-byte stores follow d's alignment grid and each is fed from s with one
// load per aligned source block (the next lane's block by DPP; see below).
// A tile stores the grid units that start in [lo, hi); its last one may run
// past hi into the next tile's elements (up to the segment's end e), and the
// next tile starts at the grid point where it ended, so no 16-byte unit is
// written in parts by two workgroups.  Only the segment's first elements
// before the grid (in its first tile) and a last unit cut by e are written
// element by element.
template <int kSteps>
__device__ __forceinline__ void seg_copy_any(const uint16_t* __restrict__ s, uint16_t* __restrict__ d, int64_t lo,
                                             int64_t hi, int64_t v, int64_t e) {
    const int64_t h = (8 - int64_t((reinterpret_cast<uintptr_t>(d + lo) >> 1) & 7)) & 7;
    const int64_t a = lo + h;                          // the first grid point at or after lo
    const int t = threadIdx.x;
    if (lo == 0 && t < 8) {                            // the segment's elements before the grid
        const int64_t k = t;
        if (k < min(a, hi)) d[k] = k < v ? s[k] : uint16_t(0);
    }
    const int64_t nu = hi > a ? (hi - a + kVec - 1) / kVec : 0;   // grid units starting in [a, hi)
    uint4 x[kSteps];
#if FSDP_ANY_NEIGHBOUR
    // Unit i reads source bytes [s + a + 16 i, + 16): offset r into its aligned
    // block, the same r for every unit.  For r != 0 it also needs the next
    // block, which is the block of unit i + 1, loaded by the next lane; that
    // block is taken from the next lane, so each block is loaded once.  Lane 63
    // of a wave, and a lane whose next unit is not loaded, load it themselves
    // (it holds bytes of the unit's own range, as in ld16_any).
    const uint32_t r = uint32_t(reinterpret_cast<uintptr_t>(s + a)) & 15u;
    const bool last_lane = (t & 63) == 63;
    u32x4 b0[kSteps], b1[kSteps];
    bool ok[kSteps], own[kSteps];
#pragma unroll
    for (int u = 0; u < kSteps; ++u) {
        const int64_t i = int64_t(u) * kCopyBlock + t;
        const int64_t g = a + i * kVec;
        ok[u] = i < nu && g + kVec <= v && g + kVec <= e;
        const bool next_ok = i + 1 < nu && g + 2 * kVec <= v && g + 2 * kVec <= e;
        own[u] = r != 0 && (last_lane || !next_ok);
        const u32x4* q = reinterpret_cast<const u32x4*>(reinterpret_cast<const char*>(s + g) - r);
        if (ok[u]) b0[u] = ld_block(q);
        if (ok[u] && own[u]) b1[u] = ld_block(q + 1);
    }
    if (r == 0) {
#pragma unroll
        for (int u = 0; u < kSteps; ++u) x[u] = make_uint4(b0[u].x, b0[u].y, b0[u].z, b0[u].w);
    } else {
#pragma unroll
        for (int u = 0; u < kSteps; ++u) {
            const u32x4 n = next_lane(b0[u]);
            if (ok[u]) x[u] = join16(b0[u], own[u] ? b1[u] : n, r);
        }
    }
#else
#pragma unroll
    for (int u = 0; u < kSteps; ++u) {
        const int64_t i = int64_t(u) * kCopyBlock + t;
        const int64_t g = a + i * kVec;
        if (i < nu && g + kVec <= v && g + kVec <= e) x[u] = ld16_any(s + g);
    }
#endif
#pragma unroll
    for (int u = 0; u < kSteps; ++u) {
        const int64_t i = int64_t(u) * kCopyBlock + t;
        const int64_t g = a + i * kVec;
        if (i >= nu) continue;
        if (g + kVec <= e) {
            if (g + kVec <= v) st16(d + g, x[u]);
            else if (g >= v) st16(d + g, make_uint4(0, 0, 0, 0));
            else for (int k = 0; k < kVec; ++k) d[g + k] = g + k < v ? s[g + k] : uint16_t(0);
        } else {                                       // the segment's last unit, cut by e
            for (int64_t k = g; k < e; ++k) d[k] = k < v ? s[k] : uint16_t(0);
        }
    }
}

// kAny: the launch has segments off the 16-byte grid, which take
// seg_copy_any; without it such a tile is copied element by element (the
// host picks kAny only when some segment needs it, so that the aligned
// kernels keep their own code).
// (vs, e): the segment's valid elements and its end, for seg_copy_any, whose
// units may run past hi.
template <int kSteps, bool kAny>
__device__ __forceinline__ void seg_copy(const uint16_t* __restrict__ s, uint16_t* __restrict__ d, int64_t lo,
                                         int64_t hi, int64_t v, bool vec, int64_t vs, int64_t e) {
    constexpr int64_t kTile = int64_t(kCopyBlock) * kVec * kSteps;
    if constexpr (kAny) {
        if (!vec) {
            seg_copy_any<kSteps>(s, d, lo, hi, vs, e);
            return;
        }
    }
    if (vec && hi - lo == kTile && (hi <= v || lo >= v)) {
        if (hi <= v) {
            uint4 x[kSteps];
#pragma unroll
            for (int u = 0; u < kSteps; ++u) x[u] = ld16(s + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec);
#pragma unroll
            for (int u = 0; u < kSteps; ++u) st16(d + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec, x[u]);
        } else {
#pragma unroll
            for (int u = 0; u < kSteps; ++u)
                st16(d + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec, make_uint4(0, 0, 0, 0));
        }
        return;
    }
    for (int u = 0; u < kSteps; ++u) {
        const int64_t g = lo + (int64_t(u) * kCopyBlock + threadIdx.x) * kVec;
        if (g >= hi) break;
        if (vec && g + kVec <= hi && (g + kVec <= v || g >= v)) {
            st16(d + g, g < v ? ld16(s + g) : make_uint4(0, 0, 0, 0));
            continue;
        }
        for (int e = 0; e < kVec; ++e) {
            const int64_t k = g + e;
            if (k >= hi) break;
            d[k] = k < v ? s[k] : uint16_t(0);
        }
    }
}

// As seg_copy, but 16-bit elements (bf16 or fp16, kFrom) in and their exact
// fp32 values out.  Each thread handles 4 elements per sub-step (8 bytes in,
// 16 bytes out), so that every load and store instruction of a wave covers
// one contiguous run.
template <int kSteps, int kFrom>
__device__ __forceinline__ void seg_widen(const uint16_t* __restrict__ s, float* __restrict__ d, int64_t lo,
                                          int64_t hi, int64_t v, bool vec) {
    constexpr int kSub = kSteps;
    constexpr int64_t kTile = int64_t(kCopyBlock) * 4 * kSub;
    if (vec && hi - lo == kTile && (hi <= v || lo >= v)) {
        if (hi <= v) {
            uint2 x[kSub];
#pragma unroll
            for (int u = 0; u < kSub; ++u) x[u] = ld8(s + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * 4);
#pragma unroll
            for (int u = 0; u < kSub; ++u)
                st16f(d + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * 4,
                      make_float4(widen_lo<kFrom>(x[u].x), widen_hi<kFrom>(x[u].x), widen_lo<kFrom>(x[u].y), widen_hi<kFrom>(x[u].y)));
        } else {
#pragma unroll
            for (int u = 0; u < kSub; ++u)
                st16f(d + lo + (int64_t(u) * kCopyBlock + threadIdx.x) * 4, make_float4(0.f, 0.f, 0.f, 0.f));
        }
        return;
    }
    for (int u = 0; u < kSub; ++u) {
        const int64_t g = lo + (int64_t(u) * kCopyBlock + threadIdx.x) * 4;
        if (g >= hi) break;
        if (vec && g + 4 <= hi && (g + 4 <= v || g >= v)) {
            const uint2 x = g < v ? ld8(s + g) : make_uint2(0, 0);
            st16f(d + g, make_float4(widen_lo<kFrom>(x.x), widen_hi<kFrom>(x.x),
                                      widen_lo<kFrom>(x.y), widen_hi<kFrom>(x.y)));
            continue;
        }
        for (int e = 0; e < 4; ++e) {
            const int64_t k = g + e;
            if (k >= hi) break;
            d[k] = k < v ? widen_lo<kFrom>(s[k]) : 0.f;
        }
    }
}

// ------------------------------------------------------------------ ag_pack

// One destination chunk (the rank's send chunk).
struct OneChunk {
    char* ptr;
    __device__ __forceinline__ char* at(int) const { return ptr; }
};

// Dst is OneChunk, or TableChunks when the packed chunk is pushed to W
// destinations (the peers' gathered buffers), each receiving the same bytes.
template <class Dst>
struct PackArgs {
    const float* src[PMAX];
    int64_t off[PMAX + 1];       // off[P] = S
    int64_t valid[PMAX];         // n_{p,rank} * inner_p
    int32_t tile_start[PMAX];    // first tile of parameter p; INT_MAX past the last parameter
    Dst dst;                     // bf16 or fp32 chunks of S elements
    int32_t ndst;                // destinations (1 for OneChunk)
    int32_t nparams;
    int32_t ntiles;
};

// One fp32 value -> its 16-bit pattern in format kOut (bf16 or fp16); four
// values -> four patterns packed in 8 bytes.
template <int kOut>
__device__ __forceinline__ uint32_t cast1(float f) { return kOut == kF16 ? f16_bits(f) : bf16_bits(f); }
template <int kOut>
__device__ __forceinline__ uint2 cast4(float4 a) {
    if constexpr (kOut == kBF16) return make_uint2(bf16x2_bits(a.x, a.y), bf16x2_bits(a.z, a.w));
    return make_uint2(cast1<kOut>(a.x) | (cast1<kOut>(a.y) << 16), cast1<kOut>(a.z) | (cast1<kOut>(a.w) << 16));
}

// The fields of the parameter a pack tile belongs to.
struct PackParam {
    const float* src;
    int64_t off;       // off_p
    int64_t region;    // off_{p+1} - off_p
    int64_t valid;     // n_{p,rank} * inner_p
};

// Lane-held argument tables.  Lane l of a wave loads entry l of each
// per-parameter table of the kernel arguments, every lane and table in one
// round of independent loads; from_lane then hands entry p to the whole wave.
// A kernel that takes its parameter's fields this way waits on one round trip
// to the argument table before its data loads, not on a chain of them (the
// tile table, then the entries of the parameter it names).  from_lane is only
// called where every lane of the wave is active, on values every lane wrote:
// a lane that is inactive when a value is computed keeps its old register,
// and readlane would return that.  The pack and the
// reduce use them.  The copies do not: their tiles are two 16-byte loads per
// lane, and the tables' extra vector loads per wave made them 3-5 % slower.
__device__ __forceinline__ int lane_index() { return int(threadIdx.x & 63); }
// The table entry a lane loads: its own, or the last one for the lanes past
// PMAX (none while PMAX is the wavefront width; their tile start is INT_MAX,
// so the lookup never selects them).
__device__ __forceinline__ int table_lane() { return min(lane_index(), PMAX - 1); }
__device__ __forceinline__ int32_t from_lane(int32_t v, int p) { return __builtin_amdgcn_readlane(v, p); }
__device__ __forceinline__ int64_t from_lane(int64_t v, int p) {
    const uint64_t u = uint64_t(v);
    const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u)), p));
    const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u >> 32)), p));
    return int64_t((uint64_t(hi) << 32) | lo);
}
// A pointer into device memory: the round trip through the global address
// space keeps its accesses global rather than flat instructions.
template <typename T>
__device__ __forceinline__ T* from_lane(T* v, int p) {
    typedef T __attribute__((address_space(1))) Global;
    return (T*)(Global*)(from_lane(reinterpret_cast<int64_t>(v), p));
}

// The pack's lane-held table: lane l holds parameter l's entries.
struct PackLane {
    int start;          // tile_start[lane]
    const float* src;
    int64_t off, end, valid;

    template <class Dst>
    __device__ __forceinline__ explicit PackLane(const PackArgs<Dst>& a) {
        const int l = table_lane();
#if FSDP_LDS_TABLE
        start = staged_entry(a.tile_start, PMAX);
#else
        start = lane_index() < PMAX ? a.tile_start[l] : INT_MAX;
#endif
        src = a.src[l];
        off = a.off[l];
        end = a.off[l + 1];
        valid = a.valid[l];
    }
    __device__ __forceinline__ PackParam param(int p) const {
        const int64_t o = from_lane(off, p);
        return PackParam{from_lane(src, p), o, from_lane(end, p) - o, from_lane(valid, p)};
    }
};

// Tile lt of parameter pp: its part of [off_p, off_{p+1}) of the chunk, the
// shard's values cast to bf16 or fp16 or copied as fp32 (kOut), zeros past the shard,
// written to every destination.  Each thread handles 4 elements per sub-step
// (16 bytes of fp32 in), so every load and store instruction of a wave covers
// one contiguous run; the full tiles of a 16-bit push take 8 per thread.
template <int kOut, class Dst, bool kNt = true, int kB = kPackBlock, int kS = kPackSteps>
__device__ __forceinline__ void pack_tile(const PackArgs<Dst>& a, const PackParam& pp, int lt) {
    constexpr int64_t kTile = int64_t(kB) * kVec * kS;
    constexpr bool kCast = kOut != kF32;
    typedef typename std::conditional<kCast, uint16_t, uint32_t>::type Out;
    constexpr int kSub = 2 * kS;
    constexpr bool kOne = std::is_same<Dst, OneChunk>::value;
    const int ndst = kOne ? 1 : a.ndst;
    const int64_t off = pp.off;
    const int64_t region = pp.region;
    const int64_t valid = pp.valid;
    const float* __restrict__ src = pp.src;
    const int64_t lo = int64_t(lt) * kTile;
    const int64_t hi = min(lo + kTile, region);
    if (lo >= hi) return;
    // every destination chunk is 16-byte aligned, so one test covers them all
    const bool vec = is_aligned16(src) && is_aligned16(reinterpret_cast<Out*>(a.dst.at(0)) + off);
    if constexpr (!kOne && kCast) {
        // Pushed to W destinations, the stores outnumber the loads W to 1:
        // each thread casts 8 consecutive elements and writes them with one
        // 16-byte store per destination.
        if (vec && hi - lo == kTile && lo + kTile <= valid) {
            uint4 y[kS];
#pragma unroll
            for (int u = 0; u < kS; ++u) {
                const float* s8 = src + lo + (int64_t(u) * kB + threadIdx.x) * 8;
                const uint2 c0 = cast4<kOut>(ld16f(s8));
                const uint2 c1 = cast4<kOut>(ld16f(s8 + 4));
                y[u] = make_uint4(c0.x, c0.y, c1.x, c1.y);
            }
            for (int j = 0; j < ndst; ++j) {
                Out* __restrict__ dst = reinterpret_cast<Out*>(a.dst.at(j)) + off;
#pragma unroll
                for (int u = 0; u < kS; ++u) st16<kNt>(dst + lo + (int64_t(u) * kB + threadIdx.x) * 8, y[u]);
            }
            return;
        }
    }
    if (vec && hi - lo == kTile && lo + kTile <= valid) {
        float4 x[kSub];
#pragma unroll
        for (int u = 0; u < kSub; ++u) x[u] = ld16f(src + lo + (int64_t(u) * kB + threadIdx.x) * 4);
        for (int j = 0; j < ndst; ++j) {
            Out* __restrict__ dst = reinterpret_cast<Out*>(a.dst.at(j)) + off;
#pragma unroll
            for (int u = 0; u < kSub; ++u) {
                const int64_t g = lo + (int64_t(u) * kB + threadIdx.x) * 4;
                if (kCast) st8<kNt>(dst + g, cast4<kOut>(x[u]));
                else st16f<kNt>(reinterpret_cast<float*>(dst + g), x[u]);
            }
        }
        return;
    }
    for (int u = 0; u < kSub; ++u) {
        const int64_t g = lo + (int64_t(u) * kB + threadIdx.x) * 4;
        if (g >= hi) break;
        if (vec && g + 4 <= hi && (g + 4 <= valid || g >= valid)) {
            const float4 x = g < valid ? ld16f(src + g) : make_float4(0.f, 0.f, 0.f, 0.f);
            for (int j = 0; j < ndst; ++j) {
                Out* __restrict__ dst = reinterpret_cast<Out*>(a.dst.at(j)) + off;
                if (kCast) st8<kNt>(dst + g, g < valid ? cast4<kOut>(x) : make_uint2(0, 0));
                else st16<kNt>(dst + g, g < valid ? make_uint4(__float_as_uint(x.x), __float_as_uint(x.y),
                                                          __float_as_uint(x.z), __float_as_uint(x.w))
                                             : make_uint4(0, 0, 0, 0));
            }
            continue;
        }
        for (int e = 0; e < 4; ++e) {
            const int64_t k = g + e;
            if (k >= hi) break;
            const Out v = k < valid ? Out(kCast ? cast1<kOut>(src[k]) : __float_as_uint(src[k])) : Out(0);
            for (int j = 0; j < ndst; ++j) (reinterpret_cast<Out*>(a.dst.at(j)) + off)[k] = v;
        }
    }
}

// Tiles numbered across the bucket; the parameter of a tile comes from the
// wave-ballot lookup.  The pack moves few bytes per launch, so its start-up
// chain is kept short: tile_start holds INT_MAX past the last parameter (no
// wait for the parameter count before the table load), the grid never exceeds
// the tile count (the first tile needs no bound check), and every field of
// the tile's parameter comes from the looked-up lane (PackLane), so the only
// wait before the data loads is the one round of table loads.  The big tile's
// registers are held to 64 so that 8 waves fit on each SIMD (the extra lane
// fields had cost one wave).  A tile is kB threads x kS steps of 8 elements.
template <int kOut, class Dst, int kB, int kS>
__global__ void __launch_bounds__(kB) __attribute__((amdgpu_waves_per_eu(8))) ag_pack_kernel(const PackArgs<Dst> a) {
    const PackLane lane(a);
    int64_t step = blockIdx.x;
    do {
        const int t = int(step);
        const int p = param_of_tile(lane.start, t);
        pack_tile<kOut, Dst, true, kB, kS>(a, lane.param(p), t - __builtin_amdgcn_readlane(lane.start, p));
        step += gridDim.x;
    } while (step < a.ntiles);
}

// The first half of a wide push: the rank's own chunk, stored through the
// cache so that the copies to the other destinations read it back from L2 and
// the MALL.  (Read back at once by many workgroups, a chunk just written with
// non-temporal stores streamed at little more than half the rate.)
template <int kOut>
__global__ void __launch_bounds__(kPackBlock) push_pack_kernel(const PackArgs<OneChunk> a) {
    const PackLane lane(a);
    int64_t step = blockIdx.x;
    do {
        const int t = int(step);
        const int p = param_of_tile(lane.start, t);
        pack_tile<kOut, OneChunk, false>(a, lane.param(p), t - __builtin_amdgcn_readlane(lane.start, p));
        step += gridDim.x;
    } while (step < a.ntiles);
}

// The second half of a wide push: chunk `from` copied to the other W - 1
// chunks of a table.  One work item is one tile of 16-byte units of one
// destination.  Workgroups are dealt to the 8 XCDs round-robin (workgroup b
// runs on XCD b mod 8; a grid-stride step is a multiple of 8), so the items are
// numbered to put all destinations of a tile on one XCD: the tile is read into
// that XCD's L2 once (cached loads) and written to each destination
// (non-temporal stores), each workgroup writing one contiguous run.
//
// From kRepGroup destinations up, they are copied in groups of kRepGroup,
// one group per grid row (blockIdx.y).  Workgroups are dispatched row by row,
// so the workgroups in flight write long runs into few destinations instead
// of short runs into all W - 1; the chunk is read once per group.
#ifndef FSDP_PUSH_REPLICATE_MIN_W
#define FSDP_PUSH_REPLICATE_MIN_W 8
#endif
constexpr int64_t kRepTile = kCopyBlock;          // 16-byte units per tile (2 KB)
constexpr int kReplicateMinW = FSDP_PUSH_REPLICATE_MIN_W;
constexpr int kRepGroupLog2 = 4;
constexpr int kRepGroup = 1 << kRepGroupLog2;     // destinations per grid row

struct ReplicateArgs {
    TableChunks dst;
    int64_t units;        // whole 16-byte units of a chunk
    int32_t tail;         // 2-byte elements after them
    int32_t from;         // the source chunk
    int32_t ndst;         // W - 1 destinations
    int32_t ntiles;
    int32_t nitems;
};

// Tile t of the source to destination index j (0 .. ndst-1, skipping `from`).
__device__ __forceinline__ void replicate_tile(const ReplicateArgs& a, const u32x4* __restrict__ src, int t, int j) {
    j += j >= a.from;                                // every chunk but the source
    u32x4* __restrict__ d = reinterpret_cast<u32x4*>(a.dst.ptr[j]);
    const int64_t g = int64_t(t) * kRepTile + threadIdx.x;
    if (g < a.units) {
        __builtin_nontemporal_store(src[g], d + g);
    } else if (g == a.units && a.tail > 0) {         // one thread copies the partial unit
        const uint16_t* s2 = reinterpret_cast<const uint16_t*>(src + a.units);
        uint16_t* d2 = reinterpret_cast<uint16_t*>(d + a.units);
        for (int e = 0; e < a.tail; ++e) d2[e] = s2[e];
    }
}

// Fewer than kRepGroup destinations: item i is tile round (i / 8) / ndst,
// destination (i / 8) mod ndst.
__global__ void __launch_bounds__(kCopyBlock) replicate_kernel(const ReplicateArgs a) {
    const u32x4* __restrict__ src = reinterpret_cast<const u32x4*>(a.dst.ptr[a.from]);
    for (int64_t step = blockIdx.x; step < a.nitems; step += gridDim.x) {
        const int i = int(step);
        const int k = i / kXcds;
        const int t = (k / a.ndst) * kXcds + i % kXcds;
        if (t >= a.ntiles) continue;
        replicate_tile(a, src, t, k % a.ndst);
    }
}

// kRepGroup destinations or more: row blockIdx.y holds destinations
// y*kRepGroup .. y*kRepGroup + kRepGroup - 1 (the last row may be short);
// item i of a row is tile round (i / 8) / kRepGroup.  `nitems` counts one row.
__global__ void __launch_bounds__(kCopyBlock) replicate_grouped_kernel(const ReplicateArgs a) {
    const u32x4* __restrict__ src = reinterpret_cast<const u32x4*>(a.dst.ptr[a.from]);
    for (int64_t step = blockIdx.x; step < a.nitems; step += gridDim.x) {
        const int i = int(step);
        const int k = i >> 3;
        const int t = ((k >> kRepGroupLog2) << 3) + (i & 7);
        const int j = int(blockIdx.y) * kRepGroup + (k & (kRepGroup - 1));
        if (t >= a.ntiles || j >= a.ndst) continue;
        replicate_tile(a, src, t, j);
    }
}

// ------------------------------------------------------------------ copy tile order

// The copy tile of workgroup-order index b.  Workgroups are dealt to the 8
// dies (XCDs) round-robin, so in tile order b each die would take every 8th
// 4 KB tile.  Instead, within each group of 8 * kXcdRun tiles, the workgroups
// of one die (b, b + 8, b + 16, ...) take kXcdRun consecutive tiles, a 1 MB
// run per die (1.4 % faster rs_pack and 1 % faster unpack on the 70B block,
// 1-3 % on the other Llama blocks and the uneven bucket; runs of 16 tiles
// were 8 % slower, and the reduce gained nothing from such an order); the
// tiles past the last whole group keep order b.  A bijection
// on [0, n), so a grid-stride loop over b still covers every tile once.
__device__ __forceinline__ int copy_tile(int64_t b, int n) {
    constexpr int64_t kGroup = int64_t(kXcds) * kXcdRun;
    if (b >= int64_t(n) / kGroup * kGroup) return int(b);
    const int64_t r = b % kGroup;
    return int(b - r + (r % kXcds) * kXcdRun + r / kXcds);
}

// ------------------------------------------------------------------ ag_unpack

// Sizes in 2-byte units (an fp32 element is two units).
template <class Chunks>
struct UnpackArgs {
    uint16_t* dst[PMAX];
    int64_t off[PMAX];
    int64_t seg[PMAX];           // L_p
    int64_t elems[PMAX];         // N_p * inner_p
    int32_t tiles_per_seg[PMAX]; // ceil(L_p / tile)
    int32_t tile_start[PMAX];
    Chunks src;                  // gathered chunks, one per source rank
    int32_t nparams;
    int32_t ntiles;
};

template <class Chunks, bool kAny>
__global__ void __launch_bounds__(kCopyBlock) ag_unpack_kernel(const UnpackArgs<Chunks> a) {
    const int lane = threadIdx.x & 63;
#if FSDP_LDS_TABLE
    const int my_start = staged_entry(a.tile_start, a.nparams);
#else
    const int my_start = lane < a.nparams ? a.tile_start[lane] : INT_MAX;
#endif
    for (int64_t step = blockIdx.x; step < a.ntiles; step += gridDim.x) {
        const int t = copy_tile(step, a.ntiles);
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
        const uint16_t* s = reinterpret_cast<const uint16_t*>(a.src.at(i)) + a.off[p];
        uint16_t* d = a.dst[p] + int64_t(i) * L;
        seg_copy<kCopySteps, kAny>(s, d, lo, hi, hi, is_aligned16(s) && is_aligned16(d), v, v);
    }
}

// ------------------------------------------------------------------ rs_pack

// Sizes in units of the source gradient: 2-byte units for a plain copy, 16-bit
// elements when kWiden (kBF16 or kF16; kF32 = no widening) casts them to an
// fp32 wire.  Tiles are numbered parameter by parameter and, within a
// parameter, destination by destination; for W above kDestMajorW they are
// numbered destination by destination and, within a destination, parameter by
// parameter, so that the workgroups running at one time write one destination
// chunk front to front instead of the segments of many chunks at once.
constexpr int kDestMajorW = 64;

template <class Chunks>
struct RsPackArgs {
    const uint16_t* src[PMAX];   // full gradients
    int64_t off[PMAX + 1];       // off[P] = S
    int64_t seg[PMAX];
    int64_t elems[PMAX];
    int32_t tiles_per_seg[PMAX]; // ceil((off_{p+1} - off_p) / tile)
    int32_t tile_start[PMAX];    // first tile of parameter p (within one destination if dest_major)
    Chunks dst;                  // send chunks, one per destination rank
    int32_t nparams;
    int32_t dest_major;
    int32_t tiles_per_dest;      // tiles of one destination chunk
    int32_t ntiles;              // W * tiles_per_dest
};

template <class Chunks, int kWiden, bool kAny>
__global__ void __launch_bounds__(kCopyBlock) rs_pack_kernel(const RsPackArgs<Chunks> a) {
    const int lane = threadIdx.x & 63;
#if FSDP_LDS_TABLE
    const int my_start = staged_entry(a.tile_start, a.nparams);
#else
    const int my_start = lane < a.nparams ? a.tile_start[lane] : INT_MAX;
#endif
    for (int64_t step = blockIdx.x; step < a.ntiles; step += gridDim.x) {
        const int t = copy_tile(step, a.ntiles);
        int p, j;                                        // parameter, destination rank
        int64_t st;                                      // tile within the segment
        if (a.dest_major) {
            j = t / a.tiles_per_dest;
            const int r = t - j * a.tiles_per_dest;
            p = param_of_tile(my_start, r);
            st = r - a.tile_start[p];
        } else {
            p = param_of_tile(my_start, t);
            const int lt = t - a.tile_start[p];
            j = lt / a.tiles_per_seg[p];
            st = lt - int64_t(j) * a.tiles_per_seg[p];
        }
        const int64_t region = a.off[p + 1] - a.off[p];
        const int64_t L = a.seg[p];
        const int64_t rest = a.elems[p] - int64_t(j) * L;
        const int64_t v = rest < L ? (rest > 0 ? rest : 0) : L;
        constexpr int64_t kTile = kWiden != kF32 ? kWidenTile : kCopyTile;
        const int64_t lo = st * kTile;
        const int64_t hi = min(lo + kTile, region);
        const uint16_t* s = a.src[p] + int64_t(j) * L;
        if constexpr (kWiden != kF32) {
            float* d = reinterpret_cast<float*>(a.dst.at(j)) + a.off[p];
            seg_widen<kCopySteps, kWiden>(s, d, lo, hi, v, is_aligned16(s) && is_aligned16(d));
        } else {
            uint16_t* d = reinterpret_cast<uint16_t*>(a.dst.at(j)) + a.off[p];
            seg_copy<kCopySteps, kAny>(s, d, lo, hi, v, is_aligned16(s) && is_aligned16(d), v, region);
        }
    }
}

// ------------------------------------------------------------------ rs_reduce

template <class Chunks>
struct ReduceArgs {
    float* dst[PMAX];
    int64_t off[PMAX];
    int64_t valid[PMAX];         // n_{p,rank} * inner_p
    int32_t tile_start[PMAX];    // first tile of parameter p; INT_MAX past the last parameter
    Chunks src;                  // received chunks, one per source rank
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

// One thread's 8 values of a tile row (kB * 8 elements, kB threads) of one
// source, as loaded.  bf16 sources: elements [8t, 8t+8) of the row, one
// 16-byte load.  fp32 sources: elements [4t, 4t+4) and [4kB + 4t, 4kB + 4t + 4),
// two 16-byte loads that each cover one contiguous run across the wave.
// Addresses are a wave-uniform row pointer plus a 32-bit byte offset.
template <typename T, int kB> struct Raw8;
template <int kB> struct Raw8<uint16_t, kB> {
    uint4 x;
    __device__ __forceinline__ static uint32_t pos(uint32_t t, int e) { return t * 8 + e; }
    __device__ __forceinline__ void load(const uint16_t* row, uint32_t t) { x = ld16(row + t * 8); }
    __device__ __forceinline__ void load_any(const uint16_t* row, uint32_t t) { x = ld16_any(row + t * 8); }
    __device__ __forceinline__ void init(float (&acc)[8]) const { init8(acc, x); }
    __device__ __forceinline__ void add(float (&acc)[8]) const { add8(acc, x); }
};
template <int kB> struct Raw8<_Float16, kB> {
    uint4 x;
    __device__ __forceinline__ static uint32_t pos(uint32_t t, int e) { return t * 8 + e; }
    __device__ __forceinline__ void load(const _Float16* row, uint32_t t) { x = ld16(row + t * 8); }
    __device__ __forceinline__ void load_any(const _Float16* row, uint32_t t) { x = ld16_any(row + t * 8); }
    __device__ __forceinline__ void init(float (&acc)[8]) const {
        acc[0] = f16_lo(x.x); acc[1] = f16_hi(x.x); acc[2] = f16_lo(x.y); acc[3] = f16_hi(x.y);
        acc[4] = f16_lo(x.z); acc[5] = f16_hi(x.z); acc[6] = f16_lo(x.w); acc[7] = f16_hi(x.w);
    }
    __device__ __forceinline__ void add(float (&acc)[8]) const {
        acc[0] += f16_lo(x.x); acc[1] += f16_hi(x.x); acc[2] += f16_lo(x.y); acc[3] += f16_hi(x.y);
        acc[4] += f16_lo(x.z); acc[5] += f16_hi(x.z); acc[6] += f16_lo(x.w); acc[7] += f16_hi(x.w);
    }
};
template <int kB> struct Raw8<float, kB> {
    float4 a, b;
    __device__ __forceinline__ static uint32_t pos(uint32_t t, int e) {
        return e < 4 ? t * 4 + e : uint32_t(kB) * 4 + t * 4 + (e - 4);
    }
    __device__ __forceinline__ void load(const float* row, uint32_t t) {
        a = ld16f(row + t * 4);
        b = ld16f(row + uint32_t(kB) * 4 + t * 4);
    }
    __device__ __forceinline__ void load_any(const float* row, uint32_t t) {
        const uint4 u = ld16_any(row + t * 4);
        const uint4 w = ld16_any(row + uint32_t(kB) * 4 + t * 4);
        a = make_float4(__uint_as_float(u.x), __uint_as_float(u.y), __uint_as_float(u.z), __uint_as_float(u.w));
        b = make_float4(__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z), __uint_as_float(w.w));
    }
    __device__ __forceinline__ void init(float (&acc)[8]) const {
        acc[0] = a.x; acc[1] = a.y; acc[2] = a.z; acc[3] = a.w;
        acc[4] = b.x; acc[5] = b.y; acc[6] = b.z; acc[7] = b.w;
    }
    __device__ __forceinline__ void add(float (&acc)[8]) const {
        acc[0] += a.x; acc[1] += a.y; acc[2] += a.z; acc[3] += a.w;
        acc[4] += b.x; acc[5] += b.y; acc[6] += b.z; acc[7] += b.w;
    }
};

// Store the 8 averages of thread t at the positions Raw8<T, kB>::pos gives.
template <typename T, int kB>
__device__ __forceinline__ void store_avg8(float* row, uint32_t t, const float (&acc)[8], float wf) {
    const float4 lo = make_float4(acc[0] / wf, acc[1] / wf, acc[2] / wf, acc[3] / wf);
    const float4 hi = make_float4(acc[4] / wf, acc[5] / wf, acc[6] / wf, acc[7] / wf);
    st16f(row + Raw8<T, kB>::pos(t, 0), lo);
    st16f(row + Raw8<T, kB>::pos(t, 4), hi);
}

// Typed pointer to the tile of source i: through the chunk table, or as a
// strided tile of one contiguous buffer.
template <typename T>
__device__ __forceinline__ const T* source(const TableChunks& c, int64_t off, int i) {
    return reinterpret_cast<const T*>(c.at(i)) + off;
}
template <typename T>
__device__ __forceinline__ const T* source(const StridedTile<T>& c, int64_t off, int i) {
    return c.at(i) + off;
}

// Loads of sources i0 .. i0+kReduceBatch-1 (those below W unless kFull) of a
// full tile; all are issued before any of them is used.  `off` is the tile's
// element offset inside every chunk.  kAny: the sources are not 16-byte
// aligned there (a dense bucket), so each 16 bytes come from ld16_any.
template <bool kFull, bool kAny, typename T, int kB, class Src>
__device__ __forceinline__ void load_sources(Raw8<T, kB> (&x)[kReduceBatch][kReduceSteps], const Src& src,
                                             int64_t off, int i0, int W, uint32_t t) {
    constexpr uint32_t kRow = uint32_t(kB) * kVec;
#pragma unroll
    for (int b = 0; b < kReduceBatch; ++b) {
        if (kFull || i0 + b < W) {
            const T* s = source<T>(src, off, i0 + b);
#pragma unroll
            for (int u = 0; u < kReduceSteps; ++u) {
                if constexpr (kAny) x[b][u].load_any(s + u * kRow, t);
                else x[b][u].load(s + u * kRow, t);
            }
        }
    }
}

// A full tile of kReduceSteps rows.  The W sources of every output are added
// in rank order 0..W-1, starting from source 0; the loads of kReduceBatch
// sources are issued ahead of their adds.
template <typename T, int kB, bool kAny, class Src>
__device__ __forceinline__ void reduce_tile_vec(const Src& src, int64_t off, float* __restrict__ dtile,
                                                int W, float wf) {
    constexpr uint32_t kRow = uint32_t(kB) * kVec;
    const uint32_t t = threadIdx.x;
    float acc[kReduceSteps][8];
    Raw8<T, kB> x[kReduceBatch][kReduceSteps];
    if (W >= kReduceBatch) load_sources<true, kAny>(x, src, off, 0, W, t);
    else load_sources<false, kAny>(x, src, off, 0, W, t);
#pragma unroll
    for (int u = 0; u < kReduceSteps; ++u) x[0][u].init(acc[u]);
#pragma unroll
    for (int b = 1; b < kReduceBatch; ++b)
        if (b < W) {
#pragma unroll
            for (int u = 0; u < kReduceSteps; ++u) x[b][u].add(acc[u]);
        }
    int i = kReduceBatch;
    for (; i + kReduceBatch <= W; i += kReduceBatch) {
        load_sources<true, kAny>(x, src, off, i, W, t);
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b)
#pragma unroll
            for (int u = 0; u < kReduceSteps; ++u) x[b][u].add(acc[u]);
    }
    if (i < W) {
        load_sources<false, kAny>(x, src, off, i, W, t);
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b)
            if (i + b < W) {
#pragma unroll
                for (int u = 0; u < kReduceSteps; ++u) x[b][u].add(acc[u]);
            }
    }
    if constexpr (sizeof(T) == 2) {
        // Thread t holds outputs [8t, 8t + 8) of each row: staged through LDS
        // so that every store instruction of a wave covers one contiguous run.
        __shared__ float4 stage[kReduceSteps * kB * 2];
#pragma unroll
        for (int u = 0; u < kReduceSteps; ++u) {
            stage[(u * kB + t) * 2] = make_float4(acc[u][0] / wf, acc[u][1] / wf, acc[u][2] / wf, acc[u][3] / wf);
            stage[(u * kB + t) * 2 + 1] = make_float4(acc[u][4] / wf, acc[u][5] / wf, acc[u][6] / wf, acc[u][7] / wf);
        }
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kReduceSteps; ++u)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                st16f(dtile + u * kRow + (h * kB + t) * 4, stage[u * kB * 2 + h * kB + t]);
        __syncthreads();
        return;
    }
#pragma unroll
    for (int u = 0; u < kReduceSteps; ++u) store_avg8<T, kB>(dtile + u * kRow, t, acc[u], wf);
}

__device__ __forceinline__ float widen(uint16_t x) { return bf16_lo(x); }
__device__ __forceinline__ float widen(_Float16 x) { return static_cast<float>(x); }
__device__ __forceinline__ float widen(float x) { return x; }

// One thread's group of 8 outputs of one row whose group lies wholly inside
// the shard (partial tiles): the same rank-ordered sum, loads issued
// kReduceBatch sources ahead.
template <typename T, int kB, bool kAny, class Src>
__device__ __forceinline__ void reduce_group_vec(const Src& src, int64_t off, float* __restrict__ drow, int W,
                                                 float wf, uint32_t t) {
    float acc[8];
    Raw8<T, kB> x[kReduceBatch];
    for (int i = 0; i < W; i += kReduceBatch) {
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b)
            if (i + b < W) {
                if constexpr (kAny) x[b].load_any(source<T>(src, off, i + b), t);
                else x[b].load(source<T>(src, off, i + b), t);
            }
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b) {
            if (i + b >= W) break;
            if (i + b == 0) x[b].init(acc);
            else x[b].add(acc);
        }
    }
    store_avg8<T, kB>(drow, t, acc, wf);
}

// One output element at element offset `g` of every chunk (unaligned or
// ragged parts), loads issued kReduceBatch sources ahead.
template <typename T, class Src>
__device__ __forceinline__ float reduce_one(const Src& src, int64_t g, int W, float wf) {
    float acc = 0.f;
    T x[kReduceBatch];
    for (int i = 0; i < W; i += kReduceBatch) {
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b)
            if (i + b < W) x[b] = source<T>(src, g, i + b)[0];
#pragma unroll
        for (int b = 0; b < kReduceBatch; ++b) {
            if (i + b >= W) break;
            acc = (i + b == 0) ? widen(x[b]) : acc + widen(x[b]);
        }
    }
    return acc / wf;
}

// kB threads per workgroup, each owning kReduceSteps groups of 8 outputs: a
// tile of kB * 8 * kReduceSteps outputs.  kAny: some parameter's sources are
// off the 16-byte grid (the host picks it only then).  The parameter of each
// tile and its fields come from lane-held tables.
template <class Chunks, typename T, int kB, bool kAny>
__global__ void __launch_bounds__(kB) rs_reduce_kernel(const ReduceArgs<Chunks> a) {
    constexpr int64_t kRow = int64_t(kB) * kVec;
    constexpr int64_t kTile = kRow * kReduceSteps;
    const int l = table_lane();
#if FSDP_LDS_TABLE
    const int my_start = staged_entry(a.tile_start, a.nparams);
#else
    const int my_start = lane_index() < PMAX ? a.tile_start[l] : INT_MAX;
#endif
    const int64_t my_valid = a.valid[l], my_off = a.off[l];
    float* const my_dst = a.dst[l];
    const int W = a.world;
    const float wf = float(W);
    const uint32_t t = threadIdx.x;
    for (int64_t step = blockIdx.x; step < a.ntiles; step += gridDim.x) {
        const int tile = int(step);
        const int p = param_of_tile(my_start, tile);
        const int64_t v = from_lane(my_valid, p);
        const int64_t lo = int64_t(tile - from_lane(my_start, p)) * kTile;
        const int64_t off = from_lane(my_off, p);
        float* __restrict__ d0 = from_lane(my_dst, p);
        // Outputs are stored 16 bytes at a time when d0 is 16-byte aligned
        // and the sources loaded 16 bytes at a time: directly when they are
        // 16-byte aligned, through ld16_any otherwise (kAny only).
        bool vec, svec;
        if constexpr (kAny) {
            vec = is_aligned16(d0);
            svec = a.src.aligned() && ((off * int64_t(sizeof(T))) & 15) == 0;
        } else {
            vec = is_aligned16(d0) && a.src.aligned() && ((off * int64_t(sizeof(T))) & 15) == 0;
            svec = true;
        }
        if (vec && lo + kTile <= v) {
            if (std::is_same<Chunks, ContigChunks>::value) {
                const ContigChunks& c = reinterpret_cast<const ContigChunks&>(a.src);
                const StridedTile<T> st{reinterpret_cast<const T*>(c.base) + off + lo,
                                        c.stride / int64_t(sizeof(T))};
                if (!kAny || svec) reduce_tile_vec<T, kB, false>(st, 0, d0 + lo, W, wf);
                else reduce_tile_vec<T, kB, kAny>(st, 0, d0 + lo, W, wf);
            } else {
                const TableChunks& c = reinterpret_cast<const TableChunks&>(a.src);
                if (!kAny || svec) reduce_tile_vec<T, kB, false>(c, off + lo, d0 + lo, W, wf);
                else reduce_tile_vec<T, kB, kAny>(c, off + lo, d0 + lo, W, wf);
            }
            continue;
        }
        // partial tile: row by row; a thread's group vectorised when all of it is in range
        for (int u = 0; u < kReduceSteps; ++u) {
            const int64_t row = lo + u * kRow;
            if (row >= v) break;
            if (vec && row + Raw8<T, kB>::pos(t, 7) < v) {
                if (std::is_same<Chunks, ContigChunks>::value) {
                    const ContigChunks& c = reinterpret_cast<const ContigChunks&>(a.src);
                    const StridedTile<T> st{reinterpret_cast<const T*>(c.base) + off + row,
                                            c.stride / int64_t(sizeof(T))};
                    if (!kAny || svec) reduce_group_vec<T, kB, false>(st, 0, d0 + row, W, wf, t);
                    else reduce_group_vec<T, kB, kAny>(st, 0, d0 + row, W, wf, t);
                } else {
                    const TableChunks& c = reinterpret_cast<const TableChunks&>(a.src);
                    if (!kAny || svec) reduce_group_vec<T, kB, false>(c, off + row, d0 + row, W, wf, t);
                    else reduce_group_vec<T, kB, kAny>(c, off + row, d0 + row, W, wf, t);
                }
                continue;
            }
            for (int e = 0; e < kVec; ++e) {
                const int64_t g = row + Raw8<T, kB>::pos(t, e);
                if (g >= v) continue;
                if (std::is_same<Chunks, ContigChunks>::value) {
                    const ContigChunks& c = reinterpret_cast<const ContigChunks&>(a.src);
                    const StridedTile<T> st{reinterpret_cast<const T*>(c.base), c.stride / int64_t(sizeof(T))};
                    d0[g] = reduce_one<T>(st, off + g, W, wf);
                } else {
                    d0[g] = reduce_one<T>(reinterpret_cast<const TableChunks&>(a.src), off + g, W, wf);
                }
            }
        }
    }
}

// ------------------------------------------------------------------ host side

// Below this many full-size reduce tiles per CU, the reduce uses half-size tiles.
constexpr int kSmallShardTilesPerCU = 4;
// From this many big pack tiles per CU up, a single-chunk pack uses them.
constexpr int kPackBigTilesPerCU = 4;

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
};

// The byte spans of one call's inputs or outputs, on the stack: at most one
// per parameter or one per chunk of a table, so the hot calls allocate
// nothing on the host either.
constexpr int kMaxSpans = (PMAX > kMaxChunks ? PMAX : kMaxChunks) + 1;
struct Spans {
    Span s[kMaxSpans];
    int n = 0;
    bool full = false;   // more spans than kMaxSpans were added (the call is refused)
    void add(const void* p, int64_t bytes) {
        if (n < kMaxSpans) s[n++] = {uintptr_t(p), uintptr_t(p) + uintptr_t(bytes)};
        else full = true;
    }
};

// Outputs must be pairwise disjoint and disjoint from every input.
fsdp_status check_overlap(const Spans& out_spans, const Spans& ins) {
    if (out_spans.full || ins.full) return fail(FSDP_ERR_TOO_MANY, "too many buffers to check for overlap");
    Spans outs = out_spans;
    Span* const b = outs.s;
    Span* const e = outs.s + outs.n;
    std::sort(b, e, [](const Span& x, const Span& y) { return x.lo < y.lo; });
    for (int k = 1; k < outs.n; ++k)
        if (b[k].lo < b[k - 1].hi) return fail(FSDP_ERR_OVERLAP, "two outputs overlap");
    for (int k = 0; k < ins.n; ++k) {
        const Span& in = ins.s[k];
        // first output ending after in.lo
        const Span* it = std::upper_bound(b, e, in.lo, [](uintptr_t v, const Span& x) { return v < x.hi; });
        if (it != e && it->lo < in.hi) return fail(FSDP_ERR_OVERLAP, "an output overlaps an input");
    }
    return FSDP_OK;
}

// `index` >= 0 names element `index` of the array `name`.
fsdp_status check_bucket_ptr(const void* ptr, int64_t elems, const char* name, int index = -1) {
    const bool null = elems > 0 && ptr == nullptr;
    if (!null && (reinterpret_cast<uintptr_t>(ptr) & 15) == 0) return FSDP_OK;
    const std::string what = index < 0 ? std::string(name) : std::string(name) + "[" + std::to_string(index) + "]";
    if (null) return fail(FSDP_ERR_INVALID, what + " is NULL");
    return fail(FSDP_ERR_ALIGN, what + " is not 16-byte aligned");
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

bool known_dtype(fsdp_dtype t) { return t == FSDP_DTYPE_BF16 || t == FSDP_DTYPE_F32 || t == FSDP_DTYPE_F16; }
int elem_bytes(fsdp_dtype t) { return t == FSDP_DTYPE_F32 ? 4 : 2; }

// A host array of W chunk pointers, each 16-byte aligned and non-NULL when
// chunks have elements.
fsdp_status load_chunk_table(const Plan& pl, const void* const* chunks, int esize, TableChunks* out,
                             Spans* spans) {
    if (chunks == nullptr) return fail(FSDP_ERR_INVALID, "chunks is NULL");
    if (pl.world > kMaxChunks) return fail(FSDP_ERR_TOO_MANY, "world size exceeds FSDP_MAX_CHUNKS");
    fsdp_status st;
    for (int i = 0; i < pl.world; ++i) {
        if ((st = check_bucket_ptr(chunks[i], pl.chunk, "chunks", i)) != FSDP_OK) return st;
        out->ptr[i] = static_cast<char*>(const_cast<void*>(chunks[i]));
        if (pl.chunk > 0) spans->add(chunks[i], pl.chunk * esize);
    }
    return FSDP_OK;
}

// One launch of `kernel` over `ntiles` work tiles, one tile per workgroup up
// to kBlocksPerCU workgroups per CU (grid-stride beyond that).  The grid also
// keeps its work-item count below 2^31, and below the plan's max_workgroups
// when that is positive.
template <typename Args>
fsdp_status launch(const Plan& pl, void (*kernel)(const Args), const Args& args, int ntiles, int block,
                   hipStream_t stream, int rows = 1) {
    if (ntiles <= 0 || rows <= 0) return FSDP_OK;
    fsdp_status st = FSDP_OK;
    const int cus = cu_count(&st);
    if (st != FSDP_OK) return st;
    int64_t cap = std::min<int64_t>(int64_t(cus) * kBlocksPerCU, (int64_t(1) << 31) / block);
    if (pl.max_workgroups > 0) cap = std::min<int64_t>(cap, pl.max_workgroups);
    const dim3 grid(unsigned(std::min<int64_t>(ntiles, cap)), unsigned(rows));
    void* kargs[] = {const_cast<Args*>(&args)};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, dim3(block), kargs, 0, stream);
    if (e != hipSuccess) return fail(FSDP_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e));
    return FSDP_OK;
}

int64_t tiles(int64_t n, int64_t tile) { return (n + tile - 1) / tile; }

// Whether every chunk of a bucket buffer starts on the 16-byte grid (the host
// has checked the base and every table entry; a contiguous buffer's stride
// may still be off the grid in a dense bucket).
bool chunks_aligned(const ContigChunks& c) { return ((uintptr_t(c.base) | uintptr_t(c.stride)) & 15) == 0; }
bool chunks_aligned(const TableChunks&) { return true; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// ---- ag_pack

// `dst` is the send chunk (OneChunk) or the W destination chunks
// (TableChunks); `outs` holds their byte spans for the overlap check.
template <class Dst>
fsdp_status do_ag_pack(const Plan& pl, int32_t rank, const float* const* shards, fsdp_dtype wire, const Dst& dst,
                       int ndst, const Spans& outs, hipStream_t stream, bool cached = false) {
    fsdp_status st;
    if (rank < 0 || rank >= pl.world) return fail(FSDP_ERR_INVALID, "rank out of range");
    if (shards == nullptr) return fail(FSDP_ERR_INVALID, "shards is NULL");
    PackArgs<Dst> a{};
    Spans ins;
    int64_t nt = 0, nt_big = 0;   // at most the planner's checked pack tile count
    for (int p = 0; p < pl.nparams; ++p) {
        const int64_t v = pl.local_elems(p, rank);
        if ((st = check_param_ptr(shards[p], v, 4, p, "shards")) != FSDP_OK) return st;
        a.src[p] = shards[p];
        a.off[p] = pl.off[p];
        a.valid[p] = v;
        nt += tiles(pl.off[p + 1] - pl.off[p], kPackTile);
        nt_big += tiles(pl.off[p + 1] - pl.off[p], kPackBigTile);
        if (v > 0) ins.add(shards[p], v * 4);
    }
    a.off[pl.nparams] = pl.chunk;
    a.dst = dst;
    a.ndst = ndst;
    a.nparams = pl.nparams;
    if (nt > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
    if ((st = check_overlap(outs, ins)) != FSDP_OK) return st;
    // A single-chunk pack of at least kPackBigTilesPerCU big tiles per CU
    // takes the big tiles (more bytes in flight per wave); smaller buckets keep
    // the small ones, which spread evenly over the CUs.  (The first HIP call:
    // every argument is checked.)
    bool big = false;
    if constexpr (std::is_same<Dst, OneChunk>::value) {
        if (!cached) {
            const int cus = cu_count(&st);
            if (st != FSDP_OK) return st;
            big = nt_big >= int64_t(kPackBigTilesPerCU) * cus;
        }
    }
    const int64_t tile = big ? kPackBigTile : kPackTile;
    int64_t t0 = 0;
    for (int p = 0; p < pl.nparams; ++p) {
        a.tile_start[p] = int32_t(t0);
        t0 += tiles(pl.off[p + 1] - pl.off[p], tile);
    }
    for (int p = pl.nparams; p < PMAX; ++p) a.tile_start[p] = INT32_MAX;   // never a tile's parameter
    a.ntiles = int32_t(t0);
    if (big) {
        if (wire == FSDP_DTYPE_BF16)
            return launch(pl, ag_pack_kernel<kBF16, Dst, kPackBigBlock, kPackBigSteps>, a, a.ntiles, kPackBigBlock, stream);
        if (wire == FSDP_DTYPE_F16)
            return launch(pl, ag_pack_kernel<kF16, Dst, kPackBigBlock, kPackBigSteps>, a, a.ntiles, kPackBigBlock, stream);
        return launch(pl, ag_pack_kernel<kF32, Dst, kPackBigBlock, kPackBigSteps>, a, a.ntiles, kPackBigBlock, stream);
    }
    if constexpr (std::is_same<Dst, OneChunk>::value) {
        if (cached) {
            if (wire == FSDP_DTYPE_BF16) return launch(pl, push_pack_kernel<kBF16>, a, a.ntiles, kPackBlock, stream);
            if (wire == FSDP_DTYPE_F16) return launch(pl, push_pack_kernel<kF16>, a, a.ntiles, kPackBlock, stream);
            return launch(pl, push_pack_kernel<kF32>, a, a.ntiles, kPackBlock, stream);
        }
    }
    if (wire == FSDP_DTYPE_BF16)
        return launch(pl, ag_pack_kernel<kBF16, Dst, kPackBlock, kPackSteps>, a, a.ntiles, kPackBlock, stream);
    if (wire == FSDP_DTYPE_F16)
        return launch(pl, ag_pack_kernel<kF16, Dst, kPackBlock, kPackSteps>, a, a.ntiles, kPackBlock, stream);
    return launch(pl, ag_pack_kernel<kF32, Dst, kPackBlock, kPackSteps>, a, a.ntiles, kPackBlock, stream);
}

fsdp_status do_ag_pack_one(const fsdp_plan* h, int32_t rank, const float* const* shards, fsdp_dtype wire,
                           void* send_chunk, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (!known_dtype(wire)) return fail(FSDP_ERR_INVALID, "unknown dtype");
    if ((st = check_bucket_ptr(send_chunk, pl->chunk, "send_chunk")) != FSDP_OK) return st;
    Spans outs;
    if (pl->chunk > 0) outs.add(send_chunk, pl->chunk * elem_bytes(wire));
    return do_ag_pack(*pl, rank, shards, wire, OneChunk{static_cast<char*>(send_chunk)}, 1, outs, stream);
}

// ---- ag_unpack: u = 2-byte units per element

template <class Chunks>
fsdp_status do_ag_unpack(const Plan& pl, const Chunks& src, const Spans& ins, int u,
                         void* const* params, hipStream_t stream) {
    fsdp_status st;
    if (params == nullptr) return fail(FSDP_ERR_INVALID, "params is NULL");
    UnpackArgs<Chunks> a{};
    Spans outs;
    int64_t nt = 0;
    for (int p = 0; p < pl.nparams; ++p) {
        const int64_t e = pl.elems[p];
        if ((st = check_param_ptr(params[p], e, 2 * u, p, "params")) != FSDP_OK) return st;
        a.dst[p] = static_cast<uint16_t*>(params[p]);
        a.off[p] = pl.off[p] * u;
        a.seg[p] = pl.seg[p] * u;
        a.elems[p] = e * u;
        const int64_t tps = tiles(a.seg[p], kCopyTile);
        if (tps > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
        a.tiles_per_seg[p] = int32_t(tps);
        a.tile_start[p] = int32_t(nt);
        nt += int64_t(pl.world) * a.tiles_per_seg[p];
        if (nt > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
        if (e > 0) outs.add(params[p], e * 2 * u);
    }
    a.src = src;
    a.nparams = pl.nparams;
    a.ntiles = int32_t(nt);
    if ((st = check_overlap(outs, ins)) != FSDP_OK) return st;
    // Every tile of segment i of parameter p reads chunk i at off_p and writes
    // params[p] at i * L_p: all on the 16-byte grid unless a stride, offset,
    // length or pointer is not.
    bool any = !chunks_aligned(src);
    for (int p = 0; p < pl.nparams; ++p)
        if (((a.off[p] * 2) & 15) || ((a.seg[p] * 2) & 15) || !aligned16(a.dst[p])) any = true;
    if (any) return launch(pl, ag_unpack_kernel<Chunks, true>, a, a.ntiles, kCopyBlock, stream);
    return launch(pl, ag_unpack_kernel<Chunks, false>, a, a.ntiles, kCopyBlock, stream);
}

// ---- rs_pack: gradient elements of `gsize` bytes; kWiden (kBF16 / kF16) casts
// 16-bit gradients to fp32, kF32 copies

template <class Chunks, int kWiden>
fsdp_status do_rs_pack(const Plan& pl, const void* const* grads, int gsize, const Chunks& dst,
                       const Spans& outs, hipStream_t stream) {
    fsdp_status st;
    if (grads == nullptr) return fail(FSDP_ERR_INVALID, "grads is NULL");
    const int u = kWiden != kF32 ? 1 : gsize / 2;     // kernel units per element
    RsPackArgs<Chunks> a{};
    Spans ins;
    int64_t nt = 0;
    for (int p = 0; p < pl.nparams; ++p) {
        const int64_t e = pl.elems[p];
        if ((st = check_param_ptr(grads[p], e, gsize, p, "grads")) != FSDP_OK) return st;
        a.src[p] = static_cast<const uint16_t*>(grads[p]);
        a.off[p] = pl.off[p] * u;
        a.seg[p] = pl.seg[p] * u;
        a.elems[p] = e * u;
        const int64_t tps = tiles((pl.off[p + 1] - pl.off[p]) * u, kWiden != kF32 ? kWidenTile : kCopyTile);
        if (tps * pl.world > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
        a.tiles_per_seg[p] = int32_t(tps);
        a.tile_start[p] = int32_t(nt);                  // rescaled below for the parameter-major order
        nt += tps;
        if (nt * pl.world > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
        if (e > 0) ins.add(grads[p], e * gsize);
    }
    a.dest_major = pl.world > kDestMajorW;
    if (!a.dest_major)
        for (int p = 0; p < pl.nparams; ++p) a.tile_start[p] *= pl.world;
    a.off[pl.nparams] = pl.chunk * u;
    a.dst = dst;
    a.nparams = pl.nparams;
    a.tiles_per_dest = int32_t(nt);
    a.ntiles = int32_t(nt * pl.world);
    if ((st = check_overlap(outs, ins)) != FSDP_OK) return st;
    // Tiles read grads[p] at j * L_p and write chunk j at off_p (the widening
    // pack has its own checks and no misaligned vector path).
    bool any = false;
    if constexpr (kWiden == kF32) {
        any = !chunks_aligned(dst);
        for (int p = 0; p < pl.nparams; ++p)
            if (((a.off[p] * 2) & 15) || ((a.seg[p] * 2) & 15) || !aligned16(a.src[p])) any = true;
    }
    if (any) return launch(pl, rs_pack_kernel<Chunks, kWiden, true>, a, a.ntiles, kCopyBlock, stream);
    return launch(pl, rs_pack_kernel<Chunks, kWiden, false>, a, a.ntiles, kCopyBlock, stream);
}

// ---- rs_reduce: received elements of type T

template <class Chunks, typename T>
fsdp_status do_rs_reduce(const Plan& pl, int32_t rank, const Chunks& src, const Spans& ins,
                         float* const* grad_shards, hipStream_t stream) {
    fsdp_status st = FSDP_OK;
    if (grad_shards == nullptr) return fail(FSDP_ERR_INVALID, "grad_shards is NULL");
    Spans outs;
    int64_t full_tiles = 0;
    for (int p = 0; p < pl.nparams; ++p) {
        const int64_t v = pl.local_elems(p, rank);
        if ((st = check_param_ptr(grad_shards[p], v, 4, p, "grad_shards")) != FSDP_OK) return st;
        if (v > 0) outs.add(grad_shards[p], v * 4);
        full_tiles += tiles(v, kReduceTile);
    }
    if ((st = check_overlap(outs, ins)) != FSDP_OK) return st;
    if (full_tiles == 0) return FSDP_OK;                 // nothing to write: no launch
    // A rank's shard that makes fewer than kSmallShardTilesPerCU full-size
    // tiles per CU is cut into half-size tiles (half as many threads per
    // workgroup, the same work per thread), so that the workgroups spread
    // evenly over the CUs.  (The first HIP call: every argument is checked.)
    const int cus = cu_count(&st);
    if (st != FSDP_OK) return st;
    bool small = full_tiles < int64_t(kSmallShardTilesPerCU) * cus;
    if (pl.reduce_tiles == FSDP_REDUCE_TILES_FULL) small = false;
    if (pl.reduce_tiles == FSDP_REDUCE_TILES_HALF) small = true;
    const int64_t tile = small ? kReduceTile / 2 : kReduceTile;
    // Tiles of the parameters with the fewest tiles are numbered (and so
    // dispatched) first: a ragged last tile sums its W sources in a longer
    // dependent chain, which then overlaps the bulk instead of trailing it.
    // (A stable insertion sort of at most FSDP_MAX_PARAMS entries: equal
    // counts keep the bucket order, and nothing is allocated.)
    int order[PMAX];
    int64_t nts[PMAX];
    for (int p = 0; p < pl.nparams; ++p) {
        nts[p] = tiles(pl.local_elems(p, rank), tile);
        int q = p;
        for (; q > 0 && nts[order[q - 1]] > nts[p]; --q) order[q] = order[q - 1];
        order[q] = p;
    }
    ReduceArgs<Chunks> a{};
    int64_t nt = 0;
    for (int q = 0; q < pl.nparams; ++q) {
        const int p = order[q];
        a.dst[q] = grad_shards[p];
        a.off[q] = pl.off[p];
        a.valid[q] = pl.local_elems(p, rank);
        a.tile_start[q] = int32_t(nt);
        nt += nts[p];
        if (nt > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
    }
    for (int q = pl.nparams; q < PMAX; ++q) a.tile_start[q] = INT32_MAX;   // never a tile's parameter
    a.src = src;
    a.world = pl.world;
    a.nparams = pl.nparams;
    a.ntiles = int32_t(nt);
    // Sources of parameter p start at off_p in every chunk.
    bool any = false;
    for (int p = 0; p < pl.nparams; ++p)
        if (!chunks_aligned(src) || ((pl.off[p] * int64_t(sizeof(T))) & 15)) any = true;
    if (small) {
        if (any) return launch(pl, rs_reduce_kernel<Chunks, T, kReduceBlock / 2, true>, a, a.ntiles, kReduceBlock / 2, stream);
        return launch(pl, rs_reduce_kernel<Chunks, T, kReduceBlock / 2, false>, a, a.ntiles, kReduceBlock / 2, stream);
    }
    if (any) return launch(pl, rs_reduce_kernel<Chunks, T, kReduceBlock, true>, a, a.ntiles, kReduceBlock, stream);
    return launch(pl, rs_reduce_kernel<Chunks, T, kReduceBlock, false>, a, a.ntiles, kReduceBlock, stream);
}

}  // namespace
}  // namespace fsdp

using namespace fsdp;

extern "C" fsdp_status fsdp_ag_pack(const fsdp_plan* h, int32_t rank, const float* const* shards,
                                    uint16_t* send_chunk, hipStream_t stream) {
    return do_ag_pack_one(h, rank, shards, FSDP_DTYPE_BF16, send_chunk, stream);
}

extern "C" fsdp_status fsdp_ag_pack_ex(const fsdp_plan* h, int32_t rank, const float* const* shards,
                                       fsdp_dtype param_dtype, void* send_chunk, hipStream_t stream) {
    return do_ag_pack_one(h, rank, shards, param_dtype, send_chunk, stream);
}

extern "C" fsdp_status fsdp_ag_pack_push(const fsdp_plan* h, int32_t rank, const float* const* shards,
                                         fsdp_dtype param_dtype, void* const* chunks, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (!known_dtype(param_dtype)) return fail(FSDP_ERR_INVALID, "unknown dtype");
    if (rank < 0 || rank >= pl->world) return fail(FSDP_ERR_INVALID, "rank out of range");
    const int esize = elem_bytes(param_dtype);
    TableChunks dst{};
    Spans outs;
    if ((st = load_chunk_table(*pl, const_cast<const void* const*>(chunks), esize, &dst, &outs)) != FSDP_OK)
        return st;
    if (pl->world < kReplicateMinW || pl->chunk == 0)
        return do_ag_pack(*pl, rank, shards, param_dtype, dst, pl->world, outs, stream);
    // Many destinations: pack once into the rank's own chunk (through the
    // cache), then copy that chunk to the other W - 1.  Every chunk's span is
    // in the overlap check of the pack.
    ReplicateArgs r{};
    r.dst = dst;
    const int64_t bytes = pl->chunk * esize;
    r.units = bytes / 16;
    r.tail = int32_t(bytes % 16 / 2);
    r.from = rank;
    r.ndst = pl->world - 1;
    const int64_t nt = tiles(r.units + (r.tail > 0), kRepTile);
    const bool grouped = r.ndst >= kRepGroup;
    const int64_t items = tiles(nt, kXcds) * kXcds * (grouped ? kRepGroup : r.ndst);
    if (items > INT32_MAX) return fail(FSDP_ERR_OVERFLOW, "too many work tiles");
    r.ntiles = int32_t(nt);
    r.nitems = int32_t(items);
    if ((st = do_ag_pack(*pl, rank, shards, param_dtype, OneChunk{dst.ptr[rank]}, 1, outs, stream, true)) != FSDP_OK)
        return st;
    if (grouped)
        return launch(*pl, replicate_grouped_kernel, r, r.nitems, kCopyBlock, stream, int(tiles(r.ndst, kRepGroup)));
    return launch(*pl, replicate_kernel, r, r.nitems, kCopyBlock, stream);
}

extern "C" fsdp_status fsdp_ag_unpack(const fsdp_plan* h, const uint16_t* gathered, uint16_t* const* params,
                                      hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    const int64_t total = int64_t(pl->world) * pl->chunk;
    if ((st = check_bucket_ptr(gathered, total, "gathered")) != FSDP_OK) return st;
    Spans ins;
    if (total > 0) ins.add(gathered, total * 2);
    const ContigChunks src{reinterpret_cast<char*>(const_cast<uint16_t*>(gathered)), pl->chunk * 2};
    return do_ag_unpack(*pl, src, ins, 1, reinterpret_cast<void* const*>(params), stream);
}

extern "C" fsdp_status fsdp_ag_unpack_ex(const fsdp_plan* h, fsdp_dtype param_dtype, const void* const* chunks,
                                         void* const* params, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (!known_dtype(param_dtype)) return fail(FSDP_ERR_INVALID, "unknown dtype");
    const int esize = elem_bytes(param_dtype);
    TableChunks src{};
    Spans ins;
    if ((st = load_chunk_table(*pl, chunks, esize, &src, &ins)) != FSDP_OK) return st;
    return do_ag_unpack(*pl, src, ins, esize / 2, params, stream);
}

extern "C" fsdp_status fsdp_rs_pack(const fsdp_plan* h, const uint16_t* const* grads, uint16_t* send_buf,
                                    hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    const int64_t total = int64_t(pl->world) * pl->chunk;
    if ((st = check_bucket_ptr(send_buf, total, "send_buf")) != FSDP_OK) return st;
    Spans outs;
    if (total > 0) outs.add(send_buf, total * 2);
    const ContigChunks dst{reinterpret_cast<char*>(send_buf), pl->chunk * 2};
    return do_rs_pack<ContigChunks, kF32>(*pl, reinterpret_cast<const void* const*>(grads), 2, dst, outs, stream);
}

extern "C" fsdp_status fsdp_rs_pack_ex(const fsdp_plan* h, fsdp_dtype grad_dtype, const void* const* grads,
                                       fsdp_dtype reduce_dtype, void* const* chunks, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (!known_dtype(grad_dtype) || !known_dtype(reduce_dtype)) return fail(FSDP_ERR_INVALID, "unknown dtype");
    // the wire keeps the gradients' type or widens 16-bit gradients to fp32;
    // any other pair would be a rounding step the method does not describe
    if (reduce_dtype != grad_dtype && reduce_dtype != FSDP_DTYPE_F32)
        return fail(FSDP_ERR_INVALID, "the wire must have the gradients' type or be fp32");
    TableChunks dst{};
    Spans outs;
    if ((st = load_chunk_table(*pl, chunks, elem_bytes(reduce_dtype), &dst, &outs)) != FSDP_OK) return st;
    if (grad_dtype == FSDP_DTYPE_BF16 && reduce_dtype == FSDP_DTYPE_F32)
        return do_rs_pack<TableChunks, kBF16>(*pl, grads, 2, dst, outs, stream);
    if (grad_dtype == FSDP_DTYPE_F16 && reduce_dtype == FSDP_DTYPE_F32)
        return do_rs_pack<TableChunks, kF16>(*pl, grads, 2, dst, outs, stream);
    return do_rs_pack<TableChunks, kF32>(*pl, grads, elem_bytes(grad_dtype), dst, outs, stream);
}

extern "C" fsdp_status fsdp_rs_reduce(const fsdp_plan* h, int32_t rank, const uint16_t* recv,
                                      float* const* grad_shards, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (rank < 0 || rank >= pl->world) return fail(FSDP_ERR_INVALID, "rank out of range");
    const int64_t total = int64_t(pl->world) * pl->chunk;
    if ((st = check_bucket_ptr(recv, total, "recv")) != FSDP_OK) return st;
    Spans ins;
    if (total > 0) ins.add(recv, total * 2);
    const ContigChunks src{reinterpret_cast<char*>(const_cast<uint16_t*>(recv)), pl->chunk * 2};
    return do_rs_reduce<ContigChunks, uint16_t>(*pl, rank, src, ins, grad_shards, stream);
}

extern "C" fsdp_status fsdp_rs_reduce_ex(const fsdp_plan* h, int32_t rank, fsdp_dtype reduce_dtype,
                                         const void* const* chunks, float* const* grad_shards, hipStream_t stream) {
    clear_error();
    fsdp_status st = FSDP_OK;
    const Plan* pl = get_plan(h, &st);
    if (!pl) return st;
    if (!known_dtype(reduce_dtype)) return fail(FSDP_ERR_INVALID, "unknown dtype");
    if (rank < 0 || rank >= pl->world) return fail(FSDP_ERR_INVALID, "rank out of range");
    TableChunks src{};
    Spans ins;
    if ((st = load_chunk_table(*pl, chunks, elem_bytes(reduce_dtype), &src, &ins)) != FSDP_OK) return st;
    if (reduce_dtype == FSDP_DTYPE_F32) return do_rs_reduce<TableChunks, float>(*pl, rank, src, ins, grad_shards, stream);
    if (reduce_dtype == FSDP_DTYPE_F16)
        return do_rs_reduce<TableChunks, _Float16>(*pl, rank, src, ins, grad_shards, stream);
    return do_rs_reduce<TableChunks, uint16_t>(*pl, rank, src, ins, grad_shards, stream);
}
