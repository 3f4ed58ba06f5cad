// Internal view of a bucket plan, shared by the planner and the launchers.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "fsdp_bucket.h"

namespace fsdp {

// Work tiles.  The copy kernels (ag_unpack, rs_pack) run kCopyBlock threads
// that move 8 elements (16 bytes of bf16) per thread and step, kCopySteps
// steps per tile; ag_pack runs kPackBlock threads that cast 8 elements per
// thread and step, kPackSteps steps per tile (kPackBigBlock and kPackBigSteps
// for a large single-chunk pack); the reduction runs kReduceBlock
// threads that each own kReduceSteps groups of 8 outputs.  One tile per
// workgroup (small tiles, many workgroups) measured fastest for these HBM
// streams.
#ifndef FSDP_COPY_BLOCK
#define FSDP_COPY_BLOCK 128
#endif
#ifndef FSDP_COPY_STEPS
#define FSDP_COPY_STEPS 2
#endif
#ifndef FSDP_PACK_STEPS
#define FSDP_PACK_STEPS 1
#endif
#ifndef FSDP_PACK_BLOCK
#define FSDP_PACK_BLOCK 128
#endif
#ifndef FSDP_PACK_BIG_BLOCK
#define FSDP_PACK_BIG_BLOCK 256
#endif
#ifndef FSDP_PACK_BIG_STEPS
#define FSDP_PACK_BIG_STEPS 4
#endif
#ifndef FSDP_REDUCE_BLOCK
#define FSDP_REDUCE_BLOCK 256
#endif
#ifndef FSDP_REDUCE_STEPS
#define FSDP_REDUCE_STEPS 2
#endif
constexpr int kVec = 8;
constexpr int kCopyBlock = FSDP_COPY_BLOCK;
constexpr int kCopySteps = FSDP_COPY_STEPS;
constexpr int64_t kCopyTile = int64_t(kCopyBlock) * kVec * kCopySteps;
// The widening pack (bf16 in, fp32 out) moves 4 elements per thread and step,
// so its tiles read half and write the same bytes as a copy tile.
constexpr int64_t kWidenTile = int64_t(kCopyBlock) * 4 * kCopySteps;
constexpr int kPackBlock = FSDP_PACK_BLOCK;
constexpr int kPackSteps = FSDP_PACK_STEPS;
constexpr int64_t kPackTile = int64_t(kPackBlock) * kVec * kPackSteps;
// The single-chunk pack of a large bucket uses bigger tiles.
constexpr int kPackBigBlock = FSDP_PACK_BIG_BLOCK;
constexpr int kPackBigSteps = FSDP_PACK_BIG_STEPS;
constexpr int64_t kPackBigTile = int64_t(kPackBigBlock) * kVec * kPackBigSteps;
constexpr int kReduceBlock = FSDP_REDUCE_BLOCK;
constexpr int kReduceSteps = FSDP_REDUCE_STEPS;
constexpr int64_t kReduceTile = int64_t(kReduceBlock) * kVec * kReduceSteps;

struct Plan {
    int32_t world;     // W
    int32_t nparams;   // P
    int32_t align;     // A (elements)
    int64_t chunk;     // S
    std::vector<int64_t> rows;     // N_p
    std::vector<int64_t> inner;    // inner_p
    std::vector<int64_t> cpr;      // c_p
    std::vector<int64_t> seg;      // L_p
    std::vector<int64_t> off;      // off_p, with off[P] = S
    std::vector<int64_t> elems;    // N_p * inner_p
    // Launch options fixed at planning (fsdp_plan_options); results never
    // depend on them.
    int64_t max_workgroups = 0;    // > 0: cap on every launch's grid
    int32_t reduce_tiles = FSDP_REDUCE_TILES_AUTO;

    int64_t local_rows(int p, int r) const {
        int64_t c = cpr[p];
        int64_t rest = rows[p] - int64_t(r) * c;
        return rest <= 0 ? 0 : (rest < c ? rest : c);
    }
    int64_t local_elems(int p, int r) const { return local_rows(p, r) * inner[p]; }
};

// Plans handed out by fsdp_bucket_plan and not yet freed.
bool plan_is_live(const fsdp_plan* h);
const Plan* plan_of(const fsdp_plan* h);

// Thread-local detail for fsdp_last_error.
fsdp_status fail(fsdp_status s, const std::string& msg);
void clear_error();

}  // namespace fsdp
