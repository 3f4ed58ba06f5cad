// Bucket planner: per-parameter offsets, dim-0 padding to W * c_p rows and
// alignment of every parameter's start (SimpleFSDP section 3.2.1 bucketing,
// section 3.1 Shard(0) sharding).  Host code only; makes no HIP call.

#include <mutex>
#include <new>
#include <unordered_set>

#include "plan_impl.h"

struct fsdp_plan {
    fsdp::Plan plan;
};

namespace fsdp {
namespace {

std::mutex g_mu;
std::unordered_set<const fsdp_plan*>& live() {
    static std::unordered_set<const fsdp_plan*> s;
    return s;
}
thread_local std::string t_err;

constexpr int64_t kMaxBytes = int64_t(1) << 62;

bool mul_ok(int64_t a, int64_t b, int64_t* out) { return !__builtin_mul_overflow(a, b, out); }
bool add_ok(int64_t a, int64_t b, int64_t* out) { return !__builtin_add_overflow(a, b, out); }

bool round_up_ok(int64_t x, int64_t a, int64_t* out) {
    int64_t t;
    if (!add_ok(x, a - 1, &t)) return false;
    *out = t / a * a;
    return true;
}

}  // namespace

bool plan_is_live(const fsdp_plan* h) {
    std::lock_guard<std::mutex> lk(g_mu);
    return h != nullptr && live().count(h) != 0;
}

const Plan* plan_of(const fsdp_plan* h) { return plan_is_live(h) ? &h->plan : nullptr; }

fsdp_status fail(fsdp_status s, const std::string& msg) {
    t_err = msg;
    return s;
}

void clear_error() { t_err.clear(); }

}  // namespace fsdp

using namespace fsdp;

extern "C" fsdp_status fsdp_bucket_plan(int32_t world_size, int32_t num_params,
                                        const int64_t* dim0, const int64_t* inner,
                                        int32_t align_elems, fsdp_plan** out) {
    return fsdp_bucket_plan_ex(world_size, num_params, dim0, inner, align_elems, nullptr, out);
}

extern "C" fsdp_status fsdp_bucket_plan_ex(int32_t world_size, int32_t num_params,
                                           const int64_t* dim0, const int64_t* inner,
                                           int32_t align_elems, const fsdp_plan_options* options,
                                           fsdp_plan** out) {
    clear_error();
    if (out == nullptr) return fail(FSDP_ERR_INVALID, "out is NULL");
    *out = nullptr;
    if (options != nullptr) {
        if (options->max_workgroups < 0) return fail(FSDP_ERR_INVALID, "max_workgroups must be >= 0");
        if (options->reduce_tiles != FSDP_REDUCE_TILES_AUTO && options->reduce_tiles != FSDP_REDUCE_TILES_FULL &&
            options->reduce_tiles != FSDP_REDUCE_TILES_HALF)
            return fail(FSDP_ERR_INVALID, "unknown reduce_tiles");
        if (options->reserved != 0) return fail(FSDP_ERR_INVALID, "reserved must be 0");
    }
    if (world_size < 1) return fail(FSDP_ERR_INVALID, "world_size must be >= 1");
    if (num_params < 1) return fail(FSDP_ERR_INVALID, "num_params must be >= 1");
    if (num_params > FSDP_MAX_PARAMS)
        return fail(FSDP_ERR_TOO_MANY, "num_params exceeds FSDP_MAX_PARAMS");
    if (dim0 == nullptr || inner == nullptr) return fail(FSDP_ERR_INVALID, "dim0/inner is NULL");
    if (align_elems < 1 || (align_elems & (align_elems - 1)) != 0)
        return fail(FSDP_ERR_INVALID, "align_elems must be a power of two");

    Plan pl;
    pl.world = world_size;
    pl.nparams = num_params;
    pl.align = align_elems;
    const int64_t W = world_size, A = align_elems;
    int64_t pos = 0;
    for (int p = 0; p < num_params; ++p) {
        const int64_t n = dim0[p], k = inner[p];
        if (n < 0 || k < 1)
            return fail(FSDP_ERR_INVALID, "parameter " + std::to_string(p) + ": dim0 < 0 or inner < 1");
        int64_t e, c, L, e4;
        if (!mul_ok(n, k, &e) || !mul_ok(e, 4, &e4) || e4 >= kMaxBytes)
            return fail(FSDP_ERR_OVERFLOW, "parameter " + std::to_string(p) + ": N*inner too large");
        c = n / W + (n % W != 0);
        if (!mul_ok(c, k, &L)) return fail(FSDP_ERR_OVERFLOW, "segment too large");
        if (!round_up_ok(pos, A, &pos)) return fail(FSDP_ERR_OVERFLOW, "offset overflow");
        pl.rows.push_back(n);
        pl.inner.push_back(k);
        pl.cpr.push_back(c);
        pl.seg.push_back(L);
        pl.off.push_back(pos);
        pl.elems.push_back(e);
        if (!add_ok(pos, L, &pos)) return fail(FSDP_ERR_OVERFLOW, "chunk overflow");
    }
    int64_t S, WS, WS4;
    if (!round_up_ok(pos, A, &S)) return fail(FSDP_ERR_OVERFLOW, "chunk overflow");
    if (!mul_ok(W, S, &WS) || !mul_ok(WS, 4, &WS4) || WS4 >= kMaxBytes)
        return fail(FSDP_ERR_OVERFLOW, "W*S too large");
    pl.chunk = S;
    pl.off.push_back(S);
    if (options != nullptr) {
        pl.max_workgroups = options->max_workgroups;
        pl.reduce_tiles = options->reduce_tiles;
    }

    // Work tiles of each kernel must be countable in 31 bits.
    int64_t t_pack = 0, t_copy = 0, t_reduce = 0;
    for (int p = 0; p < num_params; ++p) {
        const int64_t region = pl.off[p + 1] - pl.off[p];
        t_pack += (region + kPackTile - 1) / kPackTile;
        t_copy += W * ((region + kCopyTile - 1) / kCopyTile);
        t_reduce += (pl.seg[p] + kReduceTile - 1) / kReduceTile;
    }
    if (t_pack > INT32_MAX || t_copy > INT32_MAX || t_reduce > INT32_MAX)
        return fail(FSDP_ERR_OVERFLOW, "too many work tiles");

    fsdp_plan* h = new (std::nothrow) fsdp_plan;
    if (h == nullptr) return fail(FSDP_ERR_NOMEM, "plan allocation failed");
    h->plan = std::move(pl);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        live().insert(h);
    }
    *out = h;
    return FSDP_OK;
}

extern "C" void fsdp_plan_free(fsdp_plan* h) {
    if (h == nullptr) return;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (live().erase(h) == 0) return;   // unknown or already freed: ignore
    }
    delete h;
}

extern "C" int64_t fsdp_plan_chunk_elems(const fsdp_plan* h) {
    const Plan* pl = plan_of(h);
    return pl ? pl->chunk : -1;
}

extern "C" int32_t fsdp_plan_world_size(const fsdp_plan* h) {
    const Plan* pl = plan_of(h);
    return pl ? pl->world : -1;
}

extern "C" int32_t fsdp_plan_num_params(const fsdp_plan* h) {
    const Plan* pl = plan_of(h);
    return pl ? pl->nparams : -1;
}

extern "C" fsdp_status fsdp_plan_param(const fsdp_plan* h, int32_t p, int64_t* rows_per_rank,
                                       int64_t* offset, int64_t* seg_elems) {
    clear_error();
    const Plan* pl = plan_of(h);
    if (!pl) return fail(FSDP_ERR_INVALID, "unknown plan");
    if (p < 0 || p >= pl->nparams) return fail(FSDP_ERR_INVALID, "parameter index out of range");
    if (rows_per_rank) *rows_per_rank = pl->cpr[p];
    if (offset) *offset = pl->off[p];
    if (seg_elems) *seg_elems = pl->seg[p];
    return FSDP_OK;
}

extern "C" int64_t fsdp_plan_local_rows(const fsdp_plan* h, int32_t p, int32_t rank) {
    const Plan* pl = plan_of(h);
    if (!pl || p < 0 || p >= pl->nparams || rank < 0 || rank >= pl->world) return -1;
    return pl->local_rows(p, rank);
}

extern "C" const char* fsdp_status_str(fsdp_status s) {
    switch (s) {
        case FSDP_OK: return "ok";
        case FSDP_ERR_INVALID: return "invalid argument";
        case FSDP_ERR_ALIGN: return "misaligned buffer";
        case FSDP_ERR_OVERFLOW: return "size overflow";
        case FSDP_ERR_TOO_MANY: return "too many parameters in one bucket";
        case FSDP_ERR_NOMEM: return "out of host memory";
        case FSDP_ERR_HIP: return "HIP runtime error";
        case FSDP_ERR_OVERLAP: return "output overlaps an input or another output";
        default: return "unknown status";
    }
}

extern "C" const char* fsdp_last_error(void) { return fsdp::t_err.c_str(); }
