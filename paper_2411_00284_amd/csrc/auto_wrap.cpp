// Auto-wrapping: SimpleFSDP's greedy bucketing of one pass's all-gathers
// (section 3.3.2 "Auto-wrapping": the profiling model T_m = alpha + beta*n,
// Algorithm 1, and the variables of Table 1).  Host code only; makes no HIP
// call.
//
// The walk is O(n): it keeps running sums for the bucket being built
// (B_{k+1}: all-gather words, memory, compute time) and for the two buckets
// closed last (B_k: compute time; B_{k-1}: reduce-scatter words).  Every
// floating-point value is formed by the same operations in the same order as
// the definition: compute times are summed in node order starting from 0.0,
// a collective costs alpha + beta * double(words) (product and sum each
// rounded; the library is built with -ffp-contract=off), and the backward
// left-hand side adds the reduce-scatter time to the all-gather time.

#include <cmath>
#include <string>

#include "plan_impl.h"

namespace fsdp {
namespace {

constexpr int64_t kMaxWords = int64_t(1) << 53;   // words convert to double exactly

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

}  // namespace
}  // namespace fsdp

using namespace fsdp;

extern "C" fsdp_status fsdp_auto_wrap(int32_t num_nodes, int32_t backward, const int64_t* ag_words,
                                      const int64_t* rs_words, const double* compute_time,
                                      const int64_t* compute_mem, double alpha_ag, double beta_ag,
                                      double alpha_rs, double beta_rs, int64_t mem_max,
                                      int32_t* bucket_of, int32_t* num_buckets) {
    clear_error();
    if (num_buckets == nullptr) return fail(FSDP_ERR_INVALID, "num_buckets is NULL");
    if (num_nodes < 0) return fail(FSDP_ERR_INVALID, "num_nodes must be >= 0");
    if (backward != 0 && backward != 1) return fail(FSDP_ERR_INVALID, "backward must be 0 or 1");
    if (num_nodes > 0 && (ag_words == nullptr || compute_time == nullptr || compute_mem == nullptr ||
                          bucket_of == nullptr))
        return fail(FSDP_ERR_INVALID, "a node array is NULL");
    if (backward && num_nodes > 0 && rs_words == nullptr)
        return fail(FSDP_ERR_INVALID, "rs_words is NULL in a backward pass");
    if (!finite_nonneg(alpha_ag) || !finite_nonneg(beta_ag) || !finite_nonneg(alpha_rs) ||
        !finite_nonneg(beta_rs))
        return fail(FSDP_ERR_INVALID, "alpha and beta must be finite and >= 0");
    if (mem_max < 0) return fail(FSDP_ERR_INVALID, "mem_max must be >= 0");

    // Validate every node first, so that an error leaves bucket_of untouched.
    int64_t total_ag = 0, total_rs = 0, total_mem = 0;
    for (int32_t i = 0; i < num_nodes; ++i) {
        const std::string at = "node " + std::to_string(i) + ": ";
        if (ag_words[i] < 0 || (backward && rs_words[i] < 0))
            return fail(FSDP_ERR_INVALID, at + "words must be >= 0");
        if (!finite_nonneg(compute_time[i])) return fail(FSDP_ERR_INVALID, at + "compute_time must be finite, >= 0");
        if (compute_mem[i] < 0) return fail(FSDP_ERR_INVALID, at + "compute_mem must be >= 0");
        total_ag += ag_words[i];
        if (backward) total_rs += rs_words[i];
        if (total_ag > kMaxWords || total_rs > kMaxWords)
            return fail(FSDP_ERR_OVERFLOW, at + "total words exceed 2^53");
        if (__builtin_add_overflow(total_mem, compute_mem[i], &total_mem))
            return fail(FSDP_ERR_OVERFLOW, at + "total compute_mem overflows int64");
    }

    int32_t k = -1;                // index of the bucket being built
    // the bucket being built, B_{k}
    int64_t cur_ag = 0, cur_rs = 0, cur_mem = 0;
    double cur_tc = 0.0;
    // the last closed bucket (its compute hides the next all-gather) and the
    // one before it (its reduce-scatter is in flight meanwhile)
    bool have_last = false, have_prev = false;
    double last_tc = 0.0;
    int64_t last_rs = 0, prev_rs = 0;
    for (int32_t i = 0; i < num_nodes; ++i) {
        bool join = false;
        if (k >= 0) {
            const double t_c = have_last ? last_tc : 0.0;
            const double t_ag = alpha_ag + beta_ag * double(cur_ag + ag_words[i]);
            bool time_ok;
            if (backward) {
                const double t_rs = have_prev ? alpha_rs + beta_rs * double(prev_rs) : 0.0;
                time_ok = t_rs + t_ag <= t_c;
            } else {
                time_ok = t_ag <= t_c;
            }
            const bool mem_ok = cur_mem + compute_mem[i] <= mem_max;
            join = time_ok && mem_ok;
        }
        if (!join) {
            if (k >= 0) {          // close the bucket being built
                prev_rs = last_rs;
                have_prev = have_last;
                last_rs = cur_rs;
                last_tc = cur_tc;
                have_last = true;
            }
            ++k;
            cur_ag = cur_rs = cur_mem = 0;
            cur_tc = 0.0;
        }
        cur_ag += ag_words[i];
        if (backward) cur_rs += rs_words[i];
        cur_mem += compute_mem[i];
        cur_tc += compute_time[i];
        bucket_of[i] = k;
    }
    *num_buckets = k + 1;
    return FSDP_OK;
}
