/*
 * fsdp_bucket.h - one rank's share of SimpleFSDP's bucketed FSDP
 * communication path (arXiv 2411.00284) on an AMD Instinct MI355X (gfx950).
 *
 * The paper makes every parameter a DTensor sharded on dim 0 over the W
 * data-parallel ranks (section 3.1), all-gathers it to a replicated 16-bit
 * copy before use and reduce-scatters its gradient with averaging in fp32
 * (section 4, mixed precision and the replicate_compute listing), and groups
 * the collectives of several parameters into one bucket: one flat buffer is
 * filled before the collective (copy-in) and read back by each parameter's
 * size after it (copy-out / read-out) (section 3.2.1).  This library runs
 * the parts of that path that are local to one rank:
 *
 *   forward   fsdp_ag_pack    fp32 shards  -> bf16 send chunk       (copy-in)
 *             [all-gather of the chunks: not part of this library]
 *             fsdp_ag_unpack  gathered W chunks -> full bf16 params (copy-out)
 *   backward  fsdp_rs_pack    full bf16 grads -> W destination chunks (copy-in)
 *             [exchange of the chunks: not part of this library]
 *             fsdp_rs_reduce  W received chunks -> fp32 grad shards (average + read-out)
 *
 * World size W is a layout parameter of the plan; no call communicates.
 *
 * Notation (all sizes in elements):
 *   parameter p has shape (N_p, inner_p), row-major, inner_p = product of
 *   the trailing dims; c_p = ceil(N_p / W) rows per rank (torch.chunk split);
 *   rank r holds n_{p,r} = min(c_p, max(0, N_p - r*c_p)) rows;
 *   L_p = c_p * inner_p; off_0 = 0, off_{p+1} = roundup(off_p + L_p, A);
 *   S = roundup(off_{P-1} + L_{P-1}, A) is one rank's chunk.
 *   Pad rows, alignment gaps and the tail of every chunk are written as +0.
 *
 * Conventions for every call:
 *   - Device pointers are HIP device memory on the current device.  The
 *     caller owns every buffer and every host pointer array; the library owns
 *     only plans.  The hot calls allocate nothing, never synchronise, and
 *     enqueue exactly one kernel on `stream` (0 = the null stream), or none
 *     when there is nothing to write (the push at W >= 8: two).
 *   - All arguments are validated on the host before any HIP call; on any
 *     error nothing is enqueued and no output is touched.
 *   - Bucket buffers (send_chunk, gathered, send_buf, recv) must be 16-byte
 *     aligned.  Per-parameter pointers need only element alignment (4 bytes
 *     for fp32, 2 for bf16); unaligned ones take a slower element-wise path.
 *     A per-parameter pointer may be NULL only when it has no elements.
 *   - Outputs must not overlap inputs or each other (checked on the host).
 *   - A plan is needed only while a call runs: the kernel arguments are
 *     copied at launch, so the plan may be freed once the call returns, even
 *     with its launches still in flight.  Plans are immutable and may be
 *     shared between threads and streams.
 *   - bf16 values are passed as uint16_t bit patterns.
 *   - A launch uses one workgroup per work tile, up to a per-device cap;
 *     past the cap every workgroup loops over several tiles.  The reduction
 *     cuts a small shard (fewer than 4 full-size tiles per CU) into
 *     half-size tiles.  A plan made by fsdp_bucket_plan_ex may lower the cap
 *     or force the tile size; results never depend on either.
 */
#ifndef FSDP_BUCKET_H
#define FSDP_BUCKET_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t fsdp_status;

enum {
    FSDP_OK = 0,
    FSDP_ERR_INVALID = 1,   /* bad argument value, NULL where data is needed, unknown plan */
    FSDP_ERR_ALIGN = 2,     /* bucket buffer not 16-byte aligned, or element misalignment */
    FSDP_ERR_OVERFLOW = 3,  /* a size does not fit the library's 64-bit / tile limits */
    FSDP_ERR_TOO_MANY = 4,  /* more than FSDP_MAX_PARAMS parameters, or W > FSDP_MAX_CHUNKS in a chunk table */
    FSDP_ERR_NOMEM = 5,     /* host allocation of a plan failed */
    FSDP_ERR_HIP = 6,       /* the HIP runtime reported an error at launch */
    FSDP_ERR_OVERLAP = 7    /* an output overlaps an input or another output */
};

/* Parameters per bucket: the per-parameter table travels in the kernel
 * arguments (a Llama block has 9 parameters). */
#define FSDP_MAX_PARAMS 64

/* World size limit of the chunk-table entry points (*_ex), whose W chunk
 * pointers also travel in the kernel arguments. */
#define FSDP_MAX_CHUNKS 128

/* Element types of the *_ex entry points (section 4: param_dtype and
 * reduce_dtype).  BF16 and F16 (IEEE binary16) are the two 16-bit floats;
 * fp32 -> 16-bit casts round to nearest even (NaN -> a NaN), 16-bit -> fp32
 * is exact. */
typedef int32_t fsdp_dtype;
enum { FSDP_DTYPE_BF16 = 0, FSDP_DTYPE_F32 = 1, FSDP_DTYPE_F16 = 2 };

typedef struct fsdp_plan fsdp_plan;

/*
 * Plan a bucket (section 3.2.1: the bucket flattens and concatenates the
 * parameters; section 3.1: each is sharded on dim 0 over W ranks).
 *   world_size   W >= 1
 *   num_params   1 <= P <= FSDP_MAX_PARAMS
 *   dim0[P]      N_p >= 0 (host array)
 *   inner[P]     inner_p >= 1 (host array)
 *   align_elems  A, a power of two; 8 (16 bytes of bf16) enables the vector
 *                path, 1 gives the dense concatenation
 *   out          receives the plan (host memory owned by the library)
 * Errors: FSDP_ERR_INVALID, FSDP_ERR_TOO_MANY, FSDP_ERR_OVERFLOW
 * (N_p*inner_p, W*S or any byte size reaching 2^62, or more than 2^31-1
 * kernel tiles), FSDP_ERR_NOMEM.  Makes no HIP call.
 */
fsdp_status fsdp_bucket_plan(int32_t world_size, int32_t num_params,
                             const int64_t* dim0, const int64_t* inner,
                             int32_t align_elems, fsdp_plan** out);

/* Launch options of a plan (fsdp_bucket_plan_ex).  They change how the work
 * is cut into workgroups, never a result bit. */
enum {
    FSDP_REDUCE_TILES_AUTO = 0,   /* half-size tiles below 4 full-size tiles per CU */
    FSDP_REDUCE_TILES_FULL = 1,   /* always 256-thread tiles */
    FSDP_REDUCE_TILES_HALF = 2    /* always 128-thread tiles */
};
typedef struct fsdp_plan_options {
    int64_t max_workgroups;   /* > 0: no launch of the plan has a larger grid
                                 (workgroups loop over tiles); 0: the default */
    int32_t reduce_tiles;     /* FSDP_REDUCE_TILES_*; 0 is the default */
    int32_t reserved;         /* must be 0 */
} fsdp_plan_options;

/* fsdp_bucket_plan with launch options (NULL = all defaults), fixed for the
 * plan's lifetime.  Errors: those of fsdp_bucket_plan, and FSDP_ERR_INVALID
 * for a negative max_workgroups, an unknown reduce_tiles or a non-zero
 * reserved field.  Makes no HIP call. */
fsdp_status fsdp_bucket_plan_ex(int32_t world_size, int32_t num_params,
                                const int64_t* dim0, const int64_t* inner,
                                int32_t align_elems, const fsdp_plan_options* options,
                                fsdp_plan** out);

/* Release a plan (NULL is ignored). */
void fsdp_plan_free(fsdp_plan* plan);

/* S, the elements of one rank's chunk; -1 for an unknown plan. */
int64_t fsdp_plan_chunk_elems(const fsdp_plan* plan);

/* W and P of a plan; -1 for an unknown plan. */
int32_t fsdp_plan_world_size(const fsdp_plan* plan);
int32_t fsdp_plan_num_params(const fsdp_plan* plan);

/* c_p, off_p and L_p of parameter p (any output pointer may be NULL). */
fsdp_status fsdp_plan_param(const fsdp_plan* plan, int32_t p, int64_t* rows_per_rank,
                            int64_t* offset, int64_t* seg_elems);

/* n_{p,rank}, the rows of parameter p that rank holds; -1 on a bad argument. */
int64_t fsdp_plan_local_rows(const fsdp_plan* plan, int32_t p, int32_t rank);

/* Static description of a status code. */
const char* fsdp_status_str(fsdp_status status);

/* Detail of the last failed call on this thread ("" if none). */
const char* fsdp_last_error(void);

/*
 * Forward copy-in of rank `rank` (section 3.2.1, all-gather bucketing;
 * section 4, parameters cast to param_dtype = bf16 before the all-gather).
 *   shards[P]    host array of device pointers: rank's fp32 Shard(0) slab of
 *                each parameter, n_{p,rank} x inner_p, contiguous, unpadded
 *   send_chunk   device, S bf16 elements, 16-byte aligned; fully written:
 *                send_chunk[off_p + k] = bf16_rne(shards[p][k]) for
 *                k < n_{p,rank}*inner_p, +0 everywhere else
 * The cast is IEEE round-half-to-even; a NaN becomes the quiet NaN
 * (bits >> 16) | 0x0040 of the same sign.
 */
fsdp_status fsdp_ag_pack(const fsdp_plan* plan, int32_t rank,
                         const float* const* shards, uint16_t* send_chunk,
                         hipStream_t stream);

/*
 * Forward copy-out (section 3.2.1: gathered data copied out by each
 * parameter's original size).
 *   gathered     device, W*S bf16, rank-major (chunk i at gathered + i*S),
 *                16-byte aligned; only valid rows are read
 *   params[P]    host array of device pointers: full bf16 parameter p,
 *                N_p x inner_p, written as
 *                params[p][row*inner_p + col] =
 *                  gathered[(row / c_p)*S + off_p + (row % c_p)*inner_p + col]
 */
fsdp_status fsdp_ag_unpack(const fsdp_plan* plan, const uint16_t* gathered,
                           uint16_t* const* params, hipStream_t stream);

/*
 * Backward copy-in (section 3.2.1, reduce-scatter bucketing: each gradient
 * split into W chunks, chunks concatenated per destination).
 *   grads[P]     host array of device pointers: full bf16 gradient of
 *                parameter p, N_p x inner_p
 *   send_buf     device, W*S bf16, destination-major, 16-byte aligned; fully
 *                written: send_buf[j*S + off_p + k] = grads[p][j*L_p + k] when
 *                row j*c_p + k/inner_p < N_p, +0 otherwise (pad rows, gaps,
 *                tail)
 */
fsdp_status fsdp_rs_pack(const fsdp_plan* plan, const uint16_t* const* grads,
                         uint16_t* send_buf, hipStream_t stream);

/*
 * Rank-local average and read-out of rank `rank` (section 3.2.1: the bucket
 * is averaged across ranks and the gradients are read out; section 4: the
 * reduction runs in reduce_dtype = fp32; Partial("avg") -> Shard(0)).
 *   recv         device, W*S bf16, source-major (chunk from rank i at
 *                recv + i*S), 16-byte aligned; only valid rows are read
 *   grad_shards[P]  host array of device pointers: fp32 output, n_{p,rank} x
 *                inner_p each, written as
 *                a = x_0; a = fl32(a + x_i) for i = 1..W-1; out = fl32(a / W)
 *                with x_i = recv[i*S + off_p + k] widened exactly to fp32,
 *                additions in rank order, a correctly rounded division and
 *                subnormals kept.  A NaN among the x_i gives a NaN output;
 *                which NaN (its payload) is left open, as IEEE 754 leaves it.
 */
fsdp_status fsdp_rs_reduce(const fsdp_plan* plan, int32_t rank, const uint16_t* recv,
                           float* const* grad_shards, hipStream_t stream);

/*
 * ---------------------------------------------------------------------------
 * Element-type and chunk-table forms.
 *
 * These generalise the four calls above in two ways:
 *   - the element type on the wire: param_dtype = fp32 trains without mixed
 *     precision, and reduce_dtype = fp32 casts the gradients to fp32 before
 *     the reduce-scatter.  Section 4 makes both dtypes parameters of the
 *     redistribute; mixed precision is the bf16/fp32 setting.
 *   - the bucket buffers as W separate chunks.  chunks[i] points at rank i's
 *     chunk of S elements, so an exchange can be fused with the copy: pull
 *     the gathered chunks straight from the peers' send chunks, push each
 *     destination's chunk straight into that peer's receive buffer, pull
 *     the W received chunks from the peers' send buffers, or push one
 *     packed chunk into every peer's gathered buffer.
 * Layouts, zero filling, numerics and error behaviour are those of the
 * calls above; chunks[] is a host array of W <= FSDP_MAX_CHUNKS device
 * pointers, each 16-byte aligned.  Errors: as above, plus FSDP_ERR_TOO_MANY
 * for W > FSDP_MAX_CHUNKS and FSDP_ERR_INVALID for an unknown dtype.
 * ---------------------------------------------------------------------------
 */

/* fsdp_ag_pack with param_dtype BF16 or F16 (the cast) or F32 (a bit copy
 * of the fp32 shards).  send_chunk holds S elements of param_dtype. */
fsdp_status fsdp_ag_pack_ex(const fsdp_plan* plan, int32_t rank, const float* const* shards,
                            fsdp_dtype param_dtype, void* send_chunk, hipStream_t stream);

/* fsdp_ag_pack_ex pushing the packed chunk to W destinations: chunks[i] is
 * where rank i receives this rank's chunk (slot `rank` of rank i's gathered
 * buffer), so the one-shot all-gather is fused with the copy-in.  Each of the
 * W chunks receives the same S elements of param_dtype; the shards are read
 * once.  The chunks must not overlap each other or the shards.  At W >= 8
 * the call enqueues two kernels: the pack into chunks[rank], then its copy to
 * the other W - 1 chunks (which reads chunks[rank] back); below 8, one. */
fsdp_status fsdp_ag_pack_push(const fsdp_plan* plan, int32_t rank, const float* const* shards,
                              fsdp_dtype param_dtype, void* const* chunks, hipStream_t stream);

/* fsdp_ag_unpack from W chunk pointers (rank i's chunk at chunks[i]); params
 * and chunks hold param_dtype elements. */
fsdp_status fsdp_ag_unpack_ex(const fsdp_plan* plan, fsdp_dtype param_dtype, const void* const* chunks,
                              void* const* params, hipStream_t stream);

/* fsdp_rs_pack into W chunk pointers (destination j's chunk at chunks[j]).
 * reduce_dtype is grad_dtype (a copy) or F32 (16-bit gradients widened
 * exactly); any other pair, such as F32 gradients on a 16-bit wire, would
 * be a rounding step and is refused (FSDP_ERR_INVALID). */
fsdp_status fsdp_rs_pack_ex(const fsdp_plan* plan, fsdp_dtype grad_dtype, const void* const* grads,
                            fsdp_dtype reduce_dtype, void* const* chunks, hipStream_t stream);

/* fsdp_rs_reduce from W chunk pointers (source i's chunk at chunks[i]) of
 * reduce_dtype elements; the sum and division are as in fsdp_rs_reduce. */
fsdp_status fsdp_rs_reduce_ex(const fsdp_plan* plan, int32_t rank, fsdp_dtype reduce_dtype,
                              const void* const* chunks, float* const* grad_shards, hipStream_t stream);

/*
 * ---------------------------------------------------------------------------
 * Auto-wrapping (section 3.3.2 "Auto-wrapping": Algorithm 1, the variables
 * of Table 1, and the profiling model T_m = alpha + beta * n).  Host code:
 * no HIP call, no device memory.
 *
 * Cuts one pass's all-gather nodes, given in the order the pass computes
 * them, into consecutive buckets B_0, B_1, ...; step k computes B_k while
 * the all-gather of B_{k+1} is in flight and, in the backward pass, the
 * reduce-scatter of B_{k-1}.  Node i joins the bucket being built (B_{k+1})
 * exactly when
 *   forward   alpha_ag + beta_ag * (words(B_{k+1}) + ag_words[i]) <= T_c
 *   backward  T_rs + alpha_ag + beta_ag * (words(B_{k+1}) + ag_words[i]) <= T_c
 *   and       mem(B_{k+1}) + compute_mem[i] <= mem_max,
 * where T_c is the sum of compute_time over B_k (0 for the first bucket,
 * which therefore holds one node unless communication is free), mem() sums
 * compute_mem, and T_rs = alpha_rs + beta_rs * (rs_words summed over
 * B_{k-1}), 0 while there is no B_{k-1}.  Otherwise node i starts the next
 * bucket.  Sums of times run in node order from 0.0 in binary64; each
 * alpha + beta * n rounds the product and the sum separately.
 *
 *   num_nodes     n >= 0
 *   backward      0 = forward pass, 1 = backward pass
 *   ag_words      host [n], >= 0: words each node's all-gather moves (n_i)
 *   rs_words      host [n], >= 0: words of its gradient's reduce-scatter;
 *                 read in the backward pass only (may be NULL otherwise)
 *   compute_time  host [n], finite, >= 0: T_ci, in the unit of alpha/beta
 *   compute_mem   host [n], >= 0: M_ci (e.g. bytes)
 *   alpha_*, beta_*  finite, >= 0: the collectives' cost model
 *   mem_max       >= 0: M_max, in the unit of compute_mem
 *   bucket_of     host [n], out: the bucket number of every node
 *                 (0-based, non-decreasing, steps of 0 or 1)
 *   num_buckets   out: the number of buckets (0 when n = 0)
 * Errors: FSDP_ERR_INVALID for a NULL array, a negative or non-finite
 * value, or backward not 0/1; FSDP_ERR_OVERFLOW when the words of either
 * kind sum above 2^53 or the memories overflow int64.  On error no output
 * is written.  The call keeps no state and is thread-safe.
 */
fsdp_status fsdp_auto_wrap(int32_t num_nodes, int32_t backward, const int64_t* ag_words,
                           const int64_t* rs_words, const double* compute_time,
                           const int64_t* compute_mem, double alpha_ag, double beta_ag,
                           double alpha_rs, double beta_rs, int64_t mem_max,
                           int32_t* bucket_of, int32_t* num_buckets);

#ifdef __cplusplus
}
#endif

#endif /* FSDP_BUCKET_H */
