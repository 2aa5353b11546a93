/*
 * mla_sparse.h -- C ABI of libmla_sparse.so: sparse absorbed-MLA partial
 * attention (the holder side of routing the query) and the log-sum-exp merge
 * of partials (the requester side), on an AMD Instinct MI355X (gfx950).
 *
 * Method: "Move the Query, Not the Cache" (arXiv 2606.01502).  A requester
 * ships absorbed-MLA query rows, each d_qk = 576 wide (a 512-wide latent part
 * and a 64-wide decoupled-RoPE part), to the instance holding a cached chunk;
 * the holder attends them over the chunk's latent cache that it keeps in
 * memory and returns a d_v = 512 wide partial output together with softmax
 * statistics from which the requester can recombine partials exactly
 * (Section 3.2, wire format).  Under sparse selection the holder attends only
 * the entries the indexer picked, each at the position it was cached at
 * (Sections 3.3, 5.4, 6.3).  The requester recombines partials by
 * online softmax; the merge is commutative and has a zero-weight identity
 * (Sections 2.2 and 3.3).
 *
 * Conventions shared by every entry point
 *   - Tensors are passed as mla_tensor_t descriptors.  `data` is a DEVICE
 *     pointer owned by the caller; the library never frees or keeps it past
 *     the work it enqueues.  Descriptors and pointer arrays are read during
 *     the call only and may be freed when it returns.
 *   - Every call enqueues its kernels on `stream` (a hipStream_t; NULL is the
 *     legacy default stream) and returns without synchronising.  Outputs are
 *     valid once the stream reaches the enqueued work.  Inputs and outputs
 *     must stay allocated until then.
 *   - Calls return MLA_OK or a negative status.  Problems the host can see
 *     (null pointers, dtypes, shapes, strides, alignment, aliasing) return
 *     before anything is enqueued and write nothing; mla_last_error() then
 *     describes the problem.  No C++ exception crosses the ABI.
 *   - Device memory for split-K partials is allocated by the library on first
 *     need and reused (one grow-only buffer per device and stream; see
 *     "Split-K workspace" below).  Calls on different streams are
 *     independent; calls on one stream are ordered by the stream.
 */
#ifndef MLA_SPARSE_H
#define MLA_SPARSE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MLA_SPARSE_VERSION 4

#define MLA_DLAT 512  /* latent width = d_v (Section 3.2)                    */
#define MLA_DPE 64    /* decoupled-RoPE width = d_qk - d_v (Section 3.2)      */
#define MLA_BLOCK 64  /* tokens per selectable cache block                   */
#define MLA_MAX_PARTS 64

typedef enum {
  MLA_OK = 0,
  MLA_ERR_INVALID_ARGUMENT = -1, /* null pointer, dtype, shape, stride, alignment, aliasing */
  MLA_ERR_UNSUPPORTED = -2,      /* valid request this build does not implement       */
  MLA_ERR_HIP = -3,              /* a HIP runtime call or a kernel launch failed      */
  MLA_ERR_OUT_OF_MEMORY = -4     /* the split-K workspace could not be allocated      */
} mla_status_t;

typedef enum {
  MLA_DTYPE_BF16 = 1,
  MLA_DTYPE_FP8_E4M3FN = 2, /* OCP E4M3FN: bias 7, max 448, no infinities */
  MLA_DTYPE_FP32 = 3,
  MLA_DTYPE_INT32 = 4
} mla_dtype_t;

/* A strided view of device memory.  shape/stride beyond ndim are ignored;
 * strides are in elements and the innermost stride must be 1. */
typedef struct {
  void* data;               /* device pointer, owned by the caller             */
  int32_t dtype;            /* mla_dtype_t                                     */
  int32_t ndim;             /* 1..4                                            */
  int64_t shape[4];
  int64_t stride[4];
  const float* block_scale; /* fp8 cache pools only: device pointer to [P] fp32
                               per-64-token-block scales (value = code * scale);
                               must be NULL for every other tensor             */
} mla_tensor_t;

/*
 * Sparse absorbed-MLA partial attention (the holder's partial, Sections 3.2,
 * 3.3, 6.3).  R independent jobs (one per (request, chunk)); job r has
 * Mq x H query rows that all share one selection of 64-token blocks.
 *
 *   q_lat             [R_q, Mq, H, 512] bf16 latent part of the absorbed query
 *   q_pe              [R_q, Mq, H, 64]  bf16 decoupled-RoPE part (already rotated
 *                                            by the requester; no rotation here)
 *                                     R_q = R (a q per job), or any R_q dividing
 *                                     R: job r then reads q row r mod R_q, so a
 *                                     request routed to several chunks of this
 *                                     holder (jobs b, b + R_q, ... in slot-major
 *                                     order) sends its q once; those jobs are
 *                                     scheduled next to each other
 *   ckv_pool          [P, 64, 512]    bf16 or fp8-e4m3fn (+block_scale), contiguous
 *   kpe_pool          [P, 64, 64]     same dtype as ckv_pool, contiguous
 *                                     fp8: both descriptors carry a block_scale;
 *                                     passing the same array for both (one scale
 *                                     per block for the whole 576-wide entry) is
 *                                     the fast layout, two arrays (separate
 *                                     latent and RoPE scales) are also accepted.
 *                                     Scales must be finite; 0 is allowed (the
 *                                     block's values are then 0).  With two
 *                                     arrays, a block whose latent scale is 0 or
 *                                     below 2^-64 of its RoPE scale has its
 *                                     latent score part weighted by 2^-64 times
 *                                     the RoPE scale instead (an absolute score
 *                                     error of at most 2^-63 |RoPE scale| |q_lat .
 *                                     latent codes|); its values keep the latent
 *                                     scale.
 *   chunk_block_table [R, NB] int32   logical block of job r's chunk -> pool block
 *   sel_block_ids     [R, K]  int32   selected logical blocks; -1 marks an empty
 *                                     slot; a block listed twice counts twice
 *                 or  [R, Mq, K] int32   one selection per query row: a holder
 *                                     serving Mq routed requesters (or query
 *                                     rows) on the job's chunk, each with its
 *                                     own selection (Section 6.3).  Blocks that
 *                                     several rows select are read once for
 *                                     all of them.  NB times
 *                                     the query rows one row tile spans (128
 *                                     rows, or 64 when 128 would span more
 *                                     than 64 query rows) must not exceed
 *                                     73696 (MLA_ERR_UNSUPPORTED)
 *   scale                              multiplies q_lat.ckv + q_pe.kpe: any
 *                                     value with |scale| <= 2^64 (0 weights
 *                                     every token alike), else
 *                                     MLA_ERR_INVALID_ARGUMENT.  Scores are
 *                                     formed in fp32: the result is defined
 *                                     while |q_lat.ckv + q_pe.kpe| < 2^63 for
 *                                     every selected token (bf16 products
 *                                     accumulated in fp32)
 *   out_lat           [R, Mq, H, 512] fp32   written: normalised partial output
 *   out_lse           [R, Mq, H]      fp32   written: natural-log log-sum-exp
 *                 (with opts.out_format = MLA_OUT_BF16_WIRE, the wire form of
 *                 Section 3.2, 1032 bytes per row: out_lat [R, Mq, H, 512]
 *                 bf16, the normalised output rounded to nearest even, and
 *                 out_lse [R, Mq, H, 2] fp32 holding (m, l): the largest score
 *                 m of the row's tokens and l = sum_T exp(s_t - m), so that
 *                 out_lse = m + ln l; an empty T gives (-inf, 0))
 *
 * For each row, with T the multiset of tokens of the blocks selected for it
 * (by its job, or by its query row),
 *   s_t = scale * (q_lat . ckv_t + q_pe . kpe_t),
 *   out_lse = ln sum_T exp(s_t),   out_lat = sum_T exp(s_t - out_lse) * ckv_t,
 * and for an empty T: out_lat = 0, out_lse = -inf.  No mask, no positions.
 *
 * Layout: q and out rows may be strided on the R, Mq and H dims (16-byte
 * aligned rows); pools must be contiguous and 16-byte aligned.  Slot order
 * does not change the result beyond rounding.  A selected id outside
 * [0, NB), or a table entry outside [0, P), is a caller error that this call
 * does not detect on the host: such a slot is skipped (treated as empty).
 *
 * Split-K workspace: when a job is split, the library keeps one grow-only
 * device buffer per (device, stream), allocated on first need
 * (MLA_ERR_OUT_OF_MEMORY if that fails).  A larger need allocates a new
 * buffer of at least twice the size; the old one is kept, not freed, until
 * the process ends, so a HIP graph captured with it stays valid.  Calls may
 * come from several host threads, also on one stream: each call queues its
 * two kernels without another call's kernels between them.
 * Graph capture: a call captured on a stream uses that stream's workspace
 * as it was at capture time.  The workspace cannot grow while the stream is
 * being captured (MLA_ERR_UNSUPPORTED): make the same call, or a larger one,
 * on the stream before capturing.  Replay the graph on the stream it was
 * captured on, or keep other calls on that stream from running at the same
 * time as the replay (they share the buffer).  Under global-mode capture,
 * a call on another stream that has to grow its workspace allocates device
 * memory, which that capture mode forbids.
 */
mla_status_t mla_sparse_partial_attn(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                     const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                                     const mla_tensor_t* chunk_block_table,
                                     const mla_tensor_t* sel_block_ids, float scale,
                                     const mla_tensor_t* out_lat, const mla_tensor_t* out_lse,
                                     void* stream);

/* Tuning and test controls for mla_sparse_partial_attn_ex.  Zero fields mean
 * "library's choice"; the result is the same up to rounding for any value. */
typedef struct {
  /* split-K: work splits per job (0 = automatic).  A shared selection, or
   * per-row selections whose K slots times the query rows of a row tile
   * exceed 1024, split into ranges of slots (1..K); other per-row selections
   * split by logical block, split s taking blocks s, s + n, s + 2n, ...
   * (1..NB). */
  int32_t n_splits;
  /* rows per work item: 64 or 128 (0 = automatic: 128 when Mq * H > 64 and
   * the splits are long, else 64). */
  int32_t row_tile;
  /* output form: MLA_OUT_FP32 (0) or MLA_OUT_BF16_WIRE (see the partial
   * call's out_lat / out_lse). */
  int32_t out_format;
  int32_t reserved[5]; /* must be zero */
} mla_partial_opts_t;

enum { MLA_OUT_FP32 = 0, MLA_OUT_BF16_WIRE = 1 };

/* mla_sparse_partial_attn with explicit options (opts may be NULL). */
mla_status_t mla_sparse_partial_attn_ex(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                        const mla_tensor_t* ckv_pool,
                                        const mla_tensor_t* kpe_pool,
                                        const mla_tensor_t* chunk_block_table,
                                        const mla_tensor_t* sel_block_ids, float scale,
                                        const mla_tensor_t* out_lat, const mla_tensor_t* out_lse,
                                        const mla_partial_opts_t* opts, void* stream);

/*
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, serving loops that must not call hipMalloc, harnesses that
 * forbid allocation.  mla_sparse_partial_attn_ex with the same arguments,
 * layout rules, result and errors, except that its split-K workspace is a
 * static device array of MLA_NOALLOC_SCRATCH_BYTES (64 MiB) that the library
 * holds on each GPU it runs on until the process ends, instead of memory it
 * allocates.  The call allocates nothing (no hipMalloc, no allocating library
 * routine).  A call whose split partials need more than the array (about
 * 64K partial rows, jobs x row tiles x splits x 128 rows, once they are
 * stored as scaled fp16, which they are from a megabyte of fp32 rows on;
 * about 32K below that) returns
 * MLA_ERR_UNSUPPORTED before anything is enqueued.  Every call on one GPU
 * shares that GPU's array: calls that overlap in time on one GPU (on
 * different streams, or from graphs replayed concurrently) race on it and
 * must be ordered by the caller; calls on one stream are ordered by the
 * stream.  Nothing in the array needs clearing between calls (each call
 * writes every workspace entry it reads).
 */
#define MLA_NOALLOC_SCRATCH_BYTES (64ll << 20)
mla_status_t mla_sparse_partial_attn_noalloc(const mla_tensor_t* q_lat,
                                             const mla_tensor_t* q_pe,
                                             const mla_tensor_t* ckv_pool,
                                             const mla_tensor_t* kpe_pool,
                                             const mla_tensor_t* chunk_block_table,
                                             const mla_tensor_t* sel_block_ids, float scale,
                                             const mla_tensor_t* out_lat,
                                             const mla_tensor_t* out_lse,
                                             const mla_partial_opts_t* opts, void* stream);

/*
 * The same partial attention over single selected tokens: an indexer's top-k
 * tokens of the chunk (the selection budgets of Section 6.3, k = 512 .. 2048
 * attended entries) rather than whole 64-token blocks.
 *
 *   sel_token_ids     [R, K]  int32   selected logical tokens of job r's chunk:
 *                                     id s names token s % 64 of logical
 *                                     block s / 64, i.e. pool token
 *                                     chunk_block_table[r, s / 64] * 64 + s % 64;
 *                                     -1 marks an empty slot; a token listed
 *                                     twice counts twice
 *
 * Every other argument, the result (T = the multiset of selected tokens)
 * and the layout rules are those of mla_sparse_partial_attn_ex; opts.n_splits
 * counts splits of the token slots (each split takes whole 64-token groups
 * of slots, at most 1024 slots).  bf16 or fp8 caches (a token takes the
 * scales of its pool block); NB and P must not exceed 2^25 blocks
 * (MLA_ERR_UNSUPPORTED).  An id
 * outside [0, 64 NB), or a table entry outside [0, P), is a caller error that
 * the call does not detect on the host: such a slot is skipped.
 */
mla_status_t mla_sparse_partial_attn_tokens(const mla_tensor_t* q_lat, const mla_tensor_t* q_pe,
                                            const mla_tensor_t* ckv_pool,
                                            const mla_tensor_t* kpe_pool,
                                            const mla_tensor_t* chunk_block_table,
                                            const mla_tensor_t* sel_token_ids, float scale,
                                            const mla_tensor_t* out_lat,
                                            const mla_tensor_t* out_lse,
                                            const mla_partial_opts_t* opts, void* stream);

/*
 * Log-sum-exp merge of n_parts partials of the same rows (the requester's
 * online-softmax recombination, Sections 2.2, 3.3 and 4.2).
 *
 *   out_lat[j]  [B, Mq, H, 512] fp32  normalised partial outputs, j < n_parts
 *   out_lse[j]  [B, Mq, H]      fp32  their natural-log log-sum-exps
 *   n_parts     1..MLA_MAX_PARTS
 *   out         [B, Mq, H, 512] fp32  written
 *
 * Per row, over the live parts (lse != -inf): L = max lse_j,
 * lse = L + ln sum exp(lse_j - L), out = sum exp(lse_j - lse) * out_lat[j].
 * A part whose lse is -inf is skipped whatever its out_lat holds (even NaN);
 * if no part is live the row is 0.  The parts may live anywhere but must
 * share one set of strides; out may not overlap any input.
 * Parts in the bf16 wire form (Section 3.2; see mla_partial_opts_t
 * out_format) are accepted too: out_lat[j] [B, Mq, H, 512] bf16 with
 * out_lse[j] [B, Mq, H, 2] fp32 pairs (m, l), whose lse is m + ln l (-inf
 * when l = 0); every part must then be in that form.  out stays fp32.
 */
mla_status_t mla_merge_partials(const mla_tensor_t* const* out_lat,
                                const mla_tensor_t* const* out_lse, int32_t n_parts,
                                const mla_tensor_t* out, void* stream);

/* As mla_merge_partials, and also writes the merged log-sum-exp to
 * merged_lse ([B, Mq, H] fp32, -inf for rows with no live part) unless it is
 * NULL.  Merging merged partials again is exact (the merge is associative). */
mla_status_t mla_merge_partials_ex(const mla_tensor_t* const* out_lat,
                                   const mla_tensor_t* const* out_lse, int32_t n_parts,
                                   const mla_tensor_t* out, const mla_tensor_t* merged_lse,
                                   void* stream);

/* Text describing the last non-OK status returned on the calling thread
 * ("" if none).  Owned by the library; valid until the thread's next call. */
const char* mla_last_error(void);

/* MLA_SPARSE_VERSION of the loaded library. */
int32_t mla_version(void);

/*
 * FETCH-side copies on one GPU (Section 2.2): what the move-the-cache
 * primitive does with the latent cache instead of routing the query.  Both
 * run every layer of a chunk in one launch.  Pools hold L layers,
 * [L, P, 64, 512] and [L, P, 64, 64] bf16, contiguous, 16-byte aligned.
 *
 * mla_fetch_gather: the scattered gather of a selected token set into a
 * contiguous payload (FETCH's residual work under sparse selection).
 *   chunk_block_table [NB] int32    logical block of the chunk -> pool block
 *   sel_token_ids     [K]  int32    logical tokens (block * 64 + t); -1 = empty
 *   out_ckv [L, K, 512], out_kpe [L, K, 64] bf16, written: entry j is pool
 *                                   token table[s / 64] * 64 + s % 64 of slot
 *                                   j's id s, copied bit for bit; an empty
 *                                   slot, an id outside [0, 64 NB) or a table
 *                                   entry outside [0, P) gives a zero row
 */
mla_status_t mla_fetch_gather(const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                              const mla_tensor_t* chunk_block_table,
                              const mla_tensor_t* sel_token_ids, const mla_tensor_t* out_ckv,
                              const mla_tensor_t* out_kpe, void* stream);

/* mla_fetch_splice: scatter a pulled chunk into the requester's paged pools,
 * re-homed at a new position.
 *   chunk_ckv [L, n, 512], chunk_kpe [L, n, 64] bf16   the chunk, token t
 *   ckv_pool, kpe_pool                                 written in place
 *   block_table [NB] int32    the requester's logical blocks -> pool blocks
 *   dst_start                 position of token 0 in the requester's
 *                             sequence: token t goes to row (dst_start + t)
 *                             % 64 of block block_table[(dst_start + t) / 64];
 *                             dst_start + n <= 64 NB
 *   delta                     positions the chunk moves (new - old start)
 *   rope_base, pairing        the RoPE layout (a reading; the paper gives
 *                             none): pair i turns at rope_base^(-2i/64);
 *                             pairing 0 pairs dims (2i, 2i+1), 1 pairs
 *                             (i, i+32)
 * The latent row is copied bit for bit; each RoPE pair (x, y) becomes
 * (x cos a - y sin a, x sin a + y cos a), a = delta * rope_base^(-2i/64)
 * (cos and sin in double on the host, the products in fp32, one rounding
 * to bf16).  A token whose table entry is outside [0, P) is skipped; no
 * other pool row is touched. */
mla_status_t mla_fetch_splice(const mla_tensor_t* chunk_ckv, const mla_tensor_t* chunk_kpe,
                              const mla_tensor_t* ckv_pool, const mla_tensor_t* kpe_pool,
                              const mla_tensor_t* block_table, int64_t dst_start, int64_t delta,
                              float rope_base, int32_t pairing, void* stream);

/*
 * The closed-form cost model of the three redistribution primitives and the
 * selection predicate (Sections 4.1-4.2 and 5.1-5.2).  Host-only arithmetic:
 * no device, no stream; a scheduler evaluates it per (chunk, request).
 * Times in microseconds, throughputs in GB/s (1e9 bytes per second), sizes
 * in bytes.  The paper's measured constants are given in brackets.
 */
typedef struct {
  double probe_us;     /* T_probe(F): the fabric's signalled round trip [16]      */
  double route_bw_gbs; /* BW(F): routing's effective bidirectional throughput [25] */
  double compute_us;   /* T_compute: the holder's partial attention (0: transport
                          only, as the paper's fitted round trip)                */
  double merge_us;     /* T_merge: the requester's merge (0: transport only)      */
  double pull_bw_gbs;  /* FETCH's bulk pull throughput [25]                       */
  double splice_us;    /* T_splice: FETCH's position adaptation [3000]; 0 under
                          sparse selection                                       */
  double prefill_us;   /* c: LOCAL's re-prefill cost per token and layer
                          [0.5 .. 1.5]                                           */
  int32_t layers;      /* L: layers FETCH pulls and LOCAL re-prefills [27]        */
  int32_t reserved;    /* must be zero                                           */
} mla_cost_model_t;

typedef struct {
  int64_t mq;           /* Mq: query rows routed to the chunk                    */
  int64_t chunk_tokens; /* c_t: tokens of the chunk                               */
  int64_t q_bytes;      /* q: bytes per routed query row [576 x 2 = 1152]         */
  int64_t p_bytes;      /* p: bytes per returned partial row [512 x 2 + 2 x 4 =
                           1032]                                                  */
  int64_t kv_bytes;     /* b_KV: cached bytes per token and layer [1152]          */
} mla_cost_case_t;

enum { MLA_PRIMITIVE_ROUTE = 0, MLA_PRIMITIVE_FETCH = 1, MLA_PRIMITIVE_LOCAL = 2 };

typedef struct {
  double route_us;  /* T_probe + Mq (q + p) / BW + T_compute + T_merge            */
  double fetch_us;  /* L c_t b_KV / pull BW + T_splice                            */
  double local_us;  /* c_t L c                                                     */
  int32_t choice;   /* the argmin: MLA_PRIMITIVE_*; ties go to ROUTE, then FETCH   */
  int32_t reserved;
  double wire_crossover_mq;       /* Mq at which routing and pulling one layer move
                                     equal bytes: c_t b_KV / (q + p)               */
  double wire_saving;             /* 1 - Mq (q + p) / (c_t b_KV): the share of one
                                     layer's pull bytes routing does not move      */
  double congestion_bw_gbs;       /* BW below which routing's transfer exceeds the
                                     splice: Mq (q + p) / T_splice (inf if no
                                     splice)                                       */
  double splice_crossover_tokens; /* c_t above which the splice undercuts
                                     re-prefill: T_splice / (L c) (inf if c = 0)   */
} mla_cost_t;

/* Evaluate the model for one case.  MLA_ERR_INVALID_ARGUMENT for a null
 * pointer, a negative or non-finite constant, a non-positive throughput, a
 * negative size, layers < 1, chunk_tokens or kv_bytes of 0, or nonzero
 * reserved fields. */
mla_status_t mla_primitive_costs(const mla_cost_model_t* model, const mla_cost_case_t* c,
                                 mla_cost_t* out);

#ifdef __cplusplus
}
#endif

#endif /* MLA_SPARSE_H */
