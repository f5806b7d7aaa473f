/*
 * albireo.h -- C ABI of the MI355X (gfx950) per-sequence sampling library.
 *
 * The operation is the sampling step Y = Sample(Pr) of the paper's sequence-parallel sampling
 * (sec. 6.1, Eq. opt_sample): every rank holds a row-share Pr^s of the logits matrix at full
 * vocabulary width, samples each row independently, and consumes its slice of pre-generated random
 * numbers (sec. 6.2, "Deterministic random number generation").  The per-row features are the ones
 * the paper lists as enabled in its workload (sec. 8.1): repetition, frequency and presence
 * penalties, temperature, top-k, top-p (nucleus) and min-p, plus greedy decoding (sec. 2.1, T4).
 * The result per row is a token id and its log-probability (App. A, "update sequence" appends the
 * sampled id with its probability).
 *
 * Per row i the library computes, in this order (all fp32 except where noted):
 *   1. x = logits[i] (bf16 widened exactly).
 *   2. penalties over the row's history h_i (count c_v of token v in h_i):
 *        for c_v > 0:  x_v = x_v > 0 ? x_v / rep : x_v * rep;  x_v -= freq * c_v;  x_v -= pres.
 *   3. temperature T < 1e-5 => greedy: id = lowest index among the maxima of x; logprobs use T = 1.
 *      otherwise r = (float)(1 / (double)T), z_v = x_v * r (-0 -> +0; -inf stays -inf).
 *   4. m = max z, LSE = m + log sum_v exp(z_v - m) over the full vocabulary.
 *   5. min-p:  keep z >= m + (float)log(min(min_p, 1))            (when min_p > 0)
 *      top-k:  keep z >= the k-th largest z, ties kept            (when 0 < k < V)
 *      top-p:  over the kept set S2, renormalised, take whole groups of equal z in descending order
 *              until the cumulative mass reaches p                (when p < 1)
 *   6. id = first token in ascending id order whose cumulative probability over the kept set S
 *      exceeds u = uniforms[i]; logprob = z_id - LSE.
 *
 * Conventions for every entry point:
 *   - All array arguments are DEVICE pointers unless marked [host].  The caller owns every buffer.
 *   - Row-major logits [B, ld]; ld >= V elements; row i starts at logits + i * ld.  Rows need not be
 *     16-byte aligned; logits must be aligned to its element size.
 *   - All work is enqueued on `stream`; no entry point synchronises with the host, allocates or frees
 *     device memory.  Scratch memory comes from the caller's workspace.
 *   - Host-checkable problems return a non-OK status and enqueue nothing.  Problems that depend on
 *     device data produce a defined result and a per-row flag bit (ALBIREO_FLAG_*).
 *   - Results are bit-identical from run to run (no floating-point atomics), and identical for a row
 *     whether it is sampled alone or inside any batch as long as the row starts at the same address
 *     modulo 16 bytes (always the case when ld * element size is a multiple of 16 and the buffers are
 *     16-byte aligned): the reduction order is fixed by V, dtype and that alignment.
 */
#ifndef ALBIREO_H
#define ALBIREO_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { ALBIREO_F32 = 0, ALBIREO_BF16 = 1 } albireo_dtype_t;

typedef enum {
  ALBIREO_OK = 0,
  ALBIREO_E_INVALID = 1,     /* bad pointer, size, stride, dtype or n_top                       */
  ALBIREO_E_UNSUPPORTED = 2, /* shape this build does not handle (e.g. V >= 2^31)                */
  ALBIREO_E_WORKSPACE = 3,   /* workspace NULL, misaligned or smaller than albireo_workspace_size */
  ALBIREO_E_LAUNCH = 4,      /* the HIP runtime refused the launch                               */
  ALBIREO_E_SCRATCH = 5      /* albireo_sample_noalloc: the shape needs more device scratch than
                                ALBIREO_NOALLOC_SCRATCH_BYTES                                     */
} albireo_status_t;

/* Per-row flag bits written to out_flags. */
#define ALBIREO_FLAG_GREEDY 1u    /* temperature < 1e-5: argmax, uniform ignored                   */
#define ALBIREO_FLAG_EMPTY 2u     /* no finite logit: id = -1, logprob = -inf                      */
#define ALBIREO_FLAG_BAD_INPUT 4u /* NaN or +inf logit (after penalties/temperature), or a history id
                                     outside [0, V) (skipped); other outputs of the row unspecified  */
#define ALBIREO_FLAG_BAD_PARAM 8u /* malformed per-row parameter, replaced by its "off" value:
                                     temperature NaN or inf -> 1; rep <= 0, NaN or inf -> 1; freq/pres not
                                     finite -> 0; top_p NaN -> 1; min_p NaN -> 0; history offsets
                                     decreasing, negative or past hist_len -> no penalties        */
#define ALBIREO_FLAG_LIMIT 16u    /* a row's history has more distinct ids in one row chunk than
                                     this build handles on chip (ALBIREO_MAX_UNIQUE_HISTORY); the
                                     extra ids are ignored                                        */
#define ALBIREO_FLAG_TIMEOUT 32u  /* a bounded wait gave up (a value another workgroup or wave
                                     publishes never became visible within the spin limit); the
                                     row's other outputs are unspecified.  The waits: between the
                                     workgroups of a wide row (albireo_topk_topp, and the cooperative
                                     sampling route ALBIREO_ROUTE_COOPERATIVE), and, in the
                                     one-workgroup kernel, between the waves of a penalised row for
                                     its presence bitmap.  The streaming route never waits.       */

#define ALBIREO_MAX_TOP_N 32
#define ALBIREO_MAX_UNIQUE_HISTORY 2048

/*
 * Per-row sampling metadata (the paper's per-sequence metadata, sec. 3 Challenge 3 and sec. 6.2).
 * The struct itself lives in host memory and is read during the call only; every member is a device
 * pointer to a [B] array (or NULL, which turns the feature off for all rows).
 */
typedef struct {
  const float* temperature;        /* [B]  T < 1e-5 (incl. 0 and negatives) => greedy; NULL => 1  */
  const int32_t* top_k;            /* [B]  k <= 0 or k >= V => off                                 */
  const float* top_p;              /* [B]  p >= 1 => off; p <= 0 keeps the top group               */
  const float* min_p;              /* [B]  <= 0 => off; > 1 behaves as 1                           */
  const float* repetition_penalty; /* [B]  1 => off                                               */
  const float* frequency_penalty;  /* [B]  0 => off                                               */
  const float* presence_penalty;   /* [B]  0 => off                                               */
  const int64_t* hist_offsets;     /* [B+1] CSR row pointers into hist_ids; NULL => no penalties   */
  const int32_t* hist_ids;         /* [hist_len] token ids; ids outside [0, V) are skipped+flagged */
  int64_t hist_len;                /* [host value] number of entries in hist_ids                   */
  /* Optional prompt history.  When given, hist_* holds each row's generated (output) tokens only and
   * the penalties split as the OpenAI definition the paper cites for frequency and presence does:
   * the repetition penalty covers every id of the prompt or the output, the frequency and presence
   * penalties count the output only.  Without it hist_* feeds all three penalties. */
  const int64_t* prompt_offsets;   /* [B+1] CSR row pointers into prompt_ids, or NULL              */
  const int32_t* prompt_ids;       /* [prompt_len] token ids; ids outside [0, V) are skipped+flagged */
  int64_t prompt_len;              /* [host value] number of entries in prompt_ids                 */
  /* Optional per-sequence penalty state (below) in place of the histories: the rows' distinct ids
   * with their output counts and prompt marks, kept on the device from step to step.  When given,
   * hist_* and prompt_* must be NULL. */
  const struct albireo_penalty_state_s* state; /* [host] or NULL                                  */
} albireo_params_t;

/*
 * Per-sequence penalty state (host struct of device arrays, read during a call only).  Row i holds
 * the distinct token ids of its prompt and output in ids[i * cap + e], e < len[i], in ascending
 * order, with counts[i * cap + e] = the id's number of occurrences in the output (bits 0-30) and bit 31
 * set when the id occurs in the prompt.  Sampling from the state gives the same penalties as sampling
 * from the prompt and output histories it was built from, without re-counting H ids per call; the
 * state follows the sequence by albireo_penalty_state_append after every step.  Ids that find no free
 * entry are left out and set ALBIREO_FLAG_LIMIT in flags[i]; ids outside [0, V) are skipped and set
 * ALBIREO_FLAG_BAD_INPUT; malformed history offsets set ALBIREO_FLAG_BAD_PARAM.  The sampling entry
 * points copy flags[i] into out_flags[i].
 */
typedef struct albireo_penalty_state_s {
  int32_t cap;       /* [host value] entries per row, 1 .. ALBIREO_MAX_STATE_ENTRIES              */
  int32_t* ids;      /* [B, cap] device                                                          */
  uint32_t* counts;  /* [B, cap] device                                                          */
  int32_t* len;      /* [B] device                                                               */
  uint32_t* flags;   /* [B] device                                                               */
} albireo_penalty_state_t;

#define ALBIREO_MAX_STATE_ENTRIES 8192

/*
 * Build the state of B rows from their prompt and output histories (CSR as in albireo_params_t; either
 * may be NULL).  Overwrites ids, counts, len and flags of every row.  A row whose two histories hold
 * more than ALBIREO_MAX_STATE_ENTRIES ids in all keeps the state of their first that many (prompt
 * first) and sets ALBIREO_FLAG_LIMIT.
 */
albireo_status_t albireo_penalty_state_init(const albireo_penalty_state_t* state, int64_t B, int64_t V,
                                            const int64_t* prompt_offsets, const int32_t* prompt_ids,
                                            int64_t prompt_len, const int64_t* out_offsets,
                                            const int32_t* out_ids, int64_t out_len, hipStream_t stream);

/*
 * Fold one sampled token per row into the state (the step's output): ids[i] gains one output
 * occurrence; an id not yet in the row takes a new entry in order.  ids[i] outside [0, V) (an EMPTY
 * row's -1, padding rows) changes nothing.  Stream-ordered after the sampling call that produced ids.
 */
albireo_status_t albireo_penalty_state_append(const albireo_penalty_state_t* state, int64_t B, int64_t V,
                                              const int32_t* ids, hipStream_t stream);

/* Which kernels a sampling call takes (albireo_sample_route). */
typedef enum {
  ALBIREO_ROUTE_NONE = 0,          /* no kernel of this build takes the shape (ALBIREO_E_UNSUPPORTED) */
  ALBIREO_ROUTE_ONE_WORKGROUP = 1, /* one launch, one workgroup per row, the row held in registers    */
  ALBIREO_ROUTE_STREAM = 2,        /* a workgroup per row chunk, then one per row (six launches)     */
  ALBIREO_ROUTE_COOPERATIVE = 3    /* one cooperative launch of chunk workgroups (B x chunks >= 2^31) */
} albireo_route_t;

/*
 * The kernels albireo_sample, albireo_sample_step, albireo_sample_sharded (sharded != 0) and
 * albireo_sample_noalloc take for B rows of V logits of this dtype with these parameters.  Host only:
 * reads params (host struct, may be NULL; only whether a prompt history or a penalty state is given)
 * and makes no HIP call, so it works with no device present.  The choice depends on V, dtype and
 * whether a prompt history or a penalty state is given, and on B only when B x chunks reaches 2^31:
 * rows of 16 to 38 x 512 x 16 bytes take one workgroup each, other rows up to 64 x 4864 x 16 bytes
 * and rows with a prompt or a state take the streaming kernels.  ALBIREO_ROUTE_NONE for an invalid dtype, V <= 0, B < 0 or V at or
 * above 2^31 - 16.
 */
albireo_route_t albireo_sample_route(int64_t B, int64_t V, albireo_dtype_t dtype, const albireo_params_t* params,
                                    int32_t sharded);

/*
 * Bytes of device workspace needed by any entry point for this shape on the current device.
 * The workspace must be 256-byte aligned and zero-filled before its first use; every call leaves it
 * zero-filled again on return (stream order).  One workspace per stream: two calls that run
 * concurrently must not share one.  A call that returns ALBIREO_E_LAUNCH may have enqueued part of its
 * launches: zero-fill the workspace again before its next use (the Python binding does so for its own).
 */
size_t albireo_workspace_size(int64_t B, int64_t V, albireo_dtype_t dtype, int32_t n_top);

/*
 * Sample one token per row.
 *   logits       [B, ld] bf16 bit patterns or fp32 (dtype)
 *   params       [host] per-row metadata; NULL => every feature off (pure softmax sampling at T = 1)
 *   uniforms     [B] fp32 in [0, 1): the row's pre-generated random number.  Rank j of a
 *                sequence-parallel group passes uniforms + its row offset (sec. 6.2).
 *   out_ids      [B] int32 sampled token id (-1 for an EMPTY row)
 *   out_logprobs [B] fp32 log-softmax of the processed logits (after penalties and temperature) over
 *                the full vocabulary, at the sampled id
 *   n_top        0..ALBIREO_MAX_TOP_N; when > 0, out_top_ids / out_top_logprobs [B, n_top] get the n_top
 *                largest processed logits (ties -> lower id) with their logprobs; slots beyond the
 *                number of finite logits get id -1 and -inf
 *   out_flags    [B] ALBIREO_FLAG_* bits, or NULL
 * Returns ALBIREO_OK once the work is enqueued.
 */
albireo_status_t albireo_sample(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                                const albireo_params_t* params, const float* uniforms, int32_t* out_ids,
                                float* out_logprobs, int32_t n_top, int32_t* out_top_ids,
                                float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                                size_t workspace_bytes, hipStream_t stream);

/*
 * albireo_sample for callers that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  The same kernels and the same results as
 * albireo_sample; the workspace is a fixed array in the library's device memory instead of a caller
 * buffer, so the call allocates nothing (no hipMalloc, no allocating library routine).
 *   Arguments and outputs as albireo_sample, without workspace / workspace_bytes.
 *   Limit: a shape whose albireo_sample workspace exceeds ALBIREO_NOALLOC_SCRATCH_BYTES (96 MiB: about
 *   12.1 KB per row chunk, so B * P up to about 8100 row chunks, P = ceil(floor(V / 8) / 4864) for bf16
 *   and ceil(floor(V / 4) / 4864) for fp32) returns ALBIREO_E_SCRATCH before anything is enqueued.
 *   Every GPU the library runs on holds one such array until the process ends, shared by all calls on
 *   that GPU: two calls that overlap in time on one GPU (different streams, or threads) race on it and
 *   must be serialised by the caller.  Nothing in it needs to be zero between calls: every call leaves
 *   it zero-filled, and after a call that returns ALBIREO_E_LAUNCH (the runtime refused a launch
 *   part-way) the next call on that GPU first zero-fills the whole array with one more launch.
 */
#define ALBIREO_NOALLOC_SCRATCH_BYTES (96u << 20)
albireo_status_t albireo_sample_noalloc(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V,
                                        int64_t ld, const albireo_params_t* params, const float* uniforms,
                                        int32_t* out_ids, float* out_logprobs, int32_t n_top,
                                        int32_t* out_top_ids, float* out_top_logprobs, uint32_t* out_flags,
                                        hipStream_t stream);

/*
 * Apply steps 1-2 (penalties only) and write the penalised logits as fp32.
 *   params      [host] uses the repetition/frequency/presence penalties and the output history, the prompt
 *               history or the penalty state as albireo_sample does; other members ignored
 *   out_logits  [B, V] fp32, row stride V.  It may alias `logits` only when dtype is F32 and ld == V.
 */
albireo_status_t albireo_apply_penalties(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V,
                                         int64_t ld, const albireo_params_t* params, float* out_logits,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Apply steps 3-5 to already-penalised fp32 logits and report the filtered distribution.
 *   params         [host] uses temperature, top_k, top_p, min_p; penalty members are ignored
 *   out_probs      [B, V] fp32 (row stride V) renormalised probabilities over the kept set S, 0 outside
 *                  S, or NULL.  A greedy row keeps only its argmax (probability 1).
 *   out_threshold  [B] fp32 min z over S (-inf for an EMPTY row), or NULL
 *   out_kept       [B] int32 |S|, or NULL
 *   out_log_norm   [B] fp32 m + log sum_{v in S} exp(z_v - m), or NULL
 *   out_flags      [B] ALBIREO_FLAG_* bits, or NULL
 */
albireo_status_t albireo_topk_topp(const float* logits, int64_t B, int64_t V, int64_t ld,
                                   const albireo_params_t* params, float* out_probs, float* out_threshold,
                                   int32_t* out_kept, float* out_log_norm, uint32_t* out_flags,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * One decoding step's extras for albireo_sample_step (host struct, read during the call only).
 *
 * Device random numbers replace the caller's uniforms.  The paper pre-generates the random numbers of
 * a request on every GPU so that each worker's draws match a single worker's (sec. 6.2, "Deterministic
 * random number generation"); here they come from a counter-based generator instead, so any worker
 * produces the same number for the same row without storing or exchanging them.  The uniform of row
 * i is Philox-4x32 with 10 rounds (Salmon et al., SC 2011) of the counter (step, seq_ids[i]), four
 * 32-bit words low word first, under the key seed: the top 24 bits of the first output word times
 * 2^-24, in [0, 1).
 *
 * Early-feedback backfill (sec. 5, "Early-feedback backfill" and "Input processing"): the next
 * iteration's last-token tensor X_T is laid out by the scheduler before sampling ends, and each
 * scheduled sequence's new token is written into its slot by the sampler.  When next_tokens is not
 * NULL, the sampled id of row i is also written to next_tokens[backfill_dest[i]] whenever
 * 0 <= backfill_dest[i] < next_len (an EMPTY row writes -1); rows with any other value (padding rows,
 * sequences not scheduled next) write nothing, and slots no row names keep their contents.  Two rows
 * naming the same slot leave one of their ids there (which one is unspecified).
 */
typedef struct {
  uint64_t seed;                /* generator key                                                   */
  uint64_t step;                /* decoding step (counter words 0-1)                               */
  const int64_t* seq_ids;       /* [B] device sequence ids (counter words 2-3), or NULL: row index  */
  int32_t* next_tokens;         /* [next_len] device, or NULL: no backfill                         */
  const int32_t* backfill_dest; /* [B] device slot of each row in next_tokens (needed with it)      */
  int64_t next_len;             /* [host value] number of slots in next_tokens                     */
} albireo_step_t;

/*
 * albireo_sample with the uniforms generated on the device and the optional backfill, in the same
 * launch.  step [host] must not be NULL.  Every other argument is as for albireo_sample, and the
 * results equal albireo_sample's on the uniforms albireo_philox_uniforms returns for the same
 * (seed, step, seq_ids).
 */
albireo_status_t albireo_sample_step(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                                     const albireo_params_t* params, const albireo_step_t* step, int32_t* out_ids,
                                     float* out_logprobs, int32_t n_top, int32_t* out_top_ids,
                                     float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream);

/*
 * The all-to-all receive layout (host struct, read during the call only).  Before sampling, each of t
 * workers holds a vocabulary shard [s, V/t] of the whole batch; the all-to-all that replaces the gather
 * (sec. 6.1, Eq. opt_sample, the exchange written g-hat; sec. 6.2, "Efficient logit exchange") sends
 * every worker the shard columns of its own s/t rows, so worker j receives t blocks [s/t, V/t], one
 * from each worker, one after another.  This struct describes such a buffer so that it can be sampled
 * in place, with no repack:
 * element v of row i lies at
 *     logits + (v / shard_len) * shard_stride + i * ld + (v % shard_len)        (elements)
 * The packed receive buffer [t][B][shard_len] has shard_stride = B * shard_len and ld = shard_len.
 * The number of blocks is ceil(V / shard_len); the last block may be partly used (a worker's padded
 * vocabulary columns past V are never read).
 */
typedef struct {
  int64_t shard_len;    /* vocabulary columns per block (elements), > 0                       */
  int64_t shard_stride; /* elements from the start of one block to the next, >= shard_len     */
} albireo_shards_t;

/*
 * albireo_sample / albireo_sample_step on logits in the layout `shards` describes.  Exactly one of
 * `uniforms` (as albireo_sample) and `step` (as albireo_sample_step) is given.  The row's 16-byte
 * slots must each lie inside one block: logits 16-byte aligned, and shard_len, shard_stride and ld
 * times the element size multiples of 16 (else ALBIREO_E_UNSUPPORTED).  ld >= min(shard_len, V).
 * The results, including the reduction order, equal albireo_sample's on the same rows stored
 * row-major with 16-byte aligned rows.  Batch padding rows (sec. 6.2, "Batch padding": the batch is
 * padded to a multiple of t and the padded outputs are discarded before the backfill) are sampled
 * like any other row; a backfill slot of -1 keeps their ids out of the next iteration.
 */
albireo_status_t albireo_sample_sharded(const void* logits, albireo_dtype_t dtype, int64_t B, int64_t V, int64_t ld,
                                        const albireo_shards_t* shards, const albireo_params_t* params,
                                        const float* uniforms, const albireo_step_t* step, int32_t* out_ids,
                                        float* out_logprobs, int32_t n_top, int32_t* out_top_ids,
                                        float* out_top_logprobs, uint32_t* out_flags, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/*
 * The device uniforms alone: out_uniforms[i] (device, [B] fp32) = the uniform described above for
 * (seed, step, seq_ids[i]) (seq_ids NULL: i).  No workspace.
 */
albireo_status_t albireo_philox_uniforms(uint64_t seed, uint64_t step, const int64_t* seq_ids, int64_t B,
                                         float* out_uniforms, hipStream_t stream);

/*
 * The backfill alone: next_tokens[dest[i]] = ids[i] for every row i with 0 <= dest[i] < next_len
 * (ids, dest: [B] device; next_tokens: [next_len] device).  No workspace.
 */
albireo_status_t albireo_backfill(const int32_t* ids, const int32_t* dest, int64_t B, int32_t* next_tokens,
                                  int64_t next_len, hipStream_t stream);

/* Static description of a status code. */
const char* albireo_status_string(albireo_status_t status);

#ifdef __cplusplus
}
#endif
#endif /* ALBIREO_H */
