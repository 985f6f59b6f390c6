/*
 * sage.h - C ABI of the SageSched scheduling-decision path on MI355X (gfx950).
 *
 * For a batch of pending LLM requests the path predicts an output-length
 * distribution from the most similar past prompts (paper Sec. 3.1), turns it
 * into a service-cost distribution with C = O^2/2 + I*O (Sec. 3.2), computes
 * the Gittins index of that distribution and orders the queue by it, smaller
 * index first (Sec. 3.3).
 *
 * Conventions shared by every entry point:
 *  - Every pointer is a DEVICE pointer (HBM of the current HIP device) unless
 *    stated otherwise; all arrays are dense, row-major, and at least 16-byte
 *    aligned. bf16 values travel as their raw 16-bit patterns (uint16_t).
 *  - The caller owns every buffer, including the workspace. The library
 *    allocates nothing on these paths and keeps no pointer after returning.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *    the call returns without synchronising. Arguments are validated before
 *    anything is enqueued: a call that returns an error has enqueued nothing.
 *    Faults while kernels run surface at the caller's synchronisation.
 *  - Q = 0 is a valid no-op. Entry points are re-entrant on distinct streams
 *    and distinct buffers.
 *  - Return value: SAGE_OK or a negative sage_status; sage_last_error() gives
 *    a human-readable detail for the calling thread.
 */
#ifndef SAGE_H
#define SAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* sage_stream_t; /* == hipStream_t */

enum sage_status {
  SAGE_OK = 0,
  SAGE_EINVAL = -1,      /* bad argument: null pointer, size or range */
  SAGE_EWORKSPACE = -2,  /* workspace smaller than the *_workspace_bytes query */
  SAGE_EUNSUPPORTED = -3,/* device is not gfx950 */
  SAGE_EHIP = -4         /* a HIP runtime call failed (see sage_last_error) */
};

/* Limits checked by validation. */
#define SAGE_MAX_K 256
#define SAGE_MAX_BINS 4096

/*
 * sage_ingest_bf16 - store fp32 embeddings as bf16 (round to nearest, ties
 * to even): the resident history store and the query batch are kept in bf16
 * (the paper fixes no precision; Sec. 3.1 only needs cosine similarity).
 *   src [n] fp32 finite values; dst [n] bf16 bit patterns. src and dst must
 *   not overlap. n = 0 is a no-op.
 */
int sage_ingest_bf16(const float* src, size_t n, uint16_t* dst, sage_stream_t stream);

/*
 * Layouts of an embedding matrix of `rows` x d bf16 values (d % 32 == 0).
 *   SAGE_LAYOUT_ROWS    row-major [rows, d]
 *   SAGE_LAYOUT_PANELS  panel-major [d / 32][rows][32]: the d axis is cut into
 *                       32-column panels, each holding its columns of every
 *                       row contiguously; element (r, c) is at
 *                       (c / 32) * rows * 32 + r * 32 + c % 32
 * The similarity kernels walk d in 32-column slices of consecutive rows;
 * panel-major makes each slice of 16 rows one contiguous kilobyte (whole
 * 128-byte lines), which halves the L2 requests of the search. Results do not
 * depend on the layout (bit-identical outputs).
 */
enum { SAGE_LAYOUT_ROWS = 0, SAGE_LAYOUT_PANELS = 1 };

/*
 * sage_ingest_bf16_panels - sage_ingest_bf16 into the panel-major layout.
 *   src [rows, d] fp32 row-major finite values; dst [d / 32][rows][32] bf16
 *   bits (round to nearest, ties to even). src and dst must not overlap.
 * SAGE_EINVAL: rows < 0 or above 2^29, d not a positive multiple of 32, NULL
 * or misaligned pointer. rows = 0 is a no-op.
 */
int sage_ingest_bf16_panels(const float* src, int rows, int d, uint16_t* dst, sage_stream_t stream);

/*
 * sage_panels_from_rows - rearrange bf16 embeddings [rows, d] (row-major)
 * into the panel-major layout (bits copied unchanged). Errors as for
 * sage_ingest_bf16_panels.
 */
int sage_panels_from_rows(const uint16_t* src, int rows, int d, uint16_t* dst, sage_stream_t stream);

/*
 * sage_store_insert - FIFO maintenance of the history store (Sec. 3.1: the
 * records of recently served requests, prompt embedding and output length,
 * kept in a window updated first-in first-out). The store is a ring of
 * `capacity` rows: record t (counting every record ever inserted from 0)
 * lives in row t mod capacity, so the newest record overwrites the oldest,
 * and the rows in use are [0, min(total, capacity)), contiguous: pass that
 * many rows to sage_predict.
 *   emb [n, d] f32 (rounded to bf16, RNE), out_len [n] int32: the batch
 *   total: records inserted before this batch (kept by the caller; it becomes
 *          total + n); of a batch larger than the ring, only its last
 *          `capacity` records are written
 *   ring_emb [capacity, d] bf16 bits, ring_len [capacity] int32: updated
 * SAGE_EINVAL: n < 0, d not a positive multiple of 32, capacity < 1,
 * total < 0, NULL or misaligned pointer.
 */
int sage_store_insert(const float* emb, const int32_t* out_len, int n, int d, long long total,
                      int capacity, uint16_t* ring_emb, int32_t* ring_len, sage_stream_t stream);

/*
 * sage_queue_admit / sage_queue_dispatch - per-decision bookkeeping of a
 * standing queue of `slots` pending requests (Sec. 3.3: the queue is
 * re-ranked at every scheduling decision; each decision admits `batch` new
 * arrivals into the slots the previous one freed and dispatches `batch`).
 *   admit: new request i takes slot free_slots[i]: mass[s, :] = new_mass[i, :],
 *          plen[s] = new_plen[i], request[s] = next_request + i. Slots
 *          outside [0, slots) are skipped (device data, not checked on the
 *          host).
 *          free_slots [batch] int64, new_mass [batch, B] f32, new_plen [batch]
 *          int32 in; mass [slots, B] f32, plen [slots] int32, request [slots]
 *          int64 updated.
 *   dispatch: the first `batch` entries of order (a sage_rank result over
 *          the slots) leave: free_slots[i] = order[i], dispatched[i] =
 *          request[order[i]] (-1 for an entry outside [0, slots)).
 *          order [slots] int32, request [slots] int64 in; free_slots [batch],
 *          dispatched [batch] int64 out.
 * SAGE_EINVAL: batch < 0, slots < batch, B outside [1, SAGE_MAX_BINS],
 * next_request < 0, NULL or misaligned pointer (when batch > 0).
 */
int sage_queue_admit(const int64_t* free_slots, int batch, const float* new_mass, const int32_t* new_plen,
                     int B, long long next_request, int slots, float* mass, int32_t* plen, int64_t* request,
                     sage_stream_t stream);
int sage_queue_dispatch(const int32_t* order, int batch, const int64_t* request, int slots,
                        int64_t* free_slots, int64_t* dispatched, sage_stream_t stream);

/*
 * sage_predict_workspace_bytes - bytes of device workspace sage_predict needs
 * for these sizes (holds the per-stream partial neighbour lists). Returns 0
 * for invalid sizes.
 */
size_t sage_predict_workspace_bytes(int Q, int N, int d, int k, int B);

/*
 * sage_predict - semantic-aware history-based predictor (Sec. 3.1).
 *   queries  [Q, d] bf16  prompt embeddings of the pending requests (unit norm
 *                         expected; no renormalisation is applied)
 *   hist_emb [N, d] bf16  history store: embeddings of past prompts
 *   hist_len [N]   int32  their recorded output lengths (>= 1)
 *   k                     neighbours per request, 1..SAGE_MAX_K
 *   tau                   similarity threshold in [2^-20, 1]; neighbours
 *                         below it get zero weight (paper default 0.8)
 *   bin_edges [B+1] f64   strictly increasing length-bin edges; a length L
 *                         falls in the largest b in [0, B-1] with
 *                         edges[b] <= L (lengths below edges[0] go to bin 0).
 *                         The order is a precondition that is not checked
 *                         before enqueue (device array): see
 *                         sage_check_inputs
 *   B                     1..SAGE_MAX_BINS
 * Outputs (row q = request q):
 *   nbr_ids  [Q, k] int32 the k history indices with the largest similarity
 *                         s = <query, hist_emb[n]> (fp32 accumulation of bf16
 *                         products), ordered by (s desc, index asc); if
 *                         N < k the tail is padded with -1
 *   nbr_sims [Q, k] f32   their similarities (padding: -inf)
 *   counts   [Q, B] int32 neighbours (valid ids) per length bin
 *   mass     [Q, B] f32   similarity-weighted share per bin: sum of s_i over
 *                         the bin's neighbours with s_i >= tau, divided by the
 *                         same sum over all neighbours; if no neighbour reaches
 *                         tau, counts / (number of valid neighbours)
 *   workspace             >= sage_predict_workspace_bytes(Q, N, d, k, B) bytes
 * Constraints: Q >= 0, N >= 1, d >= 32 and d % 32 == 0.
 */
int sage_predict(const uint16_t* queries, int Q,
                 const uint16_t* hist_emb, const int32_t* hist_len, int N, int d,
                 int k, float tau, const double* bin_edges, int B,
                 int32_t* nbr_ids, float* nbr_sims, int32_t* counts, float* mass,
                 void* workspace, size_t workspace_bytes, sage_stream_t stream);

/*
 * sage_predict_layout - sage_predict with the layout of each embedding
 * matrix given: queries [Q, d] and hist_emb [N, d] are each SAGE_LAYOUT_ROWS
 * or SAGE_LAYOUT_PANELS (the panel-major store is the fast one; outputs are
 * identical). sage_predict is this call with both SAGE_LAYOUT_ROWS.
 * SAGE_EINVAL also for a layout that is not a SAGE_LAYOUT_* value.
 */
int sage_predict_layout(const uint16_t* queries, int query_layout, int Q,
                        const uint16_t* hist_emb, int hist_layout, const int32_t* hist_len, int N, int d,
                        int k, float tau, const double* bin_edges, int B,
                        int32_t* nbr_ids, float* nbr_sims, int32_t* counts, float* mass,
                        void* workspace, size_t workspace_bytes, sage_stream_t stream);

/*
 * sage_length_index - the store's records ordered by input length, for the
 * semantic-unaware predictor below (Sec. 4.3's predictor ablation). Build it
 * once per store (and again after records change).
 *   hist_prompt_len [N] int32  input lengths of the stored records, clamped
 *                              to [1, max_len]
 *   max_len                    1..2^20
 *   by_len [N] int32 out       record indices sorted by clamped length, equal
 *                              lengths by ascending index
 *   sorted_len [N] int32 out   their clamped lengths
 *   len_off [max_len + 2] int32 out  len_off[L] = first position in by_len
 *                              whose length is >= L (N if none)
 *   workspace                  >= sage_length_index_workspace_bytes(N) bytes
 * SAGE_EINVAL: N < 1, max_len outside [1, 2^20], NULL or misaligned pointers;
 * SAGE_EWORKSPACE: workspace too small.
 */
size_t sage_length_index_workspace_bytes(int N);
int sage_length_index(const int32_t* hist_prompt_len, int N, int max_len, int32_t* by_len, int32_t* sorted_len,
                      int32_t* len_off, void* workspace, size_t workspace_bytes, sage_stream_t stream);

/*
 * sage_predict_by_length - the semantic-unaware history-based predictor
 * (Sec. 4.3): neighbours are the stored records with the most similar INPUT
 * LENGTH rather than the most similar prompt. The similarity of input
 * lengths I and L is s = min(I, L) / max(I, L) (fp32, correctly rounded;
 * I below 1 counts as 1), so the threshold tau keeps its meaning for the
 * predictor ("the same filtering method"). The k records with the largest s
 * (ties to the lower index; padding -1 / -inf when N < k) then go through
 * the histogram of sage_predict: counts and s-weighted masses with tau.
 *   prompt_len [Q] int32       input lengths of the pending requests
 *   by_len, sorted_len, len_off, max_len   the index from sage_length_index
 *   hist_len [N] int32         recorded output lengths of the stored records
 *   other arguments and outputs as in sage_predict (nbr_sims holds s).
 * Q = 0 is a no-op. SAGE_EINVAL for sizes as in sage_predict, max_len outside
 * [1, 2^20], NULL or misaligned pointers.
 */
int sage_predict_by_length(const int32_t* prompt_len, int Q, const int32_t* by_len, const int32_t* sorted_len,
                           const int32_t* len_off, int max_len, const int32_t* hist_len, int N, int k, float tau,
                           const double* bin_edges, int B, int32_t* nbr_ids, float* nbr_sims, int32_t* counts,
                           float* mass, sage_stream_t stream);

/*
 * sage_predict_stats - what the last sage_predict / sage_predict_layout call
 * with this workspace and these sizes did in its neighbour search, for
 * measurement (the candidate keys are the select stage's input; their count
 * depends on the data). Copies a few counters from the workspace to the host
 * and SYNCHRONISES `stream`: not for the decision path itself.
 *   stats [5] host, out:
 *     [0] search path: 0 exact per-chunk lists, 1 filtered (k <= 64),
 *         2 few-query stream search
 *     [1] candidate keys written for the select stage (list path: every
 *         list entry, Q * [3] * [4])
 *     [2] queries sent to the exact fallback
 *     [3] candidate segments (lists) per query
 *     [4] capacity of a segment (list length)
 * SAGE_EINVAL for sizes as in sage_predict or stats NULL; SAGE_EWORKSPACE
 * when the workspace is smaller than that call needs.
 */
int sage_predict_stats(const void* workspace, size_t workspace_bytes, int Q, int N, int d, int k, int B,
                       long long* stats, sage_stream_t stream);

/*
 * sage_predict_noalloc - sage_predict_layout for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same search with no workspace
 * argument. Its scratch memory is a static device array of
 * SAGE_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held until the
 * process ends; the call allocates and frees nothing. Inputs and outputs are
 * the caller's, as in sage_predict_layout, and the outputs are identical to
 * that call's.
 *   SAGE_EWORKSPACE (nothing enqueued) when the search needs more scratch
 *   than the array holds: sage_predict_workspace_bytes(Q, N, d, k, B) must
 *   not exceed SAGE_NOALLOC_SCRATCH_BYTES (few-query decisions against a
 *   store of millions of rows fit; so do batches of a few hundred queries).
 * Every call on one GPU shares that GPU's array: calls that overlap in time
 * on one GPU (other streams, other host threads) race and must be ordered by
 * the caller. Nothing in the array needs to start cleared: each call writes
 * every scratch value before reading it.
 */
#define SAGE_NOALLOC_SCRATCH_BYTES (64u << 20)
int sage_predict_noalloc(const uint16_t* queries, int query_layout, int Q,
                         const uint16_t* hist_emb, int hist_layout, const int32_t* hist_len, int N, int d,
                         int k, float tau, const double* bin_edges, int B,
                         int32_t* nbr_ids, float* nbr_sims, int32_t* counts, float* mass,
                         sage_stream_t stream);

/*
 * sage_histogram - the predicted output-length distribution alone (the last
 * stage of sage_predict, Sec. 3.1), for neighbour lists obtained elsewhere.
 *   nbr_ids [Q, k] int32 history indices; entries outside [0, N) mean "no
 *                 neighbour" and are skipped
 *   nbr_sims [Q, k] f32 their similarities, each below 2048 in magnitude
 *   hist_len [N] int32 recorded output lengths of the history store
 *   other arguments and outputs as in sage_predict.
 * Weights are summed exactly (fixed point, 2^-43 resolution, which is exact
 * for every fp32 weight >= tau >= 2^-20), so results do not depend on the
 * order of the neighbours.
 */
int sage_histogram(const int32_t* nbr_ids, const float* nbr_sims, int Q, int k,
                   const int32_t* hist_len, int N, float tau, const double* bin_edges, int B,
                   int32_t* counts, float* mass, sage_stream_t stream);

/*
 * sage_cost - unified compute/memory cost model (Sec. 3.2): the cost of
 * serving request q with output length r_b is x[q, b] = r_b^2/2 + I_q * r_b,
 * evaluated in fp64 and rounded to fp32.
 *   prompt_len [Q] int32 (>= 0), bin_repr [B] f64 representative output
 *   length of each bin (positive, increasing), cost [Q, B] f32 out.
 *   Both orders are preconditions checked on the device by
 *   sage_check_inputs, not before enqueue.
 */
int sage_cost(const int32_t* prompt_len, int Q, const double* bin_repr, int B,
              float* cost, sage_stream_t stream);

/*
 * sage_index - Gittins index of each request's cost distribution (Sec. 3.3):
 *   G = inf over Delta > 0 of E[min(X, Delta)] / P(X <= Delta), X ~ D,
 * where D puts mass[q, b] on cost x[q, b]. The masses need not sum to one
 * (the index does not depend on their scale). The cost support must be
 * non-decreasing along each row (true for sage_cost on increasing bin_repr);
 * the index is then the minimum over the support points b with F_b > 0 of
 * (S_b + T_b x_b) / F_b (F, S: prefix sums of p and p*x; T: mass above b).
 *   mass [Q, B] f32, non-negative
 *   cost [Q, B] f32, or NULL: then x is computed in fp64 from prompt_len [Q]
 *        and bin_repr [B] as in sage_cost (fused, nothing materialised)
 *   index [Q] f32 out: the Gittins index (+inf for a row with no mass)
 *   argmin_bin [Q] int32 out or NULL: smallest b attaining the minimum
 *        (-1 for a row with no mass)
 * Accumulation is in fp64; one division per request.
 */
int sage_index(const float* mass, const float* cost, const int32_t* prompt_len,
               const double* bin_repr, int Q, int B,
               float* index, int32_t* argmin_bin, sage_stream_t stream);

/*
 * sage_index_attained - the index of running requests, refreshed with the
 * service they have already received (Sec. 3.3: the index of each active
 * request is updated with its remaining cost distribution, only at bucket
 * boundaries; bucket size 200 by default, Sec. 4). For request q with
 * generated[q] output tokens so far, o = bucket * floor(generated[q] / bucket)
 * and the service received is a = o^2 / 2 + I_q o (the cost model of
 * sage_cost). Support points x <= a are ruled out and the remaining cost is
 * X - a, so
 *   G = inf over Delta > 0 of E[min(X - a, Delta); X > a] / P(a < X <= a + Delta),
 * the minimum over the support points above a. generated[q] = 0 gives
 * sage_index's result; a row with no mass above a gets +inf (argmin -1).
 *   mass [Q, B] f32, prompt_len [Q] int32, bin_repr [B] f64 (as sage_index
 *        with the fused cost), generated [Q] int32 >= 0, bucket >= 1
 *   index [Q] f32 out, argmin_bin [Q] int32 out or NULL
 * Errors as sage_index; SAGE_EINVAL also for bucket < 1.
 */
int sage_index_attained(const float* mass, const int32_t* prompt_len, const double* bin_repr,
                        const int32_t* generated, int bucket, int Q, int B,
                        float* index, int32_t* argmin_bin, sage_stream_t stream);

/*
 * sage_index_attained_table - sage_index_attained for every request at each
 * refresh level at once: index[lv * Q + q] is request q's index after
 * o = lv * bucket generated tokens (a = o^2 / 2 + I_q o), lv = 0 .. levels-1,
 * the values sage_index_attained gives with generated[q] = lv * bucket. One
 * read of each row serves all its levels (the table a trace replay orders
 * by, Sec. 3.3: indices change only at bucket boundaries).
 *   mass [Q, B] f32, prompt_len [Q] int32, bin_repr [B] f64, bucket >= 1,
 *   levels >= 1 (levels * bucket within int32); index [levels, Q] f32 out.
 * Errors as sage_index_attained; SAGE_EINVAL also for levels < 1.
 */
int sage_index_attained_table(const float* mass, const int32_t* prompt_len, const double* bin_repr,
                              int bucket, int levels, int Q, int B, float* index, sage_stream_t stream);

/*
 * Variants of the method that the paper compares against (Sec. 4 ablation).
 *
 * sage_histogram_variant - sage_histogram with a choice of neighbour weight:
 *   SAGE_WEIGHT_SIMILARITY: w = s if s >= tau (sage_histogram's form);
 *   SAGE_WEIGHT_UNIFORM:    w = 1 if s >= tau, the paper's own form (Sec. 3.1:
 *                           the outputs of the similar requests form the
 *                           distribution, each counting once).
 * Same arguments, fallback and errors as sage_histogram; SAGE_EINVAL for an
 * unknown weighting.
 */
enum { SAGE_WEIGHT_SIMILARITY = 0, SAGE_WEIGHT_UNIFORM = 1 };
int sage_histogram_variant(const int32_t* nbr_ids, const float* nbr_sims, int Q, int k,
                           const int32_t* hist_len, int N, float tau, const double* bin_edges, int B,
                           int weighting, int32_t* counts, float* mass, sage_stream_t stream);

/*
 * sage_index_variant - a priority index under the paper's alternative
 * choices, on the fused cost (support at O = bin_repr[b]):
 *   cost_model SAGE_COST_RESOURCE: O^2/2 + I O (the adopted model, sage_cost)
 *              SAGE_COST_OUTPUT:   O (output length alone)
 *              SAGE_COST_OVERALL:  I + 2 O (input plus doubled output length)
 *   index_kind SAGE_INDEX_GITTINS: as sage_index
 *              SAGE_INDEX_MEAN:    E[X] = sum p x / sum p (the Mean baseline;
 *                                  argmin_bin is -1)
 *   noise_weight in [0, 1): the distribution is first mixed with the uniform
 *              one, p' = (1 - w) p / sum(p) + w / B (w = 0.2 is the paper's
 *              1:4 inaccurate prediction); rows with no mass stay empty.
 * mass [Q, B] f32, prompt_len [Q] int32, bin_repr [B] f64; index [Q] f32 out
 * (+inf for a row with no mass), argmin_bin [Q] int32 out or NULL.
 * SAGE_EINVAL for unknown enums or noise_weight outside [0, 1).
 */
/*
 * sage_mix_uniform - a deliberately inaccurate prediction (Sec. 4.3 merges a
 * uniform distribution into the predicted one at 1:4): each row becomes
 *   out[q, b] = (1 - weight) * mass[q, b] / sum_b mass[q, b] + weight / B
 * (fp64, rounded to fp32); weight = 0.2 is the paper's 1:4. A row with no
 * mass stays zero. Any index entry point can then take `out`.
 *   mass [Q, B] f32 (non-negative), out [Q, B] f32: the same buffer (in
 *   place) or one that does not overlap it; weight in [0, 1].
 * SAGE_EINVAL for a weight outside [0, 1], partial overlap, B outside
 * [1, SAGE_MAX_BINS], NULL or misaligned pointers.
 */
int sage_mix_uniform(const float* mass, int Q, int B, float weight, float* out, sage_stream_t stream);

enum { SAGE_COST_RESOURCE = 0, SAGE_COST_OUTPUT = 1, SAGE_COST_OVERALL = 2 };
enum { SAGE_INDEX_GITTINS = 0, SAGE_INDEX_MEAN = 1 };
int sage_index_variant(const float* mass, const int32_t* prompt_len, const double* bin_repr, int Q, int B,
                       int cost_model, int index_kind, float noise_weight,
                       float* index, int32_t* argmin_bin, sage_stream_t stream);

/*
 * sage_check_inputs - device check of the preconditions that the binning and
 * the index scan rely on but that validation before enqueue cannot see (the
 * arrays are device-resident, and reading them on the host would synchronise
 * the stream):
 *   SAGE_CHECK_EDGES       bin_edges [B+1] finite and strictly increasing
 *                          (the bins of Sec. 3.1's length histogram)
 *   SAGE_CHECK_REPR        bin_repr [B] finite, bin_repr[0] >= 0, and
 *                          non-decreasing
 *   SAGE_CHECK_PROMPT_LEN  prompt_len [Q] >= 0
 * With the last two the cost support r (I + r/2) of Sec. 3.2 is
 * non-decreasing along every row, which the Gittins scan of Sec. 3.3 needs:
 * on unsorted support sage_index returns a value that is not the index, and
 * on unsorted edges the histogram bins by a search over an unsorted array.
 * Any of the three arrays may be NULL (not checked). One small kernel writes
 * the OR of the failed conditions' bits to *status (int32, device), 0 when
 * all hold; the caller reads it at its next synchronisation and treats a
 * non-zero value as SAGE_EINVAL. The Python layer's Store runs it on its
 * bins once, at construction.
 * SAGE_EINVAL (nothing enqueued): B outside [1, SAGE_MAX_BINS], Q < 0,
 * status NULL, misaligned pointers.
 */
enum { SAGE_CHECK_EDGES = 1, SAGE_CHECK_REPR = 2, SAGE_CHECK_PROMPT_LEN = 4 };
int sage_check_inputs(const double* bin_edges, const double* bin_repr, int B, const int32_t* prompt_len, int Q,
                      int32_t* status, sage_stream_t stream);

/*
 * sage_debug_theta_floor - test hook, not for production use. Later
 * sage_predict calls (any thread) raise each query's pre-pass threshold
 * theta0 to at least `floor` on the filtered (k <= 64) and few-query paths,
 * which forces queries onto their exact fallback (a query left with fewer
 * than min(k, N) candidates is answered there); results must not change.
 * -inf turns it off (the default). SAGE_EINVAL for NaN. Host-only state.
 */
int sage_debug_theta_floor(float floor);

/* sage_rank_workspace_bytes - device workspace bytes for sage_rank(Q). */
size_t sage_rank_workspace_bytes(int Q);

/*
 * sage_rank - queue order (Sec. 3.3: the smaller Gittins index is served
 * first): order[0..Q) is the stable ascending argsort of index (ties keep
 * the lower request id first; +inf sorts last). NaN is not allowed.
 *   index [Q] f32, order [Q] int32 out (a permutation of 0..Q-1).
 */
int sage_rank(const float* index, int Q, int32_t* order,
              void* workspace, size_t workspace_bytes, sage_stream_t stream);

/*
 * sage_simulate - replay of a request trace against a queue served in a
 * given priority order: a discrete-event simulation run on the HOST (all
 * pointers are host pointers, nothing is enqueued on a stream). It measures
 * the paper's metric, the time-to-last-token (TTLT = finish - arrival,
 * Sec. 2), of an ordering.
 *
 * Model. Requests arrive at arrival[r] (Sec. 4.1 uses Poisson arrivals).
 * Request r needs C = O^2/2 + I*O cost units (the unified cost of Sec. 3.2
 * at its true lengths I = prompt_len[r], O = output_len[r]); after g
 * generated tokens it has received a(g) = g^2/2 + I*g. `servers` identical
 * servers each run one request at a time at `rate` cost units per second.
 * After every event instant (completions, then bucket boundaries, then
 * arrivals at that instant) the `servers` admitted requests with the
 * smallest keys run; a running request that drops out is preempted and keeps
 * its service (preemption is enabled at negligible cost, Sec. 3.3). At most
 * queue_cap requests wait besides those running (Sec. 4.4 buffers up to
 * 1,000); later arrivals wait outside in arrival order and are admitted as
 * requests finish.
 *
 * Keys. order[0 .. levels*R) is a permutation of the entries e = k*R + r,
 * best first (sage_rank's output over an index table with one row per
 * level); request r's key is the position of entry (k, r), k being the
 * number of bucket boundaries it has crossed (one every `bucket` generated
 * tokens, Sec. 3.3 refreshes the index only there). bucket = 0: keys are
 * never refreshed and levels must be 1 (FCFS, Mean, Gittins at arrival);
 * bucket > 0: levels >= ceil(max O / bucket). Positions informed .. levels*R
 * of the order hold entries without information: a refreshed index of +inf
 * (sage_index_attained's value when no predicted mass lies above the service
 * received) ranks last; a request reaching such a level keeps its key.
 * Pass informed = levels * R when every entry is meaningful.
 *
 *   arrival [R] f64 seconds, finite and non-decreasing
 *   prompt_len [R] int32 >= 0, output_len [R] int32 >= 1
 *   order [levels * R] int32, 0 <= informed <= levels * R
 *   servers >= 1, rate > 0 finite, queue_cap >= 0
 *   finish [R] f64 out (completion time), preemptions [R] int32 out or NULL
 * SAGE_EINVAL for a NULL required pointer, R < 0, levels * R >= 2^31, a
 * decreasing or non-finite arrival, out-of-range lengths, too few levels, an
 * order that is not a permutation, or bad servers / rate / queue_cap. R = 0
 * is a no-op. The caller owns every buffer; nothing is retained.
 */
int sage_simulate(const double* arrival, const int32_t* prompt_len, const int32_t* output_len, int R,
                  const int32_t* order, int levels, int informed, int bucket, int servers, double rate,
                  int queue_cap, double* finish, int32_t* preemptions);

/* Static, thread-safe name of a status code. Host pointer. */
const char* sage_status_string(int status);

/* Detail of the calling thread's last failed call ("" if none). Host pointer. */
const char* sage_last_error(void);

/*
 * Stage timer (measurement only). While a timer is attached to the calling
 * thread, every kernel the library enqueues from that thread is bracketed by
 * two HIP events recorded on the same stream. After synchronising, read the
 * per-kernel totals. The timer owns its events (created once, up to
 * `capacity` launches between resets).
 */
typedef struct sage_timer sage_timer;
int sage_timer_create(int capacity, sage_timer** out);
int sage_timer_destroy(sage_timer* t);
int sage_timer_attach(sage_timer* t);   /* NULL detaches */
/* Time only the launches named `label` (a kernel name as sage_timer_get
 * reports it); NULL or "" times every launch again. Fewer events keep the
 * timed work closer to the untimed one. Host string, copied. */
int sage_timer_only(sage_timer* t, const char* label);
int sage_timer_reset(sage_timer* t);
/* Number of distinct kernel names seen since the last reset. */
int sage_timer_count(sage_timer* t);
/* i-th kernel: its name (host string owned by the library), launches and
 * total elapsed milliseconds. The caller must have synchronised the streams. */
int sage_timer_get(sage_timer* t, int i, const char** name, int* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* SAGE_H */
