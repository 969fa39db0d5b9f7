/*
 * luffy.h - C ABI of the token-condensation MoE layer on one MI355X (gfx950).
 *
 * The layer is the single-GPU data-parallel path of the token condensation of
 * Luffy (arXiv 2411.15419): route tokens to experts (Sec. 2.1), inside every
 * expert's bucket find tokens whose cosine similarity clears a threshold and
 * keep one representative per group (Sec. 5.1 steps 1 and 3, Sec. 5.2), run
 * the expert FFN on the representatives only (Sec. 3), and give every
 * condensed token its representative's expert output when combining
 * (Sec. 6, the token_to_token table; Sec. 2.1 combine).
 *
 * Conventions for every call
 *  - Pointers named as device pointers point to device memory owned by the
 *    caller; the library allocates nothing.  Scratch memory is passed in
 *    through a workspace pointer whose minimum size the matching
 *    *_workspace_size function returns (256-byte alignment required).
 *  - Matrices are row-major.  Weights use the [out, in] layout, so the
 *    contraction index is contiguous in every operand.
 *  - dtype (luffy_dtype) selects the element type of activations and
 *    weights: LUFFY_F32 (float) or LUFFY_BF16 (bfloat16 bit patterns,
 *    uint16).  Gates, norms and accumulations are float32.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream) and never synchronises the device.  Counts that depend on the
 *    data (bucket sizes, representative counts) stay on the device; grids are
 *    sized from upper bounds and kernels read the counts they need.
 *  - Arguments are checked on the host before anything is enqueued; a
 *    rejected call enqueues nothing and returns a negative status.  Launch
 *    failures return LUFFY_E_HIP.  luffy_last_error() gives a message for the
 *    most recent failure on the calling thread.  No C++ exception crosses the
 *    ABI.
 *  - Outputs must not alias inputs.  Integer outputs are deterministic: the
 *    same inputs give bit-identical indices on every run.
 *  - Supported sizes: d and d_ff multiples of 64 and at most 32768,
 *    1 <= E <= 64, k in {1, 2}, T*k < 2^31 (luffy_condense: T*k <= 2^24),
 *    every activation matrix and every expert's weight matrix smaller than
 *    4 GiB - 64 KiB.  Other sizes return LUFFY_E_UNSUPPORTED where the call
 *    can see them (x of luffy_expert_ffn, read through row_index, is the
 *    caller's to keep within the limit).
 */
#ifndef LUFFY_H
#define LUFFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LUFFY_ABI_VERSION 6

typedef enum {
  LUFFY_OK = 0,
  LUFFY_E_INVALID = -1,     /* null pointer, bad size, k > E, k not 1 or 2 */
  LUFFY_E_UNSUPPORTED = -2, /* a size the library does not handle         */
  LUFFY_E_WORKSPACE = -3,   /* workspace missing, too small or misaligned  */
  LUFFY_E_HIP = -4          /* a HIP runtime call or launch failed         */
} luffy_status;

typedef enum { LUFFY_F32 = 0, LUFFY_BF16 = 1 } luffy_dtype;

/* Expert activation (Sec. 2.1: an expert is an FFN).
 * GELU is the exact form 0.5 z (1 + erf(z / sqrt 2)); SiLU is z / (1 + e^-z). */
typedef enum { LUFFY_ACT_GELU = 0, LUFFY_ACT_SILU = 1 } luffy_act;

int luffy_abi_version(void);
const char* luffy_status_string(int status);
const char* luffy_last_error(void);

/* ------------------------------------------------------------------------
 * luffy_route - gate, top-k and the stable dispatch order (Sec. 2.1: the gate
 * network selects experts for every token and tokens are grouped by expert).
 *
 *   x          [T, d] dtype, device          token embeddings
 *   w_gate     [E, d] dtype, device          gate weights
 *   b_gate     [E] float, device, or NULL    gate bias
 *   capacity_factor  > 0: each expert keeps at most C slots, C =
 *                    luffy_capacity(T, k, E, capacity_factor); <= 0: no limit
 * Outputs (device):
 *   topk_idx   [T, k] int32   experts by descending logit, ties to the lower
 *                             id; logits are float32 sums, and a choice
 *                             whose float32 margin is small is re-decided on
 *                             float64 logits
 *   topk_gate  [T, k] float   softmax probability of the expert (k = 1), or
 *                             the two probabilities renormalised to sum to 1
 *                             (k = 2)
 *   slot_pos   [T, k] int32   bucket position of slot (t, j), -1 if dropped
 *   perm_token [T*k]  int32   token of every bucket position; only the first
 *                             offsets[E] entries are written
 *   offsets    [E+1]  int32   bucket e holds positions offsets[e] ..
 *                             offsets[e+1]-1
 *   inv_norm   [T] float or NULL   1/|x_t| (0 for a zero row), for
 *                             luffy_condense: the gate pass reads every
 *                             row anyway, so the similarity pass need not
 * A slot is (token t, choice j) with id s = j*T + t.  Buckets are stable in
 * s (all first choices in token order, then all second choices); with a
 * capacity the first C slots of a bucket stay and later ones are dropped.
 * ---------------------------------------------------------------------- */
size_t luffy_route_workspace_size(int T, int E, int k);
int luffy_route(const void* x, int T, int d, int dtype,
                const void* w_gate, const float* b_gate, int E, int k,
                double capacity_factor,
                int32_t* topk_idx, float* topk_gate, int32_t* slot_pos,
                int32_t* perm_token, int32_t* offsets, float* inv_norm,
                void* workspace, size_t workspace_bytes, void* stream);

/* luffy_route_noalloc - luffy_route for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments and results without the workspace, whose
 * role is taken by a scratch array the library holds in device memory, one
 * per GPU, for the life of the process (luffy_route_noalloc_max_bytes()
 * bytes, 4 MiB).  Calls whose luffy_route_workspace_size(T, E, k) exceeds it
 * return LUFFY_E_UNSUPPORTED and enqueue nothing (at E = 64, k = 2 that is
 * T above 131056).  It allocates nothing on any call.  Every call on a GPU
 * uses that GPU's one array, so calls that can overlap on one GPU (several
 * streams, several host threads) race and must be ordered by the caller.  On
 * its first call on a device (the current device) it looks up the array's
 * address there, which can fail with LUFFY_E_HIP. */
size_t luffy_route_noalloc_max_bytes(void);
int luffy_route_noalloc(const void* x, int T, int d, int dtype,
                        const void* w_gate, const float* b_gate, int E, int k,
                        double capacity_factor,
                        int32_t* topk_idx, float* topk_gate, int32_t* slot_pos,
                        int32_t* perm_token, int32_t* offsets, float* inv_norm,
                        void* stream);

/* Per-expert slot capacity used by luffy_route: ceil(cf*k*T/E - 1e-9),
 * evaluated in double precision left to right (the 1e-9 keeps a product that
 * is an integer but for the binary rounding of a decimal factor, such as
 * 1.1*2*4000/8, at that integer).  0 (no limit) for cf <= 0 or a
 * non-positive size; at most INT_MAX.  Host arithmetic.  A caller sizing
 * luffy_condense's max_bucket as min(T, C) gets the same C as the routing. */
int luffy_capacity(int T, int k, int E, double capacity_factor);

/* ------------------------------------------------------------------------
 * luffy_condense - per-bucket similarity, representative selection and
 * compaction (Sec. 5.1 steps 1 and 3, Sec. 5.2, Sec. 6).
 *
 * Inside each bucket, positions a != b are joined when the cosine of their
 * embeddings is >= threshold (pairs in different buckets are never
 * compared).  A token with a zero embedding has cosine 0 with every token
 * (so it joins nothing for threshold > 0).  The degree of a
 * position is its number of edges.  Positions are then visited by
 * descending degree (lower position first on ties): a position not yet
 * decided becomes a representative and absorbs every undecided direct
 * neighbour.  Each absorbed position maps to the first representative
 * visited among its neighbours.
 *
 *   x            [T, d] dtype, device     embeddings (same as luffy_route)
 *   perm_token, offsets                   as written by luffy_route
 *   max_bucket   upper bound on any bucket size (min(T, C) for outputs of
 *                luffy_route, C from luffy_capacity); sizes the workspace.
 *                If a bucket is larger (the bound was wrong), the call still
 *                writes nothing past the workspace: no position is condensed
 *                (every position is its own representative, degrees are not
 *                written) and the compaction below runs as usual.
 *   threshold    cosine threshold h (a value > 1 disables condensation)
 *   inv_norm     [T] float, device, or NULL: 1/|x_t| as written by
 *                luffy_route for the same x; NULL computes the norms here
 * Outputs (device):
 *   rep_of_pos   [T*k] int32  position of the representative of every
 *                             position (representatives map to themselves)
 *   rep_row      [T*k] int32  row of that representative in the compacted
 *                             list (representatives in position order)
 *   rep_offsets  [E+1] int32  representatives of expert e are rows
 *                             rep_offsets[e] .. rep_offsets[e+1]-1
 *   rep_token    [T*k] int32  token of every representative row
 *   x_rep        [T*k, d] dtype or NULL   gathered representative rows
 *   degree       [T*k] int32 or NULL      degree of every position
 * Only the first offsets[E] (positions) or rep_offsets[E] (rows) entries are
 * written.
 * ---------------------------------------------------------------------- */
size_t luffy_condense_workspace_size(int T, int d, int E, int k, int max_bucket);
int luffy_condense(const void* x, int T, int d, int dtype,
                   const int32_t* perm_token, const int32_t* offsets,
                   int E, int k, int max_bucket, float threshold,
                   int32_t* rep_of_pos, int32_t* rep_row,
                   int32_t* rep_offsets, int32_t* rep_token,
                   void* x_rep, int32_t* degree, const float* inv_norm,
                   void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Similarity screen of luffy_condense (bf16 calls with d >= 2048, d a
 * multiple of 128 and T*k >= 512*E; not luffy_condense_history).  The
 * cosines of Sec. 5.1 are first estimated on fp8 (E4M3) copies of the rows,
 * each scaled by a power of two, with a bound derived from every row's
 * quantisation error: |c~ - c| <= rho_a + rho_b + rho_a*rho_b (plus room for
 * float32 rounding), rho = |x - x^| / |x|.  A 256 x 256 tile whose every
 * estimate lies outside that band around the threshold is decided by the
 * estimates, which then agree with the exact comparison for every pair; any
 * other tile is recomputed from the bf16 rows.  The outputs are the same
 * with the screen on or off.  The workspace of such calls holds the fp8
 * rows (T*d bytes).
 *
 * luffy_set_similarity_screen  on != 0 enables the screen (the default),
 *                              0 disables it for later calls in this
 *                              process; returns the previous setting.
 * luffy_similarity_screen_applies
 *                              1 if a luffy_condense call of this shape and
 *                              dtype would take the screen now, else 0.
 * ---------------------------------------------------------------------- */
int luffy_set_similarity_screen(int on);
int luffy_similarity_screen_applies(int T, int d, int E, int k, int dtype);

/* ------------------------------------------------------------------------
 * luffy_condense_history - luffy_condense with the historical similarity of
 * Sec. 5.1 step 2, for a stack of MoE blocks over the same tokens.
 *
 * The weight of a pair of tokens in one bucket is 1 when the pair's weight in
 * the previous block was above S1, 0 when it was below S2 (S1 first when both
 * hold), and the cosine otherwise (in particular when the two tokens did not
 * share a bucket in the previous block, or there is no previous block).  An
 * edge joins the pair when its weight is >= threshold; selection and
 * compaction are those of luffy_condense.
 *
 *   x ... inv_norm, max_bucket, threshold  as for luffy_condense
 *   slot_pos   [T, k] int32, device (luffy_route's): needed with hist_out
 *   hist_in    record left by the previous block (a luffy_condense_history
 *              call with the same T, E, k and max_bucket), or NULL for the
 *              first block (every pair computed).  A record from another
 *              shape, or one whose writer hit an oversized bucket, counts as
 *              empty.
 *   hist_out   record this block leaves for the next one, or NULL; it holds
 *              this block's weight classes (w > S1, w < S2) of every pair of
 *              every bucket, so the next block must use the same S1 and S2.
 *              Must not alias hist_in.  Records are luffy_history_size(T, E,
 *              k, max_bucket) bytes of device memory, 256-byte aligned,
 *              written entirely by the call.
 *   S1, S2     the two thresholds of the rule above (not NaN)
 *   stats      [4] uint64, device, or NULL: pairs (a < b of one bucket) the
 *              record left undecided, pairs it decided, 256 x 256 similarity
 *              tiles computed and tiles skipped because every pair in them
 *              was decided (bf16; float32 computes every tile)
 *   workspace  luffy_condense_history_workspace_size(T, d, E, k, max_bucket)
 * Record layout (for inspection; sections in this order, each starting at a
 * multiple of 256 bytes): int32 info[8] (a format tag, T, E, k, max_bucket);
 * int32 slot_pos[T*k]; int32 offsets[E+1]; int64 word_off[E+1]; uint64
 * hi[W]; uint64 lo[W], W = T*k*ceil(max_bucket/64).  Bit c % 64 of word
 * word_off[e] + a*ceil(n_e/64) + c/64 of hi (lo) is the class w > S1
 * (w < S2) of positions a and c of bucket e, n_e its size.
 * ---------------------------------------------------------------------- */
size_t luffy_history_size(int T, int E, int k, int max_bucket);
size_t luffy_condense_history_workspace_size(int T, int d, int E, int k, int max_bucket);
int luffy_condense_history(const void* x, int T, int d, int dtype,
                           const int32_t* perm_token, const int32_t* offsets,
                           const int32_t* slot_pos, int E, int k, int max_bucket,
                           float threshold, const void* hist_in, void* hist_out,
                           float S1, float S2,
                           int32_t* rep_of_pos, int32_t* rep_row,
                           int32_t* rep_offsets, int32_t* rep_token,
                           void* x_rep, int32_t* degree, const float* inv_norm,
                           unsigned long long* stats,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * luffy_expert_ffn - expert FFN on the representatives only (Sec. 2.1: an
 * expert is an FFN; Sec. 3: only one token of a similar group goes through
 * the expert).
 *
 *   y_rep[r] = W2_e act(W1_e x_r)   for the rows r of expert e, no biases
 *
 *   x            [*, d] dtype, device   input rows
 *   row_index    [max_rows] int32, device, or NULL: row r of the FFN reads
 *                x[row_index[r]] (pass rep_token and the embeddings to skip
 *                the gathered copy); NULL reads x[r] (e.g. x_rep)
 *   rep_offsets  [E+1] int32, device    rows of expert e
 *   w1           [E, d_ff, d] dtype, device
 *   w2           [E, d, d_ff] dtype, device
 *   max_rows     upper bound on rep_offsets[E] (T*k)
 *   y_rep        [max_rows, d] dtype, device (first rep_offsets[E] rows written)
 * The hidden activations are rounded to dtype between the two products.
 * ---------------------------------------------------------------------- */
size_t luffy_expert_ffn_workspace_size(int max_rows, int E, int d_ff, int dtype);
int luffy_expert_ffn(const void* x, const int32_t* row_index,
                     const int32_t* rep_offsets, int E, int d, int d_ff,
                     int dtype, const void* w1, const void* w2, int act,
                     int max_rows, void* y_rep,
                     void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * luffy_combine - give every slot its representative's expert output and
 * un-permute with the gates (Sec. 2.1 combine; Sec. 6 token_to_token).
 *
 *   y[t] = sum over kept slots j of topk_gate[t,j] * y_rep[rep_row[slot_pos[t,j]]]
 * A token with no kept slot gets zeros.  Sums are float32, stored as dtype.
 *   y_rep [*, d] dtype; rep_row [T*k]; slot_pos, topk_gate [T, k];
 *   y [T, d] dtype, device.
 * ---------------------------------------------------------------------- */
int luffy_combine(const void* y_rep, const int32_t* rep_row,
                  const int32_t* slot_pos, const float* topk_gate,
                  int T, int k, int d, int dtype, void* y, void* stream);

/* ------------------------------------------------------------------------
 * Backward of the condensed layer.  The paper trains the layer but does not
 * say how a gradient passes a condensed token; these calls differentiate the
 * function the forward computes with every discrete decision (routing,
 * capacity, similarity graph, representatives) held fixed, so a condensed
 * slot's gradient reaches its representative's row.
 *
 * luffy_combine_backward - transpose of luffy_combine (Sec. 2.1 combine,
 * Sec. 6 token_to_token), for dy = dL/dy:
 *   dgate[t,j] = <dy[t], y_rep[r]>,  r = rep_row[slot_pos[t,j]]  (0 if dropped)
 *   dy_rep[r]  = sum over kept slots (t,j) of representative r of
 *                topk_gate[t,j] * dy[t]
 *   dy [T, d] dtype; y_rep [max_rows, d] dtype (the forward's output);
 *   rep_row, perm_token [T*k], slot_pos, topk_gate [T, k], offsets,
 *   rep_offsets [E+1], all as the forward left them (R = rep_offsets[E]
 *   rows in use, R <= max_rows); dy_rep [max_rows, d] dtype: rows 0..R-1
 *   written; dgate [T, k] float32.  E <= 64.
 * Row sums are float32; the members of a group are added in an order that
 * is not fixed, so dy_rep may differ in the last bits between runs; dgate
 * is a fixed-order sum.  Workspace (the member lists):
 * luffy_combine_backward_workspace_size(T, k, max_rows) bytes.
 * ---------------------------------------------------------------------- */
size_t luffy_combine_backward_workspace_size(int T, int k, int max_rows);
int luffy_combine_backward(const void* dy, const void* y_rep, const int32_t* rep_row,
                           const int32_t* perm_token, const int32_t* slot_pos,
                           const float* topk_gate, const int32_t* offsets,
                           const int32_t* rep_offsets, int E, int T, int k, int d, int dtype,
                           int max_rows, void* dy_rep, float* dgate,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * luffy_expert_ffn_backward - gradients of luffy_expert_ffn (Sec. 2.1: an
 * expert is an FFN; Sec. 3: it runs on the representatives only) for
 * dy_rep = dL/dY_rep, with Z = X W1_e^T and A = act(Z) per expert e:
 *   dx_rep = (dY W2_e * act'(Z)) W1_e,  dW1_e = (dY W2_e * act'(Z))^T X,
 *   dW2_e = dY^T A  (zero for an expert without representatives).
 *   x, row_index, rep_offsets, w1, w2, act, max_rows: as for
 *   luffy_expert_ffn (Z is recomputed, nothing of the forward is kept);
 *   dy_rep [max_rows, d] bf16 (rows 0..R-1 used); dx_rep [max_rows, d] bf16
 *   (rows 0..R-1 written); dw1 [E, d_ff, d] and dw2 [E, d, d_ff] of type
 *   dw_dtype: LUFFY_F32, or LUFFY_BF16 (the weights' own type, as a bf16
 *   parameter's gradient; the float32 sums rounded once, half the bytes);
 *   another dw_dtype is LUFFY_E_INVALID.
 * bf16 only (LUFFY_E_UNSUPPORTED for float32).  Intermediates (Z, act(Z),
 * dZ and, with row_index, the gathered rows of x) are bf16 in the
 * workspace: luffy_expert_ffn_backward_workspace_size(max_rows, E, d, d_ff,
 * dtype) bytes (no copy of the weights).
 * ---------------------------------------------------------------------- */
size_t luffy_expert_ffn_backward_workspace_size(int max_rows, int E, int d, int d_ff, int dtype);
int luffy_expert_ffn_backward(const void* x, const int32_t* row_index, const int32_t* rep_offsets,
                              int E, int d, int d_ff, int dtype, const void* w1, const void* w2,
                              int act, int max_rows, const void* dy_rep, void* dx_rep,
                              void* dw1, void* dw2, int dw_dtype, void* workspace,
                              size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * luffy_adaptive_threshold - the condensation threshold h_t of training
 * iteration t from the losses of the first and of the previous iteration
 * (Sec. 5.2, Eq. 2):
 *   l_norm = (l_ini - l_prev) / l_ini,   h_t = 1 / (1 + exp(l_norm)).
 * Taken as printed: h_t = 1/2 while the loss has not moved, and it falls
 * toward 1/(1+e) (about 0.269) as the loss falls to 0; a loss above l_ini
 * gives h_t above 1/2.  For the first iteration, which has no previous loss,
 * pass l_prev = l_ini (h_1 = 1/2).  The result is what luffy_condense takes
 * as `threshold` for that iteration.  Host arithmetic in double precision;
 * no device work, no stream.
 *   l_ini   loss of the first iteration: finite and non-zero;
 *   l_prev  loss of the previous iteration: finite;
 *   h_out   host pointer that receives h_t, in [0, 1].
 * Returns LUFFY_E_INVALID, leaving *h_out unchanged, for a null h_out, a zero
 * or non-finite l_ini or a non-finite l_prev.
 * ---------------------------------------------------------------------- */
int luffy_adaptive_threshold(double l_ini, double l_prev, double* h_out);

/* ------------------------------------------------------------------------
 * Measurement hook (not part of the layer).  luffy_profile_kernel(name)
 * makes every later launch of the named kernel record a pair of HIP events
 * on the stream it runs on; NULL or "" turns this off.  luffy_profile_read
 * waits for the recorded events and returns the summed kernel time in
 * milliseconds and the number of launches since the previous read.
 * Kernel names: gate, slot_scan, slot_scatter, norm, gram, gram_recheck,
 * hist_cols, hist_gather, hist_header, greedy_round, greedy_more,
 * greedy_finish, rep_local, rep_finalize, gather, ffn_queue, ffn1, ffn2,
 * ffn2_reduce, combine; backward: cbwd_group, cbwd_rows, cbwd_gate,
 * bwd_z, bwd_act, bwd_da, bwd_dx, bwd_dx_reduce, bwd_gather, bwd_dw2,
 * bwd_dw1.
 * ---------------------------------------------------------------------- */
int luffy_profile_kernel(const char* name);
int luffy_profile_read(double* total_ms, int* launches);

#ifdef __cplusplus
}
#endif
#endif /* LUFFY_H */
