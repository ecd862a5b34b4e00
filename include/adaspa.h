/*
 * adaspa.h - C ABI of the AdaSpa attention hot path for AMD MI355X (gfx950).
 *
 * AdaSpa (arXiv 2502.21079) accelerates the 3D full attention of video
 * diffusion transformers with blockified sparse attention whose block pattern
 * is found by a precise online search that reuses log-sum-exp values across
 * denoising steps.  This library exposes the three operations of that path:
 *
 *   adaspa_dense_attn_lse     dense softmax attention + per-row LSE
 *                             (Sec. 2.2; first pass of Algorithm 1)
 *   adaspa_block_search       block attention mass W_sum_attn from a given
 *                             LSE (second pass of Algorithm 1 / Algorithm 2,
 *                             Sec. 4.1-4.2) and per-head block selection
 *                             (optimal sparse indices of Sec. 4.1, text sink
 *                             and row-wise uniform selection of Sec. 4.3)
 *   adaspa_block_sparse_attn  blockified sparse attention over the selected
 *                             key blocks (Sec. 4.1, bias form with c -> inf)
 *
 * and adaspa_fused_online_search, the first two in one launch as Algorithm 1
 * describes them (dense attention + LSE, then the masses of the same rows),
 * and adaspa_single_pass_online_search, the same results with one pass over
 * Q K^T instead of two.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Tensors are DEVICE pointers, contiguous, 16-byte aligned.
 *    Q, K, V, O: bf16 [B, H, L, D] (D innermost).  LSE: fp32 [B, H, L],
 *    natural logarithm.  W_sum_attn: fp32 [B, H, NB, NB] with NB = ceil(L/Bs).
 *  - Block rows of the sparse pattern are numbered r = (b*H + h)*NB + p for
 *    query block p; the pattern is CSR: row_ptr int32 [B*H*NB + 1] and col_idx
 *    int32, key-block indices strictly ascending within a row.
 *  - A block is a TEXT block when its token range overlaps
 *    [text_start, text_start + text_len).
 *  - Ownership: the caller owns every buffer.  No call allocates device
 *    memory, keeps a pointer after it returns, or synchronises the device:
 *    each call validates its arguments on the host, enqueues kernels on
 *    `stream` (a hipStream_t; NULL means the default stream) and returns.
 *    Counters are cleared by kernels, not memsets, so a sequence of calls
 *    with caller-allocated outputs and workspaces can be captured in a HIP
 *    graph and replayed.
 *  - Errors: invalid arguments are reported synchronously with a status code
 *    before anything is enqueued.  A failed launch returns ADASPA_ERR_HIP.
 *    A fault inside a kernel surfaces at the caller's next synchronisation.
 *  - Calls are stateless and may be issued from several host threads on
 *    different streams; calls that share an output buffer must be ordered by
 *    the caller.  (adaspa_block_sparse_attn_noalloc is the exception: its calls
 *    on one GPU share that GPU's counters and must not overlap.)
 */
#ifndef ADASPA_H_
#define ADASPA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ADASPA_OK = 0,
  ADASPA_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, bad size or range */
  ADASPA_ERR_UNSUPPORTED = 2,   /* head_dim or block outside what is built,
                                   L * D >= 2^30, or B * H >= 65536            */
  ADASPA_ERR_CAPACITY = 3,      /* col_idx capacity too small                 */
  ADASPA_ERR_WORKSPACE = 4,     /* workspace missing or too small             */
  ADASPA_ERR_HIP = 5            /* a HIP launch reported an error             */
} adaspa_status;

/* Shape of one attention call: B batches x H heads of L tokens with head
 * dimension D; square sparse blocks of Bs tokens.  Supported: D in {64, 128},
 * Bs in {64, 128}, L >= 1 (L need not be a multiple of Bs: the last block is
 * ragged and out-of-range keys never contribute), L * D < 2^30 and B * H <
 * 65536 (larger shapes return ADASPA_ERR_UNSUPPORTED).  softmax_scale <= 0 selects
 * 1/sqrt(D) (the attention-weights equation, Sec. 2.2). */
typedef struct {
  int32_t batch, heads, seqlen, head_dim;
  int32_t block;
  int32_t text_start, text_len;   /* text range for the text sink; len may be 0 */
  float softmax_scale;
} adaspa_problem;

/* Selection modes (Sec. 4.1 optimal sparse indices; Sec. 4.2 head-adaptive
 * sparsity; Sec. 4.3 row-wise uniform selection).  In every mode each video
 * query-block row of head h keeps the same count k_h of key blocks: text key
 * blocks first (text sink), then the remaining blocks by mass descending with
 * ties to the lower index.  Text query-block rows keep all NB blocks. */
enum {
  /* k_h = clamp(ceil(head_param_bp[h] * NB / 10000), max(1, #text blocks), NB) */
  ADASPA_SELECT_TOPK = 0,
  /* k_h = smallest count whose head Recall (Sec. 2.3, text rows counted as
   * fully kept) reaches head_param_bp[h] / 10000. */
  ADASPA_SELECT_COVERAGE = 1,
  /* Head-adaptive hierarchical sparsity (Sec. 4.2).  At base sparsity s
   * (base_sparsity_bp) every head keeps k(s) blocks per row; n = number of
   * heads whose Recall there exceeds recall_threshold_bp (strictly), capped at
   * floor(H/2).  The n heads of highest Recall (ties: lower head index) move
   * to sparsity (1+s)/2, the n of lowest Recall to (3s-1)/2 (at least 0);
   * k(x) is the TOPK count of keep fraction 1-x.  Heads are ranked within each
   * batch element; Recall is compared exactly.  head_param_bp is unused. */
  ADASPA_SELECT_HIERARCHICAL = 2
};

/* Flags */
enum {
  ADASPA_F_TEXT_SINK = 1,       /* force text blocks (Sec. 4.3); usually set   */
  ADASPA_F_SCORES_GIVEN = 2     /* block_mass is an INPUT: skip the mass pass  */
};

typedef struct {
  int32_t mode;                 /* ADASPA_SELECT_*                                */
  int32_t flags;                /* ADASPA_F_*                                     */
  const int32_t* head_param_bp; /* HOST array [H]: keep fraction (TOPK) or Recall
                                   target (COVERAGE) in basis points, 0..10000;
                                   applies to every batch element; may be NULL
                                   for HIERARCHICAL                              */
  int32_t base_sparsity_bp;     /* HIERARCHICAL: base sparsity s, 0..10000        */
  int32_t recall_threshold_bp;  /* HIERARCHICAL: Recall threshold, 0..10000       */
} adaspa_select;

/* Human-readable name of a status code (static storage). */
const char* adaspa_status_string(adaspa_status s);

/* Device bytes of the optional workspace of adaspa_dense_attn_lse (0 for
 * invalid arguments). */
size_t adaspa_dense_attn_workspace(const adaspa_problem* prob);

/* Dense attention with LSE (Sec. 2.2; Algorithm 1, first pass).
 *   out[b,h,i,:] = sum_j softmax_j(scale * q_i . k_j) v_j        bf16 (RNE)
 *   lse[b,h,i]   = log sum_j exp(scale * q_i . k_j)             fp32
 * q, k, v, out: bf16 [B,H,L,D]; lse: fp32 [B,H,L] (may be NULL to skip).
 * workspace (optional, caller-owned, 16-byte aligned, at least
 * adaspa_dense_attn_workspace() bytes, contents need not be initialised)
 * holds the counters of a work queue per XCD, so that the XCDs that run
 * faster take more of the work; with NULL the work is split statically.  The
 * results are bitwise the same either way.  The call clears the counters
 * itself (with a kernel on `stream`); calls that may run concurrently need
 * separate workspaces.  ADASPA_ERR_WORKSPACE if it is too small or
 * misaligned. */
adaspa_status adaspa_dense_attn_lse(const adaspa_problem* prob, const void* q,
                                    const void* k, const void* v, void* out,
                                    float* lse, void* workspace,
                                    size_t workspace_bytes, void* stream);

/* Device bytes of workspace adaspa_block_search needs for this problem and
 * selection (0 for invalid arguments). */
size_t adaspa_block_search_workspace(const adaspa_problem* prob,
                                     const adaspa_select* sel);

/* Number of col_idx entries the selection may write: the exact count for
 * TOPK, an upper bound for HIERARCHICAL (every head at the largest of its
 * three counts), B*H*NB*NB for COVERAGE (the counts depend on the data and
 * the library never synchronises to learn them).  Returns -1 for invalid
 * arguments. */
int64_t adaspa_block_search_capacity(const adaspa_problem* prob,
                                     const adaspa_select* sel);

/* Block search (Sec. 4.1-4.3; Algorithm 1 second pass / Algorithm 2).
 *   1. Unless ADASPA_F_SCORES_GIVEN: block_mass[b,h,p,c] =
 *        sum_{i in block p} sum_{j in block c} exp(scale * q_i . k_j - lse[b,h,i])
 *      with the LSE given by the caller (fresh from adaspa_dense_attn_lse, or
 *      cached from an earlier step); no renormalisation.
 *   2. Per-head count k_h (see the modes) and per-row selection, emitted as CSR
 *      into row_ptr / col_idx.  head_k int32 [B,H] and head_recall fp32 [B,H]
 *      (the head Recall at k_h) are optional outputs (may be NULL).
 * Ranking compares fp32 masses (-0 == +0, NaN last).  Cumulative masses are
 * exact: each mass m >= 0 becomes min(round_half_even(m * 2^32), cap) with
 * cap = floor(2^62 / (NB*NB)) (NaN and m <= 0 give 0); coverage holds when
 * kept * 10000 >= total * tau_bp; recall = (float)((double)kept/(double)total),
 * 1 when total is 0.
 * Supported: NB <= 8192 key blocks, H <= 512 heads and B*H*NB*NB < 2^31
 * (ADASPA_ERR_UNSUPPORTED otherwise).
 * q, k, lse may be NULL with ADASPA_F_SCORES_GIVEN.  col_capacity must be at
 * least adaspa_block_search_capacity(); workspace must hold
 * adaspa_block_search_workspace() bytes, 256-byte aligned. */
adaspa_status adaspa_block_search(const adaspa_problem* prob, const void* q,
                                  const void* k, const float* lse,
                                  const adaspa_select* sel, float* block_mass,
                                  int32_t* row_ptr, int32_t* col_idx,
                                  int64_t col_capacity, int32_t* head_k,
                                  float* head_recall, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* Fused online search (Algorithm 1, Sec. 4.2): dense attention with LSE and
 * the block masses of that fresh LSE in ONE kernel launch, then the
 * selection.  Each workgroup computes the output and LSE of 256 query rows
 * (first pass) and then the block masses of the same rows (second pass)
 * while their Q and LSE are still in registers, so Q is read once and the
 * LSE is not read back.  It produces exactly (bit for bit) what
 * adaspa_dense_attn_lse followed by adaspa_block_search with that LSE
 * produces:
 *   out, lse          as adaspa_dense_attn_lse (lse may be NULL: the masses
 *                     still use the fresh LSE)
 *   block_mass, row_ptr, col_idx, head_k, head_recall
 *                     as adaspa_block_search (ADASPA_F_SCORES_GIVEN is not
 *                     allowed: ADASPA_ERR_INVALID_ARG)
 * The workspace, its size (adaspa_block_search_workspace), the capacity
 * rule, the alignment rules and the errors are those of the two calls; the
 * workspace also holds the per-XCD work-queue counters of the fused kernel,
 * which the call clears itself. */
adaspa_status adaspa_fused_online_search(const adaspa_problem* prob, const void* q,
                                         const void* k, const void* v, void* out,
                                         float* lse, const adaspa_select* sel,
                                         float* block_mass, int32_t* row_ptr,
                                         int32_t* col_idx, int64_t col_capacity,
                                         int32_t* head_k, float* head_recall,
                                         void* workspace, size_t workspace_bytes,
                                         void* stream);

/* Device bytes of the workspace of adaspa_single_pass_online_search: the
 * workspace of adaspa_block_search plus B*H*NB*L floats of per-row block
 * masses (NB = ceil(L/Bs); 9.1 GB for B=1, H=24, L=110,336, Bs=128), rounded
 * up to 256 bytes.  0 for invalid arguments or ADASPA_F_SCORES_GIVEN. */
size_t adaspa_single_pass_online_search_workspace(const adaspa_problem* prob,
                                                  const adaspa_select* sel);

/* The least workspace adaspa_single_pass_online_search accepts: the
 * search's workspace plus the per-row block masses and row LSEs of ONE
 * (batch, head) pair (NB*L + L floats), each part rounded up to 256 bytes.
 * Given less than adaspa_single_pass_online_search_workspace() but at least
 * this, the call runs the attention pass over groups of as many (batch,
 * head) pairs as fit, one after another, then the selection of all of them;
 * the results are the same as with the full workspace.  0 for invalid
 * arguments or ADASPA_F_SCORES_GIVEN. */
size_t adaspa_single_pass_online_search_min_workspace(const adaspa_problem* prob,
                                                      const adaspa_select* sel);

/* Single-pass online search (Algorithm 1, Sec. 4.1-4.2, with one pass over
 * Q K^T): the outputs of adaspa_fused_online_search, computed differently.
 * The block mass W[p][c] is the sum over rows i of p of exp(s_ij - LSE_i)
 * over the keys j of c.  The attention pass already forms
 * exp(s_ij - m_i) for its softmax (m_i the row's running reference), so it
 * also adds those terms per (row, key block) in fp32 and keeps
 * log2 of each sum plus m_i in the workspace; once a row's LSE is known the
 * kernel turns them into the row's shares exp(y - LSE_i) and sums them over
 * the rows of each query block.  The second recomputation of Q K^T that the
 * two-pass form needs is not taken.
 *   out, lse          bit for bit those of adaspa_dense_attn_lse (lse may be
 *                     NULL: the masses still use the fresh LSE)
 *   block_mass        the masses of the fresh LSE, within 1e-3 relative of
 *                     the exact values.  They are normalised by the LSE of
 *                     the unrounded fp32 row sum; the stored lse normalises
 *                     the bf16-rounded weights of the output, so
 *                     adaspa_block_search given that lse returns masses
 *                     that differ from these by up to 2^-9 relative
 *   row_ptr, col_idx, head_k, head_recall
 *                     the selection of those masses, as adaspa_block_search
 *                     (ADASPA_F_SCORES_GIVEN is not allowed:
 *                     ADASPA_ERR_INVALID_ARG)
 * workspace must hold at least adaspa_single_pass_online_search_min_workspace()
 * bytes, 256-byte aligned (ADASPA_ERR_WORKSPACE otherwise); with
 * adaspa_single_pass_online_search_workspace() bytes every (batch, head)
 * pair runs in one launch.  It holds the selection's scratch, the per-XCD
 * work-queue counters (cleared by the call) and the per-row block masses,
 * and its contents need not be kept between calls.  Capacity, alignment and the other errors as adaspa_block_search. */
adaspa_status adaspa_single_pass_online_search(const adaspa_problem* prob, const void* q,
                                               const void* k, const void* v, void* out,
                                               float* lse, const adaspa_select* sel,
                                               float* block_mass, int32_t* row_ptr,
                                               int32_t* col_idx, int64_t col_capacity,
                                               int32_t* head_k, float* head_recall,
                                               void* workspace, size_t workspace_bytes,
                                               void* stream);

/* Device bytes of the optional workspace of adaspa_block_sparse_attn (0 for
 * invalid arguments). */
size_t adaspa_block_sparse_attn_workspace(const adaspa_problem* prob);

/* Blockified sparse attention (Sec. 4.1, bias -c(1-M) with c -> inf).
 *   out[b,h,i,:] = sum_{j in kept(p(i))} exp(scale*q_i.k_j - lseM_i) v_j
 *   lseM[b,h,i]  = log sum_{j in kept(p(i))} exp(scale * q_i . k_j)
 * where kept(p) are the key blocks col_idx[row_ptr[r] .. row_ptr[r+1]) of
 * row r = (b*H+h)*NB + p.  A row that keeps nothing gives out = 0 and
 * lseM = -inf.  Keeping every block reproduces adaspa_dense_attn_lse bit for
 * bit (both run the same main loop).  lse_out may be NULL.  col_count is
 * the number of readable col_idx entries: row bounds are clamped to
 * [0, col_count] and entries outside [0, NB) are skipped, so malformed
 * patterns never read out of bounds.  Rows should be strictly ascending
 * (a repeated block would be counted twice).  prob->text_start/text_len only
 * order the work (the text query blocks, which keep every key block under the
 * text sink, are started first) and name the block every row is expected to
 * begin with (its first tiles are loaded before the row's indices are read,
 * and reloaded if the row begins elsewhere); the results do not depend on
 * them.
 * Block 64 supports NB <= 8192 key blocks (ADASPA_ERR_UNSUPPORTED otherwise).
 * workspace (optional, caller-owned, 16-byte aligned, at least
 * adaspa_block_sparse_attn_workspace() bytes, contents need not be
 * initialised) holds per-XCD work-queue counters: the last tenth of the query
 * blocks then goes to the XCDs that run ahead; with NULL all work is split
 * statically.  The results are bitwise the same either way.  The call clears
 * the counters itself (with a kernel on `stream`); calls that may run
 * concurrently need separate workspaces.  ADASPA_ERR_WORKSPACE if it is too
 * small or misaligned. */
adaspa_status adaspa_block_sparse_attn(const adaspa_problem* prob, const void* q,
                                       const void* k, const void* v,
                                       const int32_t* row_ptr,
                                       const int32_t* col_idx, int64_t col_count,
                                       void* out, float* lse_out, void* workspace,
                                       size_t workspace_bytes, void* stream);

/* adaspa_block_sparse_attn without a workspace argument and without any
 * allocation, for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc).  It
 * computes exactly what adaspa_block_sparse_attn computes with a workspace
 * (bitwise the same outputs) and takes the same arguments and checks, except
 * that the per-XCD work-queue counters live in a 256-byte array inside the
 * library, one per GPU, held from the library's load until the process ends.
 * The current device must be the one `stream` belongs to.  Every call on a
 * GPU shares that GPU's counters (the call clears them itself with a kernel
 * on `stream`), so calls on one GPU must not overlap: issue them on one
 * stream, or order them; overlapping calls race on the counters.  Returns
 * ADASPA_ERR_WORKSPACE if a problem ever needed more than the 256 bytes (no
 * supported problem does) and ADASPA_ERR_HIP if the array's device address
 * cannot be obtained.  No hipMalloc, hipFree or allocating library routine is
 * called. */
adaspa_status adaspa_block_sparse_attn_noalloc(const adaspa_problem* prob, const void* q,
                                               const void* k, const void* v,
                                               const int32_t* row_ptr,
                                               const int32_t* col_idx, int64_t col_count,
                                               void* out, float* lse_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ADASPA_H_ */
