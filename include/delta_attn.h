/*
 * delta_attn.h -- C ABI of the MI355X (gfx950) Delta Attention prefill library.
 *
 * Delta Attention (arXiv 2505.11254, Sec. 3, Algorithm 1) corrects a sparse
 * attention output with the difference between dense and sparse attention
 * taken at every gamma-th query row:
 *
 *   out_i = (A*V)_i + [ (A~V)_a - (A*V)_a ],   a = floor(i/gamma)*gamma   (Eq. 6)
 *
 * where A*V is StreamingLLM attention (sink tokens + sliding window, softmax
 * normalised over the selected keys) and A~V is dense causal attention
 * evaluated only at the anchor rows a (Eq. 4).  Rows past the last whole
 * group of gamma rows are computed densely (implementation-details appendix).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tensors are token-major, contiguous, IEEE bfloat16 (bit patterns):
 *   q, out : [T, Hq, d]      k, v : [T, Hkv, d]
 * T = B*N for the fixed-length calls; T = cu_seqlens[B] for the _varlen
 * calls, where sequence b occupies token rows [cu_seqlens[b], cu_seqlens[b+1]).
 * All positions (causality, sinks, window, anchors) are local to a sequence;
 * sequences never attend to each other.
 *   - scale 1/sqrt(d) (Eq. 1), causal with the diagonal included (Sec. 2);
 *   - GQA: query head h reads kv head floor(h / (Hq/Hkv));
 *   - sparse key set of row i: { j <= i : j < n_sink  or  i - j < window };
 *   - anchors: rows i with i mod gamma = 0 and i < floor(L/gamma)*gamma.
 * d must be 64 or 128.  Every pointer is a device pointer, 16-byte aligned;
 * the caller owns all memory.  `out` must not overlap q, k, v or the
 * workspace.  `stream` is a hipStream_t (NULL: the null stream).
 *
 * Calls validate every argument before any HIP call; on error nothing is
 * enqueued and `out` is untouched.  On success the work is only enqueued on
 * `stream`; nothing synchronises.  Device faults surface at the caller's
 * next synchronisation.  cu_seqlens (int32, B+1 entries, device) must start
 * at 0 and be non-decreasing with every length <= max_seqlen; the library
 * cannot check device-resident values, and violating this is undefined.
 * Concurrent calls must not share a workspace.  No call keeps a pointer.
 */
#ifndef DELTA_ATTN_H
#define DELTA_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DA_ABI_VERSION 2

typedef enum {
  DA_OK = 0,
  DA_ERR_NULL = 1,        /* a required pointer is NULL */
  DA_ERR_SHAPE = 2,       /* B, N/max_seqlen, Hq or Hkv < 1, Hq % Hkv != 0, or sizes overflow */
  DA_ERR_PARAM = 3,       /* window < 1, n_sink < 0 or gamma < 1 */
  DA_ERR_UNSUPPORTED = 4, /* d not in {64, 128}, or the current device is not gfx950 */
  DA_ERR_ALIGN = 5,       /* a tensor or workspace pointer is not 16-byte aligned */
  DA_ERR_WORKSPACE = 6,   /* workspace NULL or smaller than da_workspace_bytes() */
  DA_ERR_HIP = 7          /* a HIP runtime call failed; see da_last_hip_error() */
} da_status;

/*
 * Delta Attention prefill (Algorithm 1), fixed-length batch of B sequences
 * of N tokens.  Writes the corrected output to `out`.
 * workspace: device memory of at least da_workspace_bytes(B, N, Hq, Hkv, d,
 * gamma) bytes, used for the strided rows' partial results and fp32 rows at
 * the anchors; its contents on entry do not matter.
 * Two launch schedules compute the result (see delta_attn_prefill_steps);
 * this call takes the fused one whenever da_fused_supported(Hq, Hkv, gamma),
 * else the unfused one.  The fused schedule rounds a corrected row to bf16
 * once (bf16(sparse + Delta)); the unfused one rounds the sparse row first
 * and again after adding Delta.  Anchor rows, covered groups and dense tail
 * rows are bitwise the same under both.
 */
da_status delta_attn_prefill(const void* q, const void* k, const void* v, void* out,
                             int B, int Hq, int Hkv, int N, int d,
                             int window, int n_sink, int gamma,
                             void* workspace, size_t workspace_bytes, void* stream);

/* As delta_attn_prefill for a ragged batch packed with cu_seqlens (device, int32). */
da_status delta_attn_prefill_varlen(const void* q, const void* k, const void* v, void* out,
                                    const int32_t* cu_seqlens, int B, int max_seqlen,
                                    int Hq, int Hkv, int d, int window, int n_sink, int gamma,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * The steps of Algorithm 1 one at a time, for measuring each kernel on its
 * own.  `steps` is a non-empty subset of DA_STEP_SPARSE, DA_STEP_DENSE_ROWS
 * and DA_STEP_CORRECT, optionally with DA_STEP_FUSED; the steps it names run
 * in the schedule's order, on `stream`, with the same buffers.  A later step
 * reads what earlier calls left in `out` and the workspace.
 * Unfused schedule (no DA_STEP_FUSED), in this order:
 *   DA_STEP_SPARSE      step 1: A*V for every row into `out`, plus an fp32 copy
 *                       of the anchor rows in the workspace;
 *   DA_STEP_DENSE_ROWS  steps 2-3: A~V at the anchors (Eq. 4) and at the dense
 *                       tail rows, as key-chunk partial results in the workspace;
 *   DA_STEP_CORRECT     steps 4-5 (Eq. 6): merge the partials, form Delta and
 *                       add it to the gamma rows of each group in `out`.
 * Fused schedule (DA_STEP_FUSED), in this order:
 *   DA_STEP_DENSE_ROWS  as above;
 *   DA_STEP_CORRECT     merge the partials into fp32 dense rows (workspace);
 *   DA_STEP_SPARSE      steps 1, 4-5: A*V for every row, stored as
 *                       bf16(A*V + Delta) (Eq. 6) with Delta formed from the
 *                       anchor's fp32 sparse row inside the kernel; anchor and
 *                       tail rows store the dense row.
 * The fused schedule needs every group of gamma rows inside one head's row
 * slab of a sparse-kernel workgroup (da_fused_supported); otherwise
 * DA_STEP_FUSED gives DA_ERR_UNSUPPORTED.  All steps of one schedule, in
 * order (or one call with DA_STEP_ALL, plus DA_STEP_FUSED for the fused
 * one), equal one delta_attn_prefill[_varlen] call that takes that schedule.
 * cu_seqlens may be NULL: then B sequences of max_seqlen tokens each.
 * Other arguments and errors as delta_attn_prefill_varlen; a `steps` value
 * with none of the three step bits, or with other bits, gives DA_ERR_PARAM.
 */
#define DA_STEP_SPARSE 1u
#define DA_STEP_DENSE_ROWS 2u
#define DA_STEP_CORRECT 4u
#define DA_STEP_ALL 7u
#define DA_STEP_FUSED 8u
da_status delta_attn_prefill_steps(const void* q, const void* k, const void* v, void* out,
                                   const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                   int Hkv, int d, int window, int n_sink, int gamma,
                                   void* workspace, size_t workspace_bytes, void* stream,
                                   unsigned steps);

/*
 * 1 if the fused schedule serves these sizes, else 0: some power of two h
 * dividing Hq/Hkv, h <= 8, has 256/h (the rows per query head of one sparse
 * workgroup) a multiple of gamma.  The fused schedule swaps the in-place
 * correction pass over `out` for a merge of the dense rows before the
 * sparse kernel, which then stores the corrected rows itself.
 */
int da_fused_supported(int Hq, int Hkv, int gamma);

/*
 * Correction variants of step 5 of Algorithm 1 (Sec. 3 and the interpolation
 * appendix): Steps 1-4 as in delta_attn_prefill; then, for the rows r of the
 * whole groups, out_r = (A*V)_r + c_r with, for anchor a_i = i*gamma and
 * Delta_i = (A~V)_{a_i} - (A*V)_{a_i}:
 *   DA_CORR_DELTA      c_r = Delta_{floor(r/gamma)}                    (Eq. 6)
 *   DA_CORR_RECOMPUTE  c_r = Delta_i at r = a_i, 0 elsewhere: the dense row
 *                      replaces the sparse one at anchors only         (Eq. 5)
 *   DA_CORR_INTERP     c_{a_i+k} = (1-b_k) Delta_i + b_k Delta_{i+1},
 *                      b_k = k/(gamma-1) rising from 0 to 1 over the group;
 *                      the last group keeps Delta_i.  Uses the next anchor,
 *                      so it is not causal.
 *   DA_CORR_EMA        exponential moving average with weight p0 in [0,1]
 *                      over repeat(Delta, gamma): E_r = (1-p0) E_{r-1} +
 *                      p0 D_r, E_{-1} = D_0; c_r = E_r
 *   DA_CORR_ABG        alpha-beta-gamma filter over Delta_0, Delta_1, ...
 *                      with coefficients (p0, p1, p2) for position, velocity
 *                      and acceleration; c_r = filtered Delta_{floor(r/gamma)}.
 *                      The recursion is unstable where the spectral radius of
 *                      (I - g e0^T) F exceeds 1 (gain g = (p0, p1, p2), F the
 *                      constant-acceleration transition with unit step), as
 *                      for (0.05, 1.25e-4, 2.08e-5): 1.0023 per anchor.  Its
 *                      output then grows geometrically with the anchor count,
 *                      and so do its rounding differences from an exact
 *                      evaluation.
 * Rows past the last whole group take the dense result.  DA_CORR_DELTA and
 * DA_CORR_RECOMPUTE take the fused schedule when da_fused_supported() (as
 * delta_attn_prefill does), the other modes the unfused one.  cu_seqlens may be
 * NULL (B sequences of max_seqlen tokens).  workspace needs
 * da_workspace_bytes_correction(..., mode) bytes.  Errors as
 * delta_attn_prefill_varlen, plus DA_ERR_PARAM for an unknown mode, a
 * non-finite parameter or an EMA weight outside [0,1].
 */
#define DA_CORR_DELTA 0
#define DA_CORR_RECOMPUTE 1
#define DA_CORR_INTERP 2
#define DA_CORR_EMA 3
#define DA_CORR_ABG 4
da_status delta_attn_prefill_correction(const void* q, const void* k, const void* v, void* out,
                                        const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                        int Hkv, int d, int window, int n_sink, int gamma,
                                        int mode, float p0, float p1, float p2, void* workspace,
                                        size_t workspace_bytes, void* stream);

/*
 * Delta Attention over other sparse bases (Sec. 3: the correction applies to
 * any sparse attention f*; Sec. 4 pairs it with StreamingLLM, MInference, HiP
 * and Star Attention).  f* is given by key-block lists: keys are grouped in
 * tiles of 64 positions and query rows in blocks of block_q rows, both local
 * to each sequence.  For sequence b, kv head g and query block qb the list
 * names the key tiles that the block's rows attend to; the tiles overlapping
 * the query block itself (tile >= qb*block_q/64) are always attended.  Row i
 * of a query head of group g then sees
 *   S(i) = { j <= i : tile(j) listed for (b, g, i/block_q), or
 *                     tile(j) >= (i/block_q)*block_q/64 },
 * normalised over S(i) only; Algorithm 1 runs on top unchanged.
 *
 * block_ptr: int32 [B][Hkv][nqb + 1], nqb = ceil(max_seqlen / block_q):
 *   offsets into block_idx; the list of (b, g, qb) is
 *   block_idx[block_ptr[(b*Hkv + g)*(nqb+1) + qb] .. block_ptr[... + qb + 1]).
 * block_idx: int32 key tile indices, ascending and unique within each list.
 *   Entries outside [0, qb*block_q/64) are skipped.
 * Both arrays are device memory owned by the caller; like cu_seqlens, their
 * consistency (offsets non-decreasing and inside block_idx, lists ascending
 * without repeats) is the caller's responsibility: the library cannot check
 * device-resident values, and violating it is undefined.
 * block_q must be 64, 128 or 256, and 256/h rows, h the largest power of two
 * dividing Hq/Hkv (at most 8), must not exceed it (one sparse workgroup's rows
 * per head lie in one query block); otherwise DA_ERR_UNSUPPORTED.
 */

/* f* alone under key-block lists, for every row.  cu_seqlens may be NULL (B
 * sequences of max_seqlen tokens).  Errors as sparse_attn_prefill_varlen,
 * plus DA_ERR_NULL (no lists), DA_ERR_PARAM (block_q) and DA_ERR_UNSUPPORTED. */
da_status blocksparse_attn_prefill(const void* q, const void* k, const void* v, void* out,
                                   const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                   int Hkv, int d, int block_q, const int32_t* block_ptr,
                                   const int32_t* block_idx, void* stream);

/* Delta Attention with f* under key-block lists.  steps = 0 runs the whole
 * path in the schedule the library picks (fused when
 * da_fused_supported_blocksparse()); other values select steps and schedule
 * as in delta_attn_prefill_steps.  Anchors are never assumed covered: Delta
 * is formed at every anchor.  workspace: da_workspace_bytes(B, max_seqlen,
 * Hq, Hkv, d, gamma) bytes. */
da_status delta_attn_prefill_blocksparse(const void* q, const void* k, const void* v, void* out,
                                         const int32_t* cu_seqlens, int B, int max_seqlen,
                                         int Hq, int Hkv, int d, int block_q,
                                         const int32_t* block_ptr, const int32_t* block_idx,
                                         int gamma, void* workspace, size_t workspace_bytes,
                                         void* stream, unsigned steps);

/* As da_fused_supported, with the sparse workgroup's rows per head also
 * within one query block of block_q rows (256/h <= block_q). */
int da_fused_supported_blocksparse(int Hq, int Hkv, int gamma, int block_q);

/* Workspace bytes delta_attn_prefill_correction needs (0 if the sizes or mode are invalid). */
size_t da_workspace_bytes_correction(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma,
                                     int mode);

/*
 * Sparse attention alone (f*, StreamingLLM sink + window; the first step of
 * Algorithm 1): out_i = (A*V)_i for every row.  Needs no workspace.
 */
da_status sparse_attn_prefill(const void* q, const void* k, const void* v, void* out,
                              int B, int Hq, int Hkv, int N, int d, int window, int n_sink,
                              void* stream);
da_status sparse_attn_prefill_varlen(const void* q, const void* k, const void* v, void* out,
                                     const int32_t* cu_seqlens, int B, int max_seqlen,
                                     int Hq, int Hkv, int d, int window, int n_sink,
                                     void* stream);

/*
 * Dense causal attention for every row (f, Eq. 1): the quadratic baseline the
 * method is compared with (Sec. 4.1 latency study).  Needs no workspace.
 */
da_status dense_causal_attn_prefill(const void* q, const void* k, const void* v, void* out,
                                    int B, int Hq, int Hkv, int N, int d, void* stream);
da_status dense_causal_attn_prefill_varlen(const void* q, const void* k, const void* v,
                                           void* out, const int32_t* cu_seqlens, int B,
                                           int max_seqlen, int Hq, int Hkv, int d,
                                           void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the whole
 * Delta path of delta_attn_prefill[_varlen] (cu_seqlens NULL: B sequences of
 * max_seqlen tokens each), with its workspace in a static device array of
 * DA_NOALLOC_SCRATCH_BYTES that every device the library runs on holds until
 * the process ends.  The call allocates nothing.  The strided rows split
 * their key axis into as many chunks as fit that array (fewer than
 * delta_attn_prefill takes when its workspace would not fit), so the two
 * calls can differ by rounding.  Returns DA_ERR_WORKSPACE when even one key
 * chunk does not fit (for instance a single 1M-token sequence with 32 query
 * heads); otherwise the statuses of delta_attn_prefill.  All calls on one
 * device share its array, which keeps the last call's contents: calls that
 * overlap on one device (other streams, other threads) race, so serialise
 * them.
 */
#define DA_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
da_status delta_attn_prefill_noalloc(const void* q, const void* k, const void* v, void* out,
                                     const int32_t* cu_seqlens, int B, int max_seqlen, int Hq,
                                     int Hkv, int d, int window, int n_sink, int gamma,
                                     void* stream);

/*
 * Workspace bytes delta_attn_prefill[_varlen] needs for these sizes
 * (max_seqlen = N for the fixed-length call).  0 if the sizes are invalid.
 */
size_t da_workspace_bytes(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma);

/*
 * Checks, on the GPU, the device-resident inputs the other calls take on
 * trust, and waits for the answer (this call synchronises `stream`; it is a
 * debugging aid, not for the hot path):
 *   cu_seqlens (when not NULL, B+1 entries): starts at 0, is non-decreasing,
 *     and no length exceeds max_seqlen;
 *   block_ptr / block_idx (when block_ptr is not NULL; the layout of
 *     delta_attn_prefill_blocksparse with nqb = ceil(max_seqlen / block_q),
 *     block_idx holding block_nnz entries): per (sequence, kv head) the
 *     offsets lie in [0, block_nnz] and do not decrease, and every list is
 *     strictly ascending.
 * `result` (device, int32, 4-byte aligned, caller-owned) receives the number
 * of violations.  Returns DA_OK when there are none and DA_ERR_PARAM when
 * there are some; DA_ERR_NULL without result or without anything to check,
 * DA_ERR_SHAPE / DA_ERR_PARAM for bad sizes or block_q, DA_ERR_HIP when a HIP
 * call fails.  The arrays must have the sizes stated above.
 */
da_status da_check_inputs(const int32_t* cu_seqlens, int B, int max_seqlen, int Hkv, int block_q,
                          const int32_t* block_ptr, const int32_t* block_idx, int64_t block_nnz,
                          int32_t* result, void* stream);

/*
 * How the library tiles a problem, as the launch sequence of
 * delta_attn_prefill[_varlen] uses it (block_q = 0), or of the key-block-list
 * calls (block_q = 64, 128 or 256): a host-only query, no HIP call.  A caller
 * counts the work the kernels execute (whole tiles of key_tile keys by
 * rows_per_wave query rows per wavefront) from these numbers instead of
 * restating the plan.  Each attention workgroup holds waves_per_block
 * wavefronts: heads query heads of one GQA group, each with waves_per_block /
 * heads row sub-tiles of rows_per_wave rows.  The strided dense rows split
 * their key axis into key_chunks chunks of chunk_keys keys.
 * Returns DA_ERR_NULL without `plan`, otherwise the status the whole-path
 * call would return for these sizes before touching the device.
 */
typedef struct {
  int fused;            /* 1: the whole-path call takes the fused schedule */
  int sparse_heads;     /* query heads per sparse workgroup in that schedule */
  int rows_heads;       /* query heads per strided-row (and dense causal) workgroup */
  int key_chunks;       /* key chunks of the strided dense rows */
  int chunk_keys;       /* keys per chunk, a multiple of key_tile */
  int key_tile;         /* keys per tile */
  int rows_per_wave;    /* query rows per wavefront */
  int waves_per_block;  /* wavefronts per attention workgroup */
  int sparse_slab_rows; /* rows per query head of a sparse workgroup in that schedule:
                           waves_per_block / sparse_heads * rows_per_wave (a multiple of gamma
                           when fused) */
} da_plan;

da_status da_launch_plan(int B, int max_seqlen, int Hq, int Hkv, int d, int gamma, int block_q,
                         da_plan* plan);

/* Static, NUL-terminated name of a status code. */
const char* da_status_string(da_status s);

/* The hipError_t of the last DA_ERR_HIP on the calling thread (0 if none). */
int da_last_hip_error(void);

/* DA_ABI_VERSION of the loaded library. */
int da_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DELTA_ATTN_H */
