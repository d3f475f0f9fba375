/*
 * gt_attn.h -- fused graph-transformer attention forward over a CSR graph,
 * for AMD Instinct MI355X (gfx950).
 *
 * Operation (paper: Section 2.2, attention-based family (iii) with the
 * graph-transformer logits e_ij = q_i . k_j / sqrt(D); fused single-pass
 * evaluation: Section 3.2 and Appendix D.2, "Fused forward in CSR" and
 * "Online softmax and fused aggregation"):
 *
 *   for every destination row i in [0, N) and head h in [0, H):
 *     s_e           = scale * sum_d Q[i,h,d] * K[j_e,h,d]   for each CSR entry e of row i,
 *                                                           j_e = colidx[e]
 *     out[i,h,:]    = sum_e softmax_e(s) * V[j_e,h,:]
 *
 *   Every CSR entry is one softmax term (a repeated entry counts twice); no
 *   self-loop is added beyond what the CSR lists.  A row with no entries
 *   yields out[i,h,:] = 0.  Scores, probabilities and per-edge messages are
 *   never written to memory: each row is streamed once with a running
 *   (max, sum, accumulator) state, and partial states of split rows are
 *   merged by rescaling with exp(m_part - m_total) (Appendix D.2, "Cross-warp
 *   merge and normalization").
 *
 * Layouts (all row-major, dense):
 *   rowptr  int64  [N+1]   rowptr[0] = 0, non-decreasing, rowptr[N] = E
 *   colidx  int32  [E]     source ids in [0, N); rows need not be sorted
 *   Q, K, V, out  [N][H][D] elements; fp32, or bf16 as raw uint16 bit patterns
 *
 * Precision: loads fp32 or bf16 (bf16 is widened exactly), accumulates in
 * fp32, exponentials in base 2 on a log2(e)-prescaled score; bf16 outputs
 * are rounded to nearest even from the fp32 result.  Inf and NaN in the K or
 * V row of a node reach only the rows whose entries name that node (there
 * the output is non-finite where the exact result is, elementwise for V).
 *
 * Ownership and memory: every pointer argument is DEVICE memory owned by the
 * caller; the library neither frees nor retains it past the enqueued work.
 * A call works on the calling thread's current device: `stream` (0 for the
 * null stream) must belong to it, else GT_ERROR_INVALID_VALUE.
 * `out` must not overlap Q, K or V.  Q, K, V and out must be 16-byte aligned.
 * Workspace (degree-bin lists, the light-row order of narrow-row shapes,
 * partial softmax states of split rows and the work-list counters) is owned
 * by the library and private to each call while its kernels run: a call
 * takes a free workspace block of the device and, after enqueueing its
 * kernels, hands it back tagged with an event recorded on `stream`.  A later
 * call (any stream, any host thread) reuses a free block only once that
 * event has completed, or, for a block last used on its own stream, behind a
 * device-side wait on the event; otherwise it allocates a new block from the
 * library's memory pool of the device (hipMallocFromPoolAsync on `stream`).
 * The host never waits for the device, nothing is kept per stream, and free
 * blocks above 256 MiB per device go back to the pool; gt_workspace_release()
 * returns all free blocks to the device.  On a stream being captured into a
 * graph the workspace is allocated and freed stream-ordered instead (both
 * become graph nodes).
 *
 * Semantics: asynchronous.  GT_SUCCESS means the work was enqueued on
 * `stream`; device faults surface at the caller's next synchronisation.
 * N == 0 enqueues nothing.  The CSR structure is a precondition (checked by
 * gt_csr_validate, never on this path); a malformed CSR is undefined behaviour.
 *
 * Errors: arguments are validated on the host before any device work;
 * failures return a gt_status and set a thread-local message readable with
 * gt_last_error_message().  Validation never reads device memory.
 *
 * Supported shapes: H in {1, 2, 4, 8} with D in {32, 64, 128, 256}, and for
 * bf16 features also D = 512 with H in {1, 2, 4} (one head's D elements must
 * fit 64 lanes of 16 bytes); 0 <= E < 2^31; 0 <= N < 2^31.
 */
#ifndef GT_ATTN_H
#define GT_ATTN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
/* In C++ the enumerations below have int as their fixed underlying type, so
 * any int a C caller passes is a valid value there (and is refused by the
 * argument checks) rather than an out-of-range enumeration value. */
#define GT_ENUM_BASE : int
#else
#define GT_ENUM_BASE
#endif

typedef enum gt_status GT_ENUM_BASE {
    GT_SUCCESS = 0,
    GT_ERROR_INVALID_VALUE = 1, /* null pointer, bad size, misalignment, aliasing, non-finite scale */
    GT_ERROR_NOT_SUPPORTED = 2, /* (H, D) or dtype outside the compiled set */
    GT_ERROR_OUT_OF_MEMORY = 3, /* workspace allocation failed */
    GT_ERROR_HIP = 4            /* a HIP runtime call or kernel launch failed */
} gt_status;

typedef enum gt_dtype GT_ENUM_BASE {
    GT_DTYPE_F32 = 0,
    GT_DTYPE_BF16 = 1
} gt_dtype;

/*
 * fp32 features.  out[i,h,:] as defined above.  scale is typically 1/sqrt(D)
 * (the paper's logit scaling, Section 2.2) and must be finite.
 */
gt_status gt_attn_fwd(const int64_t* rowptr, const int32_t* colidx, const float* Q,
                      const float* K, const float* V, float* out, int64_t N, int64_t E,
                      int32_t H, int32_t D, float scale, hipStream_t stream);

/*
 * bf16 features given as uint16 bit patterns; fp32 accumulation; bf16 output
 * rounded to nearest even.  Scores are bf16 dot products accumulated in fp32;
 * the fp32 softmax weights multiply the exactly widened value rows (in dense
 * tiles, each weight as the sum of two bf16 terms); the largest weight of a
 * row is exactly 1, so a single-entry row returns its value exactly.
 * Otherwise identical to gt_attn_fwd.
 */
gt_status gt_attn_fwd_bf16(const int64_t* rowptr, const int32_t* colidx, const uint16_t* Q,
                           const uint16_t* K, const uint16_t* V, uint16_t* out, int64_t N,
                           int64_t E, int32_t H, int32_t D, float scale, hipStream_t stream);

/*
 * Work-partition overrides (Appendix B.1 and D.1: degree-aware allocation of
 * rows to wavefronts, with light/heavy thresholds and per-chunk edge counts
 * that the paper tunes by grid search).  A field <= 0 selects the default.
 *   light_max_deg : rows of degree <= this are handled by one lane group
 *                   (a sub-wavefront) each (default 8 steps of the group)
 *   heavy_min_deg : rows of degree >= this are scheduled first; those longer
 *                   than one chunk are split into chunks processed by
 *                   different wavefronts and merged afterwards; rows in
 *                   between get one wavefront each (default 256; on graphs
 *                   whose default chunk exceeds 1024 and where a wavefront
 *                   holds two or more rows, a quarter of that chunk, except
 *                   for the GATv2 forward)
 *   chunk_edges   : CSR entries per chunk of a split row, rounded up to a
 *                   multiple of 64; a row is cut into at most 32 chunks, so
 *                   very long rows get longer chunks (default: from the
 *                   call's gather time at about 7 TB/s and one microsecond
 *                   per step: up to half of it in steps, at most 1024
 *                   entries, down to 64 on small graphs; where an eighth of
 *                   it exceeds 1024 entries, that eighth, up to 8192 (not for
 *                   the GATv2 forward).  With fp32 4x32 features the
 *                   graph-transformer forward gets 1024 on the arxiv-shaped
 *                   169K-node graph and 8192 on R-MAT scale 21; the GATv2
 *                   forward 768 and 1024)
 *   grid_blocks   : workgroups of the attention kernel, rounded up to a
 *                   multiple of 8 (default: about two light work items per
 *                   wavefront, within 4x..64x the resident workgroups)
 *   dense_tiles   : threshold of the matrix-core path for locally dense
 *                   graphs (Section 3.3 and Appendix D.3: block-sparse
 *                   tiles); bf16 features with H*D <= 128 only, ignored
 *                   otherwise.  0 (default) selects 256; a negative value
 *                   turns the path off.  Rows are grouped in aligned windows
 *                   of 64 ids.  The partition estimates each window's
 *                   entries that point inside the window from a sample (the
 *                   middle entry of every 8th light row) and lists the
 *                   windows estimated to hold at least `dense_tiles` of them
 *                   (with 1: every window with a light row).  The light rows
 *                   of a listed window are computed by the tile kernel: their
 *                   in-window entries as masked 64x64 tiles with bf16 MFMA
 *                   (scores and P*V), then each row's remaining entries
 *                   streamed; all other rows by the CSR kernel.  The
 *                   normaliser and lse sum the fp32 weights (for P*V see
 *                   bf16_weights).
 *   bf16_weights  : bf16 features only (ignored for fp32).  0 (default):
 *                   the softmax weights stay fp32 and multiply the exactly
 *                   widened value rows in fp32 (in dense tiles: each weight
 *                   as the sum of two bf16 terms, exact to 2^-17 relative,
 *                   with two P*V products).  Nonzero: each weight is rounded
 *                   to bf16 before it multiplies its value row, two entries
 *                   per bf16 dot2 (fewer vector instructions where the step
 *                   is arithmetic-bound); out is then within
 *                   2^-8 sum_e alpha_e |v_e| of the fp32-weight result.
 * Fields above 2^31 - 2^16 are refused (GT_ERROR_INVALID_VALUE).
 * Results are bitwise reproducible for fixed settings; different settings
 * change only the rounding.
 */
typedef struct gt_tuning {
    int32_t light_max_deg;
    int32_t heavy_min_deg;
    int32_t chunk_edges;
    int32_t grid_blocks;
    int32_t dense_tiles;
    int32_t bf16_weights;
} gt_tuning;

/*
 * Generic entry: dtype selects fp32 (void* = float*) or bf16 (void* =
 * uint16_t*); tuning may be NULL (defaults).  Same contract as gt_attn_fwd.
 * lse (may be NULL): device float [N][H], receives the natural-log
 * logsumexp of each row's scaled scores, ln(sum_e exp(s_e)), -inf for an
 * empty row -- the per-node statistic the paper stores so the backward pass
 * can recompute the attention weights (Appendix D.2).  4-byte aligned, must
 * not overlap the other buffers.
 */
gt_status gt_attn_fwd_ex(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx,
                         const void* Q, const void* K, const void* V, void* out, float* lse,
                         int64_t N, int64_t E, int32_t H, int32_t D, float scale,
                         const gt_tuning* tuning, hipStream_t stream);

/*
 * Allocation-free variant of gt_attn_fwd_ex, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation.  Same arguments, results (bit-identical to
 * gt_attn_fwd_ex with the same settings), validation and asynchrony; it calls
 * no hipMalloc, hipFree or other allocating routine, and records no
 * profiling events.  Its workspace is a 256 MiB device array of the library
 * (one per device, held from the library's load until the process ends):
 * a call whose workspace would exceed it (very large graphs, or tunings with
 * many short chunks) returns GT_ERROR_INVALID_VALUE and enqueues nothing.
 * All calls of this entry point on one device share that array, and each
 * call leaves its contents behind: calls that overlap in time on one device
 * (concurrent streams, or host threads) race and give undefined results, so
 * serialise them (one stream, or events between streams).
 */
gt_status gt_attn_fwd_noalloc(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx,
                              const void* Q, const void* K, const void* V, void* out, float* lse,
                              int64_t N, int64_t E, int32_t H, int32_t D, float scale,
                              const gt_tuning* tuning, hipStream_t stream);

/*
 * GATv2 forward (paper Section 2.2, the GATv2 member of the attention family;
 * Appendix D.2, "Fused forward in CSR (GATv2)"), on the same fused streaming
 * pass and degree-aware partition as gt_attn_fwd_ex:
 *
 *     s_e        = sum_d att[h,d] * LeakyReLU(L[i,h,d] + R[j_e,h,d])
 *     out[i,h,:] = sum_e softmax_e(s) * R[j_e,h,:]
 *
 * with LeakyReLU(x) = x for x > 0, else slope * x.  L and R are the
 * precomputed per-node features (the two linear maps of the layer applied to
 * the node states); R gives both the score operand and the value, so each CSR
 * entry gathers one row.  No logit scaling.  An empty row yields zeros.
 * Layouts: L, R, out [N][H][D] in `dtype` (16-byte aligned; out must not
 * overlap L or R); att fp32 [H][D] device memory, 16-byte aligned; lse
 * (may be NULL) float [N][H], ln(sum_e exp(s_e)), -inf for an empty row.
 * slope must be finite.  tuning as for gt_attn_fwd_ex, except dense_tiles,
 * which is ignored.  Same ownership, workspace, asynchrony and error contract
 * as gt_attn_fwd.
 */
gt_status gt_gatv2_fwd(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx, const void* L,
                       const void* R, const float* att, float slope, void* out, float* lse,
                       int64_t N, int64_t E, int32_t H, int32_t D, const gt_tuning* tuning,
                       hipStream_t stream);

/*
 * Backward pass (paper Appendix D.2, backward of the graph transformer):
 * gradients dQ, dK, dV of sum(out * dout) for the forward defined above.
 * The attention weights are recomputed from lse, the forward's per-row
 * statistic (gt_attn_fwd_ex), as alpha_e = exp(s_e - lse_i); with
 * Delta_i = <out_i, dout_i> per head and ds_e = alpha_e (<dout_i, V_j> - Delta_i):
 *     dQ_i = scale sum_e ds_e K_j,   dK_j = scale sum_e ds_e Q_i,
 *     dV_j = sum_e alpha_e dout_i    (e = (i, j) over CSR entries).
 * rowptr_t / colidx_t is the transposed structure: row j lists, once per
 * CSR entry, every destination i whose row holds j (the order within a row
 * fixes the summation order; a fixed structure gives bitwise-reproducible
 * gradients).  out and lse must come from the forward of the same inputs.
 * Layouts: Q, K, V, out, dout, dQ, dK, dV [N][H][D] in `dtype`, 16-byte
 * aligned; lse float [N][H].  Gradients are accumulated in fp32 and written
 * in `dtype` (bf16 rounded to nearest even); they must not overlap the
 * inputs or each other.  With bf16 features the two dot products per entry
 * are bf16 dot products accumulated in fp32, and each entry's coefficients
 * (ds and alpha) are rounded to bf16 before they multiply its vectors.
 * Asynchronous on `stream`; workspace as for gt_attn_fwd.
 */
gt_status gt_attn_bwd(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx,
                      const int64_t* rowptr_t, const int32_t* colidx_t, const void* Q,
                      const void* K, const void* V, const void* out, const void* dout,
                      const float* lse, void* dQ, void* dK, void* dV, int64_t N, int64_t E,
                      int32_t H, int32_t D, float scale, hipStream_t stream);

/*
 * Segment min/max aggregation (paper Section 2.2, reduction family (ii):
 * h_i <- REDUCE over the sources j of row i of h_j; Appendix, degree-aware
 * reduction-based aggregation with the order-preserving (value, index) merge):
 *
 *     out[i,f] = the min (or max) over the CSR entries e of row i of X[j_e,f]
 *     arg[i,f] = the source j_e that attains it
 *
 * Values are ordered by the paper's order-preserving key (the fp32 bit pattern
 * with every bit inverted when the sign bit is set and the sign bit set
 * otherwise, compared unsigned): non-NaN values in their real order, -0 below
 * +0, a NaN with the sign bit clear above +inf and one with it set below -inf.
 * Equal values resolve to the smallest source index, for min and for max.  An
 * empty row gives out = 0 and arg = -1.  The result is exact (a selected input
 * value) and does not depend on the row's entry order or on the tuning.
 * Layouts: X, out [N][F] in `dtype` (16-byte aligned, no overlap); arg int32
 * [N][F] (16-byte aligned) or NULL to skip it.  Supported F: rows of 64 B to
 * 4 KiB in powers of two (fp32 F in {16, ..., 1024}, bf16 F in {32, ..., 2048}).
 * tuning: light_max_deg, heavy_min_deg, chunk_edges and grid_blocks as for
 * the attention forward (the degree-aware split of Appendix B.1 / D.1);
 * dense_tiles is ignored.  Same ownership, workspace, asynchrony and error
 * contract as gt_attn_fwd.
 */
typedef enum gt_reduce_op GT_ENUM_BASE {
    GT_REDUCE_MIN = 0,
    GT_REDUCE_MAX = 1
} gt_reduce_op;

gt_status gt_segment_reduce(gt_dtype dtype, gt_reduce_op op, const int64_t* rowptr,
                            const int32_t* colidx, const void* X, void* out, int32_t* arg,
                            int64_t N, int64_t E, int32_t F, const gt_tuning* tuning,
                            hipStream_t stream);

/*
 * Locality microbenchmark of the paper's reordering study (Section 4, graph
 * reordering; the appendix figure of the reordering gap): the "dot-aggr"
 * kernel, read here as
 *
 *     out[i] = sum over the CSR entries e of row i of sum_f X[i,f] * X[j_e,f]
 *
 * (fp32; an empty row gives 0), evaluated by one wavefront per row under one
 * of two mappings with identical arithmetic:
 *   mapping 0, feature-parallel: lanes span the features, neighbours are
 *              scanned in turn (coalesced loads of one neighbour row);
 *   mapping 1, neighbour-parallel: each lane takes its own neighbours and
 *              reads their whole rows (gather-like loads).
 * load_bytes selects scalar (4) or vectorised (16) loads per lane.  F in {32,
 * 64, 128, 256, 512}.  X [N][F] fp32, 16-byte aligned; out float [N].  The
 * sum order differs between variants (fp32 accumulation per lane, then a tree
 * over the wavefront).  Asynchronous on `stream`; no workspace.
 */
gt_status gt_dot_aggr(const int64_t* rowptr, const int32_t* colidx, const float* X, float* out,
                      int64_t N, int64_t E, int32_t F, int32_t mapping, int32_t load_bytes,
                      hipStream_t stream);

/*
 * Debug utility, never on the attention path: checks on the device that
 * rowptr[0] == 0, rowptr is non-decreasing, rowptr[N] == E and every colidx
 * entry lies in [0, N).  Synchronous on `stream`; *valid (host memory) is set
 * to 1 for a well-formed CSR, else 0.
 */
gt_status gt_csr_validate(const int64_t* rowptr, const int32_t* colidx, int64_t N, int64_t E,
                          int32_t* valid, hipStream_t stream);

/* Static description of a status code. */
const char* gt_status_string(gt_status status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* gt_last_error_message(void);

/*
 * Kernel timing for benchmarking.  While enabled, every attention call
 * records HIP events on its stream around its three phases: [0] partition
 * (counter reset + degree binning), [1] the attention kernels (the dense-tile
 * kernel, when enabled, and the CSR kernel), [2] the merge of split rows.  gt_profile_collect waits for the recorded events, adds their
 * elapsed milliseconds into ms[0..2], sets *calls, and clears the record.
 * Enabling or disabling also clears it.  Process-wide, thread-safe.
 */
gt_status gt_profile_enable(int32_t enable);
gt_status gt_profile_collect(double ms[3], int64_t* calls);

/*
 * Memory of the library's workspace on `device` (host outputs): bytes the
 * pool holds from the device (free blocks kept for reuse included), and bytes
 * of workspace blocks held by calls still being enqueued on the host (0 when
 * no call is in progress; a returned call's block is free for reuse once its
 * kernels are done).  Both 0 before the device's first call.
 */
gt_status gt_workspace_pool_stats(int32_t device, uint64_t* reserved_bytes, uint64_t* used_bytes);

/*
 * Returns the free workspace blocks and the unused memory of the library's
 * workspace pools to the devices: waits for each free block's last use
 * (hipEventSynchronize), frees it, then trims the pool (hipMemPoolTrimTo).
 * Blocks held by calls in progress are not affected; safe to call at any time
 * from any thread.  Blocking: it waits for the device work that last used a
 * free block.
 */
gt_status gt_workspace_release(void);

#undef GT_ENUM_BASE

#ifdef __cplusplus
}
#endif

#endif /* GT_ATTN_H */
