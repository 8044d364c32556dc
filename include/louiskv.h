/*
 * libLouisKV: KV clustering and retrieval for long input/output decoding on
 * AMD Instinct MI355X (gfx950).
 *
 * The calls follow the method of "LouisKV: Efficient KV Cache Retrieval for
 * Long Input-Output Sequences" (arXiv 2510.11292):
 *   louiskv_cluster_prefill     k-means of prompt keys per (layer, KV head),
 *                               centroids as index vectors, cluster-packed
 *                               KV pool             (Section 4.2 prefill stage;
 *                                                    Algorithm 1 store_cache)
 *   louiskv_segment_output      decode-stage store_cache: local window append,
 *                               oldest-segment mean and offload
 *                                                   (Section 4.2 decode stage;
 *                                                    Algorithm 1 store_cache)
 *   louiskv_boundary_check      head-averaged query cosine vs threshold
 *                                                   (Section 4.1 equation for r_t;
 *                                                    Algorithm 1 decode loop)
 *   louiskv_retrieve            group-consistent unit scores, budgeted top
 *                               units, gather of their KV rows
 *                                                   (Appendix B equation for A_t;
 *                                                    Section 3.1 budget;
 *                                                    Algorithm 1 Retrieve)
 *   louiskv_retrieve_rows       the same selection as a list of pool rows
 *                               (zero-copy KV_critical for device pools)
 *   louiskv_sparse_decode_attn  attention over [KV_critical : KV_local]
 *   louiskv_sparse_decode_attn_rows  the same over listed pool rows
 *                                                   (Section 3.1 attention;
 *                                                    Algorithm 1 decode loop)
 *
 * Conventions shared by every call
 * --------------------------------
 * Ownership   The caller owns every buffer, including workspaces; the library
 *             never allocates or frees memory and keeps no state except a
 *             thread-local last-error string, and the static device array of
 *             the one allocation-free call
 *             (louiskv_sparse_decode_attn_rows_noalloc).
 * Pointers    Device pointers, except KV pools that the caller declares host
 *             resident (pool_on_host = 1): those must be pinned, device-mapped
 *             host memory (hipHostMalloc), which kernels read and write
 *             directly over the host link.  Such pools are checked with
 *             hipPointerGetAttributes; any other pointer is refused with
 *             LOUISKV_ERR_UNSUPPORTED before anything is launched.
 * Streams     `stream` is a hipStream_t (NULL = the legacy default stream).
 *             Arguments are validated on the host; the work is then enqueued
 *             and the call returns without synchronising.
 * Errors      Every call returns a louiskv_status.  On a validation error
 *             nothing is launched and no output is touched.  LOUISKV_ERR_HIP
 *             reports a failed HIP runtime call or launch; the text is in
 *             louiskv_last_error().  No C++ exception crosses the ABI.
 * Types       dtype LOUISKV_F32 (float32) or LOUISKV_BF16 (bfloat16 stored as
 *             uint16).  Centroids and segment means are always float32,
 *             indices always int32.  Only head dimension d = 128 is supported
 *             (LOUISKV_ERR_UNSUPPORTED otherwise).
 * Indexing    A slice is one (sequence, layer, KV head): s = (seq*L + layer)*Hkv
 *             + kv_head.  A group is one (sequence, layer): G = s / Hkv.  Query
 *             heads of group G are [Hkv*g]; heads h*g .. h*g+g-1 share KV head h
 *             (grouped-query attention, Appendix B).
 * Units       Retrieval units of a slice are its C clusters (unit 0..C-1, in
 *             cluster order) followed by its evicted output segments (unit C+e
 *             for the e-th eviction).  unit_start/unit_size give each unit's
 *             run of rows in the slice's pool; reps holds its index vector.
 */
#ifndef LOUISKV_H
#define LOUISKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LOUISKV_ABI_VERSION 1

typedef enum louiskv_status {
  LOUISKV_OK = 0,
  LOUISKV_ERR_NULL = 1,           /* a required pointer is NULL */
  LOUISKV_ERR_SHAPE = 2,          /* sizes are inconsistent or out of range */
  LOUISKV_ERR_DTYPE = 3,          /* unknown dtype code */
  LOUISKV_ERR_UNSUPPORTED = 4,    /* valid request the library does not serve (d != 128 ...) */
  LOUISKV_ERR_WORKSPACE = 5,      /* workspace NULL or smaller than *_workspace_size() */
  LOUISKV_ERR_HIP = 6             /* HIP runtime or launch failure */
} louiskv_status;

typedef enum louiskv_dtype { LOUISKV_F32 = 0, LOUISKV_BF16 = 1 } louiskv_dtype;

typedef enum louiskv_ref_mode {
  LOUISKV_REF_PREV = 0,    /* reference = previous step's query (Section 4.1 equation) */
  LOUISKV_REF_ANCHOR = 1   /* reference = query of the last boundary */
} louiskv_ref_mode;

/* Library ABI version (LOUISKV_ABI_VERSION of the build). */
int louiskv_abi_version(void);
/* Static text for a status code. */
const char* louiskv_status_str(int status);
/* Text of the last error recorded on the calling thread ("" if none). */
const char* louiskv_last_error(void);

/*
 * Local-window bookkeeping of the decode stage (Section 4.2 decode stage;
 * Algorithm 1 store_cache), a pure host function shared by callers and
 * louiskv_segment_output so both apply the same rule.
 *
 * The window keeps the most recent generated tokens in a ring of `window`
 * slots; generated token j lives in slot j % window.  When token `step`
 * (0-based) is stored while the window already holds `window` tokens, the
 * oldest `seg_len` tokens leave first and become one segment unit.
 * Outputs (any may be NULL): *evicted_segment = index e of the segment that
 * leaves while storing token `step` (its tokens are e*seg_len .. +seg_len-1),
 * or -1; *n_evicted = segments evicted after storing it; *n_local and
 * *local_start = live tokens in the window after storing it and the ring slot
 * of the oldest one.  Requires window % seg_len == 0, seg_len >= 1, step >= 0.
 */
int louiskv_window_info(int32_t step, int32_t window, int32_t seg_len,
                        int32_t* evicted_segment, int32_t* n_evicted,
                        int32_t* n_local, int32_t* local_start);

/* ------------------------------------------------------------------------ */
/* Prefill: k-means of the prompt keys of every slice.                       */
/* ------------------------------------------------------------------------ */

size_t louiskv_cluster_prefill_workspace_size(int64_t n_slices, int32_t n_tokens,
                                              int32_t d, int32_t n_clusters,
                                              int32_t dtype);

/*
 * Section 4.2 prefill stage and Algorithm 1 store_cache(prefill): group the
 * prompt keys of each slice with k-means, keep each cluster's centroid (the
 * mean of its keys) as its index vector, and store the prompt K/V rows in a
 * unified pool with each cluster as one contiguous run of rows.
 *
 * Lloyd iterations, `n_iters` times: assign every key to the nearest centroid
 * operand in squared Euclidean distance (ties to the lower index), then replace
 * every non-empty centroid by the mean of its keys (float64 sum, one rounding
 * to float32); an empty cluster keeps its centroid.  For LOUISKV_BF16 keys the
 * distance is taken to the bfloat16 rounding of each float32 centroid (the
 * matrix-core operand); for LOUISKV_F32 keys to the float32 centroid.
 *
 * keys        [n_slices][n_tokens][d] dtype, prompt keys.
 * init_idx    [n_slices][n_clusters] int32, token index of each initial centroid
 *             (values in [0, n_tokens); out-of-range values are clamped).
 * reps        out [n_slices][units_cap][d] float32: rows 0..C-1 = final centroids.
 * unit_start, unit_size
 *             out [n_slices][units_cap] int32: entries 0..C-1 = first pool row
 *             and member count of each cluster (unit_start is the CSR offset).
 * assign      out [n_slices][n_tokens] int32: cluster of each key after the
 *             last assignment (the centroids above are the means of these).
 * perm        out [n_slices][n_tokens] int32: token ids grouped by cluster,
 *             ascending inside a cluster; pool row r holds token perm[r].
 * values      [n_slices][n_tokens][d] dtype or NULL.
 * k_pool, v_pool
 *             out [n_slices][pool_rows][d] dtype or NULL: rows 0..n_tokens-1
 *             are written in perm order (keys from `keys`, values from
 *             `values`; v_pool requires values).  pool_on_host: see Pointers.
 * iter_events NULL or an array of 2*n_iters hipEvent_t recorded on `stream`
 *             just before and after each iteration's assignment kernel, for
 *             callers that time it.
 * Requires 1 <= n_clusters <= n_tokens, n_clusters <= units_cap, n_iters >= 1,
 * pool_rows >= n_tokens when a pool is given.
 */
int louiskv_cluster_prefill(const void* keys, int32_t dtype, int64_t n_slices,
                            int32_t n_tokens, int32_t d, int32_t n_clusters,
                            int32_t n_iters, const int32_t* init_idx,
                            float* reps, int32_t units_cap,
                            int32_t* unit_start, int32_t* unit_size,
                            int32_t* assign, int32_t* perm,
                            const void* values, void* k_pool, void* v_pool,
                            int64_t pool_rows, int32_t pool_on_host,
                            void* const* iter_events,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * The pool write of louiskv_cluster_prefill on its own (Algorithm 1 offload of
 * the prompt K/V): rows 0..n_tokens-1 of each slice's pools receive the keys
 * (and values) in perm order, so that each cluster is one contiguous run.
 * Lets a caller run the clustering without a pool and write the pool later,
 * on another stream, or time the two apart.
 *
 * keys, values [n_slices][n_tokens][d] dtype (values may be NULL when v_pool is).
 * perm        [n_slices][n_tokens] int32 as written by louiskv_cluster_prefill;
 *             entries are clamped into [0, n_tokens).
 * k_pool, v_pool  out [n_slices][pool_rows][d] dtype (v_pool may be NULL);
 *             pool_on_host: see Pointers.  Requires pool_rows >= n_tokens.
 */
int louiskv_pack_pool(const void* keys, const void* values, int32_t dtype,
                      int64_t n_slices, int32_t n_tokens, int32_t d,
                      const int32_t* perm, void* k_pool, void* v_pool,
                      int64_t pool_rows, int32_t pool_on_host, void* stream);

/*
 * louiskv_cluster_prefill with the pool write overlapped (Section 4.2 prefill
 * stage: clustering and offload run asynchronously; Algorithm 1
 * store_cache(prefill), asynchronous offload of (K, V)).  The slices are
 * taken in chunks of `slices_per_chunk` (one layer's KV heads is the natural
 * chunk).  Each chunk is clustered on `stream`; its pool write then runs on
 * `copy_stream`, beside the clustering of the following chunks.  Outputs and
 * pool contents are those of louiskv_cluster_prefill, bit for bit.
 *
 * Arguments as louiskv_cluster_prefill, with k_pool required, plus:
 * slices_per_chunk  >= 1; n_chunks = ceil(n_slices / min(slices_per_chunk, n_slices)).
 * copy_engine  host pools only: 1 = permute each chunk into HBM staging (in the
 *             workspace) and write it with the DMA copy engines
 *             (hipMemcpy2DAsync), leaving the compute units to the clustering;
 *             0 = a pack kernel on copy_stream writes the pool directly through
 *             the mapping, with a bounded grid.  Device pools always use the
 *             pack kernel.
 * chunk_events  n_events >= n_chunks + 1 hipEvent_t created by the caller
 *             (hipEventDisableTiming suffices); the library records event i on
 *             `stream` after chunk i and the last one on `copy_stream` after the
 *             last pool write, and makes `stream` wait for it, so that work
 *             enqueued on `stream` after this call sees the whole pool.
 * workspace   louiskv_cluster_prefill_pipelined_workspace_size(slices_per_chunk,
 *             ...) bytes; reused by every chunk.
 * stream, copy_stream  may be the same stream (no overlap).
 * Errors as louiskv_cluster_prefill; a NULL event is ERR_NULL.
 */
size_t louiskv_cluster_prefill_pipelined_workspace_size(int64_t slices_per_chunk,
                                                        int32_t n_tokens, int32_t d,
                                                        int32_t n_clusters, int32_t dtype,
                                                        int32_t pool_on_host,
                                                        int32_t copy_engine);

int louiskv_cluster_prefill_pipelined(const void* keys, int32_t dtype, int64_t n_slices,
                                      int32_t n_tokens, int32_t d, int32_t n_clusters,
                                      int32_t n_iters, const int32_t* init_idx,
                                      float* reps, int32_t units_cap,
                                      int32_t* unit_start, int32_t* unit_size,
                                      int32_t* assign, int32_t* perm,
                                      const void* values, void* k_pool, void* v_pool,
                                      int64_t pool_rows, int32_t pool_on_host,
                                      int64_t slices_per_chunk, int32_t copy_engine,
                                      void* const* chunk_events, int64_t n_events,
                                      void* workspace, size_t workspace_bytes,
                                      void* stream, void* copy_stream);

/*
 * One assignment step alone (the first half of a Lloyd iteration above), for
 * step-by-step checking: assign[s][i] = argmin_c ||keys[s][i] - op(c)||^2 over
 * the n_clusters float32 centroids at centroids[s][0..C-1] (slice stride
 * `centroid_stride` rows), op = bfloat16 rounding for LOUISKV_BF16 keys,
 * identity for LOUISKV_F32.  Ties go to the lower index.  Same workspace as
 * louiskv_cluster_prefill.
 */
int louiskv_kmeans_assign(const void* keys, int32_t dtype, int64_t n_slices,
                          int32_t n_tokens, int32_t d, int32_t n_clusters,
                          const float* centroids, int32_t centroid_stride,
                          int32_t* assign, void* workspace, size_t workspace_bytes,
                          void* stream);

/*
 * One update step alone (the second half of a Lloyd iteration): centroids_out
 * [s][c] = float32(mean of keys with assign == c), float64 sum; clusters with
 * no key copy centroids_in.  counts (out, nullable) [n_slices][n_clusters].
 * centroids_in and centroids_out may alias.  Same workspace as
 * louiskv_cluster_prefill.
 */
int louiskv_kmeans_update(const void* keys, int32_t dtype, int64_t n_slices,
                          int32_t n_tokens, int32_t d, int32_t n_clusters,
                          const int32_t* assign, const float* centroids_in,
                          float* centroids_out, int32_t centroid_stride,
                          int32_t* counts, void* workspace, size_t workspace_bytes,
                          void* stream);

/* ------------------------------------------------------------------------ */
/* Decode stage                                                              */
/* ------------------------------------------------------------------------ */

/*
 * Algorithm 1 store_cache(decode) and Section 4.2 decode stage: store this
 * step's key and value of every slice in its local window.  If the window
 * already holds `window` tokens (louiskv_window_info), its oldest `seg_len`
 * tokens leave first: their mean key (float64 sum, one rounding to float32)
 * becomes the index vector of unit n_clusters + e (reps, unit_start =
 * prompt_len + e*seg_len, unit_size = seg_len) and their K/V rows are copied
 * to pool rows prompt_len + e*seg_len .. +seg_len-1.
 *
 * k_new, v_new   [n_slices][d] dtype, this step's key and value.
 * k_local, v_local  in/out [n_slices][window][d] dtype ring buffers.
 * step           number of generated tokens stored before this one (0-based).
 * reps, unit_start, unit_size  in/out unit tables (see louiskv_cluster_prefill),
 *                capacity units_cap >= n_clusters + segments evicted.
 * k_pool, v_pool [n_slices][pool_rows][d] dtype; pool_rows >= prompt_len +
 *                step + 1 when a segment is evicted.
 */
int louiskv_segment_output(const void* k_new, const void* v_new, int32_t dtype,
                           int64_t n_slices, int32_t d,
                           void* k_local, void* v_local, int32_t window,
                           int32_t step, int32_t seg_len,
                           float* reps, int32_t* unit_start, int32_t* unit_size,
                           int32_t units_cap, int32_t n_clusters,
                           void* k_pool, void* v_pool, int64_t pool_rows,
                           int32_t prompt_len, int32_t pool_on_host, void* stream);

/*
 * Section 4.1 and Algorithm 1 decode loop: per group, r = (1/H) sum_h
 * cos(q_ref^h, q^h) over its H = n_q_heads query heads (float64, the cosine's
 * denominator clamped at 1e-30); fire = first_step || r < tau.  The reference
 * becomes q for every group in LOUISKV_REF_PREV mode, and for the groups that
 * fire in LOUISKV_REF_ANCHOR mode.
 *
 * q        [n_groups][n_q_heads][d] dtype, this step's queries.
 * q_ref    in/out [n_groups][n_q_heads][d] dtype (not read when first_step).
 * r_out    out [n_groups] float64 or NULL (NaN when first_step).
 * fire_out out [n_groups] uint8 (1 = boundary: retrieval runs this step).
 */
int louiskv_boundary_check(const void* q, void* q_ref, int32_t dtype,
                           int64_t n_groups, int32_t n_q_heads, int32_t d,
                           double tau, int32_t mode, int32_t first_step,
                           double* r_out, uint8_t* fire_out, void* stream);

size_t louiskv_retrieve_workspace_size(int64_t n_slices, int32_t units_cap,
                                       int32_t budget);

/*
 * Algorithm 1 Retrieve with the group-consistent score of Appendix B, for the
 * slices whose group fired (all slices when fire is NULL):
 *   A_u = (1/g) sum_j softmax_u(q_j . reps_u * scale) over units 0..n_units-1
 *   (float64), units ranked by A descending, equal scores by lower unit id
 *   (scores within 2^-39 of each other count as equal);
 *   the longest prefix of the ranking whose total unit_size is <= budget is
 *   selected (Section 3.1 constraint |I_t| <= B); the rows of the selected
 *   units, in rank order and ascending inside a unit, are copied from the
 *   pools into the dense KV_critical buffers.
 * Slices of groups that did not fire are left untouched (KV_critical is reused
 * until the next boundary).
 *
 * q            [n_groups][n_kv_heads*group_size][d] dtype.
 * scale        softmax temperature, normally 1/sqrt(d).
 * reps         [n_slices][units_cap][d] float32; unit_start, unit_size
 *              [n_slices][units_cap] int32; n_units <= units_cap.
 * k_pool, v_pool  [n_slices][pool_rows][d] dtype (pool_on_host: see Pointers).
 * fire         [n_groups] uint8 or NULL.
 * sel_units    out [n_slices][units_cap] int32, selected unit ids in rank order.
 * n_sel_units  out [n_slices] int32.
 * n_sel        out [n_slices] int32, selected tokens (<= budget).
 * k_buf, v_buf out [n_slices][budget][d] dtype, rows 0..n_sel-1 written.
 * scores_out   out [n_slices][units_cap] float64 or NULL.
 * Requires 1 <= group_size <= 8, 1 <= n_units <= 8192, budget >= 0.
 */
int louiskv_retrieve(const void* q, int32_t dtype, int64_t n_slices,
                     int32_t n_kv_heads, int32_t group_size, int32_t d, double scale,
                     const float* reps, const int32_t* unit_start,
                     const int32_t* unit_size, int32_t units_cap, int32_t n_units,
                     const void* k_pool, const void* v_pool, int64_t pool_rows,
                     int32_t pool_on_host, int32_t budget, const uint8_t* fire,
                     int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                     void* k_buf, void* v_buf, double* scores_out,
                     void* workspace, size_t workspace_bytes, void* stream);

size_t louiskv_retrieve_rows_workspace_size(int64_t n_slices, int32_t units_cap);

/*
 * louiskv_retrieve without the copy (zero-copy retrieval for pools in device
 * memory): the same scores, ranking and prefix-stop selection (Appendix B;
 * Section 3.1 budget; Algorithm 1 Retrieve), but instead of gathering K/V rows
 * into KV_critical it writes, per fired slice, the list of the selected pool
 * rows (rank order, ascending inside a unit).  louiskv_sparse_decode_attn_rows
 * then reads those rows from the pool directly: KV_critical becomes a list of
 * row indices rather than a copy.  Slices whose group did not fire keep their
 * previous list.
 *
 * sel_rows   out [n_slices][budget] int32, entries 0..n_sel-1 written
 *            (may be NULL when budget == 0).
 * Other arguments as louiskv_retrieve; the workspace is
 * louiskv_retrieve_rows_workspace_size() bytes.
 */
int louiskv_retrieve_rows(const void* q, int32_t dtype, int64_t n_slices,
                          int32_t n_kv_heads, int32_t group_size, int32_t d, double scale,
                          const float* reps, const int32_t* unit_start,
                          const int32_t* unit_size, int32_t units_cap, int32_t n_units,
                          int32_t budget, const uint8_t* fire, int32_t* sel_units,
                          int32_t* n_sel_units, int32_t* n_sel, int32_t* sel_rows,
                          double* scores_out, void* workspace, size_t workspace_bytes,
                          void* stream);

size_t louiskv_sparse_decode_attn_workspace_size(int64_t n_slices, int32_t group_size,
                                                 int32_t d, int32_t buf_rows,
                                                 int32_t window);

/*
 * Section 3.1 attention over Algorithm 1's KV_attn = [KV_critical : KV_local]:
 * for each query head j of KV head h, o_j = softmax(q_j K^T * scale) V with K,V
 * the rows 0..n_sel[s]-1 of k_buf/v_buf followed by the n_local live rows of
 * the local ring (slots (local_start + i) % window).  float32 arithmetic.
 *
 * q          [n_groups][n_kv_heads*group_size][d] dtype.
 * k_buf, v_buf [n_slices][buf_rows][d] dtype; n_sel [n_slices] int32 (<= buf_rows).
 * k_local, v_local [n_slices][window][d] dtype; 0 <= n_local <= window.
 * out        out [n_groups][n_kv_heads*group_size][d] in out_dtype.
 * lse_out    out [n_groups][n_kv_heads*group_size] float32 or NULL: natural log of
 *            each head's softmax denominator (max included); -inf and o = 0
 *            when a slice has no row.
 * workspace  louiskv_sparse_decode_attn_workspace_size() bytes for split-KV
 *            partials; the size is 0 (and workspace may be NULL) when there are
 *            enough slices for one block per slice.
 */
int louiskv_sparse_decode_attn(const void* q, int32_t dtype, int64_t n_slices,
                               int32_t n_kv_heads, int32_t group_size, int32_t d,
                               float scale, const void* k_buf, const void* v_buf,
                               const int32_t* n_sel, int32_t buf_rows,
                               const void* k_local, const void* v_local,
                               int32_t window, int32_t local_start, int32_t n_local,
                               void* out, int32_t out_dtype, float* lse_out,
                               void* workspace, size_t workspace_bytes, void* stream);

size_t louiskv_sparse_decode_attn_rows_workspace_size(int64_t n_slices, int32_t group_size,
                                                      int32_t d, int32_t budget,
                                                      int32_t window);

/*
 * louiskv_sparse_decode_attn over rows read straight from the pool: the
 * attended rows are the pool rows sel_rows[s][0..n_sel[s]-1] (as written by
 * louiskv_retrieve_rows) followed by the live rows of the local ring.  Same
 * arithmetic, layouts and outputs as louiskv_sparse_decode_attn.
 *
 * k_pool, v_pool  [n_slices][pool_rows][d] dtype, device memory.
 * sel_rows   [n_slices][budget] int32; entries are clamped into [0, pool_rows).
 * n_sel      [n_slices] int32 (<= budget).
 */
int louiskv_sparse_decode_attn_rows(const void* q, int32_t dtype, int64_t n_slices,
                                    int32_t n_kv_heads, int32_t group_size, int32_t d,
                                    float scale, const void* k_pool, const void* v_pool,
                                    int64_t pool_rows, const int32_t* sel_rows,
                                    const int32_t* n_sel, int32_t budget,
                                    const void* k_local, const void* v_local,
                                    int32_t window, int32_t local_start, int32_t n_local,
                                    void* out, int32_t out_dtype, float* lse_out,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * One decode step of Algorithm 1 for n_groups (sequence, layer) groups, with
 * fixed output segments and the KV pool in device memory, in one launch for
 * bf16 and two for float32: the boundary test (Section 4.1 equation for r_t), the decode-stage
 * store_cache (Section 4.2: window append, oldest-segment eviction), the
 * group-consistent retrieval of the groups that fired (Appendix B scores,
 * Section 3.1 budget, Algorithm 1 Retrieve; KV_critical kept as the list of
 * selected pool rows) and the attention over [KV_critical : KV_local]
 * (Section 3.1), current token included.  Meant for few groups per call (one
 * layer of a model at a time): every kernel spreads a slice over many
 * blocks, and the blocks of a slice hand over through the workspace (the
 * last one to finish a phase completes it) instead of through extra
 * launches.  In the one-launch form each block of a slice scores a part of
 * the units and attends a chunk of the rows; when the group fires, blocks
 * wait (bounded) for the slice's last scoring block to publish the
 * selection.
 *
 * Results equal, bit for bit, louiskv_decode_prologue + louiskv_retrieve_rows
 * + louiskv_sparse_decode_attn_rows (the selected units, rows, scores, r,
 * decisions, reference queries, window, unit table and pool), except the
 * attention output and lse, which split each slice's rows differently
 * (float32 summation order; same tolerance as those calls).
 *
 * Arguments are those of the three calls: q, q_ref, tau, mode, r_out,
 * fire_out as louiskv_boundary_check (the first step is step == 0); k_new,
 * v_new, k_local, v_local, window, seg_len, reps, unit_start, unit_size,
 * units_cap, n_clusters, k_pool, v_pool, pool_rows, prompt_len as
 * louiskv_segment_output (device pools only); budget, sel_units,
 * n_sel_units, n_sel, sel_rows [n_slices][max(budget, 1)], scores_out
 * (nullable) as louiskv_retrieve_rows; out, out_dtype, lse_out (nullable) as
 * louiskv_sparse_decode_attn_rows.  n_slices = n_groups * n_kv_heads and the
 * group size n_q_heads / n_kv_heads is 1, 2, 4 or 8.  The units scored at
 * step t are the clusters and the segments evicted before step t.
 *
 * workspace  louiskv_decode_step_workspace_size() bytes.  It must be zero
 *            before its first use (for example allocated zeroed); every call
 *            leaves its arrival counters and flags at zero again, so it is
 *            reused without clearing.  Calls that share it must not overlap.
 *            Its first (4 * n_slices + 1) * 64 int32 words are those
 *            counters and flags; the last of them is a status word that a
 *            block sets to 1 if its wait for a selection ever gave up (after
 *            about a million polls, which a correct launch never reaches;
 *            the environment variable LOUISKV_STEP_SPIN_LIMIT lowers that
 *            bound, for tests of this path), and that the library never
 *            clears.  The outputs of a step that set it are undefined and
 *            the workspace must be zeroed before its next use.
 */
size_t louiskv_decode_step_workspace_size(int64_t n_slices, int32_t dtype, int32_t group_size,
                                          int32_t units_cap, int32_t budget, int32_t window);

int louiskv_decode_step(const void* q, void* q_ref, int32_t dtype, int64_t n_groups,
                        int32_t n_q_heads, int32_t n_kv_heads, int32_t d, double tau,
                        int32_t mode, int32_t step, double* r_out, uint8_t* fire_out,
                        const void* k_new, const void* v_new, void* k_local, void* v_local,
                        int32_t window, int32_t seg_len, float* reps, int32_t* unit_start,
                        int32_t* unit_size, int32_t units_cap, int32_t n_clusters,
                        void* k_pool, void* v_pool, int64_t pool_rows, int32_t prompt_len,
                        int32_t budget, int32_t* sel_units, int32_t* n_sel_units,
                        int32_t* n_sel, int32_t* sel_rows, double* scores_out, void* out,
                        int32_t out_dtype, float* lse_out, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * louiskv_decode_step with KV_critical kept as an LRU cache of pool rows in
 * device memory (louiskv_retrieve_cached), for a pool in device or pinned host
 * memory (Algorithm 1 offloads the KV cache; Appendix A names the transfer
 * as the bottleneck): the boundary test, store and selection launch as in
 * louiskv_decode_step (the store writes the pool through pool_on_host's
 * device mapping), then the transfer plan of the fired slices and the copy
 * of the rows the cache lacks, then the attention over the cached rows
 * through slot_list.  Four launches.
 *
 * Results equal louiskv_decode_prologue + louiskv_retrieve_cached +
 * louiskv_sparse_decode_attn_rows over (k_buf, v_buf, slot_list) bit for
 * bit (selection, scores, r, decisions, reference queries, window, unit
 * table, pool, buffer rows, slot steps, slot list, fetch counts and cached
 * rows), except the attention output and lse (float32 summation order).
 *
 * Arguments as louiskv_decode_step, plus: pool_on_host as
 * louiskv_retrieve_cached (k_pool, v_pool in pinned host memory); budget >= 1;
 * cache_rows, k_buf, v_buf, buf_row, slot_step, slot_list, n_fetched
 * (nullable) as louiskv_retrieve_cached (budget <= cache_rows <= 65536,
 * pool_rows <= 524288, step <= 2^24 - 2).  sel_rows [n_slices][budget]
 * receives the selected pool rows (the plan's input).
 *
 * workspace  louiskv_decode_step_cached_workspace_size() bytes, zero before
 *            its first use, as louiskv_decode_step's.
 */
size_t louiskv_decode_step_cached_workspace_size(int64_t n_slices, int32_t dtype, int32_t group_size,
                                                 int32_t units_cap, int32_t budget, int32_t window);

int louiskv_decode_step_cached(const void* q, void* q_ref, int32_t dtype, int64_t n_groups,
                               int32_t n_q_heads, int32_t n_kv_heads, int32_t d, double tau,
                               int32_t mode, int32_t step, double* r_out, uint8_t* fire_out,
                               const void* k_new, const void* v_new, void* k_local, void* v_local,
                               int32_t window, int32_t seg_len, float* reps, int32_t* unit_start,
                               int32_t* unit_size, int32_t units_cap, int32_t n_clusters,
                               void* k_pool, void* v_pool, int64_t pool_rows, int32_t pool_on_host,
                               int32_t prompt_len, int32_t budget, int32_t cache_rows, void* k_buf,
                               void* v_buf, int32_t* buf_row, int32_t* slot_step, int32_t* slot_list,
                               int32_t* n_fetched, int32_t* sel_units, int32_t* n_sel_units,
                               int32_t* n_sel, int32_t* sel_rows, double* scores_out, void* out,
                               int32_t out_dtype, float* lse_out, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * louiskv_sparse_decode_attn_rows for callers that cannot allocate: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Arguments, arithmetic and outputs are those of
 * louiskv_sparse_decode_attn_rows (bit for bit), without the workspace: the
 * split-KV partials go to a static device array of
 * LOUISKV_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds
 * until the process ends.  The call allocates nothing; its first call on a
 * device looks up that device's copy of the array (hipGetSymbolAddress).
 *
 * Size limit  The launch's partials, louiskv_sparse_decode_attn_rows_workspace_size()
 *             of the same arguments, must fit LOUISKV_NOALLOC_SCRATCH_BYTES;
 *             larger launches return LOUISKV_ERR_WORKSPACE before anything is
 *             launched.  (A launch that fills the chip with one block per
 *             slice needs no partials at all.)
 * Sharing     Every call on one GPU uses the same array, which keeps the last
 *             call's contents (the kernels write every partial they read, so
 *             nothing needs clearing).  Calls that overlap on one GPU (two
 *             streams, two threads, two captured graphs replayed together)
 *             race on it: serialise them.
 */
#define LOUISKV_NOALLOC_SCRATCH_BYTES (8u << 20)

int louiskv_sparse_decode_attn_rows_noalloc(const void* q, int32_t dtype, int64_t n_slices,
                                            int32_t n_kv_heads, int32_t group_size, int32_t d,
                                            float scale, const void* k_pool, const void* v_pool,
                                            int64_t pool_rows, const int32_t* sel_rows,
                                            const int32_t* n_sel, int32_t budget,
                                            const void* k_local, const void* v_local,
                                            int32_t window, int32_t local_start, int32_t n_local,
                                            void* out, int32_t out_dtype, float* lse_out,
                                            void* stream);

/*
 * louiskv_boundary_check and louiskv_segment_output (fixed segments) of one
 * decode step in a single launch, for callers that run them back to back:
 * the boundary blocks and the store blocks are independent, because the store
 * writes only the unit it creates (index n_clusters + evicted segment) and
 * pool rows past every existing unit, which the step's retrieval does not
 * read; so the retrieval may follow this call directly.  Arguments as the two
 * calls (q .. fire_out as louiskv_boundary_check, k_new .. pool_on_host as
 * louiskv_segment_output); outputs are theirs, bit for bit.
 */
int louiskv_decode_prologue(const void* q, void* q_ref, int32_t dtype, int64_t n_groups,
                            int32_t n_q_heads, int32_t d, double tau, int32_t mode,
                            int32_t first_step, double* r_out, uint8_t* fire_out,
                            const void* k_new, const void* v_new, int64_t n_slices,
                            void* k_local, void* v_local, int32_t window, int32_t step,
                            int32_t seg_len, float* reps, int32_t* unit_start,
                            int32_t* unit_size, int32_t units_cap, int32_t n_clusters,
                            void* k_pool, void* v_pool, int64_t pool_rows, int32_t prompt_len,
                            int32_t pool_on_host, void* stream);

/* ------------------------------------------------------------------------ */
/* Decode stage with boundary-delimited segments                             */
/* ------------------------------------------------------------------------ */

/*
 * Section 4.2 (decode stage) partitions the generated KV cache into temporal
 * segments at the semantic boundaries of Section 4.1 (Algorithm 1's
 * is_new_segment); these calls implement that variant of store_cache,
 * Retrieve and attention.  A token starts a new segment when its group fired
 * this step, when no segment is open, or when the open segment already holds
 * seg_max tokens (the cap keeps a closed segment in every full window;
 * 1 <= seg_max < window).  Before a token is stored, if the window already
 * holds `window` tokens, its oldest segment leaves: it becomes the next unit
 * (index vector = mean key, float64 sum with one rounding to float32) and its
 * rows go to the pool.  Segment boundaries are per (sequence, layer) group,
 * so every slice of a group has the same segments.
 *
 * seg_state  [n_slices][louiskv_segment_state_ints(window)] int32, owned by
 *            the caller and private to the library: the window bounds, the
 *            unit count and the open segments of each slice.  Set it up with
 *            louiskv_segment_state_init after the prefill, before step 0.
 *            Entry 0 of a slice is its unit count (clusters plus segments
 *            evicted so far), entry 4 is 1 if a segment could not become a
 *            unit because units_cap or pool_rows was exhausted (its tokens
 *            are then no longer attended).
 */
size_t louiskv_segment_state_ints(int32_t window);

/*
 * The segment state before the first decode step: n_clusters units (the
 * clusters of the prefill), an empty window.  Enqueued on `stream`.
 */
int louiskv_segment_state_init(int32_t* seg_state, int64_t n_slices, int32_t window,
                               int32_t n_clusters, void* stream);

/*
 * Algorithm 1 store_cache(decode) with boundary-delimited segments (see
 * above), for every slice at decode step `step` (0-based; steps must be
 * issued in order, starting from 0).
 * fire       [n_groups] uint8, this step's boundary decisions
 *            (louiskv_boundary_check), n_groups = n_slices / n_kv_heads; NULL
 *            means no group fired (step 0 always opens a segment).
 * A unit created here has unit_start = prompt_len + (generation index of its
 * first token) and unit_size = its token count; the pool needs
 * pool_rows >= prompt_len + step + 1.  Other arguments as
 * louiskv_segment_output.
 */
int louiskv_segment_output_boundary(const void* k_new, const void* v_new, int32_t dtype,
                                    int64_t n_slices, int32_t n_kv_heads, int32_t d,
                                    void* k_local, void* v_local, int32_t window,
                                    int32_t step, int32_t seg_max, const uint8_t* fire,
                                    int32_t* seg_state, float* reps, int32_t* unit_start,
                                    int32_t* unit_size, int32_t units_cap, int32_t n_clusters,
                                    void* k_pool, void* v_pool, int64_t pool_rows,
                                    int32_t prompt_len, int32_t pool_on_host, void* stream);

/*
 * louiskv_retrieve (Appendix B scores, Section 3.1 budget, Algorithm 1
 * Retrieve) where each slice scores its own units 0 .. n_units[s]-1, the
 * count kept in seg_state; max_units bounds those counts for every slice
 * (1 <= max_units <= min(units_cap, 8192)) and sizes the sort.  Workspace as
 * louiskv_retrieve_workspace_size().
 */
int louiskv_retrieve_seg(const void* q, int32_t dtype, int64_t n_slices,
                         int32_t n_kv_heads, int32_t group_size, int32_t d, double scale,
                         const float* reps, const int32_t* unit_start,
                         const int32_t* unit_size, int32_t units_cap, int32_t max_units,
                         const int32_t* seg_state, int32_t window,
                         const void* k_pool, const void* v_pool, int64_t pool_rows,
                         int32_t pool_on_host, int32_t budget, const uint8_t* fire,
                         int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                         void* k_buf, void* v_buf, double* scores_out,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * louiskv_retrieve_rows with per-slice unit counts from seg_state (as
 * louiskv_retrieve_seg).  Workspace as louiskv_retrieve_rows_workspace_size().
 */
int louiskv_retrieve_rows_seg(const void* q, int32_t dtype, int64_t n_slices,
                              int32_t n_kv_heads, int32_t group_size, int32_t d, double scale,
                              const float* reps, const int32_t* unit_start,
                              const int32_t* unit_size, int32_t units_cap, int32_t max_units,
                              const int32_t* seg_state, int32_t window, int32_t budget,
                              const uint8_t* fire, int32_t* sel_units, int32_t* n_sel_units,
                              int32_t* n_sel, int32_t* sel_rows, double* scores_out,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * louiskv_sparse_decode_attn (Section 3.1 over [KV_critical : KV_local]) where
 * each slice's live window comes from seg_state: the tokens from its first
 * live token up to n_tokens - 1, with n_tokens the number of generated
 * tokens stored so far (step + 1 after this step's store).  Workspace as
 * louiskv_sparse_decode_attn_workspace_size().
 */
int louiskv_sparse_decode_attn_seg(const void* q, int32_t dtype, int64_t n_slices,
                                   int32_t n_kv_heads, int32_t group_size, int32_t d,
                                   float scale, const void* k_buf, const void* v_buf,
                                   const int32_t* n_sel, int32_t buf_rows,
                                   const void* k_local, const void* v_local, int32_t window,
                                   const int32_t* seg_state, int32_t n_tokens,
                                   void* out, int32_t out_dtype, float* lse_out,
                                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * louiskv_sparse_decode_attn_rows with per-slice windows from seg_state (as
 * louiskv_sparse_decode_attn_seg).  Workspace as
 * louiskv_sparse_decode_attn_rows_workspace_size().
 */
int louiskv_sparse_decode_attn_rows_seg(const void* q, int32_t dtype, int64_t n_slices,
                                        int32_t n_kv_heads, int32_t group_size, int32_t d,
                                        float scale, const void* k_pool, const void* v_pool,
                                        int64_t pool_rows, const int32_t* sel_rows,
                                        const int32_t* n_sel, int32_t budget,
                                        const void* k_local, const void* v_local, int32_t window,
                                        const int32_t* seg_state, int32_t n_tokens,
                                        void* out, int32_t out_dtype, float* lse_out,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Retrieval with delta transfers (host-resident pools)                      */
/* ------------------------------------------------------------------------ */

size_t louiskv_retrieve_delta_workspace_size(int64_t n_slices, int32_t units_cap,
                                             int32_t budget);

/*
 * Algorithm 1 Retrieve (scores of Appendix B, Section 3.1 budget) with
 * KV_critical kept as a cache of pool rows, so that a retrieval moves only
 * the rows the previous selection of the slice did not already hold (the
 * transfer that Appendix A names as the remaining bottleneck).  For every
 * fired slice: the same scores, ranking and prefix-stop selection as
 * louiskv_retrieve; buffer slots whose row is selected again keep it, the
 * others are freed; the newly selected rows (in rank order) go to the free
 * slots (in slot order), copied from the pool; slot_list then lists the
 * slots holding the selection.  Attend with louiskv_sparse_decode_attn_rows
 * (or _rows_seg) over k_buf/v_buf as the pool, budget rows, slot_list as the
 * row list.  Slices whose group did not fire are untouched.
 * buf_row    in/out [n_slices][budget] int32: the pool row held by each
 *            buffer slot, -1 when free; all -1 before the first retrieval.
 * slot_list  out [n_slices][budget] int32, entries 0..n_sel-1 written.
 * n_fetched  out [n_slices] int32 or NULL: rows copied this call (0 for
 *            slices that did not fire).
 * seg_state, window  NULL/ignored for fixed segments (n_units is then the
 *            unit count of every slice); with boundary-delimited segments the
 *            per-slice counts come from seg_state and n_units bounds them.
 * k_buf, v_buf  [n_slices][budget][d] dtype.  Requires budget >= 1 and
 *            pool_rows <= 524288.  Other arguments as louiskv_retrieve.
 */
int louiskv_retrieve_delta(const void* q, int32_t dtype, int64_t n_slices,
                           int32_t n_kv_heads, int32_t group_size, int32_t d, double scale,
                           const float* reps, const int32_t* unit_start,
                           const int32_t* unit_size, int32_t units_cap, int32_t n_units,
                           const int32_t* seg_state, int32_t window,
                           const void* k_pool, const void* v_pool, int64_t pool_rows,
                           int32_t pool_on_host, int32_t budget, const uint8_t* fire,
                           int32_t* sel_units, int32_t* n_sel_units, int32_t* n_sel,
                           void* k_buf, void* v_buf, int32_t* buf_row, int32_t* slot_list,
                           int32_t* n_fetched, double* scores_out,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * louiskv_retrieve_delta with a larger buffer kept as a least-recently-used
 * cache of pool rows: cache_rows >= budget slots per slice, so that rows
 * selected at earlier boundaries and selected again stay in HBM (Appendix A
 * names the transfer as the remaining bottleneck; rows tend to return because
 * adjacent selections overlap, Section 4.1 Observation 1).  For every fired
 * slice at decode step `step`: the same scores, ranking and prefix-stop
 * selection; a slot whose row is selected again keeps it; the k newly
 * selected rows (rank order) go to the k slots, among those not selected at
 * this step, with the smallest (slot_step, slot index), i.e. empty slots
 * first, then the rows selected longest ago, paired in slot order, and are
 * copied from the pool; slot_list lists the n_sel slots holding the
 * selection, in slot order.  Attend with louiskv_sparse_decode_attn_rows over
 * k_buf/v_buf as the pool (cache_rows rows) and slot_list as the row list.
 * buf_row    in/out [n_slices][cache_rows] int32: pool row of each slot, -1
 *            when empty; all -1 before the first retrieval.
 * slot_step  in/out [n_slices][cache_rows] int32: decode step at which the
 *            slot's row was last selected, -1 when empty; reset together
 *            with buf_row.  Steps must grow from call to call (0 <= step <
 *            2^24 - 1); a stale state (not reset) can leave rows without a
 *            slot, never write outside the buffers.
 * k_buf, v_buf  [n_slices][cache_rows][d] dtype.  slot_list [n_slices][budget].
 * budget <= cache_rows <= 65536 (LOUISKV_ERR_UNSUPPORTED above: the plan
 * keeps every slot's step in registers).
 * Workspace louiskv_retrieve_delta_workspace_size().  Other arguments as
 * louiskv_retrieve_delta.
 */
int louiskv_retrieve_cached(const void* q, int32_t dtype, int64_t n_slices,
                            int32_t n_kv_heads, int32_t group_size, int32_t d, double scale,
                            const float* reps, const int32_t* unit_start,
                            const int32_t* unit_size, int32_t units_cap, int32_t n_units,
                            const int32_t* seg_state, int32_t window,
                            const void* k_pool, const void* v_pool, int64_t pool_rows,
                            int32_t pool_on_host, int32_t budget, int32_t cache_rows,
                            int32_t step, const uint8_t* fire, int32_t* sel_units,
                            int32_t* n_sel_units, int32_t* n_sel, void* k_buf, void* v_buf,
                            int32_t* buf_row, int32_t* slot_step, int32_t* slot_list,
                            int32_t* n_fetched, double* scores_out,
                            void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Ablation baselines                                                        */
/* ------------------------------------------------------------------------ */

/*
 * Fixed-stride trigger (the retrieval ablation's baseline, Appendix D.3): in
 * place of louiskv_boundary_check, fire_out[g] = 1 for every group on the
 * steps where step % stride == 0 (step is the 0-based decode step, so the
 * first step fires), 0 otherwise.  fire_out [n_groups] uint8.
 * Errors: NULL fire_out, n_groups < 1, step < 0 or stride < 1.
 */
int louiskv_fire_every(uint8_t* fire_out, int64_t n_groups, int32_t step,
                       int32_t stride, void* stream);

/*
 * Page-level index for the prompt (the management ablation's coarse-grained
 * baseline, Appendix D.3), in place of louiskv_cluster_prefill: the prompt
 * of each slice is cut into pages of page_len tokens (the last page holds
 * the remainder), page p is unit p with index vector the mean of its keys
 * (float64 sum in row order, one rounding to float32), and the pool holds
 * the prompt rows in token order.
 *
 * keys, values [n_slices][n_tokens][d] dtype (values may be NULL when v_pool is).
 * reps        out [n_slices][units_cap][d] float32, rows 0..n_pages-1.
 * unit_start, unit_size  out [n_slices][units_cap] int32: p * page_len and
 *             min(page_len, n_tokens - p * page_len).
 * k_pool, v_pool  out [n_slices][pool_rows][d] dtype or NULL (rows
 *             0..n_tokens-1 written); pool_on_host as for louiskv_cluster_prefill.
 * Requires n_pages = ceil(n_tokens / page_len) <= units_cap and
 * pool_rows >= n_tokens when a pool is given.
 */
int louiskv_page_prefill(const void* keys, const void* values, int32_t dtype,
                         int64_t n_slices, int32_t n_tokens, int32_t d, int32_t page_len,
                         float* reps, int32_t units_cap, int32_t* unit_start,
                         int32_t* unit_size, void* k_pool, void* v_pool,
                         int64_t pool_rows, int32_t pool_on_host, void* stream);

/*
 * Per-head selection (the baseline that the group-consistent selection of
 * Appendix B replaces): every query head ranks its KV head's units by its own
 * softmax (the group score with a group of one) and takes its own budget
 * prefix, so the g heads of a KV head attend to different rows.  Arguments
 * as louiskv_retrieve_rows, but every per-list output has one list per query
 * head, list index s * group_size + j for query head j of slice s:
 * sel_units [n_slices * group_size][units_cap], n_sel_units and n_sel
 * [n_slices * group_size], sel_rows [n_slices * group_size][budget],
 * scores_out [n_slices * group_size][units_cap] or NULL.  Workspace:
 * louiskv_retrieve_rows_workspace_size(n_slices * group_size, units_cap).
 */
int louiskv_retrieve_rows_per_head(const void* q, int32_t dtype, int64_t n_slices,
                                   int32_t n_kv_heads, int32_t group_size, int32_t d,
                                   double scale, const float* reps,
                                   const int32_t* unit_start, const int32_t* unit_size,
                                   int32_t units_cap, int32_t n_units, int32_t budget,
                                   const uint8_t* fire, int32_t* sel_units,
                                   int32_t* n_sel_units, int32_t* n_sel, int32_t* sel_rows,
                                   double* scores_out, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * Attention for per-head selections: query head j of slice s attends to the
 * pool rows of list s * group_size + j (sel_rows, n_sel as written by
 * louiskv_retrieve_rows_per_head) followed by the live rows of slice s's
 * local window.  Other arguments, layouts and outputs as
 * louiskv_sparse_decode_attn_rows.  Workspace:
 * louiskv_sparse_decode_attn_rows_workspace_size(n_slices * group_size, 1,
 * d, budget, window).
 */
int louiskv_sparse_decode_attn_rows_per_head(const void* q, int32_t dtype, int64_t n_slices,
                                             int32_t n_kv_heads, int32_t group_size, int32_t d,
                                             float scale, const void* k_pool, const void* v_pool,
                                             int64_t pool_rows, const int32_t* sel_rows,
                                             const int32_t* n_sel, int32_t budget,
                                             const void* k_local, const void* v_local,
                                             int32_t window, int32_t local_start, int32_t n_local,
                                             void* out, int32_t out_dtype, float* lse_out,
                                             void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LOUISKV_H */
