/*
 * qcf.h -- C ABI of libqcf: one transformer layer of the QCFuse cache-fusion
 * step (arXiv 2606.05875) as hand-written HIP kernels for gfx950 (MI355X).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every tensor argument is a DEVICE pointer owned by the caller.  The
 *    library allocates nothing, keeps no pointer after the call returns and
 *    launches its kernels on the caller's stream in stream order (no implicit
 *    synchronisation).  Buffers must stay alive until the stream has passed
 *    the work.  Calls are reentrant; two calls that write the same buffer on
 *    different streams race.
 *  - Tensors are token-major: a K/V cache row holds n_kv_heads * head_dim
 *    elements (head-major inside the row); consecutive rows are `row_stride`
 *    elements apart (row_stride >= n_kv_heads * head_dim).  Query and output
 *    tensors are dense ([rows, n_q_heads, head_dim]).  Base pointers are 16-byte
 *    aligned; row strides are multiples of 16 bytes.  The attention and score
 *    kernels read one head's slice of every row; with a row of an even number
 *    of head slices those slices fall on a fraction of the L2 channels, so
 *    caches they read are best laid out with qcf_recommended_row_stride.
 *  - Index and position arrays are int32 device arrays; sizes fit int32.
 *  - dtype is QCF_F32 or QCF_BF16 (storage type of every floating tensor of the
 *    call, except score vectors, which are always float32); arithmetic is
 *    float32 (bf16 products on the matrix cores accumulate in float32); rotary
 *    angles are formed in float64.
 *  - head_dim is 64 or 128; n_q_heads is a multiple of n_kv_heads and the
 *    group size n_q_heads / n_kv_heads is a power of two no larger than 32
 *    (grouped-query attention: query head h reads KV head h / group).
 *  - Host-visible arguments are validated before anything is launched; a bad
 *    argument returns an error code and launches nothing.  The CONTENTS of
 *    device index arrays are preconditions: the kernels skip any index that
 *    falls outside the tensor bounds given in the call instead of touching
 *    memory out of bounds, but such input gives unspecified results.  A
 *    launch failure returns QCF_ERR_HIP.  Asynchronous device faults surface
 *    at the caller's next synchronisation.
 *  - Rotary embedding: rotate-half pairs (j, j + head_dim/2) turn by angle
 *    p * theta^(-2j/head_dim), no frequency scaling.
 */
#ifndef QCF_H_
#define QCF_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QCF_VERSION 102

typedef enum {
  QCF_OK = 0,
  QCF_ERR_INVALID_ARG = 1, /* null pointer, bad size, misaligned pointer or stride */
  QCF_ERR_UNSUPPORTED = 2, /* valid but not implemented (head_dim, group size, dtype) */
  QCF_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the _workspace_size query */
  QCF_ERR_HIP = 4          /* a HIP launch reported an error */
} qcf_status;

typedef enum { QCF_F32 = 0, QCF_BF16 = 1 } qcf_dtype;

/* Library version (QCF_VERSION) and a static text for a status code. */
int qcf_version(void);
const char* qcf_status_string(qcf_status status);

/*
 * qcf_recommended_row_stride -- row stride (in elements) for a K/V cache that
 * the attention and score kernels will read: n_kv_heads * head_dim when
 * n_kv_heads is odd, else (n_kv_heads + 1) * head_dim, i.e. one unused head
 * slice of padding per row.  A row of an odd number of head slices puts the
 * slice of one head in consecutive rows on different L2 channels (a row of
 * 8 slices of 256 bytes reaches only a few of them).  Host function; returns
 * 0 for n_kv_heads <= 0 or a head_dim other than 64 and 128.
 */
int64_t qcf_recommended_row_stride(int n_kv_heads, int head_dim);

/*
 * qcf_rerope -- position remapping Pi_i and stitching of the reused chunk
 * caches into the request cache (Section 2.1.2, eq. pic_online).  A stored
 * chunk key is rotated at its chunk-local position; rotating it once more by
 * the chunk's offset o_i moves it to its request position o_i + r.  The
 * chunk's values are copied in the same token order.  For segment s and row
 * r < seg_len[s], with src = (src_start ? src_start[s] : seg_start[s]) + r and
 * dst = seg_start[s] + r:
 *     k_out[dst] = rope(k_in[src], seg_delta[s])
 *     v_out[dst] = v_in[src]                       (when v_out != NULL)
 *   k_out, v_out  [n_out_rows, out_row_stride]; k_in, v_in [n_in_rows, in_row_stride]
 *                 k_out may equal k_in (in place, equal strides) when src == dst;
 *                 v_in must be non-NULL iff v_out is, and the V copy is skipped
 *                 when v_out == v_in.  Rows outside every segment are not touched.
 *   seg_start     [n_seg] first destination row of each segment (a chunk)
 *   seg_len       [n_seg] rows in each segment (<= max_seg_len)
 *   seg_delta     [n_seg] rotation offset of each segment in positions
 *   src_start     [n_seg] first source row of each segment, or NULL
 *   rope_theta    rotary base
 * Errors: null pointers, n_seg > 65535, head_dim unsupported, misalignment.
 */
qcf_status qcf_rerope(void* k_out, const void* k_in, void* v_out, const void* v_in,
                      qcf_dtype dtype, int64_t n_out_rows, int64_t n_in_rows, int n_kv_heads,
                      int head_dim, int64_t out_row_stride, int64_t in_row_stride, int n_seg,
                      const int32_t* seg_start,
                      const int32_t* seg_len, const int32_t* seg_delta, const int32_t* src_start,
                      int max_seg_len, double rope_theta, hipStream_t stream);

/*
 * qcf_gather_rows -- row copy dst[i] = src[idx[i]] (the anchor cache
 * KV^A = KV^PIC[A], Section 3.3.2, eq. anchor_cache; also the compact
 * fresh-row gather).
 *   dst  [n_rows rows, dst_stride_bytes]; src [n_src_rows rows, src_stride_bytes]
 *   idx  [n_rows] source rows; rows with idx outside [0, n_src_rows) are skipped
 *   row_bytes  bytes copied per row (multiple of 16, <= both strides)
 */
qcf_status qcf_gather_rows(void* dst, const void* src, const int32_t* idx, int64_t n_rows,
                           int64_t n_src_rows, int64_t row_bytes, int64_t src_stride_bytes,
                           int64_t dst_stride_bytes, hipStream_t stream);

/*
 * qcf_scatter_kv -- fused-cache update of eq. fuse_cache: recomputed rows
 * replace their PIC entries (Section 2.1.3).  For each r < n_rows with
 * s = src_idx ? src_idx[r] : r and p = row_pos[r]:
 *     k_cache[row_idx[r]] = rope(k_new[s], p)
 *     v_cache[row_idx[r]] = v_new[s]
 *     q_out[r]            = rope(q_new[s], p)      (when q_out != NULL)
 *   k_cache, v_cache  [n_cache_rows, cache_row_stride]
 *   k_new, v_new      [n_src_rows, n_kv_heads * head_dim] dense
 *   q_new             [n_src_rows, n_q_heads * head_dim] dense (may be NULL iff q_out is NULL)
 *   q_out             [n_rows, n_q_heads * head_dim] dense, may alias q_new only when
 *                     src_idx is NULL (in-place rotation)
 * Duplicate row_idx values give unspecified results.
 */
qcf_status qcf_scatter_kv(void* k_cache, void* v_cache, int64_t n_cache_rows,
                          int64_t cache_row_stride, const void* k_new, const void* v_new,
                          const void* q_new, void* q_out, int64_t n_src_rows,
                          const int32_t* src_idx, qcf_dtype dtype, int64_t n_rows,
                          const int32_t* row_idx, const int32_t* row_pos, int n_q_heads,
                          int n_kv_heads, int head_dim, double rope_theta, hipStream_t stream);

/*
 * qcf_assemble -- everything the query probe needs, in one launch (Section
 * 3.5, first half): the request cache from the stored chunk caches (eq.
 * pic_online), the user-query rows rotated at their positions, and the probe
 * buffer [KV^A ; K/V of the query] with KV^A = Pi(KV^PIC[A]) (eq.
 * anchor_cache).  Three independent parts, run side by side:
 *  (1) segments, exactly as qcf_rerope with values:
 *        k_cache[dst] = rope(k_pic[src], seg_delta[s]),  v_cache[dst] = v_pic[src]
 *  (2) query rows i < n_query, with s = query_src ? query_src[i] : i and
 *      p = query_pos[i]:
 *        k_cache[query_row[i]] = rope(k_new[s], p),  v_cache[query_row[i]] = v_new[s]
 *        q_u[i] = rope(q_new[s], p)
 *        and, when query_slot != NULL and j = query_slot[i] >= 0:
 *        probe_k[j] = rope(k_new[s], p),  probe_v[j] = v_new[s]
 *  (3) probe slots j < n_probe with probe_src[j] >= 0:
 *        probe_k[j] = rope(k_pic[probe_src[j]], probe_delta[j]),  probe_v[j] = v_pic[probe_src[j]]
 *      slots with probe_src[j] < 0 are left to the query rows.
 *   k_cache, v_cache [n_rows, row_stride]; k_pic, v_pic [n_pic_rows,
 *                    pic_row_stride] (read only; may not alias the outputs)
 *   probe_k, probe_v [n_probe, probe_row_stride]
 *   q_new [n_src_rows, n_q_heads * head_dim]; k_new, v_new [n_src_rows,
 *   n_kv_heads * head_dim]; q_u [n_query, n_q_heads * head_dim] (dense)
 *   max_seg_len >= every seg_len
 * The parts must write disjoint places: no query_row inside a segment's
 * destination rows, and each probe slot filled by (3) or by one query row.
 * Results of overlapping writes are unspecified.
 */
qcf_status qcf_assemble(void* k_cache, void* v_cache, int64_t n_rows, int64_t row_stride,
                        const void* k_pic, const void* v_pic, int64_t n_pic_rows,
                        int64_t pic_row_stride, int n_seg, const int32_t* seg_start,
                        const int32_t* seg_len, const int32_t* seg_delta,
                        const int32_t* src_start, int max_seg_len, const void* q_new,
                        const void* k_new, const void* v_new, int64_t n_src_rows,
                        int64_t n_query, const int32_t* query_row, const int32_t* query_pos,
                        const int32_t* query_src, const int32_t* query_slot, void* q_u,
                        void* probe_k, void* probe_v, int64_t n_probe, int64_t probe_row_stride,
                        const int32_t* probe_src, const int32_t* probe_delta,
                        qcf_dtype dtype, int n_q_heads, int n_kv_heads, int head_dim,
                        double rope_theta, hipStream_t stream);

/*
 * qcf_probe_scores -- per-token importance of one critical layer,
 * eq. single_layer_importance (Section 3.4.1); with accumulate != 0 the result
 * is added to `scores`, which sums it over the critical layers
 * (eq. critical_layer_importance).  For request b, context token t < ctx_len[b]:
 *   scores[cu_kv[b] + t] (+)= sum_{i, h} softmax_t'( q[cu_q[b]+i, h] . k[cu_kv[b]+t', h/group]
 *                                                  * softmax_scale )[t]
 * The softmax runs over the request's ctx_len[b] context keys.  Score slots
 * of other rows are not written.  The result is deterministic (fixed
 * reduction order).
 *   scores  float32 [n_kv_rows]
 *   q       [n_q_rows, n_q_heads, head_dim] rotated user-query states
 *   k       [n_kv_rows, k_row_stride] keys at their request positions
 *   cu_q    [batch+1], cu_kv [batch+1], ctx_len [batch] device arrays;
 *   max_q_len >= max_b(cu_q[b+1]-cu_q[b]), max_ctx_len >= max_b ctx_len[b]
 *   workspace  >= qcf_probe_scores_workspace_size(...) bytes, 256-byte aligned; it
 *              holds the per-split softmax statistics and per-(KV head, query tile)
 *              column sums between the kernels of the call and needs no
 *              initialisation.  A workspace sized for one shape serves every
 *              smaller one.  Calls that overlap in time need separate workspaces.
 */
size_t qcf_probe_scores_workspace_size(int batch, int max_q_len, int max_ctx_len,
                                       int n_q_heads, int n_kv_heads, int head_dim);
qcf_status qcf_probe_scores(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                            const void* k, int64_t n_kv_rows, int64_t k_row_stride,
                            qcf_dtype dtype, int batch, const int32_t* cu_q,
                            const int32_t* cu_kv, const int32_t* ctx_len, int max_q_len,
                            int max_ctx_len, int n_q_heads, int n_kv_heads, int head_dim,
                            float softmax_scale, void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/*
 * qcf_rope_table -- the rotations that move stored chunk keys to their request
 * offsets (Section 2.1.2, eq. pic_online) as a table:
 *   table[2 * (i * head_dim/2 + j) + {0, 1}] = cos, sin of pos[i] * theta^(-2j/head_dim)
 * formed in float64 and rounded to float32 -- the values every rotation of
 * this library uses for offset pos[i].  The table depends only on the
 * offsets, so one table serves every layer of a request.
 *   table  float32 [n, head_dim/2, 2] device output (16-byte aligned)
 *   pos    int32 [n] device offsets
 */
qcf_status qcf_rope_table(float* table, const int32_t* pos, int64_t n, int head_dim,
                          double rope_theta, hipStream_t stream);

/*
 * qcf_probe_scores_pic -- qcf_probe_scores over keys re-positioned on the fly
 * (eq. pic_online fused into eq. single_layer_importance): the keys are read
 * from the stored chunk caches and each is turned, in registers, by its row
 * of a qcf_rope_table table before it meets the queries:
 *   key of row t = rotate(k_pic[t], rope_table[key_rot[t]]), rounded to dtype,
 * which is bit for bit the key qcf_rerope / qcf_assemble store for a chunk
 * row whose offset is the table row's, so the scores equal those of
 * qcf_rerope followed by qcf_probe_scores on the re-positioned cache.  The
 * re-positioned keys are not written; the call depends only on the stored
 * caches and the rotated queries.
 *   k_pic    [n_kv_rows, k_row_stride] stored keys, rows laid out as the request
 *            cache (row cu_kv[b] + t holds context token t of request b)
 *   key_rot  int32 [n_kv_rows] table row of each key row (only context rows
 *            are read; values are clamped into [0, n_rot))
 *   rope_table, n_rot  a qcf_rope_table table of n_rot rows
 * Every other argument, the workspace and the result are as for
 * qcf_probe_scores (same workspace size).
 */
qcf_status qcf_probe_scores_pic(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                                const void* k_pic, int64_t n_kv_rows, int64_t k_row_stride,
                                const int32_t* key_rot, const float* rope_table, int64_t n_rot,
                                qcf_dtype dtype, int batch, const int32_t* cu_q,
                                const int32_t* cu_kv, const int32_t* ctx_len, int max_q_len,
                                int max_ctx_len, int n_q_heads, int n_kv_heads, int head_dim,
                                float softmax_scale, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * qcf_select_topk -- recomputation set of eq. critical_mask, taken per
 * segment (per chunk).  For segment s the k = seg_k[s] rows of
 * [seg_start[s], seg_start[s] + seg_len[s]) with the largest scores are
 * chosen; equal scores go to the lower row, and -0 equals +0.  The chosen
 * rows are written in ascending order to out_idx[out_start[s] .. + k); when
 * out_pos is not NULL, out_pos gets row - pos_base[s] (the position inside
 * the request).  Scores must be finite.  k > seg_len is clamped to seg_len.
 *   scores   float32 [n_scores]
 *   out_idx, out_pos  int32 [n_out]
 *   max_seg_len >= every seg_len (chooses the LDS staging path)
 */
qcf_status qcf_select_topk(int32_t* out_idx, int32_t* out_pos, int64_t n_out,
                           const float* scores, int64_t n_scores, int n_seg,
                           const int32_t* seg_start, const int32_t* seg_len,
                           const int32_t* seg_k, const int32_t* out_start,
                           const int32_t* pos_base, int max_seg_len, hipStream_t stream);

/*
 * qcf_probe_scores_select -- qcf_probe_scores followed by qcf_select_topk on
 * the scores it finishes (eq. single_layer_importance, or the last term of
 * eq. critical_layer_importance with accumulate != 0, then eq. critical_mask),
 * with the final summation of the scores done inside the selection when no
 * segment is longer than 1024 rows (chunks), so the two steps cost one launch
 * less; longer segments take the separate final pass.  The results are bit for bit those of the
 * two calls: `scores` holds the same values afterwards and the same rows are
 * chosen in the same order.
 *   scores, q, k, cu_q, cu_kv, ctx_len, max_q_len, max_ctx_len, heads,
 *   softmax_scale, workspace  as for qcf_probe_scores (same workspace size)
 *   out_idx, out_pos, n_out, n_seg, seg_start, seg_len, seg_k, out_start,
 *   max_seg_len  as for qcf_select_topk
 *   seg_req  int32 [n_seg]: the request b whose context holds segment s;
 *            out_pos gets row - cu_kv[seg_req[s]] (the position in the request)
 * A segment whose seg_req is outside [0, batch) is skipped.  A segment's rows
 * must lie in its request's context (rows cu_kv[b] ..
 * cu_kv[b] + ctx_len[b] - 1); other rows are ranked by their stored scores.
 * Errors as for the two calls; nothing is launched when any argument is
 * rejected.
 */
qcf_status qcf_probe_scores_select(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                                   const void* k, int64_t n_kv_rows, int64_t k_row_stride,
                                   qcf_dtype dtype, int batch, const int32_t* cu_q,
                                   const int32_t* cu_kv, const int32_t* ctx_len, int max_q_len,
                                   int max_ctx_len, int n_q_heads, int n_kv_heads, int head_dim,
                                   float softmax_scale, int32_t* out_idx, int32_t* out_pos,
                                   int64_t n_out, int n_seg, const int32_t* seg_start,
                                   const int32_t* seg_len, const int32_t* seg_k,
                                   const int32_t* out_start, const int32_t* seg_req,
                                   int max_seg_len, void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/*
 * qcf_probe_scores_select_noalloc -- qcf_probe_scores_select for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments and results, minus
 * the workspace: its scratch space is a fixed array of
 * QCF_NOALLOC_SCRATCH_BYTES in the library's device image, one per GPU, held
 * until the process ends.  The call allocates nothing (its first call on a
 * device looks the array's address up once).
 *   Shapes whose qcf_probe_scores_workspace_size exceeds
 *   QCF_NOALLOC_SCRATCH_BYTES are rejected with QCF_ERR_WORKSPACE before
 *   anything is launched.  The kernels read back only scratch words written
 *   earlier in the same call, so the array is never cleared.
 *   All calls on one GPU share its array: calls that may overlap on that GPU
 *   (several streams, several host threads) race and must be serialised by
 *   the caller, e.g. by issuing them on one stream.
 */
#define QCF_NOALLOC_SCRATCH_BYTES (48 << 20)
qcf_status qcf_probe_scores_select_noalloc(float* scores, int accumulate, const void* q,
                                           int64_t n_q_rows, const void* k, int64_t n_kv_rows,
                                           int64_t k_row_stride, qcf_dtype dtype, int batch,
                                           const int32_t* cu_q, const int32_t* cu_kv,
                                           const int32_t* ctx_len, int max_q_len, int max_ctx_len,
                                           int n_q_heads, int n_kv_heads, int head_dim,
                                           float softmax_scale, int32_t* out_idx, int32_t* out_pos,
                                           int64_t n_out, int n_seg, const int32_t* seg_start,
                                           const int32_t* seg_len, const int32_t* seg_k,
                                           const int32_t* out_start, const int32_t* seg_req,
                                           int max_seg_len, hipStream_t stream);

/*
 * qcf_sparse_prefill_attn -- causal grouped-query attention of the selected
 * rows over the fused cache (Section 2.1.3: a recomputed row at position p
 * reads every prefix key j <= p, itself included); with an explicit kv_pos it
 * is also the anchor-conditioned query probe over [anchor cache ; query]
 * (Section 3.3.2, eq. anchor_query_state).  For request b, row r in
 * [cu_rows[b], cu_rows[b+1]) and head h:
 *   out[r, h] = sum_j softmax_j( q[r, h] . k[cu_kv[b]+j, h/group] * softmax_scale ) v[cu_kv[b]+j, h/group]
 * over keys j < cu_kv[b+1]-cu_kv[b] with kpos(j) <= row_pos[r], where
 * kpos(j) = kv_pos[cu_kv[b]+j] if kv_pos != NULL, else j.  A row that sees no
 * key gets zeros (and lse = -inf).
 *   out  [n_rows, n_q_heads, head_dim]; lse float32 [n_rows, n_q_heads] or NULL
 *        (natural-log log-sum-exp of the scaled logits)
 *   q    [n_rows, n_q_heads, head_dim]; row_pos int32 [n_rows]
 *   k_cache, v_cache [n_kv_rows, kv_row_stride]
 *   cu_rows [batch+1], cu_kv [batch+1]; max_rows / max_kv bound the per-request counts
 *   workspace >= qcf_sparse_prefill_attn_workspace_size(...) bytes (may be 0), 256-byte
 *        aligned.  A bf16 call without kv_pos that has few row tiles shares the key
 *        steps of all its row tiles evenly over a fixed grid of blocks; the
 *        workspace then holds the work plan and the partial results of row tiles
 *        cut between two blocks, which a second kernel merges in a fixed order
 *        (deterministic).  A bf16 call without kv_pos over one request with at
 *        least four row tiles per compute unit hands the tiles out from work
 *        counters in the workspace, which the call resets itself (by a kernel on
 *        the same stream); each tile is still computed whole by one block, so the
 *        result does not depend on which block takes it.  Its contents need no
 *        initialisation; calls that overlap in time need separate workspaces.  The size query is monotone: the size
 *        for (batch, max_rows, max_kv) covers every call whose three values do
 *        not exceed them (other arguments equal).
 */
size_t qcf_sparse_prefill_attn_workspace_size(int batch, int max_rows, int max_kv,
                                              int n_q_heads, int n_kv_heads, int head_dim,
                                              qcf_dtype dtype);
qcf_status qcf_sparse_prefill_attn(void* out, float* lse, const void* q, const int32_t* row_pos,
                                   int64_t n_rows, const int32_t* cu_rows, const void* k_cache,
                                   const void* v_cache, int64_t n_kv_rows, int64_t kv_row_stride,
                                   const int32_t* cu_kv, const int32_t* kv_pos, qcf_dtype dtype,
                                   int batch, int max_rows, int max_kv, int n_q_heads,
                                   int n_kv_heads, int head_dim, float softmax_scale,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * qcf_sparse_prefill_attn_rope -- qcf_sparse_prefill_attn (bf16, recomputed
 * rows, no kv_pos) on un-rotated query rows: the kernel turns row r's query by
 * the rotation of its position row_pos[r] in registers (Section 2.1.3: the
 * recomputed rows' fresh queries are rotated at their request positions), so
 * no rotated copy of the queries is written or read.  The rotation is bit for
 * bit the one qcf_scatter_kv applies to q_new.
 *   q_raw       [n_q_raw, n_q_heads, head_dim] un-rotated queries
 *   q_src       int32 [n_rows]: row of q_raw for recomputed row r (values are
 *               clamped to [0, n_q_raw)), or NULL: row r of q_raw (n_q_raw >= n_rows)
 *   rope_table  float32 [n_table, head_dim/2, 2] from qcf_rope_table at positions
 *               0 .. n_table-1 (a constant of theta and head_dim: one table
 *               serves every layer and request); row_pos[r] must be < n_table
 *               (larger positions are clamped to the last row: a wrong
 *               rotation, never an out-of-range read)
 *   all other arguments as for qcf_sparse_prefill_attn (same workspace size).
 * QCF_ERR_UNSUPPORTED for float32; QCF_ERR_INVALID_ARG for a missing table.
 */
qcf_status qcf_sparse_prefill_attn_rope(void* out, float* lse, const void* q_raw,
                                        const int32_t* q_src, int64_t n_q_raw,
                                        const int32_t* row_pos, int64_t n_rows,
                                        const int32_t* cu_rows, const void* k_cache,
                                        const void* v_cache, int64_t n_kv_rows,
                                        int64_t kv_row_stride, const int32_t* cu_kv,
                                        const float* rope_table, int64_t n_table,
                                        qcf_dtype dtype, int batch, int max_rows, int max_kv,
                                        int n_q_heads, int n_kv_heads, int head_dim,
                                        float softmax_scale, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream);

/*
 * qcf_mfma_loop -- not a step of the method: a yardstick for the attention.
 * A grid of `blocks` four-wave blocks runs `iters` rounds of 16
 * v_mfma_f32_32x32x16_bf16 products per wave (four independent accumulators,
 * operand fragments taken from `operands` and rotated between products), the
 * attention's product instruction at its occupancy (two waves per SIMD when
 * blocks = 2 x compute units).  Each wave executes iters x 16 x 32768 FLOP.
 *   operands  bf16 [n_operands >= 16] device buffer (random values give the
 *             multipliers realistic activity; all-zero data runs cooler)
 *   sink      float32 [n_sink >= blocks * 256]: one sum of accumulators per thread
 *   clocks    uint64 [32]: blocks 0..7 each write (real-time counter at 100 MHz,
 *             shader-clock counter) at their start and end, so the clock the
 *             loop ran at is the ratio of the two differences
 *   blocks >= 8, iters >= 1.  Nothing is read back or synchronised.
 */
qcf_status qcf_mfma_loop(const void* operands, int64_t n_operands, float* sink, int64_t n_sink,
                         uint64_t* clocks, int blocks, int iters, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* QCF_H_ */
