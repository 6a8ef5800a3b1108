// C ABI of libqcf: host-side validation, then the kernel launchers.
// Every check runs before any HIP call, so a rejected call touches no device
// state (and works on a machine without a GPU).
#include <stdint.h>

#include "../../include/qcf.h"
#include "qcf_launch.h"

namespace {

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }
inline bool dtype_ok(qcf_dtype t) { return t == QCF_F32 || t == QCF_BF16; }
inline int64_t esize(qcf_dtype t) { return t == QCF_BF16 ? 2 : 4; }
// a device tensor pointer: non-null and 16-byte aligned (null allowed when empty)
inline bool tensor_ok(const void* p, bool empty) { return empty ? (p == nullptr || aligned16(p)) : (p && aligned16(p)); }
inline bool index_ok(const void* p, bool empty) {
  return empty || (p && (reinterpret_cast<uintptr_t>(p) & 3u) == 0);
}

qcf_status check_heads(int hq, int hkv, int d) {
  if (hkv <= 0 || hq <= 0) return QCF_ERR_INVALID_ARG;
  if (d != 64 && d != 128) return QCF_ERR_UNSUPPORTED;
  if (hq % hkv != 0) return QCF_ERR_INVALID_ARG;
  const int grp = hq / hkv;
  if ((grp & (grp - 1)) != 0 || grp > 32) return QCF_ERR_UNSUPPORTED;
  if (hq > 65535) return QCF_ERR_UNSUPPORTED;
  return QCF_OK;
}

inline qcf_status hip_status(hipError_t e) { return e == hipSuccess ? QCF_OK : QCF_ERR_HIP; }

// a K/V row stride: at least one row of heads, a whole number of 16-byte units
inline bool kv_stride_ok(int64_t stride, int hkv, int d, qcf_dtype t) {
  return stride >= (int64_t)hkv * d && (stride * esize(t)) % 16 == 0;
}

}  // namespace

extern "C" {

int qcf_version(void) { return QCF_VERSION; }

int64_t qcf_recommended_row_stride(int n_kv_heads, int head_dim) {
  if (n_kv_heads <= 0 || (head_dim != 64 && head_dim != 128)) return 0;
  return (int64_t)(n_kv_heads + (n_kv_heads % 2 == 0 ? 1 : 0)) * head_dim;
}

const char* qcf_status_string(qcf_status s) {
  switch (s) {
    case QCF_OK: return "ok";
    case QCF_ERR_INVALID_ARG: return "invalid argument";
    case QCF_ERR_UNSUPPORTED: return "unsupported configuration";
    case QCF_ERR_WORKSPACE: return "workspace missing or too small";
    case QCF_ERR_HIP: return "HIP launch error";
  }
  return "unknown status";
}

qcf_status qcf_rerope(void* k_out, const void* k_in, void* v_out, const void* v_in,
                      qcf_dtype dtype, int64_t n_out_rows, int64_t n_in_rows, int n_kv_heads,
                      int head_dim, int64_t out_row_stride, int64_t in_row_stride, int n_seg,
                      const int32_t* seg_start, const int32_t* seg_len, const int32_t* seg_delta,
                      const int32_t* src_start, int max_seg_len, double rope_theta,
                      hipStream_t stream) {
  if (!dtype_ok(dtype)) return QCF_ERR_UNSUPPORTED;
  if (n_out_rows < 0 || n_out_rows > INT32_MAX || n_in_rows < 0 || n_in_rows > INT32_MAX ||
      n_seg < 0 || max_seg_len < 0)
    return QCF_ERR_INVALID_ARG;
  if (n_kv_heads <= 0) return QCF_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return QCF_ERR_UNSUPPORTED;
  if (n_seg > 65535) return QCF_ERR_UNSUPPORTED;
  if (!kv_stride_ok(out_row_stride, n_kv_heads, head_dim, dtype) ||
      !kv_stride_ok(in_row_stride, n_kv_heads, head_dim, dtype))
    return QCF_ERR_INVALID_ARG;
  if (!(rope_theta > 0.0)) return QCF_ERR_INVALID_ARG;
  if ((v_out == nullptr) != (v_in == nullptr)) return QCF_ERR_INVALID_ARG;
  // in place needs the same row layout on both sides
  if ((k_out == k_in || (v_out && v_out == v_in)) && out_row_stride != in_row_stride)
    return QCF_ERR_INVALID_ARG;
  const bool empty = n_out_rows == 0 || n_in_rows == 0 || n_seg == 0 || max_seg_len == 0;
  if (!tensor_ok(k_out, empty) || !tensor_ok(k_in, empty) || !tensor_ok(v_out, true) ||
      !tensor_ok(v_in, true))
    return QCF_ERR_INVALID_ARG;
  if (!index_ok(seg_start, n_seg == 0) || !index_ok(seg_len, n_seg == 0) ||
      !index_ok(seg_delta, n_seg == 0) || (src_start && !index_ok(src_start, false)))
    return QCF_ERR_INVALID_ARG;
  if (empty) return QCF_OK;
  return hip_status(qcf::launch_rerope(k_out, k_in, v_out, v_in, dtype == QCF_BF16, n_out_rows,
                                       n_in_rows, n_kv_heads, head_dim, out_row_stride,
                                       in_row_stride, n_seg, seg_start, seg_len, seg_delta,
                                       src_start, max_seg_len, rope_theta, stream));
}

qcf_status qcf_gather_rows(void* dst, const void* src, const int32_t* idx, int64_t n_rows,
                           int64_t n_src_rows, int64_t row_bytes, int64_t src_stride_bytes,
                           int64_t dst_stride_bytes, hipStream_t stream) {
  if (n_rows < 0 || n_src_rows < 0 || row_bytes < 0 || n_rows > INT32_MAX) return QCF_ERR_INVALID_ARG;
  if (row_bytes % 16 != 0 || src_stride_bytes % 16 != 0 || dst_stride_bytes % 16 != 0)
    return QCF_ERR_INVALID_ARG;
  if (row_bytes > src_stride_bytes || row_bytes > dst_stride_bytes) return QCF_ERR_INVALID_ARG;
  const bool empty = n_rows == 0 || row_bytes == 0;
  if (!tensor_ok(dst, empty) || !tensor_ok(src, empty || n_src_rows == 0) || !index_ok(idx, empty))
    return QCF_ERR_INVALID_ARG;
  if (empty) return QCF_OK;
  return hip_status(qcf::launch_gather_rows(dst, src, idx, n_rows, n_src_rows, row_bytes,
                                            src_stride_bytes, dst_stride_bytes, stream));
}

qcf_status qcf_scatter_kv(void* k_cache, void* v_cache, int64_t n_cache_rows,
                          int64_t cache_row_stride, const void* k_new, const void* v_new,
                          const void* q_new, void* q_out, int64_t n_src_rows,
                          const int32_t* src_idx, qcf_dtype dtype, int64_t n_rows,
                          const int32_t* row_idx, const int32_t* row_pos, int n_q_heads,
                          int n_kv_heads, int head_dim, double rope_theta, hipStream_t stream) {
  if (!dtype_ok(dtype)) return QCF_ERR_UNSUPPORTED;
  qcf_status st = check_heads(n_q_heads, n_kv_heads, head_dim);
  if (st != QCF_OK) return st;
  if (n_rows < 0 || n_rows > INT32_MAX || n_cache_rows < 0 || n_src_rows < 0) return QCF_ERR_INVALID_ARG;
  if (cache_row_stride < (int64_t)n_kv_heads * head_dim || (cache_row_stride * esize(dtype)) % 16 != 0)
    return QCF_ERR_INVALID_ARG;
  if (!(rope_theta > 0.0)) return QCF_ERR_INVALID_ARG;
  if (q_out && !q_new) return QCF_ERR_INVALID_ARG;
  if (q_out && src_idx && q_out == q_new) return QCF_ERR_INVALID_ARG;
  const bool empty = n_rows == 0;
  if (!tensor_ok(k_cache, empty) || !tensor_ok(v_cache, empty) || !tensor_ok(k_new, empty) ||
      !tensor_ok(v_new, empty))
    return QCF_ERR_INVALID_ARG;
  if (q_out && (!aligned16(q_out) || !aligned16(q_new))) return QCF_ERR_INVALID_ARG;
  if (!index_ok(row_idx, empty) || !index_ok(row_pos, empty) || (src_idx && !index_ok(src_idx, false)))
    return QCF_ERR_INVALID_ARG;
  if (empty) return QCF_OK;
  return hip_status(qcf::launch_scatter_kv(k_cache, v_cache, n_cache_rows, cache_row_stride, k_new,
                                           v_new, q_new, q_out, n_src_rows, src_idx,
                                           dtype == QCF_BF16, n_rows, row_idx, row_pos, n_q_heads,
                                           n_kv_heads, head_dim, rope_theta, stream));
}

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
                        double rope_theta, hipStream_t stream) {
  if (!dtype_ok(dtype)) return QCF_ERR_UNSUPPORTED;
  qcf_status st = check_heads(n_q_heads, n_kv_heads, head_dim);
  if (st != QCF_OK) return st;
  if (n_rows < 0 || n_rows > INT32_MAX || n_pic_rows < 0 || n_pic_rows > INT32_MAX ||
      n_src_rows < 0 || n_src_rows > INT32_MAX || n_query < 0 || n_query > INT32_MAX ||
      n_probe < 0 || n_probe > INT32_MAX || n_seg < 0 || max_seg_len < 0)
    return QCF_ERR_INVALID_ARG;
  if (!kv_stride_ok(row_stride, n_kv_heads, head_dim, dtype) ||
      !kv_stride_ok(pic_row_stride, n_kv_heads, head_dim, dtype) ||
      !kv_stride_ok(probe_row_stride, n_kv_heads, head_dim, dtype))
    return QCF_ERR_INVALID_ARG;
  if (!(rope_theta > 0.0)) return QCF_ERR_INVALID_ARG;
  const bool no_seg = n_seg == 0 || max_seg_len == 0;
  const bool no_query = n_query == 0;
  const bool no_probe = n_probe == 0;
  const bool cache_used = !no_seg || !no_query;
  const bool pic_used = !no_seg || !no_probe;
  if (!tensor_ok(k_cache, !cache_used) || !tensor_ok(v_cache, !cache_used) ||
      !tensor_ok(k_pic, !pic_used) || !tensor_ok(v_pic, !pic_used))
    return QCF_ERR_INVALID_ARG;
  if (!tensor_ok(q_new, no_query) || !tensor_ok(k_new, no_query) || !tensor_ok(v_new, no_query) ||
      !tensor_ok(q_u, no_query))
    return QCF_ERR_INVALID_ARG;
  const bool probe_written = !no_probe || (query_slot != nullptr && !no_query);
  if (!tensor_ok(probe_k, !probe_written) || !tensor_ok(probe_v, !probe_written))
    return QCF_ERR_INVALID_ARG;
  if (!index_ok(seg_start, no_seg) || !index_ok(seg_len, no_seg) || !index_ok(seg_delta, no_seg) ||
      (src_start && !index_ok(src_start, false)))
    return QCF_ERR_INVALID_ARG;
  if (!index_ok(query_row, no_query) || !index_ok(query_pos, no_query) ||
      (query_src && !index_ok(query_src, false)) || (query_slot && !index_ok(query_slot, false)))
    return QCF_ERR_INVALID_ARG;
  if (!index_ok(probe_src, no_probe) || !index_ok(probe_delta, no_probe)) return QCF_ERR_INVALID_ARG;
  if (no_seg && no_query && no_probe) return QCF_OK;
  qcf::AssembleShape s{};
  s.n_rows = n_rows;
  s.row_stride = row_stride;
  s.pic_row_stride = pic_row_stride;
  s.probe_row_stride = probe_row_stride;
  s.n_pic_rows = n_pic_rows;
  s.n_src_rows = n_src_rows;
  s.n_query = n_query;
  s.n_probe = n_probe;
  s.n_seg = no_seg ? 0 : n_seg;
  s.max_seg_len = no_seg ? 0 : max_seg_len;
  s.hq = n_q_heads;
  s.hkv = n_kv_heads;
  s.d = head_dim;
  s.bf16 = dtype == QCF_BF16;
  s.theta = rope_theta;
  qcf::AssemblePtrs p{};
  p.k_cache = k_cache;
  p.v_cache = v_cache;
  p.k_pic = k_pic;
  p.v_pic = v_pic;
  p.seg_start = seg_start;
  p.seg_len = seg_len;
  p.seg_delta = seg_delta;
  p.src_start = src_start;
  p.q_new = q_new;
  p.k_new = k_new;
  p.v_new = v_new;
  p.q_u = q_u;
  p.query_row = query_row;
  p.query_pos = query_pos;
  p.query_src = query_src;
  p.query_slot = query_slot;
  p.probe_k = probe_k;
  p.probe_v = probe_v;
  p.probe_src = probe_src;
  p.probe_delta = probe_delta;
  return hip_status(qcf::launch_assemble(s, p, stream));
}

size_t qcf_probe_scores_workspace_size(int batch, int max_q_len, int max_ctx_len, int n_q_heads,
                                       int n_kv_heads, int head_dim) {
  if (batch < 0 || max_q_len < 0 || max_ctx_len < 0) return 0;
  if (check_heads(n_q_heads, n_kv_heads, head_dim) != QCF_OK) return 0;
  qcf::ProbeShape s{batch, max_q_len, max_ctx_len, n_q_heads, n_kv_heads, head_dim};
  return qcf::probe_scores_workspace(s);
}

}  // extern "C"

namespace {

qcf_status probe_scores_impl(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                             const void* k, int64_t n_kv_rows, int64_t k_row_stride,
                             const qcf::KeyRot& rot, qcf_dtype dtype, int batch,
                             const int32_t* cu_q, const int32_t* cu_kv, const int32_t* ctx_len,
                             int max_q_len, int max_ctx_len, int n_q_heads, int n_kv_heads,
                             int head_dim, float softmax_scale, void* workspace,
                             size_t workspace_bytes, hipStream_t stream,
                             const qcf::SelectArgs* sel = nullptr) {
  if (!dtype_ok(dtype)) return QCF_ERR_UNSUPPORTED;
  qcf_status st = check_heads(n_q_heads, n_kv_heads, head_dim);
  if (st != QCF_OK) return st;
  if (batch < 0 || batch > 65535 || max_q_len < 0 || max_ctx_len < 0) return QCF_ERR_INVALID_ARG;
  if (n_q_rows < 0 || n_kv_rows < 0 || n_q_rows > INT32_MAX || n_kv_rows > INT32_MAX)
    return QCF_ERR_INVALID_ARG;
  if (k_row_stride < (int64_t)n_kv_heads * head_dim || (k_row_stride * esize(dtype)) % 16 != 0)
    return QCF_ERR_INVALID_ARG;
  if (!(softmax_scale > 0.f)) return QCF_ERR_INVALID_ARG;
  const bool empty = batch == 0 || max_ctx_len == 0;
  if (!index_ok(scores, empty) || !tensor_ok(q, empty || n_q_rows == 0) ||
      !tensor_ok(k, empty || n_kv_rows == 0))
    return QCF_ERR_INVALID_ARG;
  if (!index_ok(cu_q, batch == 0) || !index_ok(cu_kv, batch == 0) || !index_ok(ctx_len, batch == 0))
    return QCF_ERR_INVALID_ARG;
  if (empty) {
    if (!sel || sel->n_seg == 0 || sel->max_seg_len == 0) return QCF_OK;
    // no scores to compute: the selection runs on the stored ones
    return hip_status(qcf::launch_select_topk(sel->out_idx, sel->out_pos, sel->n_out, scores,
                                              n_kv_rows, sel->n_seg, sel->seg_start, sel->seg_len,
                                              sel->seg_k, sel->out_start, nullptr,
                                              sel->max_seg_len, stream, sel->seg_req, cu_kv,
                                              batch));
  }
  const size_t need = qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, n_q_heads,
                                                      n_kv_heads, head_dim);
  if (workspace_bytes < need || (need > 0 && (!workspace || !aligned256(workspace))))
    return QCF_ERR_WORKSPACE;
  qcf::ProbeShape s{batch, max_q_len, max_ctx_len, n_q_heads, n_kv_heads, head_dim};
  return hip_status(qcf::launch_probe_scores(scores, accumulate, q, n_q_rows, k, n_kv_rows,
                                             k_row_stride, rot, dtype == QCF_BF16, cu_q, cu_kv,
                                             ctx_len, s, softmax_scale, workspace, stream, sel));
}

}  // namespace

extern "C" {

qcf_status qcf_probe_scores(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                            const void* k, int64_t n_kv_rows, int64_t k_row_stride,
                            qcf_dtype dtype, int batch, const int32_t* cu_q, const int32_t* cu_kv,
                            const int32_t* ctx_len, int max_q_len, int max_ctx_len, int n_q_heads,
                            int n_kv_heads, int head_dim, float softmax_scale, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  return probe_scores_impl(scores, accumulate, q, n_q_rows, k, n_kv_rows, k_row_stride,
                           qcf::KeyRot{nullptr, nullptr, 0}, dtype, batch, cu_q, cu_kv, ctx_len,
                           max_q_len, max_ctx_len, n_q_heads, n_kv_heads, head_dim, softmax_scale,
                           workspace, workspace_bytes, stream);
}

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
                                   hipStream_t stream) {
  if (n_out < 0 || n_seg < 0 || max_seg_len < 0 || n_out > INT32_MAX) return QCF_ERR_INVALID_ARG;
  if (n_seg > INT32_MAX / 2) return QCF_ERR_UNSUPPORTED;
  const bool none = n_seg == 0 || max_seg_len == 0;
  if (!index_ok(out_idx, none || n_out == 0)) return QCF_ERR_INVALID_ARG;
  if (out_pos && !index_ok(out_pos, false)) return QCF_ERR_INVALID_ARG;
  if (!index_ok(seg_start, n_seg == 0) || !index_ok(seg_len, n_seg == 0) ||
      !index_ok(seg_k, n_seg == 0) || !index_ok(out_start, n_seg == 0) ||
      !index_ok(seg_req, n_seg == 0))
    return QCF_ERR_INVALID_ARG;
  if (!none && (batch <= 0 || !index_ok(cu_kv, false) || !index_ok(scores, n_kv_rows == 0)))
    return QCF_ERR_INVALID_ARG;
  const qcf::SelectArgs sel{out_idx, out_pos, n_out, n_seg, seg_start, seg_len,
                            seg_k, out_start, seg_req, max_seg_len};
  return probe_scores_impl(scores, accumulate, q, n_q_rows, k, n_kv_rows, k_row_stride,
                           qcf::KeyRot{nullptr, nullptr, 0}, dtype, batch, cu_q, cu_kv, ctx_len,
                           max_q_len, max_ctx_len, n_q_heads, n_kv_heads, head_dim, softmax_scale,
                           workspace, workspace_bytes, stream, none ? nullptr : &sel);
}

qcf_status qcf_rope_table(float* table, const int32_t* pos, int64_t n, int head_dim,
                          double rope_theta, hipStream_t stream) {
  if (n < 0 || n > INT32_MAX) return QCF_ERR_INVALID_ARG;
  if (head_dim != 64 && head_dim != 128) return QCF_ERR_UNSUPPORTED;
  if (!(rope_theta > 0.0)) return QCF_ERR_INVALID_ARG;
  if (!tensor_ok(table, n == 0) || !index_ok(pos, n == 0)) return QCF_ERR_INVALID_ARG;
  if (n == 0) return QCF_OK;
  return hip_status(qcf::launch_rope_table(table, pos, n, head_dim, rope_theta, stream));
}

qcf_status qcf_probe_scores_pic(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                                const void* k_pic, int64_t n_kv_rows, int64_t k_row_stride,
                                const int32_t* key_rot, const float* rope_table, int64_t n_rot,
                                qcf_dtype dtype, int batch, const int32_t* cu_q,
                                const int32_t* cu_kv, const int32_t* ctx_len, int max_q_len,
                                int max_ctx_len, int n_q_heads, int n_kv_heads, int head_dim,
                                float softmax_scale, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  const bool empty = batch == 0 || max_ctx_len == 0 || n_kv_rows == 0;
  if (n_rot < 0 || n_rot > INT32_MAX) return QCF_ERR_INVALID_ARG;
  if (!empty && (n_rot == 0 || !index_ok(key_rot, false) || !tensor_ok(rope_table, false)))
    return QCF_ERR_INVALID_ARG;
  // with no key to read the table is not touched (the other checks still apply)
  const qcf::KeyRot rot{empty ? nullptr : key_rot, rope_table, n_rot};
  return probe_scores_impl(scores, accumulate, q, n_q_rows, k_pic, n_kv_rows, k_row_stride, rot,
                           dtype, batch, cu_q, cu_kv, ctx_len, max_q_len, max_ctx_len, n_q_heads,
                           n_kv_heads, head_dim, softmax_scale, workspace, workspace_bytes, stream);
}

qcf_status qcf_select_topk(int32_t* out_idx, int32_t* out_pos, int64_t n_out, const float* scores,
                           int64_t n_scores, int n_seg, const int32_t* seg_start,
                           const int32_t* seg_len, const int32_t* seg_k, const int32_t* out_start,
                           const int32_t* pos_base, int max_seg_len, hipStream_t stream) {
  if (n_out < 0 || n_scores < 0 || n_seg < 0 || max_seg_len < 0) return QCF_ERR_INVALID_ARG;
  if (n_out > INT32_MAX || n_scores > INT32_MAX) return QCF_ERR_INVALID_ARG;
  if (n_seg > INT32_MAX / 2) return QCF_ERR_UNSUPPORTED;
  const bool empty = n_seg == 0 || max_seg_len == 0;
  if (!index_ok(out_idx, empty || n_out == 0) || !index_ok(scores, empty || n_scores == 0))
    return QCF_ERR_INVALID_ARG;
  if (out_pos && !index_ok(out_pos, false)) return QCF_ERR_INVALID_ARG;
  if (!index_ok(seg_start, n_seg == 0) || !index_ok(seg_len, n_seg == 0) ||
      !index_ok(seg_k, n_seg == 0) || !index_ok(out_start, n_seg == 0))
    return QCF_ERR_INVALID_ARG;
  if (pos_base && !index_ok(pos_base, false)) return QCF_ERR_INVALID_ARG;
  if (empty) return QCF_OK;
  return hip_status(qcf::launch_select_topk(out_idx, out_pos, n_out, scores, n_scores, n_seg,
                                            seg_start, seg_len, seg_k, out_start, pos_base,
                                            max_seg_len, stream));
}

size_t qcf_sparse_prefill_attn_workspace_size(int batch, int max_rows, int max_kv, int n_q_heads,
                                              int n_kv_heads, int head_dim, qcf_dtype dtype) {
  if (batch < 0 || max_rows < 0 || max_kv < 0 || !dtype_ok(dtype)) return 0;
  if (check_heads(n_q_heads, n_kv_heads, head_dim) != QCF_OK) return 0;
  qcf::AttnShape s{batch, max_rows, max_kv, n_q_heads, n_kv_heads, head_dim};
  return qcf::attn_workspace(s, dtype == QCF_BF16);
}

}  // extern "C"

namespace {

qcf_status attn_impl(void* out, float* lse, const void* q, const int32_t* row_pos, int64_t n_rows,
                     const int32_t* cu_rows, const void* k_cache, const void* v_cache,
                     int64_t n_kv_rows, int64_t kv_row_stride, const int32_t* cu_kv,
                     const int32_t* kv_pos, qcf_dtype dtype, int batch, int max_rows, int max_kv,
                     int n_q_heads, int n_kv_heads, int head_dim, float softmax_scale,
                     void* workspace, size_t workspace_bytes, hipStream_t stream,
                     const qcf::QueryRot& qrot) {
  if (!dtype_ok(dtype)) return QCF_ERR_UNSUPPORTED;
  qcf_status st = check_heads(n_q_heads, n_kv_heads, head_dim);
  if (st != QCF_OK) return st;
  if (n_rows < 0 || n_rows > INT32_MAX || n_kv_rows < 0 || n_kv_rows > INT32_MAX)
    return QCF_ERR_INVALID_ARG;
  if (batch < 0 || batch > 65535 || max_rows < 0 || max_kv < 0) return QCF_ERR_INVALID_ARG;
  if (kv_row_stride < (int64_t)n_kv_heads * head_dim || (kv_row_stride * esize(dtype)) % 16 != 0)
    return QCF_ERR_INVALID_ARG;
  if (!(softmax_scale > 0.f)) return QCF_ERR_INVALID_ARG;
  const bool empty = n_rows == 0 || batch == 0 || max_rows == 0;
  if (!tensor_ok(out, empty) || !tensor_ok(q, empty) || !index_ok(row_pos, empty) ||
      !index_ok(cu_rows, batch == 0) || !index_ok(cu_kv, batch == 0))
    return QCF_ERR_INVALID_ARG;
  if (!tensor_ok(k_cache, empty || n_kv_rows == 0) || !tensor_ok(v_cache, empty || n_kv_rows == 0))
    return QCF_ERR_INVALID_ARG;
  if (lse && !index_ok(lse, false)) return QCF_ERR_INVALID_ARG;
  if (kv_pos && !index_ok(kv_pos, false)) return QCF_ERR_INVALID_ARG;
  if (qrot.table) {
    if (dtype != QCF_BF16 || kv_pos) return QCF_ERR_UNSUPPORTED;
    if (!tensor_ok(qrot.table, empty) || qrot.n_table <= 0 || qrot.n_table > INT32_MAX)
      return QCF_ERR_INVALID_ARG;
    if (qrot.src && (!index_ok(qrot.src, empty) || qrot.n_src <= 0 || qrot.n_src > INT32_MAX))
      return QCF_ERR_INVALID_ARG;
  }
  if (empty) return QCF_OK;
  if (dtype == QCF_F32 && n_rows > 0x7fffffff) return QCF_ERR_UNSUPPORTED;
  const size_t need = qcf_sparse_prefill_attn_workspace_size(batch, max_rows, max_kv, n_q_heads,
                                                             n_kv_heads, head_dim, dtype);
  if (workspace_bytes < need || (need > 0 && (!workspace || !aligned256(workspace))))
    return QCF_ERR_WORKSPACE;
  qcf::AttnShape s{batch, max_rows, max_kv, n_q_heads, n_kv_heads, head_dim};
  return hip_status(qcf::launch_sparse_attn(out, lse, q, row_pos, n_rows, cu_rows, k_cache, v_cache,
                                            n_kv_rows, kv_row_stride, cu_kv, kv_pos,
                                            dtype == QCF_BF16, s, softmax_scale, workspace, stream,
                                            qrot));
}

}  // namespace

extern "C" {

qcf_status qcf_sparse_prefill_attn(void* out, float* lse, const void* q, const int32_t* row_pos,
                                   int64_t n_rows, const int32_t* cu_rows, const void* k_cache,
                                   const void* v_cache, int64_t n_kv_rows, int64_t kv_row_stride,
                                   const int32_t* cu_kv, const int32_t* kv_pos, qcf_dtype dtype,
                                   int batch, int max_rows, int max_kv, int n_q_heads,
                                   int n_kv_heads, int head_dim, float softmax_scale,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return attn_impl(out, lse, q, row_pos, n_rows, cu_rows, k_cache, v_cache, n_kv_rows,
                   kv_row_stride, cu_kv, kv_pos, dtype, batch, max_rows, max_kv, n_q_heads,
                   n_kv_heads, head_dim, softmax_scale, workspace, workspace_bytes, stream,
                   qcf::QueryRot{nullptr, 0, nullptr, 0});
}

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
                                        size_t workspace_bytes, hipStream_t stream) {
  if (!rope_table) return QCF_ERR_INVALID_ARG;
  if (!q_src && n_q_raw < n_rows) return QCF_ERR_INVALID_ARG;
  return attn_impl(out, lse, q_raw, row_pos, n_rows, cu_rows, k_cache, v_cache, n_kv_rows,
                   kv_row_stride, cu_kv, nullptr, dtype, batch, max_rows, max_kv, n_q_heads,
                   n_kv_heads, head_dim, softmax_scale, workspace, workspace_bytes, stream,
                   qcf::QueryRot{q_src, q_src ? n_q_raw : n_rows, rope_table, n_table});
}

}  // extern "C"
