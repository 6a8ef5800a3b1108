// Internal launchers of libqcf (host side).  Arguments were validated by the
// C ABI layer; each launcher enqueues its kernels on `stream` and returns the
// HIP launch status.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace qcf {

hipError_t launch_rerope(void* k_out, const void* k_in, void* v_out, const void* v_in, bool bf16,
                         int64_t n_out_rows, int64_t n_in_rows, int hkv, int d,
                         int64_t out_row_stride, int64_t in_row_stride, int n_seg,
                         const int32_t* seg_start,
                         const int32_t* seg_len, const int32_t* seg_delta,
                         const int32_t* src_start, int max_seg_len, double theta,
                         hipStream_t stream);

hipError_t launch_rope_table(float* table, const int32_t* pos, int64_t n, int d, double theta,
                             hipStream_t stream);

hipError_t launch_gather_rows(void* dst, const void* src, const int32_t* idx, int64_t n_rows,
                              int64_t n_src_rows, int64_t row_bytes, int64_t src_stride,
                              int64_t dst_stride, hipStream_t stream);

hipError_t launch_scatter_kv(void* k_cache, void* v_cache, int64_t n_cache_rows,
                             int64_t cache_row_stride, const void* k_new, const void* v_new,
                             const void* q_new, void* q_out, int64_t n_src_rows,
                             const int32_t* src_idx, bool bf16, int64_t n_rows,
                             const int32_t* row_idx, const int32_t* row_pos, int hq, int hkv,
                             int d, double theta, hipStream_t stream);

// Per-segment selection.  out_pos gets row - pos_base[s] when pos_base is set,
// else row - req_base[seg_req[s]] when seg_req is set (a segment whose request
// is outside [0, n_req) is skipped), else row.
hipError_t launch_select_topk(int32_t* out_idx, int32_t* out_pos, int64_t n_out,
                              const float* scores, int64_t n_scores, int n_seg,
                              const int32_t* seg_start, const int32_t* seg_len,
                              const int32_t* seg_k, const int32_t* out_start,
                              const int32_t* pos_base, int max_seg_len, hipStream_t stream,
                              const int32_t* seg_req = nullptr, const int32_t* req_base = nullptr,
                              int n_req = 0);

// A selection run on the scores of the same call, right after they are final
// (segment s lies in request seg_req[s]; out_pos relative to cu_kv[seg_req[s]]).
struct SelectArgs {
  int32_t* out_idx;
  int32_t* out_pos;
  int64_t n_out;
  int n_seg;
  const int32_t *seg_start, *seg_len, *seg_k, *out_start, *seg_req;
  int max_seg_len;
};
// The per-(KV head, query tile) column sums of the bf16 score passes, which the
// fused selection adds per key (in the order the separate final pass uses).
struct ScoreCols {
  const float* colp;
  const int32_t *cu_q, *cu_kv, *ctx_len;
  int64_t n_kv_rows;
  int batch, hkv, lg, n_qt, max_qv, max_ctx, qv_tile, accumulate;
};
// hipErrorNotSupported when a segment is longer than 1024 rows
hipError_t launch_select_topk_cols(float* scores, int64_t n_scores, const ScoreCols& c,
                                   const SelectArgs& a, hipStream_t stream);

// Re-positioning calls whose stored chunk caches (K and V) exceed this many bytes
// read them with the non-temporal hint: sources larger than the last-level cache
// cannot stay there until the next step anyway, and hinted reads keep them from
// evicting the request cache that the scores and the recompute read next
// (c5, 939 MB: assemble 198 -> 166 us, re-position 173 -> 136 us; c4, 134 MB:
// plain reads, which the cache keeps between steps, stay faster).
constexpr int64_t kStreamSourceBytes = 256ll << 20;

struct AssembleShape {
  int64_t n_rows, row_stride, pic_row_stride, probe_row_stride, n_pic_rows, n_src_rows, n_query,
      n_probe;
  int n_seg, max_seg_len, hq, hkv, d;
  bool bf16;
  double theta;
};
struct AssemblePtrs {
  void *k_cache, *v_cache;
  const void *k_pic, *v_pic;
  const int32_t *seg_start, *seg_len, *seg_delta, *src_start;
  const void *q_new, *k_new, *v_new;
  void* q_u;
  const int32_t *query_row, *query_pos, *query_src, *query_slot;
  void *probe_k, *probe_v;
  const int32_t *probe_src, *probe_delta;
};
hipError_t launch_assemble(const AssembleShape& s, const AssemblePtrs& p, hipStream_t stream);

struct ProbeShape {
  int batch, max_q_len, max_ctx_len, hq, hkv, d;
};
// Keys rotated on the fly: key row t is turned by table row key_rot[t]
// (clamped into [0, n)); a null `row` reads the keys as stored.
struct KeyRot {
  const int32_t* row;
  const float* table;
  int64_t n;
};
size_t probe_scores_workspace(const ProbeShape& s);
hipError_t launch_probe_scores(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                               const void* k, int64_t n_kv_rows, int64_t k_row_stride,
                               const KeyRot& rot, bool bf16, const int32_t* cu_q,
                               const int32_t* cu_kv, const int32_t* ctx_len, const ProbeShape& s,
                               float scale, void* ws, hipStream_t stream,
                               const SelectArgs* sel = nullptr);

struct AttnShape {
  int batch, max_rows, max_kv, hq, hkv, d;
};
// Un-rotated queries: the rows of q are turned in the kernel by table row
// row_pos[r] (table from qcf_rope_table at positions 0..n_table-1), read
// through src[r] when src is given (n_src rows of q).  table == nullptr: q is
// already rotated and indexed by r.
struct QueryRot {
  const int32_t* src;
  int64_t n_src;
  const float* table;
  int64_t n_table;
};
size_t attn_workspace(const AttnShape& s, bool bf16);
hipError_t launch_sparse_attn(void* out, float* lse, const void* q, const int32_t* row_pos,
                              int64_t n_rows, const int32_t* cu_rows, const void* k_cache,
                              const void* v_cache, int64_t n_kv_rows, int64_t kv_row_stride,
                              const int32_t* cu_kv, const int32_t* kv_pos, bool bf16,
                              const AttnShape& s, float scale, void* ws, hipStream_t stream,
                              const QueryRot& qrot = QueryRot{nullptr, 0, nullptr, 0});

}  // namespace qcf
