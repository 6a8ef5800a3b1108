// The selector call (critical-layer scores + per-segment top-k) for callers
// that cannot allocate device memory: HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc.  Its scratch space is a fixed device array
// in this file instead of a caller workspace; everything else -- argument
// checks, kernels, results -- is qcf_probe_scores_select's.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "qcf.h"

namespace {

// The scratch array.  In host code its name is only a stand-in for the
// device symbol; its device address comes from hipGetSymbolAddress, once per
// device (every GPU holds its own copy until the process ends).
static __device__ __align__(256) uint8_t scratch[QCF_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices] = {};
std::mutex g_mutex;

// Device address of the current device's scratch array (looked up on the
// first call on that device), or nullptr with *err set.
void* scratch_ptr(qcf_status* err) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *err = QCF_ERR_HIP;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      *err = QCF_ERR_HIP;
      return nullptr;
    }
    g_scratch[dev] = p;
  }
  return g_scratch[dev];
}

}  // namespace

extern "C" qcf_status qcf_probe_scores_select_noalloc(
    float* scores, int accumulate, const void* q, int64_t n_q_rows, const void* k,
    int64_t n_kv_rows, int64_t k_row_stride, qcf_dtype dtype, int batch, const int32_t* cu_q,
    const int32_t* cu_kv, const int32_t* ctx_len, int max_q_len, int max_ctx_len, int n_q_heads,
    int n_kv_heads, int head_dim, float softmax_scale, int32_t* out_idx, int32_t* out_pos,
    int64_t n_out, int n_seg, const int32_t* seg_start, const int32_t* seg_len,
    const int32_t* seg_k, const int32_t* out_start, const int32_t* seg_req, int max_seg_len,
    hipStream_t stream) {
  const size_t need = qcf_probe_scores_workspace_size(batch, max_q_len, max_ctx_len, n_q_heads,
                                                      n_kv_heads, head_dim);
  if (need > (size_t)QCF_NOALLOC_SCRATCH_BYTES) return QCF_ERR_WORKSPACE;
  qcf_status err = QCF_OK;
  void* ws = scratch_ptr(&err);
  if (!ws) return err;
  // the kernels need no initialised scratch: every word they read back was
  // written earlier in the same call
  return qcf_probe_scores_select(scores, accumulate, q, n_q_rows, k, n_kv_rows, k_row_stride,
                                 dtype, batch, cu_q, cu_kv, ctx_len, max_q_len, max_ctx_len,
                                 n_q_heads, n_kv_heads, head_dim, softmax_scale, out_idx, out_pos,
                                 n_out, n_seg, seg_start, seg_len, seg_k, out_start, seg_req,
                                 max_seg_len, ws, (size_t)QCF_NOALLOC_SCRATCH_BYTES, stream);
}
