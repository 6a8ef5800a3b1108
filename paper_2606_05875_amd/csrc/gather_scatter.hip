// Row gather (anchor cache, eq. anchor_cache) and the fused-cache scatter
// (eq. fuse_cache) with the rotary embedding of the recomputed rows.
//
// Both are HBM-bound streams of 16-byte vectors.  The scatter gives every
// recomputed row its own block: the block forms the row's d/2 (cos, sin) pairs
// once (float64 angle) and its threads then rotate the row's key heads and
// query heads and copy its value heads, so the per-row trigonometry is shared
// by all H_q + H_kv heads of the row.
#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void gather_rows_kernel(
    uint8_t* __restrict__ dst, const uint8_t* __restrict__ src, const int32_t* __restrict__ idx,
    int64_t n_rows, int64_t n_src_rows, int64_t chunks_per_row, int64_t src_stride,
    int64_t dst_stride) {
  const int64_t total = n_rows * chunks_per_row;
  for (int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x; u < total;
       u += (int64_t)gridDim.x * kThreads) {
    const int64_t r = u / chunks_per_row;
    const int64_t c = u - r * chunks_per_row;
    const int64_t s = idx[r];
    if (s < 0 || s >= n_src_rows) continue;
    st16(dst + r * dst_stride + c * 16, ld16(src + s * src_stride + c * 16));
  }
}

// One recomputed row per block.  Every load of the row -- the value heads,
// the key heads' and the query heads' rotate-half pairs, kRound units of each
// per thread -- is issued, unmasked from clamped units, before the first
// store (a load under a lane condition gets a wait of its own); the angle
// table is formed meanwhile.  Rows wider than a round finish in later rounds.
constexpr int kRound = 2;

template <typename T, int D>
struct RopeUnits {
  static constexpr int HALF = D / 2, VEC = Vec16<T>::N, UPH = HALF / VEC;
  uint4 a[kRound], b[kRound];
  int off[kRound], jj[kRound];
  __device__ __forceinline__ void load(const T* src, int base, int units) {
#pragma unroll
    for (int k = 0; k < kRound; ++k) {
      const int u = min(base + (int)threadIdx.x + k * kThreads, units - 1);
      const int h = u / UPH;
      jj[k] = (u - h * UPH) * VEC;
      off[k] = h * D + jj[k];
      a[k] = ld16(src + off[k]);
      b[k] = ld16(src + off[k] + HALF);
    }
  }
  __device__ __forceinline__ void store(T* dst, int base, int units, const float2* cs) const {
#pragma unroll
    for (int k = 0; k < kRound; ++k) {
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Vec16<T>::unpack(a[k], x1);
      Vec16<T>::unpack(b[k], x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        rope_pair(x1[e], x2[e], cs[jj[k] + e], y1[e], y2[e]);
      }
      if (base + (int)threadIdx.x + k * kThreads < units) {
        st16(dst + off[k], Vec16<T>::pack(y1));
        st16(dst + off[k] + HALF, Vec16<T>::pack(y2));
      }
    }
  }
};

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void scatter_kv_kernel(
    T* k_cache, T* v_cache, int64_t n_cache_rows, int64_t cache_stride, const T* k_new,
    const T* v_new, const T* q_new, T* q_out, int64_t n_src_rows, const int32_t* src_idx,
    const int32_t* __restrict__ row_idx, const int32_t* __restrict__ row_pos, int hq, int hkv,
    double theta) {
  constexpr int HALF = D / 2;
  constexpr int VEC = Vec16<T>::N;
  constexpr int UPH = HALF / VEC;
  __shared__ float2 cs[HALF];
  const int64_t r = blockIdx.x;
  const int64_t s = src_idx ? (int64_t)src_idx[r] : r;
  if (s < 0 || s >= n_src_rows) return;
  const int64_t dst = row_idx[r];
  const bool dst_ok = dst >= 0 && dst < n_cache_rows;
  const int kv_row = hkv * D, q_row = hq * D;
  const int nv = kv_row / VEC, nk = hkv * UPH, nq = q_out ? hq * UPH : 0;
  const T* vs = v_new + s * kv_row;
  const T* ks = k_new + s * kv_row;
  const T* qs = q_new ? q_new + s * q_row : nullptr;
  T* vd = v_cache + (dst_ok ? dst : 0) * cache_stride;
  T* kd = k_cache + (dst_ok ? dst : 0) * cache_stride;
  for (int base = 0; base < max(max(nv, nk), nq); base += kThreads * kRound) {
    uint4 vbuf[kRound];
#pragma unroll
    for (int k = 0; k < kRound; ++k) vbuf[k] = ld16(vs + min(base + (int)threadIdx.x + k * kThreads, nv - 1) * VEC);
    RopeUnits<T, D> ku, qu;
    ku.load(ks, min(base, nk - 1), nk);
    if (nq > 0) qu.load(qs, min(base, nq - 1), nq);
    if (base == 0) {
      if (threadIdx.x < HALF) cs[threadIdx.x] = rope_cs((double)row_pos[r], threadIdx.x, D, theta);
      __syncthreads();
    }
    if (dst_ok) {
      if (base < nk) ku.store(kd, base, nk, cs);
#pragma unroll
      for (int k = 0; k < kRound; ++k) {
        const int c = base + threadIdx.x + k * kThreads;
        if (c < nv) st16(vd + c * VEC, vbuf[k]);
      }
    }
    if (base < nq) qu.store(q_out + r * q_row, base, nq, cs);
  }
}

// The scatter without queries (fresh K/V only): four rows per block, 64
// threads per row.  A thread loads its row's key rotate-half units and value
// chunks of a round (for bf16 with 8 x 128 key heads: one unit and two chunks,
// the whole row in one round), forms one (cos, sin) pair of the row meanwhile,
// and stores after the block's table is complete.  Same rotation arithmetic as
// scatter_kv_kernel, so the same bits.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void scatter_kv_rows_kernel(
    T* k_cache, T* v_cache, int64_t n_cache_rows, int64_t cache_stride, const T* k_new,
    const T* v_new, int64_t n_src_rows, const int32_t* src_idx, const int32_t* __restrict__ row_idx,
    const int32_t* __restrict__ row_pos, int64_t n_rows, int hkv, double theta) {
  constexpr int HALF = D / 2;
  constexpr int VEC = Vec16<T>::N;
  constexpr int UPH = HALF / VEC;
  constexpr int TPR = 64, RPB = kThreads / TPR;
  constexpr int KR = sizeof(T) == 2 ? 1 : 2, VR = 2 * KR;  // units per thread and round
  __shared__ float2 cs[RPB][HALF];
  const int sub = threadIdx.x / TPR, lt = threadIdx.x % TPR;
  const int64_t r = (int64_t)blockIdx.x * RPB + sub;
  const int64_t rc = min(r, n_rows - 1);
  const int64_t s = src_idx ? (int64_t)src_idx[rc] : rc;
  const bool s_ok = s >= 0 && s < n_src_rows;
  const int64_t dst = row_idx[rc];
  const bool ok = r < n_rows && s_ok && dst >= 0 && dst < n_cache_rows;
  const int kv_row = hkv * D;
  const int nv = kv_row / VEC, nk = hkv * UPH;
  const T* vs = v_new + (s_ok ? s : 0) * kv_row;
  const T* ks = k_new + (s_ok ? s : 0) * kv_row;
  T* vd = v_cache + (ok ? dst : 0) * cache_stride;
  T* kd = k_cache + (ok ? dst : 0) * cache_stride;
  for (int round = 0; round * TPR * KR < nk || round * TPR * VR < nv; ++round) {
    uint4 vb[VR], ka[KR], kb[KR];
    int koff[KR], kj[KR];
#pragma unroll
    for (int i = 0; i < VR; ++i) vb[i] = ld16(vs + min(round * TPR * VR + lt + TPR * i, nv - 1) * VEC);
#pragma unroll
    for (int i = 0; i < KR; ++i) {
      const int u = min(round * TPR * KR + lt + TPR * i, nk - 1);
      const int h = u / UPH;
      kj[i] = (u - h * UPH) * VEC;
      koff[i] = h * D + kj[i];
      ka[i] = ld16(ks + koff[i]);
      kb[i] = ld16(ks + koff[i] + HALF);
    }
    if (round == 0) {
      for (int j = lt; j < HALF; j += TPR) cs[sub][j] = rope_cs((double)row_pos[rc], j, D, theta);
      __syncthreads();
    }
    if (!ok) continue;
#pragma unroll
    for (int i = 0; i < VR; ++i) {
      const int c = round * TPR * VR + lt + TPR * i;
      if (c < nv) st16(vd + c * VEC, vb[i]);
    }
#pragma unroll
    for (int i = 0; i < KR; ++i) {
      if (round * TPR * KR + lt + TPR * i >= nk) continue;
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Vec16<T>::unpack(ka[i], x1);
      Vec16<T>::unpack(kb[i], x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) rope_pair(x1[e], x2[e], cs[sub][kj[i] + e], y1[e], y2[e]);
      st16(kd + koff[i], Vec16<T>::pack(y1));
      st16(kd + koff[i] + HALF, Vec16<T>::pack(y2));
    }
  }
}

template <typename T, int D>
hipError_t scatter_t(void* k_cache, void* v_cache, int64_t n_cache_rows, int64_t cache_stride,
                     const void* k_new, const void* v_new, const void* q_new, void* q_out,
                     int64_t n_src_rows, const int32_t* src_idx, int64_t n_rows,
                     const int32_t* row_idx, const int32_t* row_pos, int hq, int hkv,
                     double theta, hipStream_t stream) {
  if (!q_new && !q_out) {
    constexpr int RPB = kThreads / 64;
    scatter_kv_rows_kernel<T, D><<<dim3((unsigned)((n_rows + RPB - 1) / RPB)), kThreads, 0, stream>>>(
        static_cast<T*>(k_cache), static_cast<T*>(v_cache), n_cache_rows, cache_stride,
        static_cast<const T*>(k_new), static_cast<const T*>(v_new), n_src_rows, src_idx, row_idx,
        row_pos, n_rows, hkv, theta);
    return hipGetLastError();
  }
  scatter_kv_kernel<T, D><<<dim3((unsigned)n_rows), kThreads, 0, stream>>>(
      static_cast<T*>(k_cache), static_cast<T*>(v_cache), n_cache_rows, cache_stride,
      static_cast<const T*>(k_new), static_cast<const T*>(v_new), static_cast<const T*>(q_new),
      static_cast<T*>(q_out), n_src_rows, src_idx, row_idx, row_pos, hq, hkv, theta);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gather_rows(void* dst, const void* src, const int32_t* idx, int64_t n_rows,
                              int64_t n_src_rows, int64_t row_bytes, int64_t src_stride,
                              int64_t dst_stride, hipStream_t stream) {
  if (n_rows == 0 || row_bytes == 0) return hipSuccess;
  const int64_t chunks = row_bytes / 16;
  const int64_t total = n_rows * chunks;
  int64_t blocks = (total + kThreads - 1) / kThreads;
  if (blocks > 65536) blocks = 65536;
  gather_rows_kernel<<<dim3((unsigned)blocks), kThreads, 0, stream>>>(
      static_cast<uint8_t*>(dst), static_cast<const uint8_t*>(src), idx, n_rows, n_src_rows,
      chunks, src_stride, dst_stride);
  return hipGetLastError();
}

hipError_t launch_scatter_kv(void* k_cache, void* v_cache, int64_t n_cache_rows,
                             int64_t cache_row_stride, const void* k_new, const void* v_new,
                             const void* q_new, void* q_out, int64_t n_src_rows,
                             const int32_t* src_idx, bool bf16, int64_t n_rows,
                             const int32_t* row_idx, const int32_t* row_pos, int hq, int hkv,
                             int d, double theta, hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
#define QCF_SCATTER(T, D)                                                                   \
  return scatter_t<T, D>(k_cache, v_cache, n_cache_rows, cache_row_stride, k_new, v_new, q_new, \
                         q_out, n_src_rows, src_idx, n_rows, row_idx, row_pos, hq, hkv, theta, \
                         stream)
  if (bf16) {
    if (d == 64) QCF_SCATTER(uint16_t, 64);
    QCF_SCATTER(uint16_t, 128);
  }
  if (d == 64) QCF_SCATTER(float, 64);
  QCF_SCATTER(float, 128);
#undef QCF_SCATTER
}

}  // namespace qcf
