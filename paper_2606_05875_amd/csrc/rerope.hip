// Position remapping and stitching of the reused chunk caches (Section 2.1.2,
// eq. pic_online).
//
// A stored chunk key is rotated at its chunk-local position; moving the chunk
// to request offset o_i is one more rotation by o_i, and its values are copied
// in the same token order.  The rotation is the same for every row of a chunk,
// so a block works inside one chunk: every thread issues its 16-byte loads of
// rotate-half pairs (j .. j+v, j+d/2 .. j+d/2+v) of one head of one row and of
// the value rows, the block forms the chunk's d/2 (cos, sin) pairs (float64
// angle) while they are in flight, then rotates and stores.  HBM-bound: every
// byte is read once and written once with coalesced 16-byte accesses.
#include "qcf_device.h"
#include "qcf_launch.h"
#include "qcf_remap.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kUnitsPerThread = 1;  // key units (rotate-half pairs) per thread per round (swept: 1, 2, 4)

template <typename T, int D, bool kStreamIn>
__global__ __launch_bounds__(kThreads) void rerope_kernel(
    T* k_out, const T* k_in, T* v_out, const T* v_in, int64_t n_out_rows, int64_t n_in_rows,
    int hkv, int64_t out_stride, int64_t in_stride, int rows_per_block,
    const int32_t* __restrict__ seg_start,
    const int32_t* __restrict__ seg_len, const int32_t* __restrict__ seg_delta,
    const int32_t* __restrict__ src_start, double theta) {
  constexpr int HALF = D / 2;
  __shared__ float2 cs[HALF];

  const int s = blockIdx.y;
  const int len = seg_len[s];
  const int r0 = blockIdx.x * rows_per_block;
  if (r0 >= len) return;
  const int64_t dst0 = (int64_t)seg_start[s] + r0;
  const int64_t src0 = (src_start ? (int64_t)src_start[s] : (int64_t)seg_start[s]) + r0;
  // values are stitched unchanged, in the same token order (nothing to do in place)
  T* vdst = (v_out == nullptr || v_out == v_in) ? nullptr : v_out;
  remap_rows<T, D, kThreads, kUnitsPerThread, kStreamIn, true>(
      k_out, vdst, out_stride, k_in, v_in, in_stride, src0, dst0, min(rows_per_block, len - r0),
      hkv, n_in_rows, n_out_rows, cs, [&] {
        if (threadIdx.x < HALF) cs[threadIdx.x] = rope_cs((double)seg_delta[s], threadIdx.x, D, theta);
        __syncthreads();
      });
}

template <typename T, int D>
hipError_t launch_t(void* k_out, const void* k_in, void* v_out, const void* v_in,
                    int64_t n_out_rows, int64_t n_in_rows, int hkv, int64_t out_stride,
                    int64_t in_stride, int n_seg,
                    const int32_t* seg_start, const int32_t* seg_len, const int32_t* seg_delta,
                    const int32_t* src_start, int max_seg_len, double theta, hipStream_t stream) {
  const int units_per_row = hkv * (D / 2) / Vec16<T>::N;
  const int rpb = max(1, kThreads * kUnitsPerThread / units_per_row);
  dim3 grid((max_seg_len + rpb - 1) / rpb, n_seg);
  // the stored keys' (and values') bytes
  const int64_t src_bytes =
      n_in_rows * (int64_t)hkv * D * (int64_t)sizeof(T) * (v_in != nullptr && v_out != nullptr ? 2 : 1);
  auto kern = src_bytes > kStreamSourceBytes ? rerope_kernel<T, D, true> : rerope_kernel<T, D, false>;
  kern<<<grid, kThreads, 0, stream>>>(
      static_cast<T*>(k_out), static_cast<const T*>(k_in), static_cast<T*>(v_out),
      static_cast<const T*>(v_in), n_out_rows, n_in_rows, hkv, out_stride, in_stride, rpb, seg_start,
      seg_len, seg_delta, src_start, theta);
  return hipGetLastError();
}

// table[i * d/2 + j] = the (cos, sin) that every rotation of this library
// forms for offset pos[i] and frequency j (float64 angle, rounded to float32)
__global__ __launch_bounds__(64) void rope_table_kernel(float2* __restrict__ table,
                                                        const int32_t* __restrict__ pos, int d,
                                                        double theta) {
  const int64_t i = blockIdx.x;
  if ((int)threadIdx.x < d / 2)
    table[i * (d / 2) + threadIdx.x] = rope_cs((double)pos[i], threadIdx.x, d, theta);
}

}  // namespace

hipError_t launch_rope_table(float* table, const int32_t* pos, int64_t n, int d, double theta,
                             hipStream_t stream) {
  if (n == 0) return hipSuccess;
  rope_table_kernel<<<dim3((unsigned)n), 64, 0, stream>>>(reinterpret_cast<float2*>(table), pos, d,
                                                          theta);
  return hipGetLastError();
}

hipError_t launch_rerope(void* k_out, const void* k_in, void* v_out, const void* v_in, bool bf16,
                         int64_t n_out_rows, int64_t n_in_rows, int hkv, int d,
                         int64_t out_row_stride, int64_t in_row_stride, int n_seg,
                         const int32_t* seg_start,
                         const int32_t* seg_len, const int32_t* seg_delta,
                         const int32_t* src_start, int max_seg_len, double theta,
                         hipStream_t stream) {
  if (n_seg == 0 || max_seg_len == 0 || n_out_rows == 0 || n_in_rows == 0) return hipSuccess;
#define QCF_REROPE(T, D)                                                                       \
  return launch_t<T, D>(k_out, k_in, v_out, v_in, n_out_rows, n_in_rows, hkv, out_row_stride,   \
                        in_row_stride, n_seg,                                                  \
                        seg_start, seg_len, seg_delta, src_start, max_seg_len, theta, stream)
  if (bf16) {
    if (d == 64) QCF_REROPE(uint16_t, 64);
    QCF_REROPE(uint16_t, 128);
  }
  if (d == 64) QCF_REROPE(float, 64);
  QCF_REROPE(float, 128);
#undef QCF_REROPE
}

}  // namespace qcf
