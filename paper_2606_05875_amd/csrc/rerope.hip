// Position remapping of the reused chunk keys (Section 2.1.2, eq. pic_online).
//
// A stored chunk key is rotated at its chunk-local position; moving the chunk
// to request offset o_i is one more rotation by o_i.  The rotation is the same
// for every row of a chunk, so a block works inside one chunk: its first
// threads form the chunk's d/2 (cos, sin) pairs once (float64 angle), and every
// thread then streams 16-byte vectors of the rotate-half pairs (j .. j+v,
// j+d/2 .. j+d/2+v) of one head of one row.  HBM-bound: every key byte is read
// once and written once with coalesced 16-byte accesses.
#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kUnitsPerThread = 4;  // (row, head, j-vector) units each thread owns

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void rerope_kernel(T* out, const T* in,
                                                          int64_t n_tokens, int hkv,
                                                          int64_t row_stride, int rows_per_block,
                                                          const int32_t* __restrict__ seg_start,
                                                          const int32_t* __restrict__ seg_len,
                                                          const int32_t* __restrict__ seg_delta,
                                                          double theta) {
  constexpr int HALF = D / 2;
  constexpr int VEC = Vec16<T>::N;
  constexpr int UPH = HALF / VEC;  // units per head
  __shared__ float2 cs[HALF];

  const int s = blockIdx.y;
  const int len = seg_len[s];
  const int r0 = blockIdx.x * rows_per_block;
  if (r0 >= len) return;
  const int64_t start = seg_start[s];
  if (threadIdx.x < HALF) cs[threadIdx.x] = rope_cs((double)seg_delta[s], threadIdx.x, D, theta);
  __syncthreads();

  const int rows = min(rows_per_block, len - r0);
  const int units_per_row = hkv * UPH;
  const int total = rows * units_per_row;

  // Loads of all owned units are issued before any store: in-place calls
  // (out == in) stay correct because every unit is read and written by the
  // same thread.
  for (int base = 0; base < total; base += kThreads * kUnitsPerThread) {
    uint4 lo[kUnitsPerThread], hi[kUnitsPerThread];
    int64_t off[kUnitsPerThread];
    int jj[kUnitsPerThread];
#pragma unroll
    for (int k = 0; k < kUnitsPerThread; ++k) {
      const int u = base + threadIdx.x + k * kThreads;
      off[k] = -1;
      jj[k] = 0;
      if (u < total) {
        const int rr = u / units_per_row;
        const int c = u - rr * units_per_row;
        const int h = c / UPH;
        jj[k] = (c - h * UPH) * VEC;
        const int64_t row = start + r0 + rr;
        if (row >= 0 && row < n_tokens) {
          off[k] = row * row_stride + (int64_t)h * D + jj[k];
          lo[k] = ld16(in + off[k]);
          hi[k] = ld16(in + off[k] + HALF);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kUnitsPerThread; ++k) {
      if (off[k] < 0) continue;
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Vec16<T>::unpack(lo[k], x1);
      Vec16<T>::unpack(hi[k], x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float2 r = cs[jj[k] + e];
        y1[e] = x1[e] * r.x - x2[e] * r.y;
        y2[e] = x1[e] * r.y + x2[e] * r.x;
      }
      st16(out + off[k], Vec16<T>::pack(y1));
      st16(out + off[k] + HALF, Vec16<T>::pack(y2));
    }
  }
}

template <typename T, int D>
hipError_t launch_t(void* k_out, const void* k_in, int64_t n_tokens, int hkv, int64_t row_stride,
                    int n_seg, const int32_t* seg_start, const int32_t* seg_len,
                    const int32_t* seg_delta, int max_seg_len, double theta, hipStream_t stream) {
  const int units_per_row = hkv * (D / 2) / Vec16<T>::N;
  const int rpb = max(1, kThreads * kUnitsPerThread / units_per_row);
  dim3 grid((max_seg_len + rpb - 1) / rpb, n_seg);
  rerope_kernel<T, D><<<grid, kThreads, 0, stream>>>(
      static_cast<T*>(k_out), static_cast<const T*>(k_in), n_tokens, hkv, row_stride, rpb,
      seg_start, seg_len, seg_delta, theta);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_rerope(void* k_out, const void* k_in, bool bf16, int64_t n_tokens, int hkv,
                         int d, int64_t row_stride, int n_seg, const int32_t* seg_start,
                         const int32_t* seg_len, const int32_t* seg_delta, int max_seg_len,
                         double theta, hipStream_t stream) {
  if (n_seg == 0 || max_seg_len == 0 || n_tokens == 0) return hipSuccess;
  if (bf16) {
    return d == 64 ? launch_t<uint16_t, 64>(k_out, k_in, n_tokens, hkv, row_stride, n_seg,
                                            seg_start, seg_len, seg_delta, max_seg_len, theta,
                                            stream)
                   : launch_t<uint16_t, 128>(k_out, k_in, n_tokens, hkv, row_stride, n_seg,
                                             seg_start, seg_len, seg_delta, max_seg_len, theta,
                                             stream);
  }
  return d == 64 ? launch_t<float, 64>(k_out, k_in, n_tokens, hkv, row_stride, n_seg, seg_start,
                                       seg_len, seg_delta, max_seg_len, theta, stream)
                 : launch_t<float, 128>(k_out, k_in, n_tokens, hkv, row_stride, n_seg, seg_start,
                                        seg_len, seg_delta, max_seg_len, theta, stream);
}

}  // namespace qcf
