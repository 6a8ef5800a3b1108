// One launch that assembles a layer's request cache and the anchor probe
// buffer (Section 3.5, selective token localization, first half):
//  * every chunk's stored keys are re-positioned and its values stitched into
//    the request cache (eq. pic_online);
//  * the user-query rows get their fresh q/k rotated at positions N + i; k and
//    v go into the request cache and into the probe buffer, q into q_u;
//  * the anchor rows of the probe buffer are re-positioned straight from the
//    stored chunk caches (KV^A = Pi(KV^PIC[A]), eq. anchor_cache).
// The three parts touch disjoint outputs, so one grid runs them side by side:
// blocks [0, n_remap) remap chunk tiles, the next n_query blocks handle one
// query row each, the rest handle tiles of anchor slots.  All parts are
// HBM-bound 16-byte streams; rotation angles are formed in float64 once per
// block (constant per chunk) or once per row.
#include "qcf_device.h"
#include "qcf_launch.h"
#include "qcf_remap.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kUnits = 2;  // 16-byte units per thread per pass (swept: 1, 2, 4)

template <typename T, int D>
struct AssembleArgs {
  T *k_cache, *v_cache;
  int64_t n_rows, row_stride;
  const T *k_pic, *v_pic;
  int64_t n_pic_rows, pic_stride;
  const int32_t *seg_start, *seg_len, *seg_delta, *src_start;
  int n_seg, rows_per_block, tiles_per_seg;
  // query rows
  const T *k_new, *v_new, *q_new;
  T* q_u;
  int64_t n_src_rows;
  int n_query;
  const int32_t *query_row, *query_pos, *query_src, *query_slot;
  // probe buffer
  T *probe_k, *probe_v;
  int64_t n_probe, probe_stride;
  const int32_t *probe_src, *probe_delta;
  int probe_rows_per_block;
  int hq, hkv;
  double theta;
};

template <typename T, int D, bool kStreamIn>
__global__ __launch_bounds__(kThreads) void assemble_kernel(AssembleArgs<T, D> A) {
  constexpr int HALF = D / 2;
  __shared__ float2 cs[HALF];
  const int n_remap = A.n_seg * A.tiles_per_seg;
  const int bid = blockIdx.x;
  const int kvw = A.hkv * D;  // elements of a K/V row
  if (bid < n_remap) {
    // ---- a chunk tile: re-position keys, stitch values
    const int s = bid / A.tiles_per_seg;
    const int r0 = (bid - s * A.tiles_per_seg) * A.rows_per_block;
    const int len = A.seg_len[s];
    if (r0 >= len) return;
    const int64_t d0 = (int64_t)A.seg_start[s] + r0;
    const int64_t s0 = (A.src_start ? (int64_t)A.src_start[s] : (int64_t)A.seg_start[s]) + r0;
    // the angle table first: forming it while this kernel's loads are in flight
    // holds them across the float64 work and costs occupancy (measured slower)
    if (threadIdx.x < HALF) cs[threadIdx.x] = rope_cs((double)A.seg_delta[s], threadIdx.x, D, A.theta);
    __syncthreads();
    remap_rows<T, D, kThreads, kUnits, kStreamIn, true>(
        A.k_cache, A.v_cache, A.row_stride, A.k_pic, A.v_pic, A.pic_stride, s0, d0,
        min(A.rows_per_block, len - r0), A.hkv, A.n_pic_rows, A.n_rows, cs, [] {});
    return;
  }
  if (bid < n_remap + A.n_query) {
    // ---- one user-query row: rotate at its position into the cache, the probe
    //      buffer and q_u
    const int i = bid - n_remap;
    const int64_t src = A.query_src ? (int64_t)A.query_src[i] : (int64_t)i;
    if (src < 0 || src >= A.n_src_rows) return;
    const int64_t row = A.query_row[i];
    const int64_t slot = A.query_slot ? (int64_t)A.query_slot[i] : -1;
    if (threadIdx.x < HALF) cs[threadIdx.x] = rope_cs((double)A.query_pos[i], threadIdx.x, D, A.theta);
    __syncthreads();
    remap_rows<T, D, kThreads, kUnits, false, false>(A.k_cache, A.v_cache, A.row_stride, A.k_new,
                                                     A.v_new, kvw, src, row, 1, A.hkv,
                                                     A.n_src_rows, A.n_rows, cs, [] {});
    if (slot >= 0)
      remap_rows<T, D, kThreads, kUnits, false, false>(A.probe_k, A.probe_v, A.probe_stride,
                                                       A.k_new, A.v_new, kvw, src, slot, 1, A.hkv,
                                                       A.n_src_rows, A.n_probe, cs, [] {});
    // q: hq heads rotated into q_u[i]
    constexpr int VEC = Vec16<T>::N;
    constexpr int UPH = HALF / VEC;
    const T* qs = A.q_new + src * (int64_t)A.hq * D;
    T* qd = A.q_u + (int64_t)i * A.hq * D;
    for (int u = threadIdx.x; u < A.hq * UPH; u += kThreads) {
      const int h = u / UPH, j = (u - h * UPH) * VEC, off = h * D + j;
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Vec16<T>::unpack(ld16(qs + off), x1);
      Vec16<T>::unpack(ld16(qs + off + HALF), x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        rope_pair(x1[e], x2[e], cs[j + e], y1[e], y2[e]);
      }
      st16(qd + off, Vec16<T>::pack(y1));
      st16(qd + off + HALF, Vec16<T>::pack(y2));
    }
    return;
  }
  // ---- a tile of anchor slots: re-positioned straight from the stored chunk rows
  const int p0 = (bid - n_remap - A.n_query) * A.probe_rows_per_block;
  for (int pr = 0; pr < A.probe_rows_per_block; ++pr) {
    const int64_t p = p0 + pr;
    if (p >= A.n_probe) break;
    const int64_t src = A.probe_src[p];
    if (pr > 0) __syncthreads();  // the previous row's angle table is no longer read
    if (src < 0) continue;  // a query slot (written by that query row's block)
    if (threadIdx.x < HALF) cs[threadIdx.x] = rope_cs((double)A.probe_delta[p], threadIdx.x, D, A.theta);
    __syncthreads();
    remap_rows<T, D, kThreads, kUnits, false, false>(A.probe_k, A.probe_v, A.probe_stride,
                                                     A.k_pic, A.v_pic, A.pic_stride, src, p, 1,
                                                     A.hkv, A.n_pic_rows, A.n_probe, cs, [] {});
  }
}

template <typename T, int D>
hipError_t assemble_t(const AssembleShape& s, const AssemblePtrs& p, hipStream_t stream) {
  AssembleArgs<T, D> A;
  A.k_cache = static_cast<T*>(p.k_cache);
  A.v_cache = static_cast<T*>(p.v_cache);
  A.n_rows = s.n_rows;
  A.row_stride = s.row_stride;
  A.k_pic = static_cast<const T*>(p.k_pic);
  A.v_pic = static_cast<const T*>(p.v_pic);
  A.n_pic_rows = s.n_pic_rows;
  A.pic_stride = s.pic_row_stride;
  A.seg_start = p.seg_start;
  A.seg_len = p.seg_len;
  A.seg_delta = p.seg_delta;
  A.src_start = p.src_start;
  A.n_seg = s.n_seg;
  // rows per chunk tile: one round of kUnits key units per thread
  const int key_units_per_row = s.hkv * (D / 2) / Vec16<T>::N;
  A.rows_per_block = max(1, kThreads * kUnits / key_units_per_row);
  A.tiles_per_seg = (s.max_seg_len + A.rows_per_block - 1) / A.rows_per_block;
  A.k_new = static_cast<const T*>(p.k_new);
  A.v_new = static_cast<const T*>(p.v_new);
  A.q_new = static_cast<const T*>(p.q_new);
  A.q_u = static_cast<T*>(p.q_u);
  A.n_src_rows = s.n_src_rows;
  A.n_query = s.n_query;
  A.query_row = p.query_row;
  A.query_pos = p.query_pos;
  A.query_src = p.query_src;
  A.query_slot = p.query_slot;
  A.probe_k = static_cast<T*>(p.probe_k);
  A.probe_v = static_cast<T*>(p.probe_v);
  A.n_probe = s.n_probe;
  A.probe_stride = s.probe_row_stride;
  A.probe_src = p.probe_src;
  A.probe_delta = p.probe_delta;
  A.probe_rows_per_block = 1;  // one slot per block: its loads are the only round trip
  A.hq = s.hq;
  A.hkv = s.hkv;
  A.theta = s.theta;
  const int64_t n_remap = (int64_t)s.n_seg * A.tiles_per_seg;
  const int64_t n_probe_blocks = (s.n_probe + A.probe_rows_per_block - 1) / A.probe_rows_per_block;
  const int64_t blocks = n_remap + s.n_query + n_probe_blocks;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  // the stored chunk caches' K and V bytes
  const int64_t src_bytes = s.n_pic_rows * (int64_t)s.hkv * D * (int64_t)sizeof(T) * 2;
  if (src_bytes > kStreamSourceBytes)
    assemble_kernel<T, D, true><<<dim3((unsigned)blocks), kThreads, 0, stream>>>(A);
  else
    assemble_kernel<T, D, false><<<dim3((unsigned)blocks), kThreads, 0, stream>>>(A);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_assemble(const AssembleShape& s, const AssemblePtrs& p, hipStream_t stream) {
  if (s.bf16) return s.d == 64 ? assemble_t<uint16_t, 64>(s, p, stream) : assemble_t<uint16_t, 128>(s, p, stream);
  return s.d == 64 ? assemble_t<float, 64>(s, p, stream) : assemble_t<float, 128>(s, p, stream);
}

}  // namespace qcf
