// Row remapping shared by the re-positioning kernels (eq. pic_online): rows of
// hkv rotated keys and, optionally, their values, moved from a source layout
// to a destination layout.
#pragma once
#include "qcf_device.h"

namespace qcf {

// Rotate `nrows` rows (source rows s0.., destination rows d0..) of hkv heads by
// the angle table cs and copy their values alongside when vdst is set; rows
// outside the bounds are skipped.  A round covers kUnits key units
// (rotate-half pairs) and 2 kUnits value units per thread, and all of its loads
// are issued, unmasked from clamped rows, before anything waits: a load under a
// lane condition gets a wait of its own, which would serialise the round trips.
// make_cs() fills cs (and synchronises the block) once, after the first round's
// loads are in flight, so the float64 angle work overlaps them; every thread of
// the block must call this function with the same nrows.  A unit is read and
// written by the same thread, so in-place calls (same buffers, same rows) are
// safe.  kStreamIn reads the sources with the non-temporal hint; kStreamV writes
// the values with it (the recompute that reads them next hides its load latency).
template <typename T, int D, int kThreads, int kUnits, bool kStreamIn, bool kStreamV,
          typename MakeCs>
__device__ __forceinline__ void remap_rows(T* kdst, T* vdst, int64_t dst_stride, const T* ksrc,
                                           const T* vsrc, int64_t src_stride, int64_t s0,
                                           int64_t d0, int nrows, int hkv, int64_t n_src,
                                           int64_t n_dst, const float2* cs, MakeCs make_cs) {
  constexpr int HALF = D / 2;
  constexpr int VEC = Vec16<T>::N;
  constexpr int UPH = HALF / VEC;
  const int upr = hkv * UPH;  // key units per row (rotate-half pairs)
  const int vpr = 2 * upr;    // value units per row
  const int64_t s_hi = n_src - 1;
  const int total_k = nrows * upr, total_v = vdst ? nrows * vpr : 0;
  bool first = true;
  for (int kb = 0, vb = 0; kb < total_k || vb < total_v;
       kb += kThreads * kUnits, vb += 2 * kThreads * kUnits) {
    uint4 a[kUnits], b[kUnits], va[2 * kUnits];
    int64_t kofs[kUnits], vofs[2 * kUnits];
    int jj[kUnits];
    bool kok[kUnits], vok[2 * kUnits];
#pragma unroll
    for (int k = 0; k < kUnits; ++k) {
      const int u = kb + threadIdx.x + k * kThreads;
      const int uc = min(u, max(total_k - 1, 0));
      const int r = uc / upr, c = uc - r * upr;
      const int h = c / UPH;
      const int64_t s = s0 + r, d = d0 + r;
      kok[k] = u < total_k && s >= 0 && s < n_src && d >= 0 && d < n_dst;
      jj[k] = (c - h * UPH) * VEC;
      const int64_t so = min(max(s, (int64_t)0), s_hi) * src_stride + (int64_t)h * D + jj[k];
      kofs[k] = d * dst_stride + (int64_t)h * D + jj[k];
      a[k] = kStreamIn ? ld16_nt(ksrc + so) : ld16(ksrc + so);
      b[k] = kStreamIn ? ld16_nt(ksrc + so + HALF) : ld16(ksrc + so + HALF);
    }
    if (vdst) {
#pragma unroll
      for (int k = 0; k < 2 * kUnits; ++k) {
        const int u = vb + threadIdx.x + k * kThreads;
        const int uc = min(u, max(total_v - 1, 0));
        const int r = uc / vpr, c = uc - r * vpr;
        const int64_t s = s0 + r, d = d0 + r;
        vok[k] = u < total_v && s >= 0 && s < n_src && d >= 0 && d < n_dst;
        vofs[k] = d * dst_stride + (int64_t)c * VEC;
        const T* vp = vsrc + min(max(s, (int64_t)0), s_hi) * src_stride + (int64_t)c * VEC;
        va[k] = kStreamIn ? ld16_nt(vp) : ld16(vp);
      }
    }
    if (first) {
      make_cs();
      first = false;
    }
#pragma unroll
    for (int k = 0; k < kUnits; ++k) {
      float x1[VEC], x2[VEC], y1[VEC], y2[VEC];
      Vec16<T>::unpack(a[k], x1);
      Vec16<T>::unpack(b[k], x2);
#pragma unroll
      for (int e = 0; e < VEC; ++e) rope_pair(x1[e], x2[e], cs[jj[k] + e], y1[e], y2[e]);
      if (kok[k]) {
        st16(kdst + kofs[k], Vec16<T>::pack(y1));
        st16(kdst + kofs[k] + HALF, Vec16<T>::pack(y2));
      }
    }
    if (vdst) {
#pragma unroll
      for (int k = 0; k < 2 * kUnits; ++k)
        if (vok[k]) {
          if (kStreamV) st16_nt(vdst + vofs[k], va[k]);
          else st16(vdst + vofs[k], va[k]);
        }
    }
  }
}

}  // namespace qcf
