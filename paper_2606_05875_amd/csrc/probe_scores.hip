// Per-token importance of a critical layer (eq. single_layer_importance) and
// its sum over the critical layers (eq. critical_layer_importance).
//
// I(t) = sum_{i,h} softmax_t(q_{i,h} . k_{t,g(h)} * scale) needs every query
// row's softmax denominator over all N context keys before any column can be
// summed, so the bf16 path runs in two passes over the keys:
//   stats   : grid (query tile, KV head x key split, request).  Each wave holds
//             32 query vectors of one KV-head group in registers, streams 64-key
//             tiles of K through LDS and keeps an online (max, sum) per row.
//   merge   : per query vector, combines the key splits -> (max, 1/sum).
//   columns : grid (128-key chunk, KV head, request).  Each wave keeps its 32
//             keys in registers, streams 64-row tiles of the group's queries
//             (and their stats) through LDS, recomputes the logits and
//             accumulates probabilities per key; one butterfly across the
//             wave's lanes finishes the per-key sums.
//   finish  : sums the KV-head partials in a fixed order and writes (or adds
//             to) the score vector.
// QK^T runs on the matrix cores as S^T = K Q^T with v_mfma_f32_32x32x16_bf16:
// A = 32 keys x 16 d (a 16-byte row slice of K per lane), B = 16 d x 32 query
// vectors (a 16-byte row slice of Q per lane).  The fp32 path uses the vector
// ALUs.  Every reduction has a fixed order, so results are deterministic.
#include <math.h>

#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kQvPerBlock = 128;  // stats pass: 4 waves x 32 query vectors
constexpr int kKeyTile = 64;      // stats pass K tile
constexpr int kKeysPerBlock = 128;  // column pass: 4 waves x 32 keys
constexpr int kQTile = 64;          // column pass Q tile

struct WsLayout {
  size_t part_off, stats_off, cols_off, total;
  int n_splits, keys_per_split, max_qv;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(const ProbeShape& s) {
  WsLayout w{};
  const int grp = s.hq / s.hkv;
  w.max_qv = s.max_q_len * grp;
  const int row_tiles = (w.max_qv + kQvPerBlock - 1) / kQvPerBlock;
  const int64_t blocks = (int64_t)row_tiles * s.hkv * s.batch;
  int want = (int)((1024 + blocks - 1) / (blocks > 0 ? blocks : 1));
  int cap = (s.max_ctx_len + 511) / 512;
  if (cap < 1) cap = 1;
  const int grid_cap = 65535 / (s.hkv > 0 ? s.hkv : 1);
  if (cap > grid_cap) cap = grid_cap;
  if (cap < 1) cap = 1;
  w.n_splits = want < 1 ? 1 : (want > cap ? cap : want);
  int kps = (s.max_ctx_len + w.n_splits - 1) / w.n_splits;
  w.keys_per_split = ((kps + kKeyTile - 1) / kKeyTile) * kKeyTile;
  if (w.keys_per_split == 0) w.keys_per_split = kKeyTile;
  const size_t nb = (size_t)s.batch * s.hkv;
  w.part_off = 0;
  w.stats_off = align256(nb * w.n_splits * w.max_qv * sizeof(float2));
  w.cols_off = w.stats_off + align256(nb * w.max_qv * sizeof(float2));
  w.total = w.cols_off + align256(nb * (size_t)s.max_ctx_len * sizeof(float));
  return w;
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float2 combine_ml(float2 a, float2 b) {
  const float m = fmaxf(a.x, b.x);
  if (m == -INFINITY) return make_float2(-INFINITY, 0.f);
  return make_float2(m, a.y * exp2f(a.x - m) + b.y * exp2f(b.x - m));
}

// ---------------------------------------------------------------- bf16 stats
template <int D>
__global__ __launch_bounds__(kThreads) void probe_stats_bf16(
    float2* __restrict__ part, const uint16_t* __restrict__ q, int64_t n_q_rows,
    const uint16_t* __restrict__ k, int64_t n_kv_rows, int64_t k_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
    const int32_t* __restrict__ ctx_len, int hq, int hkv, int lg, int n_splits,
    int keys_per_split, int max_qv, float scale2) {
  constexpr int KSTR = D + 8;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kKeyTile * KSTR];

  const int tile = blockIdx.x;
  const int g = blockIdx.y % hkv, split = blockIdx.y / hkv, b = blockIdx.z;
  const int64_t q0 = cu_q[b];
  const int nqv = (cu_q[b + 1] - (int)q0) << lg;
  if (tile * kQvPerBlock >= nqv) return;
  const int64_t k0 = cu_kv[b];
  const int N = ctx_len[b];
  const int key_lo = split * keys_per_split;
  const int key_hi = min(N, key_lo + keys_per_split);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int qv = tile * kQvPerBlock + 32 * w + lq;
  const int64_t qrow = q0 + (qv >> lg);
  const bool valid = qv < nqv && qv < max_qv && qrow < n_q_rows;
  const int head = g * (1 << lg) + (qv & ((1 << lg) - 1));

  bf16x8 qreg[D / 16];
  {
    const uint16_t* qp = q + qrow * (int64_t)hq * D + (int64_t)head * D + 8 * hi;
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      qreg[st] = as_bf16x8(valid ? ld16(qp + 16 * st) : make_uint4(0, 0, 0, 0));
  }
  float m = -INFINITY, ls = 0.f;
  constexpr int CPR = D / 8;  // 16-byte chunks per K row
  for (int kt0 = key_lo; kt0 < key_hi; kt0 += kKeyTile) {
    for (int c = threadIdx.x; c < kKeyTile * CPR; c += kThreads) {
      const int key = c / CPR, ch = c - key * CPR;
      const int64_t row = k0 + kt0 + key;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (kt0 + key < key_hi && row < n_kv_rows) v = ld16(k + row * k_stride + (int64_t)g * D + ch * 8);
      st16(&k_lds[key * KSTR + ch * 8], v);
    }
    __syncthreads();
    f32x16 s[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
      s[blk] = f32x16{};
#pragma unroll
      for (int st = 0; st < D / 16; ++st) {
        const bf16x8 a = as_bf16x8(ld16(&k_lds[(blk * 32 + lq) * KSTR + 8 * hi + 16 * st]));
        s[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[st], s[blk], 0, 0, 0);
      }
    }
    float mt = -INFINITY;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int key = kt0 + blk * 32 + 8 * (v >> 2) + 4 * hi + (v & 3);
        float x = s[blk][v] * scale2;
        if (key >= key_hi) x = -INFINITY;
        s[blk][v] = x;
        mt = fmaxf(mt, x);
      }
    const float mn = fmaxf(m, mt);
    if (mn != -INFINITY) {
      float acc = 0.f;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc += exp2f(s[blk][v] - mn);
      ls = ls * exp2f(m - mn) + acc;
      m = mn;
    }
    __syncthreads();
  }
  // lanes l and l^32 hold disjoint keys of the same query vector
  float2 ml = combine_ml(make_float2(m, ls), make_float2(__shfl_xor(m, 32, 64), __shfl_xor(ls, 32, 64)));
  if (valid && hi == 0)
    part[((int64_t)(b * hkv + g) * n_splits + split) * max_qv + qv] = ml;
}

// ---------------------------------------------------------------- merge
__global__ __launch_bounds__(kThreads) void probe_merge(const float2* __restrict__ part,
                                                        float2* __restrict__ stats,
                                                        const int32_t* __restrict__ cu_q, int hkv,
                                                        int lg, int n_splits, int max_qv) {
  const int qv = blockIdx.x * kThreads + threadIdx.x;
  const int g = blockIdx.y, b = blockIdx.z;
  const int nqv = (cu_q[b + 1] - cu_q[b]) << lg;
  if (qv >= nqv || qv >= max_qv) return;
  const float2* p = part + (int64_t)(b * hkv + g) * n_splits * max_qv + qv;
  float2 ml = make_float2(-INFINITY, 0.f);
  for (int s = 0; s < n_splits; ++s) ml = combine_ml(ml, p[(int64_t)s * max_qv]);
  stats[(int64_t)(b * hkv + g) * max_qv + qv] = make_float2(ml.x, ml.y > 0.f ? 1.f / ml.y : 0.f);
}

// ---------------------------------------------------------------- bf16 columns
template <int D>
__global__ __launch_bounds__(kThreads) void probe_cols_bf16(
    float* __restrict__ cols, const float2* __restrict__ stats, const uint16_t* __restrict__ q,
    int64_t n_q_rows, const uint16_t* __restrict__ k, int64_t n_kv_rows, int64_t k_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
    const int32_t* __restrict__ ctx_len, int hq, int hkv, int lg, int max_qv, int max_ctx,
    float scale2) {
  constexpr int QSTR = D + 8;
  __shared__ __attribute__((aligned(16))) uint16_t q_lds[kQTile * QSTR];
  __shared__ float2 st_lds[kQTile];

  const int g = blockIdx.y, b = blockIdx.z;
  const int N = ctx_len[b];
  const int kc0 = blockIdx.x * kKeysPerBlock;
  if (kc0 >= N) return;
  const int64_t q0 = cu_q[b];
  const int nqv = (cu_q[b + 1] - (int)q0) << lg;
  const int64_t k0 = cu_kv[b];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int kw = kc0 + 32 * w;

  bf16x8 kreg[D / 16];
  {
    const int key = kw + lq;
    const bool ok = key < N && k0 + key < n_kv_rows;
    const uint16_t* kp = k + (k0 + key) * k_stride + (int64_t)g * D + 8 * hi;
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      kreg[st] = as_bf16x8(ok ? ld16(kp + 16 * st) : make_uint4(0, 0, 0, 0));
  }
  const float2* stg = stats + (int64_t)(b * hkv + g) * max_qv;
  float col[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) col[v] = 0.f;

  constexpr int CPR = D / 8;
  for (int qt0 = 0; qt0 < nqv; qt0 += kQTile) {
    for (int c = threadIdx.x; c < kQTile * CPR; c += kThreads) {
      const int r = c / CPR, ch = c - r * CPR;
      const int qv = qt0 + r;
      const int64_t qrow = q0 + (qv >> lg);
      const int head = g * (1 << lg) + (qv & ((1 << lg) - 1));
      uint4 v = make_uint4(0, 0, 0, 0);
      if (qv < nqv && qrow < n_q_rows) v = ld16(q + qrow * (int64_t)hq * D + (int64_t)head * D + ch * 8);
      st16(&q_lds[r * QSTR + ch * 8], v);
    }
    if (threadIdx.x < kQTile) {
      const int qv = qt0 + threadIdx.x;
      st_lds[threadIdx.x] = (qv < nqv && qv < max_qv) ? stg[qv] : make_float2(0.f, 0.f);
    }
    __syncthreads();
#pragma unroll
    for (int sub = 0; sub < kQTile / 32; ++sub) {
      f32x16 s = f32x16{};
#pragma unroll
      for (int st = 0; st < D / 16; ++st) {
        const bf16x8 bq = as_bf16x8(ld16(&q_lds[(sub * 32 + lq) * QSTR + 8 * hi + 16 * st]));
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kreg[st], bq, s, 0, 0, 0);
      }
      const float2 ml = st_lds[sub * 32 + lq];  // (max, 1/sum); 1/sum == 0 for padding
#pragma unroll
      for (int v = 0; v < 16; ++v) col[v] += exp2f(s[v] * scale2 - ml.x) * ml.y;
    }
    __syncthreads();
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) col[v] += __shfl_xor(col[v], o, 64);
  }
  if (lq == 0) {
    float* cg = cols + (int64_t)(b * hkv + g) * max_ctx;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = kw + 8 * (v >> 2) + 4 * hi + (v & 3);
      if (key < N && key < max_ctx) cg[key] = col[v];
    }
  }
}

// ---------------------------------------------------------------- finish
__global__ __launch_bounds__(kThreads) void probe_finish(float* __restrict__ scores, int accumulate,
                                                         const float* __restrict__ cols,
                                                         const int32_t* __restrict__ cu_kv,
                                                         const int32_t* __restrict__ ctx_len,
                                                         int64_t n_kv_rows, int hkv, int max_ctx) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  const int b = blockIdx.y;
  if (t >= ctx_len[b] || t >= max_ctx) return;
  const int64_t row = (int64_t)cu_kv[b] + t;
  if (row >= n_kv_rows) return;
  float acc = 0.f;
  for (int g = 0; g < hkv; ++g) acc += cols[(int64_t)(b * hkv + g) * max_ctx + t];
  scores[row] = accumulate ? scores[row] + acc : acc;
}

// ---------------------------------------------------------------- fp32 path
template <int D>
__global__ __launch_bounds__(64) void probe_stats_f32(float2* __restrict__ stats,
                                                      const float* __restrict__ q, int64_t n_q_rows,
                                                      const float* __restrict__ k, int64_t n_kv_rows,
                                                      int64_t k_stride, const int32_t* __restrict__ cu_q,
                                                      const int32_t* __restrict__ cu_kv,
                                                      const int32_t* __restrict__ ctx_len, int hq,
                                                      int hkv, int max_q_len, float scale2) {
  __shared__ float qs[D];
  const int i = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int64_t q0 = cu_q[b];
  if (i >= cu_q[b + 1] - q0 || q0 + i >= n_q_rows) return;
  const int g = h / (hq / hkv);
  for (int e = threadIdx.x; e < D; e += 64) qs[e] = q[(q0 + i) * (int64_t)hq * D + (int64_t)h * D + e];
  __syncthreads();
  const int64_t k0 = cu_kv[b];
  const int N = ctx_len[b];
  float m = -INFINITY, ls = 0.f;
  for (int t = threadIdx.x; t < N; t += 64) {
    if (k0 + t >= n_kv_rows) break;
    const float* kp = k + (k0 + t) * k_stride + (int64_t)g * D;
    float acc = 0.f;
    for (int e = 0; e < D; ++e) acc += qs[e] * kp[e];
    const float x = acc * scale2;
    const float mn = fmaxf(m, x);
    ls = ls * exp2f(m - mn) + exp2f(x - mn);
    m = mn;
  }
  float2 ml = make_float2(m, ls);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
    ml = combine_ml(ml, make_float2(__shfl_xor(ml.x, o, 64), __shfl_xor(ml.y, o, 64)));
  if (threadIdx.x == 0)
    stats[((int64_t)b * hq + h) * max_q_len + i] = make_float2(ml.x, ml.y > 0.f ? 1.f / ml.y : 0.f);
}

template <int D>
__global__ __launch_bounds__(kThreads) void probe_cols_f32(
    float* __restrict__ scores, int accumulate, const float2* __restrict__ stats,
    const float* __restrict__ q, int64_t n_q_rows, const float* __restrict__ k, int64_t n_kv_rows,
    int64_t k_stride, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
    const int32_t* __restrict__ ctx_len, int hq, int hkv, int max_q_len, float scale2) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  const int b = blockIdx.y;
  const int N = ctx_len[b];
  const int64_t k0 = cu_kv[b];
  const bool ok = t < N && k0 + t < n_kv_rows;
  const int64_t q0 = cu_q[b];
  const int nq = cu_q[b + 1] - (int)q0;
  const int grp = hq / hkv;
  float acc = 0.f;
  float kr[D];
  for (int h = 0; h < hq; ++h) {
    if (h % grp == 0) {
      const int g = h / grp;
#pragma unroll
      for (int e = 0; e < D; ++e) kr[e] = ok ? k[(k0 + t) * k_stride + (int64_t)g * D + e] : 0.f;
    }
    for (int i = 0; i < nq && i < max_q_len; ++i) {
      if (q0 + i >= n_q_rows) break;
      const float* qp = q + (q0 + i) * (int64_t)hq * D + (int64_t)h * D;
      float dot = 0.f;
#pragma unroll
      for (int e = 0; e < D; ++e) dot += qp[e] * kr[e];
      const float2 ml = stats[((int64_t)b * hq + h) * max_q_len + i];
      acc += exp2f(dot * scale2 - ml.x) * ml.y;
    }
  }
  if (!ok) return;
  scores[k0 + t] = accumulate ? scores[k0 + t] + acc : acc;
}

}  // namespace

size_t probe_scores_workspace(const ProbeShape& s) {
  if (s.batch <= 0 || s.max_q_len <= 0 || s.max_ctx_len <= 0) return 256;
  const WsLayout w = ws_layout(s);
  const size_t f32 = align256((size_t)s.batch * s.hq * s.max_q_len * sizeof(float2));
  return w.total > f32 ? w.total : f32;
}

hipError_t launch_probe_scores(float* scores, int accumulate, const void* q, int64_t n_q_rows,
                               const void* k, int64_t n_kv_rows, int64_t k_row_stride,
                               bool bf16, const int32_t* cu_q, const int32_t* cu_kv,
                               const int32_t* ctx_len, const ProbeShape& s, float scale,
                               void* ws, hipStream_t stream) {
  if (s.batch == 0 || s.max_ctx_len == 0) return hipSuccess;
  const float scale2 = scale * kLog2e;
  int lg = 0;
  while ((1 << lg) < s.hq / s.hkv) ++lg;
  if (!bf16) {
    float2* stats = static_cast<float2*>(ws);
    if (s.max_q_len > 0) {
      dim3 g1(s.max_q_len, s.hq, s.batch);
      if (s.d == 64)
        probe_stats_f32<64><<<g1, 64, 0, stream>>>(stats, (const float*)q, n_q_rows, (const float*)k,
                                                   n_kv_rows, k_row_stride, cu_q, cu_kv, ctx_len,
                                                   s.hq, s.hkv, s.max_q_len, scale2);
      else
        probe_stats_f32<128><<<g1, 64, 0, stream>>>(stats, (const float*)q, n_q_rows, (const float*)k,
                                                    n_kv_rows, k_row_stride, cu_q, cu_kv, ctx_len,
                                                    s.hq, s.hkv, s.max_q_len, scale2);
    }
    dim3 g2((s.max_ctx_len + kThreads - 1) / kThreads, s.batch);
    if (s.d == 64)
      probe_cols_f32<64><<<g2, kThreads, 0, stream>>>(scores, accumulate, stats, (const float*)q,
                                                      n_q_rows, (const float*)k, n_kv_rows,
                                                      k_row_stride, cu_q, cu_kv, ctx_len, s.hq,
                                                      s.hkv, s.max_q_len, scale2);
    else
      probe_cols_f32<128><<<g2, kThreads, 0, stream>>>(scores, accumulate, stats, (const float*)q,
                                                       n_q_rows, (const float*)k, n_kv_rows,
                                                       k_row_stride, cu_q, cu_kv, ctx_len, s.hq,
                                                       s.hkv, s.max_q_len, scale2);
    return hipGetLastError();
  }
  const WsLayout w = ws_layout(s);
  char* base = static_cast<char*>(ws);
  float2* part = reinterpret_cast<float2*>(base + w.part_off);
  float2* stats = reinterpret_cast<float2*>(base + w.stats_off);
  float* cols = reinterpret_cast<float*>(base + w.cols_off);
  const uint16_t* qb = static_cast<const uint16_t*>(q);
  const uint16_t* kb = static_cast<const uint16_t*>(k);
  if (w.max_qv > 0) {
    dim3 ga((w.max_qv + kQvPerBlock - 1) / kQvPerBlock, s.hkv * w.n_splits, s.batch);
    if (s.d == 64)
      probe_stats_bf16<64><<<ga, kThreads, 0, stream>>>(part, qb, n_q_rows, kb, n_kv_rows,
                                                        k_row_stride, cu_q, cu_kv, ctx_len, s.hq,
                                                        s.hkv, lg, w.n_splits, w.keys_per_split,
                                                        w.max_qv, scale2);
    else
      probe_stats_bf16<128><<<ga, kThreads, 0, stream>>>(part, qb, n_q_rows, kb, n_kv_rows,
                                                         k_row_stride, cu_q, cu_kv, ctx_len, s.hq,
                                                         s.hkv, lg, w.n_splits, w.keys_per_split,
                                                         w.max_qv, scale2);
    dim3 gm((w.max_qv + kThreads - 1) / kThreads, s.hkv, s.batch);
    probe_merge<<<gm, kThreads, 0, stream>>>(part, stats, cu_q, s.hkv, lg, w.n_splits, w.max_qv);
  }
  dim3 gc((s.max_ctx_len + kKeysPerBlock - 1) / kKeysPerBlock, s.hkv, s.batch);
  if (s.d == 64)
    probe_cols_bf16<64><<<gc, kThreads, 0, stream>>>(cols, stats, qb, n_q_rows, kb, n_kv_rows,
                                                     k_row_stride, cu_q, cu_kv, ctx_len, s.hq,
                                                     s.hkv, lg, w.max_qv, s.max_ctx_len, scale2);
  else
    probe_cols_bf16<128><<<gc, kThreads, 0, stream>>>(cols, stats, qb, n_q_rows, kb, n_kv_rows,
                                                      k_row_stride, cu_q, cu_kv, ctx_len, s.hq,
                                                      s.hkv, lg, w.max_qv, s.max_ctx_len, scale2);
  dim3 gf((s.max_ctx_len + kThreads - 1) / kThreads, s.batch);
  probe_finish<<<gf, kThreads, 0, stream>>>(scores, accumulate, cols, cu_kv, ctx_len, n_kv_rows,
                                            s.hkv, s.max_ctx_len);
  return hipGetLastError();
}

}  // namespace qcf
