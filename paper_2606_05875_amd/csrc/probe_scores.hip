// Per-token importance of a critical layer (eq. single_layer_importance) and
// its sum over the critical layers (eq. critical_layer_importance).
//
// I(t) = sum_{i,h} softmax_t(q_{i,h} . k_{t,g(h)} * scale) needs every query
// row's softmax denominator over all N context keys before any column can be
// summed, so the bf16 path runs in two launches:
//   stats   : grid (128-query-vector tile, KV head x key split, request), at
//             most 16 key splits.  Each wave holds 32 query vectors of one
//             KV-head group in registers; the split's keys pass through LDS in
//             128-key sub-tiles (the next one prefetched into registers while
//             the current one is in use) and every row keeps an online
//             (max, sum); the split's base-2 log-sum-exp is written.  The
//             first split's blocks also store their Q registers in MFMA
//             operand order, so the column pass reads them contiguously.
//   columns : grid (32-key chunk, request).  The block's eight waves share out
//             the (KV head, 32-query-vector) items of the request, one head at
//             a time per wave; for each item a wave merges the query vectors'
//             split log-sum-exps in a fixed order, recomputes the logits
//             against its keys (held in registers per head) and adds the
//             probabilities 2^(logit - lse) per key.  The waves' per-key sums are added in wave order in LDS and
//             written (or added) to the scores.
// No block waits for another: the two launches are the only global
// synchronisation.  QK^T runs on the matrix cores as S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16: A = 32 keys x 16 d (a 16-byte row slice of K per
// lane), B = 16 d x 32 query vectors (a 16-byte row slice of Q per lane).  The
// fp32 path uses the vector ALUs.  Every reduction has a fixed order, so
// results are deterministic.
#include <math.h>

#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kQvPerBlock = 128;  // stats pass: 4 waves x 32 query vectors
constexpr int kSubKeys = 128;     // stats pass: keys per LDS sub-tile
constexpr int kMaxSplits = 16;    // stats pass: key splits per query tile
constexpr int kColKeys = 32;      // column pass: keys per block

struct WsLayout {
  size_t part_off, frag_off, total;
  int n_splits, n_sub, max_qv, n_qt;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(const ProbeShape& s) {
  WsLayout w{};
  const int grp = s.hq / s.hkv;
  w.max_qv = s.max_q_len * grp;
  w.n_qt = (w.max_qv + kQvPerBlock - 1) / kQvPerBlock;
  const int sub_tiles = (s.max_ctx_len + kSubKeys - 1) / kSubKeys;
  w.n_sub = (sub_tiles + kMaxSplits - 1) / kMaxSplits;
  if (w.n_sub < 1) w.n_sub = 1;
  w.n_splits = (sub_tiles + w.n_sub - 1) / w.n_sub;
  if (w.n_splits < 1) w.n_splits = 1;
  const size_t nb = (size_t)s.batch * s.hkv;
  w.part_off = 0;
  w.frag_off = align256(nb * w.n_splits * w.max_qv * sizeof(float));
  // Q in MFMA B-fragment order: per (request, head, 32-vector item, 16-wide k
  // step), the 64 lanes' 16-byte slices back to back
  w.total = w.frag_off + nb * (size_t)w.n_qt * 4 * (s.d / 16) * 64 * 16;
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
    float* __restrict__ part, uint16_t* __restrict__ qfrag, const uint16_t* __restrict__ q,
    int64_t n_q_rows,
    const uint16_t* __restrict__ k, int64_t n_kv_rows, int64_t k_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
    const int32_t* __restrict__ ctx_len, int hq, int hkv, int lg, int n_splits, int n_sub,
    int max_qv, float scale2) {
  constexpr int KSTR = D + 8;
  constexpr int CPR = D / 8;                        // 16-byte chunks per K row
  constexpr int PER = kSubKeys * CPR / kThreads;    // chunks per thread per sub-tile
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kSubKeys * KSTR];

  const int tile = blockIdx.x;
  const int g = blockIdx.y % hkv, split = blockIdx.y / hkv, b = blockIdx.z;
  const int64_t q0 = cu_q[b];
  const int nqv = min((cu_q[b + 1] - (int)q0) << lg, max_qv);
  if (tile * kQvPerBlock >= nqv) return;
  const int64_t k0 = cu_kv[b];
  const int N = ctx_len[b];
  const int key_lo = split * n_sub * kSubKeys;
  const int key_hi = min(N, key_lo + n_sub * kSubKeys);
  const int n_here = key_hi > key_lo ? (key_hi - key_lo + kSubKeys - 1) / kSubKeys : 0;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int qv = tile * kQvPerBlock + 32 * w + lq;
  const int64_t qrow = q0 + (qv >> lg);
  const bool valid = qv < nqv && qrow < n_q_rows;
  const int head = g * (1 << lg) + (qv & ((1 << lg) - 1));

  uint4 buf[PER];
  auto fetch = [&](int sub) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * kThreads;
      const int key = key_lo + sub * kSubKeys + c / CPR, ch = c % CPR;
      const int64_t row = k0 + key;
      buf[i] = (key < key_hi && row < n_kv_rows) ? ld16(k + row * k_stride + (int64_t)g * D + ch * 8)
                                                 : make_uint4(0, 0, 0, 0);
    }
  };
  if (n_here > 0) fetch(0);
  bf16x8 qreg[D / 16];
  {
    const uint16_t* qp = q + qrow * (int64_t)hq * D + (int64_t)head * D + 8 * hi;
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      qreg[st] = as_bf16x8(valid ? ld16(qp + 16 * st) : make_uint4(0, 0, 0, 0));
  }
  if (split == 0) {  // one block per (tile, head, request) stores the fragments
    const int item = tile * 4 + w;
    uint16_t* fp = qfrag + ((((int64_t)(b * hkv + g) * gridDim.x * 4 + item) * (D / 16)) * 64 + l) * 8;
#pragma unroll
    for (int st = 0; st < D / 16; ++st) st16(fp + st * 64 * 8, __builtin_bit_cast(uint4, qreg[st]));
  }
  float m = -INFINITY, ls = 0.f;
  for (int sub = 0; sub < n_here; ++sub) {
    if (sub > 0) __syncthreads();  // the previous sub-tile is no longer read
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = threadIdx.x + i * kThreads;
      st16(&k_lds[(c / CPR) * KSTR + (c % CPR) * 8], buf[i]);
    }
    __syncthreads();
    if (sub + 1 < n_here) fetch(sub + 1);  // in flight during this sub-tile's work
    // two halves of 64 keys, each folded into the running (max, sum); logits are
    // scaled into the log2 domain, masked only in the split's last sub-tile
    const bool tail = key_lo + (sub + 1) * kSubKeys > key_hi;
#pragma unroll
    for (int half = 0; half < kSubKeys / 64; ++half) {
      const int kt0 = key_lo + sub * kSubKeys + half * 64;
      f32x16 sacc[2];
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        sacc[blk] = f32x16{};
#pragma unroll
        for (int st = 0; st < D / 16; ++st) {
          const bf16x8 a =
              as_bf16x8(ld16(&k_lds[(half * 64 + blk * 32 + lq) * KSTR + 8 * hi + 16 * st]));
          sacc[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[st], sacc[blk], 0, 0, 0);
        }
      }
      if (tail) {
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (kt0 + blk * 32 + 8 * (v >> 2) + 4 * hi + (v & 3) >= key_hi) sacc[blk][v] = -INFINITY;
      }
      float mt = -INFINITY;
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[blk][v]);
      const float mn = fmaxf(m, mt * scale2);
      if (mn != -INFINITY) {
        float acc = 0.f;
#pragma unroll
        for (int blk = 0; blk < 2; ++blk)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc += __builtin_amdgcn_exp2f(fmaf(sacc[blk][v], scale2, -mn));
        ls = ls * __builtin_amdgcn_exp2f(m - mn) + acc;
        m = mn;
      }
    }
  }
  // lanes l and l^32 hold disjoint keys of the same query vector; the split's
  // base-2 log-sum-exp log2(sum_t 2^(logit_t)) = max + log2(sum) (-inf: no keys)
  const float2 ml = combine_ml(make_float2(m, ls), make_float2(__shfl_xor(m, 32, 64), __shfl_xor(ls, 32, 64)));
  if (valid && hi == 0)
    part[((int64_t)(b * hkv + g) * n_splits + split) * max_qv + qv] =
        ml.y > 0.f ? ml.x + __builtin_amdgcn_logf(ml.y) : -INFINITY;
}

// ---------------------------------------------------------------- bf16 columns
constexpr int kColWaves = 8;

// Operands of one (KV head, 32-query-vector) item of the column pass: the Q
// slice (B operand) of the lane's query vector and its per-split log-sum-exps
// (even splits in lanes 0-31, odd splits in lanes 32-63).
template <int D>
struct ColItem {
  bf16x8 q[D / 16];
  float p[kMaxSplits / 2];
  bool live;
};

template <int D>
__global__ __launch_bounds__(kColWaves * 64) void probe_cols_bf16(
    float* __restrict__ scores, int accumulate, const float* __restrict__ part,
    const uint16_t* __restrict__ qfrag, int n_items_max, int64_t n_q_rows,
    const uint16_t* __restrict__ k, int64_t n_kv_rows, int64_t k_stride,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
    const int32_t* __restrict__ ctx_len, int hkv, int lg, int n_splits, int max_qv,
    float scale2) {
  __shared__ float red[kColWaves][kColKeys];
  const int chunk = blockIdx.x, b = blockIdx.y;
  const int N = ctx_len[b];
  const int kc0 = chunk * kColKeys;
  const int64_t k0 = cu_kv[b];
  if (kc0 >= N || k0 + kc0 >= n_kv_rows) return;
  const int64_t q0 = cu_q[b];
  // query vectors whose rows exist (the rest of a 32-wide item is padding)
  const int nqv = min(min((cu_q[b + 1] - (int)q0) << lg, max_qv), (int)max<int64_t>(0, n_q_rows - q0) << lg);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int nsub = (nqv + 31) >> 5;
  // waves per KV head (heads beyond the waves are taken in turns), and this
  // wave's share of the head's 32-query-vector items
  const int wpg = hkv >= kColWaves ? 1 : kColWaves / hkv;
  const int spw = (nsub + wpg - 1) / wpg;
  const int part_w = w % wpg;
  const int s0 = part_w * spw, s1 = min(nsub, s0 + spw);
  // keys past the context (or the tensor) read the last real row; their sums are dropped
  const int64_t krow = min(k0 + min(kc0 + lq, N - 1), n_kv_rows - 1);

  float col[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) col[v] = 0.f;

  if (w < hkv * wpg && s0 < s1) {
    for (int g = w / wpg; g < hkv; g += kColWaves / wpg) {
      bf16x8 kreg[D / 16];
      {
        const uint16_t* kp = k + krow * k_stride + (int64_t)g * D + 8 * hi;
#pragma unroll
        for (int st = 0; st < D / 16; ++st) kreg[st] = as_bf16x8(ld16(kp + 16 * st));
      }
      const float* pg = part + ((int64_t)(b * hkv + g) * n_splits) * max_qv;
      const uint16_t* fg = qfrag + (int64_t)(b * hkv + g) * n_items_max * (D / 16) * 64 * 8 + l * 8;
      // every load below is unconditional (indices clamped), so the hardware's
      // in-order load counter lets two items stay in flight while one is used
      auto load_item = [&](int sub, ColItem<D>& c) {
        const int qv_raw = sub * 32 + lq;
        c.live = sub < s1 && qv_raw < nqv;
        const int qv = min(qv_raw, nqv - 1);
        const uint16_t* fp = fg + (int64_t)min(sub, nsub - 1) * (D / 16) * 64 * 8;
#pragma unroll
        for (int st = 0; st < D / 16; ++st) c.q[st] = as_bf16x8(ld16(fp + st * 64 * 8));
#pragma unroll
        for (int j = 0; j < kMaxSplits / 2; ++j)
          c.p[j] = pg[(int64_t)min(2 * j + hi, n_splits - 1) * max_qv + qv];
      };
      auto use_item = [&](const ColItem<D>& c) {
        // the query vector's log-sum-exp over all keys from the splits', in a
        // fixed order: global max, then the even and odd splits' sums (lanes
        // 0-31 / 32-63), even + odd; copies past the last split are masked
        float pv[kMaxSplits / 2];
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < kMaxSplits / 2; ++j) {
          pv[j] = 2 * j + hi < n_splits ? c.p[j] : -INFINITY;
          mx = fmaxf(mx, pv[j]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        float ls = 0.f;
        if (mx != -INFINITY) {
#pragma unroll
          for (int j = 0; j < kMaxSplits / 2; ++j) ls += __builtin_amdgcn_exp2f(pv[j] - mx);
        }
        const float lo = __shfl_xor(ls, 32, 64);
        const float lsum = hi == 0 ? ls + lo : lo + ls;
        // padding (and a request without keys) get a reference that sends every
        // exponential to 0
        const float lse = (c.live && lsum > 0.f) ? mx + __builtin_amdgcn_logf(lsum) : 1e30f;
        f32x16 sacc = f32x16{};
#pragma unroll
        for (int st = 0; st < D / 16; ++st)
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kreg[st], c.q[st], sacc, 0, 0, 0);
        // S^T layout: value v of this lane is key 8(v>>2)+4hi+(v&3) of query vector
        // lq, whose log-sum-exp this lane holds: probability = 2^(logit - lse)
#pragma unroll
        for (int v = 0; v < 16; ++v) col[v] += __builtin_amdgcn_exp2f(fmaf(sacc[v], scale2, -lse));
      };
      ColItem<D> ca, cb, cc;
      load_item(s0, ca);
      load_item(s0 + 1, cb);
      for (int sub = s0; sub < s1; sub += 3) {
        load_item(sub + 2, cc);
        use_item(ca);
        load_item(sub + 3, ca);
        if (sub + 1 < s1) use_item(cb);
        load_item(sub + 4, cb);
        if (sub + 2 < s1) use_item(cc);
      }
    }
  }
  // per-key sums over the wave's 32 query-vector columns (lanes with the same hi)
#pragma unroll
  for (int v = 0; v < 16; ++v) {
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) col[v] += __shfl_xor(col[v], o, 64);
  }
  if (lq == 0) {
#pragma unroll
    for (int v = 0; v < 16; ++v) red[w][8 * (v >> 2) + 4 * hi + (v & 3)] = col[v];
  }
  __syncthreads();
  if (threadIdx.x < kColKeys) {
    const int t = kc0 + threadIdx.x;
    const int64_t row = k0 + t;
    if (t < N && row < n_kv_rows) {
      float acc = 0.f;
#pragma unroll
      for (int ww = 0; ww < kColWaves; ++ww) acc += red[ww][threadIdx.x];
      scores[row] = accumulate ? scores[row] + acc : acc;
    }
  }
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
  if ((int64_t)s.hkv * w.n_splits > 65535) return hipErrorInvalidConfiguration;
  float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + w.part_off);
  uint16_t* qfrag = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + w.frag_off);
  const uint16_t* qb = static_cast<const uint16_t*>(q);
  const uint16_t* kb = static_cast<const uint16_t*>(k);
  if (w.max_qv > 0) {
    dim3 ga(w.n_qt, s.hkv * w.n_splits, s.batch);
#define QCF_STATS(D)                                                                             \
  probe_stats_bf16<D><<<ga, kThreads, 0, stream>>>(part, qfrag, qb, n_q_rows, kb, n_kv_rows,     \
                                                   k_row_stride, cu_q, cu_kv, ctx_len, s.hq,     \
                                                   s.hkv, lg, w.n_splits, w.n_sub, w.max_qv, scale2)
    if (s.d == 64) QCF_STATS(64); else QCF_STATS(128);
#undef QCF_STATS
  }
  dim3 gc((s.max_ctx_len + kColKeys - 1) / kColKeys, s.batch);
#define QCF_COLS(D)                                                                             \
  probe_cols_bf16<D><<<gc, kColWaves * 64, 0, stream>>>(scores, accumulate, part, qfrag,       \
                                                  w.n_qt * 4, n_q_rows, kb, n_kv_rows,           \
                                                  k_row_stride, cu_q, cu_kv, ctx_len, s.hkv, lg,  \
                                                  w.n_splits, w.max_qv, scale2)
  if (s.d == 64) QCF_COLS(64); else QCF_COLS(128);
#undef QCF_COLS
  return hipGetLastError();
}

}  // namespace qcf
