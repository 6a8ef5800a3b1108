// Per-token importance of a critical layer (eq. single_layer_importance) and
// its sum over the critical layers (eq. critical_layer_importance).
//
// I(t) = sum_{i,h} softmax_t(q_{i,h} . k_{t,g(h)} * scale) needs every query
// row's softmax denominator over all N context keys before any column can be
// summed, so the bf16 path runs in three launches over the same grid of
// (KV head, 256-query-vector tile, key split, request) blocks, the head
// fastest, with the splits chosen for about 512 blocks:
//   stats   : each of the 8 waves holds 32 query vectors of one KV-head group
//             in registers; the split's keys pass through LDS (128 at a time,
//             the next ones prefetched into registers) in 32-key products,
//             and every vector keeps an online (max, sum); the split's base-2
//             log-sum-exp is written.
//   columns : the same tiles again.  Each vector's log-sum-exp over all splits
//             is merged once per block (its partials loaded together, folded
//             in split order); the logits are recomputed and each key's
//             probabilities 2^(logit - lse) summed over the tile's vectors
//             into a per-(head, tile) column buffer.
//   final   : scores[t] (+)= those column sums in (head, tile) order.
// Every block issues its loads together and waits once per K chunk: on this
// part a dependent round trip to memory costs microseconds under load.
// No block waits for another: the launches are the only global
// synchronisation.  QK^T runs on the matrix cores (v_mfma_f32_32x32x16_bf16)
// with the same operand registers either way round: the statistics take S^T =
// K Q^T (a lane owns one query vector, so its max and sum stay in the lane),
// the columns take S = Q K^T (a lane owns one key, so its sum over the query
// vectors is 16 in-lane additions and one lane swap).  The fp32 path uses the
// vector ALUs.  Every reduction has a fixed order, so results are
// deterministic.
//
// With a rotation table (kRot) the keys come from the stored chunk caches and
// each is moved to its request offset on the fly (eq. pic_online): a thread
// loads rotate-half piece pairs of a key, turns them by the key's table row in
// float32 and rounds to bf16 before the LDS store -- the very bits a stored
// re-positioned key has -- so no re-positioned copy is read or waited for.
#include <math.h>

#include <algorithm>

#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;      // fp32 path, final pass
constexpr int kW = 8;              // bf16 path: waves per block
constexpr int kQvTile = 32 * kW;   // query vectors per block
constexpr int kChunkKeys = 128;    // keys staged in LDS at a time
constexpr int kMaxSplits = 64;     // key splits per query tile
constexpr int kPassBlocks = 512;   // blocks aimed for when choosing the splits
constexpr int kCUs = 256;          // compute units of MI355X

struct WsLayout {
  size_t part_off, col_off, total;
  int n_qt, n_splits, split_keys, max_qv;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(const ProbeShape& s) {
  WsLayout w{};
  const int grp = s.hq / s.hkv;
  w.max_qv = s.max_q_len * grp;
  w.n_qt = (w.max_qv + kQvTile - 1) / kQvTile;
  // key splits of whole 32-key groups, about kPassBlocks blocks per pass -- or half as
  // many when rounding the splits to 32 keys would leave more of the last round of
  // kCUs-block slots idle (blocks of equal work then finish together)
  const int64_t per_split = (int64_t)std::max(1, w.n_qt) * s.hkv * std::max(1, s.batch);
  const int ctx = std::max(1, s.max_ctx_len);
  auto splits_for = [&](int64_t target, int& keys) {
    const int want = (int)std::min<int64_t>(
        kMaxSplits, std::max<int64_t>(1, (target + per_split - 1) / per_split));
    keys = ((ctx + want - 1) / want + 31) / 32 * 32;
    return (ctx + keys - 1) / keys;
  };
  auto idle = [&](int splits) {
    const int64_t blocks = per_split * splits;
    return (double)(((blocks + kCUs - 1) / kCUs) * kCUs - blocks) / (double)blocks;
  };
  int keys_a = 0, keys_b = 0;
  // a batch aims at four times as many blocks: the splits are cut from the longest context,
  // so shorter requests leave splits empty, and shorter splits even out the busy blocks
  // (ragged 16-request batch: scores + selection 0.34 -> 0.30 ms)
  const int64_t target = (int64_t)kPassBlocks * (s.batch > 1 ? 4 : 1);
  const int sa = splits_for(target, keys_a), sb = splits_for(target / 2, keys_b);
  const bool half = idle(sb) < idle(sa);
  w.split_keys = half ? keys_b : keys_a;
  w.n_splits = half ? sb : sa;
  const size_t nb = (size_t)s.batch * s.hkv;
  // both regions grow with the shape (the split region is sized for the most
  // splits), so a workspace sized for one call serves any smaller one
  w.part_off = 0;
  w.col_off = align256(nb * kMaxSplits * w.max_qv * sizeof(float));
  w.total = w.col_off + align256(nb * (size_t)w.n_qt * s.max_ctx_len * sizeof(float));
  return w;
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ float2 combine_ml(float2 a, float2 b) {
  const float m = fmaxf(a.x, b.x);
  if (m == -INFINITY) return make_float2(-INFINITY, 0.f);
  return make_float2(m, a.y * exp2f(a.x - m) + b.y * exp2f(b.x - m));
}

// ---------------------------------------------------------------- bf16 passes
template <int D, bool kCols, bool kRot>
__global__ __launch_bounds__(kW * 64) void scores_pass_bf16(
    float* __restrict__ part, float* __restrict__ colp, const uint16_t* __restrict__ q,
    int64_t n_q_rows, const uint16_t* __restrict__ k, int64_t n_kv_rows, int64_t k_stride,
    const int32_t* __restrict__ key_rot, const float2* __restrict__ rot_tab, int n_rot,
    const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
    const int32_t* __restrict__ ctx_len, int hq, int hkv, int lg, int n_qt, int n_splits,
    int split_keys, int max_qv, int max_ctx, float scale2) {
  constexpr int KSTR = D + 8;                          // padded LDS row (conflict-free reads)
  constexpr int CPR = D / 8;                           // 16-byte pieces per K row
  constexpr int PER = kChunkKeys * CPR / (kW * 64);    // pieces per thread per chunk
  constexpr int SPL = kMaxSplits / 2;                  // splits per lane in the merge
  constexpr int HP = CPR / 2;                          // 16-byte pieces per rotate-half
  constexpr int PU = PER / 2;                          // piece pairs per thread per chunk
  static_assert(PER % 2 == 0, "rotation works on whole piece pairs");
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kChunkKeys * KSTR];
  __shared__ float lse_l[kCols ? kQvTile : 1];
  __shared__ float red[kCols ? kW : 1][kCols ? kChunkKeys : 1];

  // block -> (KV head, query tile, split, request) with the head fastest:
  // blocks are dealt to the XCDs in turn, so with 8 KV heads every block of a
  // head runs on one XCD and its Q and split statistics are shared in that L2
  const int g = blockIdx.x % hkv;
  const int rest = blockIdx.x / hkv;
  const int qt = rest % n_qt, split = (rest / n_qt) % n_splits, b = rest / (n_qt * n_splits);
  const int64_t q0 = cu_q[b];
  const int nqv = min((cu_q[b + 1] - (int)q0) << lg, max_qv);
  if (qt * kQvTile >= nqv) return;
  const int64_t k0 = cu_kv[b];
  const int N = ctx_len[b];
  const int key_lo = split * split_keys;
  const int key_hi = min(N, key_lo + split_keys);
  if (kCols && key_lo >= key_hi) return;  // no keys: no columns (an empty split's statistics are still written)
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int qv = qt * kQvTile + 32 * w + lq;
  const int64_t qrow = q0 + (qv >> lg);
  const bool valid = qv < nqv && qrow < n_q_rows;
  const bool live = __ballot(valid) != 0;  // the wave has a real query vector
  const int head = g * (1 << lg) + (qv & ((1 << lg) - 1));

  // Every load below is unconditional, its indices clamped to real rows: a
  // load under a lane condition gets a wait of its own, which serialises the
  // round trips.  Keys past the split and query vectors past the tile are
  // masked where their products are used, so the rows read for them only
  // have to be finite.
  uint4 buf[PER];
  // with kRot a thread owns piece pairs (j .. j+7, j+D/2 .. j+D/2+7) of a key,
  // and the key's rotation-table row is loaded ahead of its pieces, so its
  // (cos, sin) can be fetched (fetch_cs) while the pieces are still in flight
  int rot_i[kRot ? PU : 1];
  uint4 csv[kRot ? 4 * PU : 1];
  auto fetch = [&](int c0) {
    if constexpr (kRot) {
      int64_t rows[PU];
#pragma unroll
      for (int i = 0; i < PU; ++i) {
        const int c = threadIdx.x + i * kW * 64;
        rows[i] = min(k0 + min(c0 + c / HP, key_hi - 1), n_kv_rows - 1);
        rot_i[i] = key_rot[rows[i]];
      }
#pragma unroll
      for (int i = 0; i < PU; ++i) {
        const int ch = (threadIdx.x + i * kW * 64) % HP;
        const uint16_t* kp = k + rows[i] * k_stride + (int64_t)g * D + ch * 8;
        buf[2 * i] = ld16(kp);
        buf[2 * i + 1] = ld16(kp + D / 2);
      }
    } else {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int c = threadIdx.x + i * kW * 64;
        const int key = min(c0 + c / CPR, key_hi - 1), ch = c % CPR;
        const int64_t row = min(k0 + key, n_kv_rows - 1);
        buf[i] = ld16(k + row * k_stride + (int64_t)g * D + ch * 8);
      }
    }
  };
  auto fetch_cs = [&]() {
    if constexpr (kRot) {
#pragma unroll
      for (int i = 0; i < PU; ++i) {
        const int ch = (threadIdx.x + i * kW * 64) % HP;
        const float2* cp = rot_tab + (int64_t)min(max(rot_i[i], 0), n_rot - 1) * (D / 2) + ch * 8;
#pragma unroll
        for (int v = 0; v < 4; ++v) csv[4 * i + v] = ld16(cp + 2 * v);
      }
    }
  };
  if (key_lo < key_hi) fetch(key_lo);
  bf16x8 qreg[D / 16];
  {
    const uint16_t* qp = q + min(qrow, n_q_rows - 1) * (int64_t)hq * D + (int64_t)head * D + 8 * hi;
#pragma unroll
    for (int st = 0; st < D / 16; ++st) qreg[st] = as_bf16x8(ld16(qp + 16 * st));
  }
  if (kRot && key_lo < key_hi) fetch_cs();
  float lse_v[kCols ? 16 : 1];
  if (kCols) {
    // the vector's base-2 log-sum-exp over every split: lanes l (even splits)
    // and l^32 (odd splits) fold theirs in split order, then even + odd; its
    // padding rows get a reference that sends every exponential to 0
    // (branch-free, so every load is issued before the first one is used;
    // an empty split's -inf and a masked slot count as a floor with weight 0)
    const float* pg = part + (int64_t)(b * hkv + g) * n_splits * max_qv + min(qv, max_qv - 1);
    float x[SPL];
#pragma unroll
    for (int j = 0; j < SPL; ++j) x[j] = pg[min(2 * j + hi, n_splits - 1) * max_qv];
    asm volatile("" ::: "memory");  // all of them in flight before the first is used
    constexpr float kFloor = -1e30f;
    float mx = kFloor, ls = 0.f;
#pragma unroll
    for (int j = 0; j < SPL; ++j) {
      const bool ok = valid && 2 * j + hi < n_splits && x[j] > kFloor;
      const float xj = ok ? x[j] : kFloor;
      const float mn = fmaxf(mx, xj);
      ls = ls * __builtin_amdgcn_exp2f(mx - mn) + (ok ? __builtin_amdgcn_exp2f(xj - mn) : 0.f);
      mx = mn;
    }
    if (ls == 0.f) mx = -INFINITY;
    const float2 mine = make_float2(mx, ls);
    const float2 other = make_float2(__shfl_xor(mx, 32, 64), __shfl_xor(ls, 32, 64));
    const float2 ml = hi == 0 ? combine_ml(mine, other) : combine_ml(other, mine);
    if (hi == 0) lse_l[32 * w + lq] = (valid && ml.y > 0.f) ? ml.x + __builtin_amdgcn_logf(ml.y) : 1e30f;
    __syncthreads();
    // S layout: value v of a lane belongs to query vector 8(v>>2)+4hi+(v&3) of the wave
#pragma unroll
    for (int v = 0; v < 16; ++v) lse_v[v] = lse_l[32 * w + 8 * (v >> 2) + 4 * hi + (v & 3)];
  }
  float m = -INFINITY, ls = 0.f;
  for (int c0 = key_lo; c0 < key_hi; c0 += kChunkKeys) {
    if (c0 > key_lo) __syncthreads();  // the previous chunk (and its sums) are no longer read
    if constexpr (kRot) {
      // the re-positioned key, rounded to bf16 as a stored re-positioned key is
#pragma unroll
      for (int i = 0; i < PU; ++i) {
        const int c = threadIdx.x + i * kW * 64;
        float x1[8], x2[8], y1[8], y2[8];
        Vec16<uint16_t>::unpack(buf[2 * i], x1);
        Vec16<uint16_t>::unpack(buf[2 * i + 1], x2);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint4 cv = csv[4 * i + e / 2];
          const float2 cs = (e & 1) ? make_float2(__uint_as_float(cv.z), __uint_as_float(cv.w))
                                    : make_float2(__uint_as_float(cv.x), __uint_as_float(cv.y));
          rope_pair(x1[e], x2[e], cs, y1[e], y2[e]);
        }
        uint16_t* dst = &k_lds[(c / HP) * KSTR + (c % HP) * 8];
        st16(dst, Vec16<uint16_t>::pack(y1));
        st16(dst + D / 2, Vec16<uint16_t>::pack(y2));
      }
    } else {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int c = threadIdx.x + i * kW * 64;
        st16(&k_lds[(c / CPR) * KSTR + (c % CPR) * 8], buf[i]);
      }
    }
    __syncthreads();
    const bool more = c0 + kChunkKeys < key_hi;
    if (more) fetch(c0 + kChunkKeys);  // in flight during this chunk's work
    const int n_keys = min(key_hi - c0, kChunkKeys);
    const int n_grp = (n_keys + 31) / 32;
    for (int kg = 0; kg < n_grp; ++kg) {
      if (kRot && more && kg == 1) fetch_cs();  // the next chunk's rotations, behind its pieces
      if (!live) {
        // a wave whose 32 query vectors are all padding (the request's last tile is
        // partly filled) adds nothing: it only takes part in the loads and barriers
        if (kCols && hi == 0) red[w][kg * 32 + lq] = 0.f;
        continue;
      }
      bf16x8 a[D / 16];
#pragma unroll
      for (int st = 0; st < D / 16; ++st) a[st] = as_bf16x8(ld16(&k_lds[(kg * 32 + lq) * KSTR + 8 * hi + 16 * st]));
      const int kt0 = c0 + kg * 32;
      f32x16 sacc = f32x16{};
      if (!kCols) {
        // S^T: value v of this lane is key 8(v>>2)+4hi+(v&3) of the group for the
        // lane's query vector; logits go to the log2 domain, keys past the split
        // are masked
#pragma unroll
        for (int st = 0; st < D / 16; ++st)
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[st], qreg[st], sacc, 0, 0, 0);
        if (kt0 + 32 > key_hi) {
#pragma unroll
          for (int v = 0; v < 16; ++v)
            if (kt0 + 8 * (v >> 2) + 4 * hi + (v & 3) >= key_hi) sacc[v] = -INFINITY;
        }
        float mt = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sacc[v]);
        const float mn = fmaxf(m, mt * scale2);
        if (mn != -INFINITY) {
          float acc = 0.f;
#pragma unroll
          for (int v = 0; v < 16; ++v) acc += __builtin_amdgcn_exp2f(fmaf(sacc[v], scale2, -mn));
          ls = ls * __builtin_amdgcn_exp2f(m - mn) + acc;
          m = mn;
        }
      } else {
        // S: this lane's key kt0 + lq, value v for query vector 8(v>>2)+4hi+(v&3)
#pragma unroll
        for (int st = 0; st < D / 16; ++st)
          sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qreg[st], a[st], sacc, 0, 0, 0);
        float cs = 0.f;
#pragma unroll
        for (int v = 0; v < 16; ++v) cs += __builtin_amdgcn_exp2f(fmaf(sacc[v], scale2, -lse_v[v]));
        const float cs_other = __shfl_xor(cs, 32, 64);
        if (hi == 0) red[w][kg * 32 + lq] = kt0 + lq < key_hi ? cs + cs_other : 0.f;
      }
    }
    if (kCols) {
      __syncthreads();
      if (threadIdx.x < n_keys) {
        float acc = 0.f;
#pragma unroll
        for (int ww = 0; ww < kW; ++ww) acc += red[ww][threadIdx.x];
        colp[((int64_t)(b * hkv + g) * n_qt + qt) * max_ctx + c0 + threadIdx.x] = acc;
      }
    }
  }
  if (!kCols) {
    // lanes l and l^32 hold disjoint keys of the same query vector; the split's
    // base-2 log-sum-exp log2(sum_t 2^(logit_t)) = max + log2(sum) (-inf: no keys)
    const float2 ml = combine_ml(make_float2(m, ls), make_float2(__shfl_xor(m, 32, 64), __shfl_xor(ls, 32, 64)));
    if (valid && hi == 0)
      part[((int64_t)(b * hkv + g) * n_splits + split) * max_qv + qv] =
          ml.y > 0.f ? ml.x + __builtin_amdgcn_logf(ml.y) : -INFINITY;
  }
}

// ---------------------------------------------------------------- bf16 final
// scores[t] (+)= the column sums of every (KV head, query tile) of the request
// that has query vectors, head-major
__global__ __launch_bounds__(kThreads) void scores_final(float* __restrict__ scores, int accumulate,
                                                         const float* __restrict__ colp,
                                                         const int32_t* __restrict__ cu_q,
                                                         const int32_t* __restrict__ cu_kv,
                                                         const int32_t* __restrict__ ctx_len,
                                                         int64_t n_kv_rows, int hkv, int lg,
                                                         int n_qt, int max_qv, int max_ctx) {
  const int t = blockIdx.x * kThreads + threadIdx.x, b = blockIdx.y;
  if (t >= ctx_len[b]) return;
  const int64_t row = cu_kv[b] + t;
  if (row >= n_kv_rows) return;
  const int nqv = min((cu_q[b + 1] - cu_q[b]) << lg, max_qv);
  const int nt = (nqv + kQvTile - 1) / kQvTile;
  const float* cp = colp + (int64_t)b * hkv * n_qt * max_ctx + t;
  float acc = 0.f;
  for (int g = 0; g < hkv; ++g)
    for (int j = 0; j < nt; ++j) acc += cp[((int64_t)g * n_qt + j) * max_ctx];
  scores[row] = accumulate ? scores[row] + acc : acc;
}

// ---------------------------------------------------------------- fp32 path
// key row `row` into kr[D], turned by its rotation-table row when kRot
template <int D, bool kRot>
__device__ __forceinline__ void key_f32(float* kr, const float* __restrict__ kp, int64_t row,
                                        const int32_t* __restrict__ key_rot,
                                        const float2* __restrict__ rot_tab, int n_rot) {
#pragma unroll
  for (int e = 0; e < D; ++e) kr[e] = kp[e];
  if constexpr (kRot) {
    const float2* cs = rot_tab + (int64_t)min(max(key_rot[row], 0), n_rot - 1) * (D / 2);
#pragma unroll
    for (int j = 0; j < D / 2; ++j) {
      const float x1 = kr[j], x2 = kr[j + D / 2];
      rope_pair(x1, x2, cs[j], kr[j], kr[j + D / 2]);
    }
  }
}

template <int D, bool kRot>
__global__ __launch_bounds__(64) void probe_stats_f32(float2* __restrict__ stats,
                                                      const float* __restrict__ q, int64_t n_q_rows,
                                                      const float* __restrict__ k, int64_t n_kv_rows,
                                                      int64_t k_stride, const int32_t* __restrict__ key_rot,
                                                      const float2* __restrict__ rot_tab, int n_rot,
                                                      const int32_t* __restrict__ cu_q,
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
    float kr[D];
    key_f32<D, kRot>(kr, k + (k0 + t) * k_stride + (int64_t)g * D, k0 + t, key_rot, rot_tab, n_rot);
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) acc += qs[e] * kr[e];
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

template <int D, bool kRot>
__global__ __launch_bounds__(kThreads) void probe_cols_f32(
    float* __restrict__ scores, int accumulate, const float2* __restrict__ stats,
    const float* __restrict__ q, int64_t n_q_rows, const float* __restrict__ k, int64_t n_kv_rows,
    int64_t k_stride, const int32_t* __restrict__ key_rot, const float2* __restrict__ rot_tab,
    int n_rot, const int32_t* __restrict__ cu_q, const int32_t* __restrict__ cu_kv,
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
      if (ok)
        key_f32<D, kRot>(kr, k + (k0 + t) * k_stride + (int64_t)g * D, k0 + t, key_rot, rot_tab, n_rot);
      else
#pragma unroll
        for (int e = 0; e < D; ++e) kr[e] = 0.f;
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
                               const KeyRot& rot, bool bf16, const int32_t* cu_q,
                               const int32_t* cu_kv, const int32_t* ctx_len, const ProbeShape& s,
                               float scale, void* ws, hipStream_t stream, const SelectArgs* sel) {
  if (s.batch == 0 || s.max_ctx_len == 0) return hipSuccess;
  const float scale2 = scale * kLog2e;
  int lg = 0;
  while ((1 << lg) < s.hq / s.hkv) ++lg;
  const bool rt = rot.row != nullptr;
  const float2* tab = reinterpret_cast<const float2*>(rot.table);
  const int n_rot = rt ? (int)rot.n : 1;
  if (!bf16) {
    float2* stats = static_cast<float2*>(ws);
    const float* qf = static_cast<const float*>(q);
    const float* kf = static_cast<const float*>(k);
    if (s.max_q_len > 0) {
      dim3 g1(s.max_q_len, s.hq, s.batch);
#define QCF_STATS(D, R)                                                                           \
  probe_stats_f32<D, R><<<g1, 64, 0, stream>>>(stats, qf, n_q_rows, kf, n_kv_rows, k_row_stride, \
                                               rot.row, tab, n_rot, cu_q, cu_kv, ctx_len, s.hq,  \
                                               s.hkv, s.max_q_len, scale2)
      if (s.d == 64) {
        if (rt) QCF_STATS(64, true); else QCF_STATS(64, false);
      } else {
        if (rt) QCF_STATS(128, true); else QCF_STATS(128, false);
      }
#undef QCF_STATS
    }
    dim3 g2((s.max_ctx_len + kThreads - 1) / kThreads, s.batch);
#define QCF_COLS(D, R)                                                                             \
  probe_cols_f32<D, R><<<g2, kThreads, 0, stream>>>(scores, accumulate, stats, qf, n_q_rows, kf,  \
                                                    n_kv_rows, k_row_stride, rot.row, tab, n_rot, \
                                                    cu_q, cu_kv, ctx_len, s.hq, s.hkv,            \
                                                    s.max_q_len, scale2)
    if (s.d == 64) {
      if (rt) QCF_COLS(64, true); else QCF_COLS(64, false);
    } else {
      if (rt) QCF_COLS(128, true); else QCF_COLS(128, false);
    }
#undef QCF_COLS
    if (sel) {
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      return launch_select_topk(sel->out_idx, sel->out_pos, sel->n_out, scores, n_kv_rows,
                                sel->n_seg, sel->seg_start, sel->seg_len, sel->seg_k,
                                sel->out_start, nullptr, sel->max_seg_len, stream, sel->seg_req,
                                cu_kv, s.batch);
    }
    return hipGetLastError();
  }
  const WsLayout w = ws_layout(s);
  if (s.batch > 65535) return hipErrorInvalidConfiguration;
  char* wb = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(wb + w.part_off);
  float* colp = reinterpret_cast<float*>(wb + w.col_off);
  const uint16_t* qb = static_cast<const uint16_t*>(q);
  const uint16_t* kb = static_cast<const uint16_t*>(k);
  if (w.max_qv > 0 && n_q_rows > 0 && n_kv_rows > 0) {
    const int64_t nblk = (int64_t)s.hkv * w.n_qt * w.n_splits * s.batch;
    if (nblk > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblk);
#define QCF_PASS(D, C, R)                                                                          \
  scores_pass_bf16<D, C, R><<<grid, kW * 64, 0, stream>>>(                                         \
      part, colp, qb, n_q_rows, kb, n_kv_rows, k_row_stride, rot.row, tab, n_rot, cu_q, cu_kv,     \
      ctx_len, s.hq, s.hkv, lg, w.n_qt, w.n_splits, w.split_keys, w.max_qv, s.max_ctx_len, scale2)
#define QCF_PASSES(D, R) \
  do {                   \
    QCF_PASS(D, false, R); \
    QCF_PASS(D, true, R);  \
  } while (0)
    if (s.d == 64) {
      if (rt) QCF_PASSES(64, true); else QCF_PASSES(64, false);
    } else {
      if (rt) QCF_PASSES(128, true); else QCF_PASSES(128, false);
    }
#undef QCF_PASSES
#undef QCF_PASS
  }
  if (sel && sel->max_seg_len <= 1024) {
    // the column sums are added per key by the selection itself (same order)
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const ScoreCols c{colp, cu_q, cu_kv, ctx_len, n_kv_rows, s.batch, s.hkv, lg,
                      std::max(1, w.n_qt), w.max_qv, s.max_ctx_len, kQvTile, accumulate};
    return launch_select_topk_cols(scores, n_kv_rows, c, *sel, stream);
  }
  scores_final<<<dim3((s.max_ctx_len + kThreads - 1) / kThreads, s.batch), kThreads, 0, stream>>>(
      scores, accumulate, colp, cu_q, cu_kv, ctx_len, n_kv_rows, s.hkv, lg, std::max(1, w.n_qt),
      w.max_qv, s.max_ctx_len);
  if (sel) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_select_topk(sel->out_idx, sel->out_pos, sel->n_out, scores, n_kv_rows,
                              sel->n_seg, sel->seg_start, sel->seg_len, sel->seg_k, sel->out_start,
                              nullptr, sel->max_seg_len, stream, sel->seg_req, cu_kv, s.batch);
  }
  return hipGetLastError();
}

}  // namespace qcf
