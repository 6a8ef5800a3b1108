// Per-segment top-k of the importance scores: the recomputation set of
// eq. critical_mask, taken chunk by chunk (or, with one segment per request,
// over the whole context).
//
// One block per segment.  Scores become order-preserving uint32 keys (larger
// score -> larger key, -0 == +0).  A most-significant-digit radix select (4
// passes of 8 bits, LDS histograms) finds the key tau of the k-th largest
// score and how many of the keys equal to tau are still needed.  The chosen
// rows are then written in index order, taking keys > tau and the
// lowest-index keys == tau, so the output is ascending and ties go to the
// lower row -- exactly the order (score desc, index asc).  The result is
// bit-exact and independent of scheduling.
//
// Segments of up to 65536 keys (a whole long request in global mode) stay in
// registers: key i lives in thread i % NT, slot i / NT, so one coalesced read
// feeds every pass.  The ordered write needs each selected key's rank: per
// (slot, wave) cell a ballot count, one exclusive scan of the cells in
// (slot, wave) order -- which is index order -- and the lane's position in
// its ballot.  Longer segments take the fallback kernel, which re-reads the
// scores from memory in every pass.
#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kColsMaxSeg = 1024;  // longest segment of the fused score + selection kernel

__device__ __forceinline__ uint32_t order_key(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) == 0u) b = 0u;  // -0 == +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Exclusive block-wide prefix count of `pred` (in thread order) and the total.
__device__ __forceinline__ uint32_t block_prefix(bool pred, uint32_t* wave_tot, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(pred);
  const uint32_t below = lanes_below(m);
  if (lane == 0) wave_tot[wave] = (uint32_t)__popcll(m);
  __syncthreads();
  uint32_t before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t t = wave_tot[w];
    before += (w < wave) ? t : 0u;
    total += t;
  }
  __syncthreads();
  return before + below;
}

// After a histogram pass: the digit of the k-th largest among the keys that
// match the prefix so far (hist[d] = their count with digit d) and how many
// keys with a larger digit precede it.  Run by one whole wave.
__device__ __forceinline__ void digit_search(const uint32_t* hist, int remaining, uint32_t* sh) {
  const int lane = threadIdx.x & 63;
  // lane l owns digits 255-4l .. 252-4l (descending digit order)
  uint32_t c[4];
  uint32_t own = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    c[e] = hist[255 - 4 * lane - e];
    own += c[e];
  }
  // exclusive prefix over lanes = keys with a larger digit
  uint32_t incl = own;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  uint32_t above = incl - own;
  if (above < (uint32_t)remaining && (uint32_t)remaining <= incl) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (above + c[e] >= (uint32_t)remaining) {
        sh[0] = 255u - 4u * lane - e;
        sh[1] = above;
        break;
      }
      above += c[e];
    }
  }
}

// Most-significant-digit radix select over the keys key_at(i), i < n: the key
// tau of the k-th largest (1 <= k < n) and how many of the keys equal to tau
// belong to the top k.  NT threads; hist has 256 entries.
template <int NT, typename KeyAt>
__device__ void radix_select(KeyAt key_at, int n, int k, uint32_t* hist, uint32_t* sh,
                             uint32_t& tau, int& remaining) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0u, mask = 0u;
  remaining = k;  // how many of the keys matching `prefix` are still to be taken
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += NT) hist[i] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += NT) {
      const uint32_t key = key_at(i);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) digit_search(hist, remaining, sh);
    __syncthreads();
    const uint32_t digit = sh[0];
    remaining -= (int)sh[1];
    prefix |= digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  tau = prefix;
}

// ---------------------------------------------------------------- register path
// In place: cells[0 .. nc) -> their exclusive prefix sums.  Run by one wave.
template <int NC>
__device__ __forceinline__ void scan_cells(uint32_t* cells) {
  constexpr int CPL = (NC + 63) / 64;  // consecutive cells per lane
  const int lane = threadIdx.x & 63;
  uint32_t v[CPL];
  uint32_t own = 0;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int idx = lane * CPL + c;
    v[c] = idx < NC ? cells[idx] : 0u;
    own += v[c];
  }
  uint32_t incl = own;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  uint32_t run = incl - own;
#pragma unroll
  for (int c = 0; c < CPL; ++c) {
    const int idx = lane * CPL + c;
    if (idx < NC) cells[idx] = run;
    run += v[c];
  }
}

// With kCols the scores are first made final here: each context row's column
// sums (ScoreCols) are added in the order of the separate final pass and, with
// accumulate, onto the row's previous score, then written back; rows outside
// the request's context keep their stored score.
template <int NT, int KPT, bool kCols>
__global__ __launch_bounds__(NT) void topk_reg_kernel(
    int32_t* __restrict__ out_idx, int32_t* __restrict__ out_pos, int64_t n_out,
    float* __restrict__ scores, int64_t n_scores, const int32_t* __restrict__ seg_start,
    const int32_t* __restrict__ seg_len, const int32_t* __restrict__ seg_k,
    const int32_t* __restrict__ out_start, const int32_t* __restrict__ pos_base,
    const int32_t* __restrict__ seg_req, const int32_t* __restrict__ req_base, int n_req,
    ScoreCols cols) {
  static_assert(NT >= 256 && NT % 64 == 0 && KPT >= 1 && KPT <= 64, "block shape");
  constexpr int NW = NT / 64;
  constexpr int NC = KPT * NW;  // (slot, wave) cells, slot-major = index order
  __shared__ uint32_t hist[256];
  __shared__ uint32_t cells[NC];
  __shared__ uint32_t sh[2];

  const int s = blockIdx.x;
  const int64_t start = seg_start[s];
  const int n = seg_len[s];
  int k = seg_k[s];
  const int64_t o = out_start[s];
  const int rq = seg_req ? seg_req[s] : 0;
  if (seg_req && (rq < 0 || rq >= n_req)) return;
  const int pb = pos_base ? pos_base[s] : (seg_req ? req_base[rq] : 0);
  if (n <= 0 || start < 0 || start + n > n_scores || n > NT * KPT) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  float* sc = scores + start;

  // Every slot loads (clamped index, so all loads are issued at once).  Slots
  // at or past n get key 0, the smallest key: the top k of the padded slots
  // are those of the segment, since k <= n and equal keys go to the lower
  // index, so no slot needs a validity test later.
  uint32_t key[KPT];
  if constexpr (kCols) {
    // (head, query tile) terms in groups of kG, all of a group's loads in flight
    constexpr int kG = 8;
    const int b = rq;
    const int64_t kv0 = cols.cu_kv[b];
    const int nctx = cols.ctx_len[b];
    const int nqv = min((cols.cu_q[b + 1] - cols.cu_q[b]) << cols.lg, cols.max_qv);
    const int nterm = cols.hkv * ((nqv + cols.qv_tile - 1) / cols.qv_tile);
    const int ntl = max(1, (nqv + cols.qv_tile - 1) / cols.qv_tile);
    const float* cp = cols.colp + (int64_t)b * cols.hkv * cols.n_qt * cols.max_ctx;
    float acc[KPT], prev[KPT];
    int tcl[KPT];
    bool ctx[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const int i = min(tid + j * NT, n - 1);
      const int64_t t = start + i - kv0;
      ctx[j] = t >= 0 && t < nctx && start + i < cols.n_kv_rows;
      tcl[j] = (int)min(max(t, (int64_t)0), (int64_t)cols.max_ctx - 1);
      prev[j] = sc[i];
      acc[j] = 0.f;
    }
    for (int e0 = 0; e0 < nterm; e0 += kG) {
      float v[KPT][kG];
#pragma unroll
      for (int e = 0; e < kG; ++e) {
        const int ec = min(e0 + e, nterm - 1);
        const int g = ec / ntl, tl = ec - g * ntl;
        const float* cpe = cp + ((int64_t)g * cols.n_qt + tl) * cols.max_ctx;
#pragma unroll
        for (int j = 0; j < KPT; ++j) v[j][e] = cpe[tcl[j]];
      }
#pragma unroll
      for (int e = 0; e < kG; ++e)
#pragma unroll
        for (int j = 0; j < KPT; ++j)
          if (e0 + e < nterm) acc[j] += v[j][e];
    }
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const int i = tid + j * NT;
      const float x = ctx[j] ? (cols.accumulate ? prev[j] + acc[j] : acc[j]) : prev[j];
      if (i < n && ctx[j]) sc[i] = x;
      key[j] = i < n ? order_key(x) : 0u;
    }
  } else {
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const int i = tid + j * NT;
      const uint32_t kv = order_key(sc[min(i, n - 1)]);
      key[j] = i < n ? kv : 0u;
    }
  }
  if (k <= 0) return;
  if (k > n) k = n;
  if (o < 0 || o + k > n_out) return;

  const bool take_all = (k == n);
  uint32_t tau = 0u;
  int remaining = k;
  if (!take_all) {
    uint32_t prefix = 0u, mask = 0u;
    for (int shift = 24; shift >= 0; shift -= 8) {
      if (tid < 256) hist[tid] = 0u;
      __syncthreads();
#pragma unroll
      for (int j = 0; j < KPT; ++j)
        if ((key[j] & mask) == prefix) atomicAdd(&hist[(key[j] >> shift) & 255u], 1u);
      __syncthreads();
      if (w == 0) digit_search(hist, remaining, sh);
      __syncthreads();
      prefix |= sh[0] << shift;
      remaining -= (int)sh[1];
      mask |= 255u << shift;
      __syncthreads();  // sh and hist are rewritten by the next pass
    }
    tau = prefix;
  }

  // which slots are chosen: keys > tau, and keys == tau whose rank among the
  // keys == tau (index order) is below `remaining`
  uint64_t sel = 0;
  if (take_all) {
#pragma unroll
    for (int j = 0; j < KPT; ++j)
      if (tid + j * NT < n) sel |= 1ull << j;
  } else {
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const uint64_t m = __ballot(key[j] == tau);
      if (lane == 0) cells[j * NW + w] = (uint32_t)__popcll(m);
    }
    __syncthreads();
    if (w == 0) scan_cells<NC>(cells);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const bool eq = key[j] == tau;
      const uint64_t m = __ballot(eq);
      const uint32_t rank = cells[j * NW + w] + lanes_below(m);
      if (key[j] > tau || (eq && rank < (uint32_t)remaining)) sel |= 1ull << j;
    }
    __syncthreads();  // cells are rewritten below
  }
  // output slots of the chosen keys, in index order
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const uint64_t m = __ballot((sel >> j) & 1ull);
    if (lane == 0) cells[j * NW + w] = (uint32_t)__popcll(m);
  }
  __syncthreads();
  if (w == 0) scan_cells<NC>(cells);
  __syncthreads();
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const bool chosen = (sel >> j) & 1ull;
    const uint64_t m = __ballot(chosen);
    const uint32_t slot = cells[j * NW + w] + lanes_below(m);
    if (chosen && slot < (uint32_t)k) {
      const int32_t row = (int32_t)(start + tid + j * NT);
      out_idx[o + slot] = row;
      if (out_pos) out_pos[o + slot] = row - pb;
    }
  }
}

// ---------------------------------------------------------------- fallback
// Segments longer than the register path holds: the scores are re-read from
// memory in every pass.
__global__ __launch_bounds__(kThreads) void select_topk_kernel(
    int32_t* __restrict__ out_idx, int32_t* __restrict__ out_pos, int64_t n_out,
    const float* __restrict__ scores, int64_t n_scores, const int32_t* __restrict__ seg_start,
    const int32_t* __restrict__ seg_len, const int32_t* __restrict__ seg_k,
    const int32_t* __restrict__ out_start, const int32_t* __restrict__ pos_base,
    const int32_t* __restrict__ seg_req, const int32_t* __restrict__ req_base, int n_req) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wave_tot[kWaves];
  __shared__ uint32_t sh[2];

  const int s = blockIdx.x;
  const int64_t start = seg_start[s];
  int n = seg_len[s];
  int k = seg_k[s];
  const int64_t o = out_start[s];
  const int rq = seg_req ? seg_req[s] : 0;
  if (seg_req && (rq < 0 || rq >= n_req)) return;
  const int pb = pos_base ? pos_base[s] : (seg_req ? req_base[rq] : 0);
  if (n <= 0 || k <= 0 || start < 0 || start + n > n_scores) return;
  if (k > n) k = n;
  if (o < 0 || o + k > n_out) return;
  const float* sc = scores + start;
  const int tid = threadIdx.x;

  auto key_at = [&](int i) -> uint32_t { return order_key(sc[i]); };

  const bool take_all = (k == n);
  uint32_t tau = 0u;
  int remaining = k;
  if (!take_all) radix_select<kThreads>(key_at, n, k, hist, sh, tau, remaining);

  // ordered compaction: keys > tau, then the `remaining` lowest-index keys == tau
  uint32_t eq_base = 0, sel_base = 0;
  for (int t0 = 0; t0 < n; t0 += kThreads) {
    const int i = t0 + tid;
    const bool valid = i < n;
    const uint32_t key = valid ? key_at(i) : 0u;
    const bool gt = valid && (take_all || key > tau);
    const bool eq = valid && !take_all && key == tau;
    uint32_t eq_tot, sel_tot;
    const uint32_t eq_rank = eq_base + block_prefix(eq, wave_tot, eq_tot);
    const bool sel = gt || (eq && eq_rank < (uint32_t)remaining);
    const uint32_t slot = sel_base + block_prefix(sel, wave_tot, sel_tot);
    if (sel && slot < (uint32_t)k) {
      out_idx[o + slot] = (int32_t)(start + i);
      if (out_pos) out_pos[o + slot] = (int32_t)(start + i) - pb;
    }
    eq_base += eq_tot;
    sel_base += sel_tot;
  }
}

}  // namespace

hipError_t launch_select_topk(int32_t* out_idx, int32_t* out_pos, int64_t n_out,
                              const float* scores, int64_t n_scores, int n_seg,
                              const int32_t* seg_start, const int32_t* seg_len,
                              const int32_t* seg_k, const int32_t* out_start,
                              const int32_t* pos_base, int max_seg_len, hipStream_t stream,
                              const int32_t* seg_req, const int32_t* req_base, int n_req) {
  if (n_seg == 0 || max_seg_len == 0) return hipSuccess;
  const dim3 grid(n_seg);
  float* sw = const_cast<float*>(scores);  // only the kCols form writes scores
#define QCF_TOPK(NT, KPT)                                                                         \
  topk_reg_kernel<NT, KPT, false><<<grid, NT, 0, stream>>>(out_idx, out_pos, n_out, sw, n_scores, \
                                                           seg_start, seg_len, seg_k, out_start,  \
                                                           pos_base, seg_req, req_base, n_req,    \
                                                           ScoreCols{})
  if (max_seg_len <= 1024) QCF_TOPK(256, 4);
  else if (max_seg_len <= 4096) QCF_TOPK(256, 16);
  else if (max_seg_len <= 8192) QCF_TOPK(512, 16);
  else if (max_seg_len <= 16384) QCF_TOPK(1024, 16);
  else if (max_seg_len <= 32768) QCF_TOPK(1024, 32);
  else if (max_seg_len <= 65536) QCF_TOPK(1024, 64);
  else
    select_topk_kernel<<<grid, kThreads, 0, stream>>>(out_idx, out_pos, n_out, scores, n_scores,
                                                      seg_start, seg_len, seg_k, out_start, pos_base,
                                                      seg_req, req_base, n_req);
#undef QCF_TOPK
  return hipGetLastError();
}

hipError_t launch_select_topk_cols(float* scores, int64_t n_scores, const ScoreCols& c,
                                   const SelectArgs& a, hipStream_t stream) {
  if (a.n_seg == 0 || a.max_seg_len == 0) return hipSuccess;
  const dim3 grid(a.n_seg);
#define QCF_TOPKC(NT, KPT)                                                                      \
  topk_reg_kernel<NT, KPT, true><<<grid, NT, 0, stream>>>(                                      \
      a.out_idx, a.out_pos, a.n_out, scores, n_scores, a.seg_start, a.seg_len, a.seg_k,         \
      a.out_start, nullptr, a.seg_req, c.cu_kv, c.batch, c)
  // segments of up to 1024 rows (chunks): every thread sums four rows' terms with all
  // their loads in flight; longer segments take the separate final pass
  if (a.max_seg_len <= kColsMaxSeg) QCF_TOPKC(256, 4);
  else return hipErrorNotSupported;
#undef QCF_TOPKC
  return hipGetLastError();
}

}  // namespace qcf

