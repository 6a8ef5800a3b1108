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

template <int NT, int KPT>
__global__ __launch_bounds__(NT) void topk_reg_kernel(
    int32_t* __restrict__ out_idx, int32_t* __restrict__ out_pos, int64_t n_out,
    const float* __restrict__ scores, int64_t n_scores, const int32_t* __restrict__ seg_start,
    const int32_t* __restrict__ seg_len, const int32_t* __restrict__ seg_k,
    const int32_t* __restrict__ out_start, const int32_t* __restrict__ pos_base) {
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
  const int pb = pos_base ? pos_base[s] : 0;
  if (n <= 0 || k <= 0 || start < 0 || start + n > n_scores || n > NT * KPT) return;
  if (k > n) k = n;
  if (o < 0 || o + k > n_out) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* sc = scores + start;

  // Every slot loads (clamped index, so all loads are issued at once).  Slots
  // at or past n get key 0, the smallest key: the top k of the padded slots
  // are those of the segment, since k <= n and equal keys go to the lower
  // index, so no slot needs a validity test later.
  uint32_t key[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const int i = tid + j * NT;
    const uint32_t kv = order_key(sc[min(i, n - 1)]);
    key[j] = i < n ? kv : 0u;
  }

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
    const int32_t* __restrict__ out_start, const int32_t* __restrict__ pos_base) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wave_tot[kWaves];
  __shared__ uint32_t sh[2];

  const int s = blockIdx.x;
  const int64_t start = seg_start[s];
  int n = seg_len[s];
  int k = seg_k[s];
  const int64_t o = out_start[s];
  const int pb = pos_base ? pos_base[s] : 0;
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
                              const int32_t* pos_base, int max_seg_len, hipStream_t stream) {
  if (n_seg == 0 || max_seg_len == 0) return hipSuccess;
  const dim3 grid(n_seg);
#define QCF_TOPK(NT, KPT)                                                                        \
  topk_reg_kernel<NT, KPT><<<grid, NT, 0, stream>>>(out_idx, out_pos, n_out, scores, n_scores,  \
                                                    seg_start, seg_len, seg_k, out_start, pos_base)
  if (max_seg_len <= 1024) QCF_TOPK(256, 4);
  else if (max_seg_len <= 4096) QCF_TOPK(256, 16);
  else if (max_seg_len <= 8192) QCF_TOPK(512, 16);
  else if (max_seg_len <= 16384) QCF_TOPK(1024, 16);
  else if (max_seg_len <= 32768) QCF_TOPK(1024, 32);
  else if (max_seg_len <= 65536) QCF_TOPK(1024, 64);
  else
    select_topk_kernel<<<grid, kThreads, 0, stream>>>(out_idx, out_pos, n_out, scores, n_scores,
                                                      seg_start, seg_len, seg_k, out_start, pos_base);
#undef QCF_TOPK
  return hipGetLastError();
}

}  // namespace qcf

