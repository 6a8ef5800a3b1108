// Causal grouped-query attention of the recomputed rows over the fused cache
// (Section 2.1.3: a recomputed row at position p reads every prefix key j <= p,
// itself included) and, with explicit key positions, the anchor-conditioned
// query probe (Section 3.3.2, eq. anchor_query_state).
//
// bf16 path (matrix cores, flash-style, one pass over the keys):
//  * a block owns 128 query vectors of one KV head: 128/G consecutive rows of
//    the request times the G query heads that share the KV head (GQA
//    packing), 32 vectors per wave;
//  * the keys 0 .. max(row position in the block) stream through LDS in
//    64-key tiles that arrive by direct global->LDS DMA (K two tiles ahead, V
//    one tile ahead; one barrier per tile), and the tile loop is software
//    pipelined: tile t+1's S^T runs on the matrix cores while tile t's
//    softmax runs on the vector ALUs;
//  * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (Q stays in registers as the B
//    operand), so each lane holds 16 logits of ONE query vector: row max,
//    rescale and row sum stay in the lane plus one lane^32 exchange;
//  * O^T += V^T P^T on the same instruction: P^T comes straight from the
//    logit registers (rounded to bf16), V^T from row-major LDS through the
//    gfx950 transposing LDS read, so V is never transposed in registers;
//  * online softmax in float32 (base-2 exponentials) with a lazy rescale;
//    the per-row causal limit masks only tiles that reach past the wave's
//    smallest position, and waves skip tiles past their largest position.
// fp32 path (vector ALUs): one wave per (row, head).
#include <limits.h>
#include <math.h>
#include <stdlib.h>

#include <algorithm>

#include "qcf_device.h"
#include "qcf_launch.h"

namespace qcf {
namespace {

constexpr int kThreads = 256;
constexpr int kKT = 64;  // keys per tile

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8, v); }

template <int D, bool kPos>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(
    uint16_t* __restrict__ out, float* __restrict__ lse, const uint16_t* __restrict__ q,
    const int32_t* __restrict__ row_pos, int64_t n_rows, const int32_t* __restrict__ cu_rows,
    const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, int64_t n_kv_rows,
    int64_t kv_stride, const int32_t* __restrict__ cu_kv, const int32_t* __restrict__ kv_pos,
    int batch, int max_tiles, int hkv, int hq, int lg, float scale2, int n_split_max,
    int split_tiles, float* __restrict__ part_o, float2* __restrict__ part_ml) {
  // LDS tiles, row-major, one key per row, filled by global->LDS DMA:
  //  K rows hold D/8 16-byte chunks + 1 pad chunk, so the 16-byte fragment
  //  reads of 8 consecutive keys hit distinct banks;
  //  V rows hold D/8 chunks + 4 pad chunks (a 64-byte shift per row), so the
  //  8-byte transposing reads of 8 rows x 64 bytes spread over all banks.
  constexpr int KCH = D / 8 + 1, VCH = D / 8 + 4;  // 16-byte chunks per LDS row
  constexpr int KSTR = KCH * 8, VSTR = VCH * 8;    // bf16 elements per LDS row
  constexpr int KI = (KCH + 3) / 4, VI = VCH / 4;  // DMA instructions per wave
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[2][kKT * KSTR];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[2][kKT * VSTR];
  __shared__ int kpos_lds[2][kPos ? kKT : 1];
  __shared__ int red[4];

  // Block order: consecutive block ids land on consecutive XCDs, so all
  // blocks of one KV head share an XCD (and its L2); the splits of one row
  // tile are adjacent; the tiles with the most keys (the last rows of each
  // request) are dispatched first.
  const int L = blockIdx.x;
  const int g = L % hkv;
  const int rest = L / hkv;
  const int split = rest % n_split_max;
  const int rest2 = rest / n_split_max;
  const int b = rest2 % batch;
  const int tile = max_tiles - 1 - rest2 / batch;
  const int G = 1 << lg;
  const int rpb = 128 >> lg;
  const int64_t r0 = cu_rows[b];
  const int nr = cu_rows[b + 1] - (int)r0;
  const int rbase = tile * rpb;
  if (rbase >= nr) return;
  const int64_t kv0 = cu_kv[b];
  int nkv = cu_kv[b + 1] - (int)kv0;
  if (kv0 + nkv > n_kv_rows) nkv = (int)(n_kv_rows - kv0);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int qv = 32 * w + lq;
  const int rl = rbase + (qv >> lg);
  const int head = g * G + (qv & (G - 1));
  const int64_t grow = r0 + rl;
  const bool valid = rl < nr && grow < n_rows;
  const int qpos = valid ? row_pos[grow] : INT_MIN;

  const int wmax = wave_max_i(valid ? qpos : -1);
  const int wmin = wave_min_i(valid ? qpos : INT_MAX);
  if (l == 0) red[w] = wmax;
  __syncthreads();
  const int bmax = max(max(red[0], red[1]), max(red[2], red[3]));
  const int kv_end = kPos ? nkv : min(nkv, bmax + 1);
  const int wave_end = kPos ? nkv : min(nkv, wmax + 1);
  // split-K: this block covers keys [kt_lo, kt_hi) of the row tile's range;
  // the last split also takes any remainder
  const int span = split_tiles * kKT;
  int nsp = (kv_end + span - 1) / span;
  if (nsp > n_split_max) nsp = n_split_max;
  const int kt_lo = split * span;
  if (split > 0 && kt_lo >= kv_end) return;
  const int kt_hi = split == nsp - 1 ? kv_end : min(kv_end, kt_lo + span);

  bf16x8 qreg[D / 16];
  {
    const uint16_t* qp = q + grow * (int64_t)hq * D + (int64_t)head * D + 8 * hi;
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      qreg[st] = as_bf16x8(valid ? ld16(qp + 16 * st) : make_uint4(0, 0, 0, 0));
  }
  f32x16 o[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};
  // running max in log2 units.  It starts at -1e30 (not -inf) so that a
  // masked logit (-inf) always gives p = exp2(-inf) = 0 without a guard;
  // padding lanes start at +inf so they never trigger a rescale and give p = 0.
  float m = valid ? -1e30f : INFINITY;
  float ls = 0.f;

  // DMA (global_load_lds_dwordx4: lane i of a wave writes 16 bytes at the
  // wave's LDS base + 16 i).  Instruction i of a tile fills LDS chunks
  // [64 i, 64 i + 64); wave w issues instructions w, w + 4, ...; the lane that
  // fills chunk c of row r loads key r's chunk c (pad chunks reload chunk 0).
  // Lane offsets are fixed; a full tile only moves a uniform base.  The tile
  // that crosses the end of the keys clamps its rows to the last key.
  const uint16_t* kbase = kc + kv0 * kv_stride + (int64_t)g * D;
  const uint16_t* vbase = vc + kv0 * kv_stride + (int64_t)g * D;
  const int jmax = max(nkv - 1, 0);
  int koff[KI], voff[KI > VI ? KI : VI];
#pragma unroll
  for (int t = 0; t < KI; ++t) {
    const int ci = (w + 4 * t) * 64 + l, r = ci / KCH, c = ci % KCH;
    koff[t] = r * (int)kv_stride + (c < D / 8 ? c * 8 : 0);
  }
#pragma unroll
  for (int t = 0; t < VI; ++t) {
    const int ci = (w + 4 * t) * 64 + l, r = ci / VCH, c = ci % VCH;
    voff[t] = r * (int)kv_stride + (c < D / 8 ? c * 8 : 0);
  }
  int kpos_reg = 0;
  auto dma = [&](const uint16_t* src, int off, uint16_t* dst) {
    __builtin_amdgcn_global_load_lds((const void*)(src + off),
                                     (void __attribute__((address_space(3)))*)dst, 16, 0, 0);
  };
  auto gload_k = [&](int kt0, int bfn) {
    if (kt0 + kKT <= nkv) {
      const uint16_t* kt = kbase + (int64_t)kt0 * kv_stride;
#pragma unroll
      for (int t = 0; t < KI; ++t)
        if (w + 4 * t < KCH) dma(kt, koff[t], &k_lds[bfn][(w + 4 * t) * 512]);
    } else {
#pragma unroll
      for (int t = 0; t < KI; ++t) {
        if (w + 4 * t >= KCH) continue;
        const int ci = (w + 4 * t) * 64 + l, r = ci / KCH, c = ci % KCH;
        const int j = min(kt0 + r, jmax);
        dma(kbase, j * (int)kv_stride + (c < D / 8 ? c * 8 : 0), &k_lds[bfn][(w + 4 * t) * 512]);
      }
    }
  };
  auto gload_v = [&](int kt0, int bfn) {
    if (kt0 + kKT <= nkv) {
      const uint16_t* vt = vbase + (int64_t)kt0 * kv_stride;
#pragma unroll
      for (int t = 0; t < VI; ++t) dma(vt, voff[t], &v_lds[bfn][(w + 4 * t) * 512]);
    } else {
#pragma unroll
      for (int t = 0; t < VI; ++t) {
        const int ci = (w + 4 * t) * 64 + l, r = ci / VCH, c = ci % VCH;
        const int j = min(kt0 + r, jmax);
        dma(vbase, j * (int)kv_stride + (c < D / 8 ? c * 8 : 0), &v_lds[bfn][(w + 4 * t) * 512]);
      }
    }
    if (kPos && threadIdx.x < kKT) {
      const int j = kt0 + threadIdx.x;
      kpos_reg = j < nkv ? kv_pos[kv0 + j] : INT_MAX;
    }
  };
  auto kstore = [&](int bfn) {
    if (kPos && threadIdx.x < kKT) kpos_lds[bfn][threadIdx.x] = kpos_reg;
  };
  // Transposing V reads (ds_read_b64_tr_b16): inside each 16-lane group, lane
  // j's element e comes from element (j & 3) of the 4-element segment that
  // lane 16 g + 4 e + ((j & 15) >> 2) addresses.  Lane (g, e, qd) therefore
  // addresses V row 4 (g >> 1) + e (+ 8 per read) at column 16 (g & 1) + 4 qd,
  // which hands every lane the keys of its P-operand slots for its d column.
  const int tg = l >> 4, te = (l >> 2) & 3, tq = l & 3;
  const int vrd = (4 * (tg >> 1) + te) * VSTR + 16 * (tg & 1) + 4 * tq;
  const int krd = lq * KSTR + 8 * hi;

  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef v4s __attribute__((address_space(3))) * lds_v4s;
  // V^T fragments of one 32-key half (2 k-steps x D/32 column blocks)
  auto read_v = [&](const uint16_t* vl, int hb, bf16x8* vf) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb) {
        const uint16_t* p0 = vl + (hb * 32 + 16 * k2) * VSTR + 32 * mb;
        const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p0));
        const v4s up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p0 + 8 * VSTR));
        vf[k2 * (D / 32) + mb] =
            __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
      }
  };
  // S^T = K Q^T of one 32-key half of the tile in LDS buffer kb
  auto qk_half = [&](const uint16_t* kl, int hb, f32x16& sh) {
    bf16x8 kf[D / 16];
#pragma unroll
    for (int st = 0; st < D / 16; ++st) kf[st] = as_bf16x8(ld16(kl + hb * 32 * KSTR + 16 * st));
    sh = f32x16{};
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      sh = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qreg[st], sh, 0, 0, 0);
  };
  // masks and running max of one tile (lazy rescale of O)
  auto softmax_pre = [&](f32x16 (&sc)[2], int kt0, int bfc) {
    const bool need_mask = kPos || kt0 + kKT > wmin || kt0 + kKT > nkv;
    if (need_mask) {
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int jt = hb * 32 + 8 * (v >> 2) + 4 * hi + (v & 3);
          const int j = kt0 + jt;
          const int kp = kPos ? kpos_lds[bfc][jt] : j;
          if (j >= nkv || kp > qpos) sc[hb][v] = -INFINITY;
        }
    }
    float mt = sc[0][0];
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[hb][v]);
    {
      // lanes l and l ^ 32 hold the two halves of the same query vector's keys
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt),
                                                       false, false);
      mt = fmaxf(mt, fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]))) * scale2;
    }
    // lazy rescale: keep a stale max unless some row's max grew by > 2^8
    if (__ballot(mt > m + 8.f)) {
      const float mn = fmaxf(m, mt);
      const float alpha = __builtin_amdgcn_exp2f(m - mn);
      ls *= alpha;
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;
      m = mn;
    }
  };
  // P = exp2(S * scale2 - m) of one tile -> pb (straight-line code)
  auto softmax_exp = [&](f32x16 (&sc)[2], bf16x8 (&pb)[2][2]) {
    const float nm = -m;
    float psum = 0.f;
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sc[hb][v], scale2, nm));
        psum += p;
        pb[hb][v >> 3][v & 7] = (__bf16)p;
      }
    ls += psum;
  };
  auto pv = [&](const uint16_t* vl, bf16x8 (&pb)[2][2]) {
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      bf16x8 vf[2 * (D / 32)];
      read_v(vl, hb, vf);
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
          o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[k2 * (D / 32) + mb], pb[hb][k2],
                                                          o[mb], 0, 0, 0);
    }
  };

  // Software pipeline over the key tiles of [kt_lo, kt_hi): while tile t's
  // softmax runs on the vector ALUs, tile t+1's S^T runs on the matrix cores.
  // K is fetched two tiles ahead and V one tile ahead, so two LDS buffers of
  // each and one barrier per tile suffice:
  //   step t: DMA K(t+2) -> K[t%2], V(t+1) -> V[(t+1)%2];
  //           S(t+1) from K[(t+1)%2] || softmax(t); O += P(t) V(t) from V[t%2];
  //           barrier.
  const int nt = kt_hi > kt_lo ? (kt_hi - kt_lo + kKT - 1) / kKT : 0;
  f32x16 sa[2], sb[2];
  if (nt > 0) {
    gload_k(kt_lo, 0);
    gload_v(kt_lo, 0);
    kstore(0);
  }
  if (nt > 1) gload_k(kt_lo + kKT, 1);
  __syncthreads();
  if (nt > 0 && kt_lo < wave_end) {
    qk_half(k_lds[0] + krd, 0, sa[0]);
    qk_half(k_lds[0] + krd, 1, sa[1]);
  }
  __syncthreads();
  auto step = [&](int t, f32x16 (&sc)[2], f32x16 (&sn)[2]) {
    const int cur = t & 1, nxt = cur ^ 1;
    const int kt0 = kt_lo + t * kKT;
    if (t + 2 < nt) gload_k(kt0 + 2 * kKT, cur);
    if (t + 1 < nt) gload_v(kt0 + kKT, nxt);
    const bool do_cur = kt0 < wave_end;
    const bool do_next = t + 1 < nt && kt0 + kKT < wave_end;
    bf16x8 pb[2][2];
    if (do_cur) softmax_pre(sc, kt0, cur);
    if (do_next) {
      // one basic block: the next tile's MFMAs interleave with this tile's exponentials
      qk_half(k_lds[nxt] + krd, 0, sn[0]);
      qk_half(k_lds[nxt] + krd, 1, sn[1]);
      softmax_exp(sc, pb);
#pragma unroll
      for (int i = 0; i < D / 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);   // then vector ALU work
      }
    } else if (do_cur) {
      softmax_exp(sc, pb);
    }
    if (do_cur) pv(v_lds[cur] + vrd, pb);
    if (t + 1 < nt) kstore(nxt);
    __syncthreads();
  };
  for (int t = 0; t < nt; t += 2) {
    step(t, sa, sb);
    if (t + 1 < nt) step(t + 1, sb, sa);
  }

  const float lt = ls + __shfl_xor(ls, 32, 64);
  uint16_t* op = out + grow * (int64_t)hq * D + (int64_t)head * D;
  if (nsp <= 1) {
    if (!valid) return;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = 32 * mb + 8 * i + 4 * hi;
        *reinterpret_cast<uint2*>(op + d0) =
            make_uint2(pack_bf16x2(o[mb][4 * i] * inv, o[mb][4 * i + 1] * inv),
                       pack_bf16x2(o[mb][4 * i + 2] * inv, o[mb][4 * i + 3] * inv));
      }
    if (lse && hi == 0) lse[grow * hq + head] = lt > 0.f ? (m + log2f(lt)) * kLn2 : -INFINITY;
    return;
  }
  // Several splits: write this split's unnormalised O^T, its (stale) max and
  // sum; attn_merge_kernel combines the splits after this kernel.
  if (!valid) return;
  const int64_t item = (((int64_t)b * max_tiles + tile) * hkv + g) * n_split_max + split;
  float* po = part_o + (item * 128 + qv) * D;
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<float4*>(po + 32 * mb + 8 * i + 4 * hi) =
          make_float4(o[mb][4 * i], o[mb][4 * i + 1], o[mb][4 * i + 2], o[mb][4 * i + 3]);
  if (hi == 0) part_ml[item * 128 + qv] = make_float2(m, lt);
}

// ---------------------------------------------------------------- 8-wave kernel
// The recomputed-row attention (no explicit key positions) on 8-wave blocks:
// 256 query vectors per block (256/G rows x the G heads of one KV head), 32
// per wave, with the same per-wave tile step as attn_bf16_kernel.  One block
// fills a CU (two waves per SIMD), which leaves LDS for a 4-stage ring of
// K/V tiles: K is fetched three tiles ahead and V two tiles ahead, and a step
// ends by waiting only for the tiles fetched one step earlier, so every
// global->LDS transfer has two steps to land.  The transfers are buffer loads
// with an LDS destination: a per-(request, head) descriptor bounds the key
// range, so rows past the last key and the LDS padding chunks read as zeros
// without touching memory, and a tile only moves a scalar row offset.
constexpr int kW8 = 8;                // waves per block
constexpr int kW8Qv = 32 * kW8;       // query vectors per block
constexpr int kStages = 4;            // LDS ring depth
constexpr int kW8Slots = 256;         // resident blocks: one per CU
constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every descriptor's range

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (stride 0): base address, byte range, gfx9 data format word.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)(uint32_t)(a >> 32) & 0xffff, (int)bytes, 0x00020000};
}

// 16 bytes per lane from the buffer at byte offset voff into LDS at lds + 16 * lane
// (zeros when voff is past the descriptor's range).  Issued as inline assembly
// so that the compiler adds no waits of its own for it: the caller orders the
// LDS traffic with explicit counter waits and barriers.
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t voff, const void* lds) {
  // the LDS base is wave-uniform; readfirstlane puts it in a scalar register
  const uint32_t la = __builtin_amdgcn_readfirstlane((uint32_t)reinterpret_cast<uintptr_t>(lds));
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(la), "v"(voff), "s"(rsrc)
               : "memory");
}

// s_waitcnt with vmcnt <= n and lgkmcnt == 0 (expcnt unconstrained); gfx9 encoding
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

template <int D>
__global__ __launch_bounds__(kW8 * 64, 1) void attn_w8_kernel(
    uint16_t* __restrict__ out, float* __restrict__ lse, const uint16_t* __restrict__ q,
    const int32_t* __restrict__ row_pos, int64_t n_rows, const int32_t* __restrict__ cu_rows,
    const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, int64_t n_kv_rows,
    int64_t kv_stride, const int32_t* __restrict__ cu_kv, int batch, int max_tiles, int hkv,
    int hq, int lg, float scale2, int n_split_max, int split_tiles, float* __restrict__ part_o,
    float2* __restrict__ part_ml) {
  constexpr int KCH = D / 8 + 1, VCH = D / 8 + 4;  // 16-byte chunks per LDS row (padded)
  constexpr int KSTR = KCH * 8, VSTR = VCH * 8;    // bf16 elements per LDS row
  constexpr int KST = kKT * KSTR, VST = kKT * VSTR;  // elements per stage
  constexpr int NSLOT = KCH + VCH;                   // 64-lane transfers per stage
  constexpr int SPW = (NSLOT + kW8 - 1) / kW8;       // transfers per wave (the first waves)
  constexpr int NFULL = NSLOT - (SPW - 1) * kW8;     // waves that issue SPW of them
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kStages * KST];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kStages * VST];
  __shared__ int red[kW8];

  const int L = blockIdx.x;
  const int g = L % hkv;
  const int rest = L / hkv;
  const int split = rest % n_split_max;
  const int rest2 = rest / n_split_max;
  const int b = rest2 % batch;
  const int tile = max_tiles - 1 - rest2 / batch;
  const int G = 1 << lg;
  const int rpb = kW8Qv >> lg;
  const int64_t r0 = cu_rows[b];
  const int nr = cu_rows[b + 1] - (int)r0;
  const int rbase = tile * rpb;
  if (rbase >= nr) return;
  const int64_t kv0 = cu_kv[b];
  int nkv = cu_kv[b + 1] - (int)kv0;
  if (kv0 + nkv > n_kv_rows) nkv = (int)(n_kv_rows - kv0);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int qv = 32 * w + lq;
  const int rl = rbase + (qv >> lg);
  const int head = g * G + (qv & (G - 1));
  const int64_t grow = r0 + rl;
  const bool valid = rl < nr && grow < n_rows;
  const int qpos = valid ? row_pos[grow] : INT_MIN;

  const int wmax = wave_max_i(valid ? qpos : -1);
  const int wmin = wave_min_i(valid ? qpos : INT_MAX);
  if (l == 0) red[w] = wmax;
  __syncthreads();
  int bmax = red[0];
#pragma unroll
  for (int i = 1; i < kW8; ++i) bmax = max(bmax, red[i]);
  const int kv_end = min(nkv, bmax + 1);
  const int wave_end = min(nkv, wmax + 1);
  const int span = split_tiles * kKT;
  int nsp = (kv_end + span - 1) / span;
  if (nsp > n_split_max) nsp = n_split_max;
  const int kt_lo = split * span;
  if (split > 0 && kt_lo >= kv_end) return;
  const int kt_hi = split == nsp - 1 ? kv_end : min(kv_end, kt_lo + span);

  bf16x8 qreg[D / 16];
  {
    const uint16_t* qp = q + grow * (int64_t)hq * D + (int64_t)head * D + 8 * hi;
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      qreg[st] = as_bf16x8(valid ? ld16(qp + 16 * st) : make_uint4(0, 0, 0, 0));
  }
  f32x16 o[D / 32];
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};
  float m = valid ? -1e30f : INFINITY;
  float ls = 0.f;

  // descriptors over this request's rows of KV head g: the last byte in range
  // is the end of the last key's head slice
  const uint32_t row_b = (uint32_t)(kv_stride * 2);
  const uint32_t range = nkv > 0 ? (uint32_t)(nkv - 1) * row_b + D * 2 : 0u;
  const i32x4 rk = make_rsrc(kc + kv0 * kv_stride + (int64_t)g * D, range);
  const i32x4 rv = make_rsrc(vc + kv0 * kv_stride + (int64_t)g * D, range);
  // this wave's transfer slots j = w + 8 i: slot j < KCH fills K chunks
  // [64 j, 64 j + 64) of a stage, the others V chunks; lane l of a slot fills
  // chunk 64 j + l = (row, column) of the padded tile
  uint32_t soff[SPW];
#pragma unroll
  for (int i = 0; i < SPW; ++i) {
    const int j = w + kW8 * i;
    const bool isk = j < KCH;
    const int ci = (isk ? j : j - KCH) * 64 + l;
    const int ch = isk ? KCH : VCH;
    const int r = ci / ch, c = ci % ch;
    soff[i] = (j < NSLOT && c < D / 8) ? (uint32_t)r * row_b + c * 16 : kOob;
  }
  const int nslots = w < NFULL ? SPW : SPW - 1;
  // the transfers of one step: tile r (relative to this split's first tile)
  // into stage r % 4, K and V; a tile past the split's end reads zeros
  const int t0 = kt_lo / kKT;
  const int nt = kt_hi > kt_lo ? (kt_hi - kt_lo + kKT - 1) / kKT : 0;
  auto issue = [&](int r) {
    const int sg = r & (kStages - 1);
    const uint32_t toff = (uint32_t)((t0 + r) * kKT) * row_b;
#pragma unroll
    for (int i = 0; i < SPW; ++i) {
      if (i >= nslots) break;
      const int j = w + kW8 * i;
      const uint32_t off = r < nt ? soff[i] + toff : kOob;
      if (j < KCH)
        dma16(rk, off, k_lds + sg * KST + j * 512);
      else
        dma16(rv, off, v_lds + sg * VST + (j - KCH) * 512);
    }
  };
  // end of a step: this step's transfers may stay in flight, all older ones
  // (and every LDS read) are complete, then the block meets
  auto step_barrier = [&]() {
    asm volatile("" ::: "memory");
    if (w < NFULL) wait_vm_lgkm0<SPW>();
    else wait_vm_lgkm0<SPW - 1>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  const int tg = l >> 4, te = (l >> 2) & 3, tq = l & 3;
  const int vrd = (4 * (tg >> 1) + te) * VSTR + 16 * (tg & 1) + 4 * tq;
  const int krd = lq * KSTR + 8 * hi;
  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef v4s __attribute__((address_space(3))) * lds_v4s;
  auto read_v = [&](const uint16_t* vl, int hb, bf16x8* vf) {
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb) {
        const uint16_t* p0 = vl + (hb * 32 + 16 * k2) * VSTR + 32 * mb;
        const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p0));
        const v4s up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p0 + 8 * VSTR));
        vf[k2 * (D / 32) + mb] =
            __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
      }
  };
  auto qk_half = [&](const uint16_t* kl, int hb, f32x16& sh) {
    bf16x8 kf[D / 16];
#pragma unroll
    for (int st = 0; st < D / 16; ++st) kf[st] = as_bf16x8(ld16(kl + hb * 32 * KSTR + 16 * st));
    sh = f32x16{};
#pragma unroll
    for (int st = 0; st < D / 16; ++st)
      sh = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qreg[st], sh, 0, 0, 0);
  };
  auto softmax_pre = [&](f32x16 (&sc)[2], int kt0) {
    if (kt0 + kKT > wmin || kt0 + kKT > nkv) {
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int j = kt0 + hb * 32 + 8 * (v >> 2) + 4 * hi + (v & 3);
          if (j >= nkv || j > qpos) sc[hb][v] = -INFINITY;
        }
    }
    float mt = sc[0][0];
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mt = fmaxf(mt, sc[hb][v]);
    {
      const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mt), __float_as_uint(mt),
                                                       false, false);
      mt = fmaxf(mt, fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]))) * scale2;
    }
    if (__ballot(mt > m + 8.f)) {
      const float mn = fmaxf(m, mt);
      const float alpha = __builtin_amdgcn_exp2f(m - mn);
      ls *= alpha;
#pragma unroll
      for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;
      m = mn;
    }
  };
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  auto softmax_exp = [&](f32x16 (&sc)[2], bf16x8 (&pb)[2][2]) {
    const float nm = -m;
    float psum = 0.f;
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sc[hb][v], scale2, nm));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sc[hb][v + 1], scale2, nm));
        psum += p0;
        psum += p1;
        const bf16x2_t pk = __builtin_convertvector((f32x2_t){p0, p1}, bf16x2_t);
        pb[hb][v >> 3][v & 7] = pk[0];
        pb[hb][v >> 3][(v & 7) + 1] = pk[1];
      }
    ls += psum;
  };
  auto pv = [&](const uint16_t* vl, bf16x8 (&pb)[2][2]) {
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      bf16x8 vf[2 * (D / 32)];
      read_v(vl, hb, vf);
#pragma unroll
      for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
        for (int mb = 0; mb < D / 32; ++mb)
          o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[k2 * (D / 32) + mb], pb[hb][k2],
                                                          o[mb], 0, 0, 0);
    }
  };

  // Ring: K(t) and V(t) live in stage t % 4.  Step t issues tile t+3 into the
  // stage of tile t-1 (its K was last read in step t-2, its V in step t-1),
  // computes S(t+1) while the softmax of tile t runs, then O += P(t) V(t); at
  // its end everything issued before step t -- K(t+2) and V(t+1) among it --
  // has landed.  Past the last tile the transfers still go out (zeros, no
  // memory traffic), so every step issues the same number of them.
  f32x16 sa[2], sb[2];
  issue(0);
  issue(1);
  issue(2);
  asm volatile("" ::: "memory");
  wait_vm_lgkm0<0>();
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  if (nt > 0 && kt_lo < wave_end) {
    qk_half(k_lds + krd, 0, sa[0]);
    qk_half(k_lds + krd, 1, sa[1]);
  }
  auto step = [&](int t, f32x16 (&sc)[2], f32x16 (&sn)[2]) {
    const int kt0 = kt_lo + t * kKT;
    issue(t + 3);
    const bool do_cur = kt0 < wave_end;
    const bool do_next = t + 1 < nt && kt0 + kKT < wave_end;
    bf16x8 pb[2][2];
    if (do_cur) softmax_pre(sc, kt0);
    if (do_next) {
      const uint16_t* kn = k_lds + ((t + 1) & 3) * KST + krd;
      qk_half(kn, 0, sn[0]);
      qk_half(kn, 1, sn[1]);
      softmax_exp(sc, pb);
#pragma unroll
      for (int i = 0; i < D / 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
      }
    } else if (do_cur) {
      softmax_exp(sc, pb);
    }
    if (do_cur) pv(v_lds + (t & 3) * VST + vrd, pb);
    step_barrier();
  };
  for (int t = 0; t < nt; t += 2) {
    step(t, sa, sb);
    if (t + 1 < nt) step(t + 1, sb, sa);
  }
  // drain the last (zero-row) transfers before the block's LDS can be reused
  asm volatile("" ::: "memory");
  wait_vm_lgkm0<0>();

  const float lt = ls + __shfl_xor(ls, 32, 64);
  uint16_t* op = out + grow * (int64_t)hq * D + (int64_t)head * D;
  if (nsp <= 1) {
    if (!valid) return;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d0 = 32 * mb + 8 * i + 4 * hi;
        *reinterpret_cast<uint2*>(op + d0) =
            make_uint2(pack_bf16x2(o[mb][4 * i] * inv, o[mb][4 * i + 1] * inv),
                       pack_bf16x2(o[mb][4 * i + 2] * inv, o[mb][4 * i + 3] * inv));
      }
    if (lse && hi == 0) lse[grow * hq + head] = lt > 0.f ? (m + log2f(lt)) * kLn2 : -INFINITY;
    return;
  }
  if (!valid) return;
  const int64_t item = (((int64_t)b * max_tiles + tile) * hkv + g) * n_split_max + split;
  float* po = part_o + (item * kW8Qv + qv) * D;
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<float4*>(po + 32 * mb + 8 * i + 4 * hi) =
          make_float4(o[mb][4 * i], o[mb][4 * i + 1], o[mb][4 * i + 2], o[mb][4 * i + 3]);
  if (hi == 0) part_ml[item * kW8Qv + qv] = make_float2(m, lt);
}

// Combines the split-K partials of every row tile that was split, in split
// order (deterministic).  One block per (row tile, KV head), QV query vectors
// per tile.  The block first turns each query vector's per-split (max, sum)
// into normalised split weights in LDS; then the tile's partial outputs, one
// contiguous [QV x D] float32 array per split, are streamed with consecutive
// threads on consecutive 32-byte pieces.
constexpr int kMaxSplit = 16;

template <int D, int QV>
__global__ __launch_bounds__(kThreads) void attn_merge_kernel(
    uint16_t* __restrict__ out, float* __restrict__ lse, const int32_t* __restrict__ row_pos,
    int64_t n_rows, const int32_t* __restrict__ cu_rows, const int32_t* __restrict__ cu_kv,
    int64_t n_kv_rows, int batch, int max_tiles, int hkv, int hq, int lg, int n_split_max,
    int split_tiles, const float* __restrict__ part_o, const float2* __restrict__ part_ml) {
  static_assert(QV == 128 || QV == 256, "tile width");
  __shared__ int red[4];
  __shared__ float wgt[kMaxSplit][QV];
  const int L = blockIdx.x;
  const int g = L % hkv;
  const int rest = L / hkv;
  const int b = rest % batch;
  const int tile = max_tiles - 1 - rest / batch;
  const int G = 1 << lg;
  const int rpb = QV >> lg;
  const int64_t r0 = cu_rows[b];
  const int nr = cu_rows[b + 1] - (int)r0;
  const int rbase = tile * rpb;
  if (rbase >= nr) return;
  const int64_t kv0 = cu_kv[b];
  int nkv = cu_kv[b + 1] - (int)kv0;
  if (kv0 + nkv > n_kv_rows) nkv = (int)(n_kv_rows - kv0);
  // the same key range (and split count) as the attention kernel's blocks
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  {
    int mx = -1;
    for (int qv = 64 * w + l; qv < QV; qv += kThreads) {
      const int rl = rbase + (qv >> lg);
      if (rl < nr && r0 + rl < n_rows) mx = max(mx, row_pos[r0 + rl]);
    }
    mx = wave_max_i(mx);
    if (l == 0) red[w] = mx;
  }
  __syncthreads();
  const int kv_end = min(nkv, max(max(red[0], red[1]), max(red[2], red[3])) + 1);
  const int span = split_tiles * kKT;
  int nsp = (kv_end + span - 1) / span;
  if (nsp > n_split_max) nsp = n_split_max;
  if (nsp <= 1) return;
  const int64_t base = (((int64_t)b * max_tiles + tile) * hkv + g) * n_split_max;
  for (int qv = threadIdx.x; qv < QV; qv += kThreads) {
    float mx = -1e30f;
    for (int sp = 0; sp < nsp; ++sp) mx = fmaxf(mx, part_ml[(base + sp) * QV + qv].x);
    float lsum = 0.f;
    for (int sp = 0; sp < nsp; ++sp) {
      const float2 ml = part_ml[(base + sp) * QV + qv];
      const float wsp = __builtin_amdgcn_exp2f(ml.x - mx);
      wgt[sp][qv] = wsp;
      lsum += wsp * ml.y;
    }
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    for (int sp = 0; sp < nsp; ++sp) wgt[sp][qv] *= inv;
    const int rl = rbase + (qv >> lg);
    const int64_t grow = r0 + rl;
    if (lse && rl < nr && grow < n_rows)
      lse[grow * hq + g * G + (qv & (G - 1))] = lsum > 0.f ? (mx + log2f(lsum)) * kLn2 : -INFINITY;
  }
  __syncthreads();
  // 8 consecutive floats per thread and pass; a pass covers 2048 / D query vectors
  constexpr int kPass = kThreads * 8;
  const float* pbase = part_o + base * QV * D;
#pragma unroll 2
  for (int e0 = 0; e0 < QV * D; e0 += kPass) {
    const int e = e0 + 8 * threadIdx.x;
    const int qv = e / D, dd = e % D;
    const int rl = rbase + (qv >> lg);
    const int64_t grow = r0 + rl;
    if (rl >= nr || grow >= n_rows) continue;
    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = 0.f;
    for (int sp = 0; sp < nsp; ++sp) {
      const float wv = wgt[sp][qv];
      const float4 x0 = *reinterpret_cast<const float4*>(pbase + (int64_t)sp * QV * D + e);
      const float4 x1 = *reinterpret_cast<const float4*>(pbase + (int64_t)sp * QV * D + e + 4);
      acc[0] += wv * x0.x; acc[1] += wv * x0.y; acc[2] += wv * x0.z; acc[3] += wv * x0.w;
      acc[4] += wv * x1.x; acc[5] += wv * x1.y; acc[6] += wv * x1.z; acc[7] += wv * x1.w;
    }
    const int head = g * G + (qv & (G - 1));
    *reinterpret_cast<uint4*>(out + grow * (int64_t)hq * D + (int64_t)head * D + dd) =
        make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                   pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7]));
  }
}

// ---------------------------------------------------------------- fp32 path
template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(
    float* __restrict__ out, float* __restrict__ lse, const float* __restrict__ q,
    const int32_t* __restrict__ row_pos, int64_t n_rows, const int32_t* __restrict__ cu_rows,
    int batch, const float* __restrict__ kc, const float* __restrict__ vc, int64_t n_kv_rows,
    int64_t kv_stride, const int32_t* __restrict__ cu_kv, const int32_t* __restrict__ kv_pos,
    int hq, int hkv, float scale2) {
  constexpr int E = D / 64;
  const int64_t r = blockIdx.x;
  const int h = blockIdx.y;
  const int l = threadIdx.x;
  // request of row r: last b with cu_rows[b] <= r
  int lo = 0, hi = batch - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu_rows[mid] <= r) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  if (r < cu_rows[b] || r >= cu_rows[b + 1] || r >= n_rows) return;
  const int64_t kv0 = cu_kv[b];
  int nkv = cu_kv[b + 1] - (int)kv0;
  if (kv0 + nkv > n_kv_rows) nkv = (int)(n_kv_rows - kv0);
  const int g = h / (hq / hkv);
  const int qpos = row_pos[r];
  float qr[E], o[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    qr[e] = q[r * (int64_t)hq * D + (int64_t)h * D + l + 64 * e];
    o[e] = 0.f;
  }
  float m = -INFINITY, ls = 0.f;
  const int jend = kv_pos ? nkv : min(nkv, qpos + 1);
  for (int j = 0; j < jend; ++j) {
    if (kv_pos && kv_pos[kv0 + j] > qpos) continue;
    const float* kp = kc + (kv0 + j) * kv_stride + (int64_t)g * D;
    const float* vp = vc + (kv0 + j) * kv_stride + (int64_t)g * D;
    float part = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) part += qr[e] * kp[l + 64 * e];
    const float x = wave_sum(part) * scale2;
    const float mn = fmaxf(m, x);
    const float alpha = exp2f(m - mn), p = exp2f(x - mn);
    ls = ls * alpha + p;
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = o[e] * alpha + p * vp[l + 64 * e];
    m = mn;
  }
  const float inv = ls > 0.f ? 1.f / ls : 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) out[r * (int64_t)hq * D + (int64_t)h * D + l + 64 * e] = o[e] * inv;
  if (lse && l == 0) lse[r * hq + h] = ls > 0.f ? (m + log2f(ls)) * kLn2 : -INFINITY;
}

// Split-K plan of the bf16 kernels (explicit-position calls never split).
// The estimate of the total work assumes row positions spread over each
// request (a triangle of key tiles).  A split holds about as many key tiles
// as one block slot of the chip gets on average (256 slots for the 8-wave
// kernel: one block per CU), at least 16, and at most 8 splits per row tile.
struct SplitPlan {
  int max_tiles, n_split, split_tiles;
  size_t o_off, ml_off, bytes;
};
// QCF_ATTN_SPLIT_TILES (read once) overrides the split size for tuning; 0
// disables splitting, unset (-1) keeps the automatic plan.
int forced_split_tiles() {
  static const int forced = [] {
    const char* e = getenv("QCF_ATTN_SPLIT_TILES");
    return e ? atoi(e) : -1;
  }();
  return forced;
}

// qv: query vectors per block; slots: blocks the chip holds at once
SplitPlan split_plan(const AttnShape& s, bool explicit_pos, int qv, int slots) {
  SplitPlan p{};
  int lg = 0;
  while ((1 << lg) < s.hq / s.hkv) ++lg;
  const int rpb = qv >> lg;
  p.max_tiles = (s.max_rows + rpb - 1) / rpb;
  const int kv_tiles = (s.max_kv + kKT - 1) / kKT;
  p.n_split = 1;
  p.split_tiles = kv_tiles > 0 ? kv_tiles : 1;
  const double est = 0.5 * (double)p.max_tiles * s.hkv * s.batch * kv_tiles;
  const int forced = forced_split_tiles();
  if (!explicit_pos && forced > 0 && forced < kv_tiles) {
    p.split_tiles = std::max(forced, (kv_tiles + kMaxSplit - 1) / kMaxSplit);
    p.n_split = (kv_tiles + p.split_tiles - 1) / p.split_tiles;
  } else if (!explicit_pos && forced < 0 && kv_tiles > 16) {
    int st = (int)((est + slots - 1.0) / slots);
    st = st < 16 ? 16 : st;
    const int min_st = (kv_tiles + 7) / 8;
    st = st < min_st ? min_st : st;
    if (st < kv_tiles) {
      p.split_tiles = st;
      p.n_split = (kv_tiles + st - 1) / st;
    }
  }
  if (p.n_split > 1) {
    const size_t groups = (size_t)p.max_tiles * s.hkv * s.batch;
    const size_t items = groups * p.n_split;
    auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
    p.o_off = 0;
    p.ml_off = a256(items * qv * s.d * sizeof(float));
    p.bytes = p.ml_off + a256(items * qv * sizeof(float2));
  }
  return p;
}

}  // namespace

size_t attn_workspace(const AttnShape& s, bool bf16) {
  if (!bf16 || s.batch <= 0 || s.max_rows <= 0) return 0;
  // An upper bound over every call whose batch, max_rows and max_kv do not
  // exceed these (the split count grows as the row count shrinks).  With G =
  // max_tiles * hkv * batch row groups, a plan has n_split <= 8 and, since a
  // split holds at least G * kv_tiles / (2 * slots) tiles, n_split <=
  // 2 * slots / G + 1.
  const SplitPlan mx = split_plan(s, false, kW8Qv, kW8Slots);
  const int kv_tiles = (s.max_kv + kKT - 1) / kKT;
  if (kv_tiles <= 16 && mx.n_split <= 1) return 0;
  const size_t G = (size_t)mx.max_tiles * s.hkv * s.batch;
  size_t items = std::min(8 * G, 2 * (size_t)kW8Slots + G);
  if (forced_split_tiles() > 0) items = G * kMaxSplit;  // a forced split size
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  return a256(items * kW8Qv * s.d * sizeof(float)) + a256(items * kW8Qv * sizeof(float2));
}

hipError_t launch_sparse_attn(void* out, float* lse, const void* q, const int32_t* row_pos,
                              int64_t n_rows, const int32_t* cu_rows, const void* k_cache,
                              const void* v_cache, int64_t n_kv_rows, int64_t kv_row_stride,
                              const int32_t* cu_kv, const int32_t* kv_pos, bool bf16,
                              const AttnShape& s, float scale, void* ws, hipStream_t stream) {
  if (n_rows == 0 || s.batch == 0 || s.max_rows == 0) return hipSuccess;
  const float scale2 = scale * kLog2e;
  int lg = 0;
  while ((1 << lg) < s.hq / s.hkv) ++lg;
  if (bf16 && !kv_pos) {
    // recomputed rows: the 8-wave kernel (buffer offsets of one request's rows are 32-bit)
    if ((double)s.max_kv * (double)kv_row_stride * 2.0 >= 2147483648.0) return hipErrorInvalidConfiguration;
    const SplitPlan p = split_plan(s, false, kW8Qv, kW8Slots);
    if (p.n_split > kMaxSplit) return hipErrorInvalidConfiguration;
    char* wb = static_cast<char*>(ws);
    float* part_o = p.n_split > 1 ? reinterpret_cast<float*>(wb + p.o_off) : nullptr;
    float2* part_ml = p.n_split > 1 ? reinterpret_cast<float2*>(wb + p.ml_off) : nullptr;
    const int64_t nblocks = (int64_t)p.max_tiles * s.batch * s.hkv * p.n_split;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblocks);
#define QCF_W8(D)                                                                                 \
  attn_w8_kernel<D><<<grid, kW8 * 64, 0, stream>>>(                                               \
      static_cast<uint16_t*>(out), lse, static_cast<const uint16_t*>(q), row_pos, n_rows, cu_rows, \
      static_cast<const uint16_t*>(k_cache), static_cast<const uint16_t*>(v_cache), n_kv_rows,    \
      kv_row_stride, cu_kv, s.batch, p.max_tiles, s.hkv, s.hq, lg, scale2, p.n_split,             \
      p.split_tiles, part_o, part_ml)
    if (s.d == 64) QCF_W8(64); else QCF_W8(128);
#undef QCF_W8
    if (p.n_split > 1) {
      dim3 mgrid((unsigned)((int64_t)p.max_tiles * s.batch * s.hkv));
#define QCF_MERGE(D)                                                                              \
  attn_merge_kernel<D, kW8Qv><<<mgrid, kThreads, 0, stream>>>(                                    \
      static_cast<uint16_t*>(out), lse, row_pos, n_rows, cu_rows, cu_kv, n_kv_rows, s.batch,       \
      p.max_tiles, s.hkv, s.hq, lg, p.n_split, p.split_tiles, part_o, part_ml)
      if (s.d == 64) QCF_MERGE(64); else QCF_MERGE(128);
#undef QCF_MERGE
    }
    return hipGetLastError();
  }
  if (bf16) {
    // explicit key positions (the anchor probe): the 4-wave kernel, never split
    const SplitPlan p = split_plan(s, true, 128, 512);
    if (p.n_split > kMaxSplit) return hipErrorInvalidConfiguration;
    char* wb = static_cast<char*>(ws);
    float* part_o = p.n_split > 1 ? reinterpret_cast<float*>(wb + p.o_off) : nullptr;
    float2* part_ml = p.n_split > 1 ? reinterpret_cast<float2*>(wb + p.ml_off) : nullptr;
    const int64_t nblocks = (int64_t)p.max_tiles * s.batch * s.hkv * p.n_split;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblocks);
#define QCF_ATTN(D, P)                                                                            \
  attn_bf16_kernel<D, P><<<grid, kThreads, 0, stream>>>(                                          \
      static_cast<uint16_t*>(out), lse, static_cast<const uint16_t*>(q), row_pos, n_rows, cu_rows, \
      static_cast<const uint16_t*>(k_cache), static_cast<const uint16_t*>(v_cache), n_kv_rows,    \
      kv_row_stride, cu_kv, kv_pos, s.batch, p.max_tiles, s.hkv, s.hq, lg, scale2, p.n_split,     \
      p.split_tiles, part_o, part_ml)
    if (kv_pos) {
      if (s.d == 64) QCF_ATTN(64, true); else QCF_ATTN(128, true);
    } else {
      if (s.d == 64) QCF_ATTN(64, false); else QCF_ATTN(128, false);
    }
#undef QCF_ATTN
    if (p.n_split > 1) {
      dim3 mgrid((unsigned)((int64_t)p.max_tiles * s.batch * s.hkv));
#define QCF_MERGE(D)                                                                              \
  attn_merge_kernel<D, 128><<<mgrid, kThreads, 0, stream>>>(                                      \
      static_cast<uint16_t*>(out), lse, row_pos, n_rows, cu_rows, cu_kv, n_kv_rows, s.batch,       \
      p.max_tiles, s.hkv, s.hq, lg, p.n_split, p.split_tiles, part_o, part_ml)
      if (s.d == 64) QCF_MERGE(64); else QCF_MERGE(128);
#undef QCF_MERGE
    }
    return hipGetLastError();
  }
  dim3 grid((unsigned)n_rows, s.hq);
  if (s.d == 64)
    attn_f32_kernel<64><<<grid, 64, 0, stream>>>(
        static_cast<float*>(out), lse, static_cast<const float*>(q), row_pos, n_rows, cu_rows,
        s.batch, static_cast<const float*>(k_cache), static_cast<const float*>(v_cache), n_kv_rows,
        kv_row_stride, cu_kv, kv_pos, s.hq, s.hkv, scale2);
  else
    attn_f32_kernel<128><<<grid, 64, 0, stream>>>(
        static_cast<float*>(out), lse, static_cast<const float*>(q), row_pos, n_rows, cu_rows,
        s.batch, static_cast<const float*>(k_cache), static_cast<const float*>(v_cache), n_kv_rows,
        kv_row_stride, cu_kv, kv_pos, s.hq, s.hkv, scale2);
  return hipGetLastError();
}

}  // namespace qcf
