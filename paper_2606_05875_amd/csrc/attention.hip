// Causal grouped-query attention of the recomputed rows over the fused cache
// (Section 2.1.3: a recomputed row at position p reads every prefix key j <= p,
// itself included) and, with explicit key positions, the anchor-conditioned
// query probe (Section 3.3.2, eq. anchor_query_state).
//
// bf16 path (matrix cores, flash-style, one pass over the keys).  Per wave:
//  * 32 query vectors of one KV head: consecutive rows of the request times
//    the G query heads that share the KV head (GQA packing);
//  * the keys stream through LDS in 64-key tiles, and the tile loop is
//    software pipelined: tile t+1's S^T runs on the matrix cores while tile
//    t's softmax runs on the vector ALUs;
//  * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (Q stays in registers as the B
//    operand), so each lane holds 16 logits of ONE query vector: row max,
//    rescale and row sum stay in the lane plus one lane^32 exchange;
//  * O^T += V^T P^T on the same instruction: P^T comes straight from the
//    logit registers (rounded to bf16), V^T from row-major LDS through the
//    gfx950 transposing LDS read, so V is never transposed in registers;
//  * online softmax in float32 (base-2 exponentials) with a lazy rescale;
//    the causal limit masks only tiles that reach past the wave's smallest
//    position, and waves skip tiles past their largest position.
// Recomputed rows run on attn_w8_kernel (8 waves, 256 query vectors, a
// 4-stage K/V ring filled by buffer loads; the products run as fenced
// sequences with their LDS fragment reads issued four products ahead; on the
// plain grid the two waves of a SIMD run the step a product phase apart, and
// one long request hands its row tiles out from per-XCD work queues; a
// persistent "stream" grid when the row tiles are few and unequal), the probe
// on attn_pos_kernel (4 waves, K/V
// by global->LDS loads two and one tiles ahead, key positions from a table).
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

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_pos_kernel(
    uint16_t* __restrict__ out, float* __restrict__ lse, const uint16_t* __restrict__ q,
    const int32_t* __restrict__ row_pos, int64_t n_rows, const int32_t* __restrict__ cu_rows,
    const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, int64_t n_kv_rows,
    int64_t kv_stride, const int32_t* __restrict__ cu_kv, const int32_t* __restrict__ kv_pos,
    int batch, int max_tiles, int hkv, int hq, int lg, float scale2) {
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
  __shared__ int kpos_lds[2][kKT];

  // Block order: consecutive block ids land on consecutive XCDs, so all
  // blocks of one KV head share an XCD (and its L2); the tiles with the most
  // rows are dispatched first.
  const int L = blockIdx.x;
  const int g = L % hkv;
  const int rest = L / hkv;
  const int b = rest % batch;
  const int tile = max_tiles - 1 - rest / batch;
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

  // every key is visited; the mask compares key positions with row positions
  const int kt_lo = 0, kt_hi = nkv;
  const int wave_end = nkv;
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
    if (threadIdx.x < kKT) {
      const int j = kt0 + threadIdx.x;
      kpos_reg = j < nkv ? kv_pos[kv0 + j] : INT_MAX;
    }
  };
  auto kstore = [&](int bfn) {
    if (threadIdx.x < kKT) kpos_lds[bfn][threadIdx.x] = kpos_reg;
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
    {
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int jt = hb * 32 + 8 * (v >> 2) + 4 * hi + (v & 3);
          const int j = kt0 + jt;
          const int kp = kpos_lds[bfc][jt];
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
  if (!valid) return;
  uint16_t* op = out + grow * (int64_t)hq * D + (int64_t)head * D;
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
}

// ---------------------------------------------------------------- 8-wave kernel
// The recomputed-row attention (no explicit key positions) on 8-wave blocks:
// 256 query vectors per block (256/G rows x the G heads of one KV head), 32
// per wave, with the same per-wave tile step as attn_pos_kernel.  One block
// fills a CU (two waves per SIMD), which leaves LDS for a 4-stage ring of
// K/V tiles: step t fetches K(t+3), first read in step t+2, and V(t+3) (V(t+2)
// on the split plain grid), first read in step t+3 (t+2), and a step ends by
// waiting only for the tiles fetched one step earlier, so every global->LDS
// transfer has at least two steps to land.  The transfers are buffer loads
// with an LDS destination: a per-(request, head) descriptor bounds the key
// range, so rows past the last key and the LDS padding chunks read as zeros
// without touching memory, and a tile only moves a scalar row offset.  (Tiles
// staged through registers -- 16-byte loads one step ahead, then plain LDS
// writes -- measured 3% slower on the c2 call with its inputs cold in the
// caches: one step of latency cover instead of two.)
constexpr int kW8 = 8;                // waves per block
constexpr int kW8Qv = 32 * kW8;       // query vectors per block
constexpr int kStages = 4;            // LDS ring depth
constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every descriptor's range

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (stride 0): base address, byte range, gfx9 data format word.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)(uint32_t)(a >> 32) & 0xffff, (int)bytes, 0x00020000};
}

// LDS byte address of a __shared__ object (32 bits, as the LDS instructions take it)
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p);
}

// 16 bytes per lane from the buffer at byte offset voff into LDS at byte
// address lds + 16 * lane (zeros when voff is past the descriptor's range).
// Issued as inline assembly so that the compiler adds no waits of its own for
// it: the caller orders the LDS traffic with explicit counter waits and barriers.
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t voff, uint32_t lds) {
  // the LDS address is wave-uniform; readfirstlane keeps it in a scalar register
  const uint32_t la = __builtin_amdgcn_readfirstlane(lds);
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

// Work of an 8-wave block.  Plain mode: block -> (KV head g, request b, row
// tile), the tile's whole key range (fixed by the block id, or claimed from a
// work queue for one long request).  Stream mode (few, unequal tiles): a
// persistent grid of nbg blocks per KV head; the head's work -- every row
// tile of every request in (request, row tile) order, each counted as
// kSegCost start-up steps followed by its 64-key steps -- is cut into nbg
// equal contiguous ranges, one per block, so every block does about the same
// amount of work whatever the row positions.  A row tile cut by a range
// boundary leaves partial results (at most two per block: its first and its
// last segment) that attn_stream_merge_kernel combines.
constexpr int kMaxStreamTiles = 256;  // row tiles (requests x tiles) of a stream-mode call
constexpr int kStreamBlocks = 256;    // persistent blocks (one per CU of MI355X)
// stream-mode plan in the workspace (int32): step prefix sums [0, kMaxStreamTiles],
// key ends, then the first cost-line unit of every block of a head [0, nbg]
constexpr int kPlanEndOff = kMaxStreamTiles + 1;
constexpr int kPlanBndOff = 2 * kMaxStreamTiles + 1;
constexpr int kPlanInts = kPlanBndOff + kStreamBlocks + 1;
// Start-up cost of a segment (row positions, Q and the first key tiles in
// flight before the first product, plus its output stores), in key steps:
// each row tile counts as this many extra steps when the ranges are cut, so
// a block that starts several tiles gets fewer key steps.
constexpr int kSegCost = 4;
// Plain grid over one long request: at most one work queue per XCD, their counters
// 128 bytes apart in the workspace, and the hardware register that names a wave's XCD.
constexpr int kQueues = 8;
constexpr int kQueueStride = 32;
constexpr int kHwRegXccId = (31 << 11) | 20;  // s_getreg: XCC_ID, bits [31:0]

// Turns a lane's query fragments by the rotation of its row's position (Section
// 2.1.3: a recomputed row's fresh query is rotated at its request position).  The
// lane holds pieces 16 st + 8 hi + e (e < 8) of slots st < D/16; rotate-half pairs
// (j, j + D/2) sit in slots st and st + D/32 of the same lane.  tr is the row's
// D/2 (cos, sin) pairs of qcf_rope_table, and the arithmetic is rope_pair's, so
// the result is bit for bit the scatter's rotated query.
template <int D>
__device__ __forceinline__ void rotate_query(bf16x8 (&qr)[D / 16], const float2* __restrict__ tr,
                                             int hi) {
  constexpr int H = D / 32;
#pragma unroll
  for (int st = 0; st < H; ++st) {
    const float4* t4 = reinterpret_cast<const float4*>(tr + 16 * st + 8 * hi);
    float4 c4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) c4[i] = t4[i];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float4 c = c4[e >> 1];
      const float2 cs = (e & 1) ? make_float2(c.z, c.w) : make_float2(c.x, c.y);
      float y1, y2;
      rope_pair((float)qr[st][e], (float)qr[st + H][e], cs, y1, y2);
      qr[st][e] = (__bf16)y1;
      qr[st + H][e] = (__bf16)y2;
    }
  }
}

template <int D, bool kStream, bool kRot>
__global__ __launch_bounds__(kW8 * 64, 1) void attn_w8_kernel(
    uint16_t* __restrict__ out, float* __restrict__ lse, const uint16_t* __restrict__ q,
    const int32_t* __restrict__ row_pos, int64_t n_rows, const int32_t* __restrict__ cu_rows,
    const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc, int64_t n_kv_rows,
    int64_t kv_stride, const int32_t* __restrict__ cu_kv, int batch, int max_tiles, int hkv,
    int hq, int lg, float scale2, int nbg, int32_t* __restrict__ plan_out,
    uint16_t* __restrict__ part_o, float2* __restrict__ part_ml,
    const int32_t* __restrict__ q_src, int64_t n_q_src, const float2* __restrict__ rtab,
    int n_tab, uint32_t* __restrict__ queue) {
  constexpr int KCH = D / 8 + 1, VCH = D / 8 + 4;  // 16-byte chunks per LDS row (padded)
  constexpr int KSTR = KCH * 8, VSTR = VCH * 8;    // bf16 elements per LDS row
  constexpr int KST = kKT * KSTR, VST = kKT * VSTR;  // elements per stage
  constexpr int NSLOT = KCH + VCH;                   // 64-lane transfers per stage
  constexpr int SPW = (NSLOT + kW8 - 1) / kW8;       // transfers per wave (the first waves)
  constexpr int NFULL = NSLOT - (SPW - 1) * kW8;     // waves that issue SPW of them
  // Plain mode splits the block: waves 0-3 (one per SIMD) load the K chunks of a stage and
  // multiply P(t) V(t) in step t; waves 4-7 load the V chunks and multiply P(t) V(t) at the
  // start of step t+1.  The stream grid keeps one schedule for all waves.
  constexpr bool kDefer = !kStream;
  constexpr int SPWK = (KCH + 3) / 4, SPWV = (VCH + 3) / 4;  // transfers per wave, split
  constexpr int SPWX = kDefer ? (SPWK > SPWV ? SPWK : SPWV) : SPW;
  __shared__ __attribute__((aligned(16))) uint16_t k_lds[kStages * KST];
  __shared__ __attribute__((aligned(16))) uint16_t v_lds[kStages * VST];
  __shared__ int red[kW8];
  __shared__ int q_next;  // plain grid with queues: a claimed item or a queue
  __shared__ int plan_cum[kStream ? kMaxStreamTiles + 1 : 1];
  __shared__ int plan_end[kStream ? kMaxStreamTiles : 1];
  __shared__ int req_rows[kStream ? kMaxStreamTiles + 1 : 1];  // cu_rows, cu_kv of the call
  __shared__ int req_kv[kStream ? kMaxStreamTiles + 1 : 1];

  // the wave index is uniform: readfirstlane lets everything derived from it live in
  // scalar registers
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l = threadIdx.x & 63, lq = l & 31, hi = l >> 5;
  const int G = 1 << lg;
  const int rpb = kW8Qv >> lg;
  const uint32_t k_base = lds_addr(k_lds), v_base = lds_addr(v_lds);
  const int qv = 32 * w + lq;
  int g = blockIdx.x % hkv;  // (plain grid with queues: set from the claimed item)

  const uint32_t row_b = (uint32_t)(kv_stride * 2);
  const int tg = l >> 4, te = (l >> 2) & 3, tq = l & 3;
  const int vrd = (4 * (tg >> 1) + te) * VSTR + 16 * (tg & 1) + 4 * tq;
  const int krd = lq * KSTR + 8 * hi;
  typedef short v4s __attribute__((ext_vector_type(4)));
  typedef v4s __attribute__((address_space(3))) * lds_v4s;
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

  // One segment: keys [kt_lo, kt_hi) of row tile `tile` of a request whose rows
  // start at r0 (nr of them) and whose keys start at kv0 (nkv of them); the
  // result is final (slot < 0) or partial slot `slot` of the workspace.
  auto segment = [&](int64_t r0, int nr, int64_t kv0, int nkv, int tile, int kt_lo, int kt_hi,
                     int64_t slot) {
    const int rl = tile * rpb + (qv >> lg);
    const int head = g * G + (qv & (G - 1));
    const int64_t grow = r0 + rl;
    const bool valid = rl < nr && grow < n_rows;

    // descriptors over this request's rows of KV head g: the last byte in range
    // is the end of the last key's head slice
    const uint32_t range = nkv > 0 ? (uint32_t)(nkv - 1) * row_b + D * 2 : 0u;
    const i32x4 rk = make_rsrc(kc + kv0 * kv_stride + (int64_t)g * D, range);
    const i32x4 rv = make_rsrc(vc + kv0 * kv_stride + (int64_t)g * D, range);
    // this wave's transfer slots: j = w + 8 i over the K then the V chunks of a stage,
    // or, split, j = (w & 3) + 4 i over the K chunks (waves 0-3) or the V chunks
    // (waves 4-7).  Slot j fills chunks [64 j, 64 j + 64) of its tile; lane l fills
    // chunk 64 j + l = (row, column) of the padded tile.
    const bool vwave = kDefer && w >= 4;
    uint32_t soff[SPWX];
    bool sk[SPWX];  // slot i fills K chunks
    int sj[SPWX];   // chunk slot within its tile
#pragma unroll
    for (int i = 0; i < SPWX; ++i) {
      int j;
      if (kDefer) {
        j = (w & 3) + 4 * i;
        sk[i] = !vwave;
      } else {
        j = w + kW8 * i;
        sk[i] = j < KCH;
        if (!sk[i]) j -= KCH;
      }
      const int ch = sk[i] ? KCH : VCH;  // chunks per row of the slot's tile
      sj[i] = j;
      const int ci = j * 64 + l;
      const int r = ci / ch, c = ci % ch;
      soff[i] = (j < ch && c < D / 8) ? (uint32_t)r * row_b + c * 16 : kOob;
    }
    const int nslots = kDefer ? (vwave ? (VCH - (w & 3) + 3) / 4 : (KCH - (w & 3) + 3) / 4)
                              : (w < NFULL ? SPW : SPW - 1);
    // the transfers of one step: tile r (relative to the segment's first tile)
    // into stage r % 4, K and V (split: this wave's part, K or V); a tile past the
    // segment's end reads zeros
    const int t0 = kt_lo / kKT;
    const int nt = kt_hi > kt_lo ? (kt_hi - kt_lo + kKT - 1) / kKT : 0;
    auto issue = [&](int r) {
      const int sg = r & (kStages - 1);
      const uint32_t toff = (uint32_t)((t0 + r) * kKT) * row_b;
#pragma unroll
      for (int i = 0; i < SPWX; ++i) {
        if (i >= nslots) break;
        const uint32_t off = r < nt ? soff[i] + toff : kOob;
        if (sk[i])
          dma16(rk, off, k_base + (uint32_t)(sg * KST + sj[i] * 512) * 2u);
        else
          dma16(rv, off, v_base + (uint32_t)(sg * VST + sj[i] * 512) * 2u);
      }
    };
    // The first three key tiles go out before anything waits on memory (every
    // LDS read of the previous segment ended at its last barrier), then the
    // row positions and Q.
    issue(0);
    issue(1);
    if (!vwave) issue(2);  // split: V runs two tiles ahead (see the ring below)
    // unconditional loads from a real row (a load under a lane condition gets a
    // wait of its own, which would also wait for the tiles above); a padding
    // lane's Q only has to be finite: its keys are all masked
    const int64_t crow = min(grow, n_rows - 1);
    const int pos_raw = row_pos[crow];
    bf16x8 qreg[D / 16];
    {
      // with kRot the query rows are un-rotated, read through q_src when it is given
      int64_t qrow = crow;
      if (kRot && q_src) qrow = min(max((int64_t)q_src[crow], (int64_t)0), n_q_src - 1);
      const uint16_t* qp = q + qrow * (int64_t)hq * D + (int64_t)head * D + 8 * hi;
#pragma unroll
      for (int st = 0; st < D / 16; ++st) qreg[st] = as_bf16x8(ld16(qp + 16 * st));
    }
    if (kRot) rotate_query<D>(qreg, rtab + (int64_t)min(max(pos_raw, 0), n_tab - 1) * (D / 2), hi);
    const int qpos = valid ? pos_raw : INT_MIN;
    const int wmax = wave_max_i(valid ? qpos : -1);
    const int wmin = wave_min_i(valid ? qpos : INT_MAX);
    const int wave_end = min(nkv, wmax + 1);
    f32x16 o[D / 32];
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb) o[mb] = f32x16{};
    float m = valid ? -1e30f : INFINITY;
    float ls = 0.f;

    // end of a step: this step's transfers may stay in flight, all older ones
    // (and every LDS read) are complete, then the block meets
    auto step_barrier = [&]() {
      asm volatile("" ::: "memory");
      if (nslots == SPWX) wait_vm_lgkm0<SPWX>();
      else wait_vm_lgkm0<SPWX - 1>();
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
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
    // S(t+1) = K Q^T beside P(t) = exp2(S(t) * scale2 - m), as one sequence of groups fenced
    // with sched_barrier, one product each: group i issues the K fragment of product i + 4
    // (four LDS reads in flight, where the compiler's own order waited on each read just
    // before its product), product i, the exponent arguments of group i + 1's elements, the
    // exponentials of its own and the sum and bf16 pack of group i - 1's.  Same operations
    // and the same order of the row sum as qk_half twice + softmax_exp, so bit-identical (c4
    // -1.2%, c5 -1.8%).  Plain mode only: the stream kernel has fewer registers to spare and
    // spilled with it.
    auto qk_exp_fused = [&](const uint16_t* kl, f32x16 (&sn)[2], f32x16 (&sc)[2], bf16x8 (&pb)[2][2]) {
      constexpr int NS = D / 16;    // products per 32-key half
      constexpr int NM = 2 * NS;    // products per tile
      constexpr int EG = 32 / NM;   // elements of the tile per group (2 at D = 128)
      constexpr int PF = 4;         // K fragments in flight
      static_assert(EG % 2 == 0 && EG * NM == 32, "groups cover the tile in element pairs");
      auto kfrag = [&](int i) { return as_bf16x8(ld16(kl + (i / NS) * 32 * KSTR + 16 * (i % NS))); };
      bf16x8 kf[NM];
#pragma unroll
      for (int i = 0; i < PF; ++i) kf[i] = kfrag(i);
      const float nm = -m;
      float psum = 0.f;
      float x[32], p[32];  // element e = 16 hb + v of the tile
      auto arg = [&](int g) {
#pragma unroll
        for (int e = EG * g; e < EG * (g + 1); ++e) x[e] = fmaf(sc[e / 16][e % 16], scale2, nm);
      };
      auto sum_pack = [&](int g) {
#pragma unroll
        for (int e = EG * g; e < EG * (g + 1); e += 2) {
          const int v = e % 16;
          psum += p[e];
          psum += p[e + 1];
          const bf16x2_t pk = __builtin_convertvector((f32x2_t){p[e], p[e + 1]}, bf16x2_t);
          pb[e / 16][v >> 3][v & 7] = pk[0];
          pb[e / 16][v >> 3][(v & 7) + 1] = pk[1];
        }
      };
      arg(0);
#pragma unroll
      for (int i = 0; i < NM; ++i) {
        __builtin_amdgcn_sched_barrier(0);
        if (i + PF < NM) kf[i + PF] = kfrag(i + PF);
        const int hb = i / NS, st = i % NS;
        sn[hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[i], qreg[st], st == 0 ? f32x16{} : sn[hb],
                                                         0, 0, 0);
        if (i + 1 < NM) arg(i + 1);
#pragma unroll
        for (int e = EG * i; e < EG * (i + 1); ++e) p[e] = __builtin_amdgcn_exp2f(x[e]);
        if (i > 0) sum_pack(i - 1);
      }
      __builtin_amdgcn_sched_barrier(0);
      sum_pack(NM - 1);
      ls += psum;
    };
    // O += P V as a fenced sequence of products, each issuing the V fragment (two transposed
    // reads) of the product four places ahead: the compiler's own order read eight fragments
    // at a time and waited at the head of every batch (bit-identical; c4 -0.8%, c5 -1.0%,
    // c2 (stream mode) -4%).
    auto pv = [&](const uint16_t* vl, bf16x8 (&pb)[2][2]) {
      constexpr int NB = D / 32;
      constexpr int NM = 4 * NB;  // products, ordered (hb, k2, mb)
      constexpr int PF = 4;       // V fragments in flight
      auto vfrag = [&](int j) {
        const int hb = j / (2 * NB), k2 = (j / NB) % 2, mb = j % NB;
        const uint16_t* p0 = vl + (hb * 32 + 16 * k2) * VSTR + 32 * mb;
        const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p0));
        const v4s up = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s)(p0 + 8 * VSTR));
        return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      bf16x8 vf[NM];
#pragma unroll
      for (int j = 0; j < PF; ++j) vf[j] = vfrag(j);
#pragma unroll
      for (int j = 0; j < NM; ++j) {
        __builtin_amdgcn_sched_barrier(0);
        if (j + PF < NM) vf[j + PF] = vfrag(j + PF);
        const int hb = j / (2 * NB), k2 = (j / NB) % 2, mb = j % NB;
        o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[j], pb[hb][k2], o[mb], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    };

    // Ring: K(t) and V(t) live in stage t % 4.  Step t computes S(t+1) while the
    // softmax of tile t runs, then issues tile t+3 into the stage of tile t-1
    // (its K was last read in step t-2, its V in step t-1), then O += P(t) V(t);
    // at its end everything issued before step t -- K(t+2) and V(t+1) among it
    // -- has landed.  Past the last tile the transfers still go out (zeros, no
    // memory traffic), so every step issues the same number of them.  Issued
    // at the start of the step instead, the transfers delayed the softmax
    // (c2 call +4%, c5 +1.5%).
    // Split (plain mode): waves 4-7 start step t with O += P(t-1) V(t-1), then issue
    // V(t+2) into the stage of tile t-2 (their last read of it was in step t-1; V(t-1)
    // stays in place), then run the softmax of tile t, which may rescale O, beside
    // S(t+1).  Waves 0-3 run the step as above with K(t+3) only.  On every SIMD one
    // wave's product-only part then meets the other's vector part, where the two
    // used to reach the same part together (c4 -3.4%, c5 -6.3%, bit-identical: the
    // order of the products into O is unchanged).  A last barrier after the loop
    // covers the final deferred product.
    f32x16 sa[2], sb[2];
    asm volatile("" ::: "memory");
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (nt > 0 && kt_lo < wave_end) {
      qk_half(k_lds + krd, 0, sa[0]);
      qk_half(k_lds + krd, 1, sa[1]);
    }
    bf16x8 pb[2][2];
    bool pend = false;  // split, waves 4-7: pb holds P of the previous tile
    auto step = [&](int t, f32x16 (&sc)[2], f32x16 (&sn)[2]) {
      const int kt0 = kt_lo + t * kKT;
      const bool do_cur = kt0 < wave_end;
      const bool do_next = t + 1 < nt && kt0 + kKT < wave_end;
      if (vwave) {
        if (pend) pv(v_lds + ((t - 1) & 3) * VST + vrd, pb);
        issue(t + 2);
      }
      if (do_cur) softmax_pre(sc, kt0);
      // The wave issuing this block (the next tile's products interleaved with this tile's
      // exponentials, the step's vector-heavy part) goes first at the SIMD's arbiter; the
      // other wave of the SIMD fills the remaining issue slots, often with its P.V
      // products (c4 4887 -> 4804 us, c5 -1.8%, bit-identical).
      __builtin_amdgcn_s_setprio(1);
      if (do_next) {
        const uint16_t* kn = k_lds + ((t + 1) & 3) * KST + krd;
        if constexpr (!kStream) {
          qk_exp_fused(kn, sn, sc, pb);
        } else {
          qk_half(kn, 0, sn[0]);
          qk_half(kn, 1, sn[1]);
          softmax_exp(sc, pb);
#pragma unroll
          for (int i = 0; i < D / 8; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
          }
        }
      } else if (do_cur) {
        softmax_exp(sc, pb);
      }
      __builtin_amdgcn_s_setprio(0);
      if (vwave) {
        pend = do_cur;
      } else {
        issue(t + 3);
        if (do_cur) pv(v_lds + (t & 3) * VST + vrd, pb);
      }
      step_barrier();
    };
    for (int t = 0; t < nt; t += 2) {
      step(t, sa, sb);
      if (t + 1 < nt) step(t + 1, sb, sa);
    }
    if (kDefer && nt > 0) {
      if (pend) pv(v_lds + ((nt - 1) & 3) * VST + vrd, pb);
      step_barrier();
    }
    // drain the last (zero-row) transfers before the LDS is refilled or released
    asm volatile("" ::: "memory");
    wait_vm_lgkm0<0>();

    const float lt = ls + __shfl_xor(ls, 32, 64);
    if (!valid) return;
    if (slot < 0) {
      uint16_t* op = out + grow * (int64_t)hq * D + (int64_t)head * D;
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
    // partial: this segment's O normalised by its own sum, in bf16 (half the
    // traffic of float32; |O / sum| <= max |v|, so one bf16 rounding of the
    // output scale), and its (max, sum) in float32.  Lanes l and l^32 write
    // the two halves of each 16-byte piece; the L2 joins them into full lines.
    uint16_t* po = part_o + (slot * kW8Qv + qv) * D;
    const float pinv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<uint2*>(po + 32 * mb + 8 * i + 4 * hi) =
            make_uint2(pack_bf16x2(o[mb][4 * i] * pinv, o[mb][4 * i + 1] * pinv),
                       pack_bf16x2(o[mb][4 * i + 2] * pinv, o[mb][4 * i + 3] * pinv));
    if (hi == 0) part_ml[slot * kW8Qv + qv] = make_float2(m, lt);
  };

  if (!kStream) {
    // plain: this block's row tile, all of its keys (up to its largest row
    // position).  The blocks of one KV head run the requests one after another,
    // longest (most keys) first, each request's tiles last row tile first:
    // the blocks that share an XCD then stream the same request's keys through
    // its L2, and the shortest work comes last.
    int tile, b = 0;
    if (queue) {
      // One request with many row tiles: the items (row tile, KV head) in the order
      // above are handed out by counters in the workspace.  Queue j holds the tiles
      // of KV heads j, j + nq, ...; a block takes from the queue of its XCD (whose L2
      // then serves one head's keys to all of its CUs) and, once that one is empty,
      // from another that still has items.  Under load the XCDs run at different
      // clocks, so the fast ones take over tiles that a fixed share per XCD would
      // leave to the slow ones at the end.  The grid holds spare blocks for that; a
      // block that finds every queue empty ends at once.
      const int nq = hkv < kQueues ? hkv : kQueues;
      const int home = (int)((__builtin_amdgcn_s_getreg(kHwRegXccId) & 15u) % (uint32_t)nq);
      uint32_t first_claim = 0;  // goes out before the request's row count is read
      if (threadIdx.x == 0) first_claim = atomicAdd(queue + kQueueStride * home, 1u);
      const int ntl = min(max_tiles, (max(cu_rows[1] - cu_rows[0], 0) + rpb - 1) / rpb);
      auto items_of = [&](int j) { return ntl * ((hkv - j + nq - 1) / nq); };
      // q_next is written only after a barrier that follows every wave's last read of
      // it; everything derived from it is wave-uniform (scalar registers)
      auto claim = [&](int j) {
        __syncthreads();
        if (threadIdx.x == 0) q_next = (int)atomicAdd(queue + kQueueStride * j, 1u);
        __syncthreads();
        return __builtin_amdgcn_readfirstlane(q_next);
      };
      auto next_queue = [&](int from) {  // the first queue after `from` with items left, or -1
        __syncthreads();
        if (w == 0) {
          const int c = l < nq ? (int)__hip_atomic_load(queue + kQueueStride * l, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT)
                               : 0;
          const bool left = l < nq && c < items_of(l);
          const int dist = wave_min_i(left ? (l - from - 1 + 2 * nq) % nq : INT_MAX);
          if (l == 0) q_next = dist == INT_MAX ? -1 : (from + 1 + dist) % nq;
        }
        __syncthreads();
        return __builtin_amdgcn_readfirstlane(q_next);
      };
      int qj = home;
      if (threadIdx.x == 0) q_next = (int)first_claim;
      __syncthreads();
      int item = __builtin_amdgcn_readfirstlane(q_next);
      while (item >= items_of(qj)) {  // (each failed claim finds a queue empty for good)
        qj = next_queue(home);
        if (qj < 0) return;
        item = claim(qj);
      }
      const int hj = items_of(qj) / ntl;  // KV heads of queue qj
      const int u = item / hj;
      tile = ntl - 1 - u;
      g = qj + nq * (item - u * hj);
    } else {
      const int rest = blockIdx.x / hkv;
      const int rank = rest / max_tiles;
      tile = max_tiles - 1 - (rest - rank * max_tiles);
      b = rank;
      if (batch > 1 && batch <= 64) {
        // rank of lane j's request: requests with more keys, or as many and a lower index
        const int nk = l < batch ? cu_kv[l + 1] - cu_kv[l] : -1;
        int rk = 0;
        for (int x = 0; x < batch; ++x) {
          const int nx = __shfl(nk, x, 64);
          rk += (nx > nk || (nx == nk && x < l)) ? 1 : 0;
        }
        const uint64_t hit = __ballot(l < batch && rk == rank);
        b = __builtin_amdgcn_readfirstlane(hit ? (int)__builtin_ctzll(hit) : rank);
      }
    }
    const int64_t r0 = cu_rows[b];
    const int nr = cu_rows[b + 1] - (int)r0;
    if (tile * rpb >= nr) return;
    const int64_t kv0 = cu_kv[b];
    int nkv = cu_kv[b + 1] - (int)kv0;
    if (kv0 + nkv > n_kv_rows) nkv = (int)(n_kv_rows - kv0);
    const int rl = tile * rpb + (qv >> lg);
    const int pos_raw = row_pos[min(r0 + rl, n_rows - 1)];
    const int mx = wave_max_i(rl < nr && r0 + rl < n_rows ? pos_raw : -1);
    if (l == 0) red[w] = mx;
    __syncthreads();
    int bmax = red[0];
#pragma unroll
    for (int i = 1; i < kW8; ++i) bmax = max(bmax, red[i]);
    segment(r0, nr, kv0, nkv, tile, 0, min(nkv, bmax + 1), -1);
    return;
  }

  // stream: the plan (key end and step count of every row tile), built by
  // each block in LDS.  The requests' row and key offsets come first; then
  // wave w takes tiles w, w+8, ... four at a time (their position loads are
  // independent), its lanes splitting each tile's rows.
  const int n_tiles = batch * max_tiles;
  for (int i = threadIdx.x; i <= batch; i += kW8 * 64) {
    req_rows[i] = cu_rows[i];
    req_kv[i] = cu_kv[i];
  }
  __syncthreads();
  auto req_nkv = [&](int b) {
    const int64_t kv0 = req_kv[b];
    const int nkv = req_kv[b + 1] - (int)kv0;
    return kv0 + nkv > n_kv_rows ? (int)(n_kv_rows - kv0) : nkv;
  };
  for (int i0 = w; i0 < n_tiles; i0 += 4 * kW8) {
    // all position loads of the four tiles go out before any is used (clamped
    // to a real row, masked afterwards)
    constexpr int RR = kW8Qv / 64;  // lanes' passes over a tile's rows (rows per tile <= kW8Qv)
    int pv[4][RR];
    bool ok[4][RR];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = min(i0 + u * kW8, n_tiles - 1);
      const int b = i / max_tiles, tile = i - b * max_tiles;
      const int64_t r0 = req_rows[b];
      const int nr = req_rows[b + 1] - (int)r0;
#pragma unroll
      for (int k = 0; k < RR; ++k) {
        const int rr = tile * rpb + l + 64 * k;
        ok[u][k] = i0 + u * kW8 < n_tiles && l + 64 * k < rpb && rr < nr && r0 + rr < n_rows;
        pv[u][k] = row_pos[min(r0 + rr, n_rows - 1)];
      }
    }
    int mx[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      mx[u] = -1;
#pragma unroll
      for (int k = 0; k < RR; ++k) mx[u] = max(mx[u], ok[u][k] ? pv[u][k] : -1);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = i0 + u * kW8;
      const int m_all = wave_max_i(mx[u]);
      if (l == 0 && i < n_tiles) plan_end[i] = max(0, min(req_nkv(i / max_tiles), m_all + 1));
    }
  }
  __syncthreads();
  if (w == 0) {
    // exclusive scan of the tiles' costs, start-up plus key steps
    // (kMaxStreamTiles / 64 tiles per lane)
    constexpr int PL = kMaxStreamTiles / 64;
    int loc[PL], sum = 0;
#pragma unroll
    for (int k = 0; k < PL; ++k) {
      const int i = l * PL + k;
      const int nst = i < n_tiles ? (plan_end[i] + kKT - 1) / kKT : 0;
      loc[k] = nst > 0 ? nst + kSegCost : 0;
      sum += loc[k];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, 64);
      if (l >= o) incl += y;
    }
    int run = incl - sum;
#pragma unroll
    for (int k = 0; k < PL; ++k) {
      const int i = l * PL + k;
      if (i < n_tiles) plan_cum[i] = run;
      run += loc[k];
    }
    if (l == 63) plan_cum[n_tiles] = incl;
  }
  __syncthreads();
  if (blockIdx.x == 0) {  // the merge kernel reads the same plan
    for (int i = threadIdx.x; i <= n_tiles; i += kW8 * 64) plan_out[i] = plan_cum[i];
    for (int i = threadIdx.x; i < n_tiles; i += kW8 * 64) plan_out[kPlanEndOff + i] = plan_end[i];
  }
  // this block's range [lo, hi_s) of the head's cost line; tile i occupies
  // [plan_cum[i], plan_cum[i+1]): kSegCost start-up units, then its key steps
  const int r = blockIdx.x / hkv;
  const int64_t S = plan_cum[n_tiles];
  int lo = (int)(r * S / nbg);
  const int hi_s = (int)((r + 1) * S / nbg);
  if (g == 0 && threadIdx.x == 0) {  // the range boundaries, for the merge
    plan_out[kPlanBndOff + r] = lo;
    if (r == nbg - 1) plan_out[kPlanBndOff + nbg] = hi_s;
  }
  int i = 0;
  bool first = true;
  while (lo < hi_s) {
    while (plan_cum[i + 1] <= lo) ++i;  // skip tiles without steps
    const int c1 = plan_cum[i + 1], a = plan_cum[i] + kSegCost;  // key step 0 at a
    const int s_lo = max(lo, a), s_hi = min(hi_s, c1);
    if (s_lo < s_hi) {
      const int b = i / max_tiles, tile = i - b * max_tiles;
      const bool whole = s_lo == a && s_hi == c1;
      const int64_t slot = whole ? -1 : ((int64_t)(g * nbg + r) * 2 + (first ? 0 : 1));
      const int64_t r0 = req_rows[b];
      segment(r0, req_rows[b + 1] - (int)r0, req_kv[b], req_nkv(b), tile, (s_lo - a) * kKT,
              min(plan_end[i], (s_hi - a) * kKT), slot);
      first = false;
    }
    lo = c1;
  }
}

// Sets the plain grid's work counters to zero before the grid starts (a kernel
// rather than a memset, so that the call can be captured in a graph).
__global__ void attn_queue_reset_kernel(uint32_t* __restrict__ queue) {
  if (threadIdx.x < kQueues) queue[kQueueStride * threadIdx.x] = 0u;
}

// Combines the stream-mode partials of each row tile that a range boundary
// cut: the blocks r_first .. r_last of the tile's KV head each hold one
// segment (in slot 0 if the segment is the block's first, else slot 1); they
// are combined in block order (deterministic).  One block per (row tile, KV
// head).
template <int D>
__global__ __launch_bounds__(kThreads) void attn_stream_merge_kernel(
    uint16_t* __restrict__ out, float* __restrict__ lse, int64_t n_rows,
    const int32_t* __restrict__ cu_rows, int batch, int max_tiles, int hkv, int hq, int lg,
    int nbg, const int32_t* __restrict__ plan, const uint16_t* __restrict__ part_o,
    const float2* __restrict__ part_ml) {
  constexpr int QV = kW8Qv;
  constexpr int QQ = QV / 4;  // query vectors per merge block (a quarter of the tile)
  constexpr int WS = 8;       // split weights kept in LDS; later ones are recomputed
  __shared__ float wgt[WS][QQ];
  __shared__ float mxq[QQ], invq[QQ];
  __shared__ int64_t slot_l[kStreamBlocks];
  __shared__ int bnd_l[kStreamBlocks + 1];
  __shared__ int nsp_l;
  const int quarter = blockIdx.x & 3;
  const int i = (blockIdx.x >> 2) / hkv, g = (blockIdx.x >> 2) % hkv;
  const int n_tiles = batch * max_tiles;
  if (i >= n_tiles) return;
  // the blocks' range boundaries go to LDS while the tile's own entries load
  for (int t = threadIdx.x; t <= nbg; t += kThreads) bnd_l[t] = plan[kPlanBndOff + t];
  const int S = plan[n_tiles];
  const int c0 = plan[i], c1 = plan[i + 1];
  if (c1 <= c0 || S == 0) return;
  __syncthreads();
  const int a = c0 + kSegCost;  // the tile's first key step on the cost line
  // block holding step x: the largest r whose range starts at or before x
  auto owner = [&](int x) {
    int a = 0, z = nbg - 1;
    while (a < z) {
      const int mid = (a + z + 1) >> 1;
      if (bnd_l[mid] <= x) a = mid; else z = mid - 1;
    }
    return a;
  };
  const int rf = owner(a), rlst = owner(c1 - 1);
  if (rf == rlst) return;  // one block did the whole tile
  // the blocks with a non-empty range between them, in order (with fewer steps
  // than blocks some ranges are empty); the first block's segment sits in its
  // slot 1 when its range began before this tile (it then did a segment of an
  // earlier tile first), every other one's in slot 0
  if (threadIdx.x == 0) {
    int n = 0;
    for (int rr = rf; rr <= rlst; ++rr) {
      const int lo_r = bnd_l[rr], hi_r = bnd_l[rr + 1];
      if (hi_r <= lo_r) continue;
      slot_l[n++] = (int64_t)(g * nbg + rr) * 2 + (lo_r < c0 ? 1 : 0);
    }
    nsp_l = n;
  }
  __syncthreads();
  const int nsp = nsp_l;
  const int b = i / max_tiles, tile = i - b * max_tiles;
  const int G = 1 << lg;
  const int rpb = QV >> lg;
  const int64_t r0 = cu_rows[b];
  const int nr = cu_rows[b + 1] - (int)r0;
  const int rbase = tile * rpb;
  const int qv0 = quarter * QQ;
  // Every load of the first kMR partials (their O pieces and, for the first
  // QQ threads, their (max, sum)) is issued before any is used, from clamped
  // slots; later partials (rare) follow one at a time.
  constexpr int kPass = kThreads * 8;
  constexpr int NP = QQ * D / kPass;
  constexpr int kMR = 4;
  uint4 ob[kMR][NP];
#pragma unroll
  for (int sp = 0; sp < kMR; ++sp) {
    const uint16_t* pp = part_o + (slot_l[min(sp, nsp - 1)] * QV + qv0) * D;
#pragma unroll
    for (int p = 0; p < NP; ++p) ob[sp][p] = ld16(pp + p * kPass + 8 * threadIdx.x);
  }
  if (threadIdx.x < QQ) {
    const int qv = qv0 + threadIdx.x;
    float2 mlr[kMR];
#pragma unroll
    for (int sp = 0; sp < kMR; ++sp) mlr[sp] = part_ml[slot_l[min(sp, nsp - 1)] * QV + qv];
    float mx = -1e30f;
#pragma unroll
    for (int sp = 0; sp < kMR; ++sp)
      if (sp < nsp) mx = fmaxf(mx, mlr[sp].x);
    for (int sp = kMR; sp < nsp; ++sp) mx = fmaxf(mx, part_ml[slot_l[sp] * QV + qv].x);
    // split sp's weight on its normalised partial: 2^(m_sp - max) * l_sp / total
    float lsum = 0.f;
#pragma unroll
    for (int sp = 0; sp < kMR; ++sp) {
      if (sp < nsp) {
        const float wsp = __builtin_amdgcn_exp2f(mlr[sp].x - mx) * mlr[sp].y;
        wgt[sp][threadIdx.x] = wsp;
        lsum += wsp;
      }
    }
    for (int sp = kMR; sp < nsp; ++sp) {
      const float2 ml = part_ml[slot_l[sp] * QV + qv];
      const float wsp = __builtin_amdgcn_exp2f(ml.x - mx) * ml.y;
      if (sp < WS) wgt[sp][threadIdx.x] = wsp;
      lsum += wsp;
    }
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    for (int sp = 0; sp < nsp && sp < WS; ++sp) wgt[sp][threadIdx.x] *= inv;
    mxq[threadIdx.x] = mx;
    invq[threadIdx.x] = inv;
    const int rl = rbase + (qv >> lg);
    const int64_t grow = r0 + rl;
    if (lse && rl < nr && grow < n_rows)
      lse[grow * hq + g * G + (qv & (G - 1))] = lsum > 0.f ? (mx + log2f(lsum)) * kLn2 : -INFINITY;
  }
  __syncthreads();
  // QQ x D outputs, 8 consecutive ones per thread and pass; partials combined in order
  float acc[NP][8];
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[p][k] = 0.f;
  auto add_partial = [&](int sp, const uint4* o) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const int e = p * kPass + 8 * threadIdx.x;
      const int ql = e / D;
      float wv;
      if (sp < WS) {
        wv = wgt[sp][ql];
      } else {
        const float2 ml = part_ml[slot_l[sp] * QV + qv0 + ql];
        wv = __builtin_amdgcn_exp2f(ml.x - mxq[ql]) * ml.y * invq[ql];
      }
      float x[8];
      Vec16<uint16_t>::unpack(o[p], x);
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[p][k] += wv * x[k];
    }
  };
#pragma unroll
  for (int sp = 0; sp < kMR; ++sp)
    if (sp < nsp) add_partial(sp, ob[sp]);
  for (int sp = kMR; sp < nsp; ++sp) {
    uint4 o[NP];
    const uint16_t* pp = part_o + (slot_l[sp] * QV + qv0) * D;
#pragma unroll
    for (int p = 0; p < NP; ++p) o[p] = ld16(pp + p * kPass + 8 * threadIdx.x);
    add_partial(sp, o);
  }
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int e = p * kPass + 8 * threadIdx.x;
    const int qv = qv0 + e / D, dd = e % D;
    const int rl = rbase + (qv >> lg);
    const int64_t grow = r0 + rl;
    if (rl >= nr || grow >= n_rows) continue;
    const int head = g * G + (qv & (G - 1));
    *reinterpret_cast<uint4*>(out + grow * (int64_t)hq * D + (int64_t)head * D + dd) =
        make_uint4(pack_bf16x2(acc[p][0], acc[p][1]), pack_bf16x2(acc[p][2], acc[p][3]),
                   pack_bf16x2(acc[p][4], acc[p][5]), pack_bf16x2(acc[p][6], acc[p][7]));
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

// Stream mode is used when the plain grid would hold fewer than 1.5 blocks per
// CU and the row tiles fit the block's plan.  (A c3-shaped layer, 392 plain
// blocks: plain 284 vs stream 297 us; c2, 200 blocks: plain 132 vs stream
// 103 us.)  Its workspace: the plan (step prefix sums and key ends of up to
// kMaxStreamTiles row tiles) and two partial slots per block.

bool use_stream(const AttnShape& s, int max_tiles) {
  const int64_t plain_blocks = (int64_t)max_tiles * s.batch * s.hkv;
  return 2 * plain_blocks < 3 * kStreamBlocks && (int64_t)max_tiles * s.batch <= kMaxStreamTiles &&
         s.max_kv > kKT;
}

struct StreamLayout {
  int nbg;
  size_t plan_off, o_off, ml_off, queue_off, bytes;
};

StreamLayout stream_layout(const AttnShape& s) {
  StreamLayout L{};
  L.nbg = std::max(1, kStreamBlocks / s.hkv);
  const size_t slots = (size_t)L.nbg * s.hkv * 2;
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  L.plan_off = 0;
  L.o_off = a256(kPlanInts * sizeof(int32_t));
  L.ml_off = L.o_off + a256(slots * kW8Qv * s.d * sizeof(uint16_t));
  L.queue_off = L.ml_off + a256(slots * kW8Qv * sizeof(float2));
  L.bytes = L.queue_off + kQueues * kQueueStride * sizeof(uint32_t);  // the work counters
  return L;
}

// Compute units of the current device.
int cu_count() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return kStreamBlocks;
  if (dev < 64 && cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = kStreamBlocks;
  if (dev < 64) cached[dev] = n;
  return n;
}

}  // namespace

size_t attn_workspace(const AttnShape& s, bool bf16) {
  // Every call that could choose stream mode needs the same layout (it only
  // depends on the heads and head_dim), so the size covers all smaller shapes.
  if (!bf16 || s.batch <= 0 || s.max_rows <= 0 || s.max_kv <= kKT) return 0;
  return stream_layout(s).bytes;
}

hipError_t launch_sparse_attn(void* out, float* lse, const void* q, const int32_t* row_pos,
                              int64_t n_rows, const int32_t* cu_rows, const void* k_cache,
                              const void* v_cache, int64_t n_kv_rows, int64_t kv_row_stride,
                              const int32_t* cu_kv, const int32_t* kv_pos, bool bf16,
                              const AttnShape& s, float scale, void* ws, hipStream_t stream,
                              const QueryRot& qrot) {
  if (n_rows == 0 || s.batch == 0 || s.max_rows == 0) return hipSuccess;
  const bool rot = qrot.table != nullptr;
  if (rot && (!bf16 || kv_pos)) return hipErrorInvalidValue;
  const float2* rtab = reinterpret_cast<const float2*>(qrot.table);
  const float scale2 = scale * kLog2e;
  int lg = 0;
  while ((1 << lg) < s.hq / s.hkv) ++lg;
  if (bf16 && !kv_pos) {
    // recomputed rows: the 8-wave kernel (buffer offsets of one request's rows are 32-bit)
    if ((double)s.max_kv * (double)kv_row_stride * 2.0 >= 2147483648.0) return hipErrorInvalidConfiguration;
    const int max_tiles = (s.max_rows + (kW8Qv >> lg) - 1) / (kW8Qv >> lg);
    if (use_stream(s, max_tiles)) {
      const StreamLayout L = stream_layout(s);
      char* wb = static_cast<char*>(ws);
      int32_t* plan = reinterpret_cast<int32_t*>(wb + L.plan_off);
      uint16_t* part_o = reinterpret_cast<uint16_t*>(wb + L.o_off);
      float2* part_ml = reinterpret_cast<float2*>(wb + L.ml_off);
      dim3 grid((unsigned)(L.nbg * s.hkv));
#define QCF_W8S(D, R)                                                                             \
  attn_w8_kernel<D, true, R><<<grid, kW8 * 64, 0, stream>>>(                                      \
      static_cast<uint16_t*>(out), lse, static_cast<const uint16_t*>(q), row_pos, n_rows, cu_rows, \
      static_cast<const uint16_t*>(k_cache), static_cast<const uint16_t*>(v_cache), n_kv_rows,    \
      kv_row_stride, cu_kv, s.batch, max_tiles, s.hkv, s.hq, lg, scale2, L.nbg, plan, part_o,     \
      part_ml, qrot.src, qrot.n_src, rtab, (int)qrot.n_table, nullptr);                           \
  attn_stream_merge_kernel<D><<<dim3((unsigned)(4 * max_tiles * s.batch * s.hkv)), kThreads, 0,   \
                                 stream>>>(static_cast<uint16_t*>(out), lse, n_rows, cu_rows,      \
                                           s.batch, max_tiles, s.hkv, s.hq, lg, L.nbg, plan,       \
                                           part_o, part_ml)
      if (s.d == 64) {
        if (rot) { QCF_W8S(64, true); } else { QCF_W8S(64, false); }
      } else {
        if (rot) { QCF_W8S(128, true); } else { QCF_W8S(128, false); }
      }
#undef QCF_W8S
      return hipGetLastError();
    }
    const int64_t nblocks = (int64_t)max_tiles * s.batch * s.hkv;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblocks);
    // One request with at least four row tiles per CU: the tiles come from work queues
    // (counters in the workspace, reset by a kernel on the same stream), and an eighth
    // more blocks let the fast XCDs take tiles from the slow ones.  Measured on one box:
    // 32 x 1024-token context (9.7 tiles per CU) -1.7 to -2.1%, 16 x 1024 (4.9) -1%,
    // 8 x 1024 (2.4) +1.9%, ragged 16-request batch +1 to +2%, so fewer tiles or
    // several requests keep the fixed order.
    uint32_t* queue = nullptr;
    if (ws && s.batch == 1 && nblocks >= 4 * (int64_t)cu_count() &&
        nblocks + nblocks / 8 <= 0x7fffffff) {
      queue = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + stream_layout(s).queue_off);
      attn_queue_reset_kernel<<<1, 64, 0, stream>>>(queue);
      grid = dim3((unsigned)(nblocks + nblocks / 8));
    }
#define QCF_W8(D, R)                                                                              \
  attn_w8_kernel<D, false, R><<<grid, kW8 * 64, 0, stream>>>(                                     \
      static_cast<uint16_t*>(out), lse, static_cast<const uint16_t*>(q), row_pos, n_rows, cu_rows, \
      static_cast<const uint16_t*>(k_cache), static_cast<const uint16_t*>(v_cache), n_kv_rows,    \
      kv_row_stride, cu_kv, s.batch, max_tiles, s.hkv, s.hq, lg, scale2, 0, nullptr, nullptr,     \
      nullptr, qrot.src, qrot.n_src, rtab, (int)qrot.n_table, queue)
    if (s.d == 64) {
      if (rot) QCF_W8(64, true); else QCF_W8(64, false);
    } else {
      if (rot) QCF_W8(128, true); else QCF_W8(128, false);
    }
#undef QCF_W8
    return hipGetLastError();
  }
  if (bf16) {
    // explicit key positions (the anchor probe): the 4-wave kernel
    const int max_tiles = (s.max_rows + (128 >> lg) - 1) / (128 >> lg);
    const int64_t nblocks = (int64_t)max_tiles * s.batch * s.hkv;
    if (nblocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    dim3 grid((unsigned)nblocks);
#define QCF_POS(D)                                                                                \
  attn_pos_kernel<D><<<grid, kThreads, 0, stream>>>(                                              \
      static_cast<uint16_t*>(out), lse, static_cast<const uint16_t*>(q), row_pos, n_rows, cu_rows, \
      static_cast<const uint16_t*>(k_cache), static_cast<const uint16_t*>(v_cache), n_kv_rows,    \
      kv_row_stride, cu_kv, kv_pos, s.batch, max_tiles, s.hkv, s.hq, lg, scale2)
    if (s.d == 64) QCF_POS(64); else QCF_POS(128);
#undef QCF_POS
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
