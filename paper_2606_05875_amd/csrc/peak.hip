// The matrix-core rate a plain loop of the attention's product instruction
// reaches on this part: not a step of the method, a yardstick for it.  The
// published bf16 peak assumes every SIMD issues v_mfma_f32_32x32x16_bf16 back
// to back at 2.4 GHz; under a sustained load the clock settles lower, and how
// far depends on the data the multipliers see.  The loop keeps two waves per
// SIMD (the attention's occupancy), four independent accumulators per wave,
// and operand fragments drawn from random bf16 data, rotated so that
// consecutive products see different operands.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qcf.h"
#include "qcf_device.h"

namespace qcf {
namespace {

constexpr int kLoopThreads = 256;  // four waves, one per SIMD
constexpr int kChains = 4;         // independent accumulators per wave
constexpr int kFrags = 4;          // operand fragments per lane and side
constexpr int kClockBlocks = 8;    // blocks that record clock counters (one per XCD)

__global__ __launch_bounds__(kLoopThreads) void mfma_loop_kernel(
    const uint16_t* __restrict__ ops, int64_t n_ops, float* __restrict__ sink, int64_t n_sink,
    uint64_t* __restrict__ clocks, int iters) {
  // each lane's fragments: 8 consecutive bf16 values per fragment from the operand
  // buffer, at lane- and block-dependent offsets (clamped inside the buffer)
  const int64_t base = ((int64_t)blockIdx.x * kLoopThreads + threadIdx.x) * (2 * kFrags * 8);
  bf16x8 a[kFrags], b[kFrags];
#pragma unroll
  for (int f = 0; f < kFrags; ++f) {
    const int64_t oa = (base + 16 * f) % (n_ops - 8);
    const int64_t ob = (base + 16 * f + 8) % (n_ops - 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[f][e] = __builtin_bit_cast(__bf16, ops[oa + e]);
      b[f][e] = __builtin_bit_cast(__bf16, ops[ob + e]);
    }
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  const bool stamp = blockIdx.x < kClockBlocks && threadIdx.x == 0;
  uint64_t r0 = 0, c0 = 0;
  if (stamp) {
    r0 = __builtin_amdgcn_s_memrealtime();
    c0 = __builtin_amdgcn_s_memtime();
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int u = 0; u < kFrags; ++u)
#pragma unroll
      for (int c = 0; c < kChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(u + c) % kFrags],
                                                         b[(u + 2 * c + 1) % kFrags], acc[c], 0, 0, 0);
  }
  if (stamp) {
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime(), c1 = __builtin_amdgcn_s_memtime();
    uint64_t* cl = clocks + 4 * blockIdx.x;
    cl[0] = r0;
    cl[1] = c0;
    cl[2] = r1;
    cl[3] = c1;
  }
  // every accumulator reaches memory, so no product can be dropped
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[c][v];
  const int64_t i = (int64_t)blockIdx.x * kLoopThreads + threadIdx.x;
  if (i < n_sink) sink[i] = s;
}

}  // namespace
}  // namespace qcf

extern "C" qcf_status qcf_mfma_loop(const void* operands, int64_t n_operands, float* sink,
                                    int64_t n_sink, uint64_t* clocks, int blocks, int iters,
                                    hipStream_t stream) {
  if (!operands || !sink || !clocks || n_operands < 16 || blocks <= 0 || iters <= 0 ||
      n_sink < (int64_t)blocks * qcf::kLoopThreads)
    return QCF_ERR_INVALID_ARG;
  if (blocks < qcf::kClockBlocks) return QCF_ERR_INVALID_ARG;
  qcf::mfma_loop_kernel<<<dim3((unsigned)blocks), qcf::kLoopThreads, 0, stream>>>(
      static_cast<const uint16_t*>(operands), n_operands, sink, n_sink, clocks, iters);
  return hipGetLastError() == hipSuccess ? QCF_OK : QCF_ERR_HIP;
}
