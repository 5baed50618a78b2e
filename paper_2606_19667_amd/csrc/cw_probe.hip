// Device half of libcw for gfx950 (MI355X): a measurement aid, not a step of
// the attention path. It measures the bf16 matrix-instruction rate the card
// sustains on operands of a chosen value distribution, to set beside the
// data-sheet peak of the attention kernel's roofline: under its power limit
// the card lowers its clock by an amount that depends on the operand bits, so
// random bf16 data sustain a lower rate than constant data.
//
// Each wavefront keeps 8 independent 32x32 accumulators busy with
// v_mfma_f32_32x32x16_bf16 (4 A fragments x 2 B fragments, taken from the
// caller's operand buffer), two wavefronts per SIMD as in the attention kernel,
// and writes one float per lane so the work is not dead code.

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "cw_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 512;   // 8 wavefronts: two per SIMD
constexpr int kFragA = 4, kFragB = 2;
constexpr int kVecBytes = 64 * 16;   // one fragment: 16 bytes per lane

__global__ __launch_bounds__(kProbeThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void mfma_probe_kernel(const u32x4* __restrict__ ops, int64_t n_vec, float* __restrict__ sink, int iters) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t gw = int64_t(blockIdx.x) * (kProbeThreads / 64) + (tid >> 6);
  bf16x8 a[kFragA], b[kFragB];
#pragma unroll
  for (int i = 0; i < kFragA; ++i)
    a[i] = __builtin_bit_cast(bf16x8, ops[((gw * (kFragA + kFragB) + i) % n_vec) * 64 + lane]);
#pragma unroll
  for (int j = 0; j < kFragB; ++j)
    b[j] = __builtin_bit_cast(bf16x8, ops[((gw * (kFragA + kFragB) + kFragA + j) % n_vec) * 64 + lane]);
  f32x16 acc[kFragA * kFragB];
#pragma unroll
  for (int c = 0; c < kFragA * kFragB; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kFragA; ++i)
#pragma unroll
      for (int j = 0; j < kFragB; ++j)
        acc[i * kFragB + j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i * kFragB + j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kFragA * kFragB; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  sink[int64_t(blockIdx.x) * kProbeThreads + tid] = s;
}

}  // namespace

extern "C" int64_t cw_probe_mfma_bf16_flops(int32_t iters, int32_t workgroups) {
  if (iters < 1 || workgroups < 1) return -1;
  return int64_t(workgroups) * (kProbeThreads / 64) * iters * (kFragA * kFragB) * (2LL * 32 * 32 * 16);
}

extern "C" cw_status cw_probe_mfma_bf16(const void* operands, int64_t operand_bytes, float* sink, int32_t iters,
                                        int32_t workgroups, void* stream) {
  const char* what = "probe_mfma_bf16";
  if (!operands || !sink) return cw::fail(CW_EINVAL, std::string(what) + ": operands and sink are required");
  if (operand_bytes < int64_t(kVecBytes) * (kFragA + kFragB) || operand_bytes % kVecBytes != 0)
    return cw::fail(CW_EINVAL, std::string(what) + ": operand_bytes must be a multiple of 1024 and >= 6144");
  if (iters < 1 || workgroups < 1 || workgroups > (1 << 20))
    return cw::fail(CW_EINVAL, std::string(what) + ": iters >= 1 and 1 <= workgroups <= 2^20 are required");
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(unsigned(workgroups)), dim3(kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(operands),
                     operand_bytes / kVecBytes, sink, int(iters));
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return cw::fail(CW_EHIP, std::string(what) + " launch: " + hipGetErrorString(e));
  return cw::ok();
}
