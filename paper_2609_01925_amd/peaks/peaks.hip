// Peak-rate microbenchmarks for the measurement side (not part of the CRISP path):
// the bf16 MFMA rate the chip sustains under load and the HBM bandwidth of a plain
// device copy.  The roofline fractions of the attention, estimation and selection
// kernels are reported against these measured rates beside the published ones.
//
// C ABI (libcrisp_peaks.so); every call only enqueues one kernel on `stream` and
// returns a hipError_t as int (0 = success).
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

constexpr int kChains = 4;  // independent accumulators per wave (three waves per SIMD fit)

// Each wave runs `iters` rounds of kChains independent v_mfma_f32_32x32x16_bf16
// (32768 FLOP each) on register operands and writes one float per lane so the
// work is kept.  Operands are built from the lane id: any finite values will do.
__global__ __launch_bounds__(256) void peak_mfma_bf16(int iters, float* out) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((lane + i) & 7));
    b[i] = (__bf16)(0.001f * (float)((lane * 3 + i) & 7));
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[c][i];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// dst[i] = src[i] over n16 16-byte words, grid-stride, one 16-byte load and store per
// lane and step (reads n16 * 16 bytes and writes as many).
__global__ __launch_bounds__(256) void peak_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                 size_t n16) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    dst[i] = src[i];
}

}  // namespace

extern "C" {

// FLOP issued by one crisp_peak_mfma_bf16 call: workgroups * 4 waves * iters * kChains * 32768.
double crisp_peak_mfma_flop(int workgroups, int iters) {
  return (double)workgroups * 4.0 * (double)iters * kChains * 32768.0;
}

// out: float[workgroups * 256] on the device.
int crisp_peak_mfma_bf16(int workgroups, int iters, float* out, void* stream) {
  if (workgroups <= 0 || iters <= 0 || !out) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(peak_mfma_bf16, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, iters, out);
  return (int)hipGetLastError();
}

// Copies `bytes` (a multiple of 16; both pointers 16-byte aligned) from src to dst.
int crisp_peak_copy(const void* src, void* dst, size_t bytes, int workgroups, void* stream) {
  if (!src || !dst || bytes % 16 || ((uintptr_t)src | (uintptr_t)dst) % 16 || workgroups <= 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(peak_copy, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, (const u32x4*)src,
                     (u32x4*)dst, bytes / 16);
  return (int)hipGetLastError();
}

}  // extern "C"
