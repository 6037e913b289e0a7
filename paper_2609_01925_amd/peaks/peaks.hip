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

// The same MFMA work on operands that change from one MFMA to the next: each lane holds
// 8 A and 8 B operands loaded from `ops` (any bits that are finite bf16 values, e.g.
// random normal values), and MFMA u of round-group g uses A[(u + c) % 8] and
// B[(3 u + c) % 8], so the multipliers' inputs toggle as they do on real data (the
// constant-operand loop above does not switch them and runs at a higher clock).
// ops: 64 lanes x 16 operands x 16 bytes, read by every wave.  iters is a multiple of 8.
__global__ __launch_bounds__(256) void peak_mfma_bf16_toggling(int iters, const bf16x8* __restrict__ ops,
                                                             float* out) {
  const int lane = threadIdx.x & 63;
  bf16x8 av[8], bv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    av[i] = ops[lane * 16 + i];
    bv[i] = ops[lane * 16 + 8 + i];
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.f;
  for (int it = 0; it < iters; it += 8) {
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int c = 0; c < kChains; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[(u + c) & 7], bv[(3 * u + c) & 7], acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[c][i];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

// dst[i] = src[i] over n16 16-byte words (reads n16 * 16 bytes and writes as many).  Each
// lane moves four words per step, loads first, so every lane keeps 64 bytes in flight;
// a grid-stride loop covers any size.
constexpr int kCopyUnroll = 4;

__global__ __launch_bounds__(256) void peak_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                 size_t n16) {
  const size_t lanes = (size_t)gridDim.x * blockDim.x;
  const size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t i = t;
  for (; i + (kCopyUnroll - 1) * lanes < n16; i += kCopyUnroll * lanes) {
    u32x4 r[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) r[u] = src[i + u * lanes];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) dst[i + u * lanes] = r[u];
  }
  for (; i < n16; i += lanes) dst[i] = src[i];
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

// As crisp_peak_mfma_bf16 with toggling operands; ops: 16 KiB (64 x 16 x 8 bf16, 16-byte
// aligned) of finite bf16 values; iters a multiple of 8.  Same FLOP count.
int crisp_peak_mfma_bf16_toggling(int workgroups, int iters, const void* ops, float* out, void* stream) {
  if (workgroups <= 0 || iters <= 0 || iters % 8 || !ops || !out || (uintptr_t)ops % 16)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(peak_mfma_bf16_toggling, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, iters,
                     (const bf16x8*)ops, out);
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
