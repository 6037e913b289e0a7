// Peak-rate microbenchmarks for the measurement side (not part of the CRISP path):
// the bf16 MFMA rate the chip sustains under load, the HBM bandwidth of a plain
// device copy, the LDS read rates of the attention kernel's operand reads and the
// VALU issue cost of exp2 against a full-rate FMA.  The roofline fractions of the
// attention, estimation and selection kernels are reported against these measured
// rates beside the published ones.
//
// C ABI (libcrisp_peaks.so); every call only enqueues one kernel on `stream` and
// returns a hipError_t as int (0 = success).
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "crisp_device.h"

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

// LDS read rate in the attention kernel's operand patterns, clocked by the wave itself
// (s_memtime, core clock cycles).  Each wave issues `iters` rounds of 8 reads from a 32
// KiB LDS area and folds the data into one register, which is written out so the reads
// are kept.  kind 0: ds_read_b128 at the K operand offsets (16 bytes per lane, rows l %
// 32 of a swizzled 128-dim tile); kind 1: ds_read_b64_tr_b16 at the transposing V
// operand offsets (8 bytes per lane); kind 2: ds_read_b64 at the K offsets.  Every
// address lies inside the area.  cycles[wave] = the wave's cycles for all rounds.
// The LDS area is 64 KiB (reads use the first 32 KiB), so that at most two workgroups
// share a CU: 512 workgroups put eight waves on every CU, as the attention kernel does.
constexpr int kLdsBytes = 32768;
constexpr int kLdsAlloc = 65536;
template <int KIND>
__global__ __launch_bounds__(256) void peak_lds_read(int iters, unsigned long long* cycles, unsigned* sink) {
#if defined(__HIP_DEVICE_COMPILE__)
  __shared__ __attribute__((aligned(1024))) char area[kLdsAlloc];
  typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;
  typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
  typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
  typedef __attribute__((address_space(3))) crisp::i16x4 lds_i16x4;
  const int tid = threadIdx.x, l = tid & 63;
  const uint32_t base = (uint32_t)(size_t)area;
  int off[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    if (KIND == 1) {
      const int grp = l >> 4, jj = l & 15;
      const int row = 4 * (grp >> 1) + (jj >> 2) + 8 * (k & 1) + 16 * (k >> 2);
      const int col = 32 * ((k >> 1) & 1) + 16 * (grp & 1) + 4 * (jj & 3);
      off[k] = crisp::lds_off(row, col);
    } else {
      off[k] = crisp::lds_off((l & 31) + 32 * (k & 1), 16 * (k >> 1) + 8 * (l >> 5));
    }
  }
  unsigned acc = 0u;
  __syncthreads();
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  for (int it = 0; it < iters; ++it) {
    const uint32_t b = base + (uint32_t)((it & 1) * (kLdsBytes / 2));
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if (KIND == 0) {
        const u32x4 v = *(const lds_u32x4*)(b + off[k]);
        acc ^= v[0] ^ v[3];
      } else if (KIND == 1) {
        const crisp::i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(b + off[k]));
        acc ^= (unsigned)(uint16_t)v[0] ^ ((unsigned)(uint16_t)v[3] << 16);
      } else {
        const u32x2 v = *(const lds_u32x2*)(b + off[k]);
        acc ^= v[0] ^ v[1];
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  if (l == 0) cycles[(size_t)blockIdx.x * 4 + (tid >> 6)] = t1 - t0;
  sink[(size_t)blockIdx.x * 256 + tid] = acc;
#endif
}

// VALU issue cost: each wave runs `iters` rounds of 8 independent chains of one
// instruction each, kind 0: x = exp2(-x) (v_exp_f32; values stay in [0.5, 1]), kind 1:
// x = fma(x, 0.5, 0.25) (v_fma_f32, full rate), kind 2: x = exp2(-x) in half precision
// (v_exp_f16 on the low 16 bits; values stay in [0.5, 1]).  cycles[wave] as above.  The
// launch reserves 64 KiB of LDS (unused), so two workgroups share a CU and 512 workgroups
// give two waves per SIMD.
template <int KIND>
__global__ __launch_bounds__(256) void peak_valu(int iters, unsigned long long* cycles, float* sink) {
  const int tid = threadIdx.x, l = tid & 63;
  if constexpr (KIND == 2) {
    unsigned h[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) h[k] = 0x3800u + ((l + k) & 63);  // 0.5 + a few ulp, as half bits
    __syncthreads();
    const unsigned long long t0 = __builtin_amdgcn_s_memtime();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < 8; ++k) asm volatile("v_exp_f16 %0, -%0" : "+v"(h[k]));
    }
    unsigned sh = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) sh += h[k] & 0xffffu;
    const unsigned long long t1 = __builtin_amdgcn_s_memtime();
    if (l == 0) cycles[(size_t)blockIdx.x * 4 + (tid >> 6)] = t1 - t0;
    sink[(size_t)blockIdx.x * 256 + tid] = (float)sh;
    return;
  }
  float x[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = 0.5f + 0.001f * (float)((l + k) & 63);
  __syncthreads();
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = KIND == 0 ? __builtin_amdgcn_exp2f(-x[k]) : __builtin_fmaf(x[k], 0.5f, 0.25f);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += x[k];
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  if (l == 0) cycles[(size_t)blockIdx.x * 4 + (tid >> 6)] = t1 - t0;
  sink[(size_t)blockIdx.x * 256 + tid] = s;
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

// Bytes one wave reads in a crisp_peak_lds_read call: iters x 8 reads x 64 lanes x (16
// bytes for kind 0, 8 for kinds 1 and 2).
double crisp_peak_lds_bytes_per_wave(int kind, int iters) {
  return (double)iters * 8.0 * 64.0 * (kind == 0 ? 16.0 : 8.0);
}

// cycles: uint64[workgroups * 4], sink: uint32[workgroups * 256], both on the device.
int crisp_peak_lds_read(int kind, int workgroups, int iters, unsigned long long* cycles, unsigned* sink,
                        void* stream) {
  if (workgroups <= 0 || iters <= 0 || !cycles || !sink || kind < 0 || kind > 2) return (int)hipErrorInvalidValue;
  if (kind == 0)
    hipLaunchKernelGGL(peak_lds_read<0>, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, iters, cycles, sink);
  else if (kind == 1)
    hipLaunchKernelGGL(peak_lds_read<1>, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, iters, cycles, sink);
  else
    hipLaunchKernelGGL(peak_lds_read<2>, dim3(workgroups), dim3(256), 0, (hipStream_t)stream, iters, cycles, sink);
  return (int)hipGetLastError();
}

// Instructions one wave issues in a crisp_peak_valu call: iters x 8.
// cycles: uint64[workgroups * 4], sink: float[workgroups * 256], both on the device.
int crisp_peak_valu(int kind, int workgroups, int iters, unsigned long long* cycles, float* sink, void* stream) {
  if (workgroups <= 0 || iters <= 0 || !cycles || !sink || kind < 0 || kind > 2) return (int)hipErrorInvalidValue;
  if (kind == 0)
    hipLaunchKernelGGL(peak_valu<0>, dim3(workgroups), dim3(256), kLdsAlloc, (hipStream_t)stream, iters, cycles, sink);
  else if (kind == 1)
    hipLaunchKernelGGL(peak_valu<1>, dim3(workgroups), dim3(256), kLdsAlloc, (hipStream_t)stream, iters, cycles, sink);
  else
    hipLaunchKernelGGL(peak_valu<2>, dim3(workgroups), dim3(256), kLdsAlloc, (hipStream_t)stream, iters, cycles, sink);
  return (int)hipGetLastError();
}

}  // extern "C"
