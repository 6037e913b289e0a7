// Device-side building blocks shared by the libcrisp kernels (gfx950 / CDNA4).
//
// MFMA operand layouts used throughout (v_mfma_f32_32x32x16_bf16, wave64,
// lane l):
//   A (32 x 16, M x K): lane l holds row l % 32, k = 8 * (l / 32) + [0, 8)
//   B (16 x 32, K x N): lane l holds col l % 32, k = 8 * (l / 32) + [0, 8)
//   C (32 x 32):        lane l holds col l % 32; register i holds
//                       row 8 * (i / 4) + 4 * (l / 32) + (i % 4)
// Attention scores are computed transposed (S^T = K Q^T: keys on M, queries on
// N), so each lane owns one query column and the softmax row reductions stay
// inside a lane plus one exchange with lane l ^ 32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "crisp_internal.h"

namespace crisp {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kNumXcd = 8;  // MI355X: 8 XCDs; workgroup i runs on XCD i % 8

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// Value held by lane l ^ 32.
__device__ __forceinline__ float swap_halves(float x) { return __shfl_xor(x, 32); }

// v_permlane32_swap exchanges the upper half-wave of one operand with the lower
// half-wave of the other; with both operands = x every lane receives the pair
// {x[l], x[l ^ 32]} (in some order), so a commutative combine of the pair gives
// the same value in both lanes of a query.
__device__ __forceinline__ float half_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// NaN-propagating maximum (v_maximum_f32 / v_maximum3_f32): unlike fmaxf it
// needs no canonicalisation of its operands.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float half_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return vmax(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Round-to-nearest-even pair conversion (v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16x2 pack_bf16(float a, float b) {
  bf16x2 r = {(__bf16)a, (__bf16)b};
  return r;
}

// acc + p[0] + p[1] with the bf16 values (v_dot2c_f32_bf16 against ones).
__device__ __forceinline__ float dot2_bf16_sum(bf16x2 p, float acc) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(p, ones, acc, false);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// LDS tile swizzle: a row of 128 bf16 is 16 chunks of 16 bytes; chunk c of row r
// is stored at chunk c ^ swz(r).  swz spreads 16 consecutive rows over 16
// distinct chunks (conflict-free 16-byte column reads) and 4 consecutive rows
// over 4 distinct groups of 4 chunks (the 4-row reads of the transposing load).
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

// Byte offset of element (r, d) in a swizzled [rows][128] bf16 LDS tile.
__device__ __forceinline__ int lds_off(int r, int d) {
  return r * 256 + ((((d >> 3) ^ swz(r)) & 15) << 4) + ((d & 7) << 1);
}

__device__ __forceinline__ bf16x8 lds_read16(const char* base, int off) {
  return *reinterpret_cast<const bf16x8*>(base + off);
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives element i%4
// of the 8-byte chunks addressed by lanes i/4, 4 + i/4, 8 + i/4, 12 + i/4.
__device__ __forceinline__ bf16x4 lds_read_tr(const char* base, int off) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + off));
  return __builtin_bit_cast(bf16x4, v);
}

__device__ __forceinline__ bf16x8 cat(bf16x4 a, bf16x4 b) {
  bf16x8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

__device__ __forceinline__ int div_up(int a, int b) { return (a + b - 1) / b; }

// Wave-wide sums.
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ int wave_sum_i(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// The proxy's mass in key block J summed over the b proxy rows (the vertical and slash
// scores of Alg. 3 before the 1/b): P holds one head's per-(block, row) pairs (lo, hi,
// max m they were summed under, -), and lane l takes rows l and l + 64 (ok0 / ok1: the
// row exists) with their normalisers mcl = M c + log2 L.  *slo and *shi get the sums of
// lo and hi, each a fixed-order butterfly over the wave, scaled by 2^(m c - mcl).
__device__ __forceinline__ void proxy_block_sums(const float4* P, int J, float c, float mcl0, float mcl1, bool ok0,
                                                 bool ok1, float* slo, float* shi) {
  const int l = __lane_id();
  float lo0 = 0.f, hi0 = 0.f, lo1 = 0.f, hi1 = 0.f;
  if (ok0) {
    const float4 e = P[(size_t)J * 128 + l];
    const float f = e.z == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(e.z * c - mcl0);
    lo0 = e.x * f;
    hi0 = e.y * f;
  }
  if (ok1) {
    const float4 e = P[(size_t)J * 128 + l + 64];
    const float f = e.z == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(e.z * c - mcl1);
    lo1 = e.x * f;
    hi1 = e.y * f;
  }
  *slo = wave_sum(lo0 + lo1);
  *shi = wave_sum(hi0 + hi1);
}

#if defined(__HIP_DEVICE_COMPILE__)

// Tile fetch: a 64-key x 128-dim tile goes straight from global memory into an
// LDS stage (buffer_load ... lds, 16 bytes per lane, lane t writing LDS base +
// 16 t).  Instruction (i, w') fills rows 16 i + 4 w' .. +3; lane t supplies row
// 16 i + 4 w' + t / 16, physical chunk t % 16, so it loads logical chunk
// (t % 16) ^ swz(row) -- the swizzle only depends on row % 16, so the per-lane
// source offset is the same for every i (i moves the scalar offset).  Keys at or
// past n lie outside the buffer range and read as 0.
template <int NW>
struct Fetch {
  static constexpr int kPerWave = 4 / NW;  // w' values per wave
  int voff[kPerWave];
};

template <int NW>
__device__ __forceinline__ void make_fetch(Fetch<NW>& f, int w, int t) {
#pragma unroll
  for (int x = 0; x < Fetch<NW>::kPerWave; ++x) {
    const int wp = w + NW * x;
    const int row = 4 * wp + (t >> 4);
    f.voff[x] = row * 256 + (((t & 15) ^ swz(row)) << 4);
  }
}

typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;

// Buffer descriptor (V#) over one KV head's [n, 128] bf16 tensor; num_records
// bounds the byte range, so reads at or past key n return 0.
__device__ __forceinline__ i32x4 tensor_rsrc(const uint16_t* base, int n) {
  const unsigned long long p = (unsigned long long)base;
  return i32x4{(int)(unsigned)p, (int)(unsigned)(p >> 32), n * 256, 0x00020000};
}

// One LDS-DMA load: 16 bytes per lane from rsrc + voff + soff into LDS address
// lds_addr + 16 * lane.  Issued as inline assembly so that the compiler's
// wait-count pass does not treat every later LDS read as dependent on it; the
// kernel waits explicitly (wait_dma) and publishes the tile with a workgroup
// barrier before any wave reads it.
__device__ __forceinline__ void dma16(i32x4 rsrc, int voff, int soff, int lds_addr) {
  const int m0 = __builtin_amdgcn_readfirstlane(lds_addr);
  const int so = __builtin_amdgcn_readfirstlane(soff);
  // The scalar offset may come from v_readfirstlane (a VALU write to an SGPR),
  // which a VMEM instruction may only read after 5 wait states, and M0 is written
  // just before; the compiler cannot see these reads inside the assembly, so the
  // wait states are part of it.
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds" ::"v"(voff), "s"(rsrc), "s"(so), "{m0}"(m0));
}

// One tensor's tile of BK keys into the LDS stage at address stage.
template <int NW, int BK>
__device__ __forceinline__ void fetch_tile(const Fetch<NW>& f, i32x4 rsrc, int stage, int key0, int w) {
#pragma unroll
  for (int x = 0; x < Fetch<NW>::kPerWave; ++x) {
    const int wp = w + NW * x;
#pragma unroll
    for (int i = 0; i < BK / 16; ++i) dma16(rsrc, f.voff[x], (key0 + 16 * i) * 256, stage + (16 * i + 4 * wp) * 256);
  }
}

// Waits until every LDS-DMA load of this wave has landed (s_waitcnt vmcnt(0)).
__device__ __forceinline__ void wait_dma() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

#endif  // __HIP_DEVICE_COMPILE__

}  // namespace crisp
