// Input checks of the debug build (libcrisp_debug.so, compiled with CRISP_DEBUG):
// non-finite bf16 values in Q, K, V, and caller-given block lists that break the
// list invariants (row_ptr within [0, cap] and non-decreasing; every entry of row qb
// in [0, qb], strictly increasing).  The release library never calls these.
//
// Each check clears a result word, runs one kernel that stores a nonzero code there
// when it finds a violation, copies the word to the host and waits for the stream:
// the debug build trades the library's asynchrony for a status it can return.
#include <atomic>

#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

// bf16 with all exponent bits set: infinity or NaN.
__global__ __launch_bounds__(256) void chk_nonfinite(const uint16_t* p, size_t n, int* found) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  int bad = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    bad |= (p[i] & 0x7f80u) == 0x7f80u;
  if (__ballot(bad) != 0ull && (threadIdx.x & 63) == 0) *found = 1;  // every writer stores 1
}

// One thread per (head, row): 1 = row_ptr out of range or decreasing, 2 = an entry
// outside [0, qb], 3 = entries not strictly increasing.
__global__ __launch_bounds__(256) void chk_lists(const int32_t* row_ptr, const int32_t* col_idx, int64_t cap,
                                                 int hq, int nb, int* found) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)hq * nb) return;
  const int h = (int)(t / nb), qb = (int)(t % nb);
  const int32_t* rp = row_ptr + (size_t)h * (nb + 1);
  const int64_t b = rp[qb], e = rp[qb + 1];
  if (b < 0 || e < b || e > cap) {
    *found = 1;
    return;
  }
  const int32_t* ci = col_idx + (size_t)h * cap;
  int prev = -1;
  for (int64_t i = b; i < e; ++i) {
    const int kb = ci[i];
    if (kb < 0 || kb > qb) {
      *found = 2;
      return;
    }
    if (kb <= prev) {
      *found = 3;
      return;
    }
    prev = kb;
  }
}

__device__ int g_found;

// The result word's address on the current device (each device holds its own copy),
// cached per device; threads that race on the first call store the same address.
hipError_t result_word(int** p) {
  constexpr int kMaxDevices = 64;
  static std::atomic<int*> addr[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  int* a = addr[dev].load(std::memory_order_relaxed);
  if (a == nullptr) {
    if ((e = hipGetSymbolAddress(reinterpret_cast<void**>(&a), HIP_SYMBOL(g_found))) != hipSuccess) return e;
    addr[dev].store(a, std::memory_order_relaxed);
  }
  *p = a;
  return hipSuccess;
}

hipError_t finish(int* word, hipStream_t stream, int* result) {
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = hipMemcpyAsync(result, word, sizeof(int), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  return e;
}

}  // namespace

hipError_t debug_nonfinite(const uint16_t* p, size_t n, hipStream_t stream, int* found) {
  *found = 0;
  if (n == 0) return hipSuccess;
  int* word;
  hipError_t e = result_word(&word);
  if (e != hipSuccess) return e;
  if ((e = hipMemsetAsync(word, 0, sizeof(int), stream)) != hipSuccess) return e;
  const size_t blocks = (n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096;
  hipLaunchKernelGGL(chk_nonfinite, dim3((unsigned)blocks), dim3(256), 0, stream, p, n, word);
  return finish(word, stream, found);
}

hipError_t debug_lists(const Dims& d, const int32_t* row_ptr, const int32_t* col_idx, int64_t cap,
                       hipStream_t stream, int* code) {
  *code = 0;
  const int64_t rows = (int64_t)d.hq * d.nb;
  if (rows == 0) return hipSuccess;
  int* word;
  hipError_t e = result_word(&word);
  if (e != hipSuccess) return e;
  if ((e = hipMemsetAsync(word, 0, sizeof(int), stream)) != hipSuccess) return e;
  hipLaunchKernelGGL(chk_lists, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, stream, row_ptr, col_idx, cap,
                     d.hq, d.nb, word);
  return finish(word, stream, code);
}

}  // namespace crisp
