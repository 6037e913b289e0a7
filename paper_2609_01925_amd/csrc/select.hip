// Stage 3: route each head (Alg. 2), select its key blocks (Alg. 3 with the
// sink-aware noise floor of Sec. 4.3 for VS heads, Alg. 4 for PE heads) and
// emit the per-head CSR block lists consumed by the attention kernel.
//
// Every kernel reads the route from device memory, so the host never waits on
// the GPU; kernels for the other route exit on entry.
//
// VS, per (head, direction), one workgroup:
//   floor  r = max((1 - p[0]) - p[N_b-1], 0), mu = r / (N_b - 2), thr = alpha * mu
//          (App. H variant: mu = median of p[1 .. N_b-2], by radix select)
//   count  c = #{p > thr};  k = min(max(c, k_min), N_b)
//   if k > c: radix-select the k-th largest value t on the float bit pattern
//   (p >= 0, so bit order is value order) and keep ties at t in block order.
// PE, per head:
//   pool     mean of Q (PE heads) and K (their KV groups) per block, fp32
//   logits   pooled Q . K^T * scale * log2(e), block-causal, 64 x 64 tiles
//   softmax  per row, divided by N_b (the sum of N_b row-normalised rows)
//   cutoff   the gamma prefix of the descending order is found without a sort:
//            a radix select over the float bit patterns weighted by mass
//            (11 + 11 + 10 bits), masses in 2^-60 fixed point so the
//            cumulative sums are exact and order-independent.  It yields the
//            value t* of the last pair taken and how many pairs equal to t*
//            (in flat order qb * N_b + kb) complete the gamma mass.
// CSR: count per row -> per-head scan -> fill, one wave per row, ballots for
// compaction; rows always hold the sink block 0 and the diagonal block qb.
// Short layers (N_b <= 64): after the pooling, one workgroup per head takes all of the
// above with every intermediate in LDS and the VS directions one wave each (sel_small).
#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

struct RState {
  uint32_t prefix;   // bits of t* found so far
  uint32_t all;      // 1: the total mass never reaches gamma, keep every pair
  unsigned long long need;  // mass (2^-60 units) still to cover below the current prefix
  unsigned long long ceq;   // pairs equal to t* to take, in flat order
  unsigned long long pad;
};

struct SelArgs {
  const uint16_t* q;
  const uint16_t* k;
  const float* c_struct;  // route score: C_struct, or D_JS in the pattern-search mode
  const float* p_v;
  const float* p_s;
  int8_t* route;
  int32_t* row_ptr;
  int32_t* col_idx;
  int64_t col_cap;
  uint8_t* dir_mask;
  int n, nb, B, hq, hkv, G;
  float c2;  // softmax scale * log2(e)
  float alpha, tau, gamma;
  int k_min;
  int vs_mode;   // 0: noise floor (Alg. 3), 1: gamma coverage per direction (App. A)
  int floor_mode;  // 0: mean of the non-anchor mass (Sec. 4.3), 1: their median (App. H)
  int kbar_all;  // 1: K_bar of every KV group is already in kbar (the JSD pattern search pooled it)
  int64_t cap;  // nb * (nb + 1) / 2
  uint8_t* masks;
  float* qbar;
  float* kbar;
  float* atil;
  unsigned long long* rhist;
  RState* rstate;
  int4* rowinfo;
  const float4* parts;     // short layers from prefill: the estimator's per-(block, row) sums, else null
  const float* rowfinal;   // their per-row normalisers
  int b;                   // proxy rows
};

constexpr int kRadixBins = 2048;
constexpr int64_t kSmallCap = 32768;  // causal pairs per head up to which one workgroup finds the PE cutoff
constexpr double kFix = 1152921504606846976.0;  // 2^60

__device__ __forceinline__ uint32_t fbits(float x) {
  uint32_t b = __float_as_uint(x);
  return (b & 0x80000000u) ? 0u : b;  // negatives (and -0) rank as 0
}

__device__ __forceinline__ unsigned long long fixed_mass(uint32_t bits) {
  return (unsigned long long)((double)__uint_as_float(bits) * kFix);
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Exclusive prefix count of `flag` over a 1024-thread block; *total gets the block total.
__device__ int block_scan_1024(int flag, int* wtot, int* total) {
  const int tid = threadIdx.x, w = tid >> 6;
  const uint64_t bal = __ballot(flag);
  const int within = __popcll(bal & lanemask_lt());
  if ((tid & 63) == 0) wtot[w] = __popcll(bal);
  __syncthreads();
  int before = 0, all = 0;
  for (int i = 0; i < 16; ++i) {
    const int t = wtot[i];
    if (i < w) before += t;
    all += t;
  }
  __syncthreads();
  *total = all;
  return before + within;
}

__device__ int block_sum_1024(int x, int* wtot) {
  x = wave_sum_i(x);
  const int tid = threadIdx.x;
  if ((tid & 63) == 0) wtot[tid >> 6] = x;
  __syncthreads();
  int s = 0;
  for (int i = 0; i < 16; ++i) s += wtot[i];
  __syncthreads();
  return s;
}

// Inclusive prefix sum over the 64 lanes in lane order, on DPP lane moves: within each
// row of 16 lanes by shifts of 1, 2, 4 and 8 (lanes shifted in from outside the row read
// 0), then the last lane of rows 0 and 2 broadcast into rows 1 and 3, and lane 31 into
// rows 2 and 3.  Integer sums, so the result is that of any other order.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROW_MASK, 0xf, true);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ unsigned long long dpp_move(unsigned long long x) {
  return ((unsigned long long)dpp_u32<CTRL, ROW_MASK>((uint32_t)(x >> 32)) << 32) | dpp_u32<CTRL, ROW_MASK>((uint32_t)x);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_move(uint32_t x) {
  return dpp_u32<CTRL, ROW_MASK>(x);
}
template <typename T>
__device__ __forceinline__ T wave_inclusive_scan(T x) {
  x += dpp_move<0x111, 0xf>(x);  // row_shr:1
  x += dpp_move<0x112, 0xf>(x);  // row_shr:2
  x += dpp_move<0x114, 0xf>(x);  // row_shr:4
  x += dpp_move<0x118, 0xf>(x);  // row_shr:8
  x += dpp_move<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
  x += dpp_move<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
  return x;
}

// Lane j's value of x (j uniform).
__device__ __forceinline__ uint32_t lane_value(uint32_t x, int j) {
  return (uint32_t)__builtin_amdgcn_readlane((int)x, j);
}
__device__ __forceinline__ unsigned long long lane_value(unsigned long long x, int j) {
  return ((unsigned long long)lane_value((uint32_t)(x >> 32), j) << 32) | lane_value((uint32_t)x, j);
}

// Digit search of a radix select, by one whole wave: bins[0 .. nbins) (nbins a
// power of two from 64 to 4096) hold non-negative weights (counts or fixed-point
// masses) of the candidates whose higher digits match, visited from bin nbins - 1
// down.  Returns the first bin at which the cumulative weight reaches need (>= 1), with
// *before the weight of the bins above it, or -1 when the total stays below need.
// Lane l sums its own run of nbins / 64 bins (starting at a lane-dependent offset in
// the run, so that the lanes' reads fall in different LDS banks: the sums are of
// integers, so the order does not matter); a prefix scan over the lanes finds the run
// that crosses need, and the wave then scans that run, one bin per lane.
template <typename T>
__device__ int wave_descend_find(const T* bins, int nbins, T need, T* before) {
  const int l = lane_id();
  const int per = nbins / 64;
  const int top = nbins - 1 - per * l;
  T own = 0;
  for (int i0 = 0; i0 < per; i0 += 8) {  // eight reads in flight, then their sum
    T v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = i0 + j < per ? bins[top - ((i0 + j + l) & (per - 1))] : (T)0;
#pragma unroll
    for (int j = 0; j < 8; ++j) own += v[j];
  }
  const T incl = wave_inclusive_scan(own);
  const uint64_t hit = __ballot(incl >= need);
  if (hit == 0) return -1;
  const int lw = __builtin_ctzll(hit);
  const T base = lane_value(incl, lw) - lane_value(own, lw);  // weight of the runs above run lw
  const int top_w = nbins - 1 - per * lw;
  int d = 0;
  T cum = 0;
  for (int j0 = 0; j0 < per; j0 += 64) {  // the run, 64 bins at a time from its top
    const int j = j0 + l;
    const T v = j < per ? bins[top_w - j] : (T)0;
    const T c = wave_inclusive_scan(v);
    const uint64_t cross = __ballot(j < per && base + cum + c >= need);
    if (cross) {
      const int lj = __builtin_ctzll(cross);
      d = top_w - (j0 + lj);
      cum = base + cum + lane_value(c, lj) - lane_value(v, lj);
      break;
    }
    cum += lane_value(c, 63);
  }
  *before = cum;
  return d;
}

// k-th largest bit pattern (k >= 1) among fbits(p[0..nb)).
__device__ uint32_t kth_largest(const float* p, int nb, int k, uint32_t* hist, int* sh) {
  const int tid = threadIdx.x;
  uint32_t prefix = 0, pmask = 0;
  int rem = k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += 1024) hist[i] = 0;
    __syncthreads();
    for (int J = tid; J < nb; J += 1024) {
      const uint32_t b = fbits(p[J]);
      if ((b & pmask) == prefix) atomicAdd(&hist[(b >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (tid < 64) {
      uint32_t cum = 0;
      const int d = wave_descend_find<uint32_t>(hist, 256, (uint32_t)rem, &cum);
      if (tid == 0) {  // the k-th largest exists, so d >= 0
        sh[0] = d < 0 ? 0 : d;
        sh[1] = rem - (int)cum;
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sh[0] << shift;
    pmask |= 255u << shift;
    rem = sh[1];
    __syncthreads();
  }
  return prefix;
}

// Marks the kd largest p (ties: lower block first) in m (and dm).  1024 threads.
__device__ void select_top_k(const float* p, int nb, int kd, uint8_t* m, uint8_t* dm, uint32_t* hist, int* sh,
                             int* wtot) {
  const int tid = threadIdx.x;
  const uint32_t t = kth_largest(p, nb, kd, hist, sh);
  int ngt = 0;
  for (int J = tid; J < nb; J += 1024) ngt += fbits(p[J]) > t;
  ngt = block_sum_1024(ngt, wtot);
  const int need = kd - ngt;
  int running = 0;
  for (int base = 0; base < nb; base += 1024) {
    const int J = base + tid;
    const uint32_t b = J < nb ? fbits(p[J]) : 0u;
    const int eq = J < nb && b == t;
    int tot;
    const int rank = running + block_scan_1024(eq, wtot, &tot);
    if (J < nb) {
      const uint8_t s = (b > t) || (eq && rank < need);
      m[J] = s;
      if (dm) dm[J] = s;
    }
    running += tot;
  }
}

// Gamma prefix of one direction (App. A, VS index selection): the blocks taken in
// order of decreasing p (ties: lower block first) until their mass reaches gamma.
// A mass-weighted radix select over the float bit patterns (11 + 11 + 10 bits),
// masses in 2^-60 fixed point so the sums are exact and order-independent: t is
// the value of the last block taken and `ceq` how many blocks equal to t (in
// block order) complete the mass.  Returns the number of blocks taken, or nb
// (with *all = 1) when the total mass never reaches gamma.  1024 threads.
__device__ int gamma_prefix(const float* p, int nb, float gamma, uint32_t* t_out, int* ceq_out, int* all_out,
                            unsigned long long* hist, unsigned long long* sh64, int* wtot) {
  const int tid = threadIdx.x;
  unsigned long long need = (unsigned long long)ceil((double)gamma * kFix);
  uint32_t prefix = 0, pmask = 0;
  int all = 0;
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
#pragma unroll
  for (int pass = 0; pass < 3; ++pass) {
    if (all) break;
    const int shift = shifts[pass], bins = 1 << widths[pass];
    for (int i = tid; i < bins; i += 1024) hist[i] = 0ull;
    __syncthreads();
    for (int J = tid; J < nb; J += 1024) {
      const uint32_t b = fbits(p[J]);
      if ((b & pmask) == prefix) atomicAdd(&hist[(b >> shift) & (uint32_t)(bins - 1)], fixed_mass(b));
    }
    __syncthreads();
    if (tid < 64) {
      unsigned long long cum = 0;
      const int d = wave_descend_find<unsigned long long>(hist, bins, need, &cum);
      if (tid == 0) {
        sh64[0] = d < 0 ? ~0ull : (unsigned long long)d;
        sh64[1] = d < 0 ? 0ull : need - cum;
      }
    }
    __syncthreads();
    if (sh64[0] == ~0ull) {
      all = 1;
    } else {
      prefix |= (uint32_t)sh64[0] << shift;
      pmask |= (uint32_t)(bins - 1) << shift;
      need = sh64[1];
    }
    __syncthreads();
  }
  *all_out = all;
  if (all) return nb;
  const unsigned long long mt = fixed_mass(prefix);
  // mt > 0: the digit search only stops on a bin holding mass
  const int ceq = (int)((need + mt - 1) / mt);
  int gt = 0;
  for (int J = tid; J < nb; J += 1024) gt += fbits(p[J]) > prefix;
  gt = block_sum_1024(gt, wtot);
  *t_out = prefix;
  *ceq_out = ceq;
  return gt + ceq;
}

// Shared memory of one direction's VS selection.
struct VsShared {
  uint32_t hist[256];
  unsigned long long hist64[2048];
  unsigned long long sh64[2];
  int wtot[16];
  int sh[2];
};

// Route (Alg. 2, or App. A's pattern search when the score is D_JS) and VS selection of
// direction dir (Alg. 3, or App. A's gamma coverage) of head h.  1024 threads.
__device__ void route_vs_dir(const SelArgs& a, int h, int dir, VsShared& vsh) {
  uint32_t* hist = vsh.hist;
  unsigned long long* hist64 = vsh.hist64;
  unsigned long long* sh64 = vsh.sh64;
  int* wtot = vsh.wtot;
  int* sh = vsh.sh;
  const int tid = threadIdx.x;
  const bool vs = a.c_struct[h] >= a.tau;
  if (dir == 0 && tid == 0) a.route[h] = vs ? 0 : 1;
  const int nb = a.nb;
  const float* p = (dir == 0 ? a.p_v : a.p_s) + (size_t)h * nb;
  uint8_t* m = a.masks + ((size_t)h * 2 + dir) * nb;
  uint8_t* dm = a.dir_mask ? a.dir_mask + ((size_t)h * 2 + dir) * nb : nullptr;
  if (!vs || nb <= 2) {
    for (int J = tid; J < nb; J += 1024) {
      m[J] = 0;
      if (dm) dm[J] = 0;
    }
    return;
  }
  if (a.vs_mode == 1) {
    uint32_t t = 0;
    int ceq = 0, all = 0;
    const int c = gamma_prefix(p, nb, a.gamma, &t, &ceq, &all, hist64, sh64, wtot);
    int kd = c > a.k_min ? c : a.k_min;
    kd = kd < nb ? kd : nb;
    if (kd == c) {
      int running = 0;
      for (int base = 0; base < nb; base += 1024) {
        const int J = base + tid;
        const uint32_t b = J < nb ? fbits(p[J]) : 0u;
        const int eq = J < nb && b == t;
        int tot;
        const int rank = running + block_scan_1024(eq, wtot, &tot);
        if (J < nb) {
          const uint8_t s = all || (b > t) || (eq && rank < ceq);
          m[J] = s;
          if (dm) dm[J] = s;
        }
        running += tot;
      }
      return;
    }
    select_top_k(p, nb, kd, m, dm, hist, sh, wtot);
    return;
  }
  float mu;
  if (a.floor_mode == 1) {
    // median of p[1 .. nb-2] (for an even count, the mean of the two middle values)
    const int m = nb - 2;
    const float hi = __uint_as_float(kth_largest(p + 1, m, m / 2 + (m & 1), hist, sh));
    if (m & 1) {
      mu = hi;
    } else {
      const float lo = __uint_as_float(kth_largest(p + 1, m, m / 2 + 1, hist, sh));
      mu = (lo + hi) * 0.5f;
    }
  } else {
    const float r = fmaxf((1.0f - p[0]) - p[nb - 1], 0.0f);
    mu = r / (float)(nb - 2);
  }
  const float thr = a.alpha * mu;
  int c = 0;
  for (int J = tid; J < nb; J += 1024) c += p[J] > thr;
  c = block_sum_1024(c, wtot);
  int kd = c > a.k_min ? c : a.k_min;
  kd = kd < nb ? kd : nb;
  if (kd == c) {
    for (int J = tid; J < nb; J += 1024) {
      const uint8_t s = p[J] > thr;
      m[J] = s;
      if (dm) dm[J] = s;
    }
    return;
  }
  select_top_k(p, nb, kd, m, dm, hist, sh, wtot);
}

// grid (hq, 2), 1024 threads.
__global__ __launch_bounds__(1024) void sel_route_vs(SelArgs a) {
  __shared__ VsShared vsh;
  route_vs_dir(a, blockIdx.x, blockIdx.y, vsh);
}

// Mean of rows [r0, r1) of a [rows][128] bf16 tensor into dst[0..128) (fp32).  256 threads.
__device__ void pool_rows(const uint16_t* src, int r0, int r1, float* dst, float (*red)[128]) {
  const int tid = threadIdx.x;
  const int c = tid & 15, rg = tid >> 4;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int r = r0 + rg; r < r1; r += 16) {
    const u32x4 raw = *reinterpret_cast<const u32x4*>(src + (size_t)r * kHeadDim + 8 * c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += __uint_as_float(raw[e] << 16);
      acc[2 * e + 1] += __uint_as_float(raw[e] & 0xffff0000u);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rg][8 * c + e] = acc[e];
  __syncthreads();
  if (tid < 128) {
    float s = 0.f;
    for (int i = 0; i < 16; ++i) s += red[i][tid];
    dst[tid] = s / (float)(r1 - r0);
  }
}

// Mean-pool Q of PE heads and K of KV groups with a PE head (Alg. 4).  grid (nb, hq + hkv), 256 threads.
__global__ __launch_bounds__(256) void sel_pool(SelArgs a) {
  __shared__ float red[16][128];
  const int J = blockIdx.x, y = blockIdx.y;
  const uint16_t* src;
  float* dst;
  if (y < a.hq) {
    if (a.c_struct[y] >= a.tau) return;  // VS head (the route of Alg. 2, decided from its score)
    src = a.q + (size_t)y * a.n * kHeadDim;
    dst = a.qbar + ((size_t)y * a.nb + J) * kHeadDim;
  } else {
    if (a.kbar_all) return;
    const int g = y - a.hq;
    bool any = false;
    for (int i = 0; i < a.G; ++i) any |= !(a.c_struct[g * a.G + i] >= a.tau);
    if (!any) return;
    src = a.k + (size_t)g * a.n * kHeadDim;
    dst = a.kbar + ((size_t)g * a.nb + J) * kHeadDim;
  }
  const int r0 = J * a.B;
  pool_rows(src, r0, r0 + a.B < a.n ? r0 + a.B : a.n, dst, red);
}

// ---------------------------------------------------------------------------
// FlexPrefill's pattern search (App. A): D_JS between the proxy's per-block mass
// p_v (App. A's per-query mean, sum-pooled over key blocks) and the pooled
// estimate softmax(pool(Q_hat) pool(K)^T * scale) over the N_b key blocks.
struct JsdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const float* p_v;
  float* jsd;
  float* kbar;  // [hkv][nb][128] fp32
  float* zbuf;  // [hq][nb] fp32 pooled logits
  int n, nb, B, b, hq, hkv, G;
  float scale;
};

// K_bar of every KV group.  grid (nb, hkv), 256 threads.
__global__ __launch_bounds__(256) void jsd_pool_k(JsdArgs a) {
  __shared__ float red[16][128];
  const int J = blockIdx.x, g = blockIdx.y;
  const int r0 = J * a.B;
  pool_rows(a.k + (size_t)g * a.n * kHeadDim, r0, r0 + a.B < a.n ? r0 + a.B : a.n,
            a.kbar + ((size_t)g * a.nb + J) * kHeadDim, red);
}

__device__ double block_sum_256d(double x, double* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  const int tid = threadIdx.x;
  if ((tid & 63) == 0) red[tid >> 6] = x;
  __syncthreads();
  const double s = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return s;
}

// One query head per workgroup, 256 threads: pooled last query block, logits
// against K_bar (one wave per key block), softmax and the two KL terms in fp64.
__global__ __launch_bounds__(256) void jsd_score(JsdArgs a) {
  __shared__ float red[16][128];
  __shared__ float qm[128];
  __shared__ float fred[4];
  __shared__ double dred[4];
  const int h = blockIdx.x, g = h / a.G, tid = threadIdx.x, l = tid & 63, w = tid >> 6;
  pool_rows(a.q + (size_t)h * a.n * kHeadDim, a.n - a.b, a.n, qm, red);
  __syncthreads();
  const float* kb = a.kbar + (size_t)g * a.nb * kHeadDim;
  float* z = a.zbuf + (size_t)h * a.nb;
  const float q0 = qm[2 * l], q1 = qm[2 * l + 1];
  float mx = -__builtin_inff();
  for (int J = w; J < a.nb; J += 4) {
    const float* kr = kb + (size_t)J * kHeadDim + 2 * l;
    const float d = wave_sum(q0 * kr[0] + q1 * kr[1]) * a.scale;
    if (l == 0) z[J] = d;
    mx = fmaxf(mx, d);
  }
  if (l == 0) fred[w] = mx;
  __syncthreads();  // also publishes the z written by lane 0 of every wave
  mx = fmaxf(fmaxf(fred[0], fred[1]), fmaxf(fred[2], fred[3]));
  double s = 0.0;
  for (int J = tid; J < a.nb; J += 256) s += (double)expf(z[J] - mx);
  s = block_sum_256d(s, dred);
  double t = 0.0;
  const float* pv = a.p_v + (size_t)h * a.nb;
  for (int J = tid; J < a.nb; J += 256) {
    const double ab = (double)expf(z[J] - mx) / s;
    const double ah = (double)pv[J];
    const double m = 0.5 * (ah + ab);
    if (ah > 0.0) t += ah * log(ah / m);
    if (ab > 0.0) t += ab * log(ab / m);
  }
  t = block_sum_256d(t, dred);
  if (tid == 0) a.jsd[h] = (float)sqrt(fmax(0.5 * t, 0.0));
}

constexpr int kLogitDirect = 512;
// Pooled logits for mid-size layers (kPeSmall < N_b <= kLogitDirect), where the tiles
// are few and short and staging them in LDS costs more latency than it saves: 64 x 64
// tiles of the block-causal triangle, grid (ntri, hq), 256 threads, operands streamed
// from L2; wave w computes the 32 x 32 sub-tile
// (query blocks 32 (w >> 1) .., key blocks 32 (w & 1) ..) as 64 steps of
// v_mfma_f32_32x32x2_f32.  The contraction over d is split between the half-waves:
// at step t, lanes 0..31 contribute d = t and lanes 32..63 d = 64 + t, for A (Q_bar
// rows) and B (K_bar rows) alike, so each lane streams 64 consecutive floats of its
// row with 16-byte loads.  Output row m = 8 (i / 4) + 4 (lane / 32) + i % 4 of
// register i, column = lane % 32.
__global__ __launch_bounds__(256) void sel_pe_logits_direct(SelArgs a) {
  const int h = blockIdx.y, tid = threadIdx.x;
  if (a.route[h] != 1) return;
  const int t = blockIdx.x;
  int qt = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while ((qt + 1) * (qt + 2) / 2 <= t) ++qt;
  while (qt * (qt + 1) / 2 > t) --qt;
  const int kt = t - qt * (qt + 1) / 2;
  const int w = tid >> 6, l = tid & 63;
  const int qs0 = qt * 64 + 32 * (w >> 1), ks0 = kt * 64 + 32 * (w & 1);
  if (ks0 > qs0 + 31 || qs0 >= a.nb) return;  // sub-tile wholly above the diagonal or past N_b
  const int qrow = qs0 + (l & 31), krow = ks0 + (l & 31);
  const int d0 = 64 * (l >> 5);
  const float* Qr = a.qbar + ((size_t)h * a.nb + (qrow < a.nb ? qrow : 0)) * kHeadDim + d0;
  const float* Kr = a.kbar + ((size_t)(h / a.G) * a.nb + (krow < a.nb ? krow : 0)) * kHeadDim + d0;
  const bool qok = qrow < a.nb, kok = krow < a.nb;
  f32x16 acc = zero16();
#pragma unroll 2
  for (int c = 0; c < 64; c += 16) {
    float4 qa[4], ka[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      qa[u] = qok ? *reinterpret_cast<const float4*>(Qr + c + 4 * u) : make_float4(0.f, 0.f, 0.f, 0.f);
      ka[u] = kok ? *reinterpret_cast<const float4*>(Kr + c + 4 * u) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[u].x, ka[u].x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[u].y, ka[u].y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[u].z, ka[u].z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(qa[u].w, ka[u].w, acc, 0, 0, 0);
    }
  }
  float* At = a.atil + (size_t)h * a.cap;
  const int kb = ks0 + (l & 31);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int qb = qs0 + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3);
    if (qb < a.nb && kb <= qb) At[(int64_t)qb * (qb + 1) / 2 + kb] = acc[i] * a.c2;
  }
}

// Pooled logits (log2 domain) on fp32 MFMA (v_mfma_f32_32x32x2_f32): tiles of
// 2 WT x 2 WT (query block, key block) pairs of the block-causal triangle, grid
// (ntri, hq), 256 threads.  The contraction over d runs in chunks of 16: each chunk of
// the tile's Q_bar and K_bar rows is staged in LDS (two stages; the next chunk is
// loaded into registers while the current one is multiplied), and wave w computes the
// WT x WT quarter (query blocks WT (w >> 1) .., key blocks WT (w & 1) ..) as
// (WT / 32)^2 accumulators of 32 x 32, so with WT = 64 each operand read from LDS
// serves two MFMAs (WT = 32, for short layers, keeps four waves busy on a small
// triangle).  Within a chunk lanes 0..31 take d = 0..7 and lanes 32..63 d = 8..15 (the
// same for Q_bar and K_bar, so the sum covers every d).  Output row m = 8 (i / 4) +
// 4 (lane / 32) + i % 4 of register i, column = lane % 32.
constexpr int kLogitChunk = 16, kLogitPitch = kLogitChunk + 4;  // floats per LDS row

template <int WT>
__global__ __launch_bounds__(256) void sel_pe_logits(SelArgs a) {
  constexpr int TILE = 2 * WT, NA = WT / 32, U = TILE * 4 / 256;  // float4 per thread per tensor and chunk
  __shared__ __attribute__((aligned(16))) float lq[2][TILE * kLogitPitch];
  __shared__ __attribute__((aligned(16))) float lk[2][TILE * kLogitPitch];
  const int h = blockIdx.y, tid = threadIdx.x;
  if (a.route[h] != 1) return;
  const int t = blockIdx.x;
  int qt = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
  while ((qt + 1) * (qt + 2) / 2 <= t) ++qt;
  while (qt * (qt + 1) / 2 > t) --qt;
  const int kt = t - qt * (qt + 1) / 2;
  const int w = tid >> 6, l = tid & 63;
  const int q0 = qt * TILE, k0 = kt * TILE;
  const int qs0 = q0 + WT * (w >> 1), ks0 = k0 + WT * (w & 1);
  const bool work = ks0 <= qs0 + WT - 1 && qs0 < a.nb;  // some pair of the quarter is causal
  const float* Qb = a.qbar + (size_t)h * a.nb * kHeadDim;
  const float* Kb = a.kbar + (size_t)(h / a.G) * a.nb * kHeadDim;
  // staging: thread tid moves float4 number tid + 256 u of the chunk (row (tid + 256 u) / 4,
  // columns 4 ((tid + 256 u) % 4)) of Q_bar and likewise of K_bar
  float4 rq[U], rk[U];
  auto load = [&](int c) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int f = tid + 256 * u, row = f >> 2, col = c * kLogitChunk + 4 * (f & 3);
      rq[u] = q0 + row < a.nb ? *reinterpret_cast<const float4*>(Qb + (size_t)(q0 + row) * kHeadDim + col)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
      rk[u] = k0 + row < a.nb ? *reinterpret_cast<const float4*>(Kb + (size_t)(k0 + row) * kHeadDim + col)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store = [&](int st) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int f = tid + 256 * u, row = f >> 2, col = 4 * (f & 3);
      *reinterpret_cast<float4*>(&lq[st][row * kLogitPitch + col]) = rq[u];
      *reinterpret_cast<float4*>(&lk[st][row * kLogitPitch + col]) = rk[u];
    }
  };
  f32x16 acc[NA][NA];
#pragma unroll
  for (int i = 0; i < NA; ++i)
#pragma unroll
    for (int j = 0; j < NA; ++j) acc[i][j] = zero16();
  constexpr int kChunks = kHeadDim / kLogitChunk;
  load(0);
  store(0);
  __syncthreads();
  for (int c = 0; c < kChunks; ++c) {
    if (c + 1 < kChunks) load(c + 1);
    if (work) {
      const int st = c & 1, dl = 8 * (l >> 5);
      float av[NA][8], bv[NA][8];
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        const float* qa = &lq[st][(WT * (w >> 1) + 32 * i + (l & 31)) * kLogitPitch + dl];
        const float* kbp = &lk[st][(WT * (w & 1) + 32 * i + (l & 31)) * kLogitPitch + dl];
        const float4 x0 = *reinterpret_cast<const float4*>(qa), x1 = *reinterpret_cast<const float4*>(qa + 4);
        const float4 y0 = *reinterpret_cast<const float4*>(kbp), y1 = *reinterpret_cast<const float4*>(kbp + 4);
        av[i][0] = x0.x; av[i][1] = x0.y; av[i][2] = x0.z; av[i][3] = x0.w;
        av[i][4] = x1.x; av[i][5] = x1.y; av[i][6] = x1.z; av[i][7] = x1.w;
        bv[i][0] = y0.x; bv[i][1] = y0.y; bv[i][2] = y0.z; bv[i][3] = y0.w;
        bv[i][4] = y1.x; bv[i][5] = y1.y; bv[i][6] = y1.z; bv[i][7] = y1.w;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int i = 0; i < NA; ++i)
#pragma unroll
          for (int j = 0; j < NA; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][u], bv[j][u], acc[i][j], 0, 0, 0);
    }
    if (c + 1 < kChunks) {
      store((c + 1) & 1);  // that stage was last read in chunk c - 1, before the barrier below it
      __syncthreads();
    }
  }
  if (!work) return;
  float* At = a.atil + (size_t)h * a.cap;
  {
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      const int kb = ks0 + 32 * j + (l & 31);
#pragma unroll
      for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int qb = qs0 + 32 * i + 8 * (r >> 2) + 4 * (l >> 5) + (r & 3);
          if (qb < a.nb && kb <= qb) At[(int64_t)qb * (qb + 1) / 2 + kb] = acc[i][j][r] * a.c2;
        }
    }
  }
}

// Short layers (N_b <= kPeSmall): the whole pooled triangle of one PE head in one
// workgroup of 16 waves.  Q_bar and K_bar rows go to LDS once (float4 columns swizzled by
// row so the operand reads of 32 rows spread over the banks).  Each of the triangle's
// three non-empty 32 x 32 quarters (query blocks 32 i .., key blocks 32 j .., j <= i) is
// split over d into four runs of 32: wave w < 12 computes quarter w / 4 over run w % 4
// on fp32 MFMA (within the run, the d split of sel_pe_logits), the twelve partial
// products go back to LDS, and the row softmax (divided by N_b) adds the four runs of
// each logit in run order.  The waves take the rows in turn, writing row qb at
// At[qb (qb + 1) / 2 ..] (global memory or LDS).  buf holds 2 kPeSmall kHeadDim floats.
constexpr int kPeSmall = kSmallSelectBlocks, kPartPitch = 33;

__device__ void pe_small_head(const SelArgs& a, int h, float* buf, float* At) {
  const int tid = threadIdx.x, nthr = blockDim.x, nwav = nthr >> 6;
  const int w = tid >> 6, l = tid & 63, nb = a.nb;
  float* sq = buf;
  float* sk = buf + kPeSmall * kHeadDim;
  const float* Qb = a.qbar + (size_t)h * nb * kHeadDim;
  const float* Kb = a.kbar + (size_t)(h / a.G) * nb * kHeadDim;
  auto phys = [](int r, int c4) { return r * kHeadDim + 4 * (c4 ^ (r & 31)); };
  for (int f = tid; f < kPeSmall * kHeadDim / 4; f += nthr) {  // kPeSmall rows x 32 float4
    const int r = f >> 5, c4 = f & 31;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f), y = x;
    if (r < nb) {
      x = *reinterpret_cast<const float4*>(Qb + (size_t)r * kHeadDim + 4 * c4);
      y = *reinterpret_cast<const float4*>(Kb + (size_t)r * kHeadDim + 4 * c4);
    }
    *reinterpret_cast<float4*>(&sq[phys(r, c4)]) = x;
    *reinterpret_cast<float4*>(&sk[phys(r, c4)]) = y;
  }
  __syncthreads();
  const int quarter = w >> 2, run = w & 3;
  const int qs0 = quarter == 0 ? 0 : 32, ks0 = quarter == 2 ? 32 : 0;
  const bool work = w < 12 && qs0 < nb;
  f32x16 acc = zero16();
  if (work) {
    const int qr = qs0 + (l & 31), kr = ks0 + (l & 31);
#pragma unroll
    for (int c = 2 * run; c < 2 * run + 2; ++c) {
      const int c4 = 4 * c + 2 * (l >> 5);  // lanes 0..31: d 16 c .. +7; lanes 32..63: d 16 c + 8 .. +15
      const float4 x0 = *reinterpret_cast<const float4*>(&sq[phys(qr, c4)]);
      const float4 x1 = *reinterpret_cast<const float4*>(&sq[phys(qr, c4 + 1)]);
      const float4 y0 = *reinterpret_cast<const float4*>(&sk[phys(kr, c4)]);
      const float4 y1 = *reinterpret_cast<const float4*>(&sk[phys(kr, c4 + 1)]);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x0.x, y0.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x0.y, y0.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x0.z, y0.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x0.w, y0.w, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x1.x, y1.x, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x1.y, y1.y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x1.z, y1.z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x1.w, y1.w, acc, 0, 0, 0);
    }
  }
  __syncthreads();  // every operand read is done before the partial products overwrite buf
  // partial products: [run][quarter][32 rows][kPartPitch]
  constexpr int kQuarter = 32 * kPartPitch, kRun = 3 * kQuarter;
  if (work) {
    float* P = buf + run * kRun + quarter * kQuarter + (l & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) P[(8 * (r >> 2) + 4 * (l >> 5) + (r & 3)) * kPartPitch] = acc[r];
  }
  __syncthreads();
  const float inv_nb = 1.f / (float)nb;
  for (int qb = w; qb < nb; qb += nwav) {
    const bool in = l <= qb;
    float x = -__builtin_inff();
    if (in) {
      const int qd = qb < 32 ? 0 : (l < 32 ? 1 : 2);
      const float* P = buf + qd * kQuarter + (qb & 31) * kPartPitch + (l & 31);
      x = (((P[0] + P[kRun]) + P[2 * kRun]) + P[3 * kRun]) * a.c2;
    }
    const float mx = wave_max(x);
    const float p = in ? fast_exp2(x - mx) : 0.f;
    const float sum = wave_sum(p);
    if (in) At[(int64_t)qb * (qb + 1) / 2 + l] = p / sum * inv_nb;
  }
}

// Reduction of one value per thread of a 256-thread workgroup in binary-tree order
// (t with t + 128, then t with t + 64, ..., then t with t + 1), the last six levels
// within wave 0 by shuffles; every thread gets the result.
template <typename Op>
__device__ __forceinline__ float tree_reduce(float* red, float v, Op op) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
  if (tid < 128) red[tid] = op(red[tid], red[tid + 128]);
  __syncthreads();
  if (tid < 64) {
    float x = op(red[tid], red[tid + 64]);
#pragma unroll
    for (int s = 32; s > 0; s >>= 1) x = op(x, __shfl_down(x, s, 64));
    if (tid == 0) red[0] = x;
  }
  __syncthreads();
  const float r = red[0];
  __syncthreads();  // red may be reused
  return r;
}

// Row softmax of the pooled logits, divided by N_b.  grid (nb, hq), 256 threads.
__global__ __launch_bounds__(256) void sel_pe_softmax(SelArgs a) {
  __shared__ float red[256];
  const int qb = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  if (a.route[h] != 1) return;
  float* row = a.atil + (size_t)h * a.cap + (int64_t)qb * (qb + 1) / 2;
  const int len = qb + 1;
  float mx = -__builtin_inff();
  for (int i = tid; i < len; i += 256) mx = fmaxf(mx, row[i]);
  mx = tree_reduce(red, mx, [](float x, float y) { return fmaxf(x, y); });
  float sum = 0.f;
  for (int i = tid; i < len; i += 256) sum += fast_exp2(row[i] - mx);
  sum = tree_reduce(red, sum, [](float x, float y) { return x + y; });
  const float inv_nb = 1.f / (float)a.nb;
  for (int i = tid; i < len; i += 256) row[i] = fast_exp2(row[i] - mx) / sum * inv_nb;
}

// Radix state init: need = ceil(gamma * 2^60), histogram cleared.  grid hq, 256 threads.
__global__ __launch_bounds__(256) void sel_radix_init(SelArgs a) {
  const int h = blockIdx.x, tid = threadIdx.x;
  if (a.route[h] != 1) return;
  for (int i = tid; i < kRadixBins; i += 256) a.rhist[(size_t)h * kRadixBins + i] = 0ull;
  if (tid == 0) {
    RState s;
    s.prefix = 0;
    s.all = 0;
    s.need = (unsigned long long)ceil((double)a.gamma * kFix);
    if (s.need == 0) s.need = 1;
    s.ceq = 0;
    s.pad = 0;
    a.rstate[h] = s;
  }
}

__device__ __forceinline__ void radix_digit(int pass, int& shift, int& nbits) {
  shift = pass == 0 ? 21 : (pass == 1 ? 10 : 0);
  nbits = pass == 2 ? 10 : 11;
}

// Mass histogram of one digit over the pairs whose higher digits match the prefix.
// grid (chunks, hq), 256 threads.
__global__ __launch_bounds__(256) void sel_radix_hist(SelArgs a, int pass) {
  __shared__ unsigned long long lh[kRadixBins];
  const int h = blockIdx.y, tid = threadIdx.x;
  if (a.route[h] != 1) return;
  const RState st = a.rstate[h];
  if (st.all) return;
  int shift, nbits;
  radix_digit(pass, shift, nbits);
  const int hi = shift + nbits;
  const uint64_t want = (uint64_t)st.prefix >> hi;
  for (int i = tid; i < kRadixBins; i += 256) lh[i] = 0ull;
  __syncthreads();
  const float* At = a.atil + (size_t)h * a.cap;
  const int64_t per = (a.cap + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t up = lo + per < a.cap ? lo + per : a.cap;
  const uint32_t dmask = (1u << nbits) - 1u;
  auto take = [&](float x) {
    const uint32_t b = fbits(x);
    if (((uint64_t)b >> hi) == want) atomicAdd(&lh[(b >> shift) & dmask], fixed_mass(b));
  };
  // The chunk [lo, up): up to three entries before the first 16-byte aligned one, then
  // 16-byte loads (four in flight per thread), then up to three entries after them.
  int64_t a0 = lo + (int64_t)((4 - (((uintptr_t)(At + lo) >> 2) & 3)) & 3);
  a0 = a0 < up ? a0 : up;
  const int64_t n4 = (up - a0) >> 2, a1 = a0 + 4 * n4;
  if (lo + tid < a0) take(At[lo + tid]);
  if (a1 + tid < up) take(At[a1 + tid]);
  const float4* A4 = reinterpret_cast<const float4*>(At + a0);
  for (int64_t j0 = tid; j0 < n4; j0 += 4 * 256) {
    float4 v[4];
#pragma unroll
    for (int x = 0; x < 4; ++x)
      if (j0 + 256 * x < n4) v[x] = A4[j0 + 256 * x];
#pragma unroll
    for (int x = 0; x < 4; ++x)
      if (j0 + 256 * x < n4) {
        take(v[x].x);
        take(v[x].y);
        take(v[x].z);
        take(v[x].w);
      }
  }
  __syncthreads();
  for (int i = tid; i < kRadixBins; i += 256)
    if (lh[i]) atomicAdd(&a.rhist[(size_t)h * kRadixBins + i], lh[i]);
}

// Picks the digit where the descending cumulative mass reaches `need`.  grid hq, 256 threads.
__global__ __launch_bounds__(256) void sel_radix_scan(SelArgs a, int pass) {
  __shared__ unsigned long long bins[kRadixBins];
  const int h = blockIdx.x, tid = threadIdx.x;
  if (a.route[h] != 1) return;
  RState st = a.rstate[h];
  if (st.all) return;
  int shift, nbits;
  radix_digit(pass, shift, nbits);
  const int nbins = 1 << nbits;
  unsigned long long* H = a.rhist + (size_t)h * kRadixBins;
  for (int i = tid; i < nbins; i += 256) bins[i] = H[i];
  __syncthreads();
  if (tid < 64) {
    unsigned long long cum = 0;
    const int bin = wave_descend_find<unsigned long long>(bins, nbins, st.need, &cum);
    if (tid == 0) {
      if (bin < 0) {
        st.all = 1;  // total mass below gamma: keep every pair
        st.ceq = ~0ull;
      } else {
        st.need -= cum;
        st.prefix |= (uint32_t)bin << shift;
        if (pass == 2) {
          const unsigned long long ft = fixed_mass(st.prefix);
          st.ceq = ft ? (st.need + ft - 1) / ft : ~0ull;
        }
      }
      a.rstate[h] = st;
    }
  }
  for (int i = tid; i < kRadixBins; i += 256) H[i] = 0ull;
}

// PE cutoff of a small layer (at most kSmallCap causal pairs per head) in one
// workgroup per head: the three digit passes of sel_radix_hist / sel_radix_scan
// with the histograms in LDS.  The masses are the same fixed-point integers, so
// t*, the remaining mass and the count of pairs equal to t* are the same; one
// launch replaces seven.  At holds the head's cap scores (global memory or LDS); the
// state ends in sst (LDS) and, when out is given, in *out.
__device__ void radix_small_head(const SelArgs& a, const float* At, unsigned long long* bins, RState& sst,
                                 RState* out) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  if (tid == 0) {
    sst.prefix = 0;
    sst.all = 0;
    sst.need = (unsigned long long)ceil((double)a.gamma * kFix);
    if (sst.need == 0) sst.need = 1;
    sst.ceq = 0;
    sst.pad = 0;
  }
  for (int pass = 0; pass < 3; ++pass) {
    int shift, nbits;
    radix_digit(pass, shift, nbits);
    const int nbins = 1 << nbits;
    for (int i = tid; i < nbins; i += nthr) bins[i] = 0ull;
    __syncthreads();  // bins cleared; sst of the previous pass visible
    if (sst.all) break;
    const int hi = shift + nbits;
    const uint64_t want = (uint64_t)sst.prefix >> hi;
    const uint32_t dmask = (uint32_t)nbins - 1u;
    for (int64_t i = tid; i < a.cap; i += nthr) {
      const uint32_t b = fbits(At[i]);
      if (((uint64_t)b >> hi) == want) atomicAdd(&bins[(b >> shift) & dmask], fixed_mass(b));
    }
    __syncthreads();
    if (tid < 64) {
      unsigned long long cum = 0;
      const int bin = wave_descend_find<unsigned long long>(bins, nbins, sst.need, &cum);
      if (tid == 0) {
        if (bin < 0) {
          sst.all = 1;  // total mass below gamma: keep every pair
          sst.ceq = ~0ull;
        } else {
          sst.need -= cum;
          sst.prefix |= (uint32_t)bin << shift;
          if (pass == 2) {
            const unsigned long long ft = fixed_mass(sst.prefix);
            sst.ceq = ft ? (sst.need + ft - 1) / ft : ~0ull;
          }
        }
      }
    }
    __syncthreads();  // the search is done with the bins before the next pass clears them
  }
  if (tid == 0 && out) *out = sst;
}

// grid hq, 1024 threads.
__global__ __launch_bounds__(1024) void sel_radix_small(SelArgs a) {
  __shared__ unsigned long long bins[kRadixBins];
  __shared__ RState sst;
  const int h = blockIdx.x;
  if (a.route[h] != 1) return;
  radix_small_head(a, a.atil + (size_t)h * a.cap, bins, sst, a.rstate + h);
}

// Per-row counts.  VS: x = row size.  PE: x = #(> t*), y = #(== t*), z = flags
// (1: block 0 > t*, 2: block 0 == t*, 4: block qb > t*, 8: block qb == t*).
// grid (ceil(nb / 4), hq), 256 threads, one wave per row.
__device__ __forceinline__ void csr_count_row(const SelArgs& a, int h, int qb) {
  const int l = threadIdx.x & 63;
  const int nb = a.nb;
  int4 info = make_int4(0, 0, 0, 0);
  if (a.route[h] == 0) {
    const uint8_t* vm = a.masks + (size_t)h * 2 * nb;
    const uint8_t* sm = vm + nb;
    int cnt = 0;
    for (int base = 0; base <= qb; base += 256) {  // four 64-entry chunks, their loads issued together
      bool sel[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int kb = base + 64 * x + l;
        sel[x] = kb <= qb && (kb == 0 || kb == qb || vm[kb] || sm[nb - 1 - qb + kb]);
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) cnt += __popcll(__ballot(sel[x]));
    }
    info.x = cnt;
  } else {
    const RState st = a.rstate[h];
    const float* row = a.atil + (size_t)h * a.cap + (int64_t)qb * (qb + 1) / 2;
    int ngt = 0, neq = 0, flags = 0;
    for (int base = 0; base <= qb; base += 256) {  // four 64-entry chunks, their loads issued together
      uint32_t bv[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int kb = base + 64 * x + l;
        bv[x] = kb <= qb ? fbits(row[kb]) : 0u;
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        if (base + 64 * x > qb) break;
        const int kb = base + 64 * x + l;
        const uint32_t b = bv[x];
        const bool gt = kb <= qb && (st.all || b > st.prefix);
        const bool eq = kb <= qb && !st.all && b == st.prefix;
        ngt += __popcll(__ballot(gt));
        neq += __popcll(__ballot(eq));
        if (base + 64 * x == 0 || qb - (base + 64 * x) < 64) {  // the chunk holds block 0 or block qb
          int f = 0;
          if (kb == 0) f |= (gt ? 1 : 0) | (eq ? 2 : 0);
          if (kb == qb) f |= (gt ? 4 : 0) | (eq ? 8 : 0);
          f = wave_sum_i(f);  // at most two lanes contribute, with disjoint bits
          flags |= f;
        }
      }
    }
    info = make_int4(ngt, neq, flags, 0);
  }
  if (l == 0) a.rowinfo[(size_t)h * nb + qb] = info;
}

__global__ __launch_bounds__(256) void sel_csr_count(SelArgs a) {
  const int qb = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (qb < a.nb) csr_count_row(a, blockIdx.y, qb);
}

// Ties taken per PE row, row sizes and the exclusive scan into row_ptr.  grid hq, 1024 threads.
__device__ __forceinline__ void csr_scan_head(const SelArgs& a, int h, long long* wtot) {
  const int tid = threadIdx.x, w = tid >> 6;
  const int nb = a.nb;
  const bool pe = a.route[h] == 1;
  const RState st = pe ? a.rstate[h] : RState{};
  int4* info = a.rowinfo + (size_t)h * nb;
  int32_t* rp = a.row_ptr + (size_t)h * (nb + 1);
  long long tie_carry = 0, row_carry = 0;
  for (int base = 0; base < nb; base += 1024) {
    const int qb = base + tid;
    int4 in = qb < nb ? info[qb] : make_int4(0, 0, 0, 0);
    // inclusive scans (ties, then row sizes) by waves + wave totals
    long long cnt = 0;
    if (pe) {
      long long x = in.y, incl = x;
      for (int o = 1; o < 64; o <<= 1) {
        const long long y = __shfl_up(incl, o);
        if ((tid & 63) >= o) incl += y;
      }
      if ((tid & 63) == 63) wtot[w] = incl;
      __syncthreads();
      long long before = 0, all = 0;
      for (int i = 0; i < 16; ++i) {
        if (i < w) before += wtot[i];
        all += wtot[i];
      }
      __syncthreads();
      const long long tie_prefix = tie_carry + before + incl - x;
      tie_carry += all;
      long long take = 0;
      if (qb < nb) {
        const unsigned long long ceq = st.ceq;
        if (ceq > (unsigned long long)tie_prefix) {
          const unsigned long long left = ceq - (unsigned long long)tie_prefix;
          take = left < (unsigned long long)in.y ? (long long)left : (long long)in.y;
        }
        const bool z_sel = (in.z & 1) || ((in.z & 2) && take >= 1);
        const bool d_sel = (in.z & 4) || ((in.z & 8) && take == in.y);
        cnt = in.x + take + (z_sel ? 0 : 1) + ((qb > 0 && !d_sel) ? 1 : 0);
        in.w = (int)take;
        info[qb] = in;
      }
    } else if (qb < nb) {
      cnt = in.x;
    }
    long long incl = cnt;
    for (int o = 1; o < 64; o <<= 1) {
      const long long y = __shfl_up(incl, o);
      if ((tid & 63) >= o) incl += y;
    }
    if ((tid & 63) == 63) wtot[w] = incl;
    __syncthreads();
    long long before = 0, all = 0;
    for (int i = 0; i < 16; ++i) {
      if (i < w) before += wtot[i];
      all += wtot[i];
    }
    __syncthreads();
    if (qb < nb) rp[qb] = (int32_t)(row_carry + before + incl - cnt);
    row_carry += all;
  }
  if (tid == 0) rp[nb] = (int32_t)row_carry;
}

__global__ __launch_bounds__(1024) void sel_csr_scan(SelArgs a) {
  __shared__ long long wtot[16];
  csr_scan_head(a, blockIdx.x, wtot);
}

// Write the block lists.  grid (ceil(nb / 4), hq), 256 threads, one wave per row.
__device__ __forceinline__ void csr_fill_row(const SelArgs& a, int h, int qb) {
  const int l = threadIdx.x & 63;
  const int nb = a.nb;
  int32_t* out = a.col_idx + (size_t)h * a.col_cap + a.row_ptr[(size_t)h * (nb + 1) + qb];
  const uint64_t lt = lanemask_lt();
  int pos = 0;
  if (a.route[h] == 0) {
    const uint8_t* vm = a.masks + (size_t)h * 2 * nb;
    const uint8_t* sm = vm + nb;
    for (int base = 0; base <= qb; base += 256) {  // four 64-entry chunks, their loads issued together
      bool sv[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int kb = base + 64 * x + l;
        sv[x] = kb <= qb && (kb == 0 || kb == qb || vm[kb] || sm[nb - 1 - qb + kb]);
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int kb = base + 64 * x + l;
        const uint64_t bal = __ballot(sv[x]);
        if (sv[x]) out[pos + __popcll(bal & lt)] = kb;
        pos += __popcll(bal);
      }
    }
  } else {
    const RState st = a.rstate[h];
    const int take = a.rowinfo[(size_t)h * nb + qb].w;
    const float* row = a.atil + (size_t)h * a.cap + (int64_t)qb * (qb + 1) / 2;
    int eq_seen = 0;
    for (int base = 0; base <= qb; base += 256) {  // four 64-entry chunks, their loads issued together
      uint32_t bv[4];
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        const int kb = base + 64 * x + l;
        bv[x] = kb <= qb ? fbits(row[kb]) : 0u;
      }
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        if (base + 64 * x > qb) break;
        const int kb = base + 64 * x + l;
        const uint32_t b = bv[x];
        const bool gt = kb <= qb && (st.all || b > st.prefix);
        const bool eq = kb <= qb && !st.all && b == st.prefix;
        const uint64_t eb = __ballot(eq);
        const int eq_rank = eq_seen + __popcll(eb & lt);
        eq_seen += __popcll(eb);
        const bool sel = kb <= qb && (gt || (eq && eq_rank < take) || kb == 0 || kb == qb);
        const uint64_t bal = __ballot(sel);
        if (sel) out[pos + __popcll(bal & lt)] = kb;
        pos += __popcll(bal);
      }
    }
  }
}

__global__ __launch_bounds__(256) void sel_csr_fill(SelArgs a) {
  const int qb = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (qb < a.nb) csr_fill_row(a, blockIdx.y, qb);
}

// ---------------------------------------------------------------------------
// Short layers (N_b <= kPeSmall): after the pooling, the route, the selection and the
// lists of one head in one workgroup, with every intermediate in LDS (the direction
// masks as 64-bit words, the pooled scores, the radix bins, the per-row counts and
// offsets), so no phase waits on a round trip through global memory.  With at most 64
// blocks a VS direction fits one wave, one block per lane, and both directions run at
// once on waves 0 and 1.  Their decisions are those of route_vs_dir, reached with
// ballots and lane reads instead of histogram passes: the k-th largest bit pattern is
// found bit by bit from the top as the largest t with #{b >= t} >= k, and the gamma cut
// as the largest block value t whose mass at or above t (the same 2^-60 fixed-point
// integers) reaches gamma -- the values the digit passes settle on, since both counts
// only fall as t grows.  The PE scores, softmax and cutoff are pe_small_head and
// radix_small_head on LDS, and the lists follow the rules of csr_count_row,
// csr_scan_head and csr_fill_row, one wave per row.  grid hq, kSmallThreads threads.
constexpr int kSmallThreads = 1024;

// k-th largest (k >= 1) of the bit patterns b of the lanes with `in` set (k of them at least).
__device__ __forceinline__ uint32_t wave_kth_largest(uint32_t b, bool in, int k) {
  uint32_t t = 0;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    if (__popcll(__ballot(in && b >= c)) >= k) t = c;
  }
  return t;
}

// select_top_k for one block per lane: the kd largest patterns of the lanes below nb,
// ties at the k-th taken in block order.
__device__ __forceinline__ bool wave_top_k(uint32_t b, bool in, int kd) {
  const uint32_t t = wave_kth_largest(b, in, kd);
  const int ngt = __popcll(__ballot(in && b > t));
  const bool eq = in && b == t;
  const int rank = __popcll(__ballot(eq) & lanemask_lt());
  return in && (b > t || (eq && rank < kd - ngt));
}

// The block set of one direction of a VS head with nb > 2 blocks (route_vs_dir), lane =
// block; P: the direction's scores (p_v or p_s) of the head.
__device__ bool small_vs_dir(const SelArgs& a, const float* P) {
  const int l = lane_id(), nb = a.nb;
  const bool in = l < nb;
  const float p = in ? P[l] : 0.f;
  const uint32_t b = in ? fbits(p) : 0u;
  if (a.vs_mode == 1) {
    const unsigned long long need = (unsigned long long)ceil((double)a.gamma * kFix);
    const unsigned long long m = in ? fixed_mass(b) : 0ull;
    // the mass at or above each lane's own value, summed over the blocks in lane order
    unsigned long long ge = 0ull, total = 0ull;
    for (int j = 0; j < nb; ++j) {
      const uint32_t bj = lane_value(b, j);
      const unsigned long long mj = lane_value(m, j);
      total += mj;
      ge += bj >= b ? mj : 0ull;
    }
    int c = nb, ceq = 0;
    uint32_t t = 0;
    const bool all = total < need;  // the total mass never reaches gamma
    if (!all) {
      // mass(>= x) only falls as x grows, and t* carries mass, so t* is the largest
      // block value whose mass at or above it reaches need
      uint32_t cand = in && ge >= need ? b : 0u;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t y = __shfl_xor(cand, o, 64);
        cand = y > cand ? y : cand;
      }
      t = cand;
      const uint64_t eqm = __ballot(in && b == t);
      const int first = __builtin_ctzll(eqm);
      const unsigned long long ge_t = lane_value(ge, first);
      const unsigned long long mt = fixed_mass(t);  // > 0: t carries mass
      const unsigned long long rest = need - (ge_t - (unsigned long long)__popcll(eqm) * mt);
      ceq = (int)((rest + mt - 1) / mt);
      c = __popcll(__ballot(in && b > t)) + ceq;
    }
    int kd = c > a.k_min ? c : a.k_min;
    kd = kd < nb ? kd : nb;
    if (kd != c) return wave_top_k(b, in, kd);
    const bool eq = in && b == t;
    const int rank = __popcll(__ballot(eq) & lanemask_lt());
    return in && (all || b > t || (eq && rank < ceq));
  }
  float mu;
  if (a.floor_mode == 1) {  // median of p[1 .. nb-2]
    const int m = nb - 2;
    const bool mid = l >= 1 && l <= nb - 2;
    const float hi = __uint_as_float(wave_kth_largest(b, mid, m / 2 + (m & 1)));
    if (m & 1) {
      mu = hi;
    } else {
      const float lo = __uint_as_float(wave_kth_largest(b, mid, m / 2 + 1));
      mu = (lo + hi) * 0.5f;
    }
  } else {
    const float r = fmaxf((1.0f - __shfl(p, 0, 64)) - __shfl(p, nb - 1, 64), 0.0f);
    mu = r / (float)(nb - 2);
  }
  const float thr = a.alpha * mu;
  const bool above = in && p > thr;
  const int c = __popcll(__ballot(above));
  int kd = c > a.k_min ? c : a.k_min;
  kd = kd < nb ? kd : nb;
  return kd == c ? above : wave_top_k(b, in, kd);
}

struct SmallShared {
  float ops[2 * kPeSmall * kHeadDim];  // Q_bar and K_bar rows, the partial products, then the radix bins
  float at[kPeSmall * (kPeSmall + 1) / 2];  // the head's pooled scores, row qb at qb (qb + 1) / 2
  uint64_t sel[kPeSmall];  // per row: VS the blocks taken; PE those above t*
  uint64_t eqm[kPeSmall];  // PE, per row: the blocks equal to t*
  int4 info[kPeSmall];     // per row: (#above t* or row size, #equal, flags, ties taken)
  int rp[kPeSmall];
  uint64_t dmask[2];
  RState st;
  float bsum[2][kPeSmall];  // per block: the proxy's lo and hi mass summed over rows
  float pvs[2][kPeSmall];   // p_v and p_s of the head
};

__global__ __launch_bounds__(kSmallThreads) void sel_small(SelArgs a) {
  __shared__ __attribute__((aligned(16))) SmallShared sm;
  const int h = blockIdx.x, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int nb = a.nb;
  const bool vs = a.c_struct[h] >= a.tau;
  if (tid == 0) a.route[h] = vs ? 0 : 1;
  const float* pdir[2] = {a.p_v + (size_t)h * nb, a.p_s + (size_t)h * nb};
  if (vs && a.parts) {
    // p_v and p_s from the estimator's sums, as its scale step forms them: p_v[J] = (lo[J] +
    // hi[J]) / b, p_s[J] = (lo[J] + hi[J - 1]) / b, every sum in the same order
    const bool ok0 = l < a.b, ok1 = l + 64 < a.b;
    const float mcl0 = ok0 ? a.rowfinal[(size_t)h * 128 + l] : 0.f;
    const float mcl1 = ok1 ? a.rowfinal[(size_t)h * 128 + l + 64] : 0.f;
    const float4* P = a.parts + (size_t)h * nb * 128;
    for (int J = w; J < nb; J += kSmallThreads / 64) {
      float slo, shi;
      proxy_block_sums(P, J, a.c2, mcl0, mcl1, ok0, ok1, &slo, &shi);
      if (l == 0) {
        sm.bsum[0][J] = slo;
        sm.bsum[1][J] = shi;
      }
    }
    __syncthreads();
    const float invb = 1.f / (float)a.b;
    if (tid < nb) {
      sm.pvs[0][tid] = (sm.bsum[0][tid] + sm.bsum[1][tid]) * invb;
      sm.pvs[1][tid] = (sm.bsum[0][tid] + (tid > 0 ? sm.bsum[1][tid - 1] : 0.f)) * invb;
    }
    __syncthreads();
    pdir[0] = sm.pvs[0];
    pdir[1] = sm.pvs[1];
  }
  if (w < 2) {  // wave w: direction w (no blocks on a PE head or with N_b <= 2)
    const bool s = vs && nb > 2 && small_vs_dir(a, pdir[w]);
    const uint64_t bits = __ballot(s);
    if (l == 0) sm.dmask[w] = bits;
    if (a.dir_mask && l < nb) a.dir_mask[((size_t)h * 2 + w) * nb + l] = s;
  }
  if (!vs) {
    pe_small_head(a, h, sm.ops, sm.at);
    __syncthreads();  // every score is in sm.at; sm.ops is free
    radix_small_head(a, sm.at, reinterpret_cast<unsigned long long*>(sm.ops), sm.st, nullptr);
  }
  __syncthreads();  // the direction masks, or the PE state
  const uint64_t lt = lanemask_lt();
  // per-row counts (csr_count_row); a wave's rows are w + 16 i, their scores read together
  constexpr int kRowsPerWave = kPeSmall / (kSmallThreads / 64);
  uint32_t rb[kRowsPerWave];
#pragma unroll
  for (int i = 0; i < kRowsPerWave; ++i) {
    const int qb = w + (kSmallThreads / 64) * i;
    rb[i] = !vs && qb < nb && l <= qb ? fbits(sm.at[qb * (qb + 1) / 2 + l]) : 0u;
  }
#pragma unroll
  for (int i = 0; i < kRowsPerWave; ++i) {
    const int qb = w + (kSmallThreads / 64) * i;
    if (qb >= nb) break;
    const bool on = l <= qb;
    int4 info;
    if (vs) {
      const uint64_t vm = sm.dmask[0], smk = sm.dmask[1];
      const bool sel = on && (l == 0 || l == qb || ((vm >> l) & 1) || ((smk >> (nb - 1 - qb + l)) & 1));
      const uint64_t bal = __ballot(sel);
      if (l == 0) sm.sel[qb] = bal;
      info = make_int4(__popcll(bal), 0, 0, 0);
    } else {
      const RState st = sm.st;
      const uint32_t b = rb[i];
      const uint64_t gt = __ballot(on && (st.all || b > st.prefix));
      const uint64_t eq = __ballot(on && !st.all && b == st.prefix);
      if (l == 0) {
        sm.sel[qb] = gt;
        sm.eqm[qb] = eq;
      }
      const int flags = (int)(gt & 1) | (int)((eq & 1) << 1) | (int)(((gt >> qb) & 1) << 2) |
                        (int)(((eq >> qb) & 1) << 3);
      info = make_int4(__popcll(gt), __popcll(eq), flags, 0);
    }
    if (l == 0) sm.info[qb] = info;
  }
  __syncthreads();
  // ties taken per PE row and the row offsets (csr_scan_head), wave 0, lane = row
  if (w == 0) {
    int4 in = l < nb ? sm.info[l] : make_int4(0, 0, 0, 0);
    int cnt = in.x;
    if (!vs) {
      int incl = in.y;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (l >= o) incl += y;
      }
      const unsigned long long tie_prefix = (unsigned long long)(incl - in.y);
      const unsigned long long ceq = sm.st.ceq;
      int take = 0;
      if (ceq > tie_prefix) {
        const unsigned long long left = ceq - tie_prefix;
        take = left < (unsigned long long)in.y ? (int)left : in.y;
      }
      const bool z_sel = (in.z & 1) || ((in.z & 2) && take >= 1);
      const bool d_sel = (in.z & 4) || ((in.z & 8) && take == in.y);
      cnt = in.x + take + (z_sel ? 0 : 1) + ((l > 0 && !d_sel) ? 1 : 0);
      in.w = take;
      if (l < nb) sm.info[l] = in;
    }
    if (l >= nb) cnt = 0;
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, 64);
      if (l >= o) incl += y;
    }
    int32_t* rp = a.row_ptr + (size_t)h * (nb + 1);
    if (l < nb) {
      sm.rp[l] = incl - cnt;
      rp[l] = incl - cnt;
    }
    if (l == nb - 1) rp[nb] = incl;
  }
  __syncthreads();
  // the lists (csr_fill_row)
  int32_t* out = a.col_idx + (size_t)h * a.col_cap;
#pragma unroll
  for (int i = 0; i < kRowsPerWave; ++i) {
    const int qb = w + (kSmallThreads / 64) * i;
    if (qb >= nb) break;
    const bool on = l <= qb;
    bool sel;
    if (vs) {
      sel = (sm.sel[qb] >> l) & 1;
    } else {
      const uint64_t eq = sm.eqm[qb];
      const bool e = (eq >> l) & 1;
      const int eq_rank = __popcll(eq & lt);
      sel = on && (((sm.sel[qb] >> l) & 1) || (e && eq_rank < sm.info[qb].w) || l == 0 || l == qb);
    }
    const uint64_t bal = __ballot(sel);
    if (sel) out[sm.rp[qb] + __popcll(bal & lt)] = l;
  }
}

}  // namespace

// Full causal lists (the context-length gate): route = dense, row qb = 0..qb.
// grid (nb, hq), 256 threads.
__global__ __launch_bounds__(256) void sel_dense_lists(int8_t* route, int32_t* row_ptr, int32_t* col_idx, int nb,
                                                       int64_t col_cap) {
  const int qb = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const int base = (int)((int64_t)qb * (qb + 1) / 2);
  if (tid == 0) {
    row_ptr[(size_t)h * (nb + 1) + qb] = base;
    if (qb == nb - 1) row_ptr[(size_t)h * (nb + 1) + nb] = base + qb + 1;
    if (qb == 0) route[h] = 2;
  }
  int32_t* out = col_idx + (size_t)h * col_cap + base;
  for (int i = tid; i <= qb; i += 256) out[i] = i;
}

hipError_t launch_dense_lists(const Dims& d, int8_t* route, int32_t* row_ptr, int32_t* col_idx, int64_t col_cap,
                              hipStream_t stream) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  hipLaunchKernelGGL(sel_dense_lists, dim3(d.nb, d.hq), dim3(256), 0, stream, route, row_ptr, col_idx, d.nb, col_cap);
  return hipGetLastError();
}

hipError_t launch_jsd(const Dims& d, float scale, const uint16_t* q, const uint16_t* k, const float* p_v,
                      float* jsd, char* ws, hipStream_t stream) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  const WsLayout L = ws_layout(d);
  JsdArgs a;
  a.q = q; a.k = k; a.p_v = p_v; a.jsd = jsd;
  a.kbar = reinterpret_cast<float*>(ws + L.kbar);
  a.zbuf = reinterpret_cast<float*>(ws + L.atil);  // free until the PE scores of stage 3
  a.n = d.n; a.nb = d.nb; a.B = d.B; a.b = d.b; a.hq = d.hq; a.hkv = d.hkv; a.G = d.G;
  a.scale = scale;
  hipLaunchKernelGGL(jsd_pool_k, dim3(d.nb, d.hkv), dim3(256), 0, stream, a);
  hipLaunchKernelGGL(jsd_score, dim3(d.hq), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_select(const Dims& d, float scale, float alpha, float tau, float gamma, int k_min, int vs_mode,
                         int floor_mode, bool kbar_all, const uint16_t* q, const uint16_t* k, const float* route_score,
                         const float* p_v, const float* p_s, int8_t* route, int32_t* row_ptr, int32_t* col_idx,
                         int64_t col_cap, uint8_t* dir_mask, char* ws, hipStream_t stream, bool scores_from_ws) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  const WsLayout L = ws_layout(d);
  SelArgs a;
  a.q = q; a.k = k; a.c_struct = route_score; a.p_v = p_v; a.p_s = p_s;
  a.route = route; a.row_ptr = row_ptr; a.col_idx = col_idx; a.col_cap = col_cap; a.dir_mask = dir_mask;
  a.n = d.n; a.nb = d.nb; a.B = d.B; a.hq = d.hq; a.hkv = d.hkv; a.G = d.G;
  a.c2 = scale * kLog2e;
  a.alpha = alpha; a.tau = tau; a.gamma = gamma; a.k_min = k_min;
  a.vs_mode = vs_mode; a.floor_mode = floor_mode; a.kbar_all = kbar_all ? 1 : 0;
  a.cap = d.cap;
  a.masks = reinterpret_cast<uint8_t*>(ws + L.masks);
  a.qbar = reinterpret_cast<float*>(ws + L.qbar);
  a.kbar = reinterpret_cast<float*>(ws + L.kbar);
  a.atil = reinterpret_cast<float*>(ws + L.atil);
  a.rhist = reinterpret_cast<unsigned long long*>(ws + L.rhist);
  a.rstate = reinterpret_cast<RState*>(ws + L.rstate);
  a.rowinfo = reinterpret_cast<int4*>(ws + L.rowinfo);
  const int nb = d.nb;
  const bool from_ws = scores_from_ws && nb <= kPeSmall;
  a.parts = from_ws ? reinterpret_cast<const float4*>(ws + L.parts) : nullptr;
  a.rowfinal = from_ws ? reinterpret_cast<const float*>(ws + L.rowfinal) : nullptr;
  a.b = d.b;
  if (nb <= kPeSmall) {  // short layers: pooling, then the whole selection in one launch per head
    hipLaunchKernelGGL(sel_pool, dim3(nb, d.hq + d.hkv), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sel_small, dim3(d.hq), dim3(kSmallThreads), 0, stream, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(sel_route_vs, dim3(d.hq, 2), dim3(1024), 0, stream, a);
  hipLaunchKernelGGL(sel_pool, dim3(nb, d.hq + d.hkv), dim3(256), 0, stream, a);
  if (nb <= kLogitDirect) {
    const int nt = (nb + 63) / 64;
    hipLaunchKernelGGL(sel_pe_logits_direct, dim3(nt * (nt + 1) / 2, d.hq), dim3(256), 0, stream, a);
  } else {
    const int nt = (nb + 127) / 128;
    hipLaunchKernelGGL(sel_pe_logits<64>, dim3(nt * (nt + 1) / 2, d.hq), dim3(256), 0, stream, a);
  }
  hipLaunchKernelGGL(sel_pe_softmax, dim3(nb, d.hq), dim3(256), 0, stream, a);
  if (d.cap <= kSmallCap) {
    hipLaunchKernelGGL(sel_radix_small, dim3(d.hq), dim3(1024), 0, stream, a);
  } else {
    hipLaunchKernelGGL(sel_radix_init, dim3(d.hq), dim3(256), 0, stream, a);
    int64_t chunks = (d.cap + 16383) / 16384;
    if (chunks > 1024) chunks = 1024;
    if (chunks < 1) chunks = 1;
    for (int pass = 0; pass < 3; ++pass) {
      hipLaunchKernelGGL(sel_radix_hist, dim3((unsigned)chunks, d.hq), dim3(256), 0, stream, a, pass);
      hipLaunchKernelGGL(sel_radix_scan, dim3(d.hq), dim3(256), 0, stream, a, pass);
    }
  }
  const int rows_grid = (nb + 3) / 4;
  hipLaunchKernelGGL(sel_csr_count, dim3(rows_grid, d.hq), dim3(256), 0, stream, a);
  hipLaunchKernelGGL(sel_csr_scan, dim3(d.hq), dim3(1024), 0, stream, a);
  hipLaunchKernelGGL(sel_csr_fill, dim3(rows_grid, d.hq), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace crisp
