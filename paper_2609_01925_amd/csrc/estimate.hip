// Stages 1-2: the last-block proxy attention and its reductions (Alg. 2, the
// C_struct equation of Sec. 3.2, and the vertical / slash scores of Alg. 3).
//
// The proxy A_hat (b rows x n keys per head) is never materialised.  Keys are
// split into ranges of whole blocks, one workgroup per (head, range):
//   pass 1  S^T = K Q_hat^T on MFMA, causal mask, per-row running max / sum-exp
//   combine per-row (max, sum) over ranges
//   pass 2  recompute S^T, P = exp(S - max) / sum, and reduce per key block J:
//             column mass      sum over rows and keys of J             -> p_v[J]
//             diagonal mass    split by the slash block of the diagonal
//                              through (last row, key + b - 1 - r):
//                              J itself or J + 1                      -> p_s
//             anchor mass      keys in [0, w_sink) or [n - w_local, n) -> C_struct
//   finalize p_v, p_s, C_struct (deterministic: every partial is written once
//            and summed in a fixed order; no floating-point atomics)
#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

constexpr int BK = 64;
constexpr int kTileBytes = BK * 256;
constexpr int NT = 256;  // 4 waves; wave w owns proxy rows 32w .. 32w + 31

struct EstArgs {
  const uint16_t* q;
  const uint16_t* k;
  int n, nb, B, b, hq, G, bps, splits;
  float c;  // softmax scale * log2(e)
  int w_sink, w_local;
  float* rowstat;   // [hq][splits][128][2]  (max of raw scores, sum of exp2)
  float* rowfinal;  // [hq][128][2]
  float4* parts;    // [hq][nb]  (column, diagonal-low, diagonal-high, anchor)
  float* c_struct;
  float* p_v;
  float* p_s;
};

__device__ __forceinline__ void load_q_hat(const EstArgs& a, int h, int r, int l, bf16x8 (&qf)[8]) {
  const int qi = a.n - a.b + r;
  const bool ok = r < a.b;
  const uint16_t* qrow = a.q + ((size_t)h * a.n + (ok ? qi : 0)) * kHeadDim;
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 16 * kk + 8 * (l >> 5));
    if (!ok) raw = u32x4{0, 0, 0, 0};
    qf[kk] = __builtin_bit_cast(bf16x8, raw);
  }
}

// K tile of 64 keys (keys at or past n read as 0): 16 bytes x 4 per thread into
// registers, then into an LDS buffer.  The next tile is loaded into registers
// before the current one's MFMAs, so its latency overlaps them.
__device__ __forceinline__ void load_k_regs(u32x4 (&t)[4], const uint16_t* Kg, int key0, int n, int tid) {
  const int c = tid & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int key = key0 + (tid >> 4) + 16 * i;
    t[i] = key < n ? *reinterpret_cast<const u32x4*>(Kg + (size_t)key * kHeadDim + 8 * c) : u32x4{0, 0, 0, 0};
  }
}

__device__ __forceinline__ void store_k_regs(char* buf, const u32x4 (&t)[4], int tid) {
  const int c = tid & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(buf + lds_off((tid >> 4) + 16 * i, 8 * c)) = t[i];
}

__device__ __forceinline__ void scores(const char* kbuf, const bf16x8 (&qf)[8], int l, f32x16 (&s)[2]) {
  s[0] = zero16();
  s[1] = zero16();
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    const int d = 16 * kk + 8 * (l >> 5);
    s[0] = mfma32(lds_read16(kbuf, lds_off(l & 31, d)), qf[kk], s[0]);
    s[1] = mfma32(lds_read16(kbuf, lds_off(32 + (l & 31), d)), qf[kk], s[1]);
  }
}

__device__ __forceinline__ int key_of(int key0, int mb, int i, int l) {
  return key0 + 32 * mb + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3);
}

// Pass 1: per (head, key range) running max and sum of exp2((s - max) * c) per proxy row.
__global__ __launch_bounds__(NT) void est_rowstats(EstArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kTileBytes];
  const int h = blockIdx.x / a.splits, sp = blockIdx.x % a.splits;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int r = 32 * w + (l & 31);
  const int qi = a.n - a.b + r;
  bf16x8 qf[8];
  load_q_hat(a, h, r, l, qf);
  const uint16_t* Kg = a.k + (size_t)(h / a.G) * a.n * kHeadDim;
  const int key_lo = sp * a.bps * a.B;
  int key_hi = key_lo + a.bps * a.B;
  key_hi = key_hi < a.n ? key_hi : a.n;
  float m_run = -__builtin_inff(), l_run = 0.f;
  int buf = 0;
  u32x4 pre[4];
  if (key_lo < key_hi) load_k_regs(pre, Kg, key_lo, a.n, tid);
  for (int key0 = key_lo; key0 < key_hi; key0 += BK, buf ^= 1) {
    char* kb = smem + buf * kTileBytes;
    store_k_regs(kb, pre, tid);
    if (key0 + BK < key_hi) load_k_regs(pre, Kg, key0 + BK, a.n, tid);
    __syncthreads();
    f32x16 s[2];
    scores(kb, qf, l, s);
    float mx = -__builtin_inff();
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (r >= a.b || key_of(key0, mb, i, l) > qi) s[mb][i] = -__builtin_inff();
        mx = fmaxf(mx, s[mb][i]);
      }
    mx = fmaxf(mx, swap_halves(mx));
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -__builtin_inff() ? 0.f : m_new;
    float ps = 0.f;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) ps += fast_exp2((s[mb][i] - m_use) * a.c);
    l_run = l_run * fast_exp2((m_run - m_use) * a.c) + ps;
    m_run = m_new;
  }
  l_run += swap_halves(l_run);
  if (l < 32 && r < a.b) {
    float* dst = a.rowstat + (((size_t)h * a.splits + sp) * 128 + r) * 2;
    dst[0] = m_run;
    dst[1] = l_run;
  }
}

// Combine the per-range row statistics: eight lanes per proxy row, each taking every
// eighth range, then a max and a sum over the eight (fixed order).  grid (hq, 4),
// 256 threads = 32 rows x 8 lanes.
__global__ __launch_bounds__(256) void est_combine(EstArgs a) {
  const int h = blockIdx.x, j = threadIdx.x & 7;
  const int r = 32 * blockIdx.y + (threadIdx.x >> 3);
  const float2* src = reinterpret_cast<const float2*>(a.rowstat) + (size_t)h * a.splits * 128 + r;
  float M = -__builtin_inff();
  for (int sp = j; sp < a.splits; sp += 8) M = fmaxf(M, src[(size_t)sp * 128].x);
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) M = fmaxf(M, __shfl_xor(M, o, 64));
  float L = 0.f;
  for (int sp = j; sp < a.splits; sp += 8) {
    const float2 ml = src[(size_t)sp * 128];
    if (ml.x != -__builtin_inff()) L += ml.y * fast_exp2((ml.x - M) * a.c);
  }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) L += __shfl_xor(L, o, 64);
  if (j == 0 && r < a.b) {
    a.rowfinal[((size_t)h * 128 + r) * 2] = M;
    a.rowfinal[((size_t)h * 128 + r) * 2 + 1] = L;
  }
}

__device__ __forceinline__ void block_reduce4(float4 v, float4* red, int tid, float4* out) {
  v.x = wave_sum(v.x);
  v.y = wave_sum(v.y);
  v.z = wave_sum(v.z);
  v.w = wave_sum(v.w);
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  if (tid == 0) {
    float4 t = red[0];
    for (int i = 1; i < NT / 64; ++i) {
      t.x += red[i].x; t.y += red[i].y; t.z += red[i].z; t.w += red[i].w;
    }
    *out = t;
  }
  __syncthreads();
}

// Pass 2: normalised proxy entries reduced per key block.
__global__ __launch_bounds__(NT) void est_reduce(EstArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kTileBytes];
  __shared__ float4 red[NT / 64];
  const int h = blockIdx.x / a.splits, sp = blockIdx.x % a.splits;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int r = 32 * w + (l & 31);
  const int qi = a.n - a.b + r;
  const bool row_ok = r < a.b;
  bf16x8 qf[8];
  load_q_hat(a, h, r, l, qf);
  // A_hat = 2^(s c - M c) / L = 2^(s c - mcl) with mcl = M c + log2 L; rows past b
  // (64-row blocks) get mcl = +inf, so every entry of theirs is exactly 0.
  float mcl = __builtin_inff();
  if (row_ok) mcl = a.rowfinal[((size_t)h * 128 + r) * 2] * a.c + log2f(a.rowfinal[((size_t)h * 128 + r) * 2 + 1]);
  const uint16_t* Kg = a.k + (size_t)(h / a.G) * a.n * kHeadDim;
  const int J0 = sp * a.bps;
  const int J1 = (J0 + a.bps < a.nb) ? J0 + a.bps : a.nb;
  const int diag_off = a.b - 1 - r;  // key k of row r lies on the diagonal through (last row, k + diag_off)
  int buf = 0;
  u32x4 pre[4];
  if (J0 < J1) load_k_regs(pre, Kg, J0 * a.B, a.n, tid);
  for (int J = J0; J < J1; ++J) {
    float lo = 0.f, hi = 0.f, anc = 0.f;  // diagonal mass staying in J / moving to J + 1; anchor mass
    const int blo = J * a.B;
    const int bhi = blo + a.B < a.n ? blo + a.B : a.n;
    const int ksplit = (J + 1) * a.B - diag_off;  // keys >= this lie on diagonals of slash block J + 1
    for (int key0 = blo; key0 < bhi; key0 += BK, buf ^= 1) {
      char* kb = smem + buf * kTileBytes;
      store_k_regs(kb, pre, tid);
      const int next = key0 + BK < bhi ? key0 + BK : (J + 1 < J1 ? (J + 1) * a.B : a.n);
      if (next < a.n) load_k_regs(pre, Kg, next, a.n, tid);
      __syncthreads();
      f32x16 s[2];
      scores(kb, qf, l, s);
      // Tiles wholly before the first proxy row, inside the block and outside both anchor
      // windows (all but a few) need no per-entry masks and no anchor sum.
      const bool plain = key0 + BK - 1 <= a.n - a.b && key0 + BK <= bhi && key0 >= a.w_sink &&
                         key0 + BK <= a.n - a.w_local;
      if (plain) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float p = fast_exp2(__builtin_fmaf(s[mb][i], a.c, -mcl));
            if (key_of(key0, mb, i, l) < ksplit) lo += p; else hi += p;
          }
      } else {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = key_of(key0, mb, i, l);
            float p = 0.f;
            if (key <= qi && key < bhi) p = fast_exp2(__builtin_fmaf(s[mb][i], a.c, -mcl));
            if (key < ksplit) lo += p; else hi += p;
            if (key < a.w_sink || key >= a.n - a.w_local) anc += p;
          }
      }
    }
    block_reduce4(make_float4(lo + hi, lo, hi, anc), red, tid, a.parts + (size_t)h * a.nb + J);
  }
}

// p_v[J] = column mass / b;  p_s[J] = (diag-low[J] + diag-high[J-1]) / b;  C_struct = anchor mass / b.
__global__ __launch_bounds__(256) void est_finalize(EstArgs a) {
  __shared__ float red[256];
  const int h = blockIdx.x, tid = threadIdx.x;
  const float4* P = a.parts + (size_t)h * a.nb;
  const float invb = 1.f / (float)a.b;
  float anch = 0.f;
  for (int J = tid; J < a.nb; J += 256) {
    const float4 cur = P[J];
    const float prev_hi = J > 0 ? P[J - 1].z : 0.f;
    a.p_v[(size_t)h * a.nb + J] = cur.x * invb;
    a.p_s[(size_t)h * a.nb + J] = (cur.y + prev_hi) * invb;
    anch += cur.w;
  }
  red[tid] = anch;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) red[tid] += red[tid + s];
    __syncthreads();
  }
  if (tid == 0) a.c_struct[h] = red[0] * invb;
}

}  // namespace

EstSplit est_split(const Dims& d) {
  EstSplit s;
  const int64_t want = 2048;  // target workgroups for pass 1 / pass 2
  int64_t bps = ((int64_t)d.nb * d.hq + want - 1) / want;
  if (bps < 1) bps = 1;
  s.bps = (int)bps;
  s.splits = (d.nb + s.bps - 1) / s.bps;
  if (s.splits < 1) s.splits = 1;
  return s;
}

hipError_t launch_estimate(const Dims& d, float scale, int w_sink, int w_local, const uint16_t* q,
                           const uint16_t* k, float* c_struct, float* p_v, float* p_s, char* ws,
                           hipStream_t stream) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  const WsLayout L = ws_layout(d);
  const EstSplit sp = est_split(d);
  EstArgs a;
  a.q = q; a.k = k;
  a.n = d.n; a.nb = d.nb; a.B = d.B; a.b = d.b; a.hq = d.hq; a.G = d.G;
  a.bps = sp.bps; a.splits = sp.splits;
  a.c = scale * kLog2e;
  a.w_sink = w_sink; a.w_local = w_local;
  a.rowstat = reinterpret_cast<float*>(ws + L.rowstat);
  a.rowfinal = reinterpret_cast<float*>(ws + L.rowfinal);
  a.parts = reinterpret_cast<float4*>(ws + L.parts);
  a.c_struct = c_struct; a.p_v = p_v; a.p_s = p_s;
  const int grid = d.hq * sp.splits;
  hipLaunchKernelGGL(est_rowstats, dim3(grid), dim3(NT), 0, stream, a);
  hipLaunchKernelGGL(est_combine, dim3(d.hq, 4), dim3(256), 0, stream, a);
  hipLaunchKernelGGL(est_reduce, dim3(grid), dim3(NT), 0, stream, a);
  hipLaunchKernelGGL(est_finalize, dim3(d.hq), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace crisp
