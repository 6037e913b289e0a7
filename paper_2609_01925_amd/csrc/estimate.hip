// Stages 1-2: the last-block proxy attention and its reductions (Alg. 2, the
// C_struct equation of Sec. 3.2, and the vertical / slash scores of Alg. 3).
//
// The proxy A_hat (b rows x n keys per head) is never materialised, and K is read
// once.  Keys are split into ranges of whole blocks, one workgroup per (head, range):
//   pass     S^T = K Q_hat^T on MFMA, causal mask, and per proxy row a running max
//            with, under it, sums of exp2((s - max) c): over all keys, over the
//            anchor keys ([0, w_sink) and [n - w_local, n)), and per key block J
//            split by the slash block of the diagonal through (last row,
//            key + b - 1 - r): J itself (lo) or J + 1 (hi).  Per (row, J) the pair
//            (lo, hi) is stored with the max it was summed under.
//   combine  per row: max M and sum L over ranges; C_struct = (1/b) sum_r anchor / L
//   scale    p_v[J] = (1/b) sum_r (lo + hi) 2^((m - M) c) / L,
//            p_s[J] = (1/b) sum_r (lo[J] + hi[J - 1]) scaled alike
// Deterministic: every partial is written once and summed in a fixed order; no
// floating-point atomics.
#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

constexpr int BK = 64;
constexpr int kTileBytes = BK * 256;
constexpr int NT = 256;  // 4 waves; wave w owns proxy rows 32w .. 32w + 31
constexpr float kSumLimit = 256.0f;  // a lane's tile sum above this raises the running max

struct EstArgs {
  const uint16_t* q;
  const uint16_t* k;
  int n, nb, B, b, hq, G, bps, splits;
  float c;  // softmax scale * log2(e)
  int w_sink, w_local;
  float4* rowstat;  // [hq][splits][128]  (max of raw scores, sum of exp2, anchor sum, -)
  float* rowfinal;  // [hq][128]  M c + log2 L per proxy row (+inf past b)
  float4* parts;    // [hq][nb][128]  (diagonal-low, diagonal-high, max they were summed under, -)
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

#if defined(__HIP_DEVICE_COMPILE__)
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

// S^T of one 64-key tile (keys on M, the wave's 32 proxy rows on N) from the
// swizzled K stage at LDS address kbuf.
__device__ __forceinline__ void scores(int kbuf, const bf16x8 (&qf)[8], int l, f32x16 (&s)[2]) {
  s[0] = zero16();
  s[1] = zero16();
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    const int d = 16 * kk + 8 * (l >> 5);
    // rows r and r + 32 share a swizzle: the second read is the first address + 32 rows
    const int addr = kbuf + lds_off(l & 31, d);
    const bf16x8 k0 = *(const lds_bf16x8*)(uint32_t)addr;
    const bf16x8 k1 = *(const lds_bf16x8*)(uint32_t)(addr + 32 * 256);
    s[0] = mfma32(k0, qf[kk], s[0]);
    s[1] = mfma32(k1, qf[kk], s[1]);
  }
}
#endif

__device__ __forceinline__ int key_of(int key0, int mb, int i, int l) {
  return key0 + 32 * mb + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3);
}

// One pass over K: scores, causal mask, and per proxy row, under a running max, the
// sums of exp2((s - max) c): per key block J split by slash block (lo: keys whose
// diagonal through the last proxy row stays in J, hi: those moving to J + 1), over the
// anchor keys (anchor mass), and over all its keys (l, the blocks' lo + hi added as each
// block ends).  K tiles go straight from global memory into a two-stage LDS ring
// (LDS-DMA; keys at or past n read as 0), the next tile's load issued as the current
// one is scored.  The running max is raised lazily: a tile's terms are formed against
// the current max, and only when some lane's tile sum exceeds 2^8 (or is not finite)
// is the tile's true row max taken, the open sums scaled down to it and the terms
// formed again -- until then every term is at most 2^8, which float32 holds as exactly
// as terms below 1; while a row of the wave has no max yet, the max is taken first.  A block's (lo, hi) is written with the
// max it was summed under when the block ends, and the range's (max, l, anchor) when
// the range ends.
__global__ __launch_bounds__(NT, 4) void est_pass(EstArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  __shared__ __attribute__((aligned(1024))) char smem[2 * kTileBytes];
  const int lds0 = __builtin_amdgcn_readfirstlane((int)(size_t)smem);
  // Workgroup i runs on XCD i % 8.  The G query heads of one (KV group, key range) take
  // consecutive workgroups of one XCD, so they stream the same K tiles through that
  // XCD's L2 at about the same time (K is read from HBM about once, not once per head).
  const int xcd = blockIdx.x % kNumXcd, slot = blockIdx.x / kNumXcd;
  const int pair = (slot / a.G) * kNumXcd + xcd;  // (KV group, range) pair, range fastest
  if (pair >= (a.hq / a.G) * a.splits) return;
  const int h = (pair / a.splits) * a.G + slot % a.G, sp = pair % a.splits;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
  const int r = 32 * w + (l & 31);
  const int qi = a.n - a.b + r;
  const bool row_ok = r < a.b;
  bf16x8 qf[8];
  load_q_hat(a, h, r, l, qf);
  Fetch<4> fe;
  make_fetch<4>(fe, w, l);
  const i32x4 rk = tensor_rsrc(a.k + (size_t)(h / a.G) * a.n * kHeadDim, a.n);
  const int J0 = sp * a.bps;
  const int J1 = (J0 + a.bps < a.nb) ? J0 + a.bps : a.nb;
  const int diag_off = a.b - 1 - r;  // key k of row r lies on the diagonal through (last row, k + diag_off)
  float m_run = -__builtin_inff(), l_run = 0.f, anc = 0.f;
  // tiles of the range in order: block J holds ceil(len / 64) tiles starting at J * B
  const int tpb = a.B / BK;
  const int key_end = J1 * a.B < a.n ? J1 * a.B : a.n;
  const int T = J0 < J1 ? (key_end - J0 * a.B + BK - 1) / BK : 0;
  // the first two tiles are loaded together (one latency for ranges of two tiles);
  // after that each step loads the tile after the current one
  if (T > 0) fetch_tile<4, BK>(fe, rk, lds0, J0 * a.B, w);
  if (T > 1) fetch_tile<4, BK>(fe, rk, lds0 + kTileBytes, (J0 + 1 / tpb) * a.B + (1 % tpb) * BK, w);
  float lo = 0.f, hi = 0.f;
  for (int t = 0; t < T; ++t) {
    const int J = J0 + t / tpb;
    const int key0 = J * a.B + (t % tpb) * BK;
    const int blo = J * a.B;
    const int bhi = blo + a.B < a.n ? blo + a.B : a.n;
    const int ksplit = (J + 1) * a.B - diag_off;  // keys >= this lie on diagonals of slash block J + 1
    wait_dma();
    __syncthreads();  // tile t has landed for every wave; every wave is done with tile t - 1's stage
    if (t >= 1 && t + 1 < T) {
      const int Jn = J0 + (t + 1) / tpb;
      fetch_tile<4, BK>(fe, rk, lds0 + ((t + 1) & 1) * kTileBytes, Jn * a.B + ((t + 1) % tpb) * BK, w);
    }
    f32x16 s[2];
    scores(lds0 + (t & 1) * kTileBytes, qf, l, s);
    // Tiles wholly before the first proxy row, inside the block and outside both anchor
    // windows (all but a few) need no per-entry masks and no anchor sum.
    const bool plain = key0 + BK - 1 <= a.n - a.b && key0 + BK <= bhi && key0 >= a.w_sink &&
                       key0 + BK <= a.n - a.w_local;
    if (!plain) {
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = key_of(key0, mb, i, l);
          if (!row_ok || key > qi || key >= bhi) s[mb][i] = -__builtin_inff();
        }
    }
    // In most tiles a whole wave's entries fall on one side of its rows' slash split
    // (the split sits at key offset r + 1 of the block): one sum, no per-entry test.
    const bool all_lo = __all(key0 + BK - 1 < ksplit), all_hi = __all(key0 >= ksplit);
    float tlo = 0.f, thi = 0.f, tanc = 0.f;
    // every entry tested against the slash split and the anchor windows (masked entries
    // give exp2(-inf) = 0): the tiles that need it, and the rare tile that raises the max
    auto general = [&](float mc) {
      tlo = 0.f;
      thi = 0.f;
      tanc = 0.f;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = key_of(key0, mb, i, l);
          const float p = fast_exp2(__builtin_fmaf(s[mb][i], a.c, -mc));
          if (key < ksplit) tlo += p; else thi += p;
          if (key < a.w_sink || key >= a.n - a.w_local) tanc += p;
        }
    };
    // A wave with a row that has no running max yet (its first tiles) goes straight to
    // the raise below: terms formed against no max would only be dropped there.
    const bool fresh = __ballot(row_ok && m_run == -__builtin_inff()) != 0;
    const float mc0 = m_run == -__builtin_inff() ? 0.f : m_run * a.c;
    if (fresh) {
      // the raise forms this tile's terms
    } else if (plain && (all_lo || all_hi)) {
      float t0 = 0.f, t1 = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        t0 += fast_exp2(__builtin_fmaf(s[0][i], a.c, -mc0));
        t1 += fast_exp2(__builtin_fmaf(s[1][i], a.c, -mc0));
      }
      if (all_lo) tlo = t0 + t1; else thi = t0 + t1;
    } else if (plain) {
      // The wave's rows cross the split inside one 32-key half of the tile; the other
      // half lies on one side of it.  Only the straddling half is tested per entry,
      // against a per-lane limit (the lane's keys in a half are 4 (l >> 5) plus the
      // offsets 8 (i >> 2) + (i & 3), increasing with i).
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const int c0 = key0 + 32 * mb;
        if (__all(c0 + 31 < ksplit) || __all(c0 >= ksplit)) {
          float u = 0.f;
#pragma unroll
          for (int i = 0; i < 16; ++i) u += fast_exp2(__builtin_fmaf(s[mb][i], a.c, -mc0));
          if (c0 < ksplit) tlo += u; else thi += u;
        } else {
          const int lim = ksplit - c0 - 4 * (l >> 5);
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float p = fast_exp2(__builtin_fmaf(s[mb][i], a.c, -mc0));
            if (8 * (i >> 2) + (i & 3) < lim) tlo += p; else thi += p;
          }
        }
      }
    } else {
      general(mc0);
    }
    const float tsum = tlo + thi;
    if (fresh || __ballot(row_ok && !(tsum <= kSumLimit))) {
      float mx = vmax(s[0][0], s[1][0]);
#pragma unroll
      for (int i = 1; i < 16; ++i) mx = vmax(mx, vmax(s[0][i], s[1][i]));
      mx = vmax(mx, swap_halves(mx));  // the same in both lanes of a row
      if (mx > m_run) {
        const float alpha = m_run == -__builtin_inff() ? 0.f : fast_exp2((m_run - mx) * a.c);
        l_run *= alpha;
        anc *= alpha;
        lo *= alpha;
        hi *= alpha;
        m_run = mx;
      }
      general(m_run == -__builtin_inff() ? 0.f : m_run * a.c);
    }
    lo += tlo;
    hi += thi;
    anc += tanc;
    if ((t + 1) % tpb == 0 || t + 1 == T) {  // block J ends
      l_run += lo + hi;  // the block's sum joins the row's, under the same running max
      const float slo = lo + swap_halves(lo), shi = hi + swap_halves(hi);
      if (l < 32 && row_ok) a.parts[((size_t)h * a.nb + J) * 128 + r] = make_float4(slo, shi, m_run, 0.f);
      lo = 0.f;
      hi = 0.f;
    }
  }
  l_run += swap_halves(l_run);
  anc += swap_halves(anc);
  if (l < 32 && row_ok) a.rowstat[((size_t)h * a.splits + sp) * 128 + r] = make_float4(m_run, l_run, anc, 0.f);
#endif
}

// Merges a range's (max m, sums l and anchor under m) into a running (M, L, A).
__device__ __forceinline__ void merge_stats(float& M, float& L, float& A, float m, float l, float anc, float c) {
  if (m == -__builtin_inff()) return;
  if (m > M) {
    const float f = M == -__builtin_inff() ? 0.f : fast_exp2((M - m) * c);
    L = L * f + l;
    A = A * f + anc;
    M = m;
  } else {
    const float f = fast_exp2((m - M) * c);
    L += l * f;
    A += anc * f;
  }
}

// Per query head: each proxy row's max M and sum L over all ranges (eight lanes per
// row, each merging every eighth range in one pass, then a fixed-order butterfly),
// the row's normaliser mcl = M c + log2 L for the block sums, and C_struct = (1/b)
// sum over rows of the row's anchor mass / L, summed over rows in a fixed order.
// 1024 threads.
__device__ __forceinline__ void combine_head(const EstArgs& a, int h, float* red) {
  const int j = threadIdx.x & 7, r = threadIdx.x >> 3;
  const float4* src = a.rowstat + (size_t)h * a.splits * 128 + r;
  const bool row_ok = r < a.b;
  float M = -__builtin_inff(), L = 0.f, A = 0.f;
  if (row_ok)
    for (int sp = j; sp < a.splits; sp += 8) {
      const float4 st = src[(size_t)sp * 128];
      merge_stats(M, L, A, st.x, st.y, st.z, a.c);
    }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) {
    const float m2 = __shfl_xor(M, o, 64), l2 = __shfl_xor(L, o, 64), a2 = __shfl_xor(A, o, 64);
    merge_stats(M, L, A, m2, l2, a2, a.c);
  }
  if (j == 0) {
    a.rowfinal[(size_t)h * 128 + r] = row_ok ? M * a.c + log2f(L) : __builtin_inff();
    red[r] = row_ok ? A / L : 0.f;
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    float t = red[threadIdx.x] + red[threadIdx.x + 64];
    t = wave_sum(t);
    if (threadIdx.x == 0) a.c_struct[h] = t / (float)a.b;
  }
}

__global__ __launch_bounds__(1024) void est_combine(EstArgs a) {
  __shared__ float red[128];
  combine_head(a, blockIdx.x, red);
}

// p_v[J] = (1/b) sum_r (lo + hi)[r][J] 2^(m c - mcl_r);  p_s[J] = (1/b) sum_r (lo[r][J] +
// hi[r][J - 1]) scaled alike, for the run of blocks [Ja, Jb) of head h, by one wave:
// lanes take rows l and l + 64, and a block's row sum is a fixed-order butterfly.
__device__ __forceinline__ void scale_run(const EstArgs& a, int h, int Ja, int Jb) {
  const int l = threadIdx.x & 63;
  const bool ok0 = l < a.b, ok1 = l + 64 < a.b;
  const float mcl0 = ok0 ? a.rowfinal[(size_t)h * 128 + l] : 0.f;
  const float mcl1 = ok1 ? a.rowfinal[(size_t)h * 128 + l + 64] : 0.f;
  const float4* P = a.parts + (size_t)h * a.nb * 128;
  float prev_hi = 0.f;
  if (Ja > 0) {
    float slo;
    proxy_block_sums(P, Ja - 1, a.c, mcl0, mcl1, ok0, ok1, &slo, &prev_hi);
  }
  const float invb = 1.f / (float)a.b;
  for (int J = Ja; J < Jb; ++J) {
    float slo, shi;
    proxy_block_sums(P, J, a.c, mcl0, mcl1, ok0, ok1, &slo, &shi);
    if (l == 0) {
      a.p_v[(size_t)h * a.nb + J] = (slo + shi) * invb;
      a.p_s[(size_t)h * a.nb + J] = (slo + prev_hi) * invb;
    }
    prev_hi = shi;
  }
}

// Each wave takes kScaleRun consecutive blocks.  grid (hq, ceil(runs / 4)), 256 threads.
constexpr int kScaleRun = 2;
__global__ __launch_bounds__(256) void est_scale(EstArgs a) {
  const int Ja = (blockIdx.y * 4 + (threadIdx.x >> 6)) * kScaleRun;
  if (Ja >= a.nb) return;
  scale_run(a, blockIdx.x, Ja, Ja + kScaleRun < a.nb ? Ja + kScaleRun : a.nb);
}

// Short layers (N_b <= kFinishSmall): combine and scale of one head in one launch (the
// 16 waves then take runs of blocks; the same sums in the same order as the two
// kernels above).  grid hq, 1024 threads.
constexpr int kFinishSmall = 32;
__global__ __launch_bounds__(1024) void est_finish(EstArgs a) {
  __shared__ float red[128];
  const int h = blockIdx.x;
  combine_head(a, h, red);
  __syncthreads();  // rowfinal of every row is visible to the whole workgroup
  for (int Ja = (threadIdx.x >> 6) * kScaleRun; Ja < a.nb; Ja += 16 * kScaleRun)
    scale_run(a, h, Ja, Ja + kScaleRun < a.nb ? Ja + kScaleRun : a.nb);
}

}  // namespace

EstSplit est_split(const Dims& d) {
  EstSplit s;
  // Target: one resident round of workgroups (4 per CU), never more.  Each head gets at
  // most want / hq ranges, so the (head, range) pairs fit one round; rounding the
  // blocks per range over all heads at once (ceil(nb hq / want)) could leave a few
  // pairs to a second round that then runs almost alone (12 of 1036 at 512k tokens,
  // 28 heads: 0.80 -> 0.72 ms).
  const int64_t want = 1024;
  int64_t per_head = want / (d.hq > 0 ? d.hq : 1);
  if (per_head < 1) per_head = 1;
  int64_t bps = ((int64_t)d.nb + per_head - 1) / per_head;
  if (bps < 1) bps = 1;
  s.bps = (int)bps;
  s.splits = (d.nb + s.bps - 1) / s.bps;
  if (s.splits < 1) s.splits = 1;
  return s;
}

hipError_t launch_estimate(const Dims& d, float scale, int w_sink, int w_local, const uint16_t* q,
                           const uint16_t* k, float* c_struct, float* p_v, float* p_s, char* ws,
                           hipStream_t stream, bool combine_only) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  const WsLayout L = ws_layout(d);
  const EstSplit sp = est_split(d);
  EstArgs a;
  a.q = q; a.k = k;
  a.n = d.n; a.nb = d.nb; a.B = d.B; a.b = d.b; a.hq = d.hq; a.G = d.G;
  a.bps = sp.bps; a.splits = sp.splits;
  a.c = scale * kLog2e;
  a.w_sink = w_sink; a.w_local = w_local;
  a.rowstat = reinterpret_cast<float4*>(ws + L.rowstat);
  a.rowfinal = reinterpret_cast<float*>(ws + L.rowfinal);
  a.parts = reinterpret_cast<float4*>(ws + L.parts);
  a.c_struct = c_struct; a.p_v = p_v; a.p_s = p_s;
  const int pairs = d.hkv * sp.splits;  // (KV group, key range) pairs, spread over the XCDs
  const int grid = kNumXcd * d.G * ((pairs + kNumXcd - 1) / kNumXcd);
  hipLaunchKernelGGL(est_pass, dim3(grid), dim3(NT), 0, stream, a);
  if (combine_only) {  // p_v and p_s are left to the caller's next launch (from parts and rowfinal)
    hipLaunchKernelGGL(est_combine, dim3(d.hq), dim3(1024), 0, stream, a);
  } else if (d.nb <= kFinishSmall) {
    hipLaunchKernelGGL(est_finish, dim3(d.hq), dim3(1024), 0, stream, a);
  } else {
    hipLaunchKernelGGL(est_combine, dim3(d.hq), dim3(1024), 0, stream, a);
    const int runs = (d.nb + kScaleRun - 1) / kScaleRun;
    hipLaunchKernelGGL(est_scale, dim3(d.hq, (runs + 3) / 4), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace crisp
