// Block-sparse causal flash attention (Eq. 1 of the paper, restricted to the
// selected key blocks) and the dense causal baseline, for gfx950.
//
// A workgroup computes one (query head, query block) unit at a time: BQ = B
// query rows, BQ / 32 waves, each wave owning 32 query rows.  Key blocks are
// streamed in tiles of 64 keys through double-buffered, swizzled LDS.  Per tile
// and wave:
//   S^T (64 keys x 32 queries) = K_tile Q^T      16 x v_mfma_f32_32x32x16_bf16
//   online softmax in fp32 (exp2, log2(e) folded into the scale)
//   O^T (128 d x 32 queries) += V^T P^T          16 x v_mfma_f32_32x32x16_bf16
// The score tile is transposed so that a lane owns one query: row maxima and
// sums are lane-local plus one v_permlane32_swap with lane l ^ 32.  The C
// layout of S^T is reused directly as the B operand of the PV product; V^T
// operands come from LDS through ds_read_b64_tr_b16, which transposes 4 keys x
// 16 dims per 16-lane group, so V needs no transposed copy.
// The score MFMAs of tile j+1 are issued before the softmax of tile j, so
// matrix cores and vector ALU can overlap within a wave.
// The running max is only raised when a row's max grows by more than 2^8
// (log2 units): until then P may exceed 1 by at most 2^8, which fp32 and bf16
// hold exactly as well, and the O accumulators are left untouched.
//
// Sparse lists are processed by a persistent grid that pulls units from a
// longest-first work list (built by attn_schedule from the list lengths), so
// long PE rows start first and short VS rows fill the tail.
#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

constexpr int BK = 64;                  // keys per tile
constexpr int kTileBytes = BK * 256;    // one K or V tile: 64 rows x 128 bf16
constexpr float kLazyRescale = 8.0f;    // log2 growth of a row max tolerated before rescaling
constexpr int kCostBuckets = 8192;

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  int64_t col_cap;
  const int32_t* order;  // persistent mode: units sorted longest first
  int* counter;          // persistent mode: next position in `order`
  int n, nb, hq, hkv, G;
  float c;        // softmax scale * log2(e)
  int map_mode;   // static grid: 0 natural order, 1 H_kv % 8 == 0, 2 8 % H_kv == 0
  int rep;        // map_mode 2: XCDs per KV group
};

// Static grid: workgroup -> (head, query block).  Units of one KV group are kept
// on one XCD (its L2 then serves the group's K/V to all G heads), and longer
// rows (higher qb) are dispatched first.
__device__ __forceinline__ bool map_unit(const AttnArgs& a, int bid, int& h, int& qb) {
  if (a.map_mode == 0) {
    if (bid >= a.hq * a.nb) return false;
    qb = a.nb - 1 - bid / a.hq;
    h = bid % a.hq;
    return true;
  }
  const int x = bid % kNumXcd, u = bid / kNumXcd;
  if (a.map_mode == 1) {
    const int gpx = a.hkv / kNumXcd;
    const int per = gpx * a.G;
    const int r = u / per;
    if (r >= a.nb) return false;
    const int w = u % per;
    qb = a.nb - 1 - r;
    h = (x + kNumXcd * (w / a.G)) * a.G + (w % a.G);
    return true;
  }
  const int g = x % a.hkv, par = x / a.hkv;
  if (par > a.nb - 1) return false;
  const int top = a.nb - 1 - ((a.nb - 1 - par) % a.rep);
  const int r = u / a.G;
  qb = top - r * a.rep;
  if (qb < 0) return false;
  h = g * a.G + (u % a.G);
  return true;
}

template <int NT>
struct TileRegs {
  static constexpr int N = (BK * 16) / NT;  // 16-byte chunks per thread per tile
  u32x4 k[N];
  u32x4 v[N];
};

template <int NT>
__device__ __forceinline__ void load_tile(TileRegs<NT>& t, const uint16_t* Kg, const uint16_t* Vg, int key0, int n,
                                          int tid) {
  const int c = tid & 15;
#pragma unroll
  for (int i = 0; i < TileRegs<NT>::N; ++i) {
    const int r = (tid >> 4) + (NT / 16) * i;
    const int key = key0 + r;
    if (key < n) {
      t.k[i] = *reinterpret_cast<const u32x4*>(Kg + (size_t)key * kHeadDim + 8 * c);
      t.v[i] = *reinterpret_cast<const u32x4*>(Vg + (size_t)key * kHeadDim + 8 * c);
    } else {
      t.k[i] = u32x4{0, 0, 0, 0};
      t.v[i] = u32x4{0, 0, 0, 0};
    }
  }
}

template <int NT>
__device__ __forceinline__ void store_tile(const TileRegs<NT>& t, char* kbuf, char* vbuf, int tid) {
  const int c = tid & 15;
#pragma unroll
  for (int i = 0; i < TileRegs<NT>::N; ++i) {
    const int r = (tid >> 4) + (NT / 16) * i;
    const int off = lds_off(r, 8 * c);
    *reinterpret_cast<u32x4*>(kbuf + off) = t.k[i];
    *reinterpret_cast<u32x4*>(vbuf + off) = t.v[i];
  }
}

// Per-lane LDS byte offsets of the MFMA operand reads, fixed for the whole kernel.
// K (A operand of S^T): row l % 32 (+32 per key sub-block, an immediate), chunk
// 2 kk + l / 32.  V^T (A operand of O^T, transposing reads): two reads per MFMA,
// rows r0 and r0 + 8 (+16 ss + 32 mb, immediates), dims 32 db + 16 (grp & 1) + 4 (jj & 3).
struct Offsets {
  int k[8];
  int v[4][2];
};

__device__ __forceinline__ void make_offsets(Offsets& off, int l) {
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) off.k[kk] = lds_off(l & 31, 16 * kk + 8 * (l >> 5));
  const int grp = l >> 4, jj = l & 15;
  const int row = 4 * (grp >> 1) + (jj >> 2);
#pragma unroll
  for (int db = 0; db < 4; ++db) {
    const int col = 32 * db + 16 * (grp & 1) + 4 * (jj & 3);
    off.v[db][0] = lds_off(row, col);
    off.v[db][1] = lds_off(row + 8, col);
  }
}

// S^T for one tile: s[mb] covers keys 32 * mb + (C-layout rows), queries = lane column.
// Rows 32..63 have the same swizzle as rows 0..31, so sub-block 1 is +32 rows.
__device__ __forceinline__ void qk_tile(const char* kbuf, const bf16x8 (&qf)[8], const Offsets& off, f32x16 (&s)[2]) {
  s[0] = zero16();
  s[1] = zero16();
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    const bf16x8 a0 = lds_read16(kbuf, off.k[kk]);
    const bf16x8 a1 = lds_read16(kbuf + 32 * 256, off.k[kk]);
    s[0] = mfma32(a0, qf[kk], s[0]);
    s[1] = mfma32(a1, qf[kk], s[1]);
  }
}

// Sets masked scores to -inf: keys after the lane's query (causal, which also
// covers keys past n), and every key of an invalid list entry.
__device__ __forceinline__ void mask_tile(f32x16 (&s)[2], int key0, int qabs, bool valid, int l) {
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = key0 + 32 * mb + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3);
      if (!valid || key > qabs) s[mb][i] = -__builtin_inff();
    }
}

// One (head, query block) unit.
template <int BQ, bool DENSE>
__device__ __forceinline__ void attn_unit(const AttnArgs& a, int h, int qb, char* smem, const Offsets& off, int tid) {
  constexpr int NT = BQ * 2;
  constexpr int TPB = BQ / BK;  // tiles per key block
  const int l = tid & 63, w = tid >> 6;
  const int g = h / a.G;
  const int q0 = qb * BQ;
  const int qabs = q0 + 32 * w + (l & 31);
  const uint16_t* Kg = a.k + (size_t)g * a.n * kHeadDim;
  const uint16_t* Vg = a.v + (size_t)g * a.n * kHeadDim;

  bf16x8 qf[8];
  {
    const uint16_t* qrow = a.q + ((size_t)h * a.n + (qabs < a.n ? qabs : 0)) * kHeadDim;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 16 * kk + 8 * (l >> 5));
      if (qabs >= a.n) raw = u32x4{0, 0, 0, 0};
      qf[kk] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  int beg = 0, cnt;
  const int32_t* cols = nullptr;
  if (DENSE) {
    cnt = qb + 1;
  } else {
    const int32_t* rp = a.row_ptr + (size_t)h * (a.nb + 1);
    const int64_t cap = a.col_cap;
    int64_t b0 = rp[qb], e0 = rp[qb + 1];
    b0 = b0 < 0 ? 0 : (b0 > cap ? cap : b0);
    e0 = e0 < b0 ? b0 : (e0 > cap ? cap : e0);
    beg = (int)b0;
    cnt = (int)(e0 - b0);
    cols = a.col_idx + (size_t)h * cap;
  }
  const int T = cnt * TPB;

  auto tile_key0 = [&](int j, bool& valid, bool& needs_mask) -> int {
    int kb = DENSE ? j / TPB : cols[beg + j / TPB];
    valid = kb >= 0 && kb <= qb;
    if (!valid) kb = 0;
    needs_mask = !valid || kb == qb;
    return kb * BQ + (j % TPB) * BK;
  };

  f32x16 o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db) o[db] = zero16();
  float m_run = -__builtin_inff(), l_run = 0.f;

  if (T > 0) {
    TileRegs<NT> regs;
    bool v0, m0;
    const int k0 = tile_key0(0, v0, m0);
    load_tile<NT>(regs, Kg, Vg, k0, a.n, tid);
    store_tile<NT>(regs, smem, smem + kTileBytes, tid);
    bool vn = false, mn = false;
    int kn = 0;
    if (T > 1) {
      kn = tile_key0(1, vn, mn);
      load_tile<NT>(regs, Kg, Vg, kn, a.n, tid);
    }
    __syncthreads();
    f32x16 s[2];
    qk_tile(smem, qf, off, s);
    if (m0) mask_tile(s, k0, qabs, v0, l);

    for (int j = 0; j < T; ++j) {
      const int cur = j & 1, nxt = cur ^ 1;
      char* kcur = smem + cur * 2 * kTileBytes;
      char* knxt = smem + nxt * 2 * kTileBytes;
      __syncthreads();  // every wave is done with tile j - 1 (held in buffer nxt)
      const bool has_next = j + 1 < T;
      const bool vnext = vn, mnext = mn;
      const int knext = kn;
      if (has_next) store_tile<NT>(regs, knxt, knxt + kTileBytes, tid);
      __syncthreads();
      if (j + 2 < T) {
        kn = tile_key0(j + 2, vn, mn);
        load_tile<NT>(regs, Kg, Vg, kn, a.n, tid);
      }
      f32x16 sn[2];
      if (has_next) {
        qk_tile(knxt, qf, off, sn);
        if (mnext) mask_tile(sn, knext, qabs, vnext, l);
      }

      // online softmax of tile j (row max raised lazily)
      float mx = -__builtin_inff();
#pragma unroll
      for (int i = 0; i < 16; i += 2)
        mx = fmaxf(fmaxf(mx, fmaxf(s[0][i], s[0][i + 1])), fmaxf(s[1][i], s[1][i + 1]));
      mx = half_max(mx);
      const bool grow = mx * a.c > m_run * a.c + kLazyRescale || m_run == -__builtin_inff();
      if (__ballot(grow)) {
        const float m_new = grow ? fmaxf(m_run, mx) : m_run;
        const float alpha = m_run == -__builtin_inff() ? 0.f : fast_exp2((m_run - m_new) * a.c);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
        m_run = m_new;
      }
      const float mc = m_run == -__builtin_inff() ? 0.f : m_run * a.c;
      bf16x8 pb[2][2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          float p[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) p[e] = fast_exp2(__builtin_fmaf(s[mb][8 * hh + e], a.c, -mc));
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const bf16x2 pr = pack_bf16(p[e], p[e + 1]);
            pb[mb][hh][e] = pr[0];
            pb[mb][hh][e + 1] = pr[1];
            l_run = dot2_bf16_sum(pr, l_run);
          }
        }

      // O^T += V^T P^T
      const char* vcur = kcur + kTileBytes;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          const char* vb = vcur + (32 * mb + 16 * ss) * 256;
#pragma unroll
          for (int db = 0; db < 4; ++db) {
            const bf16x8 av = cat(lds_read_tr(vb, off.v[db][0]), lds_read_tr(vb, off.v[db][1]));
            o[db] = mfma32(av, pb[mb][ss], o[db]);
          }
        }
      if (has_next) {
        s[0] = sn[0];
        s[1] = sn[1];
      }
    }
  }

  const float l_tot = half_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qabs < a.n) {
    uint16_t* orow = a.o + ((size_t)h * a.n + qabs) * kHeadDim;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int d = 32 * db + 8 * i4 + 4 * (l >> 5);
        const bf16x2 lo = pack_bf16(o[db][4 * i4 + 0] * inv, o[db][4 * i4 + 1] * inv);
        const bf16x2 hi = pack_bf16(o[db][4 * i4 + 2] * inv, o[db][4 * i4 + 3] * inv);
        bf16x4 r;
        r[0] = lo[0]; r[1] = lo[1]; r[2] = hi[0]; r[3] = hi[1];
        *reinterpret_cast<bf16x4*>(orow + d) = r;
      }
  }
}

template <int BQ, bool DENSE>
__global__ __launch_bounds__(BQ * 2) void attn_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * kTileBytes];
  const int tid = threadIdx.x;
  Offsets off;
  make_offsets(off, tid & 63);
  if (DENSE || a.order == nullptr) {
    int h, qb;
    if (!map_unit(a, blockIdx.x, h, qb)) return;
    attn_unit<BQ, DENSE>(a, h, qb, smem, off, tid);
    return;
  }
  __shared__ int s_unit;
  const int total = a.hq * a.nb;
  for (;;) {
    __syncthreads();  // the previous unit is done with LDS and s_unit
    if (tid == 0) s_unit = atomicAdd(a.counter, 1);
    __syncthreads();
    const int u = s_unit;
    if (u >= total) break;
    const int unit = a.order[u];
    attn_unit<BQ, DENSE>(a, unit / a.nb, unit % a.nb, smem, off, tid);
  }
}

// Longest-first work list for the persistent sparse kernel: a counting sort of
// the units (h, qb) by list length, descending.  One workgroup; also resets the
// work counter.  Order within one length is arbitrary (it only affects which
// workgroup runs a unit, never a result).
__global__ __launch_bounds__(1024) void attn_schedule(AttnArgs a) {
  __shared__ int hist[kCostBuckets];
  const int tid = threadIdx.x;
  const int total = a.hq * a.nb;
  for (int i = tid; i < kCostBuckets; i += 1024) hist[i] = 0;
  __syncthreads();
  auto cost = [&](int u) {
    const int h = u / a.nb, qb = u % a.nb;
    const int32_t* rp = a.row_ptr + (size_t)h * (a.nb + 1);
    int64_t c = (int64_t)rp[qb + 1] - (int64_t)rp[qb];
    c = c < 0 ? 0 : (c >= kCostBuckets ? kCostBuckets - 1 : c);
    return (int)c;
  };
  for (int u = tid; u < total; u += 1024) atomicAdd(&hist[kCostBuckets - 1 - cost(u)], 1);
  __syncthreads();
  // exclusive scan over buckets (descending cost), 8 buckets per thread
  __shared__ int part[1024];
  int loc[kCostBuckets / 1024];
  int s = 0;
#pragma unroll
  for (int i = 0; i < kCostBuckets / 1024; ++i) {
    loc[i] = s;
    s += hist[tid * (kCostBuckets / 1024) + i];
  }
  part[tid] = s;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int x = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  const int base = part[tid] - s;
#pragma unroll
  for (int i = 0; i < kCostBuckets / 1024; ++i) hist[tid * (kCostBuckets / 1024) + i] = base + loc[i];
  __syncthreads();
  for (int u = tid; u < total; u += 1024) {
    const int pos = atomicAdd(&hist[kCostBuckets - 1 - cost(u)], 1);
    const_cast<int32_t*>(a.order)[pos] = u;
  }
  if (tid == 0) *a.counter = 0;
}

template <int BQ, bool DENSE>
hipError_t launch_t(const AttnArgs& a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL((attn_kernel<BQ, DENSE>), dim3(grid), dim3(BQ * 2), 0, stream, a);
  return hipGetLastError();
}

// Workgroups that fit on the device at once (persistent grid size).
template <int BQ>
int persistent_grid() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] > 0) return cached[dev];
  int cus = 0, per = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, attn_kernel<BQ, false>, BQ * 2, 0) != hipSuccess || per <= 0)
    per = 1;
  cached[dev] = cus * per;
  return cached[dev];
}

}  // namespace

size_t attn_schedule_bytes(const Dims& d) { return ((size_t)d.hq * d.nb + 64) * sizeof(int32_t); }

hipError_t launch_attn(const Dims& d, float scale, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                       const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, bool dense,
                       uint16_t* o, void* sched, hipStream_t stream) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  AttnArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.row_ptr = row_ptr; a.col_idx = col_idx; a.col_cap = col_cap;
  a.order = nullptr; a.counter = nullptr;
  a.n = d.n; a.nb = d.nb; a.hq = d.hq; a.hkv = d.hkv; a.G = d.G;
  a.c = scale * kLog2e;
  int grid;
  if (d.hkv % kNumXcd == 0) {
    a.map_mode = 1; a.rep = 1;
    grid = d.hq * d.nb;
  } else if (kNumXcd % d.hkv == 0) {
    a.map_mode = 2; a.rep = kNumXcd / d.hkv;
    grid = kNumXcd * d.G * ((d.nb + a.rep - 1) / a.rep);
  } else {
    a.map_mode = 0; a.rep = 1;
    grid = d.hq * d.nb;
  }
  if (!dense && sched != nullptr) {
    a.counter = reinterpret_cast<int*>(sched);
    a.order = reinterpret_cast<const int32_t*>(sched) + 64;
    hipLaunchKernelGGL(attn_schedule, dim3(1), dim3(1024), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int pg = d.B == 128 ? persistent_grid<128>() : persistent_grid<64>();
    grid = pg < d.hq * d.nb ? pg : d.hq * d.nb;
  }
  if (d.B == 128) return dense ? launch_t<128, true>(a, grid, stream) : launch_t<128, false>(a, grid, stream);
  return dense ? launch_t<64, true>(a, grid, stream) : launch_t<64, false>(a, grid, stream);
}

}  // namespace crisp
