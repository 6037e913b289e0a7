// Block-sparse causal flash attention (Eq. 1 of the paper, restricted to the
// selected key blocks) and the dense causal baseline, for gfx950.
//
// One workgroup computes one (query head, query block) unit: BQ = B query rows,
// BQ / 32 waves, each wave owning 32 query rows.  Key blocks are streamed in
// tiles of 64 keys through double-buffered, swizzled LDS.  Per tile and wave:
//   S^T (64 keys x 32 queries) = K_tile Q^T      16 x v_mfma_f32_32x32x16_bf16
//   online softmax in fp32 (exp2 with log2(e) folded into the scale)
//   O^T (128 d x 32 queries) += V^T P^T          16 x v_mfma_f32_32x32x16_bf16
// The score tile is transposed so that a lane owns one query: row maxima and
// sums are lane-local plus one exchange with lane l ^ 32.  The C-layout of S^T
// is reused directly as the B operand of the PV product; V^T operands come
// from LDS through ds_read_b64_tr_b16, which transposes 4 keys x 16 dims per
// 16-lane group, so V never needs a transposed copy.
// The score MFMAs of tile j+1 are issued before the softmax of tile j, so the
// matrix cores and the vector ALU can overlap within a wave.
#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

constexpr int BK = 64;                  // keys per tile
constexpr int kTileBytes = BK * 256;    // one K or V tile: 64 rows x 128 bf16

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  const int32_t* row_ptr;
  const int32_t* col_idx;
  int64_t col_cap;
  int n, nb, hq, hkv, G;
  float c;        // softmax scale * log2(e)
  int map_mode;   // 0 natural order, 1 H_kv % 8 == 0, 2 8 % H_kv == 0
  int rep;        // map_mode 2: XCDs per KV group
};

// Workgroup -> (head, query block).  Units of one KV group are kept on one XCD
// (its L2 then serves the group's K/V to all G heads), and longer rows (higher
// qb) are dispatched first.
__device__ __forceinline__ bool map_unit(const AttnArgs& a, int bid, int& h, int& qb) {
  if (a.map_mode == 0) {
    if (bid >= a.hq * a.nb) return false;
    qb = a.nb - 1 - bid / a.hq;
    h = bid % a.hq;
    return true;
  }
  const int x = bid % kNumXcd, u = bid / kNumXcd;
  if (a.map_mode == 1) {
    const int gpx = a.hkv / kNumXcd;  // groups per XCD: x, x + 8, ...
    const int per = gpx * a.G;
    const int r = u / per;
    if (r >= a.nb) return false;
    const int w = u % per;
    qb = a.nb - 1 - r;
    h = (x + kNumXcd * (w / a.G)) * a.G + (w % a.G);
    return true;
  }
  const int g = x % a.hkv, par = x / a.hkv;  // XCD x: group g, rows qb = par (mod rep)
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

// S^T for one tile: s[mb] covers keys 32 * mb + (C-layout rows), queries = lane column.
__device__ __forceinline__ void qk_tile(const char* kbuf, const bf16x8 (&qf)[8], int l, f32x16 (&s)[2]) {
  s[0] = zero16();
  s[1] = zero16();
#pragma unroll
  for (int kk = 0; kk < 8; ++kk) {
    const int d = 16 * kk + 8 * (l >> 5);
    const bf16x8 a0 = lds_read16(kbuf, lds_off(l & 31, d));
    const bf16x8 a1 = lds_read16(kbuf, lds_off(32 + (l & 31), d));
    s[0] = mfma32(a0, qf[kk], s[0]);
    s[1] = mfma32(a1, qf[kk], s[1]);
  }
}

// Sets masked scores to -inf: keys after the lane's query (causal), keys past n,
// and every key of an invalid list entry.
__device__ __forceinline__ void mask_tile(f32x16 (&s)[2], int key0, int qabs, bool valid, int l) {
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = key0 + 32 * mb + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3);
      if (!valid || key > qabs) s[mb][i] = -__builtin_inff();
    }
}

template <int BQ, bool DENSE>
__global__ __launch_bounds__(BQ * 2) void attn_kernel(AttnArgs a) {
  constexpr int NT = BQ * 2;
  constexpr int TPB = BQ / BK;  // tiles per key block
  __shared__ __attribute__((aligned(16))) char smem[2 * 2 * kTileBytes];

  int h, qb;
  if (!map_unit(a, blockIdx.x, h, qb)) return;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
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

  // tile j -> key0 and validity
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
    int k0 = tile_key0(0, v0, m0);
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
    qk_tile(smem, qf, l, s);
    if (m0) mask_tile(s, k0, qabs, v0, l);

    for (int j = 0; j < T; ++j) {
      const int cur = j & 1, nxt = cur ^ 1;
      char* kcur = smem + cur * 2 * kTileBytes;
      char* knxt = smem + nxt * 2 * kTileBytes;
      __syncthreads();  // everyone is done with tile j - 1 (held in buffer nxt)
      const bool has_next = j + 1 < T;
      bool vnext = vn, mnext = mn;
      const int knext = kn;
      if (has_next) store_tile<NT>(regs, knxt, knxt + kTileBytes, tid);
      __syncthreads();
      if (j + 2 < T) {
        kn = tile_key0(j + 2, vn, mn);
        load_tile<NT>(regs, Kg, Vg, kn, a.n, tid);
      }
      f32x16 sn[2];
      if (has_next) {
        qk_tile(knxt, qf, l, sn);
        if (mnext) mask_tile(sn, knext, qabs, vnext, l);
      }

      // online softmax of tile j
      float mx = -__builtin_inff();
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, fmaxf(s[0][i], s[1][i]));
      mx = fmaxf(mx, swap_halves(mx));
      const float m_new = fmaxf(m_run, mx);
      const float m_use = m_new == -__builtin_inff() ? 0.f : m_new;
      const float alpha = fast_exp2((m_run - m_use) * a.c);
      const float mc = m_use * a.c;
      float psum = 0.f;
      bf16x8 pb[2][2];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = fast_exp2(__builtin_fmaf(s[mb][i], a.c, -mc));
          psum += p;
          pb[mb][i >> 3][i & 7] = (__bf16)p;
        }
      l_run = l_run * alpha + psum;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= alpha;

      // O^T += V^T P^T
      const char* vcur = kcur + kTileBytes;
      const int grp = l >> 4, jj = l & 15;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          const int row = 32 * mb + 16 * ss + 4 * (grp >> 1) + (jj >> 2);
#pragma unroll
          for (int db = 0; db < 4; ++db) {
            const int col = 32 * db + 16 * (grp & 1) + 4 * (jj & 3);
            const bf16x8 av = cat(lds_read_tr(vcur, lds_off(row, col)), lds_read_tr(vcur, lds_off(row + 8, col)));
            o[db] = mfma32(av, pb[mb][ss], o[db]);
          }
        }
      if (has_next) {
        s[0] = sn[0];
        s[1] = sn[1];
      }
    }
  }

  const float l_tot = l_run + swap_halves(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  if (qabs < a.n) {
    uint16_t* orow = a.o + ((size_t)h * a.n + qabs) * kHeadDim;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int d = 32 * db + 8 * i4 + 4 * (l >> 5);
        bf16x4 r;
        r[0] = (__bf16)(o[db][4 * i4 + 0] * inv);
        r[1] = (__bf16)(o[db][4 * i4 + 1] * inv);
        r[2] = (__bf16)(o[db][4 * i4 + 2] * inv);
        r[3] = (__bf16)(o[db][4 * i4 + 3] * inv);
        *reinterpret_cast<bf16x4*>(orow + d) = r;
      }
  }
}

template <int BQ, bool DENSE>
hipError_t launch_t(const AttnArgs& a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL((attn_kernel<BQ, DENSE>), dim3(grid), dim3(BQ * 2), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const Dims& d, float scale, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                       const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, bool dense,
                       uint16_t* o, hipStream_t stream) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  AttnArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.row_ptr = row_ptr; a.col_idx = col_idx; a.col_cap = col_cap;
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
  if (d.B == 128) return dense ? launch_t<128, true>(a, grid, stream) : launch_t<128, false>(a, grid, stream);
  return dense ? launch_t<64, true>(a, grid, stream) : launch_t<64, false>(a, grid, stream);
}

}  // namespace crisp
