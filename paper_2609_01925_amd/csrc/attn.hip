// Block-sparse causal flash attention (Eq. 1 of the paper, restricted to the
// selected key blocks) and the dense causal baseline, for gfx950.
//
// A workgroup computes one (query head, query block) unit at a time: BQ = B
// query rows, BQ / 32 waves, each wave owning 32 query rows.  Keys are
// streamed in tiles of 64 (32 for 64-row blocks, below).  Per 64-key tile and wave:
//   S^T (64 keys x 32 queries) = K_tile Q^T      16 x v_mfma_f32_32x32x16_bf16
//   online softmax in fp32 (exp2, log2(e) folded into the scale)
//   O^T (128 d x 32 queries) += V^T P^T          16 x v_mfma_f32_32x32x16_bf16
// The score tile is transposed so that a lane owns one query: row sums and
// maxima are lane-local plus one v_permlane32_swap with lane l ^ 32.  The C
// layout of S^T is reused directly as the B operand of the PV product; V^T
// operands come from LDS through ds_read_b64_tr_b16, which transposes 4 keys x
// 16 dims per 16-lane group, so V needs no transposed copy.
//
// K and V tiles move from global memory straight into LDS with LDS-DMA loads
// (buffer_load ... lds), two 2-deep rings (K, V) of 16 KB stages: 64 KB per
// workgroup, so two workgroups share a CU and every SIMD interleaves two waves.
// A 64-row block has a two-wave workgroup, so four must share a CU: its tiles
// have 32 keys (32 KB of rings).
// Step j of a unit overlaps three things: tile j's probabilities are formed
// (against the running max) beside the PV product of tile j-1, then the scores
// of tile j+1 are computed beside the row sums.  Each ring stage is refilled
// one step before it is read, and the loop is expanded two steps at a time so
// that every stage address is a compile-time immediate.  The running max is
// only raised when some lane's tile sum of P exceeds 2^8 (no P of a lane exceeds
// its sum): until then P may exceed 1 by at most 2^8, which fp32 and bf16 hold
// as exactly as values below 1, and the O accumulators are left untouched.
//
// Sparse lists are processed longest first from work lists that attn_schedule
// builds from the list lengths, so long PE rows start first and short VS rows
// fill the tail.  Below 512k tokens a persistent grid pulls units from one list
// per KV group, and the K/V tiles of a group stay in the caches of the XCDs that
// serve it; rows much longer than the layer's work per workgroup are split into
// chunks whose partial results attn_combine merges.  From 512k tokens on, rows
// are long enough that the workgroups of a persistent grid drift apart along the
// key axis (the two workgroups sharing a CU do not advance at the same rate, and
// each keeps its place for the whole layer), so concurrent readers of a K/V tile
// no longer meet in L2: there the grid has one workgroup per unit, and every
// workgroup takes the next unit of the group lists in order (one KV group after
// the other, longest first within a group), so units that start together
// advance together over the same group's K/V.  Up to 8192 tokens (K/V of the whole
// layer within the caches) the units come from one longest-first list of all units
// without atomics; when there are at least as many units as a persistent grid has
// workgroups, the grid has one workgroup per unit, workgroup i taking item i: the
// dispatcher starts the workgroups in order, so the longest units start first and later
// ones fill the CUs as they free up, with no loop, queue or split rows around each unit
// (2k-4k layers of 32 heads 11-12% faster than the persistent grid with split rows, 8k
// 3-10% faster, 16k 14% slower).  With fewer units (few heads) the persistent grid takes
// items i, i + grid, ... of that list and splits long rows.
#include <atomic>
#include <type_traits>

#include "crisp_device.h"
#include "crisp_internal.h"

namespace crisp {

namespace {

// Key tiles: 64 keys for 128-row query blocks.  64-row blocks have two-wave
// workgroups, which need four to a CU for two waves per SIMD, so their tiles
// have 32 keys (32 KB of rings per workgroup instead of 64 KB).
template <int BQ>
struct Tile {
  static constexpr int kBK = BQ == 128 ? 64 : 32;  // keys per tile
  static constexpr int kNMB = kBK / 32;            // 32-key sub-blocks per tile
  static constexpr int kBytes = kBK * 256;         // one K or V tile: kBK rows x 128 bf16
  static constexpr int kRing = 2 * kBytes;         // one ring (K or V): 2 stages
};
constexpr float kSumLimit = 256.0f;          // a lane's tile sum of P above this forces a rescale
constexpr int kCostBuckets = 8192;
constexpr int kOneShotMinLen = 1 << 19;  // from this length on, sparse lists run one unit per workgroup
constexpr int kStaticListMaxLen = 8192;  // up to this length too, from one list by workgroup index (no atomics)
constexpr int kMinChunk = 8;             // shortest chunk of a split row, in list entries
constexpr int kItemUnitBits = 21;        // work item = unit | chunk << 21

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
  int one_shot;          // 1: one unit per workgroup, all units in one queue
  int static_list;       // 1: all units in queue 0, workgroup i takes items i, i + grid, ...
  int* slot_base;        // split rows: first partial slot of the row's chunks, else -1
  int* split_rows;       // the split rows (any order)
  float* parts;          // partial results per slot: O[BQ][128], m[BQ], l[BQ] (fp32)
  int split_slots;       // partial slots available (0: rows are never split)
  int grid;              // workgroups of the persistent grid
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

// Queue slot of head h's KV group, and the slot the workgroups on XCD x pop from
// first (XCDs beyond the groups' share start at an empty slot and go straight to
// taking work from the others; with one unit per workgroup every workgroup
// starts at slot 0, so the slots are emptied in order).
__device__ __forceinline__ int unit_queue(const AttnArgs& a, int h) {
  const int g = h / a.G;
  if (a.hkv >= kNumXcd) return g % kNumXcd;
  return g * (kNumXcd / a.hkv);
}

__device__ __forceinline__ int home_queue(const AttnArgs& a, int x) {
  if (a.one_shot) return 0;
  if (a.hkv >= kNumXcd) return x;
  const int r = kNumXcd / a.hkv;  // XCDs per group
  return x < a.hkv * r ? (x / r) * r : x;
}

// Entries of row (head, qb) of a sparse list, with row_ptr clamped to [0, col_cap]
// exactly as the attention reads it.
__device__ __forceinline__ int row_len(const AttnArgs& a, int head, int qb) {
  const int32_t* rp = a.row_ptr + (size_t)head * (a.nb + 1);
  int64_t b0 = rp[qb], e0 = rp[qb + 1];
  b0 = b0 < 0 ? 0 : (b0 > a.col_cap ? a.col_cap : b0);
  e0 = e0 < b0 ? b0 : (e0 > a.col_cap ? a.col_cap : e0);
  return (int)(e0 - b0);
}

// Workgroup geometry for query blocks of BQ rows: QH halves of 32 queries per
// wave, BQ / (32 QH) waves.  One half per wave (two waves per SIMD, at most 256
// registers each) is what runs: two halves would halve the LDS operand reads per
// MFMA, but need one wave per SIMD, which then has no other wave to hide its
// latencies behind and runs slower.
template <int BQ>
struct Geo {
  static constexpr int kQH = 1;
  static constexpr int kWaves = BQ / (32 * kQH);
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kWavesPerEU = kQH == 2 ? 1 : 2;
};

#if defined(__HIP_DEVICE_COMPILE__)

// Per-lane LDS byte offsets of the MFMA operand reads, fixed for the whole kernel.
// K (A operand of S^T): row l % 32 (+32 rows for the second key sub-block, an
// immediate), chunk 2 kk + l / 32.  V^T (A operand of O^T, transposing reads):
// two reads per MFMA, rows r0 and r0 + 8 (+16 ss + 32 mb rows, immediates),
// dims 32 db + 16 (grp & 1) + 4 (jj & 3).
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

// LDS reads at integer LDS addresses (no generic-pointer conversion).
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
__device__ __forceinline__ bf16x8 lds_ld16(int addr) { return *(const lds_bf16x8*)(uint32_t)addr; }
__device__ __forceinline__ bf16x4 lds_ld_tr(int addr) {
  return __builtin_bit_cast(bf16x4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(uint32_t)addr));
}


// Debug build: the tile pipeline serialised -- every tile load waited for and a
// barrier after each LDS phase -- so that its results, compared bit for bit with the
// pipelined kernel's, show that the rings' overlap of loads and reads never races.
// The arithmetic and its order are unchanged.
#ifdef CRISP_DEBUG
__device__ __forceinline__ void race_sync() {
  wait_dma();
  __syncthreads();
}
#else
__device__ __forceinline__ void race_sync() {}
#endif

// S^T for one tile: s[h][mb] holds keys 32 mb + (C-layout row) against the 32
// queries of half h (lane column).  Rows 32..63 have the same swizzle as rows
// 0..31, so sub-block mb is +32 mb rows, and each K operand read serves every
// half.  The sub-blocks' accumulation chains are interleaved step by step (each
// chain still sums in kk order), so consecutive MFMAs are independent.
// The K operands of the first d-step (kk = 0) are read ahead by the caller
// (k_first) and passed in as k0.
template <int NMB>
__device__ __forceinline__ void k_first(int kbuf, const Offsets& off, bf16x8 (&k0)[NMB]) {
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) k0[mb] = lds_ld16(kbuf + 32 * 256 * mb + off.k[0]);
}

template <int QH, int NMB>
__device__ __forceinline__ void qk_tile(int kbuf, const bf16x8 (&qf)[QH][8], const Offsets& off, f32x16 (&s)[QH][NMB],
                                        const bf16x8 (&k0)[NMB]) {
#pragma unroll
  for (int h = 0; h < QH; ++h)
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) s[h][mb] = zero16();
#pragma unroll
  for (int kk = 0; kk < 8; ++kk)
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      const bf16x8 ak = kk == 0 ? k0[mb] : lds_ld16(kbuf + 32 * 256 * mb + off.k[kk]);
#pragma unroll
      for (int h = 0; h < QH; ++h) s[h][mb] = mfma32(ak, qf[h][kk], s[h][mb]);
    }
}

// Sets masked scores to -inf: keys after the lane's query (causal, which also
// covers keys past n), and every key of an invalid list entry.
template <int NMB>
__device__ __forceinline__ void mask_tile(f32x16 (&s)[NMB], int key0, int qabs, bool valid, int l) {
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = key0 + 32 * mb + 8 * (i >> 2) + 4 * (l >> 5) + (i & 3);
      if (!valid || key > qabs) s[mb][i] = -__builtin_inff();
    }
}

// Maximum of the lane's 16 scores of one sub-block.
__device__ __forceinline__ float max16(const f32x16& s) {
  float m = vmax(s[0], s[1]);
#pragma unroll
  for (int i = 2; i < 16; i += 2) m = vmax(vmax(m, s[i]), s[i + 1]);
  return m;
}

// P = exp2(s c - mc) for one sub-block as bf16 B operands of the PV product:
// pb[hh] covers the keys of registers 8 hh .. 8 hh + 7.
__device__ __forceinline__ void exp_sub(const f32x16& s, float c, float mc, bf16x8 (&pb)[2]) {
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const bf16x2 pr = pack_bf16(fast_exp2(__builtin_fmaf(s[8 * hh + e], c, -mc)),
                                  fast_exp2(__builtin_fmaf(s[8 * hh + e + 1], c, -mc)));
      pb[hh][e] = pr[0];
      pb[hh][e + 1] = pr[1];
    }
}

// The lane's sum of the tile's (bf16) probabilities, in two partial sums (the
// halves hh of each sub-block) so that the dot2 chain is half as long.
template <int NMB>
__device__ __forceinline__ float sum_tile(const bf16x8 (&pb)[NMB][2]) {
  float part[2] = {0.f, 0.f};
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        bf16x2 pr;
        pr[0] = pb[mb][hh][e];
        pr[1] = pb[mb][hh][e + 1];
        part[hh] = dot2_bf16_sum(pr, part[hh]);
      }
  return part[0] + part[1];
}

// O^T[h] (128 d x 32 queries) += V^T P^T[h] for one tile; each V^T operand (two
// transposing reads) serves every half.
template <int QH, int NMB>
__device__ __forceinline__ void pv_tile(int vbuf, const Offsets& off, const bf16x8 (&pb)[QH][NMB][2], f32x16 (&o)[QH][4]) {
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int ss = 0; ss < 2; ++ss) {
      const int vb = vbuf + (32 * mb + 16 * ss) * 256;
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const bf16x8 av = cat(lds_ld_tr(vb + off.v[db][0]), lds_ld_tr(vb + off.v[db][1]));
#pragma unroll
        for (int h = 0; h < QH; ++h) o[h][db] = mfma32(av, pb[h][mb][ss], o[h][db]);
      }
    }
}

// One (head, query block) unit, or one chunk of a split row's list: entries
// [chunk * csize, chunk * csize + csize) when part is given, whose unnormalised
// O, row max and row sum then go to the partial slot part instead of o.
template <int BQ, bool DENSE>
__device__ __forceinline__ void attn_unit(const AttnArgs& a, int head, int qb, int lds0, const Offsets& off,
                                          const Fetch<Geo<BQ>::kWaves>& fe, int tid, int chunk = 0, int csize = 0,
                                          float* part = nullptr) {
  constexpr int QH = Geo<BQ>::kQH;
  constexpr int NW = Geo<BQ>::kWaves;
  constexpr int BK = Tile<BQ>::kBK, NMB = Tile<BQ>::kNMB;
  constexpr int TPB = BQ / BK;  // tiles per key block
  const int l = tid & 63, w = tid >> 6;
  const int g = head / a.G;
  const int q0 = qb * BQ;
  int qabs[QH];
#pragma unroll
  for (int h = 0; h < QH; ++h) qabs[h] = q0 + 32 * (QH * w + h) + (l & 31);
  const i32x4 rk = tensor_rsrc(a.k + (size_t)g * a.n * kHeadDim, a.n);
  const i32x4 rv = tensor_rsrc(a.v + (size_t)g * a.n * kHeadDim, a.n);

  int beg = 0, cnt;
  const int32_t* cols = nullptr;
  if (DENSE) {
    cnt = qb + 1;
  } else {
    const int32_t* rp = a.row_ptr + (size_t)head * (a.nb + 1);
    const int64_t cap = a.col_cap;
    int64_t b0 = rp[qb], e0 = rp[qb + 1];
    b0 = b0 < 0 ? 0 : (b0 > cap ? cap : b0);
    e0 = e0 < b0 ? b0 : (e0 > cap ? cap : e0);
    beg = (int)b0;
    cnt = (int)(e0 - b0);
    cols = a.col_idx + (size_t)head * cap;
    if (part != nullptr) {
      const int lo = chunk * csize;
      beg += lo;
      cnt = cnt - lo < csize ? cnt - lo : csize;
    }
  }
  const int T = cnt * TPB;

  // Sparse lists: the unit's column indices are held 64 to a VGPR (one per lane;
  // chunk c of the list in colv0 or colv1 by its parity), the chunk of the current tile and the
  // next one, so a lookup is a v_readlane and never waits on memory.  A chunk is
  // fetched at the end of a step, a whole chunk ahead of its first use, and lands
  // under the wait at the top of the next step.  Lanes past the list end load its
  // last entry; they are never looked up.
  int colv0 = 0, colv1 = 0;
  int chunk0 = 0;  // chunk of the current tile
  auto load_chunk = [&](int c) -> int {
    const int i = 64 * c + l;
    return cols[beg + (i < cnt ? i : cnt - 1)];
  };
  auto col_of = [&](int bi) -> int {
    return __builtin_amdgcn_readlane((bi >> 6) & 1 ? colv1 : colv0, bi & 63);
  };
  if (!DENSE && cnt > 0) {
    colv0 = load_chunk(0);
    colv1 = load_chunk(1);
  }

  // tile j -> first key, validity (entry in [0, qb]) and whether it needs the mask
  auto tile_key0 = [&](int j, bool& valid, bool& needs_mask) -> int {
    int kb = DENSE ? j / TPB : col_of(j / TPB);
    valid = kb >= 0 && kb <= qb;
    if (!valid) kb = 0;
    needs_mask = !valid || kb == qb;
    return kb * BQ + (j % TPB) * BK;
  };
  auto key0_of = [&](int j) {
    bool vv, mm;
    return tile_key0(j, vv, mm);
  };
  // ring stages by parity: K at lds0 + {0, 1} tiles, V after the K ring
  auto kst = [&](int parity) { return lds0 + parity * Tile<BQ>::kBytes; };
  auto vst = [&](int parity) { return lds0 + Tile<BQ>::kRing + parity * Tile<BQ>::kBytes; };

  bf16x8 qf[QH][8];
#pragma unroll
  for (int h = 0; h < QH; ++h) {
    const uint16_t* qrow = a.q + ((size_t)head * a.n + (qabs[h] < a.n ? qabs[h] : 0)) * kHeadDim;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      u32x4 raw = *reinterpret_cast<const u32x4*>(qrow + 16 * kk + 8 * (l >> 5));
      if (qabs[h] >= a.n) raw = u32x4{0, 0, 0, 0};
      qf[h][kk] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  f32x16 o[QH][4];
  float m_run[QH], l_run[QH];
#pragma unroll
  for (int h = 0; h < QH; ++h) {
#pragma unroll
    for (int db = 0; db < 4; ++db) o[h][db] = zero16();
    m_run[h] = -__builtin_inff();
    l_run[h] = 0.f;
  }

  f32x16 s[QH][NMB];
  if (T > 0) {
    // Step j (parity P): tile j's scores S(j) are in registers and P(j-1) is
    // formed.  At the top, K(j+1) and V(j-1), issued in step j-1 (or the
    // prologue), have landed for every wave, and every wave is done with the
    // stages of K(j) (scored in step j-1) and V(j-2), which are refilled with
    // K(j+2) and V(j).  Tile j's probabilities are formed against the running max
    // beside the PV product of tile j-1.  They stand while each lane's sum of them
    // stays at most 2^8 (so does every one of them); otherwise the (rare) branch
    // raises the running max to the tile's row max, rescales O and l, and forms
    // them again.  Last, the scores of tile j+1 replace S(j).
    auto step = [&](int j, auto par, auto first, const bf16x8 (&pp)[QH][NMB][2], bf16x8 (&pn)[QH][NMB][2]) {
      constexpr int P = decltype(par)::value;
      wait_dma();
      __syncthreads();

      if (j + 2 < T) fetch_tile<NW, BK>(fe, rk, kst(P), key0_of(j + 2), w);
      fetch_tile<NW, BK>(fe, rv, vst(P), key0_of(j), w);
      race_sync();
      // K(j+1) landed before the barrier: the first d-step's operands of its scores
      // are read now, so that their latency passes under the softmax half.
      bf16x8 k0[NMB];
      k_first<NMB>(kst(1 - P), off, k0);
      // The two waves of a SIMD come from different workgroups and drift apart:
      // while one scores a tile (MFMAs only), the other forms probabilities (VALU)
      // beside its PV MFMAs.  The softmax half runs at raised wave priority, so the
      // arbiter issues its VALU work first and the scoring wave's MFMAs fill the
      // gaps (3.7% faster at 128k than equal priority; raising the scoring half
      // instead is slower).
      __builtin_amdgcn_s_setprio(1);
      {
        bool vj, mj;
        const int kj = tile_key0(j, vj, mj);
        if (mj) {
#pragma unroll
          for (int h = 0; h < QH; ++h) mask_tile(s[h], kj, qabs[h], vj, l);
        }
      }
      float ts[QH];
      bool grow = false;
#pragma unroll
      for (int h = 0; h < QH; ++h) {
        const float mc = m_run[h] == -__builtin_inff() ? 0.f : m_run[h] * a.c;
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) exp_sub(s[h][mb], a.c, mc, pn[h][mb]);
        ts[h] = sum_tile<NMB>(pn[h]);
        grow = grow || !(ts[h] <= kSumLimit) || m_run[h] == -__builtin_inff();
      }
      if (!decltype(first)::value) pv_tile<QH, NMB>(vst(1 - P), off, pp, o);
      race_sync();
      // Keeps the probabilities formed here, beside the PV product, rather than
      // letting the compiler sink them into the no-rescale path.
#pragma unroll
      for (int h = 0; h < QH; ++h) {
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) asm volatile("" ::"v"(pn[h][mb][0]), "v"(pn[h][mb][1]));
        asm volatile("" ::"v"(ts[h]));
      }
      if (__ballot(grow)) {
#pragma unroll
        for (int h = 0; h < QH; ++h) {
          float mt = max16(s[h][0]);
#pragma unroll
          for (int mb = 1; mb < NMB; ++mb) mt = vmax(mt, max16(s[h][mb]));
          const float mx = half_max(mt);
          const float m_new = vmax(m_run[h], mx);
          const float alpha = m_run[h] == -__builtin_inff() ? 0.f : fast_exp2((m_run[h] - m_new) * a.c);
          l_run[h] *= alpha;
#pragma unroll
          for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[h][db][i] *= alpha;
          m_run[h] = m_new;
          const float mcn = m_new == -__builtin_inff() ? 0.f : m_new * a.c;
#pragma unroll
          for (int mb = 0; mb < NMB; ++mb) exp_sub(s[h][mb], a.c, mcn, pn[h][mb]);
          ts[h] = sum_tile<NMB>(pn[h]);
        }
      }
#pragma unroll
      for (int h = 0; h < QH; ++h) l_run[h] += ts[h];
      // After the last tile the stage of K(j+1) holds stale data that no DMA
      // targets; those scores are never used.  The scheduler interleaves the
      // K operand reads with the MFMAs in its LDS/MFMA pipelining mode.
      __builtin_amdgcn_s_setprio(0);
      // A use here keeps the early reads at the top of the step (1.5-2% faster on
      // the sparse 128k layer than reading them with the other K operands).
#pragma unroll
      for (int mb = 0; mb < NMB; ++mb) asm volatile("" ::"v"(k0[mb]));
      __builtin_amdgcn_iglp_opt(0);
      qk_tile<QH, NMB>(kst(1 - P), qf, off, s, k0);
      race_sync();
      if (!DENSE && (((j + 1) / TPB) >> 6) != chunk0) {  // tile j+1 starts the next chunk
        ++chunk0;
        if ((chunk0 + 1) & 1)
          colv1 = load_chunk(chunk0 + 1);
        else
          colv0 = load_chunk(chunk0 + 1);
      }
    };
    using Even = std::integral_constant<int, 0>;
    using Odd = std::integral_constant<int, 1>;

    // prologue: K(0), K(1), then the scores of tile 0
    fetch_tile<NW, BK>(fe, rk, kst(0), key0_of(0), w);
    if (T > 1) fetch_tile<NW, BK>(fe, rk, kst(1), key0_of(1), w);
    wait_dma();
    __syncthreads();
    {
      bf16x8 k0[NMB];
      k_first<NMB>(kst(0), off, k0);
      qk_tile<QH, NMB>(kst(0), qf, off, s, k0);
    }
    // two P buffers with fixed registers: steps alternate between them, and the
    // parity of every step is known where it is expanded
    bf16x8 pa[QH][NMB][2], pz[QH][NMB][2];
    step(0, Even{}, std::true_type{}, pz, pa);
    int j = 1;
    for (; j + 1 < T; j += 2) {
      step(j, Odd{}, std::false_type{}, pa, pz);
      step(j + 1, Even{}, std::false_type{}, pz, pa);
    }
    // PV of the last tile: its V stage was filled in the last step
    if (j < T) {
      step(j, Odd{}, std::false_type{}, pa, pz);
      wait_dma();
      __syncthreads();
      pv_tile<QH, NMB>(vst(1), off, pz, o);
    } else {
      wait_dma();
      __syncthreads();
      pv_tile<QH, NMB>(vst(0), off, pa, o);
    }
  }

  if (!DENSE && part != nullptr) {
    // partial result of one chunk: O unnormalised, the row max (of raw scores) and sum
#pragma unroll
    for (int h = 0; h < QH; ++h) {
      const float l_tot = half_sum(l_run[h]);
      const int r = qabs[h] - q0;
      float* po = part + (size_t)r * kHeadDim;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int d = 32 * db + 8 * i4 + 4 * (l >> 5);
          *reinterpret_cast<float4*>(po + d) =
              make_float4(o[h][db][4 * i4], o[h][db][4 * i4 + 1], o[h][db][4 * i4 + 2], o[h][db][4 * i4 + 3]);
        }
      if ((l >> 5) == 0) {
        part[BQ * kHeadDim + r] = m_run[h];
        part[BQ * kHeadDim + BQ + r] = l_tot;
      }
    }
    return;
  }
#pragma unroll
  for (int h = 0; h < QH; ++h) {
    const float l_tot = half_sum(l_run[h]);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    if (qabs[h] < a.n) {
      uint16_t* orow = a.o + ((size_t)head * a.n + qabs[h]) * kHeadDim;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i4 = 0; i4 < 4; ++i4) {
          const int d = 32 * db + 8 * i4 + 4 * (l >> 5);
          const bf16x2 lo = pack_bf16(o[h][db][4 * i4 + 0] * inv, o[h][db][4 * i4 + 1] * inv);
          const bf16x2 hi = pack_bf16(o[h][db][4 * i4 + 2] * inv, o[h][db][4 * i4 + 3] * inv);
          bf16x4 r;
          r[0] = lo[0]; r[1] = lo[1]; r[2] = hi[0]; r[3] = hi[1];
          *reinterpret_cast<bf16x4*>(orow + d) = r;
        }
    }
  }
}

#endif  // __HIP_DEVICE_COMPILE__

template <int BQ, bool DENSE>
__global__ __launch_bounds__(Geo<BQ>::kThreads, Geo<BQ>::kWavesPerEU) void attn_kernel(AttnArgs a) {
#if defined(__HIP_DEVICE_COMPILE__)
  // The rings are the kernel's only LDS object, so they start at LDS address 0
  // (LDS-DMA destinations are then 1 KB aligned); the work-queue slot sits after them.
  __shared__ __attribute__((aligned(1024))) char smem[2 * Tile<BQ>::kRing + 16];
  const int lds0 = __builtin_amdgcn_readfirstlane((int)(size_t)smem);  // LDS address of the rings
  constexpr int NW = Geo<BQ>::kWaves;
  const int tid = threadIdx.x;
  Offsets off;
  make_offsets(off, tid & 63);
  Fetch<NW> fe;
  make_fetch<NW>(fe, tid >> 6, tid & 63);
  if (DENSE || a.order == nullptr) {
    int h, qb;
    if (!map_unit(a, blockIdx.x, h, qb)) return;
    attn_unit<BQ, DENSE>(a, h, qb, lds0, off, fe, tid);
    return;
  }
  // Pop from this XCD's queue (workgroup i runs on XCD i % 8); when it is empty,
  // take work from the other queues in turn.  Every queue ends, so every
  // workgroup exits once all units are taken.
  int* s_unit = reinterpret_cast<int*>(smem + 2 * Tile<BQ>::kRing);
  const int x0 = home_queue(a, blockIdx.x % kNumXcd);
  const int* start = a.counter + 8;
  const int csize = a.counter[17];  // chunk length of split rows
  constexpr size_t kSlotFloats = (size_t)BQ * (kHeadDim + 2);
  // Queues this workgroup has seen run dry (thread 0): they are never tried again.
  // A queue whose counter already reads past its end is skipped without an atomic
  // (a stale read only costs an extra atomic: counters never decrease).
  unsigned dry = 0u;
  int spos = blockIdx.x;  // static list: the next item of this workgroup
  for (;;) {
    __syncthreads();  // the previous unit is done with LDS and the unit slot
    if (a.static_list) {
      // Short layers: items i, i + grid, ... of one longest-first list, no atomic (with one
      // unit per workgroup, item i alone; the workgroups start in index order).  On a
      // persistent grid the pop's atomic and the wait for it cost about as much as a unit's
      // tiles, and a fixed stride balances as well (each round of grid items is no longer
      // than the previous one).  Every wave computes the same item.
      const int item = spos < start[1] - start[0] ? a.order[start[0] + spos] : -1;
      spos += gridDim.x;
      if (tid == 0) *s_unit = item;
    } else if (tid == 0) {
      int unit = -1;
      for (int t = 0; t < kNumXcd && unit < 0; ++t) {
        const int x = (x0 + t) % kNumXcd;
        if (dry & (1u << x)) continue;
        const int len = start[x + 1] - start[x];
        if (len <= 0 || __hip_atomic_load(a.counter + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= len) {
          dry |= 1u << x;
          continue;
        }
        const int pos = atomicAdd(a.counter + x, 1);
        if (pos < len)
          unit = a.order[start[x] + pos];
        else
          dry |= 1u << x;
      }
      *s_unit = unit;
    }
    __syncthreads();
    const int item = *s_unit;
    if (item < 0) break;
    // items carry a chunk index only when rows may be split (fewer than 2^21 units);
    // otherwise an item is the unit itself, which may exceed 2^21
    const bool split = a.split_slots > 0;
    const int unit = split ? item & ((1 << kItemUnitBits) - 1) : item;
    const int chunk = split ? item >> kItemUnitBits : 0;
    float* part = nullptr;
    if (a.split_slots > 0) {
      const int sb = a.slot_base[unit];
      if (sb >= 0) part = a.parts + (size_t)(sb + chunk) * kSlotFloats;
    }
    attn_unit<BQ, DENSE>(a, unit / a.nb, unit % a.nb, lds0, off, fe, tid, chunk, csize, part);
    if (a.one_shot) break;
  }
#endif  // __HIP_DEVICE_COMPILE__
}

// Work lists for the sparse kernel: one queue per KV group, in queue slot g % 8
// when there are >= 8 groups.  With fewer groups each group owns r = 8 / H_kv
// XCDs that all pop from one shared queue (slot g * r): they then work on the
// same query blocks at the same time, so the K/V tiles one XCD brings in from HBM
// are still in the shared last-level cache when the other XCDs of the group ask
// for them (separate queues let the XCDs of a group drift apart over a long
// layer, and each then streams K/V from HBM on its own).  Within an XCD the
// group's heads share its L2.  One-unit-per-workgroup mode empties the slots in
// order; static-list mode (short layers) puts every unit in slot 0.  Items are
// ordered longest first within a queue (a counting sort of list lengths: exact up to
// 768 entries, then in steps of 16).
//
// Split rows (persistent mode): a workgroup runs a row's tiles one after the
// other, so when the longest row holds more entries than the layer's work per
// workgroup (short layers, few heads), that row alone would set the kernel's
// time.  With G' = min(grid, slots / 2) and T the total of all rows' entries,
// rows longer than C = max(ceil(T / G'), 8, ceil(N_b / 1024)) are cut into
// ceil(L / C) chunks, each a work item of its own that leaves a partial result
// in a slot; attn_combine merges them.  Chunks number at most T / C + (rows
// longer than C) <= 2 G' <= slots.  The decision depends only on the lists and
// the grid, so results do not depend on timing.
//
// One workgroup builds everything and resets the queue counters; the order
// within one length is arbitrary (it only decides which workgroup runs an item,
// never a result).  Schedule area: int counters[8], int start[9], int C (at 17,
// INT_MAX when no row is split), int split rows (at 18); items from int offset
// 64; then slot_base[units], split_rows[slots / 2] and the partial slots.
constexpr int kQueueBuckets = kCostBuckets / kNumXcd;  // 1024 cost buckets per queue

__device__ __forceinline__ int cost_bucket(int64_t c) {
  c = c < 0 ? 0 : c;
  const int64_t b = c < 768 ? c : 768 + ((c - 768) >> 4);
  return (int)(b < kQueueBuckets - 1 ? b : kQueueBuckets - 1);
}

// Calls f(u, row length) for the units u = tid, tid + 1024, ... in that order, the row
// lengths of eight units loaded together (one memory latency per eight units, not
// one per unit).
template <typename F>
__device__ __forceinline__ void for_units(const AttnArgs& a, int total, int tid, F f) {
  constexpr int kBatch = 8;
  for (int u0 = 0; u0 < total; u0 += 1024 * kBatch) {
    int L[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int u = u0 + 1024 * j + tid;
      L[j] = u < total ? row_len(a, u / a.nb, u % a.nb) : 0;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int u = u0 + 1024 * j + tid;
      if (u < total) f(u, L[j]);
    }
  }
}

__global__ __launch_bounds__(1024) void attn_schedule(AttnArgs a) {
  __shared__ int hist[kCostBuckets];
  __shared__ int part[1024];
  __shared__ unsigned long long s_tot;
  __shared__ int s_max, s_slots, s_split;
  const int tid = threadIdx.x;
  const int total = a.hq * a.nb;
  for (int i = tid; i < kCostBuckets; i += 1024) hist[i] = 0;
  if (tid == 0) {
    s_tot = 0ull;
    s_max = 0;
    s_slots = 0;
    s_split = 0;
  }
  // Layers of up to 8192 units read each row length once, into registers, for all
  // three passes below (one memory latency instead of three on short layers).
  constexpr int kCached = 8;
  const bool cached = total <= 1024 * kCached;
  int Lc[kCached];
  if (cached) {
#pragma unroll
    for (int j = 0; j < kCached; ++j) {
      const int u = 1024 * j + tid;
      Lc[j] = u < total ? row_len(a, u / a.nb, u % a.nb) : 0;
    }
  }
  auto each_unit = [&](auto f) {
    if (cached) {
#pragma unroll
      for (int j = 0; j < kCached; ++j) {
        const int u = 1024 * j + tid;
        if (u < total) f(u, Lc[j]);
      }
    } else {
      for_units(a, total, tid, f);
    }
  };
  __syncthreads();
  int C = 0x7fffffff;
  if (a.split_slots > 0) {
    unsigned long long t = 0;
    int mx = 0;
    each_unit([&](int, int L) {
      t += (unsigned long long)L;
      mx = L > mx ? L : mx;
    });
    // one LDS atomic per wave, not per thread
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      t += (unsigned long long)__shfl_xor((long long)t, o);
      const int m2 = __shfl_xor(mx, o);
      mx = m2 > mx ? m2 : mx;
    }
    if ((tid & 63) == 0) {
      atomicAdd(&s_tot, t);
      atomicMax(&s_max, mx);
    }
    __syncthreads();
    long long gp = a.split_slots / 2;
    gp = a.grid < gp ? a.grid : gp;
    gp = gp < 1 ? 1 : gp;
    long long c = (long long)((s_tot + (unsigned long long)gp - 1) / (unsigned long long)gp);
    c = c > kMinChunk ? c : kMinChunk;
    const long long cmin = (a.nb + 1023) / 1024;
    c = c > cmin ? c : cmin;
    if (s_max > c) C = (int)c;
  }
  auto key = [&](int h, int len) {
    return (a.static_list ? 0 : unit_queue(a, h)) * kQueueBuckets + (kQueueBuckets - 1 - cost_bucket(len));
  };
  each_unit([&](int u, int L) {
    const int h = u / a.nb;
    if (L > C) {
      const int k = (L + C - 1) / C;
      for (int c = 0; c < k; ++c) atomicAdd(&hist[key(h, L - c * C < C ? L - c * C : C)], 1);
      a.slot_base[u] = atomicAdd(&s_slots, k);
      a.split_rows[atomicAdd(&s_split, 1)] = u;
    } else {
      atomicAdd(&hist[key(h, L)], 1);
      if (a.split_slots > 0) a.slot_base[u] = -1;
    }
  });
  __syncthreads();
  // exclusive scan over the keys, 8 per thread
  constexpr int per = kCostBuckets / 1024;
  int loc[per];
  int sum = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    loc[i] = sum;
    sum += hist[tid * per + i];
  }
  // inclusive scan of the per-thread sums: within each wave by shuffles, then the
  // 16 wave totals by one wave
  int incl = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if ((tid & 63) >= o) incl += y;
  }
  if ((tid & 63) == 63) part[tid >> 6] = incl;
  __syncthreads();
  if (tid < 64) {
    int wt = tid < 16 ? part[tid] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int y = __shfl_up(wt, o, 64);
      if (tid >= o) wt += y;
    }
    if (tid < 16) part[16 + tid] = wt;  // inclusive wave totals
  }
  __syncthreads();
  incl += (tid >> 6) ? part[16 + (tid >> 6) - 1] : 0;
  const int base = incl - sum;
  const int n_items = part[16 + 15];
#pragma unroll
  for (int i = 0; i < per; ++i) hist[tid * per + i] = base + loc[i];
  __syncthreads();
  // queue x starts at the first key of x: thread x * (kQueueBuckets / per) holds it
  if (tid < kNumXcd) {
    a.counter[tid] = 0;
    a.counter[8 + tid] = hist[tid * kQueueBuckets];
  }
  if (tid == 0) {
    a.counter[8 + kNumXcd] = n_items;
    a.counter[17] = C;
    a.counter[18] = s_split;
  }
  __syncthreads();
  each_unit([&](int u, int L) {
    const int h = u / a.nb;
    if (L > C) {
      const int k = (L + C - 1) / C;
      for (int c = 0; c < k; ++c) {
        const int pos = atomicAdd(&hist[key(h, L - c * C < C ? L - c * C : C)], 1);
        const_cast<int32_t*>(a.order)[pos] = u | (c << kItemUnitBits);
      }
    } else {
      const int pos = atomicAdd(&hist[key(h, L)], 1);
      const_cast<int32_t*>(a.order)[pos] = u;
    }
  });
}

// Merges the chunks of each split row in chunk order:
//   O = sum_c w_c O_c / sum_c w_c l_c,  w_c = 2^((m_c - M) c),  M = max_c m_c
// (chunks whose keys are all masked have m_c = -inf and weigh nothing).  grid
// slots / 2 (workgroups past the number of split rows exit), kCombineThreads threads:
// BQ query rows x kCombineThreads / BQ lanes, each lane 128 BQ / kCombineThreads dims.
// The chunks' row statistics and partial rows are loaded kCombineBatch chunks at a
// time (one memory latency per batch, not per chunk) and summed in chunk order.
constexpr int kCombineThreads = 1024, kCombineBatch = 4;
template <int BQ>
__global__ __launch_bounds__(kCombineThreads) void attn_combine(AttnArgs a) {
  const int i = blockIdx.x;
  if (i >= a.counter[18]) return;
  const int C = a.counter[17];
  const int u = a.split_rows[i];
  const int head = u / a.nb, qb = u % a.nb;
  const int k = (row_len(a, head, qb) + C - 1) / C;
  constexpr int TPR = kCombineThreads / BQ, DPT = kHeadDim / TPR, NB = kCombineBatch;
  constexpr size_t kSlotFloats = (size_t)BQ * (kHeadDim + 2);
  const int r = threadIdx.x / TPR, d0 = (threadIdx.x % TPR) * DPT;
  const float* base = a.parts + (size_t)a.slot_base[u] * kSlotFloats;
  float M = -__builtin_inff();
  for (int c0 = 0; c0 < k; c0 += NB) {
    float mv[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
      mv[j] = c0 + j < k ? base[(c0 + j) * kSlotFloats + BQ * kHeadDim + r] : -__builtin_inff();
#pragma unroll
    for (int j = 0; j < NB; ++j) M = fmaxf(M, mv[j]);
  }
  float acc[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) acc[e] = 0.f;
  float lsum = 0.f;
  for (int c0 = 0; c0 < k; c0 += NB) {
    float mv[NB], lv[NB];
    float4 pv[NB][DPT / 4];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const bool in = c0 + j < k;
      const float* sl = base + (size_t)(in ? c0 + j : 0) * kSlotFloats;
      mv[j] = in ? sl[BQ * kHeadDim + r] : -__builtin_inff();
      lv[j] = in ? sl[BQ * kHeadDim + BQ + r] : 0.f;
      const float4* po = reinterpret_cast<const float4*>(sl + (size_t)r * kHeadDim + d0);
#pragma unroll
      for (int e = 0; e < DPT / 4; ++e) pv[j][e] = in ? po[e] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (mv[j] == -__builtin_inff()) continue;  // also every slot past the last chunk
      const float w = fast_exp2((mv[j] - M) * a.c);
      lsum += w * lv[j];
#pragma unroll
      for (int e = 0; e < DPT / 4; ++e) {
        acc[4 * e] += w * pv[j][e].x;
        acc[4 * e + 1] += w * pv[j][e].y;
        acc[4 * e + 2] += w * pv[j][e].z;
        acc[4 * e + 3] += w * pv[j][e].w;
      }
    }
  }
  const int q = qb * BQ + r;
  if (q >= a.n) return;
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  uint16_t* orow = a.o + ((size_t)head * a.n + q) * kHeadDim + d0;
#pragma unroll
  for (int e = 0; e < DPT / 4; ++e) {
    const bf16x2 lo = pack_bf16(acc[4 * e] * inv, acc[4 * e + 1] * inv);
    const bf16x2 hi = pack_bf16(acc[4 * e + 2] * inv, acc[4 * e + 3] * inv);
    bf16x4 v4;
    v4[0] = lo[0]; v4[1] = lo[1]; v4[2] = hi[0]; v4[3] = hi[1];
    *reinterpret_cast<bf16x4*>(orow + 4 * e) = v4;
  }
}

template <int BQ, bool DENSE>
hipError_t launch_t(const AttnArgs& a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL((attn_kernel<BQ, DENSE>), dim3(grid), dim3(Geo<BQ>::kThreads), 0, stream, a);
  return hipGetLastError();
}

// Workgroups that fit on the device at once (persistent grid size), cached per
// device; threads that race on the first call compute and store the same value.
template <int BQ>
int persistent_grid() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  const int c = cached[dev].load(std::memory_order_relaxed);
  if (c > 0) return c;
  int cus = 0, per = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, attn_kernel<BQ, false>, Geo<BQ>::kThreads, 0) != hipSuccess || per <= 0)
    per = 1;
  cached[dev].store(cus * per, std::memory_order_relaxed);
  return cus * per;
}

}  // namespace

// Schedule area of the sparse kernel: header and items, then (when rows may be
// split: persistent mode, fewer than 2^21 units) slot_base, split_rows and the
// partial slots.  Slots: min(max_slots, 2 x units).
struct SchedLayout {
  int slots;
  size_t slot_base, split_rows, parts, total;
};

SchedLayout sched_layout(const Dims& d, int max_slots) {
  SchedLayout s;
  const size_t units = (size_t)d.hq * d.nb;
  const bool split = d.n < kOneShotMinLen && units < ((size_t)1 << kItemUnitBits);
  s.slots = split ? (int)(2 * units < (size_t)max_slots ? 2 * units : (size_t)max_slots) : 0;
  size_t off = (64 + units + (size_t)s.slots) * sizeof(int32_t);
  s.slot_base = off;
  if (s.slots > 0) off += units * sizeof(int32_t);
  s.split_rows = off;
  off += (size_t)(s.slots / 2) * sizeof(int32_t);
  off = (off + 255) & ~(size_t)255;
  s.parts = off;
  off += (size_t)s.slots * d.B * (kHeadDim + 2) * sizeof(float);
  s.total = off;
  return s;
}

size_t attn_schedule_bytes(const Dims& d, int max_slots) { return sched_layout(d, max_slots).total; }

namespace {
// The library's static schedule area for callers that cannot allocate: a file-scope
// device array, one copy per device.  In host code its name is not a device address;
// kernels get the address hipGetSymbolAddress returns for the current device.
__device__ __align__(256) char scratch[kStaticSchedBytes];
}  // namespace

hipError_t static_schedule_area(void** p) {
  constexpr int kMaxDevices = 64;
  static std::atomic<void*> addr[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* a = addr[dev].load(std::memory_order_relaxed);
  if (a == nullptr) {  // first call on this device (threads that race store the same address)
    if ((e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (a == nullptr) return hipErrorInvalidSymbol;
    addr[dev].store(a, std::memory_order_relaxed);
  }
  *p = a;
  return hipSuccess;
}

hipError_t launch_attn(const Dims& d, float scale, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                       const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, bool dense,
                       uint16_t* o, void* sched, hipStream_t stream, int max_slots) {
  if (d.n == 0 || d.hq == 0) return hipSuccess;
  if (dense && d.B == 64) {
    // Dense causal attention does not depend on the query block size: 128-row
    // blocks visit the same 64-key tiles in the same order, plus, for the first
    // half of each block, one fully masked tile that adds exact zeros.
    Dims d2 = d;
    d2.B = 128;
    d2.nb = (d.n + 127) / 128;
    return launch_attn(d2, scale, q, k, v, row_ptr, col_idx, col_cap, dense, o, sched, stream, max_slots);
  }
  AttnArgs a;
  a.q = q; a.k = k; a.v = v; a.o = o;
  a.row_ptr = row_ptr; a.col_idx = col_idx; a.col_cap = col_cap;
  a.order = nullptr; a.counter = nullptr; a.one_shot = 0; a.static_list = 0;
  a.slot_base = nullptr; a.split_rows = nullptr; a.parts = nullptr; a.split_slots = 0; a.grid = 0;
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
    char* sc = reinterpret_cast<char*>(sched);
    const SchedLayout sl = sched_layout(d, max_slots);
    a.counter = reinterpret_cast<int*>(sc);
    a.order = reinterpret_cast<const int32_t*>(sc) + 64;
    const int pg = d.B == 128 ? persistent_grid<128>() : persistent_grid<64>();
    // short layers with at least a persistent grid's worth of units: one unit per workgroup
    const bool short_one = d.n <= kStaticListMaxLen && (size_t)d.hq * d.nb >= (size_t)pg;
    a.one_shot = d.n >= kOneShotMinLen || short_one ? 1 : 0;
    a.static_list = d.n <= kStaticListMaxLen ? 1 : 0;
    a.split_slots = short_one ? 0 : sl.slots;  // the slots stay reserved, unused
    if (a.split_slots > 0) {
      a.slot_base = reinterpret_cast<int*>(sc + sl.slot_base);
      a.split_rows = reinterpret_cast<int*>(sc + sl.split_rows);
      a.parts = reinterpret_cast<float*>(sc + sl.parts);
    }
    grid = a.one_shot || pg > d.hq * d.nb ? d.hq * d.nb : pg;
    a.grid = grid;
    hipLaunchKernelGGL(attn_schedule, dim3(1), dim3(1024), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipError_t e;
  if (d.B == 128)
    e = dense ? launch_t<128, true>(a, grid, stream) : launch_t<128, false>(a, grid, stream);
  else
    e = launch_t<64, false>(a, grid, stream);  // dense 64-row layers run as 128-row ones (above)
  if (e != hipSuccess || a.split_slots == 0) return e;
  if (d.B == 128)
    hipLaunchKernelGGL(attn_combine<128>, dim3(a.split_slots / 2), dim3(kCombineThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_combine<64>, dim3(a.split_slots / 2), dim3(kCombineThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace crisp
