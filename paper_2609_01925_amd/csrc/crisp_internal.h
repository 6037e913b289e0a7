// Internal launch interface between the C ABI layer (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace crisp {

constexpr int kHeadDim = 128;

// Shape-derived sizes shared by host and kernels.
struct Dims {
  int hq, hkv, G, n, B, nb, b;  // b = min(B, n) proxy rows
  int64_t cap;                  // nb * (nb + 1) / 2
};

// Estimator work split: each workgroup owns `bps` whole key blocks.
struct EstSplit {
  int bps;
  int splits;
};
EstSplit est_split(const Dims& d);

// Workspace layout (byte offsets; every region 256-byte aligned).
struct WsLayout {
  size_t rowstat, rowfinal, parts, masks, qbar, kbar, atil, rhist, rstate, rowinfo, sched, total;
};
WsLayout ws_layout(const Dims& d);

// Partial-result slots of the sparse kernel's schedule area (split rows): a caller's
// workspace provides up to kWorkspaceSlots; the library's own static area, used by the
// entry point that allocates nothing, up to kStaticSlots within kStaticSchedBytes.
constexpr int kWorkspaceSlots = 1024;
constexpr int kStaticSlots = 64;
constexpr size_t kStaticSchedBytes = (size_t)16 << 20;

// Bytes of the longest-first work list used by the persistent sparse kernel, with at
// most max_slots partial-result slots.
size_t attn_schedule_bytes(const Dims& d, int max_slots = kWorkspaceSlots);

// Device address of the library's static schedule area on the current device (its
// kStaticSchedBytes are a file-scope device array; each device holds its own copy).
hipError_t static_schedule_area(void** p);

// sched == nullptr: static grid (dense, or sparse without a work list); otherwise sched
// holds attn_schedule_bytes(d, max_slots) bytes.
hipError_t launch_attn(const Dims& d, float scale, const uint16_t* q, const uint16_t* k, const uint16_t* v,
                       const int32_t* row_ptr, const int32_t* col_idx, int64_t col_cap, bool dense,
                       uint16_t* o, void* sched, hipStream_t stream, int max_slots = kWorkspaceSlots);

// combine_only: C_struct and the per-row normalisers only; p_v and p_s stay unwritten
// (launch_select with scores_from_ws forms them from the workspace instead).
hipError_t launch_estimate(const Dims& d, float scale, int w_sink, int w_local, const uint16_t* q,
                           const uint16_t* k, float* c_struct, float* p_v, float* p_s, char* ws,
                           hipStream_t stream, bool combine_only = false);

// Layers of at most this many blocks take the one-launch-per-head selection.
constexpr int kSmallSelectBlocks = 64;

// route_score is C_struct (tau = tau_proxy) or D_JS (tau = tau_jsd); vs_mode 0 is the
// noise floor (floor_mode 0: mean, 1: median), 1 gamma coverage; kbar_all: K_bar of
// every KV group is already in ws.  scores_from_ws (layers of at most kSmallSelectBlocks
// blocks, after launch_estimate with combine_only on the same ws): p_v and p_s are not
// read; the selection forms them from the estimator's sums in ws.
hipError_t launch_select(const Dims& d, float scale, float alpha, float tau, float gamma, int k_min, int vs_mode,
                         int floor_mode, bool kbar_all, const uint16_t* q, const uint16_t* k, const float* route_score,
                         const float* p_v, const float* p_s, int8_t* route, int32_t* row_ptr, int32_t* col_idx,
                         int64_t col_cap, uint8_t* dir_mask, char* ws, hipStream_t stream, bool scores_from_ws = false);

// route = dense and full causal CSR lists (col_cap >= nb (nb + 1) / 2).
hipError_t launch_dense_lists(const Dims& d, int8_t* route, int32_t* row_ptr, int32_t* col_idx, int64_t col_cap,
                              hipStream_t stream);

// D_JS per query head into jsd[hq]; leaves K_bar of every KV group in ws.
hipError_t launch_jsd(const Dims& d, float scale, const uint16_t* q, const uint16_t* k, const float* p_v,
                      float* jsd, char* ws, hipStream_t stream);

// Debug build only (CRISP_DEBUG): these wait for the stream.  *found = 1 if any of
// the n bf16 values is infinite or NaN; *code = 0 if every row of the lists keeps the
// list invariants, else 1 (row_ptr out of range or decreasing), 2 (an entry outside
// [0, qb]) or 3 (entries not strictly increasing).
hipError_t debug_nonfinite(const uint16_t* p, size_t n, hipStream_t stream, int* found);
hipError_t debug_lists(const Dims& d, const int32_t* row_ptr, const int32_t* col_idx, int64_t cap,
                       hipStream_t stream, int* code);

}  // namespace crisp
