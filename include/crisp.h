/*
 * crisp.h -- C ABI of libcrisp: CRISP sparse prefill attention on AMD gfx950.
 *
 * CRISP (Cliff-awaRe Input-adaptive Sparse Prefilling) computes, per attention
 * head of a causal prefill layer:
 *   1. a proxy attention map from the last query block          (Alg. 2)
 *   2. C_struct, the proxy mass on sink/local anchor keys, and a
 *      route: Vertical-Slash (VS) if C_struct >= tau, else PE    (Sec. 3.2, Alg. 2)
 *   3. a key-block set per query block: VS heads by a sink-aware
 *      noise floor on vertical and slash block scores (Alg. 3,
 *      Sec. 4.3); PE heads by a gamma-cumsum over pooled scores  (Alg. 4)
 *   4. causal softmax attention restricted to that set           (Eq. 1, Sec. 2.1)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Tensors are contiguous, row-major, on the device, bf16 (raw bits):
 *   q [H_q, n, d], k and v [H_kv, n, d], o [H_q, n, d];  d = head_dim = 128.
 * GQA: query head h reads KV head h / (H_q / H_kv).  Batch is 1 (one layer of
 * one sequence); callers loop over batch entries.
 * N_b = ceil(n / B) key/query blocks of B tokens; the last block may be partial.
 * The proxy uses the last b = min(B, n) queries.
 *
 * Block lists (CSR, one region per query head):
 *   row_ptr [H_q][N_b + 1]  int32, offsets local to the head's region, row_ptr[h][0] = 0
 *   col_idx [H_q][cap]      int32, cap = col_cap_per_head >= crisp_col_capacity(shape)
 *   Row qb of head h lists key blocks col_idx[h][row_ptr[h][qb] .. row_ptr[h][qb+1]),
 *   ascending, unique, each <= qb; lists built by this library always hold 0 and qb.
 *
 * Ownership and execution: the caller allocates and owns every buffer, the
 * workspace included.  The library never allocates or frees device memory,
 * never synchronises a stream or the device and never copies to the host.
 * Every call only enqueues work on `stream` (a hipStream_t, NULL = null stream)
 * and returns; results are valid once the caller synchronises.  Inputs are
 * read-only; outputs are fully overwritten.  Calls on different streams must
 * use different workspaces and outputs.
 *
 * Errors: arguments are validated on the host before anything is enqueued, so a
 * non-OK status means nothing was launched -- except CRISP_EHIP, which reports a
 * launch failure (hipGetLastError) after earlier launches of the same call may
 * already be queued.  crisp_last_error() returns a thread-local message for the
 * last failing call of the calling thread.  Non-finite inputs give undefined
 * (but memory-safe) results.  No C++ exception crosses this interface.
 *
 * Debug build: libcrisp_debug.so exports the same functions with the same host-side
 * validation and, before each call's kernels, also checks on the device that Q, K and
 * V hold no infinite or NaN value and, for crisp_sparse_attn, that every list row
 * keeps row_ptr within [0, col_cap_per_head] and non-decreasing and its entries in
 * [0, qb] and strictly increasing; a violation is CRISP_EINVAL with a message naming
 * it.  These checks launch their own kernels and wait for the stream (the one place
 * where the library synchronises), and its attention kernels run their tile pipeline
 * serialised (same arithmetic, same results as the release build, bit for bit), so
 * the debug build is for testing, not timing.
 */
#ifndef CRISP_H
#define CRISP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t crisp_bf16;  /* raw bfloat16 bits */
typedef void* crisp_stream;   /* hipStream_t */

typedef enum {
  CRISP_OK = 0,
  CRISP_EINVAL = 1,       /* bad shape, parameter, null/misaligned pointer, capacity or workspace too small */
  CRISP_EUNSUPPORTED = 2, /* head_dim != 128 or block not in {64, 128} */
  CRISP_EHIP = 3          /* a HIP launch failed; see crisp_last_error() */
} crisp_status;

enum { CRISP_ROUTE_VS = 0, CRISP_ROUTE_PE = 1, CRISP_ROUTE_DENSE = 2 /* context-length gate */ };

/* crisp_params.route_mode: what decides a head's route.
 *   CRISP_ROUTE_BY_CSTRUCT  C_struct >= tau_proxy (Alg. 2, the paper's method)
 *   CRISP_ROUTE_BY_JSD      D_JS >= tau_jsd (App. A, FlexPrefill's pattern search)
 * crisp_params.vs_mode: how a VS head selects blocks per direction.
 *   CRISP_VS_FLOOR          sink-aware noise floor (Alg. 3, Sec. 4.3)
 *   CRISP_VS_GAMMA          shortest prefix of the blocks by decreasing score whose
 *                           mass reaches gamma (App. A, FlexPrefill's VS selection) */
enum { CRISP_ROUTE_BY_CSTRUCT = 0, CRISP_ROUTE_BY_JSD = 1 };
enum { CRISP_VS_FLOOR = 0, CRISP_VS_GAMMA = 1 };

/* crisp_params.floor_mode: the noise level mu of the floor (vs_mode CRISP_VS_FLOOR).
 *   CRISP_FLOOR_MEAN        r / (N_b - 2), the mean non-anchor mass (Sec. 4.3)
 *   CRISP_FLOOR_MEDIAN      the median of p_d[1 .. N_b-2] (App. H; for an even count
 *                           the mean of the two middle values, float32)          */
enum { CRISP_FLOOR_MEAN = 0, CRISP_FLOOR_MEDIAN = 1 };

/* Layer shape.  H_q % H_kv == 0, H_kv >= 1, n >= 0, head_dim == 128,
 * block in {64, 128}.  n == 0 or H_q == 0 is a valid empty layer: calls return
 * CRISP_OK and launch nothing. */
typedef struct {
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t seq_len;
  int32_t head_dim;
  int32_t block;
} crisp_shape;

/* Hyperparameters (Sec. 5 setup: tau_proxy = 0.2, gamma = 0.95 for PE heads,
 * alpha = 1.0, k_min = 1024 tokens per direction; Sec. 3.2: w_sink = w_local = 128).
 *   alpha          noise-floor multiplier, >= 0; block J is kept iff p[J] > alpha * mu
 *   tau_proxy      route threshold on C_struct (VS iff C_struct >= tau_proxy)
 *   gamma          PE cumulative-mass target, 0 < gamma <= 1
 *   w_sink/w_local anchor windows in tokens: keys [0, w_sink) and [n - w_local, n); >= 0
 *   k_min_blocks   minimum blocks per VS direction; 0 means ceil(1024 / block)
 *   softmax_scale  logit scale; 0 means 1 / sqrt(head_dim)
 * The FlexPrefill comparator of App. A on the same kernels (defaults: the paper's method):
 *   route_mode     CRISP_ROUTE_BY_CSTRUCT (default) or CRISP_ROUTE_BY_JSD
 *   vs_mode        CRISP_VS_FLOOR (default) or CRISP_VS_GAMMA (uses gamma)
 *   tau_jsd        D_JS route threshold, finite; default 0.1 (the paper gives none)
 *   floor_mode     CRISP_FLOOR_MEAN (default) or CRISP_FLOOR_MEDIAN (App. H)
 *   dense_below_len  context-length gate (Sec. 5, short contexts): crisp_prefill_attn
 *                  runs dense causal attention when seq_len < this; 0 (default) never */
typedef struct {
  float alpha;
  float tau_proxy;
  float gamma;
  int32_t w_sink;
  int32_t w_local;
  int32_t k_min_blocks;
  float softmax_scale;
  int32_t route_mode;
  int32_t vs_mode;
  float tau_jsd;
  int32_t floor_mode;
  int32_t dense_below_len;
} crisp_params;

/* Fills *p with the paper's defaults listed above. */
void crisp_params_default(crisp_params* p);

/* N_b * (N_b + 1) / 2: the largest number of causal key blocks a head can select;
 * the col_idx capacity per head that always suffices.  Returns -1 on a bad shape. */
int64_t crisp_col_capacity(const crisp_shape* shape);

/* Host only.  Bytes of workspace that crisp_estimate, crisp_route_select and
 * crisp_prefill_attn need for `shape` (the largest of the three).  The workspace
 * must be 256-byte aligned; its contents on entry do not matter. */
crisp_status crisp_workspace_size(const crisp_shape* shape, size_t* bytes);

/* Stages 1-2 (Alg. 2; C_struct equation of Sec. 3.2; directional scores of Alg. 3).
 * For each query head h, with A_hat = causal Softmax(Q_hat K^T * scale) over the
 * last b queries:
 *   c_struct[h]   = (1/b) sum_r sum_{j in anchors} A_hat[r, j]
 *   p_v[h][J]     = (1/b) sum_r sum_{j in block J} A_hat[r, j]              (column mass)
 *   p_s[h][J]     = (1/b) sum_r sum_{j in block J} A_hat[r, j - (b - 1 - r)] (diagonal mass;
 *                   the diagonal through the last proxy row at key j; terms with a
 *                   negative key index are absent)
 * Outputs: c_struct float[H_q], p_v and p_s float[H_q][N_b] (4-byte aligned). */
crisp_status crisp_estimate(const crisp_shape* shape, const crisp_params* params,
                            const crisp_bf16* q, const crisp_bf16* k,
                            float* c_struct, float* p_v, float* p_s,
                            void* workspace, size_t workspace_bytes, crisp_stream stream);

/* FlexPrefill's pattern search (App. A), the comparator's route score.  For each
 * query head h: a_bar = Softmax(scale * pool(Q_hat) . pool(K)^T) over the N_b key
 * blocks (Q_hat = the last b queries pooled to one row, K mean-pooled per block,
 * a partial last block over its own rows) and
 *   jsd[h] = sqrt(KL(p_v[h] || m) / 2 + KL(a_bar || m) / 2),  m = (p_v[h] + a_bar) / 2,
 * natural logarithms, p_v[h] being crisp_estimate's vertical block mass (App. A's
 * per-query mean, sum-pooled over blocks).  Output: jsd float[H_q].  Leaves the
 * pooled K in the workspace. */
crisp_status crisp_jsd(const crisp_shape* shape, const crisp_params* params,
                       const crisp_bf16* q, const crisp_bf16* k, const float* p_v, float* jsd,
                       void* workspace, size_t workspace_bytes, crisp_stream stream);

/* Stage 3 (Alg. 2 route; Alg. 3 with the noise floor of Sec. 4.3; Alg. 4).
 * c_struct is the route score: C_struct from crisp_estimate, or, with route_mode
 * CRISP_ROUTE_BY_JSD, D_JS from crisp_jsd.  route[h] = VS iff score >= tau_proxy
 * (tau_jsd for D_JS), float32 compare, else PE.  With vs_mode CRISP_VS_GAMMA a VS
 * direction takes the shortest prefix of its blocks ordered by decreasing p_d (ties:
 * lower block first) whose mass reaches gamma, then k = min(max(that, k_min), N_b)
 * as below (all blocks if the mass never reaches gamma).
 * VS head, per direction d in {v, s}: r = max((1 - p_d[0]) - p_d[N_b-1], 0),
 *   mu = r / (N_b - 2), c = #{J : p_d[J] > alpha * mu}, k = min(max(c, k_min), N_b),
 *   S_d = the k largest p_d (ties: lower block index first); nothing when N_b <= 2.
 *   Row qb then holds {0, qb} u {J in S_v : J <= qb} u {qb - (N_b-1-J) >= 0 : J in S_s}.
 * PE head: Q and K are mean-pooled per block, A_tilde = block-causal row softmax of
 *   pooled logits divided by its total; pairs are taken in order of decreasing
 *   A_tilde (ties: lower qb * N_b + kb first) until their mass reaches gamma; row qb
 *   holds its taken pairs plus {0, qb}.
 * Inputs c_struct, p_v, p_s are crisp_estimate's outputs.  Outputs: route int8[H_q];
 * row_ptr/col_idx as described above (col_cap_per_head >= crisp_col_capacity);
 * dir_mask_or_null, if given, uint8[H_q][2][N_b]: 1 where the block is in S_v
 * (index 0) or S_s (index 1) of a VS head, 0 elsewhere and for PE heads. */
crisp_status crisp_route_select(const crisp_shape* shape, const crisp_params* params,
                                const crisp_bf16* q, const crisp_bf16* k,
                                const float* c_struct, const float* p_v, const float* p_s,
                                int8_t* route, int32_t* row_ptr, int32_t* col_idx,
                                int64_t col_cap_per_head, uint8_t* dir_mask_or_null,
                                void* workspace, size_t workspace_bytes, crisp_stream stream);

/* Host only.  Bytes of the optional crisp_sparse_attn workspace (256-byte aligned). */
crisp_status crisp_sparse_workspace_size(const crisp_shape* shape, size_t* bytes);

/* Stage 4 (Eq. 1): o[h][i] = sum_{j in J(i)} softmax_j(scale * q_i . k_j) v_j with
 * J(i) = {j <= i : j / B in row (i / B) of head h's list}.  Accepts caller-built
 * lists; entries outside [0, qb] are ignored and row_ptr values are clamped to
 * [0, col_cap_per_head], so a malformed list cannot cause an out-of-bounds access.
 * Rows are read as given: the order of a row's entries only changes floating-point
 * rounding, and an entry listed twice counts its block twice (crisp_route_select
 * writes every row ascending and unique; the debug build rejects other rows).
 * A row with no visible key gets o = 0.  softmax_scale 0 means 1/sqrt(d).
 * workspace_or_null (crisp_sparse_workspace_size bytes) holds a longest-first
 * work list that balances rows of very different lengths over the GPU and, for
 * layers shorter than 512k tokens, slots for partial results: a row far longer
 * than the layer's work per workgroup is split into chunks whose softmax partials
 * are merged in chunk order (up to 8192 tokens, a layer with at least as many
 * (head, query block) units as the GPU holds workgroups at once runs one workgroup
 * per unit and splits nothing).  Results are repeatable for given lists; a split row
 * differs from an unsplit one by floating-point rounding only.  With NULL the rows
 * are processed whole, in a fixed order. */
crisp_status crisp_sparse_attn(const crisp_shape* shape, float softmax_scale,
                               const crisp_bf16* q, const crisp_bf16* k, const crisp_bf16* v,
                               const int32_t* row_ptr, const int32_t* col_idx,
                               int64_t col_cap_per_head, crisp_bf16* o,
                               void* workspace_or_null, size_t workspace_bytes, crisp_stream stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): crisp_sparse_attn with its balanced
 * work list kept in the library's own static schedule area instead of a caller's
 * workspace.  Same arguments, list semantics, output and error behaviour as
 * crisp_sparse_attn; it allocates and frees nothing.  The area is a file-scope device
 * array of 16 MiB, one per GPU the library runs on, held until the process ends; it
 * holds the work list of any layer of up to 1.5 million (head, query block) units
 * (about 4 million from 2^19 tokens on, where rows are never split; a larger layer is
 * CRISP_EINVAL before anything is enqueued) and at most 64 partial-result slots, so
 * fewer long rows are split than with a workspace (results then differ from
 * crisp_sparse_attn's by floating-point rounding only).  Every call on one GPU uses that
 * GPU's area, which is rewritten before each use: calls that overlap in time on one
 * GPU (on different streams, or from different threads) race and must be serialised
 * by the caller. */
crisp_status crisp_sparse_attn_noalloc(const crisp_shape* shape, float softmax_scale,
                                       const crisp_bf16* q, const crisp_bf16* k, const crisp_bf16* v,
                                       const int32_t* row_ptr, const int32_t* col_idx,
                                       int64_t col_cap_per_head, crisp_bf16* o, crisp_stream stream);

/* Alg. 1: all stages on `stream`: estimate, route and select, sparse attention
 * (with route_mode CRISP_ROUTE_BY_JSD, crisp_jsd's pattern search before the route).
 * route_or_null, row_ptr_or_null and col_idx_or_null, if all three are given,
 * receive the route and block lists (col_idx capacity crisp_col_capacity per
 * head); if they are all null the library keeps them in the workspace (then
 * `workspace_bytes` must be crisp_prefill_workspace_size).  Mixed null/non-null
 * is CRISP_EINVAL.  Below the context-length gate (seq_len < dense_below_len) the layer
 * is dense causal attention: route[h] = CRISP_ROUTE_DENSE and every row lists all its
 * causal blocks. */
crisp_status crisp_prefill_attn(const crisp_shape* shape, const crisp_params* params,
                                const crisp_bf16* q, const crisp_bf16* k, const crisp_bf16* v,
                                crisp_bf16* o, int8_t* route_or_null, int32_t* row_ptr_or_null,
                                int32_t* col_idx_or_null,
                                void* workspace, size_t workspace_bytes, crisp_stream stream);

/* Host only.  Workspace bytes for crisp_prefill_attn when it keeps the route and
 * block lists itself (crisp_workspace_size plus the route, row_ptr and col_idx). */
crisp_status crisp_prefill_workspace_size(const crisp_shape* shape, size_t* bytes);

/* The dense baseline of the paper's latency comparison (Sec. 5 setup: full causal
 * attention with FlashAttention, against which the sparse speedups are quoted): Eq. 1
 * with every causal key block selected, o[h][i] = sum_{j <= i} softmax_j(scale *
 * q_i . k_j) v_j, run by the same kernel as crisp_sparse_attn with every causal block
 * listed implicitly.  Same tensor layouts, ownership and error behaviour as
 * crisp_sparse_attn; no workspace.  softmax_scale 0 means 1/sqrt(d). */
crisp_status crisp_dense_attn(const crisp_shape* shape, float softmax_scale,
                              const crisp_bf16* q, const crisp_bf16* k, const crisp_bf16* v,
                              crisp_bf16* o, crisp_stream stream);

/* Static name of a status code. */
const char* crisp_status_string(crisp_status status);

/* Message of the calling thread's last failing call ("" if none). */
const char* crisp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CRISP_H */
