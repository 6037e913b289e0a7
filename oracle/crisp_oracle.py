"""CRISP oracle: a plain, slow CPU statement of the paper's definitions.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import this module.  The HIP path never calls it, shares no
code with it, and nothing here reads anything the HIP path produced.

Arithmetic is float64 on the exact float values of the bf16 inputs; every
long reduction (softmax denominators, C_struct, the directional scores, the
noise-floor residual and mean, the pooled-score normalisation and the
gamma cumulative sum) is a float64 sum.  Every floating-point comparison that
decides an integer result (route, VS block membership, PE order and cutoff) is
taken in float32, the precision of the GPU kernels, on the float64 results
rounded once to float32; the GPU side takes the same decisions in float32 on
its own values.  Where the paper is silent or
ambiguous, the reading taken is named in the function's docstring (the readings
are listed with their reasons in the design notes).

Notation (paper Sec. 2-4): n sequence length, d head dim, B block size,
N_b = ceil(n / B) blocks, b = min(B, n) proxy rows, s = 1/sqrt(d) unless given.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

ROUTE_VS = 0
ROUTE_PE = 1


@dataclass
class Params:
    """CRISP hyperparameters; defaults are the paper's universal configuration
    (Sec. 5, Setup: tau_proxy = 0.2, gamma = 0.95, alpha = 1.0, B = 128,
    k_min = 1024 tokens per direction; Sec. 3.2: w_sink = w_local = 128)."""
    alpha: float = 1.0
    tau_proxy: float = 0.2
    gamma: float = 0.95
    w_sink: int = 128
    w_local: int = 128
    k_min_blocks: int = 0          # 0 -> ceil(1024 / B) blocks
    softmax_scale: float = 0.0     # 0 -> 1 / sqrt(d)
    # FlexPrefill comparator (App. A): route by the JSD pattern search instead of
    # C_struct, and/or select VS blocks by gamma coverage instead of the noise floor.
    route_mode: str = "cstruct"    # "cstruct" (Alg. 2) or "jsd" (App. A, pattern search)
    vs_mode: str = "floor"         # "floor" (Alg. 3) or "gamma" (App. A, VS index selection)
    tau_jsd: float = 0.1           # JSD threshold; the paper gives none (reading R26)
    floor_mode: str = "mean"       # "mean" (Sec. 4.3) or "median" (App. H variant)

    def scale(self, d: int) -> float:
        return self.softmax_scale if self.softmax_scale > 0 else 1.0 / math.sqrt(d)

    def k_min(self, block: int) -> int:
        return self.k_min_blocks if self.k_min_blocks > 0 else -(-1024 // block)


def n_blocks(n: int, block: int) -> int:
    """N_b = ceil(n / B) (Sec. 4.3)."""
    return -(-n // block)


def block_range(J: int, n: int, block: int) -> range:
    return range(J * block, min((J + 1) * block, n))


# ----------------------------------------------------------------------------
# Stage 1: proxy attention and C_struct (Alg. 2, Eq. for C_struct in Sec. 3.2)
# ----------------------------------------------------------------------------

def proxy_attention(q: np.ndarray, k: np.ndarray, block: int, scale: float) -> np.ndarray:
    """A_hat = Softmax(Q_hat K^T s) with Q_hat = the last b = min(B, n) queries (Alg. 2).

    Reading: the proxy is causal -- proxy row r is query i_r = n - b + r and
    sees keys j <= i_r only; entries above the causal edge are 0.
    Returns A_hat as a [b, n] float64 array whose rows sum to 1.
    """
    n = q.shape[0]
    b = min(block, n)
    rows = np.arange(n - b, n)
    z = (q[rows] @ k.T) * scale
    z[np.arange(n)[None, :] > rows[:, None]] = -np.inf
    z = z - z.max(axis=1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=1, keepdims=True)


def anchor_mask(n: int, w_sink: int, w_local: int) -> np.ndarray:
    """S_anchor = first w_sink keys union last w_local keys (Sec. 3.2).

    Reading: the local window is absolute -- the last w_local keys of the
    sequence -- and the two windows form a set union (overlap counted once).
    """
    m = np.zeros(n, dtype=bool)
    m[: max(0, min(w_sink, n))] = True
    if w_local > 0:
        m[max(0, n - w_local):] = True
    return m


def c_struct(ahat: np.ndarray, n: int, w_sink: int, w_local: int) -> float:
    """C_struct = (1/|Q_hat|) sum_i sum_{j in S_anchor} A_hat[i, j] (Sec. 3.2 / Alg. 2)."""
    return float(ahat[:, anchor_mask(n, w_sink, w_local)].sum() / ahat.shape[0])


def route(cs: float, tau_proxy: float) -> int:
    """VS iff C_struct >= tau_proxy, else PE (Alg. 2).  Compared in float32."""
    return ROUTE_VS if np.float32(cs) >= np.float32(tau_proxy) else ROUTE_PE


# ----------------------------------------------------------------------------
# Stage 2/3, VS path: directional scores and the sink-aware floor (Alg. 3,
# noise-floor equation and selection rule in Sec. 4.3)
# ----------------------------------------------------------------------------

def vs_scores(ahat: np.ndarray, n: int, block: int):
    """a_v = colmean(A_hat), a_s = diagmean(A_hat), p_d = blockpool(a_d) (Alg. 3).

    Readings: the means divide by b (the row count), so sum(a_v) = sum(a_s) = 1;
    a_s[j] collects the diagonal through (last proxy row, key j), i.e. entry
    A_hat[r, j - (b - 1 - r)] for every row r where that key index is >= 0;
    blockpool sums the B entries of a block (p_d is a mass).
    Returns (a_v, a_s, p_v, p_s).
    """
    b = ahat.shape[0]
    a_v = ahat.sum(axis=0) / b
    a_s = np.zeros(n)
    for r in range(b):
        shift = b - 1 - r
        a_s[shift:] += ahat[r, : n - shift]
    a_s /= b
    nb = n_blocks(n, block)
    p_v = np.array([a_v[block_range(J, n, block).start: block_range(J, n, block).stop].sum() for J in range(nb)])
    p_s = np.array([a_s[block_range(J, n, block).start: block_range(J, n, block).stop].sum() for J in range(nb)])
    return a_v, a_s, p_v, p_s


def vs_floor(p: np.ndarray, alpha: float, floor: str = "mean"):
    """r_d = max(1 - p_d[0] - p_d[N_b-1], 0), mu_d = r_d / (N_b - 2), threshold alpha * mu_d
    (Alg. 3; noise-floor equation, Sec. 4.3).  r_d, mu_d and alpha * mu_d are float64,
    r_d evaluated as printed, ((1 - p[0]) - p[N_b-1]).  For the score vectors of
    vs_scores, which sum to 1, r_d is the mass of the inner blocks p[1 .. N_b-2] up to
    float64 rounding (reading R20; crisp_head checks it).  Needs N_b > 2.

    floor="median" is App. H's robust variant: mu_d is the median of the N_b - 2
    non-anchor block scores p_d[1 .. N_b-2] (reading R29: for an even count the
    mean of the two middle values, in float32).
    Returns (r_d, mu_d, threshold); the median variant returns float32 mu and threshold."""
    nb = len(p)
    p64 = np.asarray(p, dtype=np.float64)
    r = max((1.0 - p64[0]) - p64[nb - 1], 0.0)
    if floor == "median":
        p32 = np.asarray(p, dtype=np.float32)
        mid = np.sort(p32[1:nb - 1])
        m = len(mid)
        mu = mid[m // 2] if m % 2 else (mid[m // 2 - 1] + mid[m // 2]) * np.float32(0.5)
        return r, mu, np.float32(alpha) * mu
    mu = r / (nb - 2)
    return r, mu, float(alpha) * mu


def vs_select(p: np.ndarray, alpha: float, k_min: int, floor: str = "mean") -> List[int]:
    """S_d = top-k_d(p_d) with k_d = clip(|{J : p_d[J] > alpha mu_d}|, k_min, N_b) (Alg. 3).

    Readings: the floor test is strict (>), taken in float32 between the block
    score and the float64 threshold, each rounded once; k_min is in blocks;
    top-k orders by (float32 p desc, block index asc).  With N_b <= 2 the forced blocks already
    cover every causal pair, so the direction selects nothing extra.
    Returns the selected block indices, ascending.
    """
    nb = len(p)
    if nb <= 2:
        return []
    p32 = np.asarray(p, dtype=np.float32)
    _, _, thr = vs_floor(p, alpha, floor)
    c = int(np.count_nonzero(p32 > np.float32(thr)))
    kd = min(max(c, k_min), nb)
    order = sorted(range(nb), key=lambda J: (-float(p32[J]), J))
    return sorted(order[:kd])


def vs_block_sets(S_v: Sequence[int], S_s: Sequence[int], nb: int) -> List[List[int]]:
    """Expand S_v u S_s u {0, N_b - 1} into a key-block set per query block (Alg. 3 output,
    used as the index set of Eq. 1).

    Readings: vertical block J covers key block J for every query block qb >= J;
    slash block J is the block diagonal at distance N_b - 1 - J, i.e. key block
    qb - (N_b - 1 - J) when that is >= 0 (block-aligned: the neighbouring
    diagonal block is not added).  The forced {0, N_b - 1} are the sink column
    and the main diagonal, so every row holds {0, qb}.
    """
    sets = []
    for qb in range(nb):
        s = {0, qb}
        s.update(J for J in S_v if J <= qb)
        for J in S_s:
            kb = qb - (nb - 1 - J)
            if kb >= 0:
                s.add(kb)
        sets.append(sorted(s))
    return sets


# ----------------------------------------------------------------------------
# PE path (Alg. 4)
# ----------------------------------------------------------------------------

def pool_blocks(x: np.ndarray, block: int) -> np.ndarray:
    """pool(X): mean of each block of B consecutive rows (Alg. 4).  A partial last
    block is averaged over the rows it has.  Reading: pool = mean."""
    n = x.shape[0]
    return np.stack([x[block_range(J, n, block).start: block_range(J, n, block).stop].mean(axis=0)
                     for J in range(n_blocks(n, block))])


def pe_scores(q: np.ndarray, k: np.ndarray, block: int, scale: float) -> np.ndarray:
    """A_bar = Softmax(pool(Q) pool(K)^T s), then A_bar / sum(A_bar) (Alg. 4).

    Reading: the softmax is block-causal (kb <= qb, diagonal included); entries
    with kb > qb are 0.  Returns the normalised [N_b, N_b] matrix (float64).
    """
    qbar = pool_blocks(q, block)
    kbar = pool_blocks(k, block)
    L = (qbar @ kbar.T) * scale
    nb = L.shape[0]
    L[np.triu_indices(nb, 1)] = -np.inf
    L = L - L.max(axis=1, keepdims=True)
    E = np.exp(L)
    A = E / E.sum(axis=1, keepdims=True)
    return A / A.sum()


def pe_select(At: np.ndarray, gamma: float):
    """Sort the causal pairs of A_tilde descending and keep the shortest prefix whose
    cumulative mass reaches gamma (Alg. 4, K* = min{k : cumsum >= gamma}).

    Readings: the order is descending (ties by flat index qb * N_b + kb
    ascending); values are the float32-rounded A_tilde; the cumulative sum is
    float64; if it never reaches gamma every pair is kept.
    Returns (selected pair list [(qb, kb)], K*, info dict).
    """
    nb = At.shape[0]
    qb, kb = np.tril_indices(nb)
    vals = At[qb, kb].astype(np.float32)
    flat = qb.astype(np.int64) * nb + kb
    order = np.lexsort((flat, -vals.astype(np.float64)))
    csum = np.cumsum(vals[order].astype(np.float64))
    g = np.float64(np.float32(gamma))
    hit = np.nonzero(csum >= g)[0]
    kstar = int(hit[0]) + 1 if len(hit) else len(order)
    sel = order[:kstar]
    info = {
        "kstar": kstar,
        "t_star": float(vals[order[kstar - 1]]) if kstar > 0 else 0.0,
        "csum_before": float(csum[kstar - 2]) if kstar >= 2 else 0.0,
        "csum_at": float(csum[kstar - 1]) if kstar >= 1 else 0.0,
        "n_pairs": len(order),
    }
    return list(zip(qb[sel].tolist(), kb[sel].tolist())), kstar, info


def pe_block_sets(pairs, nb: int) -> List[List[int]]:
    """Per query block: the selected key blocks plus the forced {0, qb}.
    Reading: Alg. 4 forces nothing; the sink and diagonal blocks are added so
    that every row is non-empty and holds the blocks Alg. 3 always keeps."""
    sets = [{0, qb} for qb in range(nb)]
    for a, c in pairs:
        sets[a].add(c)
    return [sorted(s) for s in sets]


# ----------------------------------------------------------------------------
# Stage 4: sparse attention (Eq. 1, Sec. 2.1)
# ----------------------------------------------------------------------------

def sparse_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, sets: Sequence[Sequence[int]],
                     block: int, scale: float, qbs: Optional[Sequence[int]] = None) -> np.ndarray:
    """A(Q, K, V, S) = Softmax(Q K^T s + M_S) V with M_S = 0 on the selected key blocks
    (and j <= i), -inf elsewhere (Eq. 1).  Row i of query block qb attends to
    {j : floor(j / B) in S(qb), j <= i}.  Computes the rows of the query blocks
    `qbs` (all if None); other rows are left 0.  Returns float64 [n, d]."""
    n, d = q.shape
    out = np.zeros((n, v.shape[1]))
    for qb in (range(len(sets)) if qbs is None else qbs):
        rows = np.arange(qb * block, min((qb + 1) * block, n))
        keys = np.concatenate([np.arange(J * block, min((J + 1) * block, n)) for J in sets[qb]])
        z = (q[rows] @ k[keys].T) * scale
        z[keys[None, :] > rows[:, None]] = -np.inf
        z = z - z.max(axis=1, keepdims=True)
        e = np.exp(z)
        out[rows] = (e / e.sum(axis=1, keepdims=True)) @ v[keys]
    return out


def dense_causal_sets(nb: int) -> List[List[int]]:
    return [list(range(qb + 1)) for qb in range(nb)]


# ----------------------------------------------------------------------------
# FlexPrefill comparator (App. A): JSD pattern search and gamma-coverage VS selection
# ----------------------------------------------------------------------------

def js_distance(p: np.ndarray, q: np.ndarray) -> float:
    """D_JS = sqrt(KL(p || m) / 2 + KL(q || m) / 2) with m = (p + q) / 2 (App. A,
    pattern search).  Natural logarithms; terms with a zero numerator are 0.
    Reading: the square root is taken, as the listing writes it (a distance)."""
    p = np.asarray(p, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    m = 0.5 * (p + q)

    def kl(a, b):
        nz = a > 0
        return float(np.sum(a[nz] * np.log(a[nz] / b[nz])))

    return math.sqrt(max(0.5 * kl(p, m) + 0.5 * kl(q, m), 0.0))


def pooled_estimate(q: np.ndarray, k: np.ndarray, block: int, scale: float) -> np.ndarray:
    """a_bar = Softmax(pool(Q_hat) pool(K)^T s) over the N_b key blocks (App. A, pattern
    search): Q_hat is the last b = min(B, n) queries pooled to one row (mean), K is
    pooled per block (mean; a partial last block over its own rows).  Every key
    block lies at or before Q_hat's block, so no mask applies."""
    n = q.shape[0]
    b = min(block, n)
    qp = q[n - b:].mean(axis=0)
    z = (pool_blocks(k, block) @ qp) * scale
    e = np.exp(z - z.max())
    return e / e.sum()


def jsd_score(q: np.ndarray, k: np.ndarray, p_v: np.ndarray, block: int, scale: float) -> float:
    """The pattern-search score of App. A: D_JS(a_hat, a_bar), where a_hat is the
    per-query mean of the proxy attention sum-pooled over key blocks -- exactly the
    vertical block score p_v of Alg. 3 (each proxy row sums to 1, divided by b) --
    and a_bar the pooled estimate."""
    return js_distance(p_v, pooled_estimate(q, k, block, scale))


def route_jsd(score: float, tau: float) -> int:
    """VS iff D_JS >= tau (App. A), compared in float32."""
    return ROUTE_VS if np.float32(score) >= np.float32(tau) else ROUTE_PE


def vs_select_gamma(p: np.ndarray, gamma: float, k_min: int) -> List[int]:
    """FlexPrefill's VS index selection for one direction (App. A): sort the block
    scores descending and keep the shortest prefix whose cumulative mass reaches
    gamma; k = min(max(that length, k_min), N_b).

    Readings: the scores are the block scores p_d of Alg. 3 (they already sum to
    1, the listing's normalisation); order (p desc, block index asc) on the
    float32 values; float64 cumulative sum against float32(gamma); all blocks if
    it never reaches gamma; k_min as in Alg. 3; N_b <= 2 selects nothing extra.
    Returns the selected block indices, ascending."""
    nb = len(p)
    if nb <= 2:
        return []
    p32 = np.asarray(p, dtype=np.float32)
    order = sorted(range(nb), key=lambda J: (-float(p32[J]), J))
    csum = np.cumsum(p32[order].astype(np.float64))
    hit = np.nonzero(csum >= np.float64(np.float32(gamma)))[0]
    c = int(hit[0]) + 1 if len(hit) else nb
    kd = min(max(c, k_min), nb)
    return sorted(order[:kd])


# ----------------------------------------------------------------------------
# Whole path, per head and per layer (Alg. 1)
# ----------------------------------------------------------------------------

@dataclass
class HeadResult:
    route: int
    c_struct: float
    p_v: np.ndarray
    p_s: np.ndarray
    S_v: List[int] = field(default_factory=list)
    S_s: List[int] = field(default_factory=list)
    pe_pairs: Optional[list] = None
    pe_info: Optional[dict] = None
    A_tilde: Optional[np.ndarray] = None
    sets: List[List[int]] = field(default_factory=list)
    out: Optional[np.ndarray] = None
    jsd: Optional[float] = None


def crisp_head(q: np.ndarray, k: np.ndarray, v: Optional[np.ndarray], block: int, params: Params,
               attend: bool = True, qbs: Optional[Sequence[int]] = None) -> HeadResult:
    """Alg. 1 for one query head: PatSearch -> VSIndex or PEIndex -> A(Q, K, V, S)."""
    n, d = q.shape
    nb = n_blocks(n, block)
    s = params.scale(d)
    ahat = proxy_attention(q, k, block, s)
    cs = c_struct(ahat, n, params.w_sink, params.w_local)
    _, _, p_v, p_s = vs_scores(ahat, n, block)
    if params.route_mode == "jsd":
        res = HeadResult(route=ROUTE_PE, c_struct=cs, p_v=p_v, p_s=p_s)
        res.jsd = jsd_score(q, k, p_v, block, s)
        res.route = route_jsd(res.jsd, params.tau_jsd)
    else:
        res = HeadResult(route=route(cs, params.tau_proxy), c_struct=cs, p_v=p_v, p_s=p_s)
    if res.route == ROUTE_VS:
        km = params.k_min(block)
        if params.vs_mode == "gamma":
            res.S_v = vs_select_gamma(p_v, params.gamma, km)
            res.S_s = vs_select_gamma(p_s, params.gamma, km)
        else:
            for p in (p_v, p_s):   # R20: the residual is the inner-block mass
                if nb > 2:
                    assert abs(vs_floor(p, params.alpha)[0] - p[1:nb - 1].sum()) <= 1e-6
            res.S_v = vs_select(p_v, params.alpha, km, params.floor_mode)
            res.S_s = vs_select(p_s, params.alpha, km, params.floor_mode)
        res.sets = vs_block_sets(res.S_v, res.S_s, nb)
    else:
        At = pe_scores(q, k, block, s)
        pairs, _, info = pe_select(At, params.gamma)
        res.A_tilde, res.pe_pairs, res.pe_info = At, pairs, info
        res.sets = pe_block_sets(pairs, nb)
    if attend and v is not None:
        res.out = sparse_attention(q, k, v, res.sets, block, s, qbs)
    return res


def crisp_layer(Q: np.ndarray, K: np.ndarray, V: Optional[np.ndarray], block: int, params: Params,
                heads: Optional[Sequence[int]] = None, attend: bool = True,
                qbs: Optional[Dict[int, Sequence[int]]] = None) -> Dict[int, HeadResult]:
    """Alg. 1 over the query heads of a GQA layer: head h uses KV head h // (H_q / H_kv)."""
    Hq, Hkv = Q.shape[0], K.shape[0]
    G = Hq // Hkv
    out = {}
    for h in (range(Hq) if heads is None else heads):
        g = h // G
        out[h] = crisp_head(Q[h], K[g], None if V is None else V[g], block, params, attend,
                            None if qbs is None else qbs.get(h))
    return out
