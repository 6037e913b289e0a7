"""Property tests of the CPU oracle on random shapes (hypothesis): for any length (ragged
or whole blocks), block size, logit scale and parameters, the definitions fix

* the proxy rows: causal, each a probability vector (Alg. 2);
* C_struct in [0, 1]; p_v and p_s probability vectors whose residual r_d is the mass of
  the inner blocks (Alg. 3, Sec. 4.3);
* the VS selection: at least min(k_min, N_b) blocks per direction once N_b > 2, every
  block strictly above the floor kept, and a larger alpha never keeping more;
* the PE cutoff: the kept pairs' A_tilde mass reaches gamma (every pair when gamma = 1),
  and dropping the last kept pair falls short (Alg. 4);
* the block lists: ascending, unique, within [0, qb], always holding 0 and qb;
* the metamorphic case of every block selected (k_min = N_b for VS, gamma = 1 for PE):
  the sparse attention equals float64 causal softmax attention.
"""
import math

import numpy as np
import torch
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import crisp_oracle as O
from tests.helpers import bf16_round

SETTINGS = settings(max_examples=25, deadline=None, suppress_health_check=[HealthCheck.too_slow])


def _head(seed, n, scale, sink):
    rng = np.random.default_rng(seed)
    q = bf16_round(rng.standard_normal((n, 128)) * scale)
    k = bf16_round(rng.standard_normal((n, 128)))
    if sink:  # a strong key 0 for every query: VS-like heads
        k[0] = bf16_round(q.mean(0) * 40.0 / max(np.linalg.norm(q.mean(0)), 1e-9))
    return q, k


shapes = st.tuples(st.sampled_from([64, 128]), st.integers(1, 12), st.integers(0, 127))


@SETTINGS
@given(shape=shapes, seed=st.integers(0, 10_000), scale=st.sampled_from([0.0, 0.05, 0.3, 1.0]),
       sink=st.booleans(), alpha=st.sampled_from([0.5, 1.0, 2.0]), gamma=st.sampled_from([0.5, 0.9, 0.95, 1.0]))
def test_oracle_invariants(shape, seed, scale, sink, alpha, gamma):
    block, nbf, tail = shape
    n = max(1, nbf * block + tail % block)
    nb = O.n_blocks(n, block)
    q, k = _head(seed, n, scale, sink)
    s = 1.0 / math.sqrt(128)
    A = O.proxy_attention(q, k, block, s)
    b = A.shape[0]
    assert b == min(block, n)
    for r in range(b):
        qi = n - b + r
        assert not A[r, qi + 1:].any() and abs(A[r].sum() - 1) < 1e-12
    cs = O.c_struct(A, n, 128, 128)
    assert -1e-12 <= cs <= 1 + 1e-12
    _, _, pv, ps = O.vs_scores(A, n, block)
    for p in (pv, ps):
        assert len(p) == nb and (p >= 0).all() and abs(p.sum() - 1) < 1e-12
        if nb > 2:
            assert abs(max(1 - p[0] - p[nb - 1], 0) - p[1:nb - 1].sum()) < 1e-12
    params = O.Params(alpha=alpha, gamma=gamma)
    k_min = params.k_min(block)
    for p in (pv, ps):
        S = O.vs_select(p, alpha, k_min)
        if nb <= 2:
            assert S == []
            continue
        assert len(S) >= min(k_min, nb) and S == sorted(set(S))
        _, _, thr = O.vs_floor(p, alpha)
        above = {J for J in range(nb) if np.float32(p[J]) > np.float32(thr)}
        assert above <= set(S)
        assert len(O.vs_select(p, alpha * 2, k_min)) <= len(S)
    At = O.pe_scores(q, k, block, s)
    pairs, kstar, info = O.pe_select(At, gamma)
    vals = np.array([np.float32(At[a, c]) for a, c in pairs], dtype=np.float64)
    total = sum(np.float64(np.float32(At[a, c])) for a in range(nb) for c in range(a + 1))
    g = np.float64(np.float32(gamma))
    if gamma == 1.0 and total < g:
        assert kstar == nb * (nb + 1) // 2
    else:
        assert vals.sum() >= g - 1e-9 * max(1.0, g)
        if kstar >= 1:
            assert vals.sum() - vals.min() < g + 1e-9
    for sets in (O.vs_block_sets(O.vs_select(pv, alpha, k_min), O.vs_select(ps, alpha, k_min), nb),
                 O.pe_block_sets(pairs, nb)):
        assert len(sets) == nb
        for qb, row in enumerate(sets):
            assert row == sorted(set(row)) and row[0] == 0 and row[-1] == qb and all(0 <= c <= qb for c in row)


@SETTINGS
@given(shape=shapes, seed=st.integers(0, 10_000), scale=st.sampled_from([0.05, 0.5, 1.5]), sink=st.booleans())
def test_every_block_selected_is_dense_attention(shape, seed, scale, sink):
    block, nbf, tail = shape
    n = max(1, min(nbf, 6) * block + tail % block)
    nb = O.n_blocks(n, block)
    q, k = _head(seed, n, scale, sink)
    v = bf16_round(np.random.default_rng(seed + 1).standard_normal((n, 128)))
    for params in (O.Params(k_min_blocks=nb, tau_proxy=-1.0), O.Params(gamma=1.0, tau_proxy=2.0)):
        r = O.crisp_head(q, k, v, block, params)
        assert sum(len(s) for s in r.sets) == nb * (nb + 1) // 2
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None], torch.from_numpy(v)[None, None],
            is_causal=True, scale=1.0 / math.sqrt(128))[0, 0].numpy()
        assert np.abs(r.out - ref).max() < 1e-10
