"""The parity checks themselves, on the CPU: a check that cannot fail proves nothing, so
each one is run on the oracle's own answer (it must pass) and on answers with a planted
mistake (it must fail)."""
import numpy as np
import pytest

from oracle import crisp_oracle as O
from tests import parity as PR
from tests.helpers import bf16_round, random_head

S128 = 1.0 / np.sqrt(128.0)


def _csr(sets):
    rp = np.zeros(len(sets) + 1, np.int64)
    for qb, s in enumerate(sets):
        rp[qb + 1] = rp[qb] + len(s)
    ci = np.concatenate([np.asarray(s, np.int64) for s in sets])
    return rp, ci


def _pe_sets(nb, pairs):
    sets = [{0, qb} for qb in range(nb)]
    for qb, kb in pairs:
        sets[qb].add(kb)
    return [sorted(s) for s in sets]


def _pe_case(n, block, seed, scale):
    q, k, _ = random_head(n, seed=seed, scale=scale)
    At = O.pe_scores(q, k, block, S128)
    pairs, kstar, _ = O.pe_select(At, 0.95)
    return At, pairs, kstar


@pytest.mark.parametrize("n,block,seed,scale", [(4096, 128, 3, 4.0), (2048, 64, 4, 2.0), (3000, 128, 5, 8.0)])
def test_pe_threshold_accepts_the_oracle_and_rejects_planted_mistakes(n, block, seed, scale):
    At, pairs, kstar = _pe_case(n, block, seed, scale)
    nb = At.shape[0]
    sets = _pe_sets(nb, pairs)
    rp, ci = _csr(sets)
    got_k, _ = PR.check_pe_threshold(rp, ci, At, 0.95, where="oracle")
    assert got_k == kstar
    # the largest non-forced selected pair dropped
    free = [(a, c) for a, c in pairs if c not in (0, a)]
    top = max(free, key=lambda p: At[p])
    bad = [sorted(set(s) - ({top[1]} if qb == top[0] else set())) for qb, s in enumerate(sets)]
    with pytest.raises(AssertionError, match="not selected"):
        PR.check_pe_threshold(*_csr(bad), At, 0.95)
    # the smallest unselected causal pair added
    chosen = set(pairs)
    rest = [(a, c) for a in range(nb) for c in range(1, a) if (a, c) not in chosen]
    low = min(rest, key=lambda p: At[p])
    bad = [sorted(set(s) | ({low[1]} if qb == low[0] else set())) for qb, s in enumerate(sets)]
    with pytest.raises(AssertionError, match="below"):
        PR.check_pe_threshold(*_csr(bad), At, 0.95)
    # a pair above the diagonal, and a missing forced block
    bad = [list(s) for s in sets]
    bad[1] = sorted(set(bad[1]) | {2})
    with pytest.raises(AssertionError, match="above the diagonal"):
        PR.check_pe_threshold(*_csr(bad), At, 0.95)
    bad = [list(s) for s in sets]
    bad[5] = [c for c in bad[5] if c != 5]
    with pytest.raises(AssertionError, match="forced"):
        PR.check_pe_threshold(*_csr(bad), At, 0.95)


def test_pe_threshold_on_flat_head_ties():
    """Flat head (P4): A_tilde is constant along each row, so the cut falls inside a row of
    equal values; the oracle's flat-index tie order is one valid answer and any other
    choice of the same number of tied pairs is too (they lie in the E4 band)."""
    nb, block = 40, 128
    q = np.zeros((nb * block, 128))
    k = bf16_round(np.random.default_rng(6).standard_normal((nb * block, 128)))
    At = O.pe_scores(q, k, block, S128)
    pairs, kstar, _ = O.pe_select(At, 0.95)
    sets = _pe_sets(nb, pairs)
    PR.check_pe_threshold(*_csr(sets), At, 0.95)
    cut_row = max(a for a, _ in pairs)
    taken = [c for a, c in pairs if a == cut_row]
    alt = sorted(set(range(cut_row + 1)) - set(taken))[: len(taken)]   # the other tied pairs
    sets[cut_row] = sorted({0, cut_row} | set(alt))
    PR.check_pe_threshold(*_csr(sets), At, 0.95)
    # a whole earlier row dropped is outside the band
    sets[3] = [0, 3]
    with pytest.raises(AssertionError, match="not selected"):
        PR.check_pe_threshold(*_csr(sets), At, 0.95)
