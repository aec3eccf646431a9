"""CPU checks of the L2 model's two replacement policies (tests/l2_model.py)
against definitions: LRU on cyclic streams, and Belady's MIN against an
exhaustive search over eviction choices on tiny streams."""
import itertools

import numpy as np
import pytest

import l2_model  # noqa: E402


def test_lru_cyclic_streams():
    K = 4
    fits = [0, 1, 2, 3] * 5                 # working set == K: only cold misses
    assert l2_model.lru_hits(fits, K) == len(fits) - 4
    thrash = [0, 1, 2, 3, 4] * 5            # K + 1 lines in a cycle: LRU never hits
    assert l2_model.lru_hits(thrash, K) == 0


def _best_hits(seq, K):
    """Exhaustive: the most hits any eviction sequence reaches."""
    best = 0

    def go(i, cache, hits):
        nonlocal best
        if i == len(seq):
            best = max(best, hits)
            return
        c = seq[i]
        if c in cache:
            go(i + 1, cache, hits + 1)
        elif len(cache) < K:
            go(i + 1, cache | {c}, hits)
        else:
            for v in cache:
                go(i + 1, (cache - {v}) | {c}, hits)
    go(0, frozenset(), 0)
    return best


@pytest.mark.parametrize("seed", range(6))
def test_opt_equals_exhaustive_search(seed):
    rng = np.random.default_rng(seed)
    seq = rng.integers(0, 6, size=11).tolist()
    for K in (1, 2, 3):
        assert l2_model.opt_hits(seq, K) == _best_hits(seq, K), (seq, K)
        assert l2_model.opt_hits(seq, K) >= l2_model.lru_hits(seq, K)


def test_opt_on_the_cycle_lru_cannot_serve():
    K = 4
    seq = [0, 1, 2, 3, 4] * 6
    assert l2_model.lru_hits(seq, K) == 0
    assert l2_model.opt_hits(seq, K) > len(seq) // 2
