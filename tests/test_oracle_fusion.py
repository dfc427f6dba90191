"""Pins of the complete-list weighted RRF oracle and the certification
reference (Sec. 2.1, Sec. 2.2, Sec. 3.4 / 4.2 controlled rank streams)."""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import certify, rrf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_g_closed_forms():
    assert rrf.g(1, 1, 60) == Fraction(1, 60)
    assert rrf.g(7, 1, 60) == Fraction(1, 66)
    assert rrf.g(1, 2, 60) == Fraction(2, 119)       # 1 / (1/2 + 59)
    assert rrf.g(5, 0, 60) == 0
    assert rrf.g(3, 1, 1) == Fraction(1, 3)


def test_identical_lists_give_common_prefix():
    rng = np.random.default_rng(1)
    lst = rng.permutation(500)
    assert rrf.rrf_topk([lst, lst], [1, 1], 60, 20) == list(lst[:20])


def test_reversed_lists_alternate_ends_with_id_ties():
    n = 101
    rng = np.random.default_rng(4)
    lst = rng.permutation(n)
    rev = lst[::-1]
    got = rrf.rrf_topk([lst, rev], [1, 1], 60, 10)
    # F(item at rank r of lst) = g(r) + g(n + 1 - r): mirror pairs tie exactly
    want = []
    for r in range(1, 6):
        a, b = int(lst[r - 1]), int(lst[n - r])
        want += sorted([a, b])
    assert got == want


def test_zero_weight_gives_single_channel():
    rng = np.random.default_rng(9)
    a, b = rng.permutation(300), rng.permutation(300)
    assert rrf.rrf_topk([a, b], [1, 0], 60, 15) == list(a[:15])
    assert rrf.rrf_topk([a, b], [0, 2], 60, 15) == list(b[:15])


def test_no_zero_score_padding():
    dense_list = np.arange(100)
    sparse_list = np.array([42, 7, 99])
    assert rrf.rrf_topk([dense_list, sparse_list], [0, 1], 60, 20) == [42, 7, 99]


def test_rank_scaled_weight_changes_order():
    # x = 10: dense rank 1, sparse rank 3; y = 20: dense rank 3, sparse rank 1.
    # Rank-scaled weights divide the rank, so w_dense = 2 shrinks the dense gap:
    # F(x) = 1/(1/2+59) + 1/(3+59) = 0.032936 < F(y) = 1/(3/2+59) + 1/60 = 0.033196.
    # (Weights in the numerator would order them the other way: 2/60 + 1/62 > 2/62 + 1/60.)
    d = [10, 11, 20]
    s = [20, 12, 10]
    assert rrf.rrf_topk([d, s], [2, 1], 60, 2) == [20, 10]
    assert rrf.rrf_topk([d, s], [1, 2], 60, 2) == [10, 20]


@pytest.mark.parametrize("seed", range(30))
def test_screened_topk_equals_exhaustive(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60))
    a = rng.permutation(n)
    b = rng.permutation(n)[: int(rng.integers(0, n + 1))]
    if seed % 3 == 0:
        b = a[::-1].copy()
    wts = [int(rng.integers(0, 3)), int(rng.integers(1, 3))]
    k = int(rng.choice([1, 2, 60]))
    K = int(rng.integers(1, 25))
    assert rrf.rrf_topk([a, b], wts, k, K) == rrf.rrf_topk_exact([a, b], wts, k, K)


# ---------------------------------------------------------------- certification
def _completions(prefix, pool, open_):
    """Every list that extends ``prefix`` with distinct items of ``pool``."""
    if not open_:
        yield list(prefix)
        return
    rest = [x for x in pool if x not in prefix]
    for r in range(0, len(rest) + 1):
        for tail in itertools.permutations(rest, r):
            yield list(prefix) + list(tail)


@pytest.mark.parametrize("seed", range(25))
def test_certified_prefix_holds_in_every_completion(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(2, 5))
    items = list(range(n))
    a = list(rng.permutation(n))
    b = list(rng.permutation(n)[: int(rng.integers(1, n + 1))])
    wts = [int(rng.integers(1, 3)), int(rng.integers(0, 3))]
    k = int(rng.choice([1, 2, 3]))
    K = int(rng.integers(1, n + 1))
    da, db = int(rng.integers(0, n + 1)), int(rng.integers(0, len(b) + 1))
    A, resolved = certify.certify_ref([a, b], wts, k, K, [da, db])
    # the reference sees only the prefixes and whether each list is complete
    comps_a = list(_completions(a[:da], items, da < len(a)))
    comps_b = list(_completions(b[:db], items, db < len(b)))
    for ca in comps_a:
        for cb in comps_b:
            T = rrf.rrf_topk_exact([ca, cb], wts, k, K)
            assert T[: len(A)] == A
            if resolved:
                assert T == A
    if da == len(a) and db == len(b):
        assert resolved and A == rrf.rrf_topk_exact([a, b], wts, k, K)


def test_identical_lists_resolve_exactly_at_depth_K():
    rng = np.random.default_rng(3)
    lst = list(rng.permutation(200))
    K = 10
    for d in range(0, K):
        assert not certify.certify_ref([lst, lst], [1, 1], 60, K, [d, d])[1]
    A, ok = certify.certify_ref([lst, lst], [1, 1], 60, K, [K, K])
    assert ok and A == lst[:K]


def test_reversed_lists_never_resolve_before_exhaustion():
    rng = np.random.default_rng(8)
    n = 48
    lst = list(rng.permutation(n))
    rev = lst[::-1]
    for d in range(0, n):
        A, ok = certify.certify_ref([lst, rev], [1, 1], 60, 5, [d, d])
        assert not ok and A == []
    A, ok = certify.certify_ref([lst, rev], [1, 1], 60, 5, [n, n])
    assert ok and A == rrf.rrf_topk_exact([lst, rev], [1, 1], 60, 5)


def _first_resolved(a, b, K, step, k=60):
    n = max(len(a), len(b))
    d = step
    while True:
        A, ok = certify.certify_ref([a, b], [1, 1], k, K, [d, d])
        if ok:
            return d, A
        if d >= n:
            return None, A
        d = min(n, d + step)


def _block_permuted(rng, lst, block):
    """Permute uniformly inside every contiguous block of ``block`` items."""
    lst = np.asarray(lst)
    order = np.lexsort((rng.random(len(lst)), np.arange(len(lst)) // block))
    return lst[order]


def test_controlled_correlated_streams_resolve_at_depth_32():
    g = json.load(open(os.path.join(GOLDEN, "e5_controlled_streams.json")))
    K, step, block = g["K"], g["check_every"], g["block"]
    want = g["outcomes"]["correlated_32_block_permutation"]["first_resolved_depth"]
    for n in g["sizes"]:
        for seed in g["seeds"]:
            rng = np.random.default_rng(seed)
            a = rng.permutation(n)
            b = _block_permuted(rng, a, block)
            d, A = _first_resolved(a, b, K, step)
            assert d == want
            assert A == rrf.rrf_topk([a, b], [1, 1], 60, K)


def test_controlled_anticorrelated_streams_exhaust_both():
    g = json.load(open(os.path.join(GOLDEN, "e5_controlled_streams.json")))
    assert g["outcomes"]["anti_correlated_reversal"]["both_lists_exhausted"]
    for n, seed in ((64, 1729), (96, 2027), (80, 65537)):
        rng = np.random.default_rng(seed)
        a = rng.permutation(n)
        d, A = _first_resolved(a, a[::-1], g["K"], g["check_every"])
        assert d == n
        assert A == rrf.rrf_topk_exact([a, a[::-1]], [1, 1], 60, g["K"])


def test_all_tied_streams_resolve_at_first_checkpoint_past_K():
    n = 1000
    ids = np.arange(n)      # equal scores: both lists are identifier order
    d, A = _first_resolved(ids, ids, 20, 16)
    assert d == 32 and A == list(range(20))
