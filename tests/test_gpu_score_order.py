"""The authoritative float32 score follows one fixed order (reading R6 of the
dense channel): a group of 16 lanes scores a row; lane j takes the float4
chunks c = 16 t + j of the row and the query and accumulates their products
with a fused multiply-add in (t, x, y, z, w) order, then the 16 lane sums are
added as a balanced pairwise tree (partners j ^ 1, j ^ 2, j ^ 4, j ^ 8).
This test recomputes that order on the CPU with exactly rounded float32
operations and requires the GPU's scores (pvs_scores, and the ranks pvs_next
emits) to match bit for bit.  Rows of more than 1,024 floats are scored in
segments on the device; the order is the same."""
from fractions import Fraction

import numpy as np
import pytest

from paper_2608_07152_amd import datagen

pytestmark = pytest.mark.gpu

F32 = np.float32


def _round32(fr: Fraction) -> np.float32:
    """Float32 nearest to an exact rational, ties to even."""
    f = F32(float(fr))
    cands = [np.nextafter(f, F32(-np.inf)), f, np.nextafter(f, F32(np.inf))]
    return min(cands, key=lambda c: (abs(Fraction(float(c)) - fr),
                                     int(np.array(c, F32).view(np.int32)) & 1))


def _fma32(a, b, c) -> np.float32:
    return _round32(Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c)))


def _add32(a, b) -> np.float32:
    return _round32(Fraction(float(a)) + Fraction(float(b)))


def r6_score(q: np.ndarray, v: np.ndarray) -> np.float32:
    d = len(q)
    df = (d + 3) // 4 * 4
    qp = np.zeros(df, F32)
    vp = np.zeros(df, F32)
    qp[:d] = q
    vp[:d] = v
    df4 = df // 4
    lanes = []
    for j in range(16):
        acc = F32(0)
        c = j
        while c < df4:
            for i in range(4):
                acc = _fma32(qp[4 * c + i], vp[4 * c + i], acc)
            c += 16
        lanes.append(acc)
    for off in (1, 2, 4, 8):
        lanes = [_add32(lanes[j], lanes[j ^ off]) for j in range(16)]
    return lanes[0]


@pytest.fixture(scope="module")
def E():
    from paper_2608_07152_amd import eahr
    eahr.load()
    return eahr


@pytest.mark.parametrize("d", [100, 128, 768, 1100])
def test_scores_follow_the_fixed_order_bit_for_bit(E, d):
    w = datagen.workload("tiny", n=300, d=d)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=2)
    idx = E.pvs_build(x)
    st = E.pvs_open(idx, q)
    rng = np.random.default_rng(d)
    rows = np.sort(rng.choice(w.n, size=6, replace=False))
    for b in range(2):
        got = E.pvs_scores(st, b, rows)
        for k, r in enumerate(rows):
            want = r6_score(q[b], x[r])
            assert np.array(got[k], F32).view(np.int32) == np.array(want, F32).view(np.int32), (b, r)
    # the ranks pvs_next emits carry the same scores (rescoring's own code)
    ids, sc, cnt, _ = E.pvs_next(st, 5)
    for b in range(2):
        for k in range(cnt[b]):
            want = r6_score(q[b], x[ids[b, k]])
            assert np.array(sc[b, k], F32).view(np.int32) == np.array(want, F32).view(np.int32)


@pytest.mark.parametrize("d", [128, 768])
@pytest.mark.parametrize("B", [1, 2, 60])
def test_rescored_scores_follow_the_fixed_order_bit_for_bit(E, d, B):
    """The emitted scores come from rescoring, which holds a one-query scan's
    query row in registers, reads the query rows of a scan from LDS when they
    fit (two queries at d = 128 and 768, sixty at d = 128) and from memory
    otherwise (sixty at d = 768): every path follows the fixed order."""
    w = datagen.workload("tiny", n=400, d=d)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=B)
    idx = E.pvs_build(x)
    st = E.pvs_open(idx, q)
    ids, sc, cnt, _ = E.pvs_next(st, 4)
    for b in sorted({0, B // 2, B - 1}):
        assert cnt[b] == 4
        for k in range(cnt[b]):
            want = r6_score(q[b], x[ids[b, k]])
            assert np.array(sc[b, k], F32).view(np.int32) == np.array(want, F32).view(np.int32), (b, k)
