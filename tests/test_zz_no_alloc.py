"""pvs_scores_noalloc (the entry point that allocates nothing) against
pvs_scores, through the C ABI: two calls in a row, the second smaller, and
the size limit."""
import numpy as np
import pytest

from paper_2608_07152_amd import datagen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    from paper_2608_07152_amd import eahr
    eahr.load()
    return eahr


def test_noalloc_scores_equal_pvs_scores(E):
    w = datagen.workload("tiny", n=70000, d=128)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=3)
    idx = E.pvs_build(x)
    st = E.pvs_open(idx, q)
    rng = np.random.default_rng(5)
    big = rng.integers(0, w.n, E.NOALLOC_MAX_ROWS)          # the largest call
    small = rng.integers(0, w.n, 1000)
    for b, rows in ((2, big), (0, small)):
        got = E.pvs_scores_noalloc(st, b, rows)
        want = E.pvs_scores(st, b, rows)
        assert got.view(np.int32).tolist() == want.view(np.int32).tolist()   # bit for bit
    # the second call left the first call's larger tail in the array; a third
    # call of another query still returns exactly its own scores
    got = E.pvs_scores_noalloc(st, 1, small[:7])
    assert np.array_equal(got.view(np.int32), E.pvs_scores(st, 1, small[:7]).view(np.int32))
    assert len(E.pvs_scores_noalloc(st, 1, small[:0])) == 0
    with pytest.raises(E.EahrError) as ei:
        E.pvs_scores_noalloc(st, 0, np.zeros(E.NOALLOC_MAX_ROWS + 1, np.int64))
    assert ei.value.code == E.EAHR_E_RANGE
    with pytest.raises(E.EahrError) as ei:
        E.pvs_scores_noalloc(st, 0, np.array([w.n], np.int64))
    assert ei.value.code == E.EAHR_E_INVALID
    st.close()
    idx.free()
