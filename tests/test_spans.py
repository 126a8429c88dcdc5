"""The native reference selection (rac_span_index_* / rac_span_select in
librac.so, host code) against the brute-force oracle of oracle/spans.py.

Random streams use a small vocabulary and copy stretches of earlier requests
into later ones, so windows repeat often, more than eight occurrences of a
window are common, equal-length candidates compete on recency, and spans end
at the end of either sequence.  No GPU is involved.
"""
from __future__ import annotations

import os

import numpy as np
import pytest

import paper_2608_04991_amd as rac
from oracle.spans import select_spans
from tests import test_oracle_spans as pins


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(rac.library_path()):
        pytest.fail("librac.so is not built; run __graft_entry__.build()")


def _native(hist, tokens, window):
    ix = rac.SpanIndex(window)
    for tr, base in hist:
        ix.add(np.asarray(tr, np.int32), base)
    out, cov = ix.select(np.asarray(tokens, np.int32))
    ix.close()
    return out.tolist(), cov


def _agent_stream(rng, n_req, length, vocab):
    """Requests that share a system prompt, reuse stretches of earlier
    requests (tool schemas, earlier turns) and add fresh tokens."""
    system = rng.integers(0, vocab, rng.integers(0, length // 3 + 1)).tolist()
    reqs = []
    for _ in range(n_req):
        r = list(system)
        while len(r) < length:
            if reqs and rng.random() < 0.5:
                src = reqs[rng.integers(0, len(reqs))]
                a = int(rng.integers(0, len(src)))
                r += src[a:a + int(rng.integers(1, 40))]
            else:
                r += rng.integers(0, vocab, int(rng.integers(1, 12))).tolist()
        reqs.append(r[:length])
    return reqs


@pytest.mark.parametrize("seed,window,vocab", [(0, 4, 6), (1, 2, 3), (2, 8, 20), (3, 1, 5), (4, 16, 4),
                                               (5, 3, 50)])
def test_native_selection_matches_the_oracle(seed, window, vocab):
    rng = np.random.default_rng(seed)
    reqs = _agent_stream(rng, 7, 300, vocab)
    hist, base = [], 0
    for r in reqs[:-1]:
        hist.append((r, base))
        base += len(r) + int(rng.integers(0, 5))
    want, spans = select_spans(hist, reqs[-1], window)
    got, cov = _native(hist, reqs[-1], window)
    assert got == want
    assert cov == sum(1 for v in want if v >= 0)
    if window <= 4:
        assert spans, "the stream should produce spans"


def test_native_selection_on_the_hand_made_cases():
    cases = [
        ([([5, 6, 7, 8, 9, 10], 100)], [5, 6, 7, 8, 9, 10], 3),
        ([([1, 2, 3, 4, 5, 0], 0), ([1, 2, 3, 9], 10)], [1, 2, 3, 4, 5, 7], 3),
        ([([1, 2, 3, 8], 0), ([7, 1, 2, 3, 9], 20)], [1, 2, 3, 5], 3),
        ([([1, 2, 3, 0, 1, 2, 3, 6], 40)], [1, 2, 3, 7], 3),
        ([([1, 2, 3, 4, 0, 50, 51, 52], 0), ([2, 3, 4, 50, 51, 52, 53], 100)], [1, 2, 3, 4, 50, 51, 52, 9], 3),
        ([([1, 2, 9, 1, 2], 0)], [1, 2, 3, 1, 2], 3),
        ([([1, 2, 3, 4], 0)] + [([1, 2, 0], 10 * (r + 1)) for r in range(8)], [1, 2, 3, 4], 2),
        ([([1, 2, 3], 7)], [1, 2, 3, 4, 1, 2, 3], 2),
        ([], [1, 2, 3], 2),
        ([([1, 2], 0)], [], 2),
    ]
    for hist, tokens, w in cases:
        assert _native(hist, tokens, w)[0] == select_spans(hist, tokens, w)[0], (hist, tokens, w)
    # the oracle's own pins still hold (they are what fixes these answers)
    pins.test_only_the_eight_most_recent_occurrences_are_candidates()


def test_each_window_content_keeps_its_own_occurrences():
    """Occurrences of other windows never count against a window's eight:
    nine occurrences of [1, 1] leave the single [7, 7] occurrence indexed.
    (Entries under one hash value are told apart by their tokens, so a true
    hash collision would be handled the same way; none is constructed here.)"""
    w = 2
    hist = [([7, 7, 3, 3], 0)] + [([1, 1], 10 * (r + 1)) for r in range(9)]
    got, _ = _native(hist, [7, 7, 3, 3], w)
    assert got == [0, 1, 2, 3]


def test_span_index_errors():
    assert rac.library().rac_span_index_create(0) is None
    assert rac.library().rac_span_index_create(4097) is None
    ix = rac.SpanIndex(4)
    with pytest.raises(rac.RacError):
        ix.add(np.zeros(10, np.int32), -1)
    with pytest.raises(rac.RacError):
        ix.add(np.zeros(10, np.int32), 2 ** 31 - 5)
    L = rac.library()
    assert L.rac_span_select(None, None, 0, None, None) == 1
    assert L.rac_span_select(ix._h, None, 5, None, None) == 1
    out, cov = ix.select(np.zeros(0, np.int32))
    assert out.size == 0 and cov == 0
    ix.close()
