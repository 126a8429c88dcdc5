"""Pins of the reference-selection oracle (oracle/spans.py) on hand-made
token streams whose answer follows from the selection rule directly: longest
exact span first, recency breaks ties, the scan jumps past a chosen span,
spans shorter than the window never count, and only the eight most recent
occurrences of a window are candidates."""
from __future__ import annotations

from oracle.spans import select_spans


def test_identical_prompt_is_one_span():
    hist = [([5, 6, 7, 8, 9, 10], 100)]
    out, spans = select_spans(hist, [5, 6, 7, 8, 9, 10], window=3)
    assert out == [100, 101, 102, 103, 104, 105]
    assert spans == [(0, 0, 0, 6)]


def test_nothing_shared_means_no_reference():
    out, spans = select_spans([([1, 2, 3, 4], 0)], [4, 3, 2, 1], window=2)
    assert out == [-1, -1, -1, -1] and spans == []


def test_longest_span_wins_then_recency():
    # request 0 matches 5 tokens at position 0, request 1 only 3
    hist = [([1, 2, 3, 4, 5, 0], 0), ([1, 2, 3, 9], 10)]
    out, spans = select_spans(hist, [1, 2, 3, 4, 5, 7], window=3)
    assert spans == [(0, 0, 0, 5)] and out == [0, 1, 2, 3, 4, -1]
    # equal lengths: the later request is the more recent one
    hist = [([1, 2, 3, 8], 0), ([7, 1, 2, 3, 9], 20)]
    out, spans = select_spans(hist, [1, 2, 3, 5], window=3)
    assert spans == [(0, 1, 1, 3)] and out == [21, 22, 23, -1]
    # equal lengths inside one request: the later position is more recent
    hist = [([1, 2, 3, 0, 1, 2, 3, 6], 40)]
    out, spans = select_spans(hist, [1, 2, 3, 7], window=3)
    assert spans == [(0, 0, 4, 3)] and out == [44, 45, 46, -1]


def test_scan_jumps_past_a_span_and_restarts():
    hist = [([1, 2, 3, 4, 0, 50, 51, 52], 0), ([2, 3, 4, 50, 51, 52, 53], 100)]
    # at 0 the span [1,2,3,4] (L=4) is taken; the longer [2,3,4,50,51,52]
    # starting at 1 lies inside it and is never considered; at 4 the scan
    # finds [50,51,52] in both requests (L=3 each) and takes the more recent
    out, spans = select_spans(hist, [1, 2, 3, 4, 50, 51, 52, 9], window=3)
    assert spans == [(0, 0, 0, 4), (4, 1, 3, 3)]
    assert out == [0, 1, 2, 3, 103, 104, 105, -1]


def test_matches_shorter_than_the_window_do_not_count():
    hist = [([1, 2, 9, 1, 2], 0)]
    out, spans = select_spans(hist, [1, 2, 3, 1, 2], window=3)
    assert spans == [] and out == [-1] * 5


def test_only_the_eight_most_recent_occurrences_are_candidates():
    # the window [1, 2] occurs in nine requests; only the oldest continues
    # with 3, 4 (a longer span), but it has been dropped from the index
    hist = [([1, 2, 3, 4], 0)] + [([1, 2, 0], 10 * (r + 1)) for r in range(8)]
    out, spans = select_spans(hist, [1, 2, 3, 4], window=2)
    # (after the two-token span the scan restarts at [3, 4], still indexed)
    assert spans == [(0, 8, 0, 2), (2, 0, 2, 2)] and out == [80, 81, 2, 3]
    # with one occurrence fewer the oldest is still indexed and wins
    out, spans = select_spans(hist[:8], [1, 2, 3, 4], window=2)
    assert spans == [(0, 0, 0, 4)] and out == [0, 1, 2, 3]


def test_span_extends_to_the_end_of_either_sequence():
    hist = [([1, 2, 3], 7)]
    out, spans = select_spans(hist, [1, 2, 3, 4, 1, 2, 3], window=2)
    assert spans == [(0, 0, 0, 3), (4, 0, 0, 3)]
    assert out == [7, 8, 9, -1, 7, 8, 9]
