"""Plain reference of the prefill-uplink reference selection (subsection
"Repeated-Span Retrieval for Prefill Uplinks", Eq. prefill-reference-selection).

TEST INFRASTRUCTURE ONLY: the test suite is the only caller; the product
library never imports it and it imports nothing from the product.

Written from the definition, by brute force:
  * the index holds every w-token window of the earlier requests, grouped by
    the exact window content (a hash bucket is read as one window content);
    each group keeps its `keep` most recent occurrences, recency being the
    request order and then the position inside the request;
  * at position i of the current prompt, a candidate is an indexed
    occurrence (r, j) of the window x[i:i+w], extended forward to its longest
    exact match L >= w;
  * the chosen candidate is the lexicographic maximum of (L, recency); the
    scan then moves to i + L, or to i + 1 when there is no candidate;
  * a covered position i0 + o takes store row base_r + j + o as its
    reference, every other position -1 (encoded without a reference).
"""
from __future__ import annotations


def select_spans(history, tokens, window, keep=8):
    """history: [(tokens_r, store_row0_r), ...] in request order.
    Returns (ref_rows, spans): ref_rows[i] is the store row of position i's
    reference or -1; spans lists the chosen (i, r, j, L)."""
    occ = {}
    for r, (tr, _) in enumerate(history):
        for j in range(len(tr) - window + 1):
            lst = occ.setdefault(tuple(tr[j:j + window]), [])
            lst.append((r, j))
            if len(lst) > keep:
                lst.pop(0)
    n = len(tokens)
    out = [-1] * n
    spans = []
    i = 0
    while i < n:
        best = None
        if i + window <= n:
            for r, j in occ.get(tuple(tokens[i:i + window]), []):
                tr = history[r][0]
                L = window
                while i + L < n and j + L < len(tr) and tokens[i + L] == tr[j + L]:
                    L += 1
                cand = (L, r, j)
                if best is None or cand > best:
                    best = cand
        if best is None:
            i += 1
            continue
        L, r, j = best
        for o in range(L):
            out[i + o] = history[r][1] + j + o
        spans.append((i, r, j, L))
        i += L
    return out, spans
