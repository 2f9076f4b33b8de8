"""Per-candidate expert routes for the oracle's forced-routing check.

The library records, for a mixture-of-experts model, the experts each layer
kept for each row of the latest prefill (rows = the call's prefix tokens)
and scoring call (rows = candidate body rows in jet_candidate_layout order:
question by question, candidate by candidate, tokens y_{c,1..m-1}). The
oracle runs every candidate as its own sequence x || y_c[1..m-1]; this
assembles that sequence's rows from the two records.
"""
import numpy as np


def body_row0(wl):
    """First body row of each candidate (the documented layout)."""
    m = np.diff(wl.cand_tok_offsets)
    return np.concatenate([[0], np.cumsum(m - 1)]).astype(np.int64)


def candidate_routes(wl, pre, cand, qs):
    """{candidate index within wl.subset(qs): int [L, P + m - 1, k]}."""
    r0 = body_row0(wl)
    out, j = {}, 0
    for q in qs:
        a, b = int(wl.prefix_offsets[q]), int(wl.prefix_offsets[q + 1])
        for c in range(int(wl.q_cand_offsets[q]), int(wl.q_cand_offsets[q + 1])):
            m = int(wl.cand_tok_offsets[c + 1] - wl.cand_tok_offsets[c])
            out[j] = np.concatenate([pre[:, a:b], cand[:, r0[c]:r0[c] + m - 1]], axis=1)
            j += 1
    return out

