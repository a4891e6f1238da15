"""Comparison of GPU outputs with the oracle, with the gating rules of the parity bar.

Token ids, accepted lengths and paths must match bit for bit wherever the
oracle's top-2 cd margin exceeds MARGIN_GATE and no token lies within
BOUNDARY_GATE nats of the plausibility cutoff on every row the oracle's path
visits; log-probabilities and cd scores must agree within ATOL on such rows.
Sampled decisions must match where |u - ratio| > RATIO_GATE * ratio, and
resampled tokens where the draw is more than CDF_GATE (relative to the total)
from every breakpoint of the inverse CDF.
"""
import numpy as np

import oracle

MARGIN_GATE = 1e-3
BOUNDARY_GATE = 1e-4
ATOL = 1e-3
RATIO_GATE = 1e-4
CDF_GATE = 1e-4


def ambiguous_rows(o):
    margin = o["row_stats"][:, oracle.RS_MARGIN]
    return (margin <= MARGIN_GATE) | (o["row_gap"] <= BOUNDARY_GATE)


def compare_rows(g, o, rows, report):
    """Row outputs of GPU rows `rows` against oracle rows (same order)."""
    amb = ambiguous_rows(o) if "row_gap" in o else (o["gap"] <= BOUNDARY_GATE) | (
        o["stats"][:, oracle.RS_MARGIN] <= MARGIN_GATE)
    ostats = o["row_stats"] if "row_stats" in o else o["stats"]
    oargmax = o["row_argmax"] if "row_argmax" in o else o["argmax"]
    gs, ga = g["row_stats"][rows].astype(np.float64), g["row_argmax"][rows]
    # rows with non-finite logits have no meaningful argmax: both sides must be
    # non-finite there, nothing else is compared
    key = [oracle.RS_MAXP, oracle.RS_LSEP, oracle.RS_LSEQ, oracle.RS_LOGZ]
    o_bad = ~np.all(np.isfinite(ostats[:, key]), axis=1)
    g_bad = ~np.all(np.isfinite(gs[:, key]), axis=1)
    assert np.array_equal(o_bad, g_bad), "non-finite rows differ"
    amb = amb | o_bad
    ok = ~amb
    report["rows"] = report.get("rows", 0) + len(rows)
    report["ambiguous_rows"] = report.get("ambiguous_rows", 0) + int(amb.sum())
    bad = np.flatnonzero(ok & (ga != oargmax))
    assert len(bad) == 0, f"argmax differs on rows {np.asarray(rows)[bad][:8]}"
    assert np.array_equal(gs[ok, oracle.RS_COUNT], ostats[ok, oracle.RS_COUNT]), "mask count"
    for k in (oracle.RS_MAXP, oracle.RS_LSEP, oracle.RS_LSEQ, oracle.RS_LOGZ, oracle.RS_TOP1,
              oracle.RS_SIGNAL):
        d = np.abs(gs[ok, k] - ostats[ok, k])
        assert np.all(d <= ATOL), f"row stat {k}: max diff {d.max()}"
    m_o, m_g = ostats[ok, oracle.RS_MARGIN], gs[ok, oracle.RS_MARGIN]
    fin = np.isfinite(m_o)
    assert np.array_equal(np.isfinite(m_g), fin), "margin finiteness"
    assert np.all(np.abs(m_g[fin] - m_o[fin]) <= ATOL), "margin"
    return amb


def compare_diagnostics(g, o, rows, theta, s, V, report):
    """Per-row diagnostics of GPU rows `rows` against the oracle's (same order): the
    expert's top-1 exactly where the oracle's top-2 expert-logit gap exceeds
    MARGIN_GATE; with the untruncated target (theta = 0) D_KL(pi_p||pi_q) within
    ATOL and D_KL(pi_p||pi_CD) = log Z - s D_KL(pi_p||pi_q) within (1+s) ATOL (its
    error is log Z's plus s times the other's); with a mask the divergences are not
    computed (NaN) except D_KL(pi_p||pi_CD) = +inf when the mask leaves out a token."""
    od = o["row_diag"] if "row_diag" in o else o["diag"]
    ostats = o["row_stats"] if "row_stats" in o else o["stats"]
    ga = g["row_argmax_expert"][rows]
    gk = g["row_kl"][rows].astype(np.float64)
    key = [oracle.RS_MAXP, oracle.RS_LSEP, oracle.RS_LSEQ, oracle.RS_LOGZ]
    fin = np.all(np.isfinite(ostats[:, key]), axis=1)
    clear = fin & (od[:, oracle.RD_MARGIN_P] > MARGIN_GATE)
    bad = np.flatnonzero(clear & (ga != od[:, oracle.RD_ARGMAX_P]))
    assert len(bad) == 0, f"expert top-1 differs on rows {np.asarray(rows)[bad][:8]}"
    if theta == 0.0:
        d = np.abs(gk[fin, 0] - od[fin, oracle.RD_KL_PQ])
        assert np.all(d <= ATOL), f"KL(p||q): max diff {d.max()}"
        d = np.abs(gk[fin, 1] - od[fin, oracle.RD_KL_PCD])
        assert np.all(d <= (1 + s) * ATOL), f"KL(p||cd): max diff {d.max()}"
    else:
        assert np.all(np.isnan(gk[:, 0]))
        partial = g["row_stats"][rows, oracle.RS_COUNT] < V
        assert np.all(np.isposinf(gk[partial, 1])) and np.all(np.isnan(gk[~partial, 1]))
        assert np.all(np.isposinf(od[fin & partial, oracle.RD_KL_PCD]))
    report["diag_rows"] = report.get("diag_rows", 0) + int(clear.sum())


def compare_nodes(g, o, parents, amb, report):
    """Draft-token statistics of every node whose parent row is unambiguous."""
    B, N = parents.shape
    gn, on = g["node_stats"].astype(np.float64), o["node_stats"]
    for b in range(B):
        if o["status"][b] != oracle.SEQ_OK:
            continue
        for i in range(1, N):
            r, j = b * N + i, b * N + parents[b, i]
            if amb[j]:
                continue
            assert gn[r, oracle.NS_INMASK] == on[r, oracle.NS_INMASK], f"in_mask node {r}"
            for k in (oracle.NS_LPP, oracle.NS_LPQ, oracle.NS_CD):
                assert abs(gn[r, k] - on[r, k]) <= ATOL, f"node {r} stat {k}: {gn[r, k]} vs {on[r, k]}"
            if np.isinf(on[r, oracle.NS_LPCD]):
                assert np.isneginf(gn[r, oracle.NS_LPCD])
            else:
                assert abs(gn[r, oracle.NS_LPCD] - on[r, oracle.NS_LPCD]) <= ATOL
        assert np.all(np.isnan(gn[b * N]))
    report["nodes"] = report.get("nodes", 0) + B * (N - 1)


def compare_greedy(g, o, parents, amb, report, seqs=None):
    """Sequence outputs: status exact; path, length and next token exact up to the
    first ambiguous row on the oracle's path."""
    B, N = parents.shape
    seqs = range(B) if seqs is None else seqs
    gated = 0
    for b in seqs:
        assert g["status"][b] == o["status"][b], f"status seq {b}"
        if o["status"][b] != oracle.SEQ_OK:
            assert g["accept_len"][b] == 0 and g["next_token"][b] == -1
            assert np.all(g["accept_path"][b] == -1)
            continue
        L, path = int(o["accept_len"][b]), o["accept_path"][b]
        first_amb = next((k for k in range(L + 1) if amb[b * N + path[k]]), None)
        if first_amb is None:
            assert g["accept_len"][b] == L, f"accept_len seq {b}: {g['accept_len'][b]} vs {L}"
            assert np.array_equal(g["accept_path"][b], path), f"path seq {b}"
            assert g["next_token"][b] == o["next_token"][b], f"next token seq {b}"
        else:
            gated += 1
            assert np.array_equal(g["accept_path"][b][:first_amb + 1], path[:first_amb + 1])
    report["sequences"] = report.get("sequences", 0) + len(list(seqs))
    report["gated_sequences"] = report.get("gated_sequences", 0) + gated


def check_walk_consistent(g, parents, tokens):
    """Property that holds at any size: every accepted node carries its parent row's
    argmax, the walk stopped where no child matches, next_token is the last argmax."""
    B, N = parents.shape
    amax = g["row_argmax"].reshape(B, N)
    for b in range(B):
        if g["status"][b] != oracle.SEQ_OK:
            continue
        L, path = int(g["accept_len"][b]), g["accept_path"][b]
        assert path[0] == 0 and np.all(path[L + 1:] == -1)
        for k in range(1, L + 1):
            assert parents[b, path[k]] == path[k - 1]
            assert tokens[b, path[k]] == amax[b, path[k - 1]]
            earlier = [c for c in range(path[k - 1] + 1, path[k])
                       if parents[b, c] == path[k - 1] and tokens[b, c] == amax[b, path[k - 1]]]
            assert not earlier
        last = path[L]
        kids = np.flatnonzero(parents[b] == last)
        assert np.all(tokens[b, kids] != amax[b, last])
        assert g["next_token"][b] == amax[b, last]


def compare_sample(g, o, parents, u_acc, tokens, amb, report, seqs=None):
    """Sampled walks (chains or trees): the path and length exactly when every accept
    decision the oracle's walk took is clear (|u - ratio| > RATIO_GATE * ratio, with
    the ratio against the residual the node was tested with, on unambiguous rows),
    and the emitted token when the draw is also clear of its CDF breakpoints."""
    B, N = parents.shape
    seqs = range(B) if seqs is None else seqs
    gated = 0
    for b in seqs:
        assert g["status"][b] == o["status"][b]
        if o["status"][b] != oracle.SEQ_OK:
            continue
        r0 = b * N
        clear = True
        for i in range(1, N):
            ratio = o["walk_ratio"][r0 + i]
            if np.isnan(ratio):
                continue  # not tested on the oracle's walk
            u = float(u_acc[r0 + i])
            if amb[r0 + parents[b, i]] or (np.isfinite(ratio) and
                                             abs(u - ratio) <= RATIO_GATE * max(ratio, 1e-30)):
                clear = False
                break
        if not clear:
            gated += 1
            continue
        assert g["accept_len"][b] == o["accept_len"][b], f"seq {b}"
        assert np.array_equal(g["accept_path"][b], o["accept_path"][b]), f"path seq {b}"
        jrow = r0 + int(o["accept_path"][b][o["accept_len"][b]])
        if amb[jrow] or o["res_gap"][b] <= CDF_GATE:
            gated += 1
            continue
        assert g["next_token"][b] == o["next_token"][b], f"next token seq {b}"
    report["sequences"] = report.get("sequences", 0) + len(list(seqs))
    report["gated_sequences"] = report.get("gated_sequences", 0) + gated
