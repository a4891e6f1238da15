"""Comparison of GPU outputs with the oracle, with the gating rules of the parity bar.

Greedy.  Token ids, accepted lengths and paths must match bit for bit wherever the
oracle's top-2 cd margin exceeds MARGIN_GATE and no token lies within
BOUNDARY_GATE nats of the plausibility cutoff on every row the oracle's path
visits; log-probabilities and cd scores must agree within ATOL on such rows.

Sampled.  The GPU computes each target probability pi_CD(v) = exp(log pi_CD(v)) in
fp32, then the walk's residuals and draws from those values in fp64.  So the GPU
walk is the exact walk on a target whose every entry is off by a small relative
error.  The tests measure that error at every token: dcd_propose on the
verification's own heads writes pi_CD densely through the same kernels and the same
expression the walk weighs tokens with (measure_target_error), and DELTA_P caps it
(the fp32 budget: 1e-4 in log space).  A sampled walk is then re-run on the
oracle's target with every pi_CD(v) replaced by the interval
[pi_CD(v) e^-d, pi_CD(v) e^d], d twice the measured error, carried through Alg. 1's
accept test, each residual Normalize(max(0, p - pi_e)) and the final inverse-CDF
draw.  A decision is clear when it comes out the same for every value in the
intervals; the path must match exactly when every decision on it is clear, and
the emitted token when the draw is clear too.  Rows near the mask cutoff
(BOUNDARY_GATE) gate the walk at that row, as in greedy mode.

Every gate is counted: check_gates() bounds the ambiguous rows and the gated
sequences of a test, so a broken gate cannot turn the comparison into a no-op.
"""
import numpy as np

import oracle

MARGIN_GATE = 1e-3
BOUNDARY_GATE = 1e-4
ATOL = 1e-3
DELTA_P = 1e-4
CDF_GATE = 1e-4  # draws of dcd_propose: relative distance of u * total to every breakpoint


def ambiguous_rows(o):
    margin = o["row_stats"][:, oracle.RS_MARGIN]
    return (margin <= MARGIN_GATE) | (o["row_gap"] <= BOUNDARY_GATE)


def check_gates(report, max_ambiguous=None, max_gated=None):
    """The gates of one test stay rare, unless the test states other bounds (cases
    built on ties gate every row on purpose): at most 1% of the rows (plus one)
    ambiguous; gated sequences at most one per ambiguous row (a greedy walk is gated
    only at an ambiguous row on its path) plus 2% of the sequences (sampled walks are
    also gated by their own decisions, about 2 DELTA_P of them)."""
    rows = report.get("rows", 0)
    amb = report.get("ambiguous_rows", 0)
    limit = 0.01 * rows + 1 if max_ambiguous is None else max_ambiguous
    assert amb <= limit, f"{amb} of {rows} rows ambiguous (limit {limit})"
    gated = report.get("gated_sequences", 0)
    glimit = amb + 0.02 * report.get("sequences", 0) if max_gated is None else max_gated
    assert gated <= glimit, f"{gated} gated sequences (limit {glimit})"


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
    # log pi_CD of the argmax (top1 - log Z): its error is the error of the target
    # probability the sampled gates assume bounded
    lg = gs[ok, oracle.RS_TOP1] - gs[ok, oracle.RS_LOGZ]
    lo = ostats[ok, oracle.RS_TOP1] - ostats[ok, oracle.RS_LOGZ]
    if len(lg):
        report["max_lpcd_err"] = max(report.get("max_lpcd_err", 0.0), float(np.abs(lg - lo).max()))
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
    worst = report.get("max_lpcd_err", 0.0)
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
                d = abs(gn[r, oracle.NS_LPCD] - on[r, oracle.NS_LPCD])
                assert d <= ATOL
                worst = max(worst, d)
        assert np.all(np.isnan(gn[b * N]))
    report["nodes"] = report.get("nodes", 0) + B * (N - 1)
    report["max_lpcd_err"] = worst


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


def measure_target_error(pg, lp, boundary, report, floor=-80.0, cap=DELTA_P / 2):
    """Largest |ln pi_CD_gpu(v) - log pi_CD_oracle(v)| over every token of every row
    outside `boundary`, from the GPU's dense target rows pg [R, V] (dcd_propose on the
    verification's heads) and the oracle's lp [R, V].  Tokens below e^floor of mass
    (no draw or decision can depend on them) are left out; the support must agree
    above it.  Recorded as report["target_err"], at most `cap` (the fp32 budget
    DELTA_P / 2 when both sides read the same inputs)."""
    ok = ~np.asarray(boundary)
    g, o = pg[ok].astype(np.float64), lp[ok]
    big = o > floor
    assert np.array_equal(g[big] > 0, np.ones(int(big.sum()), bool)), "GPU target misses support"
    assert np.all(g[np.isneginf(o)] == 0), "GPU target has mass off the mask"
    err = float(np.abs(np.log(g[big]) - o[big]).max()) if big.any() else 0.0
    report["target_err"] = max(report.get("target_err", 0.0), err)
    assert err <= cap, f"target log-probability error {err} exceeds {cap}"
    return err


def _inverse_cdf(w, u):
    """Smallest index whose cumulative weight exceeds u times the total (the last
    index of positive weight if rounding leaves none)."""
    c = np.cumsum(w)
    hit = np.flatnonzero((w > 0) & (c > u * c[-1]))
    if len(hit):
        return int(hit[0])
    pos = np.flatnonzero(w > 0)
    return int(pos[-1]) if len(pos) else -1


def interval_walk(parents, tokens, lp_cd, q, u_acc, u_res, delta=DELTA_P, boundary=None):
    """The sampled walk of one sequence (children tried in index order, each against
    the residual the rejected siblings left; the emitted token drawn from what is
    left), run twice at once: on the oracle's target p = exp(lp_cd) itself, and on
    intervals [p e^-delta, p e^delta] of every target probability.

    Returns dict(path, accept_len, next_token) of the point walk, `path_clear` (every
    accept decision on the path is the same for all values in the intervals, and no
    visited row is in `boundary`) and `draw_clear` (the emitted token too)."""
    N, V = lp_cd.shape
    shrink, grow = np.exp(-delta), np.exp(delta)

    def row(j):
        p = np.exp(lp_cd[j])
        return p, p * shrink, p * grow

    cur, path, clear = 0, [0], True
    p, lo, hi = row(0)
    if boundary is not None and boundary[0]:
        clear = False
    while clear:
        nxt = None
        for c in range(cur + 1, N):
            if parents[c] != cur:
                continue
            x, qc, u = int(tokens[c]), q[c].astype(np.float64), float(u_acc[c])
            if qc[x] > 0:
                acc = p[x] > 0 and u <= p[x] / qc[x]
                sure_acc = lo[x] > 0 and u <= lo[x] / qc[x]
                sure_rej = hi[x] == 0 or u > hi[x] / qc[x]
            else:  # ratio +inf: accepted iff the token has target mass
                acc, sure_acc, sure_rej = p[x] > 0, lo[x] > 0, hi[x] == 0
            if not (sure_acc or sure_rej):
                clear = False
                break
            assert acc == sure_acc
            if acc:
                nxt = c
                break
            w = np.maximum(p - qc, 0.0)
            wlo, whi = np.maximum(lo - qc, 0.0), np.maximum(hi - qc, 0.0)
            t, tlo, thi = w.sum(), wlo.sum(), whi.sum()
            if tlo > 0:
                p, lo, hi = w / t, wlo / thi, whi / tlo
            elif thi > 0:  # whether the residual applies at all depends on the error
                clear = False
                break
        if not clear or nxt is None:
            break
        path.append(nxt)
        cur = nxt
        p, lo, hi = row(cur)
        if boundary is not None and boundary[cur]:
            clear = False
    u = float(u_res[cur])
    nt = _inverse_cdf(p, u)
    draw_clear = False
    if clear and nt >= 0:
        clo, chi = np.cumsum(lo), np.cumsum(hi)
        below = chi[nt - 1] if nt > 0 else 0.0  # mass before the token, at most
        draw_clear = below < u * clo[-1] and clo[nt] > u * chi[-1]
    out = np.full(N, -1, np.int32)
    out[:len(path)] = path
    return dict(path=out, accept_len=len(path) - 1, next_token=nt, path_clear=clear,
                draw_clear=draw_clear)


def compare_sample(g, o, lp_cd, draft_probs, parents, tokens, u_acc, u_res, boundary, report,
                   seqs=None, delta=None):
    """Sampled walks (chains or trees) of GPU sequences against the oracle's (rows of
    lp_cd, draft_probs, u_acc, u_res and boundary indexed like the oracle's rows):
    the path and length exactly when the interval walk finds every decision on it
    clear, the emitted token when the draw is clear too.  The interval walk's point
    values must reproduce the oracle's own walk.  delta: the intervals' half-width
    in log space, by default twice the error measured at every token
    (measure_target_error); the errors measured at the draft tokens and row argmaxes
    must lie within it."""
    B, N = parents.shape
    seqs = range(B) if seqs is None else seqs
    if delta is None:
        assert "target_err" in report, "measure_target_error first"
        delta = 2.0 * report["target_err"] + 1e-9
    measured = report.get("max_lpcd_err")
    assert measured is not None, "compare_rows / compare_nodes first: they measure the error"
    assert measured <= delta, f"node log-probability error {measured} exceeds the bound {delta}"
    report["walk_delta"] = delta
    gated = 0
    for b in seqs:
        assert g["status"][b] == o["status"][b]
        if o["status"][b] != oracle.SEQ_OK:
            continue
        r = slice(b * N, b * N + N)
        w = interval_walk(parents[b], tokens[b], lp_cd[r], draft_probs[r], u_acc[r], u_res[r],
                          delta, boundary[r])
        L = int(o["accept_len"][b])
        if w["path_clear"]:
            assert w["accept_len"] == L and np.array_equal(w["path"], o["accept_path"][b]), \
                f"interval walk disagrees with the oracle on seq {b}"
        if not w["path_clear"]:
            gated += 1
            continue
        assert g["accept_len"][b] == L, f"accept_len seq {b}: {g['accept_len'][b]} vs {L}"
        assert np.array_equal(g["accept_path"][b], o["accept_path"][b]), f"path seq {b}"
        if not w["draw_clear"]:
            gated += 1
            continue
        assert w["next_token"] == o["next_token"][b], f"interval draw disagrees on seq {b}"
        assert g["next_token"][b] == o["next_token"][b], f"next token seq {b}"
    report["sequences"] = report.get("sequences", 0) + len(list(seqs))
    report["gated_sequences"] = report.get("gated_sequences", 0) + gated
