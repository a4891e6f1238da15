"""Pins for the CPU oracle: checks against what the paper and the mathematics fix
(hand-derived worked examples, closed forms, the paper's lemmas and theorem,
special cases and brute force), never against a retyping of the oracle itself."""
import ast
import itertools
import operator
import os

import numpy as np
import pytest
from scipy.special import logsumexp

import oracle
from paper_2608_12913_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers
def _num(expr: str) -> float:
    """Evaluate a closed-form number written with + - * / ** and literals only."""
    ops = {ast.Add: operator.add, ast.Sub: operator.sub, ast.Mult: operator.mul,
           ast.Div: operator.truediv, ast.Pow: operator.pow, ast.USub: operator.neg}

    def ev(n):
        if isinstance(n, ast.Expression):
            return ev(n.body)
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
            return float(n.value)
        if isinstance(n, ast.BinOp):
            return ops[type(n.op)](ev(n.left), ev(n.right))
        if isinstance(n, ast.UnaryOp):
            return ops[type(n.op)](ev(n.operand))
        raise ValueError(expr)

    return ev(ast.parse(expr.strip(), mode="eval"))


def _rows(fname):
    with open(os.path.join(GOLDEN, fname)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield [c.strip() for c in line.split(";")]


def _bias_only_case(logp, logq):
    """Inputs whose logits are exactly the given fp32 biases (hidden states zero).
    The two models get separate bias vectors through separate cases of W = 0."""
    V = len(logp)
    d = 8
    hp = np.zeros((1, d), np.float32)
    hq = np.zeros((1, d), np.float32)
    wp = np.zeros((V, d), np.float32)
    wq = np.zeros((V, d), np.float32)
    return hp, hq, wp, wq, np.asarray(logp, np.float32), np.asarray(logq, np.float32)


def _random_problem(rng, V, dp, dq, R, scale=1.0):
    hp = rng.standard_normal((R, dp)).astype(np.float32) * np.float32(scale)
    hq = rng.standard_normal((R, dq)).astype(np.float32) * np.float32(scale)
    wp = rng.standard_normal((V, dp)).astype(np.float32) / np.float32(np.sqrt(dp))
    wq = rng.standard_normal((V, dq)).astype(np.float32) / np.float32(np.sqrt(dq))
    bias = (-np.log(np.arange(V) + 1.0)).astype(np.float32)
    return hp, hq, wp, wq, bias


def _softmax_log(z):
    return z - logsumexp(z, axis=-1, keepdims=True)


# ---------------------------------------------------------------- LM-head logits
def test_logits_exact_small_integers():
    """Small-integer weights and hidden states: every product and partial sum is an
    exact integer, so the oracle's logits must equal exact integer arithmetic."""
    rng = np.random.default_rng(1)
    V, dp, dq, R = 37, 24, 16, 5  # non-square so a transposed operand cannot pass
    hp = rng.integers(-2, 3, (R, dp)).astype(np.float32)
    hq = rng.integers(-2, 3, (R, dq)).astype(np.float32)
    wp = rng.integers(-2, 3, (V, dp)).astype(np.float32)
    wq = rng.integers(-2, 3, (V, dq)).astype(np.float32)
    bp = rng.integers(-3, 4, V).astype(np.float32)
    bq = rng.integers(-3, 4, V).astype(np.float32)
    out = oracle.eval_rows(hp, hq, wp, wq, bp, bq, theta=0.1, s=0.5, want_logits=True)
    exact_p = hp.astype(np.int64) @ wp.astype(np.int64).T + bp.astype(np.int64)
    exact_q = hq.astype(np.int64) @ wq.astype(np.int64).T + bq.astype(np.int64)
    assert np.array_equal(out["zp"], exact_p.astype(np.float64))
    assert np.array_equal(out["zq"], exact_q.astype(np.float64))


def test_logits_one_hot_hidden_state_selects_weight_column():
    rng = np.random.default_rng(2)
    V, dp, dq = 29, 12, 8
    wp = rng.standard_normal((V, dp)).astype(np.float32)
    wq = rng.standard_normal((V, dq)).astype(np.float32)
    b = rng.standard_normal(V).astype(np.float32)
    kp, kq = [3, 0, 11], [7, 2, 5]
    hp = np.zeros((3, dp), np.float32)
    hq = np.zeros((3, dq), np.float32)
    for r in range(3):
        hp[r, kp[r]] = 1.0
        hq[r, kq[r]] = 1.0
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=0.5, want_logits=True)
    for r in range(3):
        assert np.array_equal(out["zp"][r], wp[:, kp[r]].astype(np.float64) + b)
        assert np.array_equal(out["zq"][r], wq[:, kq[r]].astype(np.float64) + b)


def test_temperature_divides_logits():
    rng = np.random.default_rng(3)
    hp, hq, wp, wq, b = _random_problem(rng, 50, 16, 8, 2)
    o1 = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=0.5, want_logits=True)
    o2 = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=0.5, temperature=2.0,
                          want_logits=True)
    np.testing.assert_allclose(o2["zp"], o1["zp"] / 2.0, rtol=0, atol=1e-14)


# ---------------------------------------------------------------- log-softmax
def test_lse_matches_library_logsumexp():
    rng = np.random.default_rng(4)
    hp, hq, wp, wq, b = _random_problem(rng, 1031, 32, 16, 4, scale=4.0)
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.1, s=0.5, want_logits=True)
    np.testing.assert_allclose(out["stats"][:, oracle.RS_LSEP], logsumexp(out["zp"], axis=1),
                               rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(out["stats"][:, oracle.RS_LSEQ], logsumexp(out["zq"], axis=1),
                               rtol=1e-13, atol=1e-12)
    np.testing.assert_array_equal(out["stats"][:, oracle.RS_MAXP], out["zp"].max(axis=1))
    total = np.exp(out["zp"] - out["stats"][:, [oracle.RS_LSEP]]).sum(axis=1)
    np.testing.assert_allclose(total, 1.0, atol=1e-12)


# ---------------------------------------------------------------- contrastive target
@pytest.mark.parametrize("row", list(_rows("cd_worked_examples.txt")), ids=lambda r: r[0])
def test_cd_worked_examples(row):
    name, s, theta, pp, pq, pcd, amax, count = row
    pi_p = np.array([_num(x) for x in pp.split(",")])
    pi_q = np.array([_num(x) for x in pq.split(",")])
    expect = np.array([_num(x) for x in pcd.split(",")])
    hp, hq, wp, wq, bp, bq = _bias_only_case(np.log(pi_p), np.log(pi_q))
    out = oracle.eval_rows(hp, hq, wp, wq, bp, bq, theta=float(theta), s=float(s),
                           want_lpcd=True)
    got = np.exp(out["lpcd"][0])
    np.testing.assert_allclose(got, expect, atol=2e-7)
    assert int(out["argmax"][0]) == int(amax)
    assert int(out["stats"][0, oracle.RS_COUNT]) == int(count)
    assert np.all(np.isneginf(out["lpcd"][0][expect == 0]))


def test_contrast_zero_gives_masked_expert():
    """s = 0: pi_CD is the expert restricted to the mask and renormalised, and its
    argmax is the expert argmax (the paper's alpha = 0 reduction)."""
    rng = np.random.default_rng(5)
    hp, hq, wp, wq, b = _random_problem(rng, 777, 24, 16, 6, scale=4.0)
    for theta in (0.0, 0.1, 0.5):
        out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=theta, s=0.0, want_logits=True,
                               want_lpcd=True)
        lp_p = _softmax_log(out["zp"])
        pi_p = np.exp(lp_p)
        mask = pi_p >= theta * pi_p.max(axis=1, keepdims=True)
        expect = np.where(mask, lp_p - np.log(np.where(mask, pi_p, 0).sum(1, keepdims=True)),
                          -np.inf)
        np.testing.assert_allclose(out["lpcd"], expect, atol=1e-10)
        assert np.array_equal(out["argmax"], out["zp"].argmax(axis=1))


def test_identical_amateur_gives_expert_for_every_strength():
    rng = np.random.default_rng(6)
    hp, _, wp, _, b = _random_problem(rng, 300, 16, 16, 3, scale=4.0)
    for s in (0.0, 0.5, 1.0, 3.0):
        out = oracle.eval_rows(hp, hp, wp, wp, b, b, theta=0.0, s=s, want_logits=True,
                               want_lpcd=True)
        np.testing.assert_allclose(out["lpcd"], _softmax_log(out["zp"]), atol=1e-10)


def test_kl_decomposition_lemma():
    """Lemma (KL divergence to target), untruncated target:
    KL(p||cd) = log Z - s KL(p||q); KL(q||cd) = log Z + (1+s) KL(q||p);
    KL(e||cd) = log Z + (1+s) KL(e||p) - s KL(e||q), with Z = sum p^(1+s) q^(-s)."""
    rng = np.random.default_rng(7)
    hp, hq, wp, wq, b = _random_problem(rng, 500, 24, 16, 4, scale=2.0)
    for s in (0.25, 0.5, 1.0):
        out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=s, want_logits=True,
                               want_lpcd=True)
        lp, lq, lc = _softmax_log(out["zp"]), _softmax_log(out["zq"]), out["lpcd"]
        le = _softmax_log(rng.standard_normal(lp.shape) * 2.0)
        logZ = out["stats"][:, oracle.RS_LOGZ]
        kl = lambda la, lb: (np.exp(la) * (la - lb)).sum(axis=1)  # noqa: E731
        np.testing.assert_allclose(kl(lp, lc), logZ - s * kl(lp, lq), atol=1e-9)
        np.testing.assert_allclose(kl(lq, lc), logZ + (1 + s) * kl(lq, lp), atol=1e-9)
        np.testing.assert_allclose(kl(le, lc), logZ + (1 + s) * kl(le, lp) - s * kl(le, lq),
                                   atol=1e-9)
        # Z itself: log sum p^(1+s) q^(-s)
        np.testing.assert_allclose(logZ, logsumexp((1 + s) * lp - s * lq, axis=1), atol=1e-11)


def test_reconstruction_error_lemma():
    """Lemma (reconstruction error decomposition): recombining approximations
    pi_e ~ pi_p and pi_f ~ pi_q gives an exponential tilt of pi_CD by
    Delta = (1+s) eps_p - s eps_q, normalised by E_{pi_CD}[exp(Delta)]."""
    rng = np.random.default_rng(8)
    V, d = 400, 16
    hp, hq, wp, wq, b = _random_problem(rng, V, d, d, 2, scale=3.0)
    # approximating heads: perturbed copies of the true heads
    we = (wp + 0.3 * rng.standard_normal(wp.shape) / np.sqrt(d)).astype(np.float32)
    wf = (wq + 0.3 * rng.standard_normal(wq.shape) / np.sqrt(d)).astype(np.float32)
    s = 0.7
    true = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=s, want_logits=True,
                            want_lpcd=True)
    appr = oracle.eval_rows(hp, hq, we, wf, b, b, theta=0.0, s=s, want_logits=True,
                            want_lpcd=True)
    eps_p = _softmax_log(appr["zp"]) - _softmax_log(true["zp"])
    eps_q = _softmax_log(appr["zq"]) - _softmax_log(true["zq"])
    delta = (1 + s) * eps_p - s * eps_q
    pi_cd = np.exp(true["lpcd"])
    z_delta = (pi_cd * np.exp(delta)).sum(axis=1, keepdims=True)
    np.testing.assert_allclose(np.exp(appr["lpcd"]), pi_cd * np.exp(delta) / z_delta,
                               rtol=1e-9, atol=1e-15)


def test_full_threshold_is_one_hot_at_expert_argmax():
    rng = np.random.default_rng(9)
    hp, hq, wp, wq, b = _random_problem(rng, 333, 16, 16, 5, scale=4.0)
    for s in (0.0, 0.5, 2.0):
        out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=1.0, s=s, want_logits=True,
                               want_lpcd=True)
        amax_p = out["zp"].argmax(axis=1)
        assert np.array_equal(out["argmax"], amax_p)
        assert np.all(out["stats"][:, oracle.RS_COUNT] == 1)
        pi = np.exp(out["lpcd"])
        np.testing.assert_array_equal(pi, np.eye(333)[amax_p])
        assert np.all(np.isinf(out["stats"][:, oracle.RS_MARGIN]))


@pytest.mark.parametrize("theta", [0.0, 0.01, 0.1, 0.5])
def test_mask_normalisation_and_support(theta):
    rng = np.random.default_rng(10)
    hp, hq, wp, wq, b = _random_problem(rng, 1024, 32, 16, 6, scale=4.0)
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=theta, s=0.5, want_logits=True,
                           want_lpcd=True)
    pi_p = np.exp(_softmax_log(out["zp"]))
    mask = pi_p >= theta * pi_p.max(axis=1, keepdims=True)
    # membership away from the exact cutoff (within 1e-9 the log/linear forms may differ)
    clear = np.abs(pi_p - theta * pi_p.max(axis=1, keepdims=True)) > 1e-9 * pi_p.max()
    assert np.array_equal(np.isfinite(out["lpcd"]) & clear, mask & clear)
    np.testing.assert_allclose(np.exp(out["lpcd"]).sum(axis=1), 1.0, atol=1e-12)
    np.testing.assert_array_equal(out["stats"][:, oracle.RS_COUNT], np.isfinite(out["lpcd"]).sum(1))


def test_argmax_and_margin_by_full_sort():
    rng = np.random.default_rng(11)
    hp, hq, wp, wq, b = _random_problem(rng, 97, 16, 8, 20, scale=4.0)
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.05, s=0.8, want_lpcd=True)
    for r in range(20):
        lc = out["lpcd"][r]
        order = np.argsort(-lc, kind="stable")  # descending, lowest id first on ties
        assert out["argmax"][r] == order[0]
        logZ = out["stats"][r, oracle.RS_LOGZ]
        assert abs(out["stats"][r, oracle.RS_TOP1] - (lc[order[0]] + logZ)) < 1e-12
        if np.isfinite(lc[order[1]]):
            np.testing.assert_allclose(out["stats"][r, oracle.RS_MARGIN], lc[order[0]] - lc[order[1]],
                                       atol=1e-12)


def test_flat_logits_tie_breaks_to_lowest_id():
    V, d = 64, 8
    z = np.zeros((1, d), np.float32)
    w = np.zeros((V, d), np.float32)
    out = oracle.eval_rows(z, z, w, w, None, None, theta=0.1, s=0.5, want_lpcd=True)
    assert out["argmax"][0] == 0
    assert out["stats"][0, oracle.RS_COUNT] == V
    np.testing.assert_allclose(np.exp(out["lpcd"][0]), 1.0 / V, atol=1e-15)
    assert out["stats"][0, oracle.RS_MARGIN] == 0.0


def test_contrastive_signal_statistic():
    """Row slot 7 is log pi_p(x*) - log pi_q(x*) at the CD argmax x*."""
    rng = np.random.default_rng(12)
    hp, hq, wp, wq, b = _random_problem(rng, 200, 16, 8, 4, scale=4.0)
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.1, s=0.5, want_logits=True)
    lp, lq = _softmax_log(out["zp"]), _softmax_log(out["zq"])
    a = out["argmax"]
    np.testing.assert_allclose(out["stats"][:, oracle.RS_SIGNAL],
                               lp[np.arange(4), a] - lq[np.arange(4), a], atol=1e-12)


# ---------------------------------------------------------------- row diagnostics
def test_row_diagnostics_kl_by_library_and_lemma():
    """D_KL(pi_p||pi_q) equals scipy's relative entropy of the two softmaxes, and the
    oracle's D_KL(pi_p||pi_CD), summed from its definition, obeys the lemma
    KL(p||cd) = log Z - s KL(p||q) of the KL-decomposition lemma (untruncated target)."""
    from scipy.stats import entropy
    rng = np.random.default_rng(13)
    hp, hq, wp, wq, b = _random_problem(rng, 700, 24, 16, 5, scale=3.0)
    for s in (0.1, 0.5, 1.0, 2.5):
        out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=s, want_logits=True)
        d = out["diag"]
        pp, pq = np.exp(_softmax_log(out["zp"])), np.exp(_softmax_log(out["zq"]))
        np.testing.assert_allclose(d[:, oracle.RD_KL_PQ], entropy(pp, pq, axis=1), rtol=1e-10)
        logZ = out["stats"][:, oracle.RS_LOGZ]
        np.testing.assert_allclose(d[:, oracle.RD_KL_PCD], logZ - s * d[:, oracle.RD_KL_PQ],
                                   atol=1e-10)
        assert np.all(d[:, oracle.RD_KL_PQ] > 0) and np.all(d[:, oracle.RD_KL_PCD] > 0)


def test_row_diagnostics_two_token_closed_form():
    """Two tokens, z_p = (0, 1), z_q = (0, 0), s = 1: pi_p = (1, e)/(1+e), pi_q = (1/2, 1/2),
    pi_CD ∝ pi_p^2 / pi_q ∝ (1, e^2), so KL(p||q) = ln 2 + sum pi_p ln pi_p and
    KL(p||cd) = sum pi_p ln(pi_p / pi_CD), written out by hand."""
    import math
    e = math.e
    hp, hq, wp, wq, bp, bq = _bias_only_case([0.0, 1.0], [0.0, 0.0])
    out = oracle.eval_rows(hp, hq, wp, wq, bp, bq, theta=0.0, s=1.0)
    p0, p1 = 1 / (1 + e), e / (1 + e)
    c0, c1 = 1 / (1 + e * e), e * e / (1 + e * e)
    kl_pq = p0 * math.log(2 * p0) + p1 * math.log(2 * p1)
    kl_pcd = p0 * math.log(p0 / c0) + p1 * math.log(p1 / c1)
    d = out["diag"][0]
    assert abs(d[oracle.RD_KL_PQ] - kl_pq) < 1e-14
    assert abs(d[oracle.RD_KL_PCD] - kl_pcd) < 1e-14
    assert d[oracle.RD_ARGMAX_P] == 1 and abs(d[oracle.RD_MARGIN_P] - 1.0) < 1e-15


def test_row_diagnostics_special_cases():
    """s = 0 gives pi_CD = pi_p (KL(p||cd) = 0); identical models give KL = 0 for both;
    a mask that drops a token with pi_p > 0 gives KL(p||cd) = +inf; flat logits keep
    the whole vocabulary in the mask and every divergence at 0."""
    rng = np.random.default_rng(14)
    hp, hq, wp, wq, b = _random_problem(rng, 300, 16, 16, 4, scale=3.0)
    d = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=0.0)["diag"]
    np.testing.assert_allclose(d[:, oracle.RD_KL_PCD], 0.0, atol=1e-12)
    d = oracle.eval_rows(hp, hp, wp, wp, b, b, theta=0.0, s=0.8)["diag"]
    np.testing.assert_allclose(d[:, [oracle.RD_KL_PQ, oracle.RD_KL_PCD]], 0.0, atol=1e-12)
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.1, s=0.5)
    assert np.all(out["stats"][:, oracle.RS_COUNT] < 300)
    assert np.all(np.isposinf(out["diag"][:, oracle.RD_KL_PCD]))
    assert np.all(np.isfinite(out["diag"][:, oracle.RD_KL_PQ]))
    z = np.zeros((1, 8), np.float32)
    w = np.zeros((64, 8), np.float32)
    d = oracle.eval_rows(z, z, w, w, None, None, theta=0.3, s=0.5)["diag"][0]
    assert d[oracle.RD_KL_PQ] == 0.0 and abs(d[oracle.RD_KL_PCD]) < 1e-15
    assert d[oracle.RD_ARGMAX_P] == 0 and d[oracle.RD_MARGIN_P] == 0.0


def test_expert_top1_by_sort_and_agreement_with_cd():
    """The expert's top-1 is the first index of the largest expert logit (stable sort),
    its margin the gap to the runner-up; with s = 0, or with theta = 1 (a one-token
    mask), the CD argmax is the expert's top-1."""
    rng = np.random.default_rng(15)
    hp, hq, wp, wq, b = _random_problem(rng, 211, 16, 8, 12, scale=4.0)
    for theta, s in ((0.0, 0.0), (0.1, 0.0), (1.0, 0.7), (0.05, 0.9)):
        out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=theta, s=s, want_logits=True)
        d = out["diag"]
        for r in range(12):
            order = np.argsort(-out["zp"][r], kind="stable")
            assert d[r, oracle.RD_ARGMAX_P] == order[0]
            assert d[r, oracle.RD_MARGIN_P] == out["zp"][r, order[0]] - out["zp"][r, order[1]]
        if s == 0.0 or theta == 1.0:
            assert np.array_equal(d[:, oracle.RD_ARGMAX_P], out["argmax"])
    # an exact tie of the two largest expert logits goes to the lower id
    hp_, hq_, wp_, wq_, bp_, bq_ = _bias_only_case([0.0, 2.0, 1.0, 2.0], [0.0, 0.0, 0.0, 0.0])
    d = oracle.eval_rows(hp_, hq_, wp_, wq_, bp_, bq_, theta=0.0, s=0.5)["diag"][0]
    assert d[oracle.RD_ARGMAX_P] == 1 and d[oracle.RD_MARGIN_P] == 0.0


def test_verify_returns_row_diagnostics_of_every_row():
    rng = np.random.default_rng(16)
    hp, hq, wp, wq, b = _random_problem(rng, 150, 16, 8, 6, scale=3.0)
    parents = np.array([[-1, 0, 1], [-1, 0, 0]], np.int32)
    tokens = np.array([[0, 3, 4], [0, 5, 6]], np.int32)
    o = oracle.verify("greedy", 2, 3, hp, hq, wp, wq, b, b, parents, tokens, theta=0.0, s=0.5)
    d = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=0.0, s=0.5)["diag"]
    np.testing.assert_array_equal(o["row_diag"], d)


# ---------------------------------------------------------------- dual-drafter proposals
def test_propose_hand_worked_example():
    """pi_e = (0.2, 0.3, 0.5), pi_f uniform, s = 1, no mask: pi_hat ~ pi_e^2 / pi_f
    ~ (0.04, 0.09, 0.25) / 0.38; the inverse CDF at u = 0.1, 0.2, 0.5 gives tokens
    0 (0.105 > 0.1), 1 (0.342 > 0.2) and 2."""
    hp, hq, wp, wq, bp, bq = _bias_only_case(np.log([0.2, 0.3, 0.5]), [0.0, 0.0, 0.0])
    he = np.repeat(hp, 3, axis=0)
    hf = np.repeat(hq, 3, axis=0)
    o = oracle.propose(he, hf, wp, wq, bp, bq, [0.1, 0.2, 0.5], theta=0.0, s=1.0)
    np.testing.assert_allclose(o["probs"], np.tile([0.04, 0.09, 0.25], (3, 1)) / 0.38, rtol=1e-6)
    assert list(o["tokens"]) == [0, 1, 2] and list(o["argmax"]) == [2, 2, 2]


def test_propose_special_cases():
    """An amateur-side head equal to the expert-side one, or s = 0, gives the
    expert-side head's own softmax (scipy), masked and renormalised under theta."""
    rng = np.random.default_rng(17)
    he, hf, we, wf, b = _random_problem(rng, 400, 16, 16, 5, scale=3.0)
    u = rng.random(5).astype(np.float32)
    for T in (1.0, 0.7):
        ze = (he.astype(np.float64) @ we.T.astype(np.float64) + b) / T
        pe = np.exp(_softmax_log(ze))
        o = oracle.propose(he, he, we, we, b, b, u, theta=0.0, s=0.8, temperature=T)
        np.testing.assert_allclose(o["probs"], pe, rtol=1e-9, atol=1e-15)
        o = oracle.propose(he, hf, we, wf, b, b, u, theta=0.2, s=0.0, temperature=T)
        keep = pe >= 0.2 * pe.max(axis=1, keepdims=True)
        np.testing.assert_allclose(o["probs"], np.where(keep, pe, 0) / np.where(keep, pe, 0).sum(1, keepdims=True),
                                   rtol=1e-9, atol=1e-15)


def test_propose_draw_follows_the_distribution():
    """Sweeping u over a midpoint grid, the drawn tokens' frequencies are the
    proposal probabilities up to the grid resolution."""
    rng = np.random.default_rng(18)
    he, hf, we, wf, b = _random_problem(rng, 12, 8, 8, 1, scale=1.0)
    G = 2000
    u = ((np.arange(G) + 0.5) / G).astype(np.float32)
    o = oracle.propose(np.repeat(he, G, 0), np.repeat(hf, G, 0), we, wf, b, b, u, theta=0.05, s=0.5)
    freq = np.bincount(o["tokens"], minlength=12) / G
    np.testing.assert_allclose(freq, o["probs"][0], atol=1.5 / G)
    assert np.all(o["probs"][0][freq > 0] > 0)


# ---------------------------------------------------------------- final RMS normalisation
def test_rmsnorm_closed_forms():
    """Constant rows normalise to 1, so the output is g itself; a one-hot row of width
    64 normalises to +-sqrt(64) = 8, so the output is 8 g at that column and 0
    elsewhere; a power-of-two scale of the rows changes nothing (eps = 0).  All exact
    in bf16."""
    rng = np.random.default_rng(19)
    d = 64
    g = synth.bf16_bits(rng.standard_normal(d).astype(np.float32))
    gf = oracle.as_f32(g)
    x = synth.bf16_bits(np.full((3, d), [[3.0], [-0.5], [1024.0]], np.float32))
    y = oracle.as_f32(oracle.rmsnorm(x, g, 1e-6))
    np.testing.assert_array_equal(y[0], gf)
    np.testing.assert_array_equal(y[1], -gf)
    np.testing.assert_array_equal(y[2], gf)
    x = np.zeros((2, d), np.float32)
    x[0, 5], x[1, 63] = 0.75, -96.0
    y = oracle.as_f32(oracle.rmsnorm(synth.bf16_bits(x), g, 0.0))
    expect = np.zeros((2, d), np.float32)
    expect[0, 5], expect[1, 63] = 8 * gf[5], -8 * gf[63]
    np.testing.assert_array_equal(y, expect)
    x = synth.bf16_bits(rng.standard_normal((4, d)).astype(np.float32))
    x4 = synth.bf16_bits(oracle.as_f32(x) * np.float32(4.0))
    np.testing.assert_array_equal(oracle.rmsnorm(x, g, 0.0), oracle.rmsnorm(x4, g, 0.0))


def test_rmsnorm_matches_torch():
    """fp32: torch's rms_norm in fp64.  bf16: the Llama-family reference computation in
    torch (fp32 statistics, the normalised value cast to bf16, then scaled in bf16);
    the oracle, in fp64, agrees bit for bit except where the fp32 rounding of the
    reference falls on the other side of a bf16 rounding boundary (one unit)."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(20)
    R, d, eps = 16, 512, 1e-5
    x = (rng.standard_normal((R, d)) * 3).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x).double(), (d,), torch.from_numpy(g).double(),
                                       eps=eps).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, eps), ref, rtol=1e-6, atol=1e-7)
    xb, gb = synth.bf16_bits(x), synth.bf16_bits(g)
    xt = torch.from_numpy(oracle.as_f32(xb)).to(torch.bfloat16)
    gt = torch.from_numpy(oracle.as_f32(gb)).to(torch.bfloat16)
    h = xt.float()
    h = h * torch.rsqrt(h.pow(2).mean(-1, keepdim=True) + eps)
    ref = (gt * h.to(torch.bfloat16)).float().numpy()
    got = oracle.as_f32(oracle.rmsnorm(xb, gb, eps))
    ulp = np.abs(got.view(np.int32) - ref.view(np.int32)) >> 16
    assert np.all(ulp <= 1) and (ulp == 0).mean() > 0.99


# ---------------------------------------------------------------- greedy walk
def _parse_ints(s):
    return np.array([int(x) for x in s.split(",")], np.int32)


@pytest.mark.parametrize("row", list(_rows("greedy_walk_examples.txt")), ids=lambda r: r[0])
def test_greedy_walk_worked_examples(row):
    name, par, tok, amax, L, path, nxt = row
    got_L, got_path, got_next = oracle.greedy_walk(_parse_ints(par), _parse_ints(tok),
                                                   _parse_ints(amax))
    assert got_L == int(L)
    assert np.array_equal(got_path, _parse_ints(path))
    assert got_next == int(nxt)


def _brute_force_walk(parents, tokens, amax):
    """Enumerate every root-to-node path whose every node carries its parent row's
    argmax; among the maximal ones take the lexicographically smallest node sequence."""
    N = len(parents)
    paths = []

    def ext(p):
        kids = [c for c in range(N) if parents[c] == p[-1] and tokens[c] == amax[p[-1]]]
        if not kids:
            paths.append(tuple(p))
        for c in kids:
            ext(p + [c])

    ext([0])
    best = min(paths)
    return len(best) - 1, best, int(amax[best[-1]])


def test_greedy_walk_matches_brute_force_on_random_trees():
    rng = np.random.default_rng(13)
    for trial in range(300):
        N = int(rng.integers(1, 14))
        parents = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, N)], np.int32)
        V = int(rng.integers(2, 5))  # tiny vocabulary: many matches and duplicate siblings
        tokens = rng.integers(0, V, N).astype(np.int32)
        amax = rng.integers(0, V, N).astype(np.int32)
        L, path, nxt = oracle.greedy_walk(parents, tokens, amax)
        bL, bpath, bnext = _brute_force_walk(parents, tokens, amax)
        assert (L, nxt) == (bL, bnext), trial
        assert tuple(path[:L + 1]) == bpath and np.all(path[L + 1:] == -1)


def _tiny_greedy_case(seed, **kw):
    case = synth.make_case("tiny_chain8", seed, **kw)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s)
    tokens = synth.greedy_tokens(case, rows["argmax"])
    return case, tokens


@pytest.mark.parametrize("tree", ["chain", "tree"])
def test_accepted_path_is_prefix_of_cd_greedy_continuation(tree):
    kw = dict(N=24, tree="tree", depth=5, max_children=4) if tree == "tree" else {}
    for seed in range(5):
        case, tokens = _tiny_greedy_case(seed, **kw)
        o = oracle.verify("greedy", case.B, case.N, case.hp, case.hq, case.wp, case.wq, case.bias,
                          case.bias, case.parents, tokens, theta=case.theta, s=case.s)
        assert o["status"][0] == oracle.SEQ_OK
        L, path = int(o["accept_len"][0]), o["accept_path"][0]
        amax = o["row_argmax"]
        for k in range(1, L + 1):  # every accepted token is its parent row's CD argmax
            node, parent = path[k], path[k - 1]
            assert case.parents[0, node] == parent
            assert tokens[0, node] == amax[parent]
        assert o["next_token"][0] == amax[path[L]]
        # and the walk stopped: no child of the last node carries the argmax
        last = path[L]
        kids = [c for c in range(case.N) if case.parents[0, c] == last]
        assert all(tokens[0, c] != amax[last] for c in kids)


def test_masked_tokens_are_never_accepted():
    case = synth.make_case("tiny_chain8", 3, N=16)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, want_lpcd=True)
    for trial in range(3):
        # every draft token is chosen OUTSIDE its parent row's mask
        tokens = np.zeros((1, case.N), np.int32)
        for i in range(1, case.N):
            masked = np.flatnonzero(np.isneginf(rows["lpcd"][i - 1]))
            tokens[0, i] = masked[(7 * i + trial) % len(masked)]
        o = oracle.verify("greedy", 1, case.N, case.hp, case.hq, case.wp, case.wq, case.bias,
                          case.bias, case.parents, tokens, theta=case.theta, s=case.s)
        assert o["accept_len"][0] == 0
        assert np.all(o["node_stats"][1:, oracle.NS_INMASK] == 0)
        assert np.all(np.isneginf(o["node_stats"][1:, oracle.NS_LPCD]))


def test_node_statistics_follow_parent_rows():
    case, tokens = _tiny_greedy_case(4, N=20, tree="tree", depth=4, max_children=5)
    o = oracle.verify("greedy", 1, case.N, case.hp, case.hq, case.wp, case.wq, case.bias,
                      case.bias, case.parents, tokens, theta=case.theta, s=case.s)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, want_logits=True, want_lpcd=True)
    lp, lq = _softmax_log(rows["zp"]), _softmax_log(rows["zq"])
    ns = o["node_stats"]
    assert np.all(np.isnan(ns[0]))
    for i in range(1, case.N):
        j, x = case.parents[0, i], tokens[0, i]
        np.testing.assert_allclose(ns[i, :3], [lp[j, x], lq[j, x], 1.5 * lp[j, x] - 0.5 * lq[j, x]],
                                   atol=1e-12)
        assert ns[i, oracle.NS_LPCD] == rows["lpcd"][j, x]


def test_sequence_status_codes():
    case, tokens = _tiny_greedy_case(0)
    args = (case.hp, case.hq, case.wp, case.wq, case.bias, case.bias)
    par = case.parents.copy()
    par[0, 3] = 5  # parent after child
    o = oracle.verify("greedy", 1, case.N, *args, par, tokens, theta=0.1, s=0.5)
    assert o["status"][0] == oracle.SEQ_BAD_TREE and o["accept_len"][0] == 0
    assert o["next_token"][0] == -1 and np.all(o["accept_path"][0] == -1)
    bad = tokens.copy()
    bad[0, 2] = case.V
    o = oracle.verify("greedy", 1, case.N, *args, case.parents, bad, theta=0.1, s=0.5)
    assert o["status"][0] == oracle.SEQ_BAD_TOKEN
    hp = case.hp.copy()
    hp[4, 0] = np.inf
    o = oracle.verify("greedy", 1, case.N, hp, *args[1:], case.parents, tokens, theta=0.1, s=0.5)
    assert o["status"][0] == oracle.SEQ_NONFINITE
    # sampled verification takes trees as well as chains
    tree = synth.make_case("tiny_chain8", 0, N=8, tree="tree", depth=3, max_children=3)
    probs = np.full((8, case.V), 1.0 / case.V, np.float32)
    o = oracle.verify("sample", 1, 8, *args, tree.parents, tokens, theta=0.1, s=0.5,
                      draft_probs=probs, u_acc=case.u_acc, u_res=case.u_res)
    assert o["status"][0] == oracle.SEQ_OK


# ---------------------------------------------------------------- sampled verification
def _tiny_target(rng, V, theta, s, N):
    hp, hq, wp, wq, b = _random_problem(rng, V, 8, 8, N, scale=2.0)
    out = oracle.eval_rows(hp, hq, wp, wq, b, b, theta=theta, s=s, want_lpcd=True)
    return out["lpcd"]


class _ChainCall:
    """Repeated calls of the oracle's sampler on a chain, on fixed buffers (fast loop)."""

    def __init__(self, lp_cd, q):
        import ctypes
        self.lib = oracle._load()
        self.N, self.V = lp_cd.shape
        self.lp = np.ascontiguousarray(lp_cd, np.float64)
        self.q = np.ascontiguousarray(q, np.float32)
        self.par = np.arange(-1, self.N - 1, dtype=np.int32)
        self.tok = np.zeros(self.N, np.int32)
        self.ua = np.full(self.N, 0.5, np.float32)
        self.ur = np.full(self.N, 0.5, np.float32)
        self.L = np.zeros(1, np.int32)
        self.path = np.zeros(self.N, np.int32)
        self.nxt = np.zeros(1, np.int32)
        p = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731
        self.args = (self.N, self.V, p(self.par), p(self.tok), p(self.lp), p(self.q), p(self.ua),
                     p(self.ur), p(self.L), p(self.path), p(self.nxt), None, None, None)

    def __call__(self):
        self.lib.dco_sample_tree(*self.args)
        return int(self.L[0]), int(self.nxt[0])


@pytest.mark.parametrize("theta,s", [(0.0, 0.5), (0.1, 0.5), (0.3, 1.0), (0.0, 0.0)])
def test_lossless_theorem_by_enumeration(theta, s):
    """Theorem (lossless property) with the plausibility-mask remark: enumerating every
    draft token x ~ pi_e and a G x G midpoint grid of (u_acc, u_res), the emitted token
    is distributed exactly as pi_CD up to the grid resolution."""
    rng = np.random.default_rng(14)
    V, G = 6, 128
    lp_cd = _tiny_target(rng, V, theta, s, 2)
    target = np.exp(lp_cd[0])
    proposals = [rng.dirichlet(np.ones(V)), np.eye(V)[int(np.argmin(target))],
                 np.full(V, 1.0 / V), np.r_[0.0, rng.dirichlet(np.ones(V - 1))]]
    grid = ((np.arange(G) + 0.5) / G).astype(np.float32)
    for pe in proposals:
        pe = pe.astype(np.float32)
        call = _ChainCall(lp_cd, np.stack([np.zeros(V, np.float32), pe]))
        emitted = np.zeros(V)
        for x in range(V):
            if pe[x] == 0:
                continue
            call.tok[1] = x
            for ua in grid:
                call.ua[1] = ua
                for ur in grid:
                    call.ur[0] = ur
                    L, nxt = call()
                    emitted[x if L == 1 else nxt] += pe[x] / (G * G)
        np.testing.assert_allclose(emitted, target, atol=2.0 / G)
        assert np.all(emitted[target == 0] == 0)


@pytest.fixture(scope="module")
def sweep_lib(tmp_path_factory):
    """The brute-force sweep driver (tests/native/lossless_sweep.c) built against the
    oracle library."""
    import ctypes
    import subprocess
    lib = oracle.build(force=False)
    out = tmp_path_factory.mktemp("sweep") / "libsweep.so"
    src = os.path.join(os.path.dirname(__file__), "native", "lossless_sweep.c")
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", src, lib, "-o", str(out),
                           f"-Wl,-rpath,{os.path.dirname(lib)}"])
    L = ctypes.CDLL(str(out))
    P = ctypes.c_void_p
    L.sweep_star.argtypes = [ctypes.c_int, ctypes.c_int, P, P, ctypes.c_int, P]
    L.sweep_star.restype = ctypes.c_int
    return L


@pytest.mark.parametrize("K,V,G,theta,s", [(2, 5, 96, 0.0, 0.5), (2, 5, 96, 0.1, 1.0),
                                           (3, 3, 24, 0.0, 0.5)])
def test_lossless_theorem_on_trees_by_enumeration(sweep_lib, K, V, G, theta, s):
    """The lossless property with several drafted children per node: a root with K
    children drafted independently from different proposals (one of them with a zero
    entry, one one-hot on the target's least likely token).  Enumerating every token
    assignment and a midpoint grid of every uniform, the first emitted token is
    distributed as pi_CD of the root."""
    rng = np.random.default_rng(30 + K)
    lp_cd = np.zeros((K + 1, V))
    lp_cd[0] = _tiny_target(rng, V, theta, s, 1)[0]
    target = np.exp(lp_cd[0])
    props = [rng.dirichlet(np.ones(V)), np.r_[0.0, rng.dirichlet(np.ones(V - 1))],
             np.eye(V)[int(np.argmin(target))]]
    q = np.zeros((K + 1, V), np.float32)
    for k in range(K):
        q[k + 1] = props[k]
    out = np.zeros(V)
    P = lambda a: a.ctypes.data_as(__import__("ctypes").c_void_p)  # noqa: E731
    assert sweep_lib.sweep_star(K, V, P(lp_cd), P(q), G, P(out)) == 0
    np.testing.assert_allclose(out, target, atol=2.0 / G)
    assert np.all(out[target == 0] == 0)


def test_tree_sampler_hand_worked_example():
    """Root with two children, V = 2, pi_CD(root) = (1/2, 1/2).  Child 1 is one-hot on
    token 0 (q_1 = (1, 0)): ratio 1/2, rejected at u = 0.7, leaving the residual
    max(0, p - q_1) = (0, 1/2) -> (0, 1).  Child 2 (q_2 = (1/2, 1/2)) then carries
    token 0, with p(0) = 0: rejected whatever u is; the residual is
    max(0, (0, 1) - (1/2, 1/2)) = (0, 1/2) -> (0, 1), so the draw is token 1.  Carrying
    token 1 instead, its ratio is 1 / (1/2) = 2 and it is accepted; the bonus is drawn
    from pi_CD of its own row."""
    lp = np.log(np.array([[0.5, 0.5], [0.5, 0.5], [0.25, 0.75]]))
    q = np.array([[0, 0], [1, 0], [0.5, 0.5]], np.float32)
    par = [-1, 0, 0]
    o = oracle.sample_tree(par, [0, 0, 0], lp, q, [0.5, 0.7, 0.01], [0.1, 0.5, 0.5])
    assert o["accept_len"] == 0 and o["next_token"] == 1
    np.testing.assert_allclose(o["walk_ratio"][1:], [0.5, 0.0])
    o = oracle.sample_tree(par, [0, 0, 1], lp, q, [0.5, 0.7, 0.99], [0.5, 0.5, 0.2])
    assert o["accept_len"] == 1 and list(o["path"][:2]) == [0, 2]
    assert o["next_token"] == 0  # 0.2 < 0.25: the first token of (1/4, 3/4)
    np.testing.assert_allclose(o["walk_ratio"][1:], [0.5, 2.0])
    # child 1 accepted (u = 0.3 <= 1/2): child 2 is never tested
    o = oracle.sample_tree(par, [0, 0, 1], lp, q, [0.5, 0.3, 0.5], [0.5, 0.9, 0.5])
    assert o["accept_len"] == 1 and o["path"][1] == 1 and o["next_token"] == 1
    assert np.isnan(o["walk_ratio"][2])


def test_tree_walk_descends_after_acceptance():
    """Depth 2: an accepted child's own children are tested against its row."""
    lp = np.log(np.array([[0.5, 0.5], [0.9, 0.1], [0.2, 0.8], [0.5, 0.5]]))
    q = np.array([[0, 0], [0, 1], [1, 0], [0, 1]], np.float32)
    par = [-1, 0, 1, 0]
    # node 1 (token 1 under the root: ratio 1/2, u 0.4 -> accept); node 2 (token 0 under
    # row 1: ratio 0.9, u 0.5 -> accept); node 3 is a sibling of node 1, never tested
    o = oracle.sample_tree(par, [0, 1, 0, 1], lp, q, [0.5, 0.4, 0.5, 0.01], [0.5, 0.5, 0.3, 0.5])
    assert o["accept_len"] == 2 and list(o["path"][:3]) == [0, 1, 2]
    # node 2 is a leaf: the bonus comes from row 2, (0.2, 0.8), at u = 0.3 -> token 1
    assert o["next_token"] == 1 and np.isnan(o["walk_ratio"][3])
    np.testing.assert_allclose(o["walk_ratio"][1:3], [0.5, 0.9])


def test_proposal_equal_to_target_accepts_everything():
    rng = np.random.default_rng(15)
    V, N = 50, 6
    lp_cd = _tiny_target(rng, V, 0.05, 0.5, N)
    q = np.zeros((N, V), np.float32)
    q[1:] = np.exp(lp_cd[:-1])  # node i was drawn from its parent row's target
    for trial in range(20):
        tokens = [0] + [int(rng.choice(V, p=np.exp(lp_cd[i - 1]) / np.exp(lp_cd[i - 1]).sum()))
                        for i in range(1, N)]
        u = rng.uniform(0.0, 0.999, N).astype(np.float32)
        o = oracle.sample_chain(tokens, lp_cd, q, u, u)
        assert o["accept_len"] == N - 1
        assert np.isfinite(lp_cd[N - 1, o["next_token"]])  # bonus drawn inside the mask


def test_masked_one_hot_proposal_rejects_and_resamples_target():
    """A proposal that is one-hot on a masked token is rejected at node 1 and the
    residual max(0, pi_CD - pi_e) is pi_CD itself."""
    rng = np.random.default_rng(16)
    V, G = 40, 4000
    lp_cd = _tiny_target(rng, V, 0.2, 0.5, 3)
    masked = int(np.flatnonzero(np.isneginf(lp_cd[0]))[0])
    q = np.zeros((3, V), np.float32)
    q[1, masked] = 1.0
    q[2] = 1.0 / V
    counts = np.zeros(V)
    for ur in (np.arange(G) + 0.5) / G:
        o = oracle.sample_chain([0, masked, 0], lp_cd, q, [0.5, 1e-7, 0.5], [ur, 0.5, 0.5])
        assert o["accept_len"] == 0 and o["ratio"][1] == 0.0
        counts[o["next_token"]] += 1
    np.testing.assert_allclose(counts / G, np.exp(lp_cd[0]), atol=2.0 / G)


def test_sampled_never_accepts_or_emits_masked_tokens():
    rng = np.random.default_rng(17)
    V, N = 30, 5
    for trial in range(200):
        lp_cd = _tiny_target(rng, V, 0.3, float(rng.uniform(0, 2)), N)
        q = np.stack([rng.dirichlet(np.ones(V) * 0.3) for _ in range(N)]).astype(np.float32)
        tokens = [0] + [int(rng.integers(V)) for _ in range(N - 1)]
        u = rng.uniform(1e-6, 1 - 1e-6, N).astype(np.float32)
        o = oracle.sample_chain(tokens, lp_cd, q, u, u[::-1].copy())
        L = o["accept_len"]
        for i in range(1, L + 1):
            assert np.isfinite(lp_cd[i - 1, tokens[i]])
        assert np.isfinite(lp_cd[L, o["next_token"]])


def test_zero_proposal_probability_accepts_in_mask():
    rng = np.random.default_rng(18)
    V = 20
    lp_cd = _tiny_target(rng, V, 0.0, 0.5, 2)
    q = np.zeros((2, V), np.float32)
    q[1, 3] = 1.0
    o = oracle.sample_chain([0, 5], lp_cd, q, [0.5, 0.999], [0.5, 0.5])
    assert o["ratio"][1] == np.inf and o["accept_len"] == 1
    # a masked token is rejected even when its proposal probability is zero
    lp_m = _tiny_target(rng, V, 0.5, 0.5, 2)
    masked = int(np.flatnonzero(np.isneginf(lp_m[0]))[0])
    o = oracle.sample_chain([0, masked], lp_m, q, [0.5, 1e-7], [0.5, 0.5])
    assert o["accept_len"] == 0 and np.isfinite(lp_m[0, o["next_token"]])


def test_verify_sample_matches_per_row_composition():
    case = synth.make_case("tiny_chain8", 21, mode="sample", B=3, N=6)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, temperature=case.T, want_logits=True,
                            want_lpcd=True)
    par_logits = np.zeros_like(rows["zp"])
    par_logits[1:] = rows["zp"][:-1]
    probs, tokens = synth.sampled_draft(case, par_logits)
    o = oracle.verify("sample", case.B, case.N, case.hp, case.hq, case.wp, case.wq, case.bias,
                      case.bias, case.parents, tokens, theta=case.theta, s=case.s,
                      temperature=case.T, draft_probs=probs, u_acc=case.u_acc, u_res=case.u_res)
    for b in range(case.B):
        sl = slice(b * case.N, (b + 1) * case.N)
        ref = oracle.sample_chain(tokens[b], rows["lpcd"][sl], probs[sl], case.u_acc[sl],
                                  case.u_res[sl])
        assert o["status"][b] == 0
        assert o["accept_len"][b] == ref["accept_len"]
        assert o["next_token"][b] == ref["next_token"]
        np.testing.assert_array_equal(o["node_stats"][sl][1:, oracle.NS_RATIO], ref["ratio"][1:])
