"""GPU parity: libdcd (through the C ABI) against the CPU oracle on seeded inputs."""
import sys

import numpy as np
import pytest

import oracle
from paper_2608_12913_amd import synth
from tests import parity

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_12913_amd import dcd
    dcd.lib()  # loud failure if the library is missing


def _runner():
    from paper_2608_12913_amd.runner import DeviceProblem
    return DeviceProblem


def _oracle_greedy(case, tokens, **kw):
    args = dict(theta=case.theta, s=case.s)
    args.update(kw)
    return oracle.verify("greedy", case.B, case.N, case.hp, case.hq, case.wp, case.wq, case.bias,
                         case.bias, case.parents, tokens, **args)


def _greedy_tokens(case, **kw):
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=kw.get("theta", case.theta), s=kw.get("s", case.s))
    return synth.greedy_tokens(case, rows["argmax"])


def _check_greedy(case, tokens, label, gates=None, **kw):
    """Greedy parity of every row and sequence; `gates` overrides the bounds of
    parity.check_gates (cases built on ties)."""
    _say(f"{label}: B={case.B} N={case.N} V={case.V} dp={case.dp} dq={case.dq} {case.dtype} {kw}")
    o = _oracle_greedy(case, tokens, **kw)
    dp = _runner().from_case(case, tokens, **kw)
    g = dp.run("greedy")
    report = {}
    amb = parity.compare_rows(g, o, np.arange(case.R), report)
    parity.compare_diagnostics(g, o, np.arange(case.R), kw.get("theta", case.theta),
                               kw.get("s", case.s), case.V, report)
    parity.compare_nodes(g, o, case.parents, amb, report)
    parity.compare_greedy(g, o, case.parents, amb, report)
    parity.check_walk_consistent(g, case.parents, tokens)
    parity.check_gates(report, **(gates or {}))
    _say(f"{label}: ok {report}")
    return g, o, dp


# ------------------------------------------------------------------ small cases
@pytest.mark.parametrize("seed", range(5))
def test_tiny_chain8_fp32(seed):
    case = synth.make_case("tiny_chain8", seed)
    _check_greedy(case, _greedy_tokens(case), f"tiny_chain8 seed {seed}")


@pytest.mark.parametrize("seed", range(3))
def test_small_tree_bf16_ragged_vocab(seed):
    # 4099 = 16 full 256-token tiles + 3; 128 rows = 2 row blocks
    case = synth.make_case("b8_tree64", seed, B=2, V=4099, dp=512, dq=256)
    _check_greedy(case, _greedy_tokens(case), f"small tree seed {seed}")


def test_ragged_hidden_and_rows():
    # K tails (520 and 136 are not multiples of 64 elements) and 70 rows (64 + 6)
    case = synth.make_case("b8_tree64", 7, N=70, V=1000, dp=520, dq=136)
    _check_greedy(case, _greedy_tokens(case), "ragged K and rows")


@pytest.mark.parametrize("seed", range(2))
def test_many_rows_ragged(seed):
    # 9 sequences x 64 nodes = 576 rows: the many-row LM-head kernel (256-row tiles,
    # the last one ragged), a ragged vocabulary and a K tail (200 = 3 chunks + 8 bf16)
    case = synth.make_case("b8_batch32x64", 30 + seed, B=9, V=4099, dp=512, dq=200)
    _check_greedy(case, _greedy_tokens(case), f"many rows seed {seed}")


@pytest.mark.parametrize("theta", [0.1, 0.0])
def test_many_rows_tiny_hidden_and_vocabulary(theta):
    # the many-row kernel's extreme tails: 8- and 24-element rows (one K chunk, most of
    # it past the row end) and a vocabulary of one full tile plus one token
    case = synth.make_case("b8_batch32x64", 33, B=9, V=257, dp=8, dq=24, theta=theta)
    assert case.R == 576
    _check_greedy(case, _greedy_tokens(case), f"many rows, tiny rows and vocabulary, theta {theta}")


def test_ragged_fp32():
    case = synth.make_case("tiny_chain8", 8, N=19, V=777, dp=100, dq=36)
    _check_greedy(case, _greedy_tokens(case), "ragged fp32")


@pytest.mark.parametrize("theta,s", [(0.0, 0.5), (1.0, 0.5), (0.1, 0.0), (0.1, 2.0), (0.001, 1.0)])
def test_mask_and_strength_settings(theta, s):
    case = synth.make_case("b8_tree64", 11, N=24, depth=5, max_children=4, V=2000, dp=256, dq=128)
    tokens = _greedy_tokens(case, theta=theta, s=s)
    _check_greedy(case, tokens, f"theta={theta} s={s}", theta=theta, s=s)


@pytest.mark.parametrize("theta,s", [(1.0, 0.5), (0.1, 0.0), (0.3, 2.0), (0.001, 1.0), (0.0, 0.5), (0.0, 2.0)])
def test_mask_and_strength_settings_many_rows(theta, s):
    # 576 rows: the many-row LM-head kernel under every mask width and strength, and
    # without the mask (its untruncated epilogue)
    case = synth.make_case("b8_batch32x64", 12, B=9, V=2000, dp=256, dq=128)
    tokens = _greedy_tokens(case, theta=theta, s=s)
    _check_greedy(case, tokens, f"many rows theta={theta} s={s}", theta=theta, s=s)


@pytest.mark.parametrize("seed", range(2))
def test_untruncated_target_ragged(seed):
    # theta = 0: every token is in the support (dense-logit path); 16 full tiles + 3
    # tokens, 2 row blocks
    case = synth.make_case("b8_tree64", 20 + seed, B=2, V=4099, dp=512, dq=256, theta=0.0)
    g, _, _ = _check_greedy(case, _greedy_tokens(case), f"untruncated ragged seed {seed}")
    assert np.all(g["row_stats"][:, oracle.RS_COUNT] == case.V)


def test_untruncated_target_fp32_ragged_k():
    case = synth.make_case("tiny_chain8", 22, N=19, V=777, dp=100, dq=36, theta=0.0)
    _check_greedy(case, _greedy_tokens(case), "untruncated fp32")


@pytest.mark.parametrize("B,theta", [(4, 0.1), (8, 0.1), (4, 0.0), (8, 0.0)])
def test_fp32_128_row_tiles(B, theta):
    # 100 and 200 rows go to the streaming kernel's 128-row workgroups (one row
    # block with non-temporal weight loads, two with cached ones), fp32 with K tails
    case = synth.make_case("tiny_chain8", 24 + B, B=B, N=25, V=777, dp=100, dq=36, theta=theta)
    _check_greedy(case, _greedy_tokens(case), f"fp32 {case.R} rows theta={theta}")


def test_flat_logits_every_token_in_mask():
    case = synth.make_case("tiny_chain8", 12, N=8, V=1500, dp=64, dq=32)
    case.wp[:] = 0
    case.wq[:] = 0
    case.bias[:] = 0
    tokens = _greedy_tokens(case)
    # every token ties: every row is ambiguous by construction (compared exactly below)
    g, o, _ = _check_greedy(case, tokens, "flat logits", gates=dict(max_ambiguous=case.R, max_gated=1))
    assert np.all(g["row_argmax"] == 0) and np.all(g["row_argmax_expert"] == 0)
    assert np.all(g["row_stats"][:, oracle.RS_COUNT] == 1500)
    assert np.all(np.isnan(g["row_kl"]))  # the mask holds every token: not computed
    np.testing.assert_allclose(g["row_stats"][:, oracle.RS_LOGZ], o["row_stats"][:, oracle.RS_LOGZ],
                               atol=1e-4)


def test_exact_integer_logits_theta_one():
    """Small-integer bf16 weights and states make every fp32 partial sum exact, so the
    set of tokens tied at the expert max (the theta = 1 mask) must match exactly."""
    rng = np.random.default_rng(13)
    case = synth.make_case("b8_tree64", 13, N=16, depth=4, max_children=4, V=3000, dp=128, dq=64)
    for name, d in (("hp", 128), ("hq", 64)):
        setattr(case, name, synth.bf16_bits(rng.integers(-2, 3, (case.R, d)).astype(np.float32)))
    case.wp = synth.bf16_bits(rng.integers(-1, 2, (3000, 128)).astype(np.float32))
    case.wq = synth.bf16_bits(rng.integers(-1, 2, (3000, 64)).astype(np.float32))
    case.bias[:] = 0
    tokens = _greedy_tokens(case, theta=1.0)
    _say("exact integer logits")
    o = _oracle_greedy(case, tokens, theta=1.0)
    g = _runner().from_case(case, tokens, theta=1.0).run("greedy")
    assert np.array_equal(g["row_argmax"], o["row_argmax"])
    assert np.array_equal(g["row_stats"][:, oracle.RS_COUNT], o["row_stats"][:, oracle.RS_COUNT])
    assert np.array_equal(g["accept_len"], o["accept_len"])
    assert np.array_equal(g["accept_path"], o["accept_path"])
    np.testing.assert_allclose(g["row_stats"][:, oracle.RS_MAXP], o["row_stats"][:, oracle.RS_MAXP],
                               rtol=0, atol=0)
    # the expert's top-1 among the tied tokens: the lowest id, exactly
    assert np.array_equal(g["row_argmax_expert"], o["row_diag"][:, oracle.RD_ARGMAX_P])


def test_exact_integer_logits_many_rows():
    """The same exactness through the many-row LM-head kernel: 9 sequences of 64 nodes
    (576 rows, the last 256-row tile ragged), a ragged vocabulary, two K chunks of the
    expert rows and one of the amateur rows.  The theta = 1 mask (the tokens tied at the
    expert max), the argmax, the expert max and the walk must match exactly."""
    rng = np.random.default_rng(15)
    V = 3001
    case = synth.make_case("b8_batch32x64", 15, B=9, V=V, dp=128, dq=64)
    assert case.R == 576
    for name, d in (("hp", 128), ("hq", 64)):
        setattr(case, name, synth.bf16_bits(rng.integers(-2, 3, (case.R, d)).astype(np.float32)))
    case.wp = synth.bf16_bits(rng.integers(-1, 2, (V, 128)).astype(np.float32))
    case.wq = synth.bf16_bits(rng.integers(-1, 2, (V, 64)).astype(np.float32))
    case.bias[:] = 0
    tokens = _greedy_tokens(case, theta=1.0)
    _say("exact integer logits, many rows")
    o = _oracle_greedy(case, tokens, theta=1.0)
    g = _runner().from_case(case, tokens, theta=1.0).run("greedy")
    assert np.array_equal(g["row_argmax"], o["row_argmax"])
    assert np.array_equal(g["row_stats"][:, oracle.RS_COUNT], o["row_stats"][:, oracle.RS_COUNT])
    assert np.array_equal(g["accept_len"], o["accept_len"])
    assert np.array_equal(g["accept_path"], o["accept_path"])
    np.testing.assert_allclose(g["row_stats"][:, oracle.RS_MAXP], o["row_stats"][:, oracle.RS_MAXP],
                               rtol=0, atol=0)
    assert np.array_equal(g["row_argmax_expert"], o["row_diag"][:, oracle.RD_ARGMAX_P])
    assert (o["accept_len"] > 0).sum() >= 6, "most sequences must accept along their spine"


def test_exact_integer_logits_untruncated_expert_top1():
    """theta = 0 with exact integer logits: many tokens tie at the expert max across
    vocabulary tiles; the expert's top-1 is the lowest of them, merged over tiles."""
    rng = np.random.default_rng(14)
    V = 4099
    case = synth.make_case("b8_tree64", 14, N=16, depth=4, max_children=4, V=V, dp=128, dq=64,
                           theta=0.0)
    for name, d in (("hp", 128), ("hq", 64)):
        setattr(case, name, synth.bf16_bits(rng.integers(-1, 2, (case.R, d)).astype(np.float32)))
    case.wp = synth.bf16_bits(rng.integers(-1, 2, (V, 128)).astype(np.float32))
    case.wq = synth.bf16_bits(rng.integers(-1, 2, (V, 64)).astype(np.float32))
    case.bias[:] = 0
    tokens = _greedy_tokens(case)
    _say("exact integer logits, theta 0")
    o = _oracle_greedy(case, tokens)
    g = _runner().from_case(case, tokens).run("greedy")
    zp = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias, theta=0.0,
                          s=case.s, want_logits=True)["zp"]
    cross = sum(len(set(np.flatnonzero(z == z.max()) // 256)) > 1 for z in zp)
    assert cross >= 4, "the case must tie the expert max across tiles"
    assert np.array_equal(g["row_argmax_expert"], o["row_diag"][:, oracle.RD_ARGMAX_P])
    np.testing.assert_allclose(g["row_kl"][:, 0], o["row_diag"][:, oracle.RD_KL_PQ], atol=parity.ATOL)
    np.testing.assert_allclose(g["row_kl"][:, 1], o["row_diag"][:, oracle.RD_KL_PCD],
                               atol=(1 + case.s) * parity.ATOL)


def test_exact_integer_logits_untruncated_many_rows():
    """theta = 0 through the many-row kernel with exact integer logits: the expert max
    ties across vocabulary tiles and across the two token halves of a tile, so the
    expert's top-1 (the lowest tied token) and the argmax are compared exactly."""
    rng = np.random.default_rng(16)
    V = 3001
    case = synth.make_case("b8_batch32x64", 16, B=9, V=V, dp=128, dq=64, theta=0.0)
    assert case.R == 576
    for name, d in (("hp", 128), ("hq", 64)):
        setattr(case, name, synth.bf16_bits(rng.integers(-1, 2, (case.R, d)).astype(np.float32)))
    case.wp = synth.bf16_bits(rng.integers(-1, 2, (V, 128)).astype(np.float32))
    case.wq = synth.bf16_bits(rng.integers(-1, 2, (V, 64)).astype(np.float32))
    case.bias[:] = 0
    tokens = _greedy_tokens(case)
    _say("exact integer logits, theta 0, many rows")
    o = _oracle_greedy(case, tokens)
    g = _runner().from_case(case, tokens).run("greedy")
    zp = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias, theta=0.0,
                          s=case.s, want_logits=True)["zp"]
    cross = sum(len(set(np.flatnonzero(z == z.max()) // 128)) > 1 for z in zp)
    assert cross >= 20, "the case must tie the expert max across token halves"
    assert np.array_equal(g["row_argmax_expert"], o["row_diag"][:, oracle.RD_ARGMAX_P])
    assert np.array_equal(g["row_argmax"], o["row_argmax"])
    assert np.array_equal(g["accept_len"], o["accept_len"])
    np.testing.assert_allclose(g["row_stats"][:, oracle.RS_MAXP], o["row_stats"][:, oracle.RS_MAXP],
                               rtol=0, atol=0)
    np.testing.assert_allclose(g["row_kl"][:, 0], o["row_diag"][:, oracle.RD_KL_PQ], atol=parity.ATOL)


def test_duplicate_sibling_tokens():
    case = synth.make_case("b8_tree64", 14, N=32, depth=4, max_children=6, V=1024, dp=128, dq=64)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s)
    tokens = np.zeros((1, case.N), np.int32)
    for i in range(1, case.N):  # every child carries its parent's argmax
        tokens[0, i] = rows["argmax"][case.parents[0, i]]
    _check_greedy(case, tokens, "duplicate siblings")


def test_sequence_status_codes():
    case = synth.make_case("tiny_chain8", 15, B=4, N=8, V=512, dp=64, dq=32)
    tokens = _greedy_tokens(case)
    case.parents[1, 3] = 6  # parent after child
    tokens[2, 4] = 512  # out of the vocabulary
    case.hp[3 * 8 + 2, 5] = np.inf  # non-finite logits in sequence 3
    _check_greedy(case, tokens, "status codes")


@pytest.mark.parametrize("which,rows", [("separate", "few"), ("none", "few"), ("separate", "many"),
                                        ("none", "many")])
def test_bias_variants(which, rows):
    # one bias per model (the amateur's differs from the expert's), or none at all
    # (null pointers: both models' logits unbiased); "many": 576 rows, through the
    # many-row LM-head kernel
    if rows == "few":
        case = synth.make_case("b8_tree64", 70, N=20, depth=4, max_children=4, V=1500, dp=128, dq=64)
    else:
        case = synth.make_case("b8_batch32x64", 71, B=9, V=1500, dp=128, dq=64)
    zero = np.zeros(case.V, np.float32)
    if which == "separate":
        bp, bq = case.bias, (0.5 * case.bias - 0.25).astype(np.float32)
    else:
        bp = bq = None
    op = bp if bp is not None else zero
    oq = bq if bq is not None else zero
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, op, oq, theta=case.theta, s=case.s)
    tokens = synth.greedy_tokens(case, rows["argmax"])
    _say(f"bias {which}: B={case.B} N={case.N} V={case.V} R={case.R}")
    o = oracle.verify("greedy", case.B, case.N, case.hp, case.hq, case.wp, case.wq, op, oq,
                      case.parents, tokens, theta=case.theta, s=case.s)
    g = _runner().from_case(case, tokens, bias_p=bp, bias_q=bq).run("greedy")
    report = {}
    amb = parity.compare_rows(g, o, np.arange(case.R), report)
    parity.compare_nodes(g, o, case.parents, amb, report)
    parity.compare_greedy(g, o, case.parents, amb, report)
    parity.check_gates(report)
    _say(f"bias {which}: ok {report}")


def test_repeated_calls_are_bit_identical():
    case = synth.make_case("b8_tree64", 16, N=40, V=3001, dp=256, dq=128)
    tokens = _greedy_tokens(case)
    dp = _runner().from_case(case, tokens)
    a = dp.run("greedy")
    b = dp.run("greedy")
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


def test_workspace_reused_across_problems():
    """One workspace, filled with garbage, serves problems of different shapes in
    turn, some of them only through dcd_lmhead_partials.  The LM-head launch clears
    the row bounds of each call itself: a problem whose logits are four times
    smaller than the previous one's (so stale bounds would drop every tile holding
    its mask members) must come out bit for bit as on a fresh workspace."""
    from paper_2608_12913_amd import dcd
    big = synth.make_case("b8_tree64", 80, N=40, depth=5, max_children=6, V=6000, dp=256, dq=128)
    small = synth.make_case("b8_tree64", 81, B=3, N=24, depth=4, max_children=4, V=6000, dp=256,
                            dq=128, h_scale=1.0)
    runs = []
    for case in (big, small):
        dp = _runner().from_case(case, _greedy_tokens(case))
        runs.append((dp, dp.run("greedy")))
    need = max(dp.ws_bytes for dp, _ in runs)
    shared = torch.full((need,), 0xAB, dtype=torch.uint8, device="cuda:0")
    stream = torch.cuda.current_stream()
    for step, k in enumerate((0, 1, 1, 0, 1)):
        dp, ref = runs[k]
        other = runs[1 - k][0]
        # the other problem's LM heads alone on the same workspace first
        dcd.lmhead_partials(other.problem, other.inputs, False, shared, need, stream)
        dcd.verify_greedy(dp.problem, dp.inputs, dp.outputs, shared, need, stream)
        torch.cuda.synchronize()
        got = {k2: getattr(dp, k2).cpu().numpy() for k2 in ref}
        for k2 in ref:
            assert np.array_equal(ref[k2].view(np.uint8), got[k2].view(np.uint8)), (step, k2)
    _say("workspace reuse: ok")


# ------------------------------------------------------------------ sampled
def _sampled_setup(case):
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, temperature=case.T, want_logits=True)
    parent_logits = np.zeros_like(rows["zp"])
    parent_logits[1:] = rows["zp"][:-1]
    return synth.sampled_draft(case, parent_logits)


def _oracle_sample(case, probs, tokens):
    """The oracle's sampled verification and log pi_CD of every row (for the gates)."""
    o = oracle.verify("sample", case.B, case.N, case.hp, case.hq, case.wp, case.wq, case.bias,
                      case.bias, case.parents, tokens, theta=case.theta, s=case.s,
                      temperature=case.T, draft_probs=probs, u_acc=case.u_acc, u_res=case.u_res)
    lp = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                          theta=case.theta, s=case.s, temperature=case.T, want_lpcd=True)["lpcd"]
    return o, lp


def _compare_sampled(g, o, lp, case, probs, tokens, report, dev, gates=None, delta=None):
    """Rows, diagnostics, nodes and walks of a sampled verification; `dev` (the
    problem on the GPU) also gives the dense target rows that measure the error
    bound of the walk comparison."""
    amb = parity.compare_rows(g, o, np.arange(case.R), report)
    parity.compare_diagnostics(g, o, np.arange(case.R), case.theta, case.s, case.V, report)
    parity.compare_nodes(g, o, case.parents, amb, report)
    boundary = o["row_gap"] <= parity.BOUNDARY_GATE
    if delta is None:
        pg = dev.propose(case.u_res)["probs"]
        parity.measure_target_error(pg, lp, boundary, report)
        del pg
    parity.compare_sample(g, o, lp, probs, case.parents, tokens, case.u_acc, case.u_res, boundary,
                          report, delta=delta)
    # the ratio pi_CD / pi_e of every draft token: its relative error is the error of
    # log pi_CD plus the rounding of the reported ratio, an fp32 division (the walk
    # itself divides in fp64)
    gr = g["node_stats"][:, oracle.NS_RATIO].astype(np.float64)
    orat = o["node_stats"][:, oracle.NS_RATIO]
    fin = np.isfinite(orat) & (orat > 1e-30)
    assert np.all(np.abs(np.log(gr[fin] / orat[fin])) <= report["walk_delta"] + 2.0 ** -22)
    parity.check_gates(report, **(gates or {}))


def _check_sample(case, probs, tokens, label, gates=None):
    _say(f"{label}: B={case.B} N={case.N} V={case.V} {case.dtype} theta={case.theta} s={case.s}")
    o, lp = _oracle_sample(case, probs, tokens)
    dev = _runner().from_case(case, tokens, draft_probs=probs)
    g = dev.run("sample")
    report = {}
    _compare_sampled(g, o, lp, case, probs, tokens, report, dev, gates)
    _say(f"{label}: ok {report}")
    return g, o


@pytest.mark.parametrize("theta,T", [(1.0, 1.0), (0.1, 0.7), (0.0, 1.3)])
def test_sampled_chains_mask_and_temperature(theta, T):
    # theta = 1 (the target keeps only the tokens tied at the expert max) and
    # temperatures other than 1 (dividing both models' logits before the mask)
    case = synth.make_case("s8_chain16x8", 72, V=3000, dp=256, dq=128, theta=theta, T=T)
    probs, tokens = _sampled_setup(case)
    _check_sample(case, probs, tokens, f"sampled theta={theta} T={T}")


@pytest.mark.parametrize("theta", [0.1, 0.0])
def test_root_only_sequences(theta):
    # N = 1, nothing drafted: greedy emits the root row's argmax, sampled verification
    # the bonus draw from pi_CD of the root row
    case = synth.make_case("tiny_chain8", 60, B=3, N=1, V=1000, dp=64, dq=32, theta=theta)
    g, _, _ = _check_greedy(case, _greedy_tokens(case), f"root only theta={theta}")
    assert np.all(g["accept_len"] == 0)
    case = synth.make_case("s8_chain16x8", 62, B=3, N=1, V=1000, dp=64, dq=32, theta=theta)
    probs, tokens = _sampled_setup(case)
    g, _ = _check_sample(case, probs, tokens, f"root only sampled theta={theta}")
    assert np.all(g["accept_len"] == 0)


@pytest.mark.parametrize("theta", [0.5, 0.0])
def test_vocabulary_smaller_than_a_tile(theta):
    # 5 tokens and 8-element rows: one ragged vocabulary tile and one 16-byte K chunk
    case = synth.make_case("b8_tree64", 61, B=2, N=3, V=5, dp=8, dq=8, theta=theta)
    _check_greedy(case, _greedy_tokens(case), f"V=5 theta={theta}")
    case = synth.make_case("s8_chain16x8", 63, B=2, N=3, V=5, dp=8, dq=8, theta=theta)
    probs, tokens = _sampled_setup(case)
    _check_sample(case, probs, tokens, f"V=5 sampled theta={theta}")


@pytest.mark.parametrize("seed,theta,s", [(0, 0.1, 0.5), (1, 0.0, 0.5), (2, 0.3, 1.0), (3, 0.1, 0.0)])
def test_sampled_chains_small(seed, theta, s):
    case = synth.make_case("s8_chain16x8", seed, V=3000, dp=256, dq=128, theta=theta, s=s)
    probs, tokens = _sampled_setup(case)
    _check_sample(case, probs, tokens, f"sampled small seed {seed}")


def test_sampled_always_accept_and_reject():
    case = synth.make_case("s8_chain16x8", 5, B=4, N=6, V=700, dp=128, dq=64)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, want_lpcd=True)
    probs = np.zeros((case.R, case.V), np.float32)
    tokens = np.zeros((case.B, case.N), np.int32)
    for r in range(case.R):
        i = r % case.N
        if i == 0:
            continue
        p = np.exp(rows["lpcd"][r - 1])
        if r // case.N < 2:  # proposal = target: always accepted
            probs[r] = p
            tokens[r // case.N, i] = int(np.argmax(p))
        else:  # one-hot on a masked token: rejected at node 1
            t = int(np.flatnonzero(p == 0)[r % 5])
            probs[r, t] = 1.0
            tokens[r // case.N, i] = t
    case.u_acc = np.minimum(case.u_acc, np.float32(0.99))
    g, o = _check_sample(case, probs, tokens, "always accept / reject")
    assert np.all(g["accept_len"][:2] == case.N - 1) and np.all(g["accept_len"][2:] == 0)


def test_untruncated_sampled_residual_over_vocabulary():
    """theta = 0: a one-hot proposal on the target's least likely token is rejected at
    node 1 and the residual, max(0, pi_CD - pi_e), spans the whole vocabulary."""
    case = synth.make_case("s8_chain16x8", 23, B=4, N=6, V=1500, dp=128, dq=64, theta=0.0)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=0.0, s=case.s, want_lpcd=True)
    probs = np.zeros((case.R, case.V), np.float32)
    tokens = np.zeros((case.B, case.N), np.int32)
    for r in range(case.R):
        i = r % case.N
        if i == 0:
            continue
        p = np.exp(rows["lpcd"][r - 1])
        if r // case.N < 2:  # proposal = target: always accepted
            probs[r] = p
            tokens[r // case.N, i] = int(np.argmax(p))
        else:
            t = int(np.argmin(p))
            probs[r, t] = 1.0
            tokens[r // case.N, i] = t
    case.u_acc = np.maximum(np.minimum(case.u_acc, np.float32(0.99)), np.float32(1e-3))
    g, o = _check_sample(case, probs, tokens, "untruncated accept / reject")
    assert np.all(g["accept_len"][:2] == case.N - 1) and np.all(g["accept_len"][2:] == 0)
    assert np.all(g["row_stats"][:, oracle.RS_COUNT] == case.V)


def _sampled_tree_setup(case):
    """Proposals of a tree: node i's from the expert logits of its parent row."""
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, temperature=case.T, want_logits=True)
    parent_logits = np.zeros_like(rows["zp"])
    for r in range(case.R):
        i = r % case.N
        if i:
            parent_logits[r] = rows["zp"][r - i + case.parents[r // case.N, i]]
    return synth.sampled_draft(case, parent_logits)


@pytest.mark.parametrize("seed,theta,s", [(0, 0.1, 0.5), (1, 0.0, 0.5), (2, 0.3, 1.0)])
def test_sampled_trees_small(seed, theta, s):
    """Sampled verification of draft trees: siblings tried in index order against the
    residual of the rejected ones (several rejections per node occur here)."""
    case = synth.make_case("s8_chain16x8", 40 + seed, B=6, N=24, tree="tree", depth=4,
                           max_children=5, V=2500, dp=256, dq=128, theta=theta, s=s)
    probs, tokens = _sampled_tree_setup(case)
    g, o = _check_sample(case, probs, tokens, f"sampled trees seed {seed}")
    walked = np.isfinite(o["walk_ratio"]) | np.isinf(o["walk_ratio"])
    _say(f"sampled trees seed {seed}: {int(walked.sum())} nodes tested on the walks, "
         f"accept lengths {g['accept_len'].tolist()}")


@pytest.mark.parametrize("seed,theta,s", [(3, 0.1, 0.5), (4, 0.3, 1.0), (5, 0.0, 0.5)])
def test_sampled_trees_many_rows(seed, theta, s):
    """Sampled verification of 9 trees of 64 nodes (576 rows): the many-row LM-head
    kernel feeding the walk decisions settled per row."""
    case = synth.make_case("s8_chain16x8", 40 + seed, B=9, N=64, tree="tree", depth=6,
                           max_children=4, V=2500, dp=256, dq=128, theta=theta, s=s)
    assert case.R == 576 and case.dtype == "bf16"
    probs, tokens = _sampled_tree_setup(case)
    g, o = _check_sample(case, probs, tokens, f"sampled trees, many rows, seed {seed}")
    _say(f"sampled trees, many rows, seed {seed}: accept lengths {g['accept_len'].tolist()}")


@pytest.mark.parametrize("theta", [0.1, 0.0])
def test_sampled_trees_odd_node_count(theta):
    # 23 nodes per sequence: the walk's per-node LDS state at an odd count
    case = synth.make_case("s8_chain16x8", 48, B=3, N=23, tree="tree", depth=4,
                           max_children=5, V=2000, dp=128, dq=64, theta=theta)
    probs, tokens = _sampled_tree_setup(case)
    _check_sample(case, probs, tokens, f"sampled trees N=23 theta={theta}")


def test_sampled_tree_forced_paths():
    """Star trees of three children.  Sequence 0: child 1 is one-hot on a masked token
    (rejected, and its residual is pi_CD itself), child 2 proposes pi_CD exactly and
    carries its argmax (ratio 1: accepted).  Sequence 1: every child is one-hot on a
    masked token, so all are rejected and the token is drawn from pi_CD."""
    case = synth.make_case("s8_chain16x8", 50, B=2, N=4, tree="chain", V=900, dp=128, dq=64)
    case.parents[:] = np.array([-1, 0, 0, 0])
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, want_lpcd=True)
    probs = np.zeros((case.R, case.V), np.float32)
    tokens = np.zeros((case.B, case.N), np.int32)
    for b in range(2):
        p = np.exp(rows["lpcd"][b * 4])
        masked = np.flatnonzero(p == 0)
        for i in (1, 2, 3):
            t = int(masked[7 * i + b])
            if b == 0 and i == 2:
                probs[b * 4 + i] = p
                t = int(np.argmax(p))
            else:
                probs[b * 4 + i, t] = 1.0
            tokens[b, i] = t
    case.u_acc = np.minimum(case.u_acc, np.float32(0.99))
    g, o = _check_sample(case, probs, tokens, "sampled star trees")
    assert list(g["accept_path"][0][:2]) == [0, 2] and g["accept_len"][0] == 1
    assert g["accept_len"][1] == 0


@pytest.mark.parametrize("seed,B,V,dtype", [(0, 4, 2500, "bf16"), (1, 3, 1499, "f32"), (2, 1, 3001, "bf16"),
                                           (3, 2, 130, "bf16")])
def test_untruncated_sampled_trees_spread_walk(seed, B, V, dtype):
    """theta = 0 with at most 4 sequences: each sequence's walk is spread over 64
    workgroups, one slice of the vocabulary each (ragged at the vocabulary's end;
    with V = 130 most slices are empty), with several rejections per node."""
    case = synth.make_case("s8_chain16x8", 80 + seed, B=B, N=24, tree="tree", depth=4,
                           max_children=5, V=V, dp=256, dq=128, theta=0.0, dtype=dtype)
    probs, tokens = _sampled_tree_setup(case)
    g, o = _check_sample(case, probs, tokens, f"spread walk seed {seed} B={B} V={V} {dtype}")
    assert np.all(g["status"] == 0)
    walked = np.isfinite(o["walk_ratio"]) | np.isinf(o["walk_ratio"])
    _say(f"spread walk seed {seed}: {int(walked.sum())} nodes tested, accept lengths "
         f"{g['accept_len'].tolist()}")


@pytest.mark.parametrize("B", [64, 65])
def test_untruncated_sampled_many_sequences(B):
    """theta = 0: 64 sequences get 4 workgroups each for their walks (the fewest the
    spread walk takes); 65 are walked by the finish kernel, one workgroup each."""
    case = synth.make_case("s8_chain16x8", 90 + B, B=B, N=3, V=997, dp=64, dq=32, theta=0.0)
    probs, tokens = _sampled_setup(case)
    g, _ = _check_sample(case, probs, tokens, f"untruncated sampled B={B}")
    assert np.all(g["status"] == 0)


def test_sampled_tree_at_the_node_limit():
    """4096 nodes (the largest sequence): the walk's state fills most of the LDS."""
    case = synth.make_case("s8_chain16x8", 51, B=1, N=4096, tree="tree", depth=12,
                           max_children=6, V=300, dp=64, dq=32, theta=0.1)
    probs, tokens = _sampled_tree_setup(case)
    _check_sample(case, probs, tokens, "sampled tree of 4096 nodes")



def test_sampled_settled_and_walked_sequences_together():
    """theta > 0: each row settles its children's accept ratios and its terminal draw
    unless a node has more than 64 children, its children's proposals at its mask
    members exceed 4096 values, or it has more than 1024 mask members; such a sequence
    is walked in the sequence phase instead.  One call holds one sequence of each:
    0, a star of 80 children; 1, a tree that settles; 2, a star of 40 children under a
    root with more than 4096 / 40 mask members; 3, a chain with a row of more than 1024
    mask members (its hidden state scaled down, flattening the expert)."""
    N = 81
    case = synth.make_case("s8_chain16x8", 60, B=4, N=N, tree="tree", depth=4, max_children=5,
                           V=3000, dp=64, dq=32, theta=0.0005, dtype="f32")
    star = np.arange(N) - 1
    star[1:81] = 0
    case.parents[0] = star
    star40 = np.arange(N) - 1
    star40[1:41] = 0
    star40[41] = 40
    case.parents[2] = star40
    case.parents[3] = synth.chain_parents(N)
    case.hp[3 * N + 3] *= np.float32(0.02)
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s, want_lpcd=True)
    members = np.isfinite(rows["lpcd"]).sum(1).reshape(case.B, N)
    kids = np.stack([np.bincount(case.parents[b][1:], minlength=N) for b in range(case.B)])
    assert kids[0, 0] == 80 > 64
    assert kids[1].max() <= 64 and members[1].max() <= 1024 and (kids[1] * members[1]).max() <= 4096
    assert kids[2].max() <= 64 and members[2].max() <= 1024 and kids[2, 0] * members[2, 0] > 4096
    assert members[3].max() > 1024
    probs, tokens = _sampled_tree_setup(case)
    g, _ = _check_sample(case, probs, tokens, "settled and walked sequences")
    assert np.all(g["status"] == 0)

# ------------------------------------------------------------------ full-size workloads
def _spine_tokens(case, **kw):
    """Draft tokens with one full-depth path that copies the target argmax."""
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=kw.get("theta", case.theta), s=kw.get("s", case.s))
    return synth.greedy_tokens(case, rows["argmax"], spine=True)


def _depth(parents):
    return len(synth.deepest_path(parents)) - 1


@pytest.mark.slow
def test_full_b8_tree64():
    case = synth.make_case("b8_tree64", 0)
    _say("b8_tree64: oracle over all 64 rows (coin tokens)")
    _check_greedy(case, _greedy_tokens(case), "b8_tree64 seed 0")


@pytest.mark.slow
@pytest.mark.parametrize("workload", ["b8_tree64", "b70_tree64"])
def test_full_tree_accepts_full_depth(workload):
    """The headline shapes with one deepest path copying the target argmax: the walk
    accepts it to the tree's full depth (8), node by node as the oracle does."""
    case = synth.make_case(workload, 0)
    _say(f"{workload}: oracle over all 64 rows (one full-depth path)")
    g, o, _ = _check_greedy(case, _spine_tokens(case), f"{workload} full-depth path")
    depth = _depth(case.parents[0])
    assert depth == 8
    assert o["accept_len"][0] == depth and g["accept_len"][0] == depth


@pytest.mark.slow
def test_full_b8_tree64_untruncated():
    case = synth.make_case("b8_tree64", 0, theta=0.0)
    _say("b8_tree64 theta 0: oracle over all 64 rows")
    g, o, _ = _check_greedy(case, _spine_tokens(case), "b8_tree64 theta 0")
    assert g["accept_len"][0] == _depth(case.parents[0])


@pytest.mark.slow
def test_full_b70_tree64():
    case = synth.make_case("b70_tree64", 0)
    _say("b70_tree64: oracle over all 64 rows (coin tokens)")
    _check_greedy(case, _greedy_tokens(case), "b70_tree64 seed 0")


def _full_sampled_setup(case):
    # stand-in drafter: expert logits of every parent row from a plain fp32 matmul
    dev = torch.device("cuda:0")
    hp = torch.from_numpy(synth.bf16_to_f32(case.hp)).to(dev)
    wp = torch.from_numpy(synth.bf16_to_f32(case.wp)).to(dev)
    z = (hp @ wp.T + torch.from_numpy(case.bias).to(dev)).double().cpu().numpy()
    del hp, wp
    parent_logits = np.zeros_like(z)
    parent_logits[1:] = z[:-1]
    return synth.sampled_draft(case, parent_logits)


@pytest.mark.slow
@pytest.mark.parametrize("theta", [0.1, 0.0])
def test_full_s8_chain16x8(theta):
    """All 16 chains of the sampled workload against the oracle."""
    case = synth.make_case("s8_chain16x8", 0, theta=theta)
    probs, tokens = _full_sampled_setup(case)
    _say(f"s8_chain16x8 theta {theta}: oracle over all 16 sequences")
    o, lp = _oracle_sample(case, probs, tokens)
    dev = _runner().from_case(case, tokens, draft_probs=probs)
    g = dev.run("sample")
    report = {}
    _compare_sampled(g, o, lp, case, probs, tokens, report, dev)
    assert np.all(g["status"] == 0)
    _say(f"s8_chain16x8: ok {report}; accept lengths {g['accept_len'].tolist()}")


@pytest.mark.slow
@pytest.mark.parametrize("theta", [0.1, 0.0])
def test_full_b8_tree64_sampled(theta):
    """The sampled 64-node tree against the oracle (theta = 0: the walk spread over 64
    workgroups)."""
    case = synth.make_case("b8_tree64", 0, mode="sample", theta=theta)
    probs, tokens = _full_sampled_setup(case)
    _say(f"b8_tree64 sampled theta {theta}: oracle")
    o, lp = _oracle_sample(case, probs, tokens)
    dev = _runner().from_case(case, tokens, draft_probs=probs)
    g = dev.run("sample")
    report = {}
    _compare_sampled(g, o, lp, case, probs, tokens, report, dev)
    assert np.all(g["status"] == 0)
    _say(f"b8_tree64 sampled: ok {report}; accept lengths {g['accept_len'].tolist()}")


@pytest.mark.slow
@pytest.mark.parametrize("theta", [0.1, 0.0])
def test_full_b8_batch32x64(theta):
    # theta 0.1: the many-row kernel; theta 0: the streaming kernel's 64-row shape
    # with 32 row blocks per tile.  Eight sequences spread over the batch (rows in
    # every 256-row tile of the many-row kernel) are compared in full; their draft
    # trees hold a full-depth path copying the oracle's argmax.  Elsewhere the
    # tokens are random.
    case = synth.make_case("b8_batch32x64", 0, theta=theta)
    seqs = [0, 5, 9, 14, 18, 23, 27, 31]
    rows = np.concatenate([np.arange(b * 64, b * 64 + 64) for b in seqs])
    _say(f"b8_batch32x64 theta={theta}: oracle over sequences {seqs}")
    o_rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                              theta=case.theta, s=case.s, rows=rows)
    amax = np.full(case.R, -1, np.int32)
    amax[rows] = o_rows["argmax"]
    tokens = synth.greedy_tokens(case, amax, spine=True)
    o = oracle.verify("greedy", len(seqs), 64, case.hp[rows], case.hq[rows], case.wp, case.wq,
                      case.bias, case.bias, case.parents[seqs], tokens[seqs], theta=case.theta,
                      s=case.s)
    g = _runner().from_case(case, tokens).run("greedy")
    sel = dict(accept_len=g["accept_len"][seqs], accept_path=g["accept_path"][seqs],
               next_token=g["next_token"][seqs], status=g["status"][seqs],
               row_argmax=g["row_argmax"][rows], row_stats=g["row_stats"][rows],
               node_stats=g["node_stats"][rows], row_argmax_expert=g["row_argmax_expert"][rows],
               row_kl=g["row_kl"][rows])
    report = {}
    amb = parity.compare_rows(sel, o, np.arange(len(rows)), report)
    parity.compare_diagnostics(sel, o, np.arange(len(rows)), case.theta, case.s, case.V, report)
    parity.compare_nodes(sel, o, case.parents[seqs], amb, report)
    parity.compare_greedy(sel, o, case.parents[seqs], amb, report)
    parity.check_walk_consistent(g, case.parents, tokens)
    parity.check_gates(report)
    for k, b in enumerate(seqs):
        assert sel["accept_len"][k] == _depth(case.parents[b])
    _say(f"b8_batch32x64 theta={theta}: ok {report}; accept lengths "
         f"{sel['accept_len'].tolist()}")


@pytest.mark.slow
@pytest.mark.parametrize("workload,mode,theta", [("b8_tree64", "greedy", 0.1), ("s8_chain16x8", "sample", 0.1),
                                                 ("b8_tree64", "sample", 0.1), ("b8_tree64", "sample", 0.0),
                                                 ("b8_batch32x64", "greedy", 0.1)])
def test_full_size_repeated_calls_are_bit_identical(workload, mode, theta):
    """Which vocabulary tiles keep their candidates depends on when each reads the
    running bound; the outputs must not.  Full-size calls (64 rows: one row block per
    tile; 128 rows: the 128-row shape, 501 tiles on 256 CUs in two rounds; 2048 rows:
    the many-row kernel) repeated with another call of a different problem in between,
    every output compared bit for bit."""
    case = synth.make_case(workload, 0, mode=mode, theta=theta)
    if mode == "sample":
        probs, tokens = _full_sampled_setup(case)
    elif case.R > 512:  # the coin rule with every token uniform: no oracle rows needed
        probs, tokens = None, synth.greedy_tokens(case, np.full(case.R, -1, np.int32))
    else:
        probs, tokens = None, _spine_tokens(case)
    _say(f"{workload} {mode}: repeated calls")
    dp = _runner().from_case(case, tokens, draft_probs=probs)
    a = dp.run(mode)
    other = synth.make_case("b8_tree64", 3, N=32, depth=5, max_children=4)
    _runner().from_case(other, _greedy_tokens(other)).run("greedy")
    b = dp.run(mode)
    c = dp.run(mode)
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k
        assert np.array_equal(a[k].view(np.uint8), c[k].view(np.uint8)), k


# ------------------------------------------------------------------ final RMS normalisation
def _pre_norm(case, seed, eps=1e-5):
    """Un-normalised rows (the normalised synthetic states times a per-row scale in
    [0.5, 8]) and bf16/fp32 scales g ~ 1 + 0.1 N(0, 1); returns the normalised rows the
    oracle computes and the inputs the library gets."""
    rng = np.random.default_rng(seed)
    to = (lambda a: synth.bf16_bits(a)) if case.dtype == "bf16" else (lambda a: a.astype(np.float32))
    pre, norms, post = {}, {}, {}
    for name, d in (("hp", case.dp), ("hq", case.dq)):
        x = oracle.as_f32(getattr(case, name)) * rng.uniform(0.5, 8.0, (case.R, 1)).astype(np.float32)
        pre[name] = to(x)
        norms[name] = to((1 + 0.1 * rng.standard_normal(d)).astype(np.float32))
        post[name] = oracle.rmsnorm(pre[name], norms[name], eps)
    return pre, norms, post


def _check_final_norm(case, label, mode="greedy", eps=1e-5):
    pre, norms, post = _pre_norm(case, 70, eps)
    _say(f"{label}: final norm, B={case.B} N={case.N} V={case.V} {case.dtype} theta={case.theta}")
    # the oracle on the rows it normalised itself
    case.hp, case.hq = post["hp"], post["hq"]
    if mode == "greedy":
        tokens = _greedy_tokens(case)
        o = _oracle_greedy(case, tokens)
        probs = None
    else:
        probs, tokens = _sampled_tree_setup(case)
        o, lp = _oracle_sample(case, probs, tokens)
    # the library on the rows before the normalisation
    dev = _runner().from_case(case, tokens, draft_probs=probs, hp=pre["hp"], hq=pre["hq"],
                              norm_p=norms["hp"], norm_q=norms["hq"], norm_eps=eps)
    g = dev.run(mode)
    report = {}
    amb = parity.compare_rows(g, o, np.arange(case.R), report)
    parity.compare_nodes(g, o, case.parents, amb, report)
    gates = None
    if mode == "greedy":
        parity.compare_greedy(g, o, case.parents, amb, report)
    else:
        # The oracle normalises with fp64 statistics, so an element of a row can round
        # to the neighbouring bf16 value: the logits then differ by more than fp32
        # accumulation alone (up to about 2e-4, within ATOL).  The walk is gated with
        # the error measured at every token, capped at ATOL instead of DELTA_P / 2,
        # and one of the four walks may be gated by it.
        boundary = o["row_gap"] <= parity.BOUNDARY_GATE
        parity.measure_target_error(dev.propose(case.u_res)["probs"], lp, boundary, report,
                                    cap=parity.ATOL)
        parity.compare_sample(g, o, lp, probs, case.parents, tokens, case.u_acc, case.u_res,
                              boundary, report)
        gates = dict(max_gated=1)
    parity.check_gates(report, **(gates or {}))
    _say(f"{label}: ok {report}")


def test_final_norm_masked_bf16():
    case = synth.make_case("b8_tree64", 71, B=2, V=4099, dp=512, dq=256)
    _check_final_norm(case, "final norm masked")


def test_final_norm_untruncated_bf16():
    case = synth.make_case("b8_tree64", 72, B=2, V=4099, dp=512, dq=256, theta=0.0)
    _check_final_norm(case, "final norm untruncated")


def test_final_norm_fp32_many_rows_and_sampled():
    case = synth.make_case("tiny_chain8", 73, N=19, V=777, dp=100, dq=36)
    _check_final_norm(case, "final norm fp32")
    case = synth.make_case("b8_batch32x64", 74, B=9, V=4099, dp=512, dq=200)
    _check_final_norm(case, "final norm many rows")
    case = synth.make_case("s8_chain16x8", 75, B=4, N=16, tree="tree", depth=4, max_children=4,
                           V=2000, dp=256, dq=128)
    _check_final_norm(case, "final norm sampled trees", mode="sample")
