"""GPU: the allocation-free entry point (dcd_verify_greedy_noalloc) against
dcd_verify_greedy with a caller's workspace, through the C ABI: two calls in a row,
the second on a smaller problem, every output bit for bit (the same kernels on the
same inputs)."""
import numpy as np
import pytest

import oracle
from paper_2608_12913_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_12913_amd import dcd
    dcd.lib()


def _outputs_equal(a, b):
    for k in a:
        assert np.array_equal(np.asarray(a[k]).view(np.uint8), np.asarray(b[k]).view(np.uint8)), k


def _noalloc_run(dev):
    """The same problem and output buffers as `dev`, through the allocation-free call."""
    from paper_2608_12913_amd import dcd
    for t in (dev.accept_len, dev.accept_path, dev.next_token, dev.status, dev.row_argmax,
              dev.row_stats, dev.node_stats, dev.row_argmax_expert, dev.row_kl):
        t.fill_(-7)
    dcd.verify_greedy_noalloc(dev.problem, dev.inputs, dev.outputs,
                              torch.cuda.current_stream(dev.device))
    torch.cuda.synchronize(dev.device)
    return {k: getattr(dev, k).cpu().numpy() for k in
            ("accept_len", "accept_path", "next_token", "status", "row_argmax", "row_stats",
             "node_stats", "row_argmax_expert", "row_kl")}


def _tokens(case):
    rows = oracle.eval_rows(case.hp, case.hq, case.wp, case.wq, case.bias, case.bias,
                            theta=case.theta, s=case.s)
    return synth.greedy_tokens(case, rows["argmax"], spine=True)


def test_noalloc_matches_workspace_entry_point_twice_shrinking():
    from paper_2608_12913_amd.runner import DeviceProblem
    # first call: 64-row tree, ragged vocabulary; second: a smaller chain problem
    big = synth.make_case("b8_tree64", 90, V=20000, dp=512, dq=256)
    small = synth.make_case("tiny_chain8", 91, dtype="bf16", N=6, V=3001, dp=128, dq=64)
    print("[noalloc] first call: 64 rows, V=20000", flush=True)
    db = DeviceProblem.from_case(big, _tokens(big))
    ref_big = db.run("greedy")
    got_big = _noalloc_run(db)
    _outputs_equal(ref_big, got_big)
    assert got_big["status"][0] == 0 and got_big["accept_len"][0] == 8
    print("[noalloc] second call: 6 rows, V=3001", flush=True)
    ds = DeviceProblem.from_case(small, _tokens(small))
    ref_small = ds.run("greedy")
    got_small = _noalloc_run(ds)
    _outputs_equal(ref_small, got_small)
    assert got_small["accept_len"][0] == small.N - 1
    # and once more at full size after the small one (the array keeps the last
    # call's contents; every call clears what it reads)
    _outputs_equal(ref_big, _noalloc_run(db))


def test_noalloc_headline_shape_untruncated():
    """The 8B/1B 64-node tree at plaus_thresh 0 (the largest layout the array takes)."""
    from paper_2608_12913_amd.runner import DeviceProblem
    case = synth.make_case("b8_tree64", 0, theta=0.0)
    print("[noalloc] b8_tree64 theta 0", flush=True)
    dev = DeviceProblem.from_case(case, np.zeros((1, 64), np.int32))
    first = dev.run("greedy")
    dev.set_tokens(synth.greedy_tokens(case, first["row_argmax"], spine=True))
    ref = dev.run("greedy")
    _outputs_equal(ref, _noalloc_run(dev))
    assert ref["accept_len"][0] == 8
