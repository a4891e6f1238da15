"""The measurement probes on the GPU: they run, and report plausible rates."""
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _timed(fn, n):
    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(n):
        fn()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n * 1e-3


def test_stream_read_probe():
    from paper_2608_12913_amd import dcd
    nbytes = 1 << 30
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda:0")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    stream = torch.cuda.current_stream()
    t = _timed(lambda: dcd.probe_stream_read(buf, nbytes, sink, stream), 5)
    gbs = nbytes / t / 1e9
    print(f"[probe] stream read {gbs:.0f} GB/s", flush=True)
    assert 1000 < gbs < 8000
    assert int(sink.item()) == 0  # ones XOR to zero, never the sink pattern


def test_mfma_probe():
    from paper_2608_12913_amd import dcd
    wg, iters = 512, 2000
    sink = torch.zeros(wg * 256, dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.current_stream()
    flops = dcd.probe_mfma_bf16(wg, iters, sink, stream)
    assert flops == wg * 4 * iters * 8 * 16384
    t = _timed(lambda: dcd.probe_mfma_bf16(wg, iters, sink, stream), 3)
    tf = flops / t / 1e12
    print(f"[probe] bf16 MFMA {tf:.0f} TFLOP/s", flush=True)
    assert 100 < tf < 2600
    assert bool(torch.isfinite(sink).all())
