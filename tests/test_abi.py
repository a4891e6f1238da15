"""C-ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects invalid requests on the host before any launch."""
import ctypes
import glob
import os
import re

import pytest

from paper_2608_12913_amd import dcd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def _declared_functions(header=None):
    names = set()
    for h in HEADERS:
        if header and os.path.basename(h) != header:
            continue
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(dcd_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function():
    """libdcd.so exports dcd.h; the benchmark's probes (dcd_probe.h) live in
    libdcd_probe.so and nowhere in the product library."""
    assert [os.path.basename(h) for h in HEADERS] == ["dcd.h", "dcd_probe.h"]
    names = _declared_functions("dcd.h")
    assert set(names) == set(dcd.EXPORTS)
    L = dcd.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.dcd_abi_version() == 7
    probes = _declared_functions("dcd_probe.h")
    assert set(probes) == set(dcd.PROBE_EXPORTS)
    PL = dcd.probe_lib()
    for n in probes:
        assert hasattr(PL, n), n
        assert not hasattr(L, n), n


def test_struct_layouts_match_the_header(tmp_path):
    """The ctypes structs of the binding have the header's sizes and field offsets
    (a C program built with the header against the same names)."""
    import subprocess
    structs = {"dcd_problem": dcd.Problem, "dcd_inputs": dcd.Inputs, "dcd_outputs": dcd.Outputs}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "dcd.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)])
    got = {}
    for line in subprocess.check_output([str(exe)], text=True).splitlines():
        cname, field, val = line.split()
        got[(cname, field)] = int(val)
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def test_error_strings():
    for code in range(0, -9, -1):
        assert dcd.error_string(code) and dcd.error_string(code) != "unknown error code"
    assert dcd.error_string(-99) == "unknown error code"


def _problem(**kw):
    base = dict(batch=1, nodes=64, vocab=128256, d_expert=4096, d_amateur=2048, dtype="bf16",
                plaus_thresh=0.1, cd_strength=0.5, temperature=1.0)
    base.update(kw)
    return dcd.make_problem(**base)


def test_workspace_bytes():
    ws = dcd.workspace_bytes(_problem())
    R, V = 64, 128256
    # candidate logits (8 B per row and token) dominate; partials, bitmap, row results on top
    assert R * V * 8 < ws < R * V * 8 * 1.1
    assert dcd.workspace_bytes(_problem(batch=32)) > 31 * ws
    for bad in (dict(batch=0), dict(vocab=0), dict(d_expert=4100), dict(dtype=7),
                dict(plaus_thresh=1.5), dict(plaus_thresh=-0.1), dict(cd_strength=-1.0),
                dict(plaus_thresh=float("nan")), dict(cd_strength=float("inf"))):
        assert dcd.workspace_bytes(_problem(**bad)) == 0, bad
    # fp32 rows need a multiple of 4 elements, bf16 a multiple of 8
    assert dcd.workspace_bytes(_problem(dtype="f32", d_expert=4100)) > 0


def _fake_ptrs():
    # host addresses suitably aligned; never dereferenced because validation fails first
    buf = (ctypes.c_char * 4096)()
    a = (ctypes.addressof(buf) + 255) // 256 * 256
    return buf, a


def _call_greedy(problem, inputs, outputs, ws, ws_bytes):
    return dcd.lib().dcd_verify_greedy(ctypes.byref(problem), ctypes.byref(inputs),
                                       ctypes.byref(outputs), ws, ws_bytes, None)


def test_host_validation_errors():
    buf, a = _fake_ptrs()
    p = _problem(nodes=8, vocab=1024, d_expert=256, d_amateur=128)
    good_in = dcd.Inputs(a, a, a, a, a, a, a, a)
    good_out = dcd.Outputs(a, a, a, a, None, None, None)
    need = dcd.workspace_bytes(p)
    # missing required pointers
    for i in range(8):
        if i in (4, 5):  # biases are optional
            continue
        vals = [a] * 8
        vals[i] = None
        assert _call_greedy(p, dcd.Inputs(*vals), good_out, a, need) == dcd.DCD_ERR_NULL
    for i in range(4):
        vals = [a] * 4 + [None] * 3
        vals[i] = None
        assert _call_greedy(p, good_in, dcd.Outputs(*vals), a, need) == dcd.DCD_ERR_NULL
    # misaligned matrices (16 bytes) and small buffers (4 bytes)
    assert _call_greedy(p, dcd.Inputs(a + 8, a, a, a, a, a, a, a), good_out, a, need) == dcd.DCD_ERR_ALIGN
    assert _call_greedy(p, dcd.Inputs(a, a, a, a, a + 2, a, a, a), good_out, a, need) == dcd.DCD_ERR_ALIGN
    # workspace too small / missing / misaligned
    assert _call_greedy(p, good_in, good_out, a, need - 1) == dcd.DCD_ERR_WORKSPACE
    assert _call_greedy(p, good_in, good_out, None, need) == dcd.DCD_ERR_WORKSPACE
    assert _call_greedy(p, good_in, good_out, a + 16, need) == dcd.DCD_ERR_WORKSPACE
    # parameters and shapes
    assert _call_greedy(_problem(nodes=8, vocab=1024, d_expert=256, d_amateur=128, plaus_thresh=2.0),
                        good_in, good_out, a, need) == dcd.DCD_ERR_PARAM
    assert _call_greedy(_problem(nodes=0), good_in, good_out, a, need) == dcd.DCD_ERR_SHAPE
    assert _call_greedy(_problem(nodes=4097), good_in, good_out, a, need) == dcd.DCD_ERR_SHAPE
    assert _call_greedy(_problem(d_amateur=2044), good_in, good_out, a, need) == dcd.DCD_ERR_ALIGN
    # sampled mode validates temperature and its extra inputs
    L = dcd.lib()
    ps = _problem(nodes=8, vocab=1024, d_expert=256, d_amateur=128, temperature=0.0)
    rc = L.dcd_verify_sample(ctypes.byref(ps), ctypes.byref(good_in), a, a, a,
                             ctypes.byref(good_out), a, need, None)
    assert rc == dcd.DCD_ERR_PARAM
    ps = _problem(nodes=8, vocab=1024, d_expert=256, d_amateur=128)
    rc = L.dcd_verify_sample(ctypes.byref(ps), ctypes.byref(good_in), None, a, a,
                             ctypes.byref(good_out), a, need, None)
    assert rc == dcd.DCD_ERR_NULL
    del buf


def test_binding_raises():
    p = _problem(batch=0)
    with pytest.raises(dcd.DcdError) as e:
        dcd.verify_greedy(p, dcd.Inputs(), dcd.Outputs(), None, 0)
    assert e.value.code == dcd.DCD_ERR_SHAPE


def test_probe_host_validation():
    """The measurement probes reject invalid requests before any launch."""
    L = dcd.probe_lib()
    buf = (ctypes.c_char * 64)()
    a = (ctypes.addressof(buf) + 15) // 16 * 16
    flops = ctypes.c_double(0.0)
    assert L.dcd_probe_stream_read(None, 16, a, None) == dcd.DCD_ERR_NULL
    assert L.dcd_probe_stream_read(a, 0, a, None) == dcd.DCD_ERR_SHAPE
    assert L.dcd_probe_stream_read(a, 24, a, None) == dcd.DCD_ERR_SHAPE
    assert L.dcd_probe_stream_read(a + 4, 16, a, None) == dcd.DCD_ERR_ALIGN
    assert L.dcd_probe_mfma_bf16(0, 10, a, ctypes.byref(flops), None) == dcd.DCD_ERR_SHAPE
    assert L.dcd_probe_mfma_bf16(4, 0, a, ctypes.byref(flops), None) == dcd.DCD_ERR_SHAPE
    assert L.dcd_probe_mfma_bf16(4, 10, None, ctypes.byref(flops), None) == dcd.DCD_ERR_NULL


def test_propose_host_validation():
    """dcd_propose rejects a call without outputs, a draw without uniforms, misaligned
    buffers and a short workspace before any launch."""
    buf, a = _fake_ptrs()
    p = _problem(nodes=8, vocab=1024, d_expert=256, d_amateur=128)
    need = dcd.workspace_bytes(p)
    ins = dcd.Inputs(a, a, a, a, None, None, None, None)  # no tree needed

    def call(u, tokens, probs, argmax, ws=a, n=need, i=ins):
        return dcd.lib().dcd_propose(ctypes.byref(p), ctypes.byref(i), u, tokens, probs, argmax,
                                     ws, n, None)

    assert call(None, None, None, None) == dcd.DCD_ERR_NULL
    assert call(None, a, None, None) == dcd.DCD_ERR_NULL        # tokens need u
    assert call(a, a + 2, None, None) == dcd.DCD_ERR_ALIGN
    assert call(None, None, a + 1, None) == dcd.DCD_ERR_ALIGN
    assert call(None, None, None, a, n=need - 1) == dcd.DCD_ERR_WORKSPACE
    assert call(None, None, None, a, i=dcd.Inputs(a, None, a, a, None, None, None, None)) == dcd.DCD_ERR_NULL


def test_final_norm_host_validation():
    """The final RMS normalisation needs both scale vectors (16-byte aligned), a flag
    of 0 or 1 and a finite eps >= 0; its workspace holds the normalised rows."""
    buf, a = _fake_ptrs()
    kw = dict(nodes=8, vocab=1024, d_expert=256, d_amateur=128)
    p0 = _problem(**kw)
    p1 = _problem(final_norm=True, norm_eps=1e-5, **kw)
    assert dcd.workspace_bytes(p1) >= dcd.workspace_bytes(p0) + 8 * (256 + 128) * 2
    p2 = _problem(**kw)
    p2.final_norm = 2
    assert dcd.workspace_bytes(p2) == 0
    assert dcd.workspace_bytes(_problem(final_norm=True, norm_eps=-1.0, **kw)) == 0
    assert dcd.workspace_bytes(_problem(final_norm=True, norm_eps=float("nan"), **kw)) == 0
    need = dcd.workspace_bytes(p1)
    out = dcd.Outputs(a, a, a, a, None, None, None)
    assert _call_greedy(p1, dcd.Inputs(a, a, a, a, a, a, a, a), out, a, need) == dcd.DCD_ERR_NULL
    assert _call_greedy(p1, dcd.Inputs(a, a, a, a, a, a, a, a, a, None), out, a, need) == dcd.DCD_ERR_NULL
    assert _call_greedy(p1, dcd.Inputs(a, a, a, a, a, a, a, a, a + 4, a), out, a, need) == dcd.DCD_ERR_ALIGN
    assert _call_greedy(p1, dcd.Inputs(a, a, a, a, a, a, a, a, a, a), out, a, need - 1) == dcd.DCD_ERR_WORKSPACE


def test_noalloc_refuses_problems_beyond_its_array():
    """dcd_verify_greedy_noalloc checks the problem's workspace size against its static
    array before it touches a device (so this runs without a GPU)."""
    cap = dcd.noalloc_max_bytes()
    assert cap == 80 << 20
    assert dcd.workspace_bytes(_problem()) <= cap  # the 64-row 8B/1B tree fits
    assert dcd.workspace_bytes(_problem(plaus_thresh=0.0)) <= cap
    big = _problem(batch=2)
    assert dcd.workspace_bytes(big) > cap
    ins, outs = dcd.Inputs(), dcd.Outputs()
    with pytest.raises(dcd.DcdError) as e:
        dcd.verify_greedy_noalloc(big, ins, outs)
    assert e.value.code == dcd.DCD_ERR_TOO_LARGE
    with pytest.raises(dcd.DcdError) as e:  # invalid problems first
        dcd.verify_greedy_noalloc(_problem(vocab=0), ins, outs)
    assert e.value.code == dcd.DCD_ERR_SHAPE
