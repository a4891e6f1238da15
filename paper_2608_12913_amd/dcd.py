"""ctypes binding of libdcd (include/dcd.h): argument marshalling only.

Every step of the verification runs in the library's HIP kernels.  Buffers are
passed as device pointers: anything with ``data_ptr()`` (a torch tensor on the
GPU) or a plain integer address.  A missing or unloadable library raises; there
is no fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdcd.so")
PROBE_LIB_PATH = os.path.join(PKG, "libdcd_probe.so")  # the benchmark's measurement probes

DCD_OK, DCD_ERR_NULL, DCD_ERR_SHAPE, DCD_ERR_PARAM = 0, -1, -2, -3
DCD_ERR_ALIGN, DCD_ERR_WORKSPACE, DCD_ERR_UNSUPPORTED, DCD_ERR_HIP = -4, -5, -6, -7
DCD_ERR_TOO_LARGE = -8
SEQ_OK, SEQ_BAD_TREE, SEQ_BAD_TOKEN, SEQ_NONFINITE, SEQ_NOT_CHAIN, SEQ_WALK_TIMEOUT = range(6)
DCD_F32, DCD_BF16 = 0, 1
ROW_MAX_P, ROW_LSE_P, ROW_LSE_Q, ROW_LOGZ, ROW_TOP1, ROW_MARGIN, ROW_COUNT, ROW_SIGNAL = range(8)
NODE_LOGP_P, NODE_LOGP_Q, NODE_CD, NODE_LOGP_CD, NODE_IN_MASK, NODE_RATIO = range(6)

EXPORTS = ("dcd_workspace_bytes", "dcd_verify_greedy", "dcd_verify_sample",
           "dcd_lmhead_partials", "dcd_propose", "dcd_error_string", "dcd_abi_version",
           "dcd_verify_greedy_noalloc", "dcd_noalloc_max_bytes")
PROBE_EXPORTS = ("dcd_probe_stream_read", "dcd_probe_mfma_bf16")  # include/dcd_probe.h


class DcdError(RuntimeError):
    def __init__(self, code: int):
        self.code = code
        super().__init__(f"libdcd error {code}: {error_string(code)}")


class Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("nodes", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("d_expert", ctypes.c_int32), ("d_amateur", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("plaus_thresh", ctypes.c_float),
                ("cd_strength", ctypes.c_float), ("temperature", ctypes.c_float),
                ("final_norm", ctypes.c_int32), ("norm_eps", ctypes.c_float)]


class Inputs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("h_expert", "h_amateur", "w_expert", "w_amateur",
                                                "bias_expert", "bias_amateur", "parents", "tokens",
                                                "norm_expert", "norm_amateur")]


class Outputs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("accept_len", "accept_path", "next_token", "status",
                                                "row_argmax", "row_stats", "node_stats",
                                                "row_argmax_expert", "row_kl")]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                               "(or python -m paper_2608_12913_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.dcd_workspace_bytes.argtypes = [ctypes.POINTER(Problem)]
        L.dcd_workspace_bytes.restype = ctypes.c_size_t
        L.dcd_verify_greedy.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs),
                                        ctypes.POINTER(Outputs), P, ctypes.c_size_t, P]
        L.dcd_verify_greedy.restype = ctypes.c_int
        L.dcd_verify_sample.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs), P, P, P,
                                        ctypes.POINTER(Outputs), P, ctypes.c_size_t, P]
        L.dcd_verify_sample.restype = ctypes.c_int
        L.dcd_propose.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs), P, P, P, P, P,
                                  ctypes.c_size_t, P]
        L.dcd_propose.restype = ctypes.c_int
        L.dcd_lmhead_partials.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs),
                                          ctypes.c_int, P, ctypes.c_size_t, P]
        L.dcd_lmhead_partials.restype = ctypes.c_int
        L.dcd_verify_greedy_noalloc.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Inputs),
                                                ctypes.POINTER(Outputs), P]
        L.dcd_verify_greedy_noalloc.restype = ctypes.c_int
        L.dcd_noalloc_max_bytes.argtypes = []
        L.dcd_noalloc_max_bytes.restype = ctypes.c_size_t
        L.dcd_error_string.argtypes = [ctypes.c_int]
        L.dcd_error_string.restype = ctypes.c_char_p
        L.dcd_abi_version.argtypes = []
        L.dcd_abi_version.restype = ctypes.c_int
        _lib = L
    return _lib


_probe_lib = None


def probe_lib() -> ctypes.CDLL:
    """The measurement probes (include/dcd_probe.h), a library of their own."""
    global _probe_lib
    if _probe_lib is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise RuntimeError(f"{PROBE_LIB_PATH} is not built: run __graft_entry__.build()")
        L = ctypes.CDLL(PROBE_LIB_PATH)
        P = ctypes.c_void_p
        L.dcd_probe_stream_read.argtypes = [P, ctypes.c_size_t, P, P]
        L.dcd_probe_stream_read.restype = ctypes.c_int
        L.dcd_probe_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, P,
                                          ctypes.POINTER(ctypes.c_double), P]
        L.dcd_probe_mfma_bf16.restype = ctypes.c_int
        _probe_lib = L
    return _probe_lib


def error_string(code: int) -> str:
    return lib().dcd_error_string(int(code)).decode()


def ptr(x) -> int | None:
    """Device address of a buffer (None stays NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(stream) -> int | None:
    if stream is None:
        return None
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def make_problem(batch, nodes, vocab, d_expert, d_amateur, dtype="bf16", plaus_thresh=0.1,
                 cd_strength=0.5, temperature=1.0, final_norm=False, norm_eps=0.0) -> Problem:
    dt = {"bf16": DCD_BF16, "f32": DCD_F32}.get(dtype, dtype)
    return Problem(batch, nodes, vocab, d_expert, d_amateur, dt, plaus_thresh, cd_strength,
                   temperature, int(bool(final_norm)), norm_eps)


def make_inputs(h_expert, h_amateur, w_expert, w_amateur, bias_expert, bias_amateur, parents,
                tokens, norm_expert=None, norm_amateur=None) -> Inputs:
    return Inputs(*(ptr(a) for a in (h_expert, h_amateur, w_expert, w_amateur, bias_expert,
                                     bias_amateur, parents, tokens, norm_expert, norm_amateur)))


def make_outputs(accept_len, accept_path, next_token, status, row_argmax=None, row_stats=None,
                 node_stats=None, row_argmax_expert=None, row_kl=None) -> Outputs:
    return Outputs(*(ptr(a) for a in (accept_len, accept_path, next_token, status, row_argmax,
                                      row_stats, node_stats, row_argmax_expert, row_kl)))


def workspace_bytes(problem: Problem) -> int:
    return int(lib().dcd_workspace_bytes(ctypes.byref(problem)))


def verify_greedy(problem: Problem, inputs: Inputs, outputs: Outputs, workspace,
                  workspace_bytes: int, stream=None) -> None:
    rc = lib().dcd_verify_greedy(ctypes.byref(problem), ctypes.byref(inputs),
                                 ctypes.byref(outputs), ptr(workspace), int(workspace_bytes),
                                 _stream(stream))
    if rc != DCD_OK:
        raise DcdError(rc)


def verify_greedy_noalloc(problem: Problem, inputs: Inputs, outputs: Outputs, stream=None) -> None:
    """dcd_verify_greedy on the library's static per-GPU workspace (no allocation)."""
    _check(lib().dcd_verify_greedy_noalloc(ctypes.byref(problem), ctypes.byref(inputs),
                                           ctypes.byref(outputs), _stream(stream)))


def noalloc_max_bytes() -> int:
    return int(lib().dcd_noalloc_max_bytes())


def verify_sample(problem: Problem, inputs: Inputs, draft_probs, u_accept, u_resample,
                  outputs: Outputs, workspace, workspace_bytes: int, stream=None) -> None:
    rc = lib().dcd_verify_sample(ctypes.byref(problem), ctypes.byref(inputs), ptr(draft_probs),
                                 ptr(u_accept), ptr(u_resample), ctypes.byref(outputs),
                                 ptr(workspace), int(workspace_bytes), _stream(stream))
    if rc != DCD_OK:
        raise DcdError(rc)


def lmhead_partials(problem: Problem, inputs: Inputs, sampled: bool, workspace,
                    workspace_bytes: int, stream=None) -> None:
    rc = lib().dcd_lmhead_partials(ctypes.byref(problem), ctypes.byref(inputs), int(sampled),
                                   ptr(workspace), int(workspace_bytes), _stream(stream))
    if rc != DCD_OK:
        raise DcdError(rc)


def probe_stream_read(buf, nbytes: int, sink, stream=None) -> None:
    """Enqueue one streaming read of `nbytes` at `buf` (include/dcd_probe.h)."""
    _check(probe_lib().dcd_probe_stream_read(ptr(buf), int(nbytes), ptr(sink), _stream(stream)))


def probe_mfma_bf16(workgroups: int, iters: int, sink, stream=None) -> float:
    """Enqueue the bf16 MFMA loop; returns the flops one launch performs."""
    flops = ctypes.c_double(0.0)
    _check(probe_lib().dcd_probe_mfma_bf16(int(workgroups), int(iters), ptr(sink),
                                            ctypes.byref(flops), _stream(stream)))
    return flops.value


def _check(rc: int) -> None:
    if rc != DCD_OK:
        raise DcdError(rc)


def propose(problem: Problem, inputs: Inputs, u, tokens, probs, argmax, workspace,
            workspace_bytes: int, stream=None) -> None:
    """Enqueue dcd_propose (outputs may be None, but not all three)."""
    _check(lib().dcd_propose(ctypes.byref(problem), ctypes.byref(inputs), ptr(u), ptr(tokens),
                             ptr(probs), ptr(argmax), ptr(workspace), int(workspace_bytes),
                             _stream(stream)))
