"""Plain fp64 CPU oracle for contrastive-decoding tree verification.

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg are the only callers.  It shares no code with the
GPU library and never imports it.

The arithmetic lives in ``dcd_oracle.c`` (built into ``liboracle.so`` next to
this file by :func:`build`); this module only marshals numpy arrays.  Inputs are
float32 arrays holding the exact bf16 or fp32 input values; bf16 data arrives as
uint16 bit patterns and is widened exactly (bf16 is the top half of fp32).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dcd_oracle.c")
# the library the loader uses; DCD_ORACLE_LIB names another build of the same source
# (the sanitised one, see build)
_LIB = os.environ.get("DCD_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_SAN_LIB = os.path.join(_HERE, "liboracle_san.so")

# row_stats slots
RS_MAXP, RS_LSEP, RS_LSEQ, RS_LOGZ, RS_TOP1, RS_MARGIN, RS_COUNT, RS_SIGNAL = range(8)
# row diagnostics slots: argmax pi_p, D_KL(pi_p||pi_q), D_KL(pi_p||pi_CD), expert top-2 logit gap
RD_ARGMAX_P, RD_KL_PQ, RD_KL_PCD, RD_MARGIN_P = range(4)
# node_stats slots
NS_LPP, NS_LPQ, NS_CD, NS_LPCD, NS_INMASK, NS_RATIO = range(6)
SEQ_OK, SEQ_BAD_TREE, SEQ_BAD_TOKEN, SEQ_NONFINITE, SEQ_NOT_CHAIN = range(5)


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math).  sanitize: a separate
    build with AddressSanitizer and UndefinedBehaviorSanitizer (any report aborts), for
    running the pins under them; loading it needs libasan preloaded."""
    lib = _SAN_LIB if sanitize else _LIB
    if force or not os.path.exists(lib):
        tmp = lib + ".tmp"
        opt = (["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                "-fno-sanitize-recover=all"] if sanitize else ["-O2"])
        subprocess.check_call(
            ["gcc", *opt, "-std=c11", "-fPIC", "-shared", "-fopenmp", "-Wall", _SRC, "-o", tmp, "-lm"]
        )
        os.replace(tmp, lib)
    return lib


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, f64 = ctypes.c_int, ctypes.c_double
        lib.dco_eval_rows.argtypes = [i32, i32, i32, P, P, P, P, P, P, f64, f64, f64, P, i32,
                                      P, P, P, P, P, P, P, i32]
        lib.dco_eval_rows.restype = i32
        lib.dco_propose.argtypes = [i32, i32, i32, i32, P, P, P, P, P, P, f64, f64, f64, P, P, P, P,
                                    P, i32]
        lib.dco_propose.restype = i32
        lib.dco_rmsnorm.argtypes = [i32, i32, P, P, f64, i32, P]
        lib.dco_rmsnorm.restype = None
        lib.dco_greedy_walk.argtypes = [i32, P, P, P, P, P, P]
        lib.dco_greedy_walk.restype = None
        lib.dco_sample_tree.argtypes = [i32, i32, P, P, P, P, P, P, P, P, P, P, P, P]
        lib.dco_sample_tree.restype = None
        lib.dco_verify.argtypes = [i32, i32, i32, i32, i32, i32, P, P, P, P, P, P, P, P,
                                   f64, f64, f64, P, P, P, P, P, P, P, P, P, P, P, P, P, P, i32]
        lib.dco_verify.restype = i32
        _lib = lib
    return _lib


def as_f32(a) -> np.ndarray:
    """float32 view of bf16 (uint16 bits) or fp32 data, exactly."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32)
    return np.ascontiguousarray(a, dtype=np.float32)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def eval_rows(hp, hq, wp, wq, bp, bq, *, theta, s, temperature=1.0, rows=None,
              want_logits=False, want_lpcd=False, nthreads=0):
    """Per-row oracle evaluation.

    Returns dict(argmax [n], stats [n, 8], gap [n], diag [n, 4] (RD_* slots), and
    optionally zp, zq, lpcd [n, V]).
    """
    hp, hq, wp, wq = as_f32(hp), as_f32(hq), as_f32(wp), as_f32(wq)
    bp = None if bp is None else _c(bp, np.float32)
    bq = None if bq is None else _c(bq, np.float32)
    V, dp = wp.shape
    dq = wq.shape[1]
    ids = None if rows is None else _c(rows, np.int32)
    n = hp.shape[0] if ids is None else len(ids)
    out = dict(argmax=np.empty(n, np.int32), stats=np.empty((n, 8)), gap=np.empty(n),
               diag=np.empty((n, 4)))
    if want_logits:
        out["zp"] = np.empty((n, V))
        out["zq"] = np.empty((n, V))
    if want_lpcd:
        out["lpcd"] = np.empty((n, V))
    rc = _load().dco_eval_rows(V, dp, dq, _p(hp), _p(hq), _p(wp), _p(wq), _p(bp), _p(bq),
                               float(temperature), float(theta), float(s), _p(ids), n,
                               _p(out["argmax"]), _p(out["stats"]), _p(out["gap"]),
                               _p(out["diag"]), _p(out.get("zp")), _p(out.get("zq")), _p(out.get("lpcd")),
                               int(nthreads))
    if rc:
        raise RuntimeError(f"dco_eval_rows failed ({rc})")
    return out


def propose(he, hf, we, wf, be, bf, u, *, theta, s, temperature=1.0, nthreads=0):
    """Proposals from the recombined heads: dict(probs [R, V], tokens [R], gap [R],
    argmax [R])."""
    he, hf, we, wf = as_f32(he), as_f32(hf), as_f32(we), as_f32(wf)
    be = None if be is None else _c(be, np.float32)
    bf = None if bf is None else _c(bf, np.float32)
    u = _c(u, np.float32)
    V, de = we.shape
    df = wf.shape[1]
    R = he.shape[0]
    o = dict(probs=np.zeros((R, V)), tokens=np.zeros(R, np.int32), gap=np.zeros(R),
             argmax=np.zeros(R, np.int32))
    rc = _load().dco_propose(R, V, de, df, _p(he), _p(hf), _p(we), _p(wf), _p(be), _p(bf),
                             float(temperature), float(theta), float(s), _p(u), _p(o["tokens"]),
                             _p(o["probs"]), _p(o["gap"]), _p(o["argmax"]), int(nthreads))
    if rc:
        raise RuntimeError(f"dco_propose failed ({rc})")
    return o


def rmsnorm(x, g, eps):
    """Final RMS normalisation of the rows of x with scale g; bf16 data (uint16 bit
    patterns) stays bf16 (returned as uint16 bits), fp32 stays fp32."""
    bf16 = np.asarray(x).dtype == np.uint16
    xf, gf = as_f32(x), as_f32(g)
    R, d = xf.shape
    y = np.empty((R, d), np.float32)
    _load().dco_rmsnorm(R, d, _p(xf), _p(gf), float(eps), int(bf16), _p(y))
    if bf16:
        return (y.view(np.uint32) >> 16).astype(np.uint16)
    return y


def greedy_walk(parents, tokens, row_argmax):
    parents, tokens, row_argmax = (_c(parents, np.int32), _c(tokens, np.int32),
                                   _c(row_argmax, np.int32))
    N = len(parents)
    L = np.zeros(1, np.int32)
    path = np.empty(N, np.int32)
    nxt = np.zeros(1, np.int32)
    _load().dco_greedy_walk(N, _p(parents), _p(tokens), _p(row_argmax), _p(L), _p(path), _p(nxt))
    return int(L[0]), path, int(nxt[0])


def sample_tree(parents, tokens, lp_cd, draft_probs, u_acc, u_res):
    """Alg. 1 accept/residual/bonus over one draft tree, given log pi_CD rows [N, V]."""
    parents, tokens = _c(parents, np.int32), _c(tokens, np.int32)
    lp_cd = _c(lp_cd, np.float64)
    q = _c(draft_probs, np.float32)
    u_acc, u_res = _c(u_acc, np.float32), _c(u_res, np.float32)
    N, V = lp_cd.shape
    L = np.zeros(1, np.int32)
    path = np.empty(N, np.int32)
    nxt = np.zeros(1, np.int32)
    ratio = np.full(N, np.nan)
    walk = np.full(N, np.nan)
    gap = np.zeros(1)
    _load().dco_sample_tree(N, V, _p(parents), _p(tokens), _p(lp_cd), _p(q), _p(u_acc), _p(u_res),
                            _p(L), _p(path), _p(nxt), _p(ratio), _p(walk), _p(gap))
    return dict(accept_len=int(L[0]), path=path, next_token=int(nxt[0]), ratio=ratio,
                walk_ratio=walk, res_gap=float(gap[0]))


def sample_chain(tokens, lp_cd, draft_probs, u_acc, u_res):
    """sample_tree on a chain (parents[i] = i - 1)."""
    N = len(tokens)
    return sample_tree(np.arange(-1, N - 1), tokens, lp_cd, draft_probs, u_acc, u_res)


def verify(mode, B, N, hp, hq, wp, wq, bp, bq, parents, tokens, *, theta, s,
           temperature=1.0, draft_probs=None, u_acc=None, u_res=None, nthreads=0):
    """Full verification (mode "greedy" or "sample"); returns a dict of numpy outputs."""
    m = {"greedy": 0, "sample": 1}[mode]
    hp, hq, wp, wq = as_f32(hp), as_f32(hq), as_f32(wp), as_f32(wq)
    bp = None if bp is None else _c(bp, np.float32)
    bq = None if bq is None else _c(bq, np.float32)
    parents, tokens = _c(parents, np.int32).reshape(-1), _c(tokens, np.int32).reshape(-1)
    V, dp = wp.shape
    dq = wq.shape[1]
    R = B * N
    if m == 1:
        draft_probs = _c(draft_probs, np.float32)
        u_acc, u_res = _c(u_acc, np.float32), _c(u_res, np.float32)
    o = dict(accept_len=np.zeros(B, np.int32), accept_path=np.zeros((B, N), np.int32),
             next_token=np.zeros(B, np.int32), status=np.zeros(B, np.int32),
             row_argmax=np.zeros(R, np.int32), row_stats=np.zeros((R, 8)),
             node_stats=np.zeros((R, 6)), row_diag=np.zeros((R, 4)), row_gap=np.zeros(R),
             res_gap=np.zeros(B), walk_ratio=np.zeros(R))
    rc = _load().dco_verify(m, B, N, V, dp, dq, _p(hp), _p(hq), _p(wp), _p(wq), _p(bp), _p(bq),
                            _p(parents), _p(tokens), float(theta), float(s), float(temperature),
                            _p(draft_probs), _p(u_acc), _p(u_res), _p(o["accept_len"]),
                            _p(o["accept_path"]), _p(o["next_token"]), _p(o["status"]),
                            _p(o["row_argmax"]), _p(o["row_stats"]), _p(o["node_stats"]),
                            _p(o["row_diag"]), _p(o["row_gap"]), _p(o["res_gap"]),
                            _p(o["walk_ratio"]), int(nthreads))
    if rc:
        raise RuntimeError(f"dco_verify failed ({rc})")
    return o
