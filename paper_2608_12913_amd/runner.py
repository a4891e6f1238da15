"""Device buffers for one verification problem and calls through the C ABI.

PyTorch only allocates device memory and provides the stream; every step of the
verification runs in libdcd's kernels (through :mod:`paper_2608_12913_amd.dcd`).
"""
from __future__ import annotations

import numpy as np
import torch

from . import dcd


def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:  # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


class DeviceProblem:
    """Inputs, outputs and workspace of one problem, resident on `device`."""

    def __init__(self, *, hp, hq, wp, wq, bias_p, bias_q, parents, tokens, B, N, V, dtype,
                 theta, s, T=1.0, draft_probs=None, u_acc=None, u_res=None, device="cuda:0",
                 row_outputs=True, norm_p=None, norm_q=None, norm_eps=0.0):
        self.device = torch.device(device)
        dv = lambda a: None if a is None else _dev(a, self.device)  # noqa: E731
        self.B, self.N, self.V = B, N, V
        self.hp, self.hq, self.wp, self.wq = dv(hp), dv(hq), dv(wp), dv(wq)
        self.bias_p = dv(None if bias_p is None else np.asarray(bias_p, np.float32))
        self.bias_q = (self.bias_p if bias_q is bias_p
                       else dv(None if bias_q is None else np.asarray(bias_q, np.float32)))
        self.parents = dv(np.asarray(parents, np.int32).reshape(B, N))
        self.tokens = dv(np.asarray(tokens, np.int32).reshape(B, N))
        self.draft_probs = dv(None if draft_probs is None else np.asarray(draft_probs, np.float32))
        self.u_acc = dv(None if u_acc is None else np.asarray(u_acc, np.float32))
        self.u_res = dv(None if u_res is None else np.asarray(u_res, np.float32))
        # norm_p / norm_q: scales of the models' final RMS normalisation; hp / hq are
        # then the rows before it
        self.norm_p, self.norm_q = dv(norm_p), dv(norm_q)
        final_norm = norm_p is not None
        self.problem = dcd.make_problem(B, N, V, hp.shape[1], hq.shape[1], dtype, theta, s, T,
                                        final_norm, norm_eps)
        R = B * N
        i32 = dict(dtype=torch.int32, device=self.device)
        f32 = dict(dtype=torch.float32, device=self.device)
        self.accept_len = torch.empty(B, **i32)
        self.accept_path = torch.empty(B, N, **i32)
        self.next_token = torch.empty(B, **i32)
        self.status = torch.empty(B, **i32)
        self.row_argmax = torch.empty(R, **i32) if row_outputs else None
        self.row_stats = torch.empty(R, 8, **f32) if row_outputs else None
        self.node_stats = torch.empty(R, 6, **f32) if row_outputs else None
        self.row_argmax_expert = torch.empty(R, **i32) if row_outputs else None
        self.row_kl = torch.empty(R, 2, **f32) if row_outputs else None
        self.ws_bytes = dcd.workspace_bytes(self.problem)
        if self.ws_bytes == 0:
            raise dcd.DcdError(dcd.DCD_ERR_SHAPE)
        # zero-filled once: its first words are the call count the library keeps
        self.workspace = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=self.device)
        self.inputs = dcd.make_inputs(self.hp, self.hq, self.wp, self.wq, self.bias_p, self.bias_q,
                                      self.parents, self.tokens, self.norm_p, self.norm_q)
        self.outputs = dcd.make_outputs(self.accept_len, self.accept_path, self.next_token,
                                        self.status, self.row_argmax, self.row_stats,
                                        self.node_stats, self.row_argmax_expert, self.row_kl)

    @classmethod
    def from_case(cls, case, tokens, draft_probs=None, device="cuda:0", row_outputs=True,
                  **overrides):
        kw = dict(hp=case.hp, hq=case.hq, wp=case.wp, wq=case.wq, bias_p=case.bias,
                  bias_q=case.bias, parents=case.parents, tokens=tokens, B=case.B, N=case.N,
                  V=case.V, dtype=case.dtype, theta=case.theta, s=case.s, T=case.T,
                  draft_probs=draft_probs, u_acc=case.u_acc, u_res=case.u_res, device=device,
                  row_outputs=row_outputs)
        kw.update(overrides)
        return cls(**kw)

    def set_tokens(self, tokens):
        self.tokens.copy_(torch.from_numpy(np.asarray(tokens, np.int32).reshape(self.B, self.N)))

    def launch(self, mode: str, stream=None) -> None:
        """Enqueue one verification on `stream` (default: torch's current stream)."""
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        if mode == "greedy":
            dcd.verify_greedy(self.problem, self.inputs, self.outputs, self.workspace,
                              self.ws_bytes, stream)
        else:
            dcd.verify_sample(self.problem, self.inputs, self.draft_probs, self.u_acc, self.u_res,
                              self.outputs, self.workspace, self.ws_bytes, stream)

    def propose(self, u, want_probs=True) -> dict:
        """dcd_propose on this problem's heads (the expert slots hold one drafter head,
        the amateur slots the other); synchronous, host copies of the outputs."""
        R, V = self.B * self.N, self.V
        i32 = dict(dtype=torch.int32, device=self.device)
        u = torch.from_numpy(np.asarray(u, np.float32)).to(self.device)
        tokens, argmax = torch.empty(R, **i32), torch.empty(R, **i32)
        probs = torch.empty(R, V, dtype=torch.float32, device=self.device) if want_probs else None
        dcd.propose(self.problem, self.inputs, u, tokens, probs, argmax, self.workspace,
                    self.ws_bytes, torch.cuda.current_stream(self.device))
        torch.cuda.synchronize(self.device)
        out = dict(tokens=tokens.cpu().numpy(), argmax=argmax.cpu().numpy())
        if probs is not None:
            out["probs"] = probs.cpu().numpy()
        return out

    def launch_lmhead(self, mode: str, stream=None) -> None:
        """Enqueue only the LM-head projection stage (the dominant kernel)."""
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        dcd.lmhead_partials(self.problem, self.inputs, mode == "sample", self.workspace,
                            self.ws_bytes, stream)

    def run(self, mode: str) -> dict:
        """One synchronous verification; returns host copies of every output."""
        self.launch(mode)
        torch.cuda.synchronize(self.device)
        out = dict(accept_len=self.accept_len.cpu().numpy(),
                   accept_path=self.accept_path.cpu().numpy(),
                   next_token=self.next_token.cpu().numpy(), status=self.status.cpu().numpy())
        if self.row_argmax is not None:
            out.update(row_argmax=self.row_argmax.cpu().numpy(),
                       row_stats=self.row_stats.cpu().numpy(),
                       node_stats=self.node_stats.cpu().numpy(),
                       row_argmax_expert=self.row_argmax_expert.cpu().numpy(),
                       row_kl=self.row_kl.cpu().numpy())
        return out
