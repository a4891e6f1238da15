"""Seeded synthetic inputs for contrastive-decoding tree verification.

Shared by the tests, the benchmark and the oracle's callers.  Holds none of the
verification arithmetic: it draws random numbers and lays them out.  Where an
input depends on a model output (draft tokens that copy the target argmax, the
stand-in drafter that perturbs the expert logits), the caller passes that output
in and this module only applies the seeded randomness.

Distributions (the paper prints none for logits; these are the workload's):
  * LM-head weights  W_m[v, k] ~ N(0, 1/d_m), drawn in fp32, rounded to bf16 (RNE)
    for bf16 workloads;
  * hidden states    H_m[r, k] ~ N(0, 4^2), same rounding;
  * shared bias      b_v = -ln(v + 1), computed in fp64, rounded once to fp32;
  * trees            root 0, a spine reaching the maximum depth, every other node
                     attached to a uniform eligible parent (depth < max, fewer than
                     max children), relabelled breadth-first so parent[i] < i and
                     siblings are contiguous; chains have parent[i] = i - 1;
  * uniforms         (k + 0.5) * 2^-23 with k uniform in [0, 2^23): exact in fp32 and
                     strictly inside (0, 1).
Shapes follow the paper's models (Llama-3 vocabulary 128,256; hidden sizes
4096/2048 for the 8B/1B pair, 8192/4096 for 70B/8B) and its verification sizes.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

VOCAB_LLAMA3 = 128256

# name -> workload description
CONFIGS = {
    # tiny greedy chain in fp32: the oracle finishes in milliseconds
    "tiny_chain8": dict(mode="greedy", B=1, N=8, tree="chain", V=1024, dp=256, dq=128,
                        dtype="f32", theta=0.1, s=0.5, T=1.0),
    # Llama-3-8B/1B-shaped 64-node tree (depth 8, at most 8 children per node)
    "b8_tree64": dict(mode="greedy", B=1, N=64, tree="tree", depth=8, max_children=8,
                      V=VOCAB_LLAMA3, dp=4096, dq=2048, dtype="bf16", theta=0.1, s=0.5, T=1.0),
    # sampled verification of 16 chains of 8 nodes, temperature 1
    "s8_chain16x8": dict(mode="sample", B=16, N=8, tree="chain", V=VOCAB_LLAMA3, dp=4096,
                         dq=2048, dtype="bf16", theta=0.1, s=0.5, T=1.0),
    # 32 sequences x 64-node trees = 2048 rows
    "b8_batch32x64": dict(mode="greedy", B=32, N=64, tree="tree", depth=8, max_children=8,
                          V=VOCAB_LLAMA3, dp=4096, dq=2048, dtype="bf16", theta=0.1, s=0.5,
                          T=1.0),
    # Llama-3-70B/8B-shaped 64-node tree
    "b70_tree64": dict(mode="greedy", B=1, N=64, tree="tree", depth=8, max_children=8,
                       V=VOCAB_LLAMA3, dp=8192, dq=4096, dtype="bf16", theta=0.1, s=1.0, T=1.0),
}

_STREAMS = ("w_p", "w_q", "h_p", "h_q", "tree", "tokens", "uniforms", "drafter")


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest even); returns uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    flat_in, flat_out = x.reshape(-1), out.reshape(-1)
    step = 1 << 24
    for lo in range(0, flat_in.size, step):
        u = flat_in[lo:lo + step].view(np.uint32).astype(np.uint64)
        u += 0x7FFF + ((u >> 16) & 1)
        flat_out[lo:lo + step] = (u >> 16).astype(np.uint16)
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def uniforms(rng: np.random.Generator, shape) -> np.ndarray:
    k = rng.integers(0, 1 << 23, size=shape, dtype=np.int64)
    return ((k.astype(np.float64) + 0.5) * 2.0 ** -23).astype(np.float32)


def chain_parents(N: int) -> np.ndarray:
    return np.arange(-1, N - 1, dtype=np.int32)


def tree_parents(rng: np.random.Generator, N: int, depth: int, max_children: int) -> np.ndarray:
    parent, dep, nchild = [-1], [0], [0]
    for i in range(1, min(depth, N - 1) + 1):  # spine to the maximum depth
        parent.append(i - 1)
        dep.append(i)
        nchild[i - 1] += 1
        nchild.append(0)
    while len(parent) < N:
        eligible = [n for n in range(len(parent)) if dep[n] < depth and nchild[n] < max_children]
        p = eligible[int(rng.integers(len(eligible)))]
        parent.append(p)
        dep.append(dep[p] + 1)
        nchild[p] += 1
        nchild.append(0)
    children = [[] for _ in range(N)]
    for c in range(1, N):
        children[parent[c]].append(c)  # creation order
    order, head = [0], 0
    while head < len(order):
        order.extend(children[order[head]])
        head += 1
    new_id = {old: new for new, old in enumerate(order)}
    out = np.empty(N, dtype=np.int32)
    for old, new in new_id.items():
        out[new] = -1 if parent[old] < 0 else new_id[parent[old]]
    return out


@dataclass
class Case:
    name: str
    cfg: dict
    seed: int
    B: int
    N: int
    V: int
    dp: int
    dq: int
    dtype: str  # "bf16" (uint16 bit arrays) or "f32"
    hp: np.ndarray  # [B*N, dp]
    hq: np.ndarray  # [B*N, dq]
    wp: np.ndarray  # [V, dp]
    wq: np.ndarray  # [V, dq]
    bias: np.ndarray  # [V] fp32, shared by both models
    parents: np.ndarray  # [B, N] int32
    coins: np.ndarray  # [B, N] bool: draft token copies the target argmax
    u_token: np.ndarray  # [B, N] float64 in (0,1): draws for random draft tokens
    u_acc: np.ndarray  # [B*N] fp32
    u_res: np.ndarray  # [B*N] fp32
    eps: np.ndarray | None = None  # [B*N, V] fp32 drafter noise (sampled workloads)
    u_draw: np.ndarray | None = None  # [B*N] float64: draws of sampled draft tokens
    extra: dict = field(default_factory=dict)

    @property
    def R(self) -> int:
        return self.B * self.N

    @property
    def theta(self) -> float:
        return self.cfg["theta"]

    @property
    def s(self) -> float:
        return self.cfg["s"]

    @property
    def T(self) -> float:
        return self.cfg["T"]

    @property
    def mode(self) -> str:
        return self.cfg["mode"]


def _draw_matrix(rng, shape, scale, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    x *= np.float32(scale)
    return bf16_bits(x) if dtype == "bf16" else x


def make_case(name: str, seed: int = 0, **overrides) -> Case:
    """Build the seeded inputs of a named workload (overrides patch its description)."""
    cfg = dict(CONFIGS[name]) if name in CONFIGS else {}
    cfg.update(overrides)
    B, N, V, dp, dq = cfg["B"], cfg["N"], cfg["V"], cfg["dp"], cfg["dq"]
    dtype = cfg["dtype"]
    rngs = dict(zip(_STREAMS, (np.random.default_rng(s)
                               for s in np.random.SeedSequence(seed).spawn(len(_STREAMS)))))
    wp = _draw_matrix(rngs["w_p"], (V, dp), 1.0 / np.sqrt(dp), dtype)
    wq = _draw_matrix(rngs["w_q"], (V, dq), 1.0 / np.sqrt(dq), dtype)
    hp = _draw_matrix(rngs["h_p"], (B * N, dp), cfg.get("h_scale", 4.0), dtype)
    hq = _draw_matrix(rngs["h_q"], (B * N, dq), cfg.get("h_scale", 4.0), dtype)
    bias = (-np.log(np.arange(V, dtype=np.float64) + 1.0)).astype(np.float32)
    if cfg["tree"] == "chain":
        parents = np.stack([chain_parents(N) for _ in range(B)])
    else:
        parents = np.stack([tree_parents(rngs["tree"], N, cfg["depth"], cfg["max_children"])
                            for _ in range(B)])
    coins = rngs["tokens"].random((B, N)) < 0.5
    u_token = rngs["tokens"].random((B, N))
    u_acc = uniforms(rngs["uniforms"], B * N)
    u_res = uniforms(rngs["uniforms"], B * N)
    eps = u_draw = None
    if cfg["mode"] == "sample":
        eps = rngs["drafter"].standard_normal(size=(B * N, V), dtype=np.float32)
        u_draw = rngs["drafter"].random(B * N)
    return Case(name=name, cfg=cfg, seed=seed, B=B, N=N, V=V, dp=dp, dq=dq, dtype=dtype,
                hp=hp, hq=hq, wp=wp, wq=wq, bias=bias, parents=parents.astype(np.int32),
                coins=coins, u_token=u_token, u_acc=u_acc, u_res=u_res, eps=eps, u_draw=u_draw)


def _pick_excluding(u: float, V: int, excluded: set) -> int:
    """The floor(u * (V - |excluded|))-th token of [0, V) not in `excluded`."""
    k = int(u * (V - len(excluded)))
    for e in sorted(excluded):
        if e <= k:
            k += 1
        else:
            break
    return k


def deepest_path(parents: np.ndarray) -> list:
    """Nodes of the root-to-node path that ends at the deepest node (the lowest index
    among equally deep ones), root first."""
    N = len(parents)
    depth = np.zeros(N, dtype=np.int64)
    for i in range(1, N):
        depth[i] = depth[parents[i]] + 1
    node = int(np.argmax(depth))
    path = [node]
    while node > 0:
        node = int(parents[node])
        path.append(node)
    return path[::-1]


def greedy_tokens(case: Case, row_argmax: np.ndarray, spine: bool = False) -> np.ndarray:
    """Draft tokens for greedy workloads: with probability 1/2 (the case's coin) a
    node copies the target argmax of its parent's row (given by the caller), else it
    is uniform over the vocabulary; siblings never repeat a token.  An unknown argmax
    (< 0: the caller did not compute that row) makes the node's token uniform.

    spine=True: in addition, every node of one deepest root-to-leaf path copies its
    parent row's argmax (the token is reserved before its siblings draw theirs), so
    the tree holds a full-depth path that a greedy target accepts.  A sequence whose
    path crosses a row with an unknown argmax (< 0) keeps the coin rule."""
    row_argmax = np.asarray(row_argmax).reshape(case.B, case.N)
    tokens = np.zeros((case.B, case.N), dtype=np.int32)
    for b in range(case.B):
        used = {}
        forced = {}
        if spine:
            path = deepest_path(case.parents[b])
            if all(row_argmax[b, j] >= 0 for j in path[:-1]):
                for j, c in zip(path[:-1], path[1:]):
                    forced[c] = int(row_argmax[b, j])
                    used.setdefault(j, set()).add(forced[c])
        for i in range(1, case.N):
            j = int(case.parents[b, i])
            sib = used.setdefault(j, set())
            if i in forced:
                tokens[b, i] = forced[i]
                continue
            t = int(row_argmax[b, j])
            if not (case.coins[b, i] and t >= 0 and t not in sib):
                t = _pick_excluding(float(case.u_token[b, i]), case.V, sib)
            sib.add(t)
            tokens[b, i] = t
    return tokens


def sampled_draft(case: Case, expert_logits_parent: np.ndarray):
    """Stand-in proposer for sampled workloads (the drafter itself is outside the
    verification step): node i's proposal is softmax((z_p of its parent row + eps_i) / T)
    with eps ~ N(0, 1), and its token is drawn from that proposal by inverse CDF.

    expert_logits_parent: [B*N, V] expert logits of each node's PARENT row (row 0 of
    every sequence is ignored).  Returns (draft_probs [B*N, V] fp32, tokens [B, N])."""
    R, V = case.R, case.V
    probs = np.zeros((R, V), dtype=np.float32)
    tokens = np.zeros((case.B, case.N), dtype=np.int32)
    for r in range(R):
        i = r % case.N
        if i == 0:
            continue
        x = (np.asarray(expert_logits_parent[r], dtype=np.float64) + case.eps[r]) / case.T
        x -= x.max()
        p = np.exp(x)
        p /= p.sum()
        probs[r] = p.astype(np.float32)
        c = np.cumsum(p)
        t = int(np.searchsorted(c, case.u_draw[r] * c[-1], side="right"))
        tokens[r // case.N, i] = min(t, V - 1)
    return probs, tokens
