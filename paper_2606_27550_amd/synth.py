"""Seeded synthetic inputs for the tree-verification step.

This module is shared by the oracle's tests and by the HIP path's tests and
benchmark.  It only draws random numbers and arranges them into the shapes of
the paper's workloads (Vicuna-7B / 13B shapes, Medusa/Hydra-style draft trees);
it performs none of the verification step's arithmetic.  Every tensor comes
from its own PCG64 stream keyed by (123, workload, tensor, layer, step,
attempt); 123 is the prompt-sampling seed of the paper's setup (§5.2).

Floating-point tensors are drawn in fp32 and rounded to bf16 with
round-to-nearest-even; they are returned as raw uint16 bit patterns so that
both sides of a parity check start from identical bits.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Sequence

import numpy as np

SEED = 123

# Stream identifiers: one per synthetic tensor kind.
S_TREE, S_Q, S_KT, S_VT, S_KC, S_VC, S_X, S_W, S_U, S_R = range(1, 11)
S_REGIME, S_SPIKE, S_PREFIX, S_BANK = range(11, 15)


def stream(workload: int, tensor: int, layer: int = 0, step: int = 0,
           attempt: int = 0) -> np.random.Generator:
    """Independent PCG64 generator for one (workload, tensor, layer, step, attempt)."""
    ss = np.random.SeedSequence([SEED, workload, tensor, layer, step, attempt])
    return np.random.Generator(np.random.PCG64(ss))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bits.

    Inputs are finite and far from the fp32 overflow threshold.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(g: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    x = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x)


# --------------------------------------------------------------------------
# Draft-tree shapes
# --------------------------------------------------------------------------

def _depths(parent: Sequence[int]) -> list[int]:
    d = [0] * len(parent)
    for i in range(1, len(parent)):
        d[i] = d[parent[i]] + 1
    return d


def uniform_attach_tree(workload: int, n_nodes: int, depth_cap: int,
                        tensor: int = S_TREE, layer: int = 0) -> list[int]:
    """Parent array of a tree grown node by node.

    Node 0 is the root.  Node i attaches to a uniformly chosen earlier node
    whose depth is below ``depth_cap``.  If the deepest node ends up shallower
    than the cap, the tree is redrawn from the next attempt's stream, so the
    realised depth always equals the cap.
    """
    if n_nodes < 1:
        raise ValueError("a tree has at least its root")
    if n_nodes == 1:
        return [-1]
    if depth_cap < 1 or depth_cap > n_nodes - 1:
        raise ValueError("depth cap must lie in [1, n_nodes-1]")
    for attempt in range(10_000):
        g = stream(workload, tensor, layer, 0, attempt)
        parent = [-1]
        depth = [0]
        for _ in range(1, n_nodes):
            cand = [j for j in range(len(parent)) if depth[j] < depth_cap]
            p = cand[int(g.integers(len(cand)))]
            parent.append(p)
            depth.append(depth[p] + 1)
        if max(depth) == depth_cap:
            return parent
    raise RuntimeError("could not realise the requested depth")


def level_width_tree(workload: int, widths: Sequence[int],
                     tensor: int = S_TREE, layer: int = 0) -> list[int]:
    """Tree with a fixed node count per depth (root at depth 0 not counted).

    Nodes are numbered level by level; each depth-d node picks a uniform
    parent among the depth-(d-1) nodes.
    """
    g = stream(workload, tensor, layer, 0, 0)
    parent = [-1]
    prev = [0]
    for w in widths:
        cur = []
        for _ in range(w):
            parent.append(prev[int(g.integers(len(prev)))])
            cur.append(len(parent) - 1)
        prev = cur
    return parent


def chain_tree(n_nodes: int) -> list[int]:
    return [-1] + list(range(n_nodes - 1))


def star_tree(n_nodes: int) -> list[int]:
    return [-1] + [0] * (n_nodes - 1)


def tree_depth(parent: Sequence[int]) -> int:
    return max(_depths(parent))


# --------------------------------------------------------------------------
# Draft tokens
# --------------------------------------------------------------------------

def draft_tokens(parent: Sequence[int], target_argmax: np.ndarray, u: np.ndarray,
                 r: np.ndarray, p_acc: float) -> np.ndarray:
    """Synthetic drafter: node i proposes the target's greedy token at its
    parent with probability ``p_acc`` (u[i] < p_acc), else the random token
    r[i].  The root's token is never verified; it is set to -1.
    """
    T = len(parent)
    tok = np.empty(T, dtype=np.int32)
    tok[0] = -1
    for i in range(1, T):
        tok[i] = target_argmax[parent[i]] if u[i] < p_acc else r[i]
    return tok


# --------------------------------------------------------------------------
# Workload descriptions (model shapes follow the paper's base models)
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    ident: int
    name: str
    n_heads: int
    n_kv_heads: int
    head_dim: int
    hidden: int
    vocab: int
    prefix_len: int
    n_layers: int
    p_acc: float
    rope_theta: float
    w_std: float = 0.02


WORKLOADS = {
    # one attention layer + LM head, Vicuna-7B shapes, one 27-node tree
    "tree27_L256_7b": Workload(1, "tree27_L256_7b", 32, 32, 128, 4096, 32000, 256, 1, 0.7, 10000.0),
    # Vicuna-7B shapes, 5-tree bank, prefix 2048 growing, per-step scheduler
    "bank5_L2048_7b": Workload(2, "bank5_L2048_7b", 32, 32, 128, 4096, 32000, 2048, 1, 0.7, 10000.0),
    # 32 layers of 7B attention, prefix 4096, 64-node depth-5 tree
    "tree64_L4096_7b_32layer": Workload(3, "tree64_L4096_7b_32layer", 32, 32, 128, 4096, 32000, 4096, 32, 0.7, 10000.0),
    # 13B shapes, prefix 8192, 128-node depth-6 tree
    "tree128_L8192_13b": Workload(4, "tree128_L8192_13b", 40, 40, 128, 5120, 32000, 8192, 1, 0.5, 10000.0),
    # batch 8, GQA 32:8, vocab 128256, ragged trees
    "batch8_gqa_v128k": Workload(5, "batch8_gqa_v128k", 32, 8, 128, 4096, 128256, 0, 1, 0.7, 10000.0),
}

# Node counts (root included) and depth caps of the 5-tree bank of the
# scheduler workload, sorted by size.
BANK5_SIZES = (1, 8, 26, 64, 128)
BANK5_CAPS = (0, 3, 4, 5, 6)
# Ragged bank of the batched workload.
BATCH_BANK_SIZES = (8, 16, 32, 64, 128)
BATCH_BANK_CAPS = (3, 4, 4, 5, 6)
# Per-depth node counts of the 13B workload's tree (sum 127, plus root = 128).
LEVEL_WIDTHS_13B = (40, 30, 22, 16, 11, 8)


def workload_trees(wl: Workload) -> list[list[int]]:
    """Parent arrays of the topology bank used by a workload."""
    if wl.ident == 1:
        return [uniform_attach_tree(wl.ident, 27, 4)]
    if wl.ident == 2:
        return [uniform_attach_tree(wl.ident, n, c, layer=k) if n > 1 else [-1]
                for k, (n, c) in enumerate(zip(BANK5_SIZES, BANK5_CAPS))]
    if wl.ident == 3:
        return [uniform_attach_tree(wl.ident, 64, 5)]
    if wl.ident == 4:
        return [level_width_tree(wl.ident, LEVEL_WIDTHS_13B)]
    if wl.ident == 5:
        return [uniform_attach_tree(wl.ident, n, c, layer=k)
                for k, (n, c) in enumerate(zip(BATCH_BANK_SIZES, BATCH_BANK_CAPS))]
    raise KeyError(wl.ident)


@dataclasses.dataclass
class AttnInputs:
    """One layer's attention inputs, as bf16 bit patterns."""
    q: np.ndarray        # [T, Hq, d]
    k_tree: np.ndarray   # [T, Hkv, d]
    v_tree: np.ndarray   # [T, Hkv, d]
    k_cache: np.ndarray  # [Hkv, cap, d]; rows >= prefix_len are zero
    v_cache: np.ndarray  # [Hkv, cap, d]


def attn_inputs(wl_ident: int, T: int, Hq: int, Hkv: int, d: int, prefix_len: int,
                cap: int, layer: int = 0, step: int = 0) -> AttnInputs:
    if cap < prefix_len + T:
        raise ValueError("cache capacity below prefix_len + T")
    q = normal_bf16(stream(wl_ident, S_Q, layer, step), (T, Hq, d))
    kt = normal_bf16(stream(wl_ident, S_KT, layer, step), (T, Hkv, d))
    vt = normal_bf16(stream(wl_ident, S_VT, layer, step), (T, Hkv, d))
    kc = np.zeros((Hkv, cap, d), dtype=np.uint16)
    vc = np.zeros((Hkv, cap, d), dtype=np.uint16)
    if prefix_len:
        kc[:, :prefix_len] = normal_bf16(stream(wl_ident, S_KC, layer, 0), (Hkv, prefix_len, d))
        vc[:, :prefix_len] = normal_bf16(stream(wl_ident, S_VC, layer, 0), (Hkv, prefix_len, d))
    return AttnInputs(q, kt, vt, kc, vc)


def lm_head_weight(wl_ident: int, vocab: int, hidden: int, std: float = 0.02,
                   copy: int = 0) -> np.ndarray:
    """LM-head weight [vocab, hidden] (nn.Linear layout) as bf16 bits."""
    return normal_bf16(stream(wl_ident, S_W, copy, 0), (vocab, hidden), std)


def hidden_rows(wl_ident: int, n_rows: int, hidden: int, step: int = 0,
                attempt: int = 0, layer: int = 0) -> np.ndarray:
    """Final hidden states of tree nodes [n_rows, hidden] as bf16 bits."""
    return normal_bf16(stream(wl_ident, S_X, layer, step, attempt), (n_rows, hidden))


def draft_randoms(wl_ident: int, n_rows: int, vocab: int, step: int = 0,
                  layer: int = 0) -> tuple[np.ndarray, np.ndarray]:
    """Per-node acceptance coin u ~ U[0,1) and replacement token r ~ U{0..V-1}."""
    u = stream(wl_ident, S_U, layer, step).random(n_rows)
    r = stream(wl_ident, S_R, layer, step).integers(0, vocab, n_rows, dtype=np.int64)
    return u, r.astype(np.int32)


def regime_spikes(wl_ident: int, n_steps: int, n_rows: int, vocab: int,
                  hidden: int, layer: int = 0):
    """Per-step confidence regime for the scheduler workload.

    A two-state Markov chain (stay probability 0.9) picks a high or low regime
    per step; the step draws a lift Delta ~ U[11, 18] (high) or U[0, 11] (low)
    and a planted token v_i per row.  Returns (delta[n_steps], tokens[n_steps,
    n_rows]).  The lift is applied by :func:`plant_spike`.
    """
    g = stream(wl_ident, S_REGIME, layer, 0)
    hi = bool(g.random() < 0.5)
    delta = np.empty(n_steps)
    for t in range(n_steps):
        if t and g.random() >= 0.9:
            hi = not hi
        delta[t] = g.uniform(11.0, 18.0) if hi else g.uniform(0.0, 11.0)
    toks = stream(wl_ident, S_SPIKE, layer, 0).integers(0, vocab, (n_steps, n_rows))
    return delta, toks.astype(np.int64)


def plant_spike(x_bits: np.ndarray, w_bits: np.ndarray, tokens: np.ndarray,
                delta: float, w_std: float) -> np.ndarray:
    """Add (delta / E||w||^2) * w[token_i] to row i of the hidden states.

    E||w||^2 = hidden * w_std^2 is the expected squared norm of a weight row,
    so the planted token's logit rises by about ``delta``.  Works in fp32 on
    the widened bf16 values and rounds back to bf16.
    """
    x = bf16_bits_to_f32(x_bits).copy()
    hidden = x.shape[1]
    c = np.float32(delta / (hidden * w_std * w_std))
    x += c * bf16_bits_to_f32(w_bits[tokens[: x.shape[0]]])
    return f32_to_bf16_bits(x)


def batch_prefix_lens(wl_ident: int, batch: int, lo: int = 512, hi: int = 16384) -> np.ndarray:
    return stream(wl_ident, S_PREFIX).integers(lo, hi + 1, batch).astype(np.int32)


def redraw_until(make: Callable[[int], np.ndarray], ok: Callable[[np.ndarray], np.ndarray],
                 max_attempts: int = 64) -> np.ndarray:
    """Row-wise redraw helper: ``make(attempt)`` gives candidate rows and
    ``ok(rows)`` a boolean per row; failing rows are replaced by the same row of
    the next attempt until all pass.  The test for a row is supplied by the
    caller."""
    rows = make(0).copy()
    good = ok(rows)
    attempt = 1
    while not good.all():
        if attempt >= max_attempts:
            raise RuntimeError("row redraw did not converge")
        cand = make(attempt)
        bad = ~good
        rows[bad] = cand[bad]
        good[bad] = ok(rows[bad])
        attempt += 1
    return rows
