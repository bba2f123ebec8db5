"""Plain CPU oracle for the EntMTP tree-verification step (fp64, slow, obvious).

TEST INFRASTRUCTURE.  Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  The library path never
calls it, and it shares no code with the HIP kernels or the C-ABI: every
function below is written from the paper's definitions (and the readings listed
in the design notes where the paper is silent).

What the step computes, in the paper's terms:

* ``bank_entry``: the per-tree buffers a precompiled bank ships with -- the
  tree attention mask, the position offsets and the gather/retrieve indices --
  for a draft tree given as a parent array (§2.3 Independent Multi-Head
  Prediction; §4 Inference-Time Tree Scheduler, "Cost").
* ``tree_attention``: one attention layer of the single sparse verification
  pass: every draft-tree node attends to the whole prefix and to its own
  root-to-node path (§2.3; §3.2 names the mask size as a verifier cost).
* ``verify_logits``: the target model's LM head applied to the tree's final
  hidden states (§2.2 gives the LM-head form softmax(W h)).
* ``logit_stats``: the per-node softmax statistics the scheduler reads: the
  top-1 probability p0 (§4, path-value score), the argmax, and the entropy
  (the paper's entropy signal, §3 and Appendix A).
* ``accept``: greedy verification -- the longest root-to-node path whose every
  draft token equals the target's argmax at the parent (§2.1, left-to-right
  acceptance, specialised to greedy decoding), and the accept length (§5.1).
* ``accept_typical``: the same walk under Hydra's typical acceptance
  condition (posterior threshold and entropy-scaled threshold, §5.1-§5.2).
* ``accept_stochastic``: speculative-sampling verification (min(1, p/p_hat)
  acceptance with residual resampling, §2.1) over the tree's children.
* ``kv_compact``: the KV-cache update that keeps the accepted path (§3.2,
  the proposal -> tree decoding -> verification -> KV-cache update loop).
* ``ladder_next``: the hysteretic threshold policy over a size-sorted bank
  (§4, "Policy").
* ``frontier_scores`` / ``frontier_select``: Algorithm 1's inner step -- every
  one-node augmentation of a tree scored from one rollout of the tree joined
  with its frontier, and the tie-broken choice of the node to add (§3.1).

Floating point is fp64 throughout.  Tensors that the interface stores as bf16
are passed in as uint16 bit patterns and widened exactly.
"""
from __future__ import annotations

import math
from typing import Sequence

import numpy as np

T_MAX = 256          # largest tree the bank accepts (root included)
D_MAX = 31           # deepest node the bank accepts
MASK_WORDS = T_MAX // 32


# --------------------------------------------------------------------------
# bf16 helpers (oracle's own)
# --------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns: the bits are the top half of an fp32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bf16 value (ties to even), as fp64.

    bf16 keeps 8 significant bits: with x = m * 2**e and 0.5 <= |m| < 1,
    the result is rint(m * 256) / 256 * 2**e.  Normal range only.
    """
    m, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(np.rint(m * 256.0), e - 8)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Bit pattern of round_to_bf16(x)."""
    r = round_to_bf16(x).astype(np.float32)       # exact: 8 significant bits
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# --------------------------------------------------------------------------
# TopologyBank entry (§2.3; §4 "Cost")
# --------------------------------------------------------------------------

def validate_parent(parent: Sequence[int]) -> None:
    T = len(parent)
    if T < 1 or T > T_MAX:
        raise ValueError(f"tree size {T} outside [1, {T_MAX}]")
    if parent[0] != -1:
        raise ValueError("the root (node 0) must have parent -1")
    for i in range(1, T):
        if not (0 <= parent[i] < i):
            raise ValueError(f"parent[{i}] = {parent[i]} is not an earlier node")


def ancestors_or_self(parent: Sequence[int], i: int) -> list[int]:
    """anc*(i): node i and every node on its path to the root, root first."""
    chain = []
    while i != -1:
        chain.append(i)
        i = parent[i]
    return chain[::-1]


def bank_entry(parent: Sequence[int]) -> dict:
    """Buffers of one draft tree.

    * ``depth[i]``: number of edges from the root (the position offset of node
      i: it sits at sequence position prefix_len + depth[i]).
    * ``mask[i]``: MASK_WORDS uint32 words; bit j (word j // 32, bit j % 32)
      is set iff j is an ancestor of i or i itself.  Bits >= T are zero.
    * ``path[i][k]``: the ancestor of i at depth k for k <= depth[i], else -1;
      shape [T, D+1] with D the tree's depth.
    * ``leaves``: nodes without children, ascending; ``retrieve[l] =
      path[leaves[l]]`` (the gather rows of each root-to-leaf candidate).
    """
    validate_parent(parent)
    T = len(parent)
    chains = [ancestors_or_self(parent, i) for i in range(T)]
    depth = np.array([len(c) - 1 for c in chains], dtype=np.int32)
    D = int(depth.max())
    if D > D_MAX:
        raise ValueError(f"tree depth {D} exceeds {D_MAX}")
    mask = np.zeros((T, MASK_WORDS), dtype=np.uint32)
    for i, c in enumerate(chains):
        for j in c:
            mask[i, j // 32] |= np.uint32(1 << (j % 32))
    path = np.full((T, D + 1), -1, dtype=np.int32)
    for i, c in enumerate(chains):
        path[i, : len(c)] = c
    has_child = [False] * T
    for i in range(1, T):
        has_child[parent[i]] = True
    leaves = np.array([i for i in range(T) if not has_child[i]], dtype=np.int32)
    retrieve = path[leaves].copy()
    return {"T": T, "D": D, "parent": np.asarray(parent, dtype=np.int32),
            "depth": depth, "mask": mask, "path": path, "leaves": leaves,
            "retrieve": retrieve}


# --------------------------------------------------------------------------
# Rotary position embedding (reading: Llama-family rotate-half convention)
# --------------------------------------------------------------------------

def rope(x: np.ndarray, pos: float, theta: float) -> np.ndarray:
    """Rotate a head vector to sequence position ``pos``.

    Pairs (c, c + d/2) form a 2-D vector turned by the angle
    pos * theta**(-2c/d).  ``x`` has shape [..., d].
    """
    d = x.shape[-1]
    half = d // 2
    c = np.arange(half, dtype=np.float64)
    ang = pos * np.power(float(theta), -2.0 * c / d)
    cos, sin = np.cos(ang), np.sin(ang)
    lo, hi = x[..., :half], x[..., half:]
    out = np.empty_like(x, dtype=np.float64)
    out[..., :half] = lo * cos - hi * sin
    out[..., half:] = hi * cos + lo * sin
    return out


# --------------------------------------------------------------------------
# Tree-masked attention (§2.3: single sparse forward pass over the tree)
# --------------------------------------------------------------------------

def tree_attention(q_bits, k_tree_bits, v_tree_bits, k_cache_bits, v_cache_bits,
                   prefix_len: int, parent: Sequence[int], scale: float,
                   rope_theta: float):
    """One attention layer of tree verification.

    q_bits [T, Hq, d], k/v_tree_bits [T, Hkv, d], caches [Hkv, cap, d]
    (bf16 bits).  Query head h uses KV head h // (Hq // Hkv).

    1. If rope_theta > 0, q_i and k_i are rotated to position
       prefix_len + depth(i); the rotated key is rounded to bf16 because the
       cache stores bf16.
    2. The tree's keys and values are written to cache slots prefix_len + i.
    3. Node i attends to cache slots [0, prefix_len) and to prefix_len + j for
       every j in anc*(i), with logits scale * (q . k), softmax in fp64.

    Returns (out [T, Hq, d] fp64, new k_cache bits, new v_cache bits).
    """
    validate_parent(parent)
    q = bf16_to_f64(q_bits)
    kt = bf16_to_f64(k_tree_bits)
    vt = bf16_to_f64(v_tree_bits)
    T, Hq, d = q.shape
    Hkv = kt.shape[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    group = Hq // Hkv
    L = int(prefix_len)
    cap = k_cache_bits.shape[1]
    if cap < L + T:
        raise ValueError("cache capacity below prefix_len + T")
    chains = [ancestors_or_self(parent, i) for i in range(T)]
    depth = [len(c) - 1 for c in chains]

    if rope_theta > 0:
        q = np.stack([rope(q[i], L + depth[i], rope_theta) for i in range(T)])
        kt = np.stack([rope(kt[i], L + depth[i], rope_theta) for i in range(T)])
        kt = round_to_bf16(kt)

    k_cache = np.array(k_cache_bits, dtype=np.uint16, copy=True)
    v_cache = np.array(v_cache_bits, dtype=np.uint16, copy=True)
    for i in range(T):
        k_cache[:, L + i] = f64_to_bf16_bits(kt[i])
        v_cache[:, L + i] = np.asarray(v_tree_bits[i], dtype=np.uint16)

    K = bf16_to_f64(k_cache[:, : L + T])
    V = bf16_to_f64(v_cache[:, : L + T])
    out = np.zeros((T, Hq, d), dtype=np.float64)
    for h in range(Hq):
        g = h // group
        # every node sees the whole prefix: one product for all nodes
        s_prefix = scale * (q[:, h] @ K[g, :L].T)            # [T, L]
        for i in range(T):
            tree_keys = [L + j for j in chains[i]]
            s = np.concatenate([s_prefix[i], scale * (K[g, tree_keys] @ q[i, h])])
            p = np.exp(s - s.max())
            p /= p.sum()
            out[i, h] = p[:L] @ V[g, :L] + p[L:] @ V[g, tree_keys]
    return out, k_cache, v_cache


# --------------------------------------------------------------------------
# LM-head verification logits (§2.2 LM-head form; §2.3 verification pass)
# --------------------------------------------------------------------------

def verify_logits(x_bits: np.ndarray, w_bits: np.ndarray) -> np.ndarray:
    """z[i, v] = sum_k X[i, k] * W[v, k], in fp64 (X [T, hid], W [V, hid])."""
    return bf16_to_f64(x_bits) @ bf16_to_f64(w_bits).T


def verify_logits_rows(x_bits: np.ndarray, w_bits: np.ndarray, cols) -> np.ndarray:
    """The same sums restricted to vocabulary rows ``cols`` (for sampled checks)."""
    return bf16_to_f64(x_bits) @ bf16_to_f64(w_bits[np.asarray(cols)]).T


# --------------------------------------------------------------------------
# Per-node softmax statistics (§4 path-value score; §3 / App. A entropy)
# --------------------------------------------------------------------------

def logit_stats_row(z: np.ndarray, inv_temp: float = 1.0):
    """(entropy in nats, top-1 probability, argmax) of softmax(inv_temp * z).

    The argmax is the lowest index attaining max(z).  With y = inv_temp * z,
    m = max(y), e_v = exp(y_v - m) and Z = sum e_v: p1 = 1 / Z and
    H = -sum p_v log p_v = log Z - sum (y_v - m) e_v / Z.  Terms with e_v = 0
    contribute 0 (this keeps -inf logits out of 0 * inf).
    """
    z = np.asarray(z, dtype=np.float64)
    zmax = z.max()
    amax = int(np.flatnonzero(z == zmax)[0])
    y = z * float(inv_temp)
    m = y.max()
    e = np.exp(y - m)
    Z = e.sum()
    nz = e > 0
    H = math.log(Z) - float(((y[nz] - m) * e[nz]).sum()) / Z
    return H, 1.0 / Z, amax


def logit_stats(z: np.ndarray, inv_temp: float = 1.0):
    """Row-wise :func:`logit_stats_row` over z [T, V]."""
    rows = [logit_stats_row(r, inv_temp) for r in np.atleast_2d(z)]
    H = np.array([r[0] for r in rows])
    p1 = np.array([r[1] for r in rows])
    am = np.array([r[2] for r in rows], dtype=np.int32)
    return H, p1, am


# --------------------------------------------------------------------------
# Longest accepted path (§2.1 left-to-right acceptance, greedy; §5.1)
# --------------------------------------------------------------------------

def accept(parent: Sequence[int], draft_tokens: Sequence[int], target_argmax: Sequence[int]):
    """Greedy tree verification.

    Node i >= 1 is accepted when its draft token equals the target's greedy
    token at its parent and its parent is accepted (the root always is).
    The answer is the deepest accepted node (lowest index among equals); the
    accept length a is its depth, the accepted path its root-to-node chain,
    and the bonus token the target's greedy token at that node.

    Returns (a, path [a+1], bonus, best).
    """
    validate_parent(parent)
    T = len(parent)
    depth = [0] * T
    ok = [True] + [False] * (T - 1)
    for i in range(1, T):      # parents precede children
        depth[i] = depth[parent[i]] + 1
        ok[i] = ok[parent[i]] and int(draft_tokens[i]) == int(target_argmax[parent[i]])
    best = 0
    for i in range(T):
        if ok[i] and depth[i] > depth[best]:
            best = i
    path = ancestors_or_self(parent, best)
    return depth[best], path, int(target_argmax[best]), best


def typical_probs(z_row, inv_temp: float):
    """Temperature-scaled next-token distribution of one node and its entropy
    in nats (the quantities the typical acceptance condition compares)."""
    y = np.asarray(z_row, dtype=np.float64) * float(inv_temp)
    y = y - y.max()
    e = np.exp(y)
    p = e / e.sum()
    nz = p > 0
    H = float(-(p[nz] * np.log(p[nz])).sum())
    return p, H


def accept_typical(parent: Sequence[int], draft_tokens: Sequence[int], z, inv_temp: float,
                   eps: float, alpha: float):
    """Typical-acceptance tree verification (the verification condition the
    paper keeps from Hydra, §5.1, with temperature T = 1 / inv_temp, posterior
    threshold eps and mixing coefficient alpha of §5.2; the rule itself is the
    published typical acceptance of Medusa/Hydra, not restated in the paper).

    Node i >= 1 is locally acceptable when its draft token's probability under
    its parent's distribution p = softmax(z[parent] * inv_temp) exceeds
    min(eps, alpha * exp(-H(p))); it is accepted when its parent is accepted
    too (the root always is).  The answer is the deepest accepted node; where
    several accepted nodes share that depth (siblings often pass together
    under this rule), the published rule keeps the candidate whose accepted
    tokens are jointly most likely: the largest sum of log p_draft over the
    node's root-to-node path, then the lowest index.  The bonus token is the
    argmax at the chosen node.

    z: the tree's logits [T][V].  Returns (a, path, bonus, best, p_draft,
    threshold) with p_draft[i] the draft token's probability under node i's
    parent (0 for the root) and threshold[j] node j's acceptance threshold.
    """
    validate_parent(parent)
    T = len(parent)
    probs, thr = [], []
    for j in range(T):
        p, H = typical_probs(z[j], inv_temp)
        probs.append(p)
        thr.append(min(float(eps), float(alpha) * math.exp(-H)))
    depth = [0] * T
    ok = [True] + [False] * (T - 1)
    p_draft = [0.0] * T
    for i in range(1, T):
        depth[i] = depth[parent[i]] + 1
        p_draft[i] = float(probs[parent[i]][int(draft_tokens[i])])
        ok[i] = ok[parent[i]] and p_draft[i] > thr[parent[i]]
    # joint log-likelihood of each accepted node's path (the root contributes 0)
    loglik = [0.0] * T
    for i in range(1, T):
        if ok[i]:
            loglik[i] = loglik[parent[i]] + math.log(p_draft[i])
    a = max(depth[i] for i in range(T) if ok[i])
    deepest = [i for i in range(T) if ok[i] and depth[i] == a]
    best = deepest[0]
    for i in deepest[1:]:          # ascending index: a later node must be strictly more likely
        if loglik[i] > loglik[best]:
            best = i
    path = ancestors_or_self(parent, best)
    bonus = int(np.argmax(np.asarray(z[best], dtype=np.float64)))
    return depth[best], path, bonus, best, np.array(p_draft), np.array(thr)


def _inverse_cdf(r: np.ndarray, u: float) -> int:
    """The smallest index b with r[0] + ... + r[b] > u * sum(r): a draw from
    the (unnormalised) distribution r with the uniform u."""
    c = np.cumsum(r)
    hit = np.nonzero(c > u * c[-1])[0]
    return int(hit[0]) if len(hit) else int(np.nonzero(r > 0)[0][-1])


def accept_stochastic(parent: Sequence[int], draft_tokens: Sequence[int], z, q, inv_temp: float,
                      u_accept: Sequence[float], u_sample: Sequence[float]):
    """Speculative-sampling verification of a draft tree (§2.1).

    §2.1 gives the rule for one chain: the draft token t at a position is kept
    with probability min(1, p(t) / p_hat(t)) -- p the target's distribution,
    p_hat the draft's -- left to right; at the first rejection the suffix is
    dropped and a replacement is drawn from norm(max(0, p - p_hat)).  On a
    tree the walk starts at the root with r = p at that node and tries the
    node's children in index (rank) order, each drafted from the node's draft
    distribution q[node]: child c passes when u_accept[c] * q(t_c) < r(t_c)
    (u < min(1, r / q); with q(t_c) = 0, when r(t_c) > 0).  The first child
    that passes becomes the current node, with r = p at it; each child that
    fails replaces r by norm(max(0, r - q[node])) before the next sibling is
    tried (recursive rejection sampling; for a chain it is exactly the rule
    above).  When no child passes, or the current node is a leaf, the bonus
    token is drawn from r with u_sample[node] (inverse CDF over the
    vocabulary in index order).  Should a residual vanish (r = q exactly in
    arithmetic), the distribution before that subtraction is kept.

    z [T][V] target logits, p = softmax(z * inv_temp); q [T][V] draft
    distributions.  Returns (a, path, bonus, best, trace) where trace lists
    every comparison made, as (child, u * q(t), r(t)), and last the draw,
    as ('sample', u * sum(r), cumulative sums around the drawn index).
    """
    validate_parent(parent)
    T = len(parent)
    d = depths(parent)
    children = [[] for _ in range(T)]
    for i in range(1, T):
        children[parent[i]].append(i)
    trace = []
    cur = 0
    while True:
        y = np.asarray(z[cur], dtype=np.float64) * float(inv_temp)
        e = np.exp(y - y.max())
        r = e / e.sum()
        qn = np.asarray(q[cur], dtype=np.float64)
        nxt = None
        for c in children[cur]:
            t = int(draft_tokens[c])
            lhs, rhs = float(u_accept[c]) * qn[t], r[t]
            trace.append((c, lhs, rhs))
            if (qn[t] > 0 and lhs < rhs) or (qn[t] == 0 and rhs > 0):
                nxt = c
                break
            w = np.maximum(r - qn, 0.0)
            if w.sum() > 0:
                r = w / w.sum()
        if nxt is None:
            bonus = _inverse_cdf(r, float(u_sample[cur]))
            c_all = np.cumsum(r)
            lo = c_all[bonus - 1] if bonus > 0 else 0.0
            trace.append(("sample", float(u_sample[cur]) * c_all[-1], lo, c_all[bonus]))
            path = ancestors_or_self(parent, cur)
            return d[cur], path, bonus, cur, trace
        cur = nxt


# --------------------------------------------------------------------------
# KV-cache update of the accepted path (§3.2 decode loop)
# --------------------------------------------------------------------------

def kv_compact(k_cache: np.ndarray, v_cache: np.ndarray, prefix_len: int,
               path: Sequence[int]):
    """Keep the accepted path's rows.  Caches are [..., cap, d] (any leading
    layer/head axes).  Row prefix_len + j receives the old row
    prefix_len + path[j] for j = 0..a; every other row is unchanged.
    """
    L = int(prefix_len)
    k_new = np.array(k_cache, copy=True)
    v_new = np.array(v_cache, copy=True)
    for j, src in enumerate(path):
        k_new[..., L + j, :] = k_cache[..., L + src, :]
        v_new[..., L + j, :] = v_cache[..., L + src, :]
    return k_new, v_new


# --------------------------------------------------------------------------
# Scheduler (§4 "Policy": hysteresis; K-way ladder over the bank)
# --------------------------------------------------------------------------

def ladder_next(rung: int, n_rungs: int, s: float, tau_on: float, tau_off: float) -> int:
    """One step of the hysteretic ladder over a size-sorted bank: climb one
    rung when s > tau_on, descend one when s <= tau_off, else stay."""
    if s > tau_on:
        return min(rung + 1, n_rungs - 1)
    if s <= tau_off:
        return max(rung - 1, 0)
    return rung


def binary_next(current_is_big: bool, s: float, tau_on: float, tau_off: float) -> bool:
    """The two-tree policy: switch to the aggressive tree when s > tau_on and
    back to the conservative one when s <= tau_off."""
    if s > tau_on:
        return True
    if s <= tau_off:
        return False
    return current_is_big


# --------------------------------------------------------------------------
# Acceptance frontier: scoring one-node augmentations (§3.1, Algorithm 1)
# --------------------------------------------------------------------------
#
# A node of a draft tree is named, as in Medusa/Hydra tree lists, by its tuple
# of child ranks along the root-to-node path; with a parent array whose
# children appear in rank order, a node's rank is the number of earlier
# siblings.  |nu| is the node's depth and sum(nu) its rank sum, Algorithm 1's
# tie-break keys.

def child_ranks(parent: Sequence[int]) -> list[int]:
    """Rank of every node among its parent's children (index order); 0 for
    the root."""
    validate_parent(parent)
    seen: dict[int, int] = {}
    rank = [0] * len(parent)
    for i in range(1, len(parent)):
        rank[i] = seen.get(parent[i], 0)
        seen[parent[i]] = rank[i] + 1
    return rank


def rank_sums(parent: Sequence[int]) -> list[int]:
    """sum(nu): the child ranks added up along each node's root-to-node path."""
    rank = child_ranks(parent)
    return [sum(rank[j] for j in ancestors_or_self(parent, i)) for i in range(len(parent))]


def depths(parent: Sequence[int]) -> list[int]:
    validate_parent(parent)
    d = [0] * len(parent)
    for i in range(1, len(parent)):
        d[i] = d[parent[i]] + 1
    return d


def next_children(parent: Sequence[int], max_depth: int) -> list[int]:
    """NextChildren(T, D) (Algorithm 1, not spelled out in the paper): every
    node of T, the root included, whose depth is below D proposes its
    next-ranked child.  Returns the candidates' parents, in node order."""
    d = depths(parent)
    return [p for p in range(len(parent)) if d[p] < max_depth]


def joint_tree(parent: Sequence[int], max_depth: int):
    """T joined with its frontier F: T's nodes keep their indices and the
    candidates follow in the order of next_children.  Returns (parent array
    of T u F, in_tree flags)."""
    cand = next_children(parent, max_depth)
    joint = list(parent) + cand
    return joint, [True] * len(parent) + [False] * len(cand)


def _accepted(parent: Sequence[int], ok_row) -> list[bool]:
    """Accepted nodes of one sample: the node and every ancestor below the
    root locally acceptable (the root always is)."""
    acc = [True] * len(parent)
    for i in range(1, len(parent)):
        acc[i] = acc[parent[i]] and bool(ok_row[i])
    return acc


def frontier_scores(parent: Sequence[int], in_tree: Sequence[bool], local_ok) -> list[int]:
    """Algorithm 1's scoring step over one rollout of the joint tree T u F:
    for each sample (one verification of the joint tree), the accept length
    of T is the deepest accepted node of T, and that of T u {nu} for a
    candidate nu is the larger of it and depth(nu) when nu itself is
    accepted -- a candidate's only ancestors are in T, so its acceptance does
    not depend on the other candidates.  local_ok[s][i]: node i's draft token
    passes the local test in sample s (greedy: it equals the target's argmax
    at the parent).  Returns, per node, the accept length summed over the
    samples: for candidates that of T u {nu}, for members of T that of T."""
    d = depths(parent)
    J = len(parent)
    sums = [0] * J
    for row in local_ok:
        acc = _accepted(parent, row)
        a_T = max(d[i] for i in range(J) if in_tree[i] and acc[i])
        for i in range(J):
            sums[i] += a_T if in_tree[i] else max(a_T, d[i] if acc[i] else 0)
    return sums


def frontier_select(parent: Sequence[int], in_tree: Sequence[bool], sums: Sequence[int]) -> int:
    """nu* = argmax over the candidates of (mean accept length, -sum(nu),
    -|nu|) (Algorithm 1); the mean over a common sample count orders as the
    sum.  Equal keys: the lower node index.  -1 when there is no candidate."""
    rs, d = rank_sums(parent), depths(parent)
    best, best_key = -1, None
    for i in range(len(parent)):
        if in_tree[i]:
            continue
        key = (sums[i], -rs[i], -d[i])
        if best_key is None or key > best_key:
            best, best_key = i, key
    return best


# --------------------------------------------------------------------------
# Whole step
# --------------------------------------------------------------------------

def verify_step(parent, q_bits, k_tree_bits, v_tree_bits, k_cache_bits, v_cache_bits,
                prefix_len, x_bits, w_bits, draft_tokens, scale, rope_theta,
                inv_temp=1.0):
    """One tree-verification step of one layer: attention (with the tree's
    K/V appended), LM-head logits, statistics, acceptance and compaction.

    The logits interface is fp32, so the statistics read the fp64 sums rounded
    to fp32 (the precision in which the argmax decision is taken).
    """
    out, kc, vc = tree_attention(q_bits, k_tree_bits, v_tree_bits, k_cache_bits,
                                 v_cache_bits, prefix_len, parent, scale, rope_theta)
    z = verify_logits(x_bits, w_bits).astype(np.float32)
    H, p1, am = logit_stats(z, inv_temp)
    a, path, bonus, best = accept(parent, draft_tokens, am)
    kc2, vc2 = kv_compact(kc, vc, prefix_len, path)
    return {"out": out, "logits": z, "entropy": H, "top1p": p1, "argmax": am,
            "accept_len": a, "path": path, "bonus": bonus, "best": best,
            "s": float(p1[best]), "k_cache": kc2, "v_cache": vc2}
