"""Pins of the oracle's whole verification step (not the GPU): lossless
verification, the property the paper states for greedy tree decoding (§2.1:
accepted drafts plus the bonus token are exactly what the target model would
have produced one token at a time; §5.1 accept length).

The oracle's step takes the tree's final hidden states as an input of their
own.  To pin its composition (statistics, acceptance, bonus token and
compaction) against something other than itself, these tests build a tiny
one-layer model whose hidden states do come from its attention: token t at
a position has query, key and value rows Eq[t], Ek[t], Ev[t] (rotated by
RoPE), the layer's attention output is the hidden state, and an LM head maps
it to logits.  Decoding that model one token at a time (a one-node tree per
token, which the attention pins equate with ordinary decode) gives the
reference token stream and cache rows.  A verification step over a draft
tree that contains those tokens must then emit the same tokens and leave the
same cache rows.
"""
import math

import numpy as np
import pytest

from oracle import entmtp_oracle as orc
from paper_2606_27550_amd import synth

V, H, D_HEAD = 64, 2, 16
HID = H * D_HEAD
L0 = 12
THETA = 10000.0
SCALE = 1 / math.sqrt(D_HEAD)
MARGIN = 1e-2


class ToyModel:
    """Embeddings, LM head and a prefix cache, all bf16 bit patterns."""

    def __init__(self, seed, depth):
        g = synth.stream(900 + seed, 1)
        self.Eq = synth.normal_bf16(g, (V, H, D_HEAD))
        self.Ek = synth.normal_bf16(g, (V, H, D_HEAD))
        self.Ev = synth.normal_bf16(g, (V, H, D_HEAD))
        self.W = synth.normal_bf16(g, (V, HID))
        cap = L0 + 64
        self.kc = np.zeros((H, cap, D_HEAD), np.uint16)
        self.vc = np.zeros((H, cap, D_HEAD), np.uint16)
        self.kc[:, :L0] = synth.normal_bf16(g, (H, L0, D_HEAD))
        self.vc[:, :L0] = synth.normal_bf16(g, (H, L0, D_HEAD))
        self.t0 = int(g.integers(V))

    def rows(self, tokens):
        tok = np.asarray(tokens)
        return self.Eq[tok], self.Ek[tok], self.Ev[tok]

    def hidden(self, out):
        """Attention output [T, H, d] (fp64) -> hidden states [T, HID] (bf16 bits)."""
        return orc.f64_to_bf16_bits(out.reshape(out.shape[0], HID))

    def decode(self, n):
        """n tokens, one at a time, greedily; returns (tokens, k cache, v cache,
        smallest top-2 logit gap seen)."""
        kc, vc, tok, L = self.kc, self.vc, self.t0, L0
        emitted, gap = [], np.inf
        for _ in range(n):
            q, k, v = self.rows([tok])
            out, kc, vc = orc.tree_attention(q, k, v, kc, vc, L, [-1], SCALE, THETA)
            z = orc.verify_logits(self.hidden(out), self.W)[0]
            top2 = np.sort(z)[-2:]
            gap = min(gap, top2[1] - top2[0])
            tok = int(np.argmax(z))
            emitted.append(tok)
            L += 1
        return emitted, kc, vc, gap

    def verify(self, parent, tokens):
        """One verification step of the draft tree (tokens[0] is the root's,
        the last committed token): the tree's hidden states are the model's
        own (its attention over the prefix and the node's path), then the
        oracle's step."""
        q, k, v = self.rows(tokens)
        out, _, _ = orc.tree_attention(q, k, v, self.kc, self.vc, L0, parent, SCALE, THETA)
        x = self.hidden(out)
        drafts = np.asarray(tokens, np.int32).copy()
        drafts[0] = -1
        return orc.verify_step(parent, q, k, v, self.kc, self.vc, L0, x, self.W, drafts, SCALE,
                               THETA)


def model_for(seed, depth):
    """A seed whose greedy stream keeps a top-2 gap above the margin, so the
    argmax decision does not depend on rounding order."""
    for s in range(seed, seed + 50):
        m = ToyModel(s, depth)
        toks, kc, vc, gap = m.decode(depth + 1)
        if gap >= MARGIN:
            return m, toks, kc, vc
    raise RuntimeError("no seed with a clear greedy stream")


def emitted(ref, tokens):
    """Accepted drafts along the accepted path, then the bonus token."""
    return [int(tokens[i]) for i in ref["path"][1:]] + [ref["bonus"]]


@pytest.mark.parametrize("seed,depth", [(1, 1), (2, 4), (3, 6)])
def test_chain_of_greedy_drafts_equals_sequential_decoding(seed, depth):
    m, seq, kc_seq, vc_seq = model_for(seed, depth)
    parent = synth.chain_tree(depth + 1)
    tokens = [m.t0] + seq[:depth]
    ref = m.verify(parent, tokens)
    assert ref["accept_len"] == depth
    assert emitted(ref, tokens) == seq                      # depth drafts + the bonus token
    # the compacted cache holds exactly the rows sequential decoding wrote
    n = L0 + depth + 1
    np.testing.assert_array_equal(ref["k_cache"][:, :n], kc_seq[:, :n])
    np.testing.assert_array_equal(ref["v_cache"][:, :n], vc_seq[:, :n])


@pytest.mark.parametrize("seed,depth", [(4, 3), (5, 5)])
def test_branching_tree_accepts_the_greedy_branch(seed, depth):
    """The greedy stream as one branch of a tree whose every level also holds
    a wrong sibling (numbered before the right one) and a wrong grandchild
    under it: the step accepts the greedy branch, emits the sequential
    tokens, and the other branches neither leak into its attention (its
    hidden states, hence its argmax chain, would change) nor into the
    cache."""
    m, seq, kc_seq, vc_seq = model_for(seed, depth)
    parent, tokens, good = [-1], [m.t0], 0
    for lvl in range(depth):
        right = seq[lvl]
        wrong = (right + 1 + lvl) % V
        parent.append(good)                 # a wrong sibling first
        tokens.append(wrong)
        parent.append(len(parent) - 1)      # its child (never reachable)
        tokens.append(seq[lvl + 1] if lvl + 1 < len(seq) else right)
        parent.append(good)                 # then the greedy token
        tokens.append(right)
        good = len(parent) - 1
    ref = m.verify(parent, tokens)
    assert ref["accept_len"] == depth
    assert emitted(ref, tokens) == seq
    n = L0 + depth + 1
    np.testing.assert_array_equal(ref["k_cache"][:, :n], kc_seq[:, :n])
    np.testing.assert_array_equal(ref["v_cache"][:, :n], vc_seq[:, :n])


@pytest.mark.parametrize("seed", range(6))
def test_any_drafts_emit_a_prefix_of_the_sequential_stream(seed):
    """Whatever the drafts, what a step emits (its accepted drafts and the
    bonus token) is the first a + 1 tokens of sequential greedy decoding, and
    the cache rows of those tokens are the sequential ones."""
    depth = 5
    m, seq, kc_seq, vc_seq = model_for(10 + seed, depth)
    g = np.random.default_rng(seed)
    drafts = [t if g.random() < 0.6 else int(g.integers(V)) for t in seq[:depth]]
    parent = synth.chain_tree(depth + 1)
    tokens = [m.t0] + drafts
    ref = m.verify(parent, tokens)
    a = ref["accept_len"]
    k = next((i for i, (d_, s_) in enumerate(zip(drafts, seq)) if d_ != s_), depth)
    assert a == k                                # the first wrong draft stops the walk
    assert emitted(ref, tokens) == seq[: a + 1]
    n = L0 + a + 1
    np.testing.assert_array_equal(ref["k_cache"][:, :n], kc_seq[:, :n])
    np.testing.assert_array_equal(ref["v_cache"][:, :n], vc_seq[:, :n])
