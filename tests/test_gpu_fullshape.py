"""GPU parity at the shapes the benchmark times.

The closed-loop tests of test_gpu_step.py use hidden size 512 and a 1000-token
vocabulary.  There the LM head's grid stays below two workgroups per CU, so
the step takes other kernel instantiations than at the model shapes: no
paired vocabulary slices, no fully unrolled K loop, 125 partials per node.
Here each workload the benchmark times runs through the step driver (or
through the entry points the batched step calls) at its own shapes, and
every step is compared with the oracle replaying the same trees from its own
cache state (the paper's verification pass, §2.3, and the decode loop with
the tree scheduler, §4):

* the 27-node tree at prefix 256 with Vicuna-7B shapes (hidden 4096,
  vocabulary 32000, 32 x 128 heads), armed as the benchmark runs it;
* the 5-tree bank {1, 8, 26, 64, 128} at prefix 2048 with the prefix growing.
  Every tree goes through its own-size LM head and through the larger armed
  LM heads the ladder can reach (folded slice pairs up to 32 nodes, paired
  64- and 128-node tiles);
* the same bank with the tree chosen on the GPU (device-sized LM heads and
  attention, the ladder beside the statistics), its step log replayed on the
  oracle;
* the 13B shapes (hidden 5120, 40 heads, prefix 8192, the 128-node tree);
* the 128256-token vocabulary: the merge of 2048 statistics partials per node
  (the merge's two-pass branch above 512 partials) over 136 rows, and a step
  over the batched workload's bank with GQA 32:8 (1024 folded partials per
  small-tree node).

Bars: argmax, accept length, path (the whole buffer: -1 past the accept
length), bonus token and compacted cache bit-exact; attention outputs within
2e-2 absolute; entropy, top-1 probability and s within 1e-3 relative (plus
1e-6 absolute).
"""
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import entmtp_oracle as orc  # noqa: E402
from paper_2606_27550_amd import synth  # noqa: E402
from tests.helpers import dev_bf16, dev_i32, host_bits, margin_hidden  # noqa: E402

pytestmark = pytest.mark.gpu

ATOL_BF16 = 2e-2
RTOL_STATS = 1e-3
ATOL_STATS = 1e-6
TAU_ON, TAU_OFF = 0.8, 0.6


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


def say(*a):
    print("[gpu-test]", *a, flush=True)


class Weights:
    """LM-head weight of a workload: bits, exact fp64 widening, device copy."""

    def __init__(self, ident, V, hid, std):
        self.bits = synth.lm_head_weight(ident, V, hid, std=std)
        self.f64 = orc.bf16_to_f64(self.bits)
        self.dev = dev_bf16(self.bits)
        self.std = std


_WEIGHTS = {}


def weights(ident, V, hid, std=0.02):
    key = (ident, V, hid, std)
    if key not in _WEIGHTS:
        _WEIGHTS.clear()          # one model-sized weight in memory at a time
        say(f"drawing LM-head weight V={V} hid={hid}")
        _WEIGHTS[key] = Weights(ident, V, hid, std)
    return _WEIGHTS[key]


def step_host_inputs(ident, t, Tmax, Hq, Hkv, d, w, lift=None):
    """Step t's tree inputs (bit patterns): one attention layer, the tree's
    final hidden states with the top-2 margin (and the scheduler workload's
    planted lift), their target argmax and the drafter's coins."""
    a_in = synth.attn_inputs(ident, Tmax, Hq, Hkv, d, 0, Tmax, step=t + 1)
    x = margin_hidden(ident, Tmax, w.bits, step=t + 1, w64=w.f64, spikes=lift, w_std=w.std)
    am = (orc.bf16_to_f64(x) @ w.f64.T).argmax(axis=1)
    u, r = synth.draft_randoms(ident, Tmax, w.bits.shape[0], step=t + 1)
    return a_in, x, am, u, r


def check_step(st, out_h, T, a, bonus, s, ref, heads=None):
    """The step's device outputs against the oracle's step (one layer)."""
    want = ref["out"] if heads is None else ref["out"][:, heads]
    got = out_h[:T] if heads is None else out_h[:T, heads]
    err = float(np.abs(got - want).max())
    assert err <= ATOL_BF16, f"attention max abs error {err}"
    np.testing.assert_array_equal(st.argmax[:T].cpu().numpy(), ref["argmax"])
    np.testing.assert_allclose(st.entropy[:T].cpu().numpy(), ref["entropy"], rtol=RTOL_STATS,
                               atol=ATOL_STATS)
    np.testing.assert_allclose(st.top1p[:T].cpu().numpy(), ref["top1p"], rtol=RTOL_STATS,
                               atol=ATOL_STATS)
    assert (a, bonus) == (ref["accept_len"], ref["bonus"])
    assert (int(st.accept_len.item()), int(st.bonus.item())) == (a, bonus)
    path = st.path.cpu().numpy()
    assert path[: a + 1].tolist() == list(ref["path"])
    assert (path[a + 1:] == -1).all(), path          # the whole buffer, whatever the tree's depth
    assert abs(s - ref["s"]) <= RTOL_STATS * ref["s"] + ATOL_STATS
    return err


def host_scheduled_run(api, wl, trees, rungs, *, L0, grows, arm, flush_each, lifts=None,
                       heads=None, V=None):
    """Host-scheduled steps through entmtp_step_launch / _arm / _wait on the
    given tree sequence; each step against the oracle's step from the
    oracle's own cache chain, and the caches bit for bit (after every step
    when flush_each, else after the final flush).  arm: each next step's LM
    head is enqueued while the step before is pending, for the largest tree
    the ladder can reach (the next rung), as the benchmark runs it."""
    Hq, Hkv, d, hid = wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.hidden
    V = V or wl.vocab
    scale, theta = 1 / math.sqrt(d), wl.rope_theta
    bank = api.Bank(trees)
    K, Tmax, Dmax = len(trees), max(bank.T), max(bank.D)
    n = len(rungs)
    cap = L0 + (n * (Dmax + 1) if grows else 0) + Tmax + 8
    w = weights(wl.ident, V, hid, wl.w_std)
    base = synth.attn_inputs(wl.ident, 1, Hq, Hkv, d, L0, cap)
    kc_o, vc_o = base.k_cache, base.v_cache            # the oracle's cache chain
    kc, vc = dev_bf16(kc_o), dev_bf16(vc_o)
    st = api.Step(bank, kc, vc, w.dev, Hq=Hq, Hkv=Hkv, d=d, cap=cap, tree_rows=Tmax, scale=scale,
                  rope_theta=theta, keep_logits=False)
    out = torch.empty((Tmax, Hq, d), dtype=torch.bfloat16, device="cuda")

    def inputs(t):
        host = step_host_inputs(wl.ident, t, Tmax, Hq, Hkv, d, w, None if lifts is None else lifts[t])
        a_in, x = host[0], host[1]
        return host, (dev_bf16(a_in.q), dev_bf16(a_in.k_tree), dev_bf16(a_in.v_tree), dev_bf16(x))

    L, ahead, errs = L0, None, []
    for t, r in enumerate(rungs):
        T, parent = bank.T[r], trees[r]
        (a_in, x, am, u, r_tok), (q, kt, vt, X) = ahead if ahead is not None else inputs(t)
        ahead = None
        tok = synth.draft_tokens(parent, am, u, r_tok, wl.p_acc)
        say(f"{wl.name} step {t}: tree {r} ({T} nodes) prefix {L}")
        tok_d = dev_i32(tok)        # kept alive until the acceptance has read it
        st.launch(r, L, q, kt, vt, out, X, tok_d)
        if arm and t + 1 < n:
            ahead = inputs(t + 1)
            st.arm(ahead[1][3], bank.T[min(r + 1, K - 1)])
        a, bonus, s = st.wait(timeout_s=60.0)
        if flush_each:
            st.flush()
        torch.cuda.synchronize()
        out_h = out.float().cpu().numpy()
        ref = orc.verify_step(parent, a_in.q[:T], a_in.k_tree[:T], a_in.v_tree[:T], kc_o, vc_o, L,
                              x[:T], w.bits, tok, scale, theta)
        errs.append(check_step(st, out_h, T, a, bonus, s, ref, heads))
        kc_o, vc_o = ref["k_cache"], ref["v_cache"]
        end = L + a + 1
        if flush_each:
            np.testing.assert_array_equal(host_bits(kc)[:, :end], kc_o[:, :end])
            np.testing.assert_array_equal(host_bits(vc)[:, :end], vc_o[:, :end])
        if grows:
            L = end
    st.flush()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_bits(kc)[:, :end], kc_o[:, :end])
    np.testing.assert_array_equal(host_bits(vc)[:, :end], vc_o[:, :end])
    st.close()
    say(f"{wl.name}: max attention error per step {[f'{e:.1e}' for e in errs]}")


def test_step_tree27_L256_7b(api):
    """The 27-node workload as the benchmark runs it: the prefix reset to 256
    every step, each next LM head armed (27 rows: the 32-node folded tile),
    the compaction checked after every step."""
    wl = synth.WORKLOADS["tree27_L256_7b"]
    host_scheduled_run(api, wl, synth.workload_trees(wl), [0] * 4, L0=wl.prefix_len, grows=False,
                       arm=True, flush_each=True)


def test_step_bank5_L2048_7b_every_tree_and_armed_tile(api):
    """The 5-tree bank at prefix 2048, the prefix growing.  The tree sequence
    climbs and descends the ladder one rung at a time, so with arming (sized
    for the next rung) each tree runs through its own LM-head tile and
    through a larger one: 1 node through the 1-, 16- and 32-row tiles, 8
    through 8 and 64, 26 through 26 and 128, 64 through 64 and 128, 128
    through the paired 128-node tile."""
    wl = synth.WORKLOADS["bank5_L2048_7b"]
    trees = synth.workload_trees(wl)
    rungs = [0, 1, 2, 3, 4, 4, 3, 2, 1, 0, 0]
    deltas, toks = synth.regime_spikes(wl.ident, len(rungs), max(map(len, trees)), wl.vocab,
                                       wl.hidden)
    lifts = [(float(deltas[t]), toks[t]) for t in range(len(rungs))]
    host_scheduled_run(api, wl, trees, rungs, L0=wl.prefix_len, grows=True, arm=True,
                       flush_each=False, lifts=lifts)


def test_step_bank5_L2048_7b_unarmed(api):
    """The same bank without arming: every LM head sized for its own tree."""
    wl = synth.WORKLOADS["bank5_L2048_7b"]
    trees = synth.workload_trees(wl)
    rungs = [4, 3, 2, 1, 0]
    host_scheduled_run(api, wl, trees, rungs, L0=wl.prefix_len, grows=True, arm=False,
                       flush_each=True)


def test_device_scheduled_bank5_L2048_7b_replayed_on_oracle(api):
    """Device-scheduled steps at the bank's shapes (the ladder on the GPU,
    device-sized LM heads and attention; nothing read back until the end).
    The step log (tree, prefix length, accept length, s) is replayed on the
    oracle step by step: each step's tree and prefix must be the oracle's,
    its accept length exact and s within 1e-3; each next tree must be the
    ladder's choice on the oracle's s unless that s lies within 1e-3 of a
    threshold, where the GPU's choice is followed.  Attention outputs of
    every step, the final caches and the last step's statistics and path are
    compared as well.  Planted lifts far from the thresholds (2 or 16) move
    the ladder down from the 128-node tree and back up."""
    wl = synth.WORKLOADS["bank5_L2048_7b"]
    Hq, Hkv, d, hid, V = wl.n_heads, wl.n_kv_heads, wl.head_dim, wl.hidden, wl.vocab
    scale, theta = 1 / math.sqrt(d), wl.rope_theta
    trees = synth.workload_trees(wl)
    bank = api.Bank(trees)
    K, Tmax, Dmax = len(trees), max(bank.T), max(bank.D)
    lift_sched = [2.0, 2.0, 2.0, 16.0, 16.0, 2.0, 16.0, 2.0]
    n = len(lift_sched)
    L0 = wl.prefix_len
    cap = L0 + n * (Dmax + 1) + Tmax + 8
    w = weights(wl.ident, V, hid, wl.w_std)
    base = synth.attn_inputs(wl.ident, 1, Hq, Hkv, d, L0, cap)
    kc_o, vc_o = base.k_cache, base.v_cache
    kc, vc = dev_bf16(kc_o), dev_bf16(vc_o)
    st = api.Step(bank, kc, vc, w.dev, Hq=Hq, Hkv=Hkv, d=d, cap=cap, tree_rows=Tmax, scale=scale,
                  rope_theta=theta, keep_logits=False, tau_on=TAU_ON, tau_off=TAU_OFF)
    _, toks = synth.regime_spikes(wl.ident, n, Tmax, V, hid)
    host, dev_in = [], []
    for t in range(n):
        a_in, x, am, u, r = step_host_inputs(wl.ident, t, Tmax, Hq, Hkv, d, w,
                                             (lift_sched[t], toks[t]))
        drafts = np.zeros((K, Tmax), np.int32)
        for k in range(K):
            drafts[k, : bank.T[k]] = synth.draft_tokens(trees[k], am, u, r, wl.p_acc)
        host.append((a_in, x, drafts))
        dev_in.append((dev_bf16(a_in.q), dev_bf16(a_in.k_tree), dev_bf16(a_in.v_tree), dev_bf16(x),
                       dev_i32(drafts)))
    outs = [torch.zeros((Tmax, Hq, d), dtype=torch.bfloat16, device="cuda") for _ in range(n)]
    log = torch.full((n, 4), -1, dtype=torch.int32, device="cuda")
    say("device-scheduled bank5: enqueue", n, "steps")
    st.device_start(K - 1, L0)
    for t in range(n):
        q, kt, vt, X, dr = dev_in[t]
        st.launch_device(q, kt, vt, outs[t], X, dr, log)
    st.flush()
    torch.cuda.synchronize()
    log_h = log.cpu().numpy()
    say("device log", log_h[:, :3].tolist())

    rung, L, visited = K - 1, L0, set()
    for t in range(n):
        a_in, x, drafts = host[t]
        T = bank.T[rung]
        visited.add(rung)
        g_rung, g_L, g_a = (int(v) for v in log_h[t, :3])
        g_s = float(log_h[t, 3:4].view(np.float32)[0])
        assert (g_rung, g_L) == (rung, L), (t, log_h[t])
        ref = orc.verify_step(trees[rung], a_in.q[:T], a_in.k_tree[:T], a_in.v_tree[:T], kc_o, vc_o,
                              L, x[:T], w.bits, drafts[rung, :T], scale, theta)
        assert g_a == ref["accept_len"], (t, g_a, ref["accept_len"])
        assert abs(g_s - ref["s"]) <= RTOL_STATS * ref["s"] + ATOL_STATS
        err = float(np.abs(outs[t][:T].float().cpu().numpy() - ref["out"]).max())
        assert err <= ATOL_BF16, (t, err)
        kc_o, vc_o = ref["k_cache"], ref["v_cache"]
        L += g_a + 1
        nxt = orc.ladder_next(rung, K, ref["s"], TAU_ON, TAU_OFF)
        if t + 1 < n and int(log_h[t + 1, 0]) != nxt:
            near = min(abs(ref["s"] - TAU_ON) / TAU_ON, abs(ref["s"] - TAU_OFF) / TAU_OFF)
            assert near <= RTOL_STATS, (t, ref["s"], int(log_h[t + 1, 0]), nxt)
            nxt = int(log_h[t + 1, 0])
        last = (ref, T)
        rung = nxt
    assert len(visited) >= 3, visited
    ref, T = last
    np.testing.assert_array_equal(st.argmax[:T].cpu().numpy(), ref["argmax"])
    np.testing.assert_allclose(st.top1p[:T].cpu().numpy(), ref["top1p"], rtol=RTOL_STATS,
                               atol=ATOL_STATS)
    np.testing.assert_allclose(st.entropy[:T].cpu().numpy(), ref["entropy"], rtol=RTOL_STATS,
                               atol=ATOL_STATS)
    path = st.path.cpu().numpy()
    a = ref["accept_len"]
    assert path[: a + 1].tolist() == list(ref["path"]) and (path[a + 1:] == -1).all()
    np.testing.assert_array_equal(host_bits(kc)[:, :L], kc_o[:, :L])
    np.testing.assert_array_equal(host_bits(vc)[:, :L], vc_o[:, :L])
    st.close()


def test_step_tree128_L8192_13b(api):
    """13B shapes: 40 x 128 heads, hidden 5120, prefix 8192, the 128-node tree
    of six levels; the paired 128-node tile with the 40-chunk K loop beside
    the four-tile attention."""
    wl = synth.WORKLOADS["tree128_L8192_13b"]
    host_scheduled_run(api, wl, synth.workload_trees(wl), [0, 0], L0=wl.prefix_len, grows=False,
                       arm=True, flush_each=True)


def test_step_v128k_gqa_bank(api):
    """The batched workload's bank through the single-sequence step at its
    shapes (GQA 32:8, vocabulary 128256): 16- and 32-node trees merge 1024
    folded partials per node in the fused finalize-accept kernel, 64- and
    128-node trees 2048 partials (two-pass merge) in the statistics kernel,
    the 128-node tree through the paired tile."""
    wl = synth.WORKLOADS["batch8_gqa_v128k"]
    trees = synth.workload_trees(wl)
    host_scheduled_run(api, wl, trees, [1, 2, 3, 4], L0=1000, grows=True, arm=True,
                       flush_each=True)


def test_stats_v128k_two_pass_merge(api):
    """136 rows at vocabulary 128256 through the two halves of the fused
    statistics: the LM head writes 2048 partials per node (128-node tiles,
    two passes), and the finalize merges them with its read-twice branch.
    Logits on sampled columns, argmax bit-exact, entropy and top-1
    probability within 1e-3 of the oracle's statistics of the fp32 logits."""
    wl = synth.WORKLOADS["batch8_gqa_v128k"]
    T, hid, V = 136, wl.hidden, wl.vocab
    w = weights(wl.ident, V, hid, wl.w_std)
    x = margin_hidden(wl.ident, T, w.bits, step=99, w64=w.f64, w_std=w.std)
    X = dev_bf16(x)
    nbytes = api.stats_partials_bytes(T, hid, V)
    assert nbytes == T * 2048 * 16, nbytes      # 2048 partials of 16 bytes per node
    part = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    logits = torch.empty((T, V), dtype=torch.float32, device="cuda")
    H, p1 = torch.empty(T, device="cuda"), torch.empty(T, device="cuda")
    am = torch.empty(T, dtype=torch.int32, device="cuda")
    api.verify_logits_partials(X, w.dev, logits, 1.0, part)
    api.stats_finalize(part, T, V, 1.0, H, p1, am)
    torch.cuda.synchronize()
    z = orc.verify_logits(x, w.bits).astype(np.float32)
    rH, rp1, ram = orc.logit_stats(z)
    np.testing.assert_array_equal(am.cpu().numpy(), ram)
    np.testing.assert_allclose(H.cpu().numpy(), rH, rtol=RTOL_STATS, atol=ATOL_STATS)
    np.testing.assert_allclose(p1.cpu().numpy(), rp1, rtol=RTOL_STATS, atol=ATOL_STATS)
    cols = np.random.default_rng(3).choice(V, 512, replace=False)
    err = float(np.abs(logits.cpu().numpy()[:, cols] - z[:, cols]).max())
    assert err <= ATOL_BF16, err
