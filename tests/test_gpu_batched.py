"""GPU parity of the batched entry points (several sequences per call, each
with its own tree from the bank, its own prefix length and its own cache)
against the oracle, sequence by sequence.

Bars as for the single-sequence calls: max abs error 2e-2 for attention
outputs, bit-exact cache appends, acceptance and compaction.
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
WL = synth.WORKLOADS["batch8_gqa_v128k"]
D_HEAD = 128
THETA = 10000.0


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


@pytest.fixture(scope="module")
def trees():
    return synth.workload_trees(WL)


def say(*a):
    print("[gpu-test]", *a, flush=True)


def batch_inputs(trees, topo, lens, Hq, Hkv, cap, seed):
    """Per-sequence attention inputs, stacked the way the batched calls take them."""
    inp = [synth.attn_inputs(seed, len(trees[t]), Hq, Hkv, D_HEAD, L, cap, step=b + 1)
           for b, (t, L) in enumerate(zip(topo, lens))]
    cat = lambda name: np.ascontiguousarray(np.concatenate([getattr(x, name) for x in inp]))
    return inp, cat("q"), cat("k_tree"), cat("v_tree")


def run_batched_attn(api, trees, topo, lens, Hq, Hkv, cap, seed):
    bank = api.Bank(trees)
    inp, q, kt, vt = batch_inputs(trees, topo, lens, Hq, Hkv, cap, seed)
    kcs = [dev_bf16(x.k_cache) for x in inp]
    vcs = [dev_bf16(x.v_cache) for x in inp]
    rows = q.shape[0]
    out = torch.full((rows, Hq, D_HEAD), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(api.tree_attn_batched_workspace(len(topo), max(bank.T), Hq, Hkv, D_HEAD, max(lens)),
                     dtype=torch.uint8, device="cuda")
    api.tree_attn_batched(bank, topo, lens, dev_bf16(q), dev_bf16(kt), dev_bf16(vt), kcs, vcs,
                          1 / math.sqrt(D_HEAD), THETA, out, ws)
    torch.cuda.synchronize()
    return inp, out.float().cpu().numpy(), [host_bits(k) for k in kcs], [host_bits(v) for v in vcs]


def test_tree_attn_batched_small(api, trees):
    topo = [0, 4, 2, 1, 3, 4]
    lens = [0, 37, 300, 513, 90, 1000]
    Hq, Hkv = 8, 2
    cap = max(lens) + 128 + 5
    say("tree_attn_batched", topo, lens)
    inp, out, kcs, vcs = run_batched_attn(api, trees, topo, lens, Hq, Hkv, cap, 91)
    row = 0
    for b, (t, L) in enumerate(zip(topo, lens)):
        T = len(trees[t])
        ref, rk, rv = orc.tree_attention(inp[b].q, inp[b].k_tree, inp[b].v_tree, inp[b].k_cache,
                                         inp[b].v_cache, L, trees[t], 1 / math.sqrt(D_HEAD), THETA)
        err = np.abs(out[row:row + T] - ref).max()
        assert err <= ATOL_BF16, (b, err)
        np.testing.assert_array_equal(kcs[b][:, : L + T], rk[:, : L + T])
        np.testing.assert_array_equal(vcs[b][:, : L + T], rv[:, : L + T])
        row += T


def test_tree_attn_batched_full_shapes_sampled_heads(api, trees):
    """Batch of 8 at the workload's shapes (GQA 32:8, prefixes 512..16384);
    one KV head per sequence checked against the oracle."""
    B, Hq, Hkv = 8, WL.n_heads, WL.n_kv_heads
    lens = [int(x) for x in synth.batch_prefix_lens(WL.ident, B)]
    topo = [b % len(trees) for b in range(B)]
    cap = max(lens) + 128 + 8
    say("tree_attn_batched full shapes", topo, lens)
    inp, out, kcs, vcs = run_batched_attn(api, trees, topo, lens, Hq, Hkv, cap, WL.ident)
    assert np.isfinite(out).all()
    G = Hq // Hkv
    row = 0
    for b, (t, L) in enumerate(zip(topo, lens)):
        T = len(trees[t])
        g = b % Hkv
        x = inp[b]
        ref, rk, rv = orc.tree_attention(x.q[:, g * G:(g + 1) * G], x.k_tree[:, g:g + 1],
                                         x.v_tree[:, g:g + 1], x.k_cache[g:g + 1], x.v_cache[g:g + 1],
                                         L, trees[t], 1 / math.sqrt(D_HEAD), THETA)
        err = np.abs(out[row:row + T, g * G:(g + 1) * G] - ref).max()
        say(f"  seq {b}: T {T} L {L} head {g} max abs err {err:.2e}")
        assert err <= ATOL_BF16, (b, err)
        np.testing.assert_array_equal(kcs[b][g:g + 1, L:L + T], rk[:, L:L + T])
        np.testing.assert_array_equal(vcs[b][g:g + 1, L:L + T], rv[:, L:L + T])
        row += T


def test_accept_batched(api, trees):
    bank = api.Bank(trees)
    g = np.random.default_rng(17)
    B = 8
    topo = [int(t) for t in g.integers(0, len(trees), B)]
    rows = sum(bank.T[t] for t in topo)
    V = 50
    am = g.integers(0, V, rows).astype(np.int32)
    p1 = g.random(rows).astype(np.float32)
    toks = []
    row = 0
    for b, t in enumerate(topo):
        T = bank.T[t]
        u, r = g.random(T), g.integers(0, V, T)
        pa = [0.0, 1.0, 0.7, 0.7, 0.9, 0.5, 0.7, 0.3][b]   # none / all / mixed matches
        toks.append(synth.draft_tokens(trees[t], am[row:row + T], u, r, pa))
        row += T
    tok = np.concatenate(toks).astype(np.int32)
    cap_path = max(bank.D) + 3
    a = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    bon = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    best = torch.zeros(B, device="cuda")
    path = torch.full((B, cap_path), -7, dtype=torch.int32, device="cuda")
    api.accept_batched(bank, topo, dev_i32(tok), dev_i32(am), torch.from_numpy(p1).cuda(), a, path,
                       bon, best)
    torch.cuda.synchronize()
    a, bon, best, path = a.cpu().numpy(), bon.cpu().numpy(), best.cpu().numpy(), path.cpu().numpy()
    row = 0
    for b, t in enumerate(topo):
        T = bank.T[t]
        ra, rpath, rbonus, rbest = orc.accept(trees[t], tok[row:row + T], am[row:row + T])
        assert (a[b], bon[b]) == (ra, rbonus), b
        assert best[b] == p1[row + rbest]
        assert path[b, : ra + 1].tolist() == list(rpath)
        assert (path[b, ra + 1:] == -1).all()
        row += T
    assert a[1] == bank.D[topo[1]]          # all drafts match: the full depth


def test_kv_compact_batched(api, trees):
    g = np.random.default_rng(23)
    B, n_layers, Hkv, d = 5, 2, 4, 128
    lens = [0, 50, 7, 300, 129]
    topo = [4, 0, 2, 3, 1]
    cap = max(lens) + 128 + 4
    caches = [synth.f32_to_bf16_bits(g.standard_normal((2, n_layers, Hkv, cap, d)).astype(np.float32))
              for _ in range(B)]
    cap_path = 8
    paths = np.full((B, cap_path), -1, np.int32)
    acc = np.zeros(B, np.int32)
    for b, t in enumerate(topo):
        T = len(trees[t])
        am = g.integers(0, 3, T)
        tok = synth.draft_tokens(trees[t], am, g.random(T), g.integers(0, 3, T), 0.8)
        a, path, _, _ = orc.accept(trees[t], tok, am)
        acc[b] = a
        paths[b, : a + 1] = path
    kcs = [dev_bf16(c[0]) for c in caches]
    vcs = [dev_bf16(c[1]) for c in caches]
    api.kv_compact_batched(dev_i32(paths), dev_i32(acc), lens, kcs, vcs)
    torch.cuda.synchronize()
    for b in range(B):
        rk, rv = orc.kv_compact(caches[b][0], caches[b][1], lens[b], paths[b, : acc[b] + 1].tolist())
        np.testing.assert_array_equal(host_bits(kcs[b]), rk)
        np.testing.assert_array_equal(host_bits(vcs[b]), rv)


@pytest.mark.parametrize("topo,lens,V", [
    ([0, 1, 2, 0], [700, 64, 1500, 1023], 32000),
    # 64- and 128-node trees: 336 rows, three 128-row LM-head passes
    ([4, 3, 1, 4], [513, 2048, 90, 4000], 32000),
    # the benchmark's vocabulary: 2048 statistics partials per node
    ([4, 2], [1500, 777], 128256),
])
def test_batched_step_end_to_end(api, trees, topo, lens, V):
    """Attention, the LM head and statistics over the concatenated rows,
    acceptance and compaction of a batch, each sequence against the oracle's
    step on its own rows (GQA 32:8, hidden 4096)."""
    Hq, Hkv, hid = WL.n_heads, WL.n_kv_heads, WL.hidden
    say("batched step", topo, lens, V)
    B = len(topo)
    cap = max(lens) + 128 + 8
    scale = 1 / math.sqrt(D_HEAD)
    bank = api.Bank(trees)
    inp, q, kt, vt = batch_inputs(trees, topo, lens, Hq, Hkv, cap, 57)
    rows = q.shape[0]
    w = synth.lm_head_weight(57, V, hid)
    w64 = orc.bf16_to_f64(w)
    x = margin_hidden(57, rows, w, w64=w64)
    am_ref = (orc.bf16_to_f64(x) @ w64.T).argmax(axis=1)
    toks, row = [], 0
    for b, t in enumerate(topo):
        T = len(trees[t])
        u, r = synth.draft_randoms(57, T, V, step=b + 1)
        toks.append(synth.draft_tokens(trees[t], am_ref[row:row + T], u, r, 0.7))
        row += T
    tok = np.concatenate(toks).astype(np.int32)

    kcs = [dev_bf16(i.k_cache) for i in inp]
    vcs = [dev_bf16(i.v_cache) for i in inp]
    out = torch.empty((rows, Hq, D_HEAD), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(api.tree_attn_batched_workspace(B, max(bank.T), Hq, Hkv, D_HEAD, max(lens)),
                     dtype=torch.uint8, device="cuda")
    api.tree_attn_batched(bank, topo, lens, dev_bf16(q), dev_bf16(kt), dev_bf16(vt), kcs, vcs, scale,
                          THETA, out, ws)
    logits = torch.empty((rows, V), device="cuda")
    H, p1 = torch.empty(rows, device="cuda"), torch.empty(rows, device="cuda")
    am = torch.empty(rows, dtype=torch.int32, device="cuda")
    lws = torch.empty(api.verify_logits_stats_workspace(rows, hid, V), dtype=torch.uint8, device="cuda")
    api.verify_logits_stats(dev_bf16(x), dev_bf16(w), logits, 1.0, H, p1, am, lws)
    cap_path = max(bank.D) + 1
    a = torch.zeros(B, dtype=torch.int32, device="cuda")
    bon = torch.zeros(B, dtype=torch.int32, device="cuda")
    best = torch.zeros(B, device="cuda")
    path = torch.full((B, cap_path), -1, dtype=torch.int32, device="cuda")
    api.accept_batched(bank, topo, dev_i32(tok), am, p1, a, path, bon, best)
    api.kv_compact_batched(path, a, lens, kcs, vcs)
    torch.cuda.synchronize()

    out_h, z, Hh, p1h, amh = (out.float().cpu().numpy(), logits.cpu().numpy(), H.cpu().numpy(),
                              p1.cpu().numpy(), am.cpu().numpy())
    a_h, bon_h, best_h, path_h = a.cpu().numpy(), bon.cpu().numpy(), best.cpu().numpy(), path.cpu().numpy()
    row = 0
    for b, (t, L) in enumerate(zip(topo, lens)):
        T = len(trees[t])
        sl = slice(row, row + T)
        ref = orc.verify_step(trees[t], inp[b].q, inp[b].k_tree, inp[b].v_tree, inp[b].k_cache,
                              inp[b].v_cache, L, x[sl], w, tok[sl], scale, THETA)
        assert np.abs(out_h[sl] - ref["out"]).max() <= ATOL_BF16
        assert np.abs(z[sl] - ref["logits"]).max() <= ATOL_BF16
        np.testing.assert_array_equal(amh[sl], ref["argmax"])
        np.testing.assert_allclose(Hh[sl], ref["entropy"], rtol=RTOL_STATS, atol=1e-6)
        np.testing.assert_allclose(p1h[sl], ref["top1p"], rtol=RTOL_STATS, atol=1e-6)
        assert (a_h[b], bon_h[b]) == (ref["accept_len"], ref["bonus"])
        assert path_h[b, : a_h[b] + 1].tolist() == list(ref["path"])
        assert abs(best_h[b] - ref["s"]) <= RTOL_STATS * ref["s"] + 1e-6
        n = L + a_h[b] + 1
        np.testing.assert_array_equal(host_bits(kcs[b])[:, :n], ref["k_cache"][:, :n])
        np.testing.assert_array_equal(host_bits(vcs[b])[:, :n], ref["v_cache"][:, :n])
        row += T
