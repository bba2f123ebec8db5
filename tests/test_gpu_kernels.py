"""GPU parity: every kernel of the C ABI against the oracle on the same seeded
inputs.

Bars: bit-exact for masks, paths, argmax, accept results and compacted KV;
max abs error 2e-2 for bf16 attention outputs and fp32 logits; relative 1e-3
(plus 1e-6 absolute near 0) for entropy and top-1 probability.
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


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


def say(*a):
    print("[gpu-test]", *a, flush=True)


# ------------------------------------------------------------------ logits --

def random_bits(shape, seed, std=1.0):
    g = np.random.default_rng(seed)
    return synth.f32_to_bf16_bits((g.standard_normal(shape) * std).astype(np.float32))


@pytest.mark.parametrize("T,hid,V", [(1, 8, 1), (3, 64, 63), (16, 256, 4097), (17, 512, 1000),
                                     (27, 264, 301), (33, 128, 129), (64, 384, 777),
                                     (128, 256, 515), (129, 128, 260), (300, 64, 100)])
def test_verify_logits_shapes(api, T, hid, V):
    say("verify_logits", T, hid, V)
    X = random_bits((T, hid), 1)
    W = random_bits((V, hid), 2, 0.05)
    ref = orc.verify_logits(X, W)
    out = torch.full((T, V), float("nan"), device="cuda")
    api.verify_logits(dev_bf16(X), dev_bf16(W), out)
    got = out.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref).max()
    assert err <= ATOL_BF16, err
    assert err <= 1e-4 * max(1.0, np.abs(ref).max())


@pytest.fixture(scope="module")
def w7b():
    return synth.lm_head_weight(1, 32000, 4096)


@pytest.mark.parametrize("T", [27, 64, 100, 128])
def test_verify_logits_7b_full(api, w7b, T):
    say("verify_logits 7b", T)
    X = synth.hidden_rows(1, T, 4096)
    ref = orc.verify_logits(X, w7b)
    out = torch.empty((T, 32000), device="cuda")
    api.verify_logits(dev_bf16(X), dev_bf16(w7b), out)
    err = np.abs(out.cpu().numpy() - ref).max()
    assert err <= ATOL_BF16, err
    assert err <= 1e-4, err


def test_verify_logits_v128k_sampled(api):
    say("verify_logits 128k vocab, 544 rows, sampled columns")
    V, hid, T = 128256, 4096, 544
    W = synth.lm_head_weight(5, V, hid)
    X = synth.hidden_rows(5, T, hid)
    out = torch.empty((T, V), device="cuda")
    api.verify_logits(dev_bf16(X), dev_bf16(W), out)
    cols = np.unique(np.concatenate([np.random.default_rng(0).integers(0, V, 400),
                                     [0, 1, 2, 3, V - 4, V - 3, V - 2, V - 1]]))
    ref = orc.verify_logits_rows(X, W, cols)
    err = np.abs(out.cpu().numpy()[:, cols] - ref).max()
    assert err <= 1e-4, err


# ------------------------------------------------------------------- stats --

def run_stats(api, z32, inv_temp=1.0):
    T, V = z32.shape
    zt = torch.from_numpy(np.ascontiguousarray(z32)).cuda()
    H = torch.empty(T, device="cuda")
    p1 = torch.empty(T, device="cuda")
    am = torch.empty(T, dtype=torch.int32, device="cuda")
    api.logit_stats(zt, inv_temp, H, p1, am)
    return H.cpu().numpy(), p1.cpu().numpy(), am.cpu().numpy()


def check_stats(got, ref):
    H, p1, am = got
    rH, rp1, ram = ref
    np.testing.assert_array_equal(am, ram)
    assert np.all(np.abs(H - rH) <= RTOL_STATS * np.abs(rH) + 1e-6), (H, rH)
    assert np.all(np.abs(p1 - rp1) <= RTOL_STATS * np.abs(rp1) + 1e-6), (p1, rp1)


def test_logit_stats_closed_forms(api):
    say("logit_stats closed forms")
    V = 32000
    rows = [np.zeros(V), np.full(V, -3.5)]
    z = np.full(V, -np.inf); z[417] = 2.0; rows.append(z)
    z = np.full(V, -np.inf); z[[400, 17, 250]] = 1.5; rows.append(z)
    for delta in (0.0, 0.5, 3.0, 11.2, 18.0):
        z = np.zeros(V); z[12345] = delta; rows.append(z)
    z = np.random.default_rng(0).standard_normal(V) + 1000.0; rows.append(z)
    z32 = np.stack(rows).astype(np.float32)
    got = run_stats(api, z32)
    check_stats(got, orc.logit_stats(z32))
    H, p1, am = got
    assert abs(H[0] - math.log(V)) <= 1e-3 * math.log(V) and am[0] == 0 and am[1] == 0
    assert am[2] == 417 and H[2] == 0.0 and p1[2] == 1.0
    assert am[3] == 17 and abs(H[3] - math.log(3)) <= 1e-3 * math.log(3)


@pytest.mark.parametrize("V", [1, 2, 63, 64, 65, 4097, 128256])
def test_logit_stats_vocab_sizes(api, V):
    say("logit_stats V", V)
    g = np.random.default_rng(V)
    z32 = (g.standard_normal((5, V)) * 3).astype(np.float32)
    z32[1] = 0.0
    for it in (1.0, 1 / 0.7):
        check_stats(run_stats(api, z32, it), orc.logit_stats(z32, it))


def test_logit_stats_on_margin_logits(api, w7b):
    say("logit_stats on 7b-shaped logits")
    X = margin_hidden(1, 27, w7b)
    z32 = orc.verify_logits(X, w7b).astype(np.float32)
    check_stats(run_stats(api, z32), orc.logit_stats(z32))


def run_fused(api, X, W, inv_temp=1.0):
    T, hid = X.shape
    V = W.shape[0]
    logits = torch.full((T, V), float("nan"), device="cuda")
    H = torch.empty(T, device="cuda")
    p1 = torch.empty(T, device="cuda")
    am = torch.empty(T, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(16, api.verify_logits_stats_workspace(T, hid, V)), dtype=torch.uint8,
                     device="cuda")
    api.verify_logits_stats(dev_bf16(X), dev_bf16(W), logits, inv_temp, H, p1, am, ws)
    return logits.cpu().numpy(), (H.cpu().numpy(), p1.cpu().numpy(), am.cpu().numpy())


@pytest.mark.parametrize("T,hid,V", [(1, 512, 1), (3, 512, 63), (16, 1024, 4097), (27, 4096, 32000),
                                     (33, 512, 1000), (64, 512, 777), (64, 4096, 32000),
                                     (100, 4096, 32000), (128, 4096, 32000),
                                     (129, 512, 260), (7, 264, 301), (300, 2048, 100)])
def test_verify_logits_stats_fused(api, T, hid, V):
    say("verify_logits_stats", T, hid, V)
    X = random_bits((T, hid), 11)
    W = random_bits((V, hid), 12, 0.05)
    ref = orc.verify_logits(X, W)
    for it in (1.0, 1 / 0.7):
        z, st = run_fused(api, X, W, it)
        assert np.abs(z - ref).max() <= 1e-4 * max(1.0, np.abs(ref).max())
        # statistics on the kernel's own fp32 logits must match the oracle's
        # statistics of its fp32-rounded logits: identical argmax when the
        # top-2 gap exceeds the fp32 accumulation error, stats within the bar
        H, p1, am = st
        rH, rp1, ram = orc.logit_stats(ref.astype(np.float32), it)
        gap = np.sort(ref, axis=1)
        safe = (gap[:, -1] - gap[:, -2]) > 1e-4 if V > 1 else np.ones(T, bool)
        np.testing.assert_array_equal(am[safe], ram[safe])
        assert np.all(np.abs(H - rH) <= RTOL_STATS * np.abs(rH) + 1e-6), (H, rH)
        assert np.all(np.abs(p1 - rp1) <= RTOL_STATS * np.abs(rp1) + 1e-6), (p1, rp1)


@pytest.mark.parametrize("T,V", [(1, 32000), (27, 32000), (64, 4097), (200, 1000)])
def test_verify_logits_partials_then_finalize_equals_fused(api, T, V):
    say("verify_logits_partials + stats_finalize", T, V)
    hid = 1024
    X = dev_bf16(random_bits((T, hid), 21))
    W = dev_bf16(random_bits((V, hid), 22, 0.05))
    ws = torch.empty(api.stats_partials_bytes(T, hid, V), dtype=torch.uint8, device="cuda")
    out = []
    for split in (False, True):
        z = torch.full((T, V), float("nan"), device="cuda")
        H, p1 = torch.empty(T, device="cuda"), torch.empty(T, device="cuda")
        am = torch.empty(T, dtype=torch.int32, device="cuda")
        if split:
            api.verify_logits_partials(X, W, z, 1 / 0.7, ws)
            api.stats_finalize(ws, T, V, 1 / 0.7, H, p1, am)
        else:
            api.verify_logits_stats(X, W, z, 1 / 0.7, H, p1, am, ws)
        out.append([t.cpu().numpy() for t in (z, H, p1, am)])
    for a, b in zip(*out):
        np.testing.assert_array_equal(a, b)


def test_verify_logits_stats_fused_margin_7b(api, w7b):
    say("verify_logits_stats 7b margin rows")
    X = margin_hidden(1, 27, w7b)
    z, (H, p1, am) = run_fused(api, X, w7b)
    rH, rp1, ram = orc.logit_stats(orc.verify_logits(X, w7b).astype(np.float32))
    np.testing.assert_array_equal(am, ram)
    assert np.all(np.abs(H - rH) <= RTOL_STATS * np.abs(rH) + 1e-6)
    assert np.all(np.abs(p1 - rp1) <= RTOL_STATS * np.abs(rp1) + 1e-6)


def test_verify_logits_13b_hidden_5120(api):
    """The 13B shape (hidden 5120, fully unrolled 40-stage K loop): logits and
    fused statistics of a 128-node tree against the oracle."""
    say("verify_logits 13b shapes")
    V, hid, T = 32000, 5120, 128
    w = synth.lm_head_weight(4, V, hid)
    X = margin_hidden(4, T, w)
    ref = orc.verify_logits(X, w)
    z, (H, p1, am) = run_fused(api, X, w)
    assert np.abs(z - ref).max() <= 1e-4 * max(1.0, np.abs(ref).max())
    rH, rp1, ram = orc.logit_stats(ref.astype(np.float32))
    np.testing.assert_array_equal(am, ram)
    assert np.all(np.abs(H - rH) <= RTOL_STATS * np.abs(rH) + 1e-6)
    assert np.all(np.abs(p1 - rp1) <= RTOL_STATS * np.abs(rp1) + 1e-6)
    for T2 in (1, 16, 27, 64):   # the other node tiles at this hidden size
        z2, st2 = run_fused(api, X[:T2], w)
        np.testing.assert_array_equal(st2[2], ram[:T2])
        assert np.abs(z2 - ref[:T2]).max() <= 1e-4 * max(1.0, np.abs(ref).max())


# ------------------------------------------------------------------ accept --

def run_accept(api, bank, topo, tok, am, p1=None):
    T, D = bank.T[topo], bank.D[topo]
    a = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    path = torch.full((D + 1,), -7, dtype=torch.int32, device="cuda")
    bonus = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    bp = torch.full((1,), -1.0, device="cuda")
    p1t = torch.from_numpy(np.asarray(p1, np.float32)).cuda() if p1 is not None else None
    api.accept(bank, topo, dev_i32(tok), dev_i32(am), p1t, a, path, bonus, bp if p1 is not None else None)
    return int(a.item()), path.cpu().numpy(), int(bonus.item()), float(bp.item())


def test_accept_random_trees(api):
    say("accept random trees")
    g = np.random.default_rng(3)
    trees = [[-1], [-1, 0], synth.chain_tree(32), synth.star_tree(256)]
    trees += [synth.uniform_attach_tree(900 + k, n, c) for k, (n, c) in
              enumerate([(7, 3), (27, 4), (64, 5), (128, 6), (256, 8)])]
    deep = synth.chain_tree(32) + [int(x) for x in g.integers(0, 31, 60)]   # depth 31, 92 nodes
    trees.append(deep)
    trees += synth.workload_trees(synth.WORKLOADS["bank5_L2048_7b"])
    bank = api.Bank(trees)
    for topo, parent in enumerate(trees):
        T = len(parent)
        for trial in range(40):
            am = g.integers(0, 5 if trial % 2 else 32000, T).astype(np.int32)
            p_acc = [0.0, 0.5, 0.9, 1.0][trial % 4]
            u, r = g.random(T), g.integers(0, 32000, T)
            tok = synth.draft_tokens(parent, am, u, r, p_acc)
            p1 = g.random(T).astype(np.float32)
            a, path, bonus, bp = run_accept(api, bank, topo, tok, am, p1)
            ra, rpath, rbonus, rbest = orc.accept(parent, tok, am)
            assert a == ra and bonus == rbonus
            D = bank.D[topo]
            np.testing.assert_array_equal(path, np.array(rpath + [-1] * (D + 1 - len(rpath))))
            assert bp == p1[rbest]
            if p_acc == 1.0:
                assert a == D


# -------------------------------------------------------------- compaction --

@pytest.mark.parametrize("n_layers,Hkv,cap,L,d", [(1, 32, 400, 256, 128), (3, 8, 64, 20, 128),
                                                  (32, 4, 300, 100, 128), (2, 5, 50, 0, 64)])
def test_kv_compact_random(api, n_layers, Hkv, cap, L, d):
    say("kv_compact", n_layers, Hkv, cap, L, d)
    g = np.random.default_rng(n_layers * 7 + L)
    kc = g.integers(0, 0x7F00, (n_layers, Hkv, cap, d)).astype(np.uint16)
    vc = g.integers(0, 0x7F00, (n_layers, Hkv, cap, d)).astype(np.uint16)
    T = min(cap - L, 30)
    parent = synth.uniform_attach_tree(77 + L, T, min(6, T - 1)) if T > 1 else [-1]
    kd, vd = dev_bf16(kc), dev_bf16(vc)
    for best in range(T):
        path = orc.ancestors_or_self(parent, best)
        a = len(path) - 1
        pt = dev_i32(path + [-1] * (8 - len(path)) if len(path) < 8 else path)
        at = dev_i32([a])
        kd.copy_(dev_bf16(kc)); vd.copy_(dev_bf16(vc))
        api.kv_compact(pt, at, L, kd, vd)
        rk, rv = orc.kv_compact(kc, vc, L, path)
        np.testing.assert_array_equal(host_bits(kd), rk)
        np.testing.assert_array_equal(host_bits(vd), rv)


# --------------------------------------------------------------- attention --

def run_attn(api, bank, topo, inp, L, scale, theta):
    q, kt, vt = dev_bf16(inp.q), dev_bf16(inp.k_tree), dev_bf16(inp.v_tree)
    kc, vc = dev_bf16(inp.k_cache), dev_bf16(inp.v_cache)
    T, Hq, d = inp.q.shape
    Hkv = inp.k_tree.shape[1]
    out = torch.full((T, Hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(api.tree_attn_workspace(T, Hq, Hkv, d, L), dtype=torch.uint8, device="cuda")
    api.tree_attn(bank, topo, q, kt, vt, kc, vc, L, scale, theta, out, ws)
    return (out.float().cpu().numpy(), host_bits(kc), host_bits(vc))


def check_attn(api, parent, T, L, Hq, Hkv, theta, wl=50, cap_extra=5, layer=0):
    d = 128
    cap = L + T + cap_extra
    inp = synth.attn_inputs(wl, T, Hq, Hkv, d, L, cap, layer=layer)
    bank = api.Bank([parent])
    scale = 1 / math.sqrt(d)
    out, kc, vc = run_attn(api, bank, 0, inp, L, scale, theta)
    ref, rk, rv = orc.tree_attention(inp.q, inp.k_tree, inp.v_tree, inp.k_cache, inp.v_cache,
                                     L, parent, scale, theta)
    err = np.abs(out - ref).max()
    assert err <= ATOL_BF16, err
    # the append is bit-exact (fp64 rotation, one rounding), prefix untouched
    np.testing.assert_array_equal(kc[:, : L + T], rk[:, : L + T])
    np.testing.assert_array_equal(vc[:, : L + T], rv[:, : L + T])
    return err


@pytest.mark.parametrize("kind,T,L,Hq,Hkv,theta", [
    ("single", 1, 0, 2, 2, 0.0), ("single", 1, 1, 4, 4, 10000.0), ("chain", 5, 31, 2, 2, 0.0),
    ("chain", 32, 32, 2, 2, 10000.0), ("star", 9, 33, 4, 1, 10000.0), ("random", 27, 256, 8, 8, 10000.0),
    ("random", 64, 100, 8, 2, 10000.0), ("random", 128, 0, 4, 4, 0.0), ("random", 200, 70, 4, 1, 10000.0),
    ("random", 256, 513, 2, 2, 10000.0), ("star", 100, 1000, 4, 4, 10000.0), ("chain", 3, 4000, 8, 8, 10000.0),
    # four-tile kernel with idle waves: 2 tiles (40 nodes; 20 nodes x 2 heads
    # per KV head) and 3 tiles (80 nodes)
    ("random", 40, 300, 4, 4, 10000.0), ("random", 20, 777, 4, 2, 10000.0),
    ("random", 80, 1500, 8, 8, 10000.0),
    # the deepest tree in the four-tile kernel (32 levels of angles in LDS)
    ("chain", 32, 50, 8, 2, 10000.0)])
def test_tree_attn_small(api, kind, T, L, Hq, Hkv, theta):
    say("tree_attn", kind, T, L, Hq, Hkv, theta)
    if kind == "single":
        parent = [-1]
    elif kind == "chain":
        parent = synth.chain_tree(T)
    elif kind == "star":
        parent = synth.star_tree(T)
    else:
        parent = synth.uniform_attach_tree(600 + T, T, min(6, T - 1))
    check_attn(api, parent, T, L, Hq, Hkv, theta)


def test_tree_attn_mask_leakage(api):
    say("tree_attn mask leakage")
    parent = synth.uniform_attach_tree(31, 27, 4)
    T, L, H, d = 27, 70, 4, 128
    inp = synth.attn_inputs(51, T, H, H, d, L, L + T)
    bank = api.Bank([parent])
    base, _, _ = run_attn(api, bank, 0, inp, L, 0.1, 10000.0)
    anc = [set(orc.ancestors_or_self(parent, i)) for i in range(T)]
    g = np.random.default_rng(8)
    for i in (0, 5, 26):
        kt, vt = inp.k_tree.copy(), inp.v_tree.copy()
        for j in range(T):
            if j not in anc[i]:
                kt[j] = synth.f32_to_bf16_bits(g.standard_normal(kt[j].shape).astype(np.float32))
                vt[j] = synth.f32_to_bf16_bits(g.standard_normal(vt[j].shape).astype(np.float32))
        pert = synth.AttnInputs(inp.q, kt, vt, inp.k_cache, inp.v_cache)
        out, _, _ = run_attn(api, bank, 0, pert, L, 0.1, 10000.0)
        np.testing.assert_array_equal(out[i], base[i])
    # the other half: a node's own path does reach it.  Perturbing one node's
    # key and value changes exactly the rows of the nodes it is an ancestor
    # of (itself included), and leaves every other row as it was.
    for j in (0, 3, 11, 26):
        kt, vt = inp.k_tree.copy(), inp.v_tree.copy()
        kt[j] = synth.f32_to_bf16_bits(g.standard_normal(kt[j].shape).astype(np.float32))
        vt[j] = synth.f32_to_bf16_bits(g.standard_normal(vt[j].shape).astype(np.float32))
        pert = synth.AttnInputs(inp.q, kt, vt, inp.k_cache, inp.v_cache)
        out, _, _ = run_attn(api, bank, 0, pert, L, 0.1, 10000.0)
        for i in range(T):
            if j in anc[i]:
                assert not np.array_equal(out[i], base[i]), (j, i)
            else:
                np.testing.assert_array_equal(out[i], base[i])


@pytest.mark.parametrize("name,T,L,Hq,Hkv", [("7b_tree27", 27, 256, 32, 32),
                                             ("7b_bank_T128", 128, 2048, 32, 32),
                                             ("7b_bank_T1", 1, 2048, 32, 32),
                                             ("13b_tree128", 128, 8192, 40, 40),
                                             ("gqa_T128_L16384", 128, 16384, 32, 8)])
def test_tree_attn_workload_shapes(api, name, T, L, Hq, Hkv):
    say("tree_attn workload", name)
    if T == 1:
        parent = [-1]
    elif name.startswith("13b"):
        parent = synth.workload_trees(synth.WORKLOADS["tree128_L8192_13b"])[0]
    else:
        parent = synth.uniform_attach_tree(700 + T, T, 6 if T == 128 else 4)
    err = check_attn(api, parent, T, L, Hq, Hkv, 10000.0, wl=60)
    say("  max abs err", err)
