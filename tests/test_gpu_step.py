"""GPU: the step driver (entmtp_step_*) in a closed decode loop.

The driver chains the kernels that the other GPU tests check one at a time.
Here a loop runs as a decoder would: the ladder picks each tree from the
previous step's s, and the prefix grows by the accepted tokens.  Every step is
replayed from the GPU's state before it, (1) on the oracle (open-loop replay
of the GPU's tree sequence, so a near-threshold s cannot split the two runs)
and (2) through the individual entry points, which must agree bit for bit --
except, for trees of up to 32 nodes, the logits, entropy and top-1
probability: the step's LM head there takes two vocabulary slices per
workgroup (one partial for both, and its own K order), so it sums the same
fp32 terms in another order (agreement to 1e-5 relative there; the argmax
still bit for bit).
"""
# step vs. entry points: the same fp32 terms summed in another order
RTOL_ORDER, ATOL_ORDER = 1e-5, 1e-6
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import entmtp_oracle as orc  # noqa: E402
from paper_2606_27550_amd import synth  # noqa: E402
from tests.helpers import dev_bf16, dev_i32, host_bits, margin_hidden  # noqa: E402

pytestmark = pytest.mark.gpu

WL = 77
ATOL_BF16 = 2e-2
RTOL_STATS = 1e-3
W_STD = 0.05


@pytest.fixture(scope="module")
def api():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_27550_amd import api as _api
    return _api


def say(*a):
    print("[gpu-test]", *a, flush=True)


def bank_trees():
    return [[-1], synth.uniform_attach_tree(WL, 8, 3), synth.uniform_attach_tree(WL + 1, 26, 4),
            synth.uniform_attach_tree(WL + 2, 64, 5)]


def step_inputs(t, n_layers, Tmax, Hq, Hkv, d, w_bits, w64, delta, spike):
    layers = [synth.attn_inputs(WL, Tmax, Hq, Hkv, d, 0, Tmax, step=t + 1, layer=l)
              for l in range(n_layers)]
    x = margin_hidden(WL, Tmax, w_bits, step=t + 1, w64=w64, spikes=(delta, spike), w_std=W_STD)
    am = (orc.bf16_to_f64(x) @ w64.T).argmax(axis=1)
    u, r = synth.draft_randoms(WL, Tmax, w_bits.shape[0], step=t + 1)
    return layers, x, am, u, r


def stack(layers, name):
    return np.ascontiguousarray(np.stack([getattr(a, name) for a in layers]))


def run_loop(api, n_layers, n_steps, Hq=8, Hkv=2, hid=512, V=1000, L0=40, start_rung=0,
             keep_logits=True, flush_each=True, arm=None):
    """Closed loop through the step driver, each step checked (1) on the
    oracle from the cache state before it and (2) bit for bit against the same
    step through the individual entry points (whose cache is compacted every
    step).  flush_each=False leaves every compaction to the next launch and
    compares the driver's cache once, after the final flush.  arm="ladder"
    enqueues each next step's LM head while the step before is pending
    (entmtp_step_arm), sized for the largest tree the ladder can reach;
    arm="low" arms one row only, so every larger tree takes the fallback."""
    d, theta = 128, 10000.0
    scale = 1 / math.sqrt(d)
    trees = bank_trees()
    bank = api.Bank(trees)
    Tmax, Dmax = max(bank.T), max(bank.D)
    cap = L0 + n_steps * (Dmax + 1) + Tmax + 8
    w_bits = synth.lm_head_weight(WL, V, hid, std=W_STD)
    w64 = orc.bf16_to_f64(w_bits)
    W = dev_bf16(w_bits)
    base = [synth.attn_inputs(WL, 1, Hq, Hkv, d, L0, cap, layer=l) for l in range(n_layers)]
    kc = dev_bf16(stack(base, "k_cache"))          # [layers][Hkv][cap][d]
    vc = dev_bf16(stack(base, "v_cache"))
    kc2, vc2 = kc.clone(), vc.clone()              # the entry-point replay's own cache
    stride = Hkv * cap * d
    st = api.Step(bank, kc, vc, W, n_layers=n_layers, Hq=Hq, Hkv=Hkv, d=d, cap=cap,
                  tree_rows=Tmax, scale=scale, rope_theta=theta, cache_layer_stride=stride,
                  keep_logits=keep_logits)
    deltas, spikes = synth.regime_spikes(WL, n_steps, Tmax, V, hid)

    # entry-point replay buffers
    out2 = torch.empty((n_layers, Tmax, Hq, d), dtype=torch.bfloat16, device="cuda")
    lg2 = torch.empty((Tmax, V), device="cuda")
    H2, p12 = torch.empty(Tmax, device="cuda"), torch.empty(Tmax, device="cuda")
    am2 = torch.empty(Tmax, dtype=torch.int32, device="cuda")
    a2, b2 = torch.zeros(1, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.int32, device="cuda")
    s2 = torch.zeros(1, device="cuda")
    path2 = torch.full((Dmax + 1,), -1, dtype=torch.int32, device="cuda")
    aws = torch.empty(api.tree_attn_workspace(Tmax, Hq, Hkv, d, cap), dtype=torch.uint8, device="cuda")
    lws = torch.empty(api.verify_logits_stats_workspace(Tmax, hid, V), dtype=torch.uint8, device="cuda")

    def inputs(t):
        # host inputs, then the step's device buffers (enqueued on the stream
        # before the step is armed: work enqueued after arming queues behind
        # the armed LM head)
        got = step_inputs(t, n_layers, Tmax, Hq, Hkv, d, w_bits, w64, float(deltas[t]), spikes[t])
        q, kt, vt = (dev_bf16(stack(got[0], n)) for n in ("q", "k_tree", "v_tree"))
        out = torch.full((n_layers, Tmax, Hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        return got, (dev_bf16(got[1]), q, kt, vt, out)

    L, rung, topo_trace, switches = L0, start_rung, [], 0
    ahead = None   # the next step's inputs, when its LM head is armed
    for t in range(n_steps):
        T, parent = bank.T[rung], trees[rung]
        (layers, x, am, u, r), (X, q, kt, vt, out) = ahead if ahead is not None else inputs(t)
        ahead = None
        tok = synth.draft_tokens(parent, am, u, r, 0.7)
        tok_d = dev_i32(tok)   # read by the acceptance, which the launch enqueues after it
        kc_before, vc_before = host_bits(kc2), host_bits(vc2)
        say(f"step {t}: layers {n_layers} topo {rung} T {T} L {L}")

        st.launch(rung, L, q, kt, vt, out, X, tok_d)
        if arm and t + 1 < n_steps:
            ahead = inputs(t + 1)
            bound = 1 if arm == "low" else bank.T[min(rung + 1, len(trees) - 1)]
            st.arm(ahead[1][0], bound)
        a, bonus, s = st.wait(timeout_s=60.0)
        if flush_each:
            st.flush()
        torch.cuda.synchronize()

        # (2) the same step through the individual entry points, bit for bit
        for l in range(n_layers):
            api.tree_attn(bank, rung, q[l, :T], kt[l, :T], vt[l, :T], kc2[l], vc2[l], L, scale,
                          theta, out2[l, :T], aws)
        api.verify_logits_stats(X[:T], W, lg2[:T], 1.0, H2[:T], p12[:T], am2[:T], lws)
        api.accept(bank, rung, tok_d, am2, p12, a2, path2, b2, s2)
        api.kv_compact(path2, a2, L, kc2, vc2)
        torch.cuda.synchronize()
        # entmtp_accept writes its tree's D + 1 path entries; the step writes
        # its whole path buffer (-1 past the accept length, whatever the depth
        # of the tree before)
        Dt = bank.D[rung]
        pairs = [(out[:, :T], out2[:, :T]), (st.argmax[:T], am2[:T]), (st.path[:Dt + 1], path2[:Dt + 1])]
        assert (st.path[Dt + 1:] == -1).all()
        for mine, theirs in ((st.entropy[:T], H2[:T]), (st.top1p[:T], p12[:T])):
            torch.testing.assert_close(mine, theirs, rtol=RTOL_ORDER, atol=ATOL_ORDER)
        if flush_each:
            pairs += [(kc, kc2), (vc, vc2)]
        if keep_logits:
            if T <= 32:
                torch.testing.assert_close(st.logits[:T], lg2[:T], rtol=RTOL_ORDER, atol=1e-5)
            else:
                pairs.append((st.logits[:T], lg2[:T]))
        for mine, theirs in pairs:
            assert torch.equal(mine.view(torch.int16) if mine.dtype == torch.bfloat16 else mine,
                               theirs.view(torch.int16) if theirs.dtype == torch.bfloat16 else theirs)
        assert (a, bonus) == (int(a2.item()), int(b2.item()))
        assert abs(np.float32(s) - np.float32(s2.item())) <= RTOL_ORDER * abs(s) + ATOL_ORDER
        assert a == int(st.accept_len.item()) and bonus == int(st.bonus.item())

        # (1) the oracle from the GPU's state before the step
        ref = orc.verify_step(parent, layers[0].q[:T], layers[0].k_tree[:T], layers[0].v_tree[:T],
                              kc_before[0], vc_before[0], L, x[:T], w_bits, tok, scale, theta)
        assert np.abs(out[0, :T].float().cpu().numpy() - ref["out"]).max() <= ATOL_BF16
        if keep_logits:
            assert np.abs(st.logits[:T].cpu().numpy() - ref["logits"]).max() <= ATOL_BF16
        np.testing.assert_array_equal(st.argmax[:T].cpu().numpy(), ref["argmax"])
        np.testing.assert_allclose(st.entropy[:T].cpu().numpy(), ref["entropy"], rtol=RTOL_STATS,
                                   atol=1e-6)
        np.testing.assert_allclose(st.top1p[:T].cpu().numpy(), ref["top1p"], rtol=RTOL_STATS,
                                   atol=1e-6)
        assert (a, bonus) == (ref["accept_len"], ref["bonus"])
        assert st.path.cpu().numpy()[: a + 1].tolist() == list(ref["path"])
        assert abs(s - ref["s"]) <= RTOL_STATS * ref["s"] + 1e-6
        kc_now, vc_now = host_bits(kc2), host_bits(vc2)
        n = L + a + 1
        for l in range(n_layers):
            if l == 0:
                rk, rv = ref["k_cache"], ref["v_cache"]
            else:   # other layers: their own attention append, then the same path
                _, rk, rv = orc.tree_attention(layers[l].q[:T], layers[l].k_tree[:T],
                                               layers[l].v_tree[:T], kc_before[l], vc_before[l], L,
                                               parent, scale, theta)
                rk, rv = orc.kv_compact(rk, rv, L, ref["path"])
            np.testing.assert_array_equal(kc_now[l][:, :n], rk[:, :n])
            np.testing.assert_array_equal(vc_now[l][:, :n], rv[:, :n])

        topo_trace.append(rung)
        L += a + 1
        nxt = api.ladder_next(rung, len(trees), s, 0.8, 0.6)
        switches += nxt != rung
        rung = nxt
    if not flush_each:
        st.flush()
        torch.cuda.synchronize()
        assert torch.equal(kc.view(torch.int16), kc2.view(torch.int16))
        assert torch.equal(vc.view(torch.int16), vc2.view(torch.int16))
    st.close()
    return topo_trace, switches


def test_step_closed_loop_one_layer(api):
    trace, switches = run_loop(api, n_layers=1, n_steps=14)
    say("topology trace", trace)
    assert switches >= 2 and len(set(trace)) >= 3   # the loop really moved along the ladder


def test_step_closed_loop_compaction_left_to_next_launch(api):
    # the pipelined form: no flush between steps, one at the end
    trace, switches = run_loop(api, n_layers=2, n_steps=10, flush_each=False, keep_logits=False)
    assert switches >= 1


def test_step_closed_loop_three_layers(api):
    # starts on the largest tree; no logits kept (statistics from the accumulators)
    trace, _ = run_loop(api, n_layers=3, n_steps=4, start_rung=3, keep_logits=False)
    assert trace[0] == 3


@pytest.mark.parametrize("arm,flush_each", [("ladder", True), ("ladder", False), ("low", False)])
def test_step_closed_loop_armed(api, arm, flush_each):
    # the next step's LM head enqueued behind the gate while a step is pending:
    # sized by the ladder's reach, or too small (fresh LM head as fallback)
    # (no logits kept: the armed LM head of the next step reuses the buffer,
    # and may start once the gate's time limit ends its wait)
    trace, switches = run_loop(api, n_layers=2, n_steps=12, flush_each=flush_each,
                               keep_logits=False, arm=arm)
    say("armed", arm, "topology trace", trace)
    assert switches >= 2 and len(set(trace)) >= 3


def test_step_arm_errors(api):
    bank = api.Bank(bank_trees())
    Hq, Hkv, d, hid, V, cap = 4, 4, 128, 512, 300, 80
    kc = torch.zeros((Hkv, cap, d), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    W = torch.zeros((V, hid), dtype=torch.bfloat16, device="cuda")
    st = api.Step(bank, kc, vc, W, Hq=Hq, Hkv=Hkv, cap=cap, tree_rows=64, scale=0.1, rope_theta=0.0)
    X = torch.zeros((64, hid), dtype=torch.bfloat16, device="cuda")
    for bound in (0, 65):                           # outside [1, the largest tree]
        with pytest.raises(api.EntmtpError) as e:
            st.arm(X, bound)
        assert e.value.code == api.ERANGE
    st.arm(X, 8)
    with pytest.raises(api.EntmtpError) as e:       # armed twice
        st.arm(X, 8)
    assert e.value.code == api.EINVAL
    q = torch.zeros((64, Hq, d), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((64, Hkv, d), dtype=torch.bfloat16, device="cuda")
    tok = torch.zeros(64, dtype=torch.int32, device="cuda")
    ev = torch.cuda.Event(enable_timing=True)
    ev.record()                                     # (torch creates the event at its first record)
    with pytest.raises(api.EntmtpError) as e:       # events belong to the arming call
        st.launch(1, 0, q, kv, kv, q.clone(), X, tok, ev_lm_begin=ev, ev_lm_end=ev)
    assert e.value.code == api.EINVAL
    st.launch(1, 0, q, kv, kv, q.clone(), X, tok)   # an 8-node tree: the armed LM head
    a, bonus, s = st.wait(timeout_s=60.0)
    assert bonus == 0 and abs(s - 1.0 / V) <= 1e-6 and a == bank.D[1]
    st.arm(X, 8)                                    # armed, then left to the flush
    st.flush()
    torch.cuda.synchronize()
    st.close()


def test_step_errors(api):
    bank = api.Bank(bank_trees())
    Hq, Hkv, d, hid, V, cap = 4, 4, 128, 512, 300, 80
    kc = torch.zeros((Hkv, cap, d), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    W = torch.zeros((V, hid), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(api.EntmtpError) as e:       # tree_rows below the largest tree
        api.Step(bank, kc, vc, W, Hq=Hq, Hkv=Hkv, cap=cap, tree_rows=63, scale=0.1, rope_theta=0.0)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.EntmtpError) as e:       # hidden size without the fused path
        api.Step(bank, kc, vc, torch.zeros((V, 264), dtype=torch.bfloat16, device="cuda"), Hq=Hq,
                 Hkv=Hkv, cap=cap, tree_rows=64, scale=0.1, rope_theta=0.0)
    assert e.value.code == api.EINVAL
    st = api.Step(bank, kc, vc, W, Hq=Hq, Hkv=Hkv, cap=cap, tree_rows=64, scale=0.1, rope_theta=0.0)
    q = torch.zeros((64, Hq, d), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((64, Hkv, d), dtype=torch.bfloat16, device="cuda")
    X = torch.zeros((64, hid), dtype=torch.bfloat16, device="cuda")
    tok = torch.zeros(64, dtype=torch.int32, device="cuda")
    with pytest.raises(api.EntmtpError) as e:       # prefix + T beyond the cache
        st.launch(3, cap - 63, q, kv, kv, q.clone(), X, tok)
    assert e.value.code == api.ERANGE
    with pytest.raises(api.EntmtpError) as e:       # nothing in flight to wait for
        st.wait(timeout_s=0.1)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.EntmtpError) as e:
        st.launch(len(bank), 0, q, kv, kv, q.clone(), X, tok)
    assert e.value.code == api.EINVAL
    st.launch(3, cap - 64, q, kv, kv, q.clone(), X, tok)   # the largest valid prefix
    with pytest.raises(api.EntmtpError) as e:       # its result not read yet
        st.launch(3, 0, q, kv, kv, q.clone(), X, tok)
    assert e.value.code == api.EINVAL
    with pytest.raises(api.EntmtpError) as e:
        st.flush()
    assert e.value.code == api.EINVAL
    a, bonus, s = st.wait(timeout_s=60.0)
    st.flush()
    torch.cuda.synchronize()
    # all-zero logits: uniform distribution, argmax 0; zero drafts match it
    assert bonus == 0 and abs(s - 1.0 / V) <= 1e-6 and a == bank.D[3]
    st.close()


@pytest.mark.parametrize("n_layers,with128", [(1, False), (2, True)])
def test_device_scheduled_loop_matches_host_scheduled(api, n_layers, with128):
    """The same closed loop twice: the host reads each step's result and runs
    the ladder (entmtp_step_launch / _wait / ladder_next), and the GPU does it
    (entmtp_step_device_start / _launch_device, no host reads until the end).
    Trees, prefix lengths, accept lengths, s, outputs and caches agree bit for
    bit."""
    Hq, Hkv, d, hid, V, L0, n_steps = 8, 2, 128, 512, 1000, 40, 14
    theta, scale = 10000.0, 1 / math.sqrt(128)
    trees = bank_trees() + ([synth.uniform_attach_tree(WL + 3, 128, 6)] if with128 else [])
    bank = api.Bank(trees)
    K, Tmax, Dmax = len(trees), max(bank.T), max(bank.D)
    cap = L0 + n_steps * (Dmax + 1) + Tmax + 8
    rung0 = K - 1 if with128 else 0   # start on the largest tree (two LM-head passes)
    w_bits = synth.lm_head_weight(WL, V, hid, std=W_STD)
    w64 = orc.bf16_to_f64(w_bits)
    W = dev_bf16(w_bits)
    base = [synth.attn_inputs(WL, 1, Hq, Hkv, d, L0, cap, layer=l) for l in range(n_layers)]
    kc_h = dev_bf16(stack(base, "k_cache"))
    vc_h = dev_bf16(stack(base, "v_cache"))
    kc_d, vc_d = kc_h.clone(), vc_h.clone()
    stride = Hkv * cap * d
    kw = dict(n_layers=n_layers, Hq=Hq, Hkv=Hkv, d=d, cap=cap, tree_rows=Tmax, scale=scale,
              rope_theta=theta, cache_layer_stride=stride)
    st_h = api.Step(bank, kc_h, vc_h, W, keep_logits=False, **kw)
    st_d = api.Step(bank, kc_d, vc_d, W, keep_logits=False, tau_on=0.8, tau_off=0.6, **kw)
    deltas, spikes = synth.regime_spikes(WL, n_steps, Tmax, V, hid)
    steps, host_steps = [], []
    for t in range(n_steps):
        layers, x, am, u, r = step_inputs(t, n_layers, Tmax, Hq, Hkv, d, w_bits, w64,
                                          float(deltas[t]), spikes[t])
        drafts = np.zeros((K, Tmax), np.int32)
        for k in range(K):
            drafts[k, : bank.T[k]] = synth.draft_tokens(trees[k], am, u, r, 0.7)
        host_steps.append((layers, x, drafts))
        steps.append({"q": dev_bf16(stack(layers, "q")), "kt": dev_bf16(stack(layers, "k_tree")),
                      "vt": dev_bf16(stack(layers, "v_tree")), "x": dev_bf16(x),
                      "drafts": dev_i32(drafts)})
    out_h = torch.zeros((n_steps, n_layers, Tmax, Hq, d), dtype=torch.bfloat16, device="cuda")
    out_d = torch.zeros_like(out_h)

    # host-scheduled
    L, rung, trace = L0, rung0, []
    for t, e in enumerate(steps):
        st_h.launch(rung, L, e["q"], e["kt"], e["vt"], out_h[t], e["x"], e["drafts"][rung])
        a, bonus, s = st_h.wait(timeout_s=60.0)
        trace.append((rung, L, a, s))
        L += a + 1
        rung = api.ladder_next(rung, K, s, 0.8, 0.6)
    st_h.flush()
    torch.cuda.synchronize()

    # device-scheduled: every step enqueued without reading anything back
    log = torch.full((n_steps, 4), -1, dtype=torch.int32, device="cuda")
    st_d.device_start(rung0, L0)
    for t, e in enumerate(steps):
        st_d.launch_device(e["q"], e["kt"], e["vt"], out_d[t], e["x"], e["drafts"], log)
    st_d.flush()
    torch.cuda.synchronize()
    say("host trace", [(r_, a_) for r_, _, a_, _ in trace])
    log_h = log.cpu().numpy()
    for t, (r_, L_, a_, s_) in enumerate(trace):
        assert tuple(log_h[t, :3]) == (r_, L_, a_), (t, log_h[t], (r_, L_, a_))
        assert log_h[t, 3:4].view(np.float32)[0] == np.float32(s_)
    assert len({r_ for r_, *_ in trace}) >= 3
    if with128:
        assert trace[0][0] == K - 1
    for t, (r_, *_rest) in enumerate(trace):
        T = bank.T[r_]
        assert torch.equal(out_h[t, :, :T].view(torch.int16), out_d[t, :, :T].view(torch.int16)), t
    assert torch.equal(kc_h.view(torch.int16), kc_d.view(torch.int16))
    assert torch.equal(vc_h.view(torch.int16), vc_d.view(torch.int16))
    # the configuration's outputs hold the last step's result in both modes
    assert int(st_d.accept_len.item()) == trace[-1][2] == int(st_h.accept_len.item())
    a_last = trace[-1][2]
    assert torch.equal(st_d.path[: a_last + 1], st_h.path[: a_last + 1])
    assert (st_d.path[a_last + 1:] == -1).all() and (st_h.path[a_last + 1:] == -1).all()

    # the device log replayed on the oracle, step by step from the oracle's own
    # caches: tree and prefix as the oracle's ladder leaves them, accept length
    # exact, s within 1e-3; a next tree that differs from the ladder's choice on
    # the oracle's s is allowed only when that s lies within 1e-3 of a threshold
    kc_o = [b.k_cache for b in base]
    vc_o = [b.v_cache for b in base]
    rung, L = rung0, L0
    for t in range(n_steps):
        layers, x, drafts = host_steps[t]
        T = bank.T[rung]
        g_s = float(log_h[t, 3:4].view(np.float32)[0])
        assert tuple(int(v) for v in log_h[t, :2]) == (rung, L), (t, log_h[t])
        ref = orc.verify_step(trees[rung], layers[0].q[:T], layers[0].k_tree[:T],
                              layers[0].v_tree[:T], kc_o[0], vc_o[0], L, x[:T], w_bits,
                              drafts[rung, :T], scale, theta)
        assert int(log_h[t, 2]) == ref["accept_len"], t
        assert abs(g_s - ref["s"]) <= RTOL_STATS * ref["s"] + 1e-6
        assert np.abs(out_d[t, 0, :T].float().cpu().numpy() - ref["out"]).max() <= ATOL_BF16
        kc_o[0], vc_o[0] = ref["k_cache"], ref["v_cache"]
        for l in range(1, n_layers):
            _, rk, rv = orc.tree_attention(layers[l].q[:T], layers[l].k_tree[:T],
                                           layers[l].v_tree[:T], kc_o[l], vc_o[l], L, trees[rung],
                                           scale, theta)
            kc_o[l], vc_o[l] = orc.kv_compact(rk, rv, L, ref["path"])
        L += ref["accept_len"] + 1
        nxt = orc.ladder_next(rung, K, ref["s"], 0.8, 0.6)
        if t + 1 < n_steps and int(log_h[t + 1, 0]) != nxt:
            near = min(abs(ref["s"] - 0.8) / 0.8, abs(ref["s"] - 0.6) / 0.6)
            assert near <= RTOL_STATS, (t, ref["s"])
            nxt = int(log_h[t + 1, 0])
        rung = nxt
    kd = host_bits(kc_d)
    vd = host_bits(vc_d)
    for l in range(n_layers):
        np.testing.assert_array_equal(kd[l][:, :L], kc_o[l][:, :L])
        np.testing.assert_array_equal(vd[l][:, :L], vc_o[l][:, :L])
    st_h.close()
    st_d.close()


def test_step_32_layer_workload_sampled(api):
    """The 32-layer workload at its shapes (prefix 4096, 64-node tree of depth
    5, 32 x 128 heads, hidden 4096, vocab 32000): one step through the step
    driver; attention checked on the oracle for sampled (layer, KV head)
    pairs, the LM-head statistics and acceptance exactly, and the compaction
    of every layer bit for bit against the appended tree rows."""
    wl = synth.WORKLOADS["tree64_L4096_7b_32layer"]
    n_layers, H, d, hid, V, L = wl.n_layers, wl.n_heads, wl.head_dim, wl.hidden, wl.vocab, wl.prefix_len
    trees = synth.workload_trees(wl)
    bank = api.Bank(trees)
    T, D = bank.T[0], bank.D[0]
    cap = L + T + 8
    scale, theta = 1 / math.sqrt(d), wl.rope_theta
    say("32-layer step: generating inputs")
    layers = [synth.attn_inputs(wl.ident, T, H, H, d, L, cap, layer=l) for l in range(n_layers)]
    kc = dev_bf16(stack(layers, "k_cache"))
    vc = dev_bf16(stack(layers, "v_cache"))
    w = synth.lm_head_weight(wl.ident, V, hid)
    w64 = orc.bf16_to_f64(w)
    x = margin_hidden(wl.ident, T, w, w64=w64)
    am = (orc.bf16_to_f64(x) @ w64.T).argmax(axis=1)
    u, r = synth.draft_randoms(wl.ident, T, V)
    tok = synth.draft_tokens(trees[0], am, u, r, wl.p_acc)
    st = api.Step(bank, kc, vc, dev_bf16(w), n_layers=n_layers, Hq=H, Hkv=H, d=d, cap=cap,
                  tree_rows=T, scale=scale, rope_theta=theta, cache_layer_stride=H * cap * d)
    out = torch.empty((n_layers, T, H, d), dtype=torch.bfloat16, device="cuda")
    say("32-layer step: launch")
    st.launch(0, L, dev_bf16(stack(layers, "q")), dev_bf16(stack(layers, "k_tree")),
              dev_bf16(stack(layers, "v_tree")), out, dev_bf16(x), dev_i32(tok))
    a, bonus, s = st.wait(timeout_s=120.0)
    st.flush()
    torch.cuda.synchronize()
    ra, rpath, rbonus, rbest = orc.accept(trees[0], tok, am)
    assert (a, bonus) == (ra, rbonus)
    assert st.path.cpu().numpy()[: a + 1].tolist() == list(rpath)
    z = orc.verify_logits(x, w).astype(np.float32)
    rH, rp1, ram = orc.logit_stats(z)
    np.testing.assert_array_equal(st.argmax.cpu().numpy(), ram)
    np.testing.assert_allclose(st.top1p.cpu().numpy(), rp1, rtol=RTOL_STATS, atol=1e-6)
    kc_h, vc_h = host_bits(kc), host_bits(vc)
    out_h = out.float().cpu().numpy()
    for l, g in ((0, 0), (13, 7), (31, 31)):
        x_l = layers[l]
        ref, rk, rv = orc.tree_attention(x_l.q[:, g:g + 1], x_l.k_tree[:, g:g + 1],
                                         x_l.v_tree[:, g:g + 1], x_l.k_cache[g:g + 1],
                                         x_l.v_cache[g:g + 1], L, trees[0], scale, theta)
        err = np.abs(out_h[l, :, g:g + 1] - ref).max()
        say(f"  layer {l} head {g}: max abs err {err:.2e}")
        assert err <= ATOL_BF16
        rk2, rv2 = orc.kv_compact(rk, rv, L, rpath)
        np.testing.assert_array_equal(kc_h[l, g:g + 1, : L + a + 1], rk2[:, : L + a + 1])
        np.testing.assert_array_equal(vc_h[l, g:g + 1, : L + a + 1], rv2[:, : L + a + 1])
    # every layer: the prefix is untouched and row L + j holds the old tree row path[j]
    for l in range(n_layers):
        np.testing.assert_array_equal(vc_h[l, :, :L], layers[l].v_cache[:, :L])
        for j, node in enumerate(rpath):
            np.testing.assert_array_equal(vc_h[l, :, L + j], layers[l].v_tree[node])
    st.close()


def test_device_step_graph_replays_match_eager_steps(api):
    """A segment of 16 device-scheduled steps (the ring depth) captured as one
    graph and replayed three times -- with unrelated eager work and
    synchronisations between the replays -- against the same 48 steps launched
    one by one: per-replay logs, attention outputs, statistics and caches bit
    for bit.  A replay after a number of eager steps that is not a multiple
    of the ring depth is refused."""
    Hq, Hkv, d, hid, V, L0, n_seg, reps = 8, 2, 128, 512, 1000, 40, 16, 3
    theta, scale = 10000.0, 1 / math.sqrt(128)
    trees = bank_trees()
    bank = api.Bank(trees)
    K, Tmax, Dmax = len(trees), max(bank.T), max(bank.D)
    n_steps = n_seg * reps
    cap = L0 + n_steps * (Dmax + 1) + Tmax + 8
    w_bits = synth.lm_head_weight(WL, V, hid, std=W_STD)
    w64 = orc.bf16_to_f64(w_bits)
    W = dev_bf16(w_bits)
    W2 = W.clone()                       # a second weight copy, as the benchmark alternates
    base = synth.attn_inputs(WL, 1, Hq, Hkv, d, L0, cap)
    kc_e, vc_e = dev_bf16(base.k_cache), dev_bf16(base.v_cache)
    kc_g, vc_g = kc_e.clone(), vc_e.clone()
    kw = dict(Hq=Hq, Hkv=Hkv, d=d, cap=cap, tree_rows=Tmax, scale=scale, rope_theta=theta,
              keep_logits=False, stream=torch.cuda.Stream())
    st_e = api.Step(bank, kc_e, vc_e, W, **kw)
    kw["stream"] = torch.cuda.Stream()
    st_g = api.Step(bank, kc_g, vc_g, W, **kw)
    deltas, spikes = synth.regime_spikes(WL, n_seg, Tmax, V, hid)
    seg = []
    for i in range(n_seg):
        layers, x, am, u, r = step_inputs(i, 1, Tmax, Hq, Hkv, d, w_bits, w64, float(deltas[i]),
                                          spikes[i])
        drafts = np.zeros((K, Tmax), np.int32)
        for k in range(K):
            drafts[k, : bank.T[k]] = synth.draft_tokens(trees[k], am, u, r, 0.7)
        seg.append({"q": dev_bf16(layers[0].q), "k_tree": dev_bf16(layers[0].k_tree),
                    "v_tree": dev_bf16(layers[0].v_tree), "hidden": dev_bf16(x),
                    "drafts": dev_i32(drafts), "w_lm": W if i % 2 == 0 else W2,
                    "out": torch.zeros((Tmax, Hq, d), dtype=torch.bfloat16, device="cuda")})
    log_e = torch.full((n_steps, 4), -1, dtype=torch.int32, device="cuda")
    log_g = torch.full((n_steps, 4), -1, dtype=torch.int32, device="cuda")

    # eager: the 24 steps one by one, snapshotting after each segment
    snaps = []
    out_e = [torch.zeros_like(e["out"]) for e in seg]
    st_e.device_start(0, L0)
    for rep in range(reps):
        for i, e in enumerate(seg):
            st_e.launch_device(e["q"], e["k_tree"], e["v_tree"], out_e[i], e["hidden"], e["drafts"],
                               log_e, w_lm=e["w_lm"])
        st_e.flush()
        torch.cuda.synchronize()
        snaps.append({"k": kc_e.clone(), "v": vc_e.clone(), "out": [o.clone() for o in out_e],
                      "top1p": st_e.top1p.clone(), "path": st_e.path.clone()})

    # graph: one capture, three replays
    st_g.device_start(0, L0)
    graph = st_g.device_graph(seg, log_g)
    torch.cuda.synchronize()
    assert (log_g == -1).all()           # capturing ran nothing
    for rep in range(reps):
        graph.launch()
        torch.cuda.synchronize()
        junk = torch.randn(1 << 16, device="cuda").sum()   # eager work between replays
        junk.item()
        say(f"graph replay {rep}: log rows {log_g[rep * n_seg:(rep + 1) * n_seg, 0].tolist()}")
        sn = snaps[rep]
        assert torch.equal(log_g[: (rep + 1) * n_seg], log_e[: (rep + 1) * n_seg]), rep
        assert (log_g[(rep + 1) * n_seg:] == -1).all()
        assert torch.equal(kc_g.view(torch.int16), sn["k"].view(torch.int16)), rep
        assert torch.equal(vc_g.view(torch.int16), sn["v"].view(torch.int16)), rep
        for i, e in enumerate(seg):
            assert torch.equal(e["out"].view(torch.int16), sn["out"][i].view(torch.int16)), (rep, i)
        assert torch.equal(st_g.top1p, sn["top1p"]) and torch.equal(st_g.path, sn["path"])
    assert len(set(log_e[:, 0].tolist())) >= 2          # the ladder moved inside the segments
    e = seg[0]
    st_g.launch_device(e["q"], e["k_tree"], e["v_tree"], e["out"], e["hidden"], e["drafts"])
    with pytest.raises(api.EntmtpError) as err:          # one eager step: the ring slot moved
        graph.launch()
    assert err.value.code == api.EINVAL
    st_g.flush()
    torch.cuda.synchronize()
    graph.close()
    st_e.close()
    st_g.close()


def test_device_scheduled_fixed_prefix_and_cache_overflow(api):
    """(1) With device_prefix_fixed every device-scheduled step verifies at the
    prefix length it started with: the log's prefix column stays put, and the
    steps equal host-scheduled steps launched at that prefix (trees, accept
    lengths, s and caches bit for bit).  (2) A run whose prefix outgrows the
    cache (one fixed 64-node tree): the first step whose prefix plus tree
    exceeds the capacity, and every step after it, logs accept length -1 and
    keeps its tree and prefix length; the steps before it log as usual."""
    Hq, Hkv, d, hid, V, L0, n_steps = 8, 2, 128, 512, 1000, 40, 8
    theta, scale = 10000.0, 1 / math.sqrt(128)
    trees = bank_trees()
    bank = api.Bank(trees)
    K, Tmax = len(trees), max(bank.T)
    w_bits = synth.lm_head_weight(WL, V, hid, std=W_STD)
    w64 = orc.bf16_to_f64(w_bits)
    W = dev_bf16(w_bits)
    deltas, spikes = synth.regime_spikes(WL, n_steps, Tmax, V, hid)
    steps = []
    for t in range(n_steps):
        layers, x, am, u, r = step_inputs(t, 1, Tmax, Hq, Hkv, d, w_bits, w64, float(deltas[t]),
                                          spikes[t])
        drafts = np.zeros((K, Tmax), np.int32)
        for k in range(K):
            drafts[k, : bank.T[k]] = synth.draft_tokens(trees[k], am, u, r, 0.7)
        steps.append({"q": dev_bf16(layers[0].q), "kt": dev_bf16(layers[0].k_tree),
                      "vt": dev_bf16(layers[0].v_tree), "x": dev_bf16(x), "drafts": dev_i32(drafts)})
    out = torch.zeros((Tmax, Hq, d), dtype=torch.bfloat16, device="cuda")

    # (1) fixed prefix, host- and device-scheduled
    cap = L0 + Tmax + 8
    base = synth.attn_inputs(WL, 1, Hq, Hkv, d, L0, cap)
    kc_h, vc_h = dev_bf16(base.k_cache), dev_bf16(base.v_cache)
    kc_d, vc_d = kc_h.clone(), vc_h.clone()
    kw = dict(Hq=Hq, Hkv=Hkv, d=d, cap=cap, tree_rows=Tmax, scale=scale, rope_theta=theta,
              keep_logits=False)
    st_h = api.Step(bank, kc_h, vc_h, W, **kw)
    st_d = api.Step(bank, kc_d, vc_d, W, device_prefix_fixed=True, **kw)
    rung, trace = 0, []
    for e in steps:
        st_h.launch(rung, L0, e["q"], e["kt"], e["vt"], out, e["x"], e["drafts"][rung])
        a, bonus, s = st_h.wait(timeout_s=60.0)
        trace.append((rung, L0, a, s))
        rung = api.ladder_next(rung, K, s, 0.8, 0.6)
    st_h.flush()
    log = torch.full((n_steps, 4), -7, dtype=torch.int32, device="cuda")
    st_d.device_start(0, L0)
    for e in steps:
        st_d.launch_device(e["q"], e["kt"], e["vt"], out, e["x"], e["drafts"], log)
    st_d.flush()
    torch.cuda.synchronize()
    log_h = log.cpu().numpy()
    say("fixed prefix: host trace", [(r_, a_) for r_, _, a_, _ in trace])
    for t, (r_, L_, a_, s_) in enumerate(trace):
        assert tuple(log_h[t, :3]) == (r_, L_, a_), (t, log_h[t])
        assert log_h[t, 3:4].view(np.float32)[0] == np.float32(s_)
    assert len({r_ for r_, *_ in trace}) >= 2
    assert torch.equal(kc_h.view(torch.int16), kc_d.view(torch.int16))
    assert torch.equal(vc_h.view(torch.int16), vc_d.view(torch.int16))
    st_h.close()
    st_d.close()

    # (2) growing prefix, one fixed tree (thresholds that never move the
    # ladder), a cache four slots larger than the first step needs
    rung = 3
    cap = L0 + bank.T[rung] + 4
    base = synth.attn_inputs(WL, 1, Hq, Hkv, d, L0, cap)
    kc, vc = dev_bf16(base.k_cache), dev_bf16(base.v_cache)
    st = api.Step(bank, kc, vc, W, tau_on=float("inf"), tau_off=float("-inf"),
                  **dict(kw, cap=cap))
    log = torch.full((n_steps, 4), -7, dtype=torch.int32, device="cuda")
    st.device_start(rung, L0)
    for e in steps:
        st.launch_device(e["q"], e["kt"], e["vt"], out, e["x"], e["drafts"], log)
    st.flush()
    torch.cuda.synchronize()
    log_h = log.cpu().numpy()
    say("overflow run log", log_h[:, :3].tolist())
    L, over = L0, False
    for t in range(n_steps):
        r_, L_, a_ = (int(v) for v in log_h[t, :3])
        assert (r_, L_) == (rung, L), (t, log_h[t])
        over = over or L + bank.T[rung] > cap
        if over:
            assert a_ == -1, (t, log_h[t])
        else:
            assert 0 <= a_ <= bank.D[rung], (t, log_h[t])
            L += a_ + 1
    assert over                                  # the run did outgrow the cache
    np.testing.assert_array_equal(host_bits(kc)[:, :L0], base.k_cache[:, :L0])   # prefix intact
    st.close()
