"""Pins of the oracle's LM-head logits (§2.2 LM-head form) and per-node
softmax statistics (§4 path-value score p0; entropy signal of §3 / App. A).

Independent references: brute-force triple loops, one-hot selection, and the
closed forms of entropy and top-1 probability for uniform, one-hot, k-way tie
and two-level distributions; shift invariance and overflow safety.
"""
import math

import numpy as np
import pytest

from oracle import entmtp_oracle as orc
from paper_2606_27550_amd import synth


def test_lm_head_bruteforce_tiny():
    g = np.random.default_rng(0)
    X = synth.f32_to_bf16_bits(g.standard_normal((3, 5)).astype(np.float32))
    W = synth.f32_to_bf16_bits(g.standard_normal((7, 5)).astype(np.float32))
    z = orc.verify_logits(X, W)
    xf, wf = orc.bf16_to_f64(X), orc.bf16_to_f64(W)
    for i in range(3):
        for v in range(7):
            acc = 0.0
            for k in range(5):
                acc += float(xf[i, k]) * float(wf[v, k])
            assert abs(z[i, v] - acc) <= 1e-14 * max(1.0, abs(acc))


def test_lm_head_one_hot_selects_weight_column():
    g = np.random.default_rng(1)
    hid, V = 64, 50
    W = synth.f32_to_bf16_bits(g.standard_normal((V, hid)).astype(np.float32))
    X = np.zeros((hid, hid), np.uint16)
    for k in range(hid):
        X[k, k] = 0x3F80                     # bf16 1.0
    z = orc.verify_logits(X, W)
    np.testing.assert_array_equal(z, orc.bf16_to_f64(W).T)
    rows = orc.verify_logits_rows(X, W, [3, 17, 49])
    np.testing.assert_array_equal(rows, z[:, [3, 17, 49]])


@pytest.mark.parametrize("V", [1, 2, 63, 32000, 128256])
def test_uniform_logits(V):
    H, p1, am = orc.logit_stats_row(np.full(V, 3.25))
    assert am == 0
    assert abs(H - math.log(V)) <= 1e-12 * max(1, math.log(V))
    assert abs(p1 - 1.0 / V) <= 1e-15
    if V == 32000:
        assert abs(H - 10.373491181781864) < 1e-12
    if V == 128256:
        assert abs(H - 11.761783545564427) < 1e-12


def test_one_hot_logits():
    z = np.full(1000, -np.inf)
    z[417] = 2.0
    H, p1, am = orc.logit_stats_row(z)
    assert (H, p1, am) == (0.0, 1.0, 417)
    z = np.full(1000, -5.0)
    z[3] = 800.0                              # others at m - 805: exp underflows to 0
    H, p1, am = orc.logit_stats_row(z)
    assert am == 3 and p1 == 1.0 and H == 0.0
    z[3] = 300.0                              # others at m - 305: H = 999 * 305 * e^-305 (to first order)
    H, p1, am = orc.logit_stats_row(z)
    assert am == 3 and p1 == 1.0
    assert abs(H - 999 * 305 * math.exp(-305)) <= 1e-9 * H


@pytest.mark.parametrize("k", [2, 3, 7])
def test_k_way_tie(k):
    z = np.full(500, -np.inf)
    idx = [400, 17, 250, 9, 300, 111, 499][:k]
    z[idx] = 1.5
    H, p1, am = orc.logit_stats_row(z)
    assert am == min(idx)
    assert abs(H - math.log(k)) < 1e-14
    assert abs(p1 - 1.0 / k) < 1e-15


@pytest.mark.parametrize("delta", [0.0, 0.5, 3.0, 11.2, 18.0])
def test_two_level_closed_form(delta):
    V = 32000
    z = np.zeros(V)
    z[12345] = delta
    H, p1, am = orc.logit_stats_row(z)
    ed = math.exp(delta)
    S = ed + V - 1
    assert abs(p1 - ed / S) <= 1e-12 * (ed / S)
    assert abs(H - (math.log(S) - delta * ed / S)) <= 1e-12 * math.log(S)
    assert am == (12345 if delta > 0 else 0)


def test_shift_invariance_overflow_and_temperature():
    g = np.random.default_rng(3)
    z = g.standard_normal(4096)
    H, p1, am = orc.logit_stats_row(z)
    for c in (-50.0, 7.0, 1000.0):
        H2, p2, am2 = orc.logit_stats_row(z + c)
        assert am2 == am
        assert abs(H2 - H) < 1e-9 and abs(p2 - p1) < 1e-12
    # entropy from the definition -sum p log p
    p = np.exp(z - z.max())
    p /= p.sum()
    assert abs(H - float(-(p * np.log(p)).sum())) < 1e-12
    assert abs(p1 - p.max()) < 1e-15
    # inverse temperature scales the logits before the softmax
    Ht, pt, amt = orc.logit_stats_row(z, inv_temp=1 / 0.7)
    pt_ref = np.exp(z / 0.7 - (z / 0.7).max())
    pt_ref /= pt_ref.sum()
    assert amt == am
    assert abs(Ht - float(-(pt_ref * np.log(pt_ref)).sum())) < 1e-12
    # rows are independent
    Z = g.standard_normal((5, 300))
    Hs, ps, ams = orc.logit_stats(Z)
    for i in range(5):
        assert (Hs[i], ps[i], ams[i]) == orc.logit_stats_row(Z[i])
