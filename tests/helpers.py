"""Shared test plumbing: device transfer of bf16 bit patterns and the
margin-enforced hidden states (the oracle decides the margin)."""
from __future__ import annotations

import numpy as np

from oracle import entmtp_oracle as orc
from paper_2606_27550_amd import synth

MARGIN = 1e-2   # top-1 minus top-2 logit of every generated row


def dev_bf16(bits: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_bits(t) -> np.ndarray:
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def top2_gap(z: np.ndarray) -> np.ndarray:
    part = np.partition(z, -2, axis=1)[:, -2:]
    return part[:, 1] - part[:, 0]


def margin_hidden(wl_ident: int, n_rows: int, w_bits: np.ndarray, step: int = 0,
                  w64: np.ndarray | None = None, spikes=None, w_std: float = 0.02) -> np.ndarray:
    """Hidden-state rows whose oracle logits have a top-2 gap >= MARGIN.

    Failing rows are redrawn from the next attempt's stream.  ``spikes`` =
    (delta, tokens) applies the scheduler workload's planted lift."""
    hid = w_bits.shape[1]
    wf = w64 if w64 is not None else orc.bf16_to_f64(w_bits)

    def make(attempt):
        x = synth.hidden_rows(wl_ident, n_rows, hid, step=step, attempt=attempt)
        if spikes is not None:
            delta, toks = spikes
            x = synth.plant_spike(x, w_bits, toks, delta, w_std)
        return x

    def ok(rows):
        z = orc.bf16_to_f64(rows) @ wf.T
        return top2_gap(z) >= MARGIN

    return synth.redraw_until(make, ok)
