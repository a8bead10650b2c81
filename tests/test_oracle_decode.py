"""Whole decodes with the oracle on the small workloads (Section 2: iterate
until every position is unmasked; Section 4.1: semi-autoregressive blocks).

Checks the run-level invariants: the mask only shrinks, every non-idle step
commits at least one token, a fallback step commits exactly one (the
leftmost masked position of the active block), the number of steps (NFE)
is at most the generation length, everything is unmasked at the end, and
resuming from a saved state reproduces an uninterrupted run.
"""
import numpy as np
import pytest

from paper_2609_39859_amd import synth


def _decode(orc, cfg, start_step=0, state=None, max_steps=None):
    W = synth.weights(cfg)
    Wb = synth.to_bits(W)
    if state is None:
        tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    else:
        tok, msk, bs = state
    B, L, BL = cfg.B, cfg.L, cfg.block_len
    hist = []
    t = start_step
    while msk.any() and (max_steps is None or t - start_step < max_steps):
        h = synth.to_bits(synth.hidden(cfg, t, W=W))
        prev = msk.copy()
        st = orc.step(h, Wb, tok, msk, bs, B, L, BL, cfg.tau)
        tok, msk, bs = st["tokens"], st["mask"], st["block_start"]
        hist.append(dict(prev=prev, st=st))
        t += 1
        assert t <= cfg.G + 1
    return hist, (tok, msk, bs)


@pytest.mark.parametrize("name", ["tiny", "tiny_peaked"])
def test_tiny_decode_invariants(orc, name):
    cfg = synth.CONFIGS[name]
    hist, (tok, msk, bs) = _decode(orc, cfg)
    B, L, P, BL = cfg.B, cfg.L, cfg.P, cfg.block_len
    assert not msk.any()
    assert len(hist) <= cfg.G
    n_fb = 0
    for h in hist:
        st, prev = h["st"], h["prev"]
        newly = np.nonzero(prev.astype(bool) & ~st["mask"].astype(bool))[0]
        assert np.all(st["mask"] <= prev)
        assert np.all(st["tokens"][newly] == st["argmax"][newly])
        for b in range(B):
            mine = [k - b * L for k in newly if b * L <= k < (b + 1) * L]
            if st["fallback"][b] == 1:
                n_fb += 1
                left = min(k - b * L for k in np.nonzero(prev[b * L:(b + 1) * L])[0] + b * L)
                assert mine == [left]
            elif st["fallback"][b] == 0:
                assert len(mine) >= 1
                assert all(st["conf"][b * L + k] > cfg.tau for k in mine)
    # prompt positions are never touched
    init_tok = synth.initial_state(cfg)[0].numpy()
    for b in range(B):
        assert np.array_equal(tok[b * L: b * L + P], init_tok[b * L: b * L + P])
    assert n_fb >= 1


def test_resume_matches_uninterrupted(orc):
    cfg = synth.CONFIGS["tiny"]
    full, end_full = _decode(orc, cfg)
    part, state = _decode(orc, cfg, max_steps=9)
    rest, end_rest = _decode(orc, cfg, start_step=9, state=state)
    assert len(part) + len(rest) == len(full)
    for a, b in zip(end_full, end_rest):
        assert np.array_equal(a, b)


def test_mid_config_single_step(orc):
    """The mid workload (30% of generation positions masked): one step on
    every row, block skip-forward over complete blocks included."""
    cfg = synth.CONFIGS["mid"].with_(B=1)
    W = synth.weights(cfg)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    h = synth.to_bits(synth.hidden(cfg, 0))
    rows = np.arange(cfg.P, cfg.L)
    st = orc.row_stats(h, synth.to_bits(W), rows)
    assert np.all(st["entropy"] <= np.log(cfg.V) + 1e-12)
    assert np.all(st["conf"] >= 1.0 / cfg.V - 1e-15)
