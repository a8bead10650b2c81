"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded input bits (see tests/harness.py for the comparison rules).

Small workloads are checked on every row and, for decodes, in lock-step:
each step starts both sides from the oracle's state.  Full-size workloads
(d = 4096, V = 126464) are checked in the launch configuration the benchmark
times, on sampled rows the oracle evaluates one by one, plus properties that
hold for every row.
"""
import math
import types

import numpy as np
import pytest
import torch

import oracle
from paper_2609_39859_amd import _binding, synth

from harness import (Report, check_rule_on_own_stats, compare_decisions, compare_sampled,
                     compare_stats, gpu_step, host_bits, record)

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _lam(cfg_tau):
    return float(np.float32(cfg_tau))


def _say(*a):
    print(*a, flush=True)


def lockstep_decode(cfg, rule=0, max_steps=None, rows_fn=None,
                    rows_mode=_binding.FORK_ROWS_ALL, temperature=0.0, seed=0):
    """Decode cfg in lock-step; rows_fn(step, mask, block_start) picks the rows
    the oracle evaluates (default: all).  The random fallback rule draws one
    uniform per sequence and step from a seeded generator.  With
    FORK_ROWS_ACTIVE the rows outside the active blocks must come back
    untouched.  With temperature > 0 the candidates of the active blocks are
    drawn (step counter = step index) and compared with the oracle's draws.
    Returns the report and the number of steps."""
    W = synth.weights(cfg)
    Wd = W.to(DEV)
    Wb = host_bits(W)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    B, L, BL = cfg.B, cfg.L, cfg.block_len
    rep = Report()
    t = 0
    while msk[:].any() and (max_steps is None or t < max_steps):
        h = synth.hidden(cfg, t, W=W)
        hb = host_bits(h)
        rows = np.arange(cfg.M) if rows_fn is None else rows_fn(t, msk, bs)
        ref = oracle.row_stats(hb, Wb, rows)
        uni = np.random.default_rng(cfg.seed + 7000 + t).random(B).astype(np.float32)
        g = gpu_step(h.to(DEV), Wd, tok, msk, bs, B, L, BL, cfg.tau, rule=rule, uniform=uni,
                     rows_mode=rows_mode, temperature=temperature, seed=seed, counter=t)
        active = _active_rows(cfg, msk, bs)
        if rows_mode == _binding.FORK_ROWS_ACTIVE:
            _check_untouched(g, active, cfg.M)
        conf_full = np.full(cfg.M, np.nan)
        ent_full = np.full(cfg.M, np.nan)
        am_full = np.zeros(cfg.M, np.int32)
        conf_full[rows] = ref["conf"]
        ent_full[rows] = ref["entropy"]
        am_full[rows] = ref["argmax"]
        if temperature > 0:
            drawn = np.isin(rows, active)
            greedy_rows = rows[~drawn]
            ties = compare_stats(g, {k: v[~drawn] for k, v in ref.items()}, greedy_rows,
                                 hb, Wb, cfg.d, rep)
            drows = rows[drawn]
            sm = oracle.row_sample(hb, Wb, drows, temperature, seed, t)
            ties = np.concatenate([ties, compare_sampled(
                g, {k: v[drawn] for k, v in ref.items()}, sm, drows, hb, Wb, cfg.d,
                temperature, seed, t, rep)])
            conf_full[drows] = sm["conf"]
            am_full[drows] = sm["cand"]
        else:
            ties = compare_stats(g, ref, rows, hb, Wb, cfg.d, rep)
        sel = oracle.select_ex(conf_full, am_full, tok, msk, bs, B, L, BL, _lam(cfg.tau), rule,
                               entropy=ent_full, uniform=uni)
        compare_decisions(g, sel, conf_full, tok, msk, bs, B, L, BL, cfg.tau, rep,
                          rule=rule, near_tie_rows=ties, entropy_ref=ent_full, uniform=uni,
                          tie_seqs_excluded=temperature > 0)
        tok, msk, bs = sel[0], sel[1], sel[2]
        t += 1
        assert t <= cfg.G + 1
    _say("%s: %d steps, %d rows (%d near-tie), %d sequence-steps (%d near-threshold), max err %s"
         % (cfg.name, t, rep.rows, rep.near_tie_rows, rep.seqs, rep.near_threshold_seqs,
            {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, cfg.name, steps=t, rule=rule, rows_mode=rows_mode, temperature=temperature,
           tau=cfg.tau)
    return rep, t


def _active_rows(cfg, msk, bs):
    rows = []
    for b in range(cfg.B):
        masked = [k for k in range(int(bs[b]), cfg.L) if msk[b * cfg.L + k]]
        if masked:
            s = int(bs[b]) + ((masked[0] - int(bs[b])) // cfg.block_len) * cfg.block_len
            rows += [b * cfg.L + k for k in range(s, min(s + cfg.block_len, cfg.L))]
    return np.array(sorted(set(rows)), np.int64)


def _check_untouched(g, active, M):
    """Rows outside the active blocks keep the harness's sentinels."""
    other = np.setdiff1d(np.arange(M), active)
    for k in ("conf", "entropy", "logp", "lse"):
        assert np.all(np.isnan(getattr(g, k)[other])), k
    assert np.all(g.argmax[other] == -7)


def _same_on_active(a, b, active):
    """Two steps agree bit for bit on the active rows and in every decision."""
    for k in ("conf", "entropy", "logp", "lse"):
        x, y = getattr(a, k)[active], getattr(b, k)[active]
        assert np.array_equal(x.view(np.int32), y.view(np.int32)), k
    assert np.array_equal(a.argmax[active], b.argmax[active])
    for k in ("tokens", "mask", "block_start", "fallback", "ncommit", "commit_pos"):
        assert np.array_equal(getattr(a, k), getattr(b, k)), k


# ------------------------------------------------------------ small workloads

def test_crafted_ties_and_layout():
    """One-hot hidden rows against a periodic one-hot W: z_v = 3 exactly for
    every v congruent to the row's hot index, 0 elsewhere.  The candidate must
    be the lowest tied index (checks the accumulator layout and the tie-break
    across lanes, waves and vocabulary tiles); conf = 1/(k + (V-k) e^-3)."""
    _need_gpu()
    for dtype in (torch.float32, torch.bfloat16):
        d, V, B, L = 64, 1000, 3, 50
        M = B * L
        hot = (np.arange(M) * 7) % d
        h = torch.zeros(M, d)
        h[torch.arange(M), torch.as_tensor(hot)] = 3.0
        W = torch.zeros(V, d)
        W[torch.arange(V), torch.arange(V) % d] = 1.0
        h, W = h.to(dtype), W.to(dtype)
        tok = np.zeros(M, np.int32)
        msk = np.zeros(M, np.uint8)
        bs = np.zeros(B, np.int32)
        g = gpu_step(h.to(DEV), W.to(DEV), tok, msk, bs, B, L, 10, 0.5)
        assert np.array_equal(g.argmax, hot)
        k = np.array([len(range(x, V, d)) for x in hot])
        conf = 1.0 / (k + (V - k) * math.exp(-3.0))
        np.testing.assert_allclose(g.conf, conf, atol=2e-6, rtol=1e-5)
        ref = oracle.row_stats(host_bits(h), host_bits(W))
        np.testing.assert_allclose(g.entropy, ref["entropy"], atol=2e-5)
        np.testing.assert_allclose(g.logp, ref["logp"], atol=2e-5)
        assert np.all(g.fallback == -1) and np.all(g.ncommit == 0)


def test_crafted_ragged_tile_boundary():
    """V = 300: the second vocabulary tile holds 44 rows.  One-hot hidden
    rows select one column of W, so the logits of a position are that column
    exactly.  Columns: the maximum at the last row (299), at the first row of
    the ragged tile (256), tied across the tile boundary (255 and 256: the
    lower wins), all logits far below zero, a ragged tile far below the
    maximum, and all logits equal.  Checks candidate, confidence, entropy
    and log-probability against closed forms and the oracle, and the
    teacher-forced log-probability of tokens on both sides of the boundary."""
    _need_gpu()
    V, d = 300, 8
    cols = np.full((V, 6), -1.0, np.float32)
    cols[299, 0] = 1.0
    cols[256, 1] = 1.0
    cols[255, 2] = cols[256, 2] = 1.0
    cols[:, 3] = -50.0
    cols[280, 3] = -40.0
    cols[:256, 4] = 0.0
    cols[256:, 4] = -30.0
    cols[7, 4] = 2.0
    cols[:, 5] = 0.5
    want = np.array([299, 256, 255, 280, 7, 0])
    for dtype in (torch.float32, torch.bfloat16):
        B, L = 1, 12
        M = B * L
        hot = np.arange(M) % 6
        h = torch.zeros(M, d)
        h[torch.arange(M), torch.as_tensor(hot)] = 1.0
        W = torch.zeros(V, d)
        W[:, :6] = torch.as_tensor(cols)
        h, W = h.to(dtype), W.to(dtype)
        g = gpu_step(h.to(DEV), W.to(DEV), np.zeros(M, np.int32), np.zeros(M, np.uint8),
                     np.zeros(B, np.int32), B, L, L, 0.5)
        assert np.array_equal(g.argmax, want[hot])
        z = cols[:, hot].T.astype(np.float64)                 # [M, V] exact logits
        zm = z.max(axis=1, keepdims=True)
        p = np.exp(z - zm) / np.exp(z - zm).sum(axis=1, keepdims=True)
        np.testing.assert_allclose(g.conf, p.max(axis=1), atol=2e-6, rtol=1e-5)
        ent = -(p * np.log(np.where(p > 0, p, 1.0))).sum(axis=1)
        np.testing.assert_allclose(g.entropy, ent, atol=2e-5)
        lse = zm[:, 0] + np.log(np.exp(z - zm).sum(axis=1))
        np.testing.assert_allclose(g.lse, lse, atol=2e-5, rtol=1e-6)
        np.testing.assert_allclose(g.logp, z.max(axis=1) - lse, atol=2e-5)
        ref = oracle.row_stats(host_bits(h), host_bits(W))
        np.testing.assert_allclose(g.entropy, ref["entropy"], atol=2e-5)
        np.testing.assert_allclose(g.logp, ref["logp"], atol=2e-5)
        # teacher-forced tokens on both sides of the tile boundary
        tgt = np.array([255, 256, 299, 0, 298, 257, 255, 256, 299, 0, 1, 280], np.int32)
        out = torch.empty(M, dtype=torch.float32, device=DEV)
        _binding.logprob(h.to(DEV), W.to(DEV), torch.as_tensor(tgt).to(DEV), out)
        torch.cuda.synchronize()
        np.testing.assert_allclose(out.cpu().numpy(), z[np.arange(M), tgt] - lse, atol=2e-5)


@pytest.mark.parametrize("name", ["tiny", "tiny_peaked"])
def test_tiny_lockstep_decode(name):
    _need_gpu()
    cfg = synth.CONFIGS[name]
    rep, steps = lockstep_decode(cfg)
    assert steps <= cfg.G
    assert rep.near_threshold_seqs <= max(1, rep.seqs // 20)
    assert rep.near_tie_rows <= max(1, rep.rows // 50)


@pytest.mark.parametrize("lam", [0.0, 0.5, 1.0])
def test_tiny_threshold_special_cases(lam):
    """lambda = 0: whole blocks per step; lambda = 1: autoregressive order."""
    _need_gpu()
    cfg = synth.CONFIGS["tiny"].with_(tau=lam)
    rep, steps = lockstep_decode(cfg)
    if lam == 0.0:
        assert steps == math.ceil(cfg.G / cfg.block_len)
    if lam == 1.0:
        assert steps == cfg.G


def test_tiny_free_running_matches_oracle_decode():
    """Without resynchronisation the GPU decode reproduces the oracle decode
    (this workload has no near-threshold or near-tie events)."""
    _need_gpu()
    cfg = synth.CONFIGS["tiny"]
    W = synth.weights(cfg)
    Wd, Wb = W.to(DEV), host_bits(W)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    gt, gm, gb = tok.copy(), msk.copy(), bs.copy()
    for t in range(cfg.G + 1):
        if not msk.any():
            break
        h = synth.hidden(cfg, t)
        st = oracle.step(host_bits(h), Wb, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, _lam(cfg.tau))
        g = gpu_step(h.to(DEV), Wd, gt, gm, gb, cfg.B, cfg.L, cfg.block_len, cfg.tau)
        tok, msk, bs = st["tokens"], st["mask"], st["block_start"]
        gt, gm, gb = g.tokens, g.mask, g.block_start
        assert np.array_equal(g.fallback, st["fallback"])
    assert not gm.any() and np.array_equal(gt, tok)


def test_mid_step0_all_rows():
    _need_gpu()
    cfg = synth.CONFIGS["mid"]
    W = synth.weights(cfg)
    h = synth.hidden(cfg, 0)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    hb, Wb = host_bits(h), host_bits(W)
    ref = oracle.row_stats(hb, Wb)
    g = gpu_step(h.to(DEV), W.to(DEV), tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau)
    rep = Report()
    ties = compare_stats(g, ref, np.arange(cfg.M), hb, Wb, cfg.d, rep)
    sel = oracle.select(ref["conf"], ref["argmax"], tok, msk, bs, cfg.B, cfg.L, cfg.block_len,
                        _lam(cfg.tau))
    compare_decisions(g, sel, ref["conf"], tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau,
                      rep, near_tie_rows=ties)
    _say("mid step 0: near-tie rows %d / %d, max err %s" % (rep.near_tie_rows, rep.rows, rep.max_err))
    record(rep, cfg.name, steps=1, tau=cfg.tau)
    assert rep.near_tie_rows <= cfg.M // 50


@pytest.mark.parametrize("rule", [_binding.FORK_RULE_LEFTMOST, _binding.FORK_RULE_MAXCONF])
def test_mid_planted_lockstep_decode(rule):
    """Planted confident rows force multi-commit parallel steps at
    d = 1024, V = 32000; both fallback rules."""
    _need_gpu()
    cfg = synth.CONFIGS["mid_planted"]
    rep, steps = lockstep_decode(cfg, rule=rule,
                                 rows_fn=lambda t, m, b: _active_rows(cfg, m, b))
    assert steps < 0.9 * 39  # parallel steps happen


@pytest.mark.parametrize("rule", [_binding.FORK_RULE_MINCONF, _binding.FORK_RULE_MAXENT,
                                  _binding.FORK_RULE_RANDOM])
@pytest.mark.parametrize("name", ["tiny_peaked", "mid_planted"])
def test_fallback_ablations_lockstep(name, rule):
    """The fallback ablations of Section 4.1 (lowest confidence, highest
    entropy, random masked position) in lock-step with the oracle."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    rows_fn = None if name.startswith("tiny") else (lambda t, m, b: _active_rows(cfg, m, b))
    rep, steps = lockstep_decode(cfg, rule=rule, rows_fn=rows_fn)
    assert steps <= cfg.G
    assert rep.near_threshold_seqs <= max(2, rep.seqs // 10)


RAGGED = [
    # B, L, d, V, dtype, block_len
    (3, 37, 200, 1013, torch.bfloat16, 8),
    (1, 1, 8, 1, torch.bfloat16, 1),
    (2, 300, 72, 257, torch.float32, 300),
    (5, 61, 520, 2049, torch.bfloat16, 7),
    (2, 129, 1032, 777, torch.bfloat16, 64),
    (1, 257, 96, 300, torch.float32, 65),
]


@pytest.mark.parametrize("B,L,d,V,dtype,BL", RAGGED)
@pytest.mark.parametrize("rule", [0, 1, 2, 3, 4])
def test_ragged_shapes_and_random_states(B, L, d, V, dtype, BL, rule):
    """Shapes that are not multiples of the tiles, random masks and block
    starts (including idle sequences and block_start = L)."""
    _need_gpu()
    gen = torch.Generator().manual_seed(B * 1000 + L + d + V + rule)
    M = B * L
    h = (torch.randn(M, d, generator=gen) * 2.0).to(dtype)
    W = (torch.randn(V, d, generator=gen) / math.sqrt(d)).to(dtype)
    rng = np.random.default_rng(M + V)
    msk = (rng.random(M) < 0.5).astype(np.uint8)
    tok = np.where(msk, -1, rng.integers(0, V, M)).astype(np.int32)
    bs = rng.integers(0, L + 1, B).astype(np.int32)
    if B > 1:
        msk[(B - 1) * L:] = 0  # an idle sequence
    hb, Wb = host_bits(h), host_bits(W)
    ref = oracle.row_stats(hb, Wb)
    uni = rng.random(B).astype(np.float32)
    for tau in (0.05, 0.3):
        g = gpu_step(h.to(DEV), W.to(DEV), tok, msk, bs, B, L, BL, tau, rule=rule, uniform=uni)
        rep = Report()
        ties = compare_stats(g, ref, np.arange(M), hb, Wb, d, rep)
        sel = oracle.select_ex(ref["conf"], ref["argmax"], tok, msk, bs, B, L, BL, _lam(tau), rule,
                               entropy=ref["entropy"], uniform=uni)
        compare_decisions(g, sel, ref["conf"], tok, msk, bs, B, L, BL, tau, rep, rule=rule,
                          near_tie_rows=ties, entropy_ref=ref["entropy"], uniform=uni)
        record(rep, "ragged", shape=[B, L, d, V, BL], rule=rule, tau=tau)


@pytest.mark.parametrize("B,L,d,V,dtype,BL", RAGGED)
@pytest.mark.parametrize("rule", [0, 3, 4])
def test_active_rows_mode_matches_all_rows(B, L, d, V, dtype, BL, rule):
    """FORK_ROWS_ACTIVE runs the LM head on the active blocks only: on those
    rows every statistic is bit-identical to the all-rows step (each logit
    accumulates the same products in the same order), the decisions are the
    same, and every other row is left untouched."""
    _need_gpu()
    gen = torch.Generator().manual_seed(7 * B + L + d + V + rule)
    M = B * L
    h = (torch.randn(M, d, generator=gen) * 2.0).to(dtype).to(DEV)
    W = (torch.randn(V, d, generator=gen) / math.sqrt(d)).to(dtype).to(DEV)
    rng = np.random.default_rng(M + V + 1)
    msk = (rng.random(M) < 0.5).astype(np.uint8)
    tok = np.where(msk, -1, rng.integers(0, V, M)).astype(np.int32)
    bs = rng.integers(0, L + 1, B).astype(np.int32)
    if B > 1:
        msk[(B - 1) * L:] = 0  # an idle sequence
    uni = rng.random(B).astype(np.float32)
    active = _active_rows(types.SimpleNamespace(B=B, L=L, block_len=BL), msk, bs)
    for tau in (0.05, 0.3):
        a = gpu_step(h, W, tok, msk, bs, B, L, BL, tau, rule=rule, uniform=uni)
        b = gpu_step(h, W, tok, msk, bs, B, L, BL, tau, rule=rule, uniform=uni,
                     rows_mode=_binding.FORK_ROWS_ACTIVE)
        _same_on_active(a, b, active)
        _check_untouched(b, active, M)


@pytest.mark.parametrize("name,rule", [("tiny_peaked", 0), ("mid_planted", 0),
                                       ("mid_planted", 1)])
def test_active_rows_mode_lockstep_decode(name, rule):
    """A whole decode in FORK_ROWS_ACTIVE against the oracle on the active
    rows, in lock-step."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    rep, steps = lockstep_decode(cfg, rule=rule,
                                 rows_fn=lambda t, m, b: _active_rows(cfg, m, b),
                                 rows_mode=_binding.FORK_ROWS_ACTIVE)
    assert steps <= cfg.G
    assert rep.near_threshold_seqs <= max(2, rep.seqs // 10)


# ------------------------------------------------------- drawn candidates

SEED = 0x9E3779B97F4A7C15


@pytest.mark.parametrize("name,temperature,rows_mode", [
    ("tiny", 1.0, 0), ("tiny_peaked", 0.8, 0), ("tiny_peaked", 0.8, 1),
    ("mid_planted", 0.8, 0), ("mid_planted", 1.5, 1)])
def test_drawn_candidates_lockstep_decode(name, temperature, rows_mode):
    """A whole decode with candidates drawn at a sampling temperature
    (Section 2), in lock-step with the oracle's Gumbel-max draws over
    Philox4x32-10 (step counter = step index)."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    rows_fn = None if (name.startswith("tiny") and rows_mode == 0) else \
        (lambda t, m, b: _active_rows(cfg, m, b))
    rep, steps = lockstep_decode(cfg, rows_fn=rows_fn, rows_mode=rows_mode,
                                 temperature=temperature, seed=SEED)
    assert steps <= cfg.G
    assert rep.near_threshold_seqs <= max(2, rep.seqs // 10)
    assert rep.near_tie_rows <= max(2, rep.rows // 50)


@pytest.mark.parametrize("B,L,d,V,dtype,BL", RAGGED)
def test_drawn_candidates_ragged_and_mode_invariant(B, L, d, V, dtype, BL):
    """Ragged shapes with random states: drawn candidates of every active
    row against the oracle, and bit-identical results between FORK_ROWS_ALL
    and FORK_ROWS_ACTIVE (the draws are keyed by the row, not by the tile)."""
    _need_gpu()
    gen = torch.Generator().manual_seed(3 * B + L + d + V)
    M = B * L
    h = (torch.randn(M, d, generator=gen) * 2.0).to(dtype)
    W = (torch.randn(V, d, generator=gen) / math.sqrt(d)).to(dtype)
    rng = np.random.default_rng(M + V + 2)
    msk = (rng.random(M) < 0.5).astype(np.uint8)
    tok = np.where(msk, -1, rng.integers(0, V, M)).astype(np.int32)
    bs = rng.integers(0, L + 1, B).astype(np.int32)
    hb, Wb = host_bits(h), host_bits(W)
    active = _active_rows(types.SimpleNamespace(B=B, L=L, block_len=BL), msk, bs)
    temperature, counter = 0.7, 12345
    a = gpu_step(h.to(DEV), W.to(DEV), tok, msk, bs, B, L, BL, 0.3, temperature=temperature,
                 seed=SEED, counter=counter)
    b = gpu_step(h.to(DEV), W.to(DEV), tok, msk, bs, B, L, BL, 0.3, temperature=temperature,
                 seed=SEED, counter=counter, rows_mode=_binding.FORK_ROWS_ACTIVE)
    _same_on_active(a, b, active)
    _check_untouched(b, active, M)
    rep = Report()
    st = oracle.row_stats(hb, Wb)
    other = np.setdiff1d(np.arange(M), active)
    compare_stats(a, {k: v[other] for k, v in st.items()}, other, hb, Wb, d, rep)
    if active.size:
        sm = oracle.row_sample(hb, Wb, active, temperature, SEED, counter)
        compare_sampled(a, {k: v[active] for k, v in st.items()}, sm, active, hb, Wb, d,
                        temperature, SEED, counter, rep)
    _say("ragged drawn %s: %d rows (%d near-tie)" % ((B, L, d, V, BL), rep.rows, rep.near_tie_rows))
    record(rep, "ragged", shape=[B, L, d, V, BL], temperature=temperature)


@pytest.mark.parametrize("B,L,d,V,BL", [(4, 256, 1024, 32000, 32), (2, 384, 264, 1013, 16),
                                         (8, 512, 4096, 126464, 32)])
def test_drawn_all_rows_interleaved_positions(B, L, d, V, BL):
    """Drawing over all rows when B*L is a multiple of 256 (more than one
    position tile) runs the LM-head kernel whose position tiles take
    interleaved 16-row chunks.  Rows whose candidates are not drawn equal
    the greedy step bit for bit; drawn rows equal the active-rows mode bit
    for bit and the oracle's draws."""
    _need_gpu()
    M = B * L
    assert M % 256 == 0 and M // 256 > 1
    gen = torch.Generator().manual_seed(5 * B + L + d + V)
    h = (torch.randn(M, d, generator=gen) * 2.0).to(torch.bfloat16)
    W = (torch.randn(V, d, generator=gen) / math.sqrt(d)).to(torch.bfloat16)
    rng = np.random.default_rng(M + V + 7)
    msk = (rng.random(M) < 0.6).astype(np.uint8)
    tok = np.where(msk, -1, rng.integers(0, V, M)).astype(np.int32)
    bs = (rng.integers(0, L // BL, B) * BL).astype(np.int32)
    hd, Wd = h.to(DEV), W.to(DEV)
    active = _active_rows(types.SimpleNamespace(B=B, L=L, block_len=BL), msk, bs)
    other = np.setdiff1d(np.arange(M), active)
    temperature, counter = 0.8, 77
    a = gpu_step(hd, Wd, tok, msk, bs, B, L, BL, 0.9, temperature=temperature, seed=SEED,
                 counter=counter)
    g = gpu_step(hd, Wd, tok, msk, bs, B, L, BL, 0.9)
    b = gpu_step(hd, Wd, tok, msk, bs, B, L, BL, 0.9, temperature=temperature, seed=SEED,
                 counter=counter, rows_mode=_binding.FORK_ROWS_ACTIVE)
    for k in ("conf", "entropy", "logp", "lse"):
        x, y = getattr(a, k)[other], getattr(g, k)[other]
        assert np.array_equal(x.view(np.int32), y.view(np.int32)), k
    assert np.array_equal(a.argmax[other], g.argmax[other])
    _same_on_active(a, b, active)
    hb, Wb = host_bits(h), host_bits(W)
    rows = active[:: max(1, active.size // 64)] if active.size else active
    rep = Report()
    if rows.size:
        st = oracle.row_stats(hb, Wb, rows)
        sm = oracle.row_sample(hb, Wb, rows, temperature, SEED, counter)
        compare_sampled(a, st, sm, rows, hb, Wb, d, temperature, SEED, counter, rep)
    _say("interleaved drawn %s: %d active rows, %d checked (%d near-tie)" % (
        (B, L, d, V, BL), active.size, rep.rows, rep.near_tie_rows))
    record(rep, "interleaved_drawn", shape=[B, L, d, V, BL], temperature=temperature)


def test_drawn_candidates_change_with_counter_and_seed():
    """Different counters or seeds give different draws; the same ones give
    the same bits."""
    _need_gpu()
    cfg = synth.CONFIGS["mid"]
    W = synth.weights(cfg).to(DEV)
    h = synth.hidden(cfg, 0).to(DEV)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    run = lambda seed, counter: gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len,
                                         cfg.tau, temperature=1.0, seed=seed, counter=counter)
    active = _active_rows(cfg, msk, bs)
    a, a2, b, c = run(1, 0), run(1, 0), run(1, 1), run(2, 0)
    assert np.array_equal(a.argmax, a2.argmax) and np.array_equal(a.conf.view(np.int32),
                                                                  a2.conf.view(np.int32))
    assert (a.argmax[active] != b.argmax[active]).mean() > 0.5
    assert (a.argmax[active] != c.argmax[active]).mean() > 0.5
    other = np.setdiff1d(np.arange(cfg.M), active)
    assert np.array_equal(a.argmax[other], b.argmax[other])  # greedy outside


@pytest.mark.parametrize("M,d,V", [(2, 1 << 20, 257), (3, 64, 1000003)])
def test_extreme_sizes(M, d, V):
    """The largest supported hidden size (d = 2^20: 2 MiB rows, the limit of
    the kernel's 32-bit tile offsets) and a vocabulary of about a million
    entries (3907 vocabulary tiles), bf16, every row against the oracle."""
    _need_gpu()
    gen = torch.Generator().manual_seed(M + d + V)
    h = (torch.randn(M, d, generator=gen) * 2.0).to(torch.bfloat16)
    W = (torch.randn(V, d, generator=gen) / math.sqrt(d)).to(torch.bfloat16)
    hb, Wb = host_bits(h), host_bits(W)
    msk = np.ones(M, np.uint8)
    tok = np.full(M, -1, np.int32)
    bs = np.zeros(1, np.int32)
    g = gpu_step(h.to(DEV), W.to(DEV), tok, msk, bs, 1, M, M, 0.5)
    ref = oracle.row_stats(hb, Wb)
    rep = Report()
    compare_stats(g, ref, np.arange(M), hb, Wb, d, rep)
    _say("extreme sizes M=%d d=%d V=%d: max err %s" % (
        M, d, V, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, "extreme", shape=[M, d, V])


def test_caller_workspace_and_determinism():
    """Caller-provided workspace gives the same bits as the library one, and
    repeated runs are bit-identical (fixed merge order, no atomics)."""
    _need_gpu()
    cfg = synth.CONFIGS["mid"]
    W = synth.weights(cfg).to(DEV)
    h = synth.hidden(cfg, 3).to(DEV)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    a = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau)
    b = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau)
    nbytes = _binding.workspace_bytes(cfg.B, cfg.L, cfg.V)
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=DEV)
    off = (-ws.data_ptr()) % 256
    c = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau,
                 workspace=ws[off:off + nbytes])
    for x in (b, c):
        for k in ("conf", "entropy", "logp", "lse"):
            assert np.array_equal(getattr(a, k).view(np.int32), getattr(x, k).view(np.int32)), k
        for k in ("argmax", "tokens", "mask", "block_start", "fallback", "ncommit", "commit_pos"):
            assert np.array_equal(getattr(a, k), getattr(x, k)), k
    # fork_workspace_bytes covers every mode; a step that draws candidates
    # needs all of it
    with pytest.raises(_binding.ForkError):
        gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau,
                 workspace=ws[off:off + nbytes - 256], temperature=1.0)


def test_bad_block_start_is_reported_in_data():
    _need_gpu()
    B, L, d, V = 3, 16, 16, 40
    h = torch.randn(B * L, d).to(torch.bfloat16).to(DEV)
    W = torch.randn(V, d).to(torch.bfloat16).to(DEV)
    msk = np.ones(B * L, np.uint8)
    tok = np.full(B * L, -1, np.int32)
    bs = np.array([-1, 17, 16], np.int32)
    g = gpu_step(h, W, tok, msk, bs, B, L, 4, 0.5)
    assert g.fallback.tolist() == [-2, -2, -1]
    assert np.array_equal(g.mask, msk) and np.array_equal(g.tokens, tok)
    assert g.block_start.tolist() == [-1, 17, 16]
    assert np.all(g.commit_pos == -1)


# ------------------------------------------------------------- full sizes

def _sample_rows(cfg, msk, bs, n_seq=4, n_random=32, seed=0):
    rng = np.random.default_rng(seed)
    act = _active_rows(cfg.with_(B=min(cfg.B, n_seq)), msk[: min(cfg.B, n_seq) * cfg.L], bs)
    extra = rng.choice(cfg.M, n_random, replace=False)
    edge = np.array([0, 255, 256, cfg.M - 1])
    return np.array(sorted(set(act.tolist()) | set(extra.tolist()) | set(edge.tolist())), np.int64), \
        list(range(min(cfg.B, n_seq)))


@pytest.mark.parametrize("name", ["llada8b", "rollout", "long"])
def test_full_size_step_sampled(name):
    """One step at the benchmark's full sizes and launch configuration:
    sampled rows against the oracle, decisions exact on the sequences whose
    active block the oracle evaluated, and every-row properties:
    0 <= H <= log V, 1/V <= conf <= 1, log q = -log(1/conf) within float
    error.  With these distributions no position is confident (max q is far
    below lambda), so every sequence takes a fallback step at position P."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    _say("full-size %s: generating inputs" % name)
    W = synth.weights(cfg, device=DEV)
    h = synth.hidden(cfg, 0, device=DEV)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    _say("full-size %s: GPU step" % name)
    g = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau)
    rows, seqs = _sample_rows(cfg, msk, bs)
    _say("full-size %s: oracle on %d rows" % (name, rows.size))
    hb, Wb = host_bits(h), host_bits(W)
    ref = oracle.row_stats(hb, Wb, rows)
    rep = Report()
    ties = compare_stats(g, ref, rows, hb, Wb, cfg.d, rep)
    conf_full = np.full(cfg.M, np.nan)
    am_full = np.zeros(cfg.M, np.int32)
    conf_full[rows] = ref["conf"]
    am_full[rows] = ref["argmax"]
    sel = oracle.select(conf_full, am_full, tok, msk, bs, cfg.B, cfg.L, cfg.block_len,
                        _lam(cfg.tau))
    compare_decisions(g, sel, conf_full, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau,
                      rep, seqs=seqs, near_tie_rows=ties)
    check_rule_on_own_stats(g, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau, 0,
                            range(cfg.B))
    logV = math.log(cfg.V)
    assert np.all(g.entropy >= -1e-3) and np.all(g.entropy <= logV + 1e-3)
    assert np.all(g.conf >= (1.0 / cfg.V) * (1 - 1e-3)) and np.all(g.conf <= 1.0 + 1e-6)
    np.testing.assert_allclose(g.logp, np.log(g.conf.astype(np.float64)), atol=1e-4)
    assert np.all(g.fallback == 1)
    assert np.all(g.commit_pos[:, 0] == cfg.P) and np.all(g.commit_pos[:, 1:] == -1)
    _say("full-size %s: %d rows ok (%d near-tie), max err %s" % (
        name, rep.rows, rep.near_tie_rows, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, name, steps=1, tau=cfg.tau)


@pytest.mark.parametrize("name", ["llada8b", "rollout"])
def test_full_size_active_rows_mode(name):
    """FORK_ROWS_ACTIVE at full size: bit-identical to the all-rows step on
    the active rows, same decisions, other rows untouched; the active rows of
    the first sequences against the oracle."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    W = synth.weights(cfg, device=DEV)
    h = synth.hidden(cfg, 5, device=DEV)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    _say("full-size active %s: GPU steps" % name)
    a = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau)
    b = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau,
                 rows_mode=_binding.FORK_ROWS_ACTIVE)
    active = _active_rows(cfg, msk, bs)
    assert active.size == cfg.B * cfg.block_len
    _same_on_active(a, b, active)
    _check_untouched(b, active, cfg.M)
    rows = active[: 2 * cfg.block_len]
    ref = oracle.row_stats(host_bits(h), host_bits(W), rows)
    rep = Report()
    compare_stats(b, ref, rows, host_bits(h), host_bits(W), cfg.d, rep)
    _say("full-size active %s: ok, max err %s" % (
        name, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, name, steps=1, rows_mode=1, tau=cfg.tau)


@pytest.mark.parametrize("name,rows_mode", [("llada8b", 0), ("llada8b", 1), ("rollout", 0),
                                            ("rollout", 1)])
def test_full_size_drawn_candidates(name, rows_mode):
    """Drawn candidates at the full sizes (temperature 0.8, as in the
    paper's tuned Fork-dLLM setting): the active rows of the first two and
    the last sequence against the oracle's draws (over all rows, the
    rollout batch spreads its drawn blocks over 96 position tiles)."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    W = synth.weights(cfg, device=DEV)
    h = synth.hidden(cfg, 2, device=DEV)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    _say("full-size drawn %s mode %d: GPU step" % (name, rows_mode))
    g = gpu_step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, cfg.tau, rows_mode=rows_mode,
                 temperature=0.8, seed=SEED, counter=2)
    act = _active_rows(cfg, msk, bs)
    rows = np.concatenate([act[: 2 * cfg.block_len], act[-cfg.block_len:]])
    hb, Wb = host_bits(h), host_bits(W)
    st = oracle.row_stats(hb, Wb, rows)
    sm = oracle.row_sample(hb, Wb, rows, 0.8, SEED, 2)
    rep = Report()
    compare_sampled(g, st, sm, rows, hb, Wb, cfg.d, 0.8, SEED, 2, rep)
    _say("full-size drawn %s: %d rows ok (%d near-tie), max err %s" % (
        name, rep.rows, rep.near_tie_rows, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, name, steps=1, rows_mode=rows_mode, temperature=0.8, tau=cfg.tau)


def test_full_size_planted_peaks_lockstep():
    """Multi-commit parallel steps at the full LLaDA-8B shape (d = 4096,
    V = 126464): three lock-step steps with planted peaks, every active row
    against the oracle, decisions exact outside the exclusion sets."""
    _need_gpu()
    cfg = synth.CONFIGS["llada8b_planted"]
    W = synth.weights(cfg, device=DEV)
    Wb = host_bits(W)
    tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
    B, L, BL = cfg.B, cfg.L, cfg.block_len
    rep = Report()
    multi = 0
    for t in range(3):
        h = synth.hidden(cfg, t, device=DEV, W=W)
        hb = host_bits(h)
        rows = _active_rows(cfg, msk, bs)
        _say("planted full-size step %d: GPU step, oracle on %d rows" % (t, rows.size))
        g = gpu_step(h, W, tok, msk, bs, B, L, BL, cfg.tau)
        ref = oracle.row_stats(hb, Wb, rows)
        ties = compare_stats(g, ref, rows, hb, Wb, cfg.d, rep)
        conf_full = np.full(cfg.M, np.nan)
        am_full = np.zeros(cfg.M, np.int32)
        conf_full[rows], am_full[rows] = ref["conf"], ref["argmax"]
        sel = oracle.select(conf_full, am_full, tok, msk, bs, B, L, BL, _lam(cfg.tau))
        compare_decisions(g, sel, conf_full, tok, msk, bs, B, L, BL, cfg.tau, rep,
                          near_tie_rows=ties)
        multi += int(np.sum(sel[4] > 1))
        tok, msk, bs = sel[0], sel[1], sel[2]
    assert multi >= 4, "expected parallel multi-commit steps, got %d" % multi
    _say("planted full-size: %d rows (%d near-tie), %d multi-commit sequence-steps, max err %s" % (
        rep.rows, rep.near_tie_rows, multi, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, cfg.name, steps=3, multi_commit_seq_steps=multi, tau=cfg.tau)


def _decode_checks(cfg):
    """Steps of a full-size decode checked against the oracle, by kind:
    "block" = every row of the active blocks (at most 256) + 64 sampled rows,
    "commit" = the committed rows + 16 sampled rows.  They include the first
    step, the last step of the first block, the first two steps of the
    second, the middle block boundary and the final step."""
    BL, G = cfg.block_len, cfg.G
    big = cfg.B * BL > 256
    checks = {t: "commit" for t in (BL - 1, BL + 1, G // 2 - 1, G // 2)}
    for t in (0, BL, G - 1):
        checks[t] = "commit" if big else "block"
    return checks


@pytest.mark.parametrize("name", ["llada8b", "rollout", "long"])
def test_full_size_decode_is_autoregressive(name):
    """A whole decode at full size on the GPU, in the launch configuration
    the benchmark times (all B*L rows through the LM head), hidden states
    regenerated every step.  With no confident position every step is a
    fallback step and the commits follow AR order P, P+1, ... (Section 2),
    crossing every block boundary (Section 4.1).  At the steps of
    _decode_checks the GPU's statistics are compared with the oracle's on
    the committed or active-block rows plus sampled rows, and the decision
    against the oracle's selection on those rows.  Per step, the fallback
    flag and the log-probability of the committed token (the inputs of
    ForkGRPO, Section 3.2) are kept; at the end the recorded
    log-probabilities of checked steps are recomputed by fork_logprob
    (teacher forcing on the committed tokens)."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    W = synth.weights(cfg, device=DEV)
    Wb = None
    tok, msk, bs = (x.to(DEV) for x in synth.initial_state(cfg))
    B, L, BL, M, P = cfg.B, cfg.L, cfg.block_len, cfg.M, cfg.P
    f32 = dict(dtype=torch.float32, device=DEV)
    conf, ent, logp, lse = (torch.empty(M, **f32) for _ in range(4))
    am = torch.empty(M, dtype=torch.int32, device=DEV)
    fb = torch.empty(B, dtype=torch.int32, device=DEV)
    nc = torch.empty(B, dtype=torch.int32, device=DEV)
    cp = torch.empty(B * BL, dtype=torch.int32, device=DEV)
    checks = _decode_checks(cfg)
    rng = np.random.default_rng(cfg.seed + 99)
    fallbacks = np.zeros((cfg.G, B), np.int32)
    logp_commit = np.zeros((cfg.G, B), np.float32)
    rep = Report()
    lam = _lam(cfg.tau)
    max_conf = 0.0
    _say("full-size decode %s: %d steps, checks at %s" % (name, cfg.G, sorted(checks)))
    for t in range(cfg.G):
        h = synth.hidden(cfg, t, device=DEV)
        if t in checks:
            before = (tok.cpu().numpy(), msk.cpu().numpy(), bs.cpu().numpy())
        _binding.fork_step_ex(h, W, tok, msk, bs, BL, cfg.tau, conf, ent, logp, fb, B=B, L=L,
                              out_lse=lse, out_argmax=am, out_ncommit=nc, out_commit_pos=cp)
        fbh = fb.cpu().numpy()
        cph = cp.cpu().numpy().reshape(B, BL)
        assert np.all(fbh == 1), "step %d: fallback %s" % (t, fbh)
        assert np.all(cph[:, 0] == P + t) and np.all(cph[:, 1:] == -1), "step %d: commits" % t
        committed = np.arange(B) * L + P + t
        fallbacks[t] = fbh
        logp_commit[t] = logp[torch.as_tensor(committed, device=DEV)].cpu().numpy()
        # the threshold decision has a margin far wider than the 2e-3
        # statistics tolerance, so the oracle's decision is the GPU's
        max_conf = max(max_conf, float(conf.max().item()))
        if t not in checks:
            continue
        if Wb is None:
            Wb = host_bits(W)
        hb = host_bits(h)
        tok0, msk0, bs0 = before
        active = _active_rows(cfg, msk0, bs0)
        if checks[t] == "block":
            rows = np.union1d(active, rng.choice(M, 64, replace=False))
        else:
            rows = np.union1d(committed, rng.choice(M, 16, replace=False))
        _say("full-size decode %s step %d: oracle on %d rows (%s)" % (name, t, rows.size, checks[t]))
        g = types.SimpleNamespace(conf=conf.cpu().numpy(), entropy=ent.cpu().numpy(),
                                  logp=logp.cpu().numpy(), lse=lse.cpu().numpy(),
                                  argmax=am.cpu().numpy(), tokens=tok.cpu().numpy(),
                                  mask=msk.cpu().numpy(), block_start=bs.cpu().numpy(),
                                  fallback=fbh, ncommit=nc.cpu().numpy(), commit_pos=cph)
        ref = oracle.row_stats(hb, Wb, rows)
        ties = compare_stats(g, ref, rows, hb, Wb, cfg.d, rep)
        assert np.array_equal(g.tokens[committed], g.argmax[committed])
        assert msk0[committed].all() and not g.mask[committed].any()
        if checks[t] == "block":
            conf_full = np.full(M, np.nan)
            am_full = np.zeros(M, np.int32)
            conf_full[rows], am_full[rows] = ref["conf"], ref["argmax"]
            sel = oracle.select(conf_full, am_full, tok0, msk0, bs0, B, L, BL, lam)
            compare_decisions(g, sel, conf_full, tok0, msk0, bs0, B, L, BL, cfg.tau, rep,
                              near_tie_rows=ties)
        else:
            check_rule_on_own_stats(g, tok0, msk0, bs0, B, L, BL, cfg.tau, 0, range(B))
            rep.seqs += B
    assert not msk.cpu().numpy().reshape(B, L)[:, P:].any()
    assert max_conf < lam - 0.01, "a confident position (%g) near lambda" % max_conf
    assert np.all(fallbacks == 1)
    assert np.all(np.isfinite(logp_commit)) and np.all(logp_commit <= 0)
    # ForkGRPO reads the recorded log q of each fallback commit: the
    # teacher-forced likelihood of the committed tokens under the same head
    # reproduces it
    final_tok = tok
    for t in sorted(checks)[:3]:
        h = synth.hidden(cfg, t, device=DEV)
        rows_t = torch.as_tensor(np.arange(B) * L + P + t, dtype=torch.int32, device=DEV)
        out = torch.empty(B, **f32)
        _binding.logprob(h, W, final_tok[rows_t.long()].contiguous(), out, rows=rows_t)
        np.testing.assert_allclose(out.cpu().numpy(), logp_commit[t], rtol=0, atol=1e-5)
    _say("full-size decode %s: %d steps, %d rows checked (%d near-tie), %d sequence-steps, "
         "max conf %.3g, max err %s" % (name, cfg.G, rep.rows, rep.near_tie_rows, rep.seqs,
                                        max_conf, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, name, steps=cfg.G, decode=True, max_conf=max_conf, tau=cfg.tau)


def _device_decode(cfg, W, hidden_at, state, t0, t1=None):
    """Steps t0 .. t1-1 (or until nothing is masked) on device-resident
    state; per-step host copies of the outputs, and the state at the end."""
    tok, msk, bs = (torch.as_tensor(x).to(DEV) for x in state)
    B, L, BL, M = cfg.B, cfg.L, cfg.block_len, cfg.M
    f32 = dict(dtype=torch.float32, device=DEV)
    outs = []
    t = t0
    while (t1 is None and bool(msk.any())) or (t1 is not None and t < t1):
        assert t < cfg.G
        conf, ent, logp = (torch.empty(M, **f32) for _ in range(3))
        fb = torch.empty(B, dtype=torch.int32, device=DEV)
        cp = torch.empty(B * BL, dtype=torch.int32, device=DEV)
        _binding.fork_step_ex(hidden_at(t), W, tok, msk, bs, BL, cfg.tau, conf, ent, logp, fb,
                              B=B, L=L, out_commit_pos=cp)
        outs.append([x.cpu().numpy() for x in (conf, ent, logp, fb, cp)])
        t += 1
    return outs, tuple(x.cpu().numpy() for x in (tok, msk, bs))


def test_gpu_resume_matches_uninterrupted():
    """The decode's whole state is (tokens, mask, block_start): a GPU decode
    stopped after k steps, its state moved to the host, the library's
    workspaces released and the decode resumed from fresh device buffers
    gives bit-identical per-step outputs and final state to the
    uninterrupted decode (mid_planted: parallel and fallback steps, blocks
    skipped forward)."""
    _need_gpu()
    cfg = synth.CONFIGS["mid_planted"]
    W = synth.weights(cfg)
    Wd = W.to(DEV)
    cache = {}

    def hidden_at(t):
        if t not in cache:
            cache[t] = synth.hidden(cfg, t, W=W).to(DEV)
        return cache[t]

    state0 = tuple(x.numpy() for x in synth.initial_state(cfg))
    ref_outs, ref_final = _device_decode(cfg, Wd, hidden_at, state0, 0)
    T = len(ref_outs)
    assert T > 6 and not ref_final[1].any()
    fbs = np.array([o[3] for o in ref_outs])
    assert (fbs == 0).any() and (fbs == 1).any(), "expected parallel and fallback steps"
    for k in (1, T // 2, T - 1):
        a, mid = _device_decode(cfg, Wd, hidden_at, state0, 0, k)
        torch.cuda.synchronize()
        _binding.release()
        b, final = _device_decode(cfg, Wd, hidden_at, mid, k)
        assert len(a) + len(b) == T
        for t, (x, y) in enumerate(zip(a + b, ref_outs)):
            for i, (u, v) in enumerate(zip(x, y)):
                assert np.array_equal(u.view(np.int32), v.view(np.int32)), \
                    "resume after %d: step %d output %d differs" % (k, t, i)
        for u, v in zip(final, ref_final):
            assert np.array_equal(u, v)
    _say("resume: %d-step decode reproduced after stops at %s" % (T, [1, T // 2, T - 1]))


@pytest.mark.parametrize("B,L,d,V,dtype,BL", RAGGED + [(8, 512, 64, 3000, torch.bfloat16, 32),
                                                       (3, 200, 64, 700, torch.bfloat16, 64)])
@pytest.mark.parametrize("rule", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("rows_mode", [0, 1])
def test_step_decisions_equal_standalone_selection(B, L, d, V, dtype, BL, rule, rows_mode):
    """The step's own selection decides exactly what fork_select decides on
    the step's confidences, candidates and entropies from the same state,
    for every rule and both row modes, with a drawn-candidate case."""
    _need_gpu()
    gen = torch.Generator().manual_seed(11 * B + L + d + V + rule)
    M = B * L
    h = (torch.randn(M, d, generator=gen) * 2.0).to(dtype).to(DEV)
    W = (torch.randn(V, d, generator=gen) / math.sqrt(d)).to(dtype).to(DEV)
    rng = np.random.default_rng(M + V + 5 + rule)
    msk = (rng.random(M) < 0.5).astype(np.uint8)
    tok = np.where(msk, -1, rng.integers(0, V, M)).astype(np.int32)
    bs = rng.integers(0, L + 1, B).astype(np.int32)
    if B > 1:
        msk[(B - 1) * L:] = 0  # an idle sequence
    uni = rng.random(B).astype(np.float32)
    for tau, temperature in ((0.05, 0.0), (0.3, 0.0), (0.2, 0.9)):
        g = gpu_step(h, W, tok, msk, bs, B, L, BL, tau, rule=rule, uniform=uni,
                     rows_mode=rows_mode, temperature=temperature, seed=SEED, counter=3)
        t = lambda x: torch.as_tensor(np.ascontiguousarray(x)).to(DEV)
        conf = np.nan_to_num(g.conf, nan=0.0)
        ent = np.nan_to_num(g.entropy, nan=0.0)
        am = np.where(g.argmax == -7, 0, g.argmax).astype(np.int32)
        tok_d, msk_d, bs_d = t(tok.copy()), t(msk.copy()), t(bs.copy())
        fb = torch.full((B,), -9, dtype=torch.int32, device=DEV)
        nc = torch.full((B,), -9, dtype=torch.int32, device=DEV)
        cp = torch.full((B * BL,), -9, dtype=torch.int32, device=DEV)
        _binding.select(t(conf), t(am), tok_d, msk_d, bs_d, BL, tau, fb, B=B, L=L, rule=rule,
                        entropy=t(ent), uniform=t(uni), out_ncommit=nc, out_commit_pos=cp)
        torch.cuda.synchronize()
        assert np.array_equal(g.tokens, tok_d.cpu().numpy())
        assert np.array_equal(g.mask, msk_d.cpu().numpy())
        assert np.array_equal(g.block_start, bs_d.cpu().numpy())
        assert np.array_equal(g.fallback, fb.cpu().numpy())
        assert np.array_equal(g.ncommit, nc.cpu().numpy())
        assert np.array_equal(g.commit_pos, cp.cpu().numpy().reshape(B, BL))


@pytest.mark.parametrize("name", ["rollout", "long"])
def test_full_size_active_rows_decode(name):
    """A whole full-size decode with the LM head on the active blocks' rows
    only (FORK_ROWS_ACTIVE): AR-order fallback commits across every block
    boundary, rows outside the active blocks never written, and at the
    boundary steps the committed rows plus sampled active rows against the
    oracle."""
    _need_gpu()
    cfg = synth.CONFIGS[name]
    W = synth.weights(cfg, device=DEV)
    Wb = None
    tok, msk, bs = (x.to(DEV) for x in synth.initial_state(cfg))
    B, L, BL, M, P = cfg.B, cfg.L, cfg.block_len, cfg.M, cfg.P
    f32 = dict(dtype=torch.float32, device=DEV)
    conf, ent, logp, lse = (torch.full((M,), float("nan"), **f32) for _ in range(4))
    am = torch.full((M,), -7, dtype=torch.int32, device=DEV)
    fb = torch.empty(B, dtype=torch.int32, device=DEV)
    cp = torch.empty(B * BL, dtype=torch.int32, device=DEV)
    checks = _decode_checks(cfg)
    rng = np.random.default_rng(cfg.seed + 98)
    rep = Report()
    written = np.zeros(M, bool)
    _say("full-size active-rows decode %s: %d steps" % (name, cfg.G))
    for t in range(cfg.G):
        h = synth.hidden(cfg, t, device=DEV)
        bs_before = bs.cpu().numpy() if t in checks else None
        msk_before = msk.cpu().numpy() if t in checks else None
        _binding.fork_step_ex(h, W, tok, msk, bs, BL, cfg.tau, conf, ent, logp, fb, B=B, L=L,
                              out_lse=lse, out_argmax=am, out_commit_pos=cp,
                              rows_mode=_binding.FORK_ROWS_ACTIVE)
        fbh = fb.cpu().numpy()
        cph = cp.cpu().numpy().reshape(B, BL)
        assert np.all(fbh == 1), "step %d: fallback %s" % (t, fbh)
        assert np.all(cph[:, 0] == P + t) and np.all(cph[:, 1:] == -1), "step %d: commits" % t
        if t not in checks:
            continue
        if Wb is None:
            Wb = host_bits(W)
        active = _active_rows(cfg, msk_before, bs_before)
        g = types.SimpleNamespace(conf=conf.cpu().numpy(), entropy=ent.cpu().numpy(),
                                  logp=logp.cpu().numpy(), lse=lse.cpu().numpy(),
                                  argmax=am.cpu().numpy())
        written |= ~np.isnan(g.conf)
        committed = np.arange(B) * L + P + t
        rows = np.union1d(committed, rng.choice(active, 16, replace=False))
        _say("active-rows decode %s step %d: oracle on %d rows" % (name, t, rows.size))
        ref = oracle.row_stats(host_bits(h), Wb, rows)
        compare_stats(g, ref, rows, host_bits(h), Wb, cfg.d, rep)
        assert np.array_equal(tok.cpu().numpy()[committed], g.argmax[committed])
    # only rows of some step's active block were ever written (the blocks of
    # the generation region); the prompt never
    assert not written.reshape(B, L)[:, :P].any()
    assert not msk.cpu().numpy().reshape(B, L)[:, P:].any()
    _say("full-size active-rows decode %s: %d rows checked (%d near-tie), max err %s" % (
        name, rep.rows, rep.near_tie_rows, {k: "%.2e" % v for k, v in rep.max_err.items()}))
    record(rep, name, steps=cfg.G, decode=True, rows_mode=1, tau=cfg.tau)
