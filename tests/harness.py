"""Shared helpers of the GPU parity tests: run one step through the C ABI,
run the oracle on the same input bits, and compare.

Comparison rules (the bar of the parity tests):
* confidence, entropy and log-probability: |gpu - oracle| <= STAT_TOL;
* candidate token: identical, except at near-ties, where the oracle's top-2
  logit gap is below GAP_TOL; there the GPU's candidate must be a valid
  maximiser (its exact logit within GAP_TOL of the maximum), and the row is
  counted as excluded;
* decisions (tokens, mask, block_start, fallback flag, commit count): bit
  exact per sequence, except sequences whose active block holds a masked
  position with |conf - lambda| < THRESH_TOL; there the GPU's decision must
  be the rule applied to its own confidences, and the sequence is counted as
  excluded.

GAP_TOL: products of bf16 (or fp32) inputs accumulate in fp32 over d terms;
with |partial sums| up to ~10 the rounding error of one logit is below
d * 2^-24 * 10 = 2.4e-3 at d = 4096 in the worst case and ~4e-5 typically, so
two logits closer than 2e-3 (5e-3 for d > 4096) may legitimately swap.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

import oracle
from paper_2609_39859_amd import _binding, synth

STAT_TOL = 2e-3
THRESH_TOL = 1e-4


def gap_tol(d: int) -> float:
    return 2e-3 if d <= 4096 else 5e-3


@dataclasses.dataclass
class GpuOut:
    conf: np.ndarray
    entropy: np.ndarray
    logp: np.ndarray
    lse: np.ndarray
    argmax: np.ndarray
    tokens: np.ndarray
    mask: np.ndarray
    block_start: np.ndarray
    fallback: np.ndarray
    ncommit: np.ndarray
    commit_pos: np.ndarray


def gpu_step(h_dev, W_dev, tokens, mask, block_start, B, L, block_len, tau,
             rule=_binding.FORK_RULE_LEFTMOST, workspace=None, uniform=None,
             rows_mode=_binding.FORK_ROWS_ALL, temperature=0.0, seed=0, counter=0) -> GpuOut:
    """One step through fork_step_ex on the device of h_dev; host inputs for
    the state, host copies of every output.  Per-position outputs start as
    NaN (statistics) and -7 (candidates), so rows a step leaves untouched are
    visible."""
    dev = h_dev.device
    M = B * L
    tok = torch.as_tensor(np.asarray(tokens, np.int32)).to(dev)
    msk = torch.as_tensor(np.asarray(mask, np.uint8)).to(dev)
    bs = torch.as_tensor(np.asarray(block_start, np.int32)).to(dev)
    f32 = dict(dtype=torch.float32, device=dev)
    i32 = dict(dtype=torch.int32, device=dev)
    conf, ent, logp, lse = (torch.full((M,), float("nan"), **f32) for _ in range(4))
    am = torch.full((M,), -7, **i32)
    fb = torch.full((B,), -9, **i32)
    nc = torch.full((B,), -9, **i32)
    cp = torch.full((B * block_len,), -9, **i32)
    uni = None if uniform is None else torch.as_tensor(np.asarray(uniform, np.float32)).to(dev)
    _binding.fork_step_ex(h_dev, W_dev, tok, msk, bs, block_len, tau, conf, ent, logp, fb,
                          B=B, L=L, out_lse=lse, out_argmax=am, out_ncommit=nc,
                          out_commit_pos=cp, rule=rule, workspace=workspace,
                          fallback_uniform=uni, rows_mode=rows_mode,
                          temperature=temperature, seed=seed, counter=counter)
    torch.cuda.synchronize(dev)
    c = lambda t: t.cpu().numpy()
    return GpuOut(c(conf), c(ent), c(logp), c(lse), c(am), c(tok), c(msk), c(bs), c(fb),
                  c(nc), c(cp).reshape(B, block_len))


def exact_logit(hbits, Wbits, r, v) -> float:
    """<h_r, W_v> in binary64 from the stored bits (numpy dot, for validating
    a near-tie candidate)."""
    def f64(x):
        if x.dtype == np.uint16:
            return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        return x.astype(np.float64)
    return float(np.dot(f64(hbits[r]), f64(Wbits[v])))


@dataclasses.dataclass
class Report:
    rows: int = 0
    near_tie_rows: int = 0
    seqs: int = 0
    near_threshold_seqs: int = 0
    max_err: dict = dataclasses.field(default_factory=dict)


# Exclusion counts of every parity check run in this session (written out by
# tests/conftest.py at the end of the session).
RECORDS = []


def record(rep: Report, config: str, **extra) -> None:
    """Keep the counts of one parity check: rows compared and how many were
    near-ties, sequence-steps compared and how many sat near the threshold,
    the largest errors; labelled with the running test."""
    import os
    test = os.environ.get("PYTEST_CURRENT_TEST", "?").rsplit(" ", 1)[0]
    RECORDS.append(dict(test=test, config=config, rows=rep.rows,
                        near_tie_rows=rep.near_tie_rows, seqs=rep.seqs,
                        near_threshold_seqs=rep.near_threshold_seqs,
                        max_err={k: float(v) for k, v in sorted(rep.max_err.items())},
                        **extra))


def compare_stats(g: GpuOut, ref: dict, rows, hbits, Wbits, d: int, rep: Report):
    rows = np.asarray(rows)
    for k in ("conf", "entropy", "logp", "lse"):
        gv = getattr(g, k)[rows].astype(np.float64)
        ov = ref[k]
        err = np.abs(gv - ov)
        if k == "lse":
            err = err / np.maximum(1.0, np.abs(ov))  # relative for the normaliser
        rep.max_err[k] = max(rep.max_err.get(k, 0.0), float(err.max()) if err.size else 0.0)
        bad = np.nonzero(~(err <= STAT_TOL))[0]
        assert bad.size == 0, "%s: %d rows off, e.g. row %d gpu %r oracle %r" % (
            k, bad.size, rows[bad[0]], gv[bad[0]], ov[bad[0]])
    gt = gap_tol(d)
    ga = g.argmax[rows]
    mism = np.nonzero(ga != ref["argmax"])[0]
    for i in mism:
        r = int(rows[i])
        assert ref["gap"][i] < gt, "row %d: candidate %d vs oracle %d (gap %g)" % (
            r, ga[i], ref["argmax"][i], ref["gap"][i])
        zmax = exact_logit(hbits, Wbits, r, int(ref["argmax"][i]))
        zg = exact_logit(hbits, Wbits, r, int(ga[i]))
        assert zmax - zg <= gt, "row %d: candidate %d is not a maximiser" % (r, ga[i])
    rep.rows += rows.size
    rep.near_tie_rows += int(mism.size)
    return rows[mism]


def key_tol(d: int, temperature: float) -> float:
    """Two Gumbel keys closer than this may be ordered either way: the logit
    error (GAP_TOL) scaled by 1/temperature, plus binary32 rounding of the
    perturbation (|log E| < 17, relative error ~1e-7)."""
    return gap_tol(d) / temperature + 1e-4


def oracle_key(hbits, Wbits, r, v, temperature, seed, counter) -> float:
    """The oracle's Gumbel key of vocabulary entry v at row r."""
    e, _ = oracle.exp_draw(seed, counter, r, v)
    return exact_logit(hbits, Wbits, r, v) / temperature - float(np.log(e))


def compare_sampled(g: GpuOut, st: dict, sm: dict, rows, hbits, Wbits, d: int,
                    temperature: float, seed: int, counter: int, rep: Report):
    """Rows whose candidates are drawn: entropy and log-normaliser against
    the oracle's statistics `st`; the drawn token against the oracle's draw
    `sm` (identical, or both within key_tol of the best key when the
    oracle's top-2 key gap is below it); confidence and log-probability
    against the oracle's untempered q of the GPU's token.  Returns the rows
    whose token differs."""
    rows = np.asarray(rows)
    for k in ("entropy", "lse"):
        gv = getattr(g, k)[rows].astype(np.float64)
        err = np.abs(gv - st[k])
        if k == "lse":
            err = err / np.maximum(1.0, np.abs(st[k]))
        rep.max_err[k] = max(rep.max_err.get(k, 0.0), float(err.max()) if err.size else 0.0)
        assert np.all(err <= STAT_TOL), "%s off on drawn rows (max %g)" % (k, err.max())
    kt = key_tol(d, temperature)
    ga = g.argmax[rows]
    logq = sm["logp"].copy()
    mism = np.nonzero(ga != sm["cand"])[0]
    for i in mism:
        r = int(rows[i])
        assert sm["keygap"][i] < kt, "row %d: drawn %d vs oracle %d (key gap %g)" % (
            r, ga[i], sm["cand"][i], sm["keygap"][i])
        kbest = oracle_key(hbits, Wbits, r, int(sm["cand"][i]), temperature, seed, counter)
        kg = oracle_key(hbits, Wbits, r, int(ga[i]), temperature, seed, counter)
        assert kbest - kg <= kt, "row %d: drawn %d is not a maximiser of the keys" % (r, ga[i])
        logq[i] = exact_logit(hbits, Wbits, r, int(ga[i])) - st["lse"][i]
    for k, ref in (("conf", np.exp(logq)), ("logp", logq)):
        gv = getattr(g, k)[rows].astype(np.float64)
        err = np.abs(gv - ref)
        rep.max_err[k] = max(rep.max_err.get(k, 0.0), float(err.max()) if err.size else 0.0)
        bad = np.nonzero(~(err <= STAT_TOL))[0]
        assert bad.size == 0, "%s: %d drawn rows off, e.g. row %d gpu %r oracle %r" % (
            k, bad.size, rows[bad[0]], gv[bad[0]], ref[bad[0]])
    rep.rows += rows.size
    rep.near_tie_rows += int(mism.size)
    return rows[mism]


def check_rule_on_own_stats(g: GpuOut, tokens, mask, block_start, B, L, BL, tau, rule, seqs,
                            uniform=None):
    """Property check, for decisions that sit on the threshold: the GPU's
    commits are exactly what the rule gives on the GPU's own binary32
    confidences (committed set inside the active block; all masked positions
    with conf > tau there, else exactly one: the leftmost masked, or for the
    max-confidence rule one of maximal confidence, lowest position)."""
    t32 = np.float32(tau)
    for b in seqs:
        base = b * L
        masked = [k for k in range(int(block_start[b]), L) if mask[base + k]]
        committed = [k for k in range(L) if mask[base + k] and not g.mask[base + k]]
        assert all(g.tokens[base + k] == g.argmax[base + k] for k in committed)
        untouched = [k for k in range(L) if k not in committed]
        assert np.array_equal(g.tokens[base + np.array(untouched, int)],
                              np.asarray(tokens)[base + np.array(untouched, int)])
        if not masked:
            assert g.fallback[b] == -1 and not committed
            continue
        s = int(block_start[b]) + ((masked[0] - int(block_start[b])) // BL) * BL
        blk = [k for k in masked if k < s + BL]
        assert g.block_start[b] == s
        passing = [k for k in blk if np.float32(g.conf[base + k]) > t32]
        if passing:
            assert g.fallback[b] == 0 and committed == passing
        else:
            assert g.fallback[b] == 1 and len(committed) == 1
            if rule == _binding.FORK_RULE_LEFTMOST:
                assert committed == [blk[0]]
            elif rule == _binding.FORK_RULE_RANDOM:
                j = min(int(np.float32(uniform[b]) * np.float32(len(blk))), len(blk) - 1)
                assert committed == [blk[j]]
            else:
                key = {_binding.FORK_RULE_MAXCONF: g.conf, _binding.FORK_RULE_MINCONF: -g.conf,
                       _binding.FORK_RULE_MAXENT: g.entropy}[rule]
                best = max(key[base + k] for k in blk)
                assert committed == [min(k for k in blk if key[base + k] == best)]
        assert g.ncommit[b] == len(committed)


# Fallback keys closer than this (oracle values) may be ordered either way by
# the GPU's binary32 statistics: the lowest-confidence / highest-entropy pick
# is then excluded from the exact comparison (and checked on the GPU's own
# statistics instead).
KEY_TIE_TOL = {2: 1e-5, 3: 1e-4}


def compare_decisions(g: GpuOut, sel, conf_ref, tokens, mask, block_start, B, L, BL,
                      tau, rep: Report, seqs=None, rule=0, near_tie_rows=(),
                      entropy_ref=None, uniform=None, tie_seqs_excluded=False):
    """sel = oracle select output on oracle confidences and candidates.
    With tie_seqs_excluded, a sequence whose active block holds a near-tie
    row is excluded too (a drawn token that differs carries a different
    confidence, so the threshold decision may legitimately differ)."""
    tok_o, msk_o, bs_o, fb_o, nc_o = sel
    lam = float(np.float32(tau))
    seqs = list(range(B) if seqs is None else seqs)
    # GPU decisions always agree with the rule on its own statistics
    check_rule_on_own_stats(g, tokens, mask, block_start, B, L, BL, tau, rule, seqs, uniform)
    tie = set(int(r) for r in near_tie_rows)
    for b in seqs:
        sl = slice(b * L, (b + 1) * L)
        rep.seqs += 1
        s = int(bs_o[b])
        near = False
        if fb_o[b] != -1:
            e = min(s + BL, L)
            blk = [k for k in range(s, e) if mask[b * L + k]]
            near = any(abs(conf_ref[b * L + k] - lam) < THRESH_TOL for k in blk)
            if fb_o[b] == 1 and rule in KEY_TIE_TOL and len(blk) > 1:
                key = np.array([conf_ref[b * L + k] if rule == 2 else entropy_ref[b * L + k]
                                for k in blk])
                srt = np.sort(key)
                gap = srt[1] - srt[0] if rule == 2 else srt[-1] - srt[-2]
                near = near or gap < KEY_TIE_TOL[rule]
        if tie_seqs_excluded and fb_o[b] != -1:
            near = near or any(b * L + k in tie for k in range(s, min(s + BL, L)))
        if near:
            rep.near_threshold_seqs += 1
            continue
        assert g.fallback[b] == fb_o[b], "seq %d fallback gpu %d oracle %d" % (b, g.fallback[b], fb_o[b])
        assert g.block_start[b] == bs_o[b]
        assert g.ncommit[b] == nc_o[b]
        assert np.array_equal(g.mask[sl], msk_o[sl]), "seq %d mask differs" % b
        diff = np.nonzero(g.tokens[sl] != tok_o[sl])[0] + b * L
        assert all(int(k) in tie for k in diff), "seq %d tokens differ at %s" % (b, diff[:8])
        committed = sorted(k - b * L for k in range(b * L, (b + 1) * L) if mask[k] and not msk_o[k])
        cp = [int(x) for x in g.commit_pos[b] if x >= 0]
        assert cp == committed and all(x == -1 for x in g.commit_pos[b][len(cp):])


def host_bits(t: torch.Tensor):
    return synth.to_bits(t)
