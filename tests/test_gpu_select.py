"""GPU parity of the unmasking rule on its own (fork_select, Algorithm 2 and
the fallback rules of Algorithm 1 and Section 4.1): both kernel paths (one
wave per sequence, and one lane per sequence for large batches of short
blocks) against the oracle, bit for bit (both sides decide on the same
binary32 confidences)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_39859_amd import _binding

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _state(B, L, V, seed):
    rng = np.random.default_rng(seed)
    M = B * L
    conf = rng.random(M).astype(np.float32)
    conf[rng.random(M) < 0.1] = np.float32(0.9)           # values on the threshold
    ent = np.round(rng.random(M) * 4, 2).astype(np.float32)  # frequent ties
    am = rng.integers(0, V, M).astype(np.int32)
    msk = (rng.random(M) < 0.5).astype(np.uint8)
    tok = np.where(msk, -1, rng.integers(0, V, M)).astype(np.int32)
    bs = rng.integers(0, L + 1, B).astype(np.int32)
    msk[(B - 1) * L:] = 0                                  # an idle sequence
    uni = rng.random(B).astype(np.float32)
    return conf, ent, am, tok, msk, bs, uni


def _pm(x, B, L):
    """Row-major [B*L] -> position-major [L*B] (position k of sequence b at
    k*B + b)."""
    return np.ascontiguousarray(np.asarray(x).reshape(B, L).T).reshape(-1)


def _rm(x, B, L):
    return np.ascontiguousarray(np.asarray(x).reshape(L, B).T).reshape(-1)


def _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, tau, rule,
         layout=_binding.FORK_LAYOUT_ROW_MAJOR, outputs="all"):
    """fork_select on row-major host state; with the position-major layout
    the per-position arrays are transposed for the call and back after it,
    so the results compare directly.  outputs: "all" asks for the commit
    counts and positions, "ncommit" for the counts only, "none" for
    neither (their slots then come back as -9)."""
    t = lambda x: torch.as_tensor(np.ascontiguousarray(x), device=DEV)
    pm = layout == _binding.FORK_LAYOUT_POSITION_MAJOR
    lay = (lambda x: _pm(x, B, L)) if pm else (lambda x: x)
    tok_d, msk_d, bs_d = t(lay(tok).copy()), t(lay(msk).copy()), t(bs.copy())
    fb = torch.full((B,), -9, dtype=torch.int32, device=DEV)
    nc = torch.full((B,), -9, dtype=torch.int32, device=DEV)
    cp = torch.full((B * BL,), -9, dtype=torch.int32, device=DEV)
    _binding.select(t(lay(conf)), t(lay(am)), tok_d, msk_d, bs_d, BL, tau, fb, B=B, L=L,
                    rule=rule, entropy=t(lay(ent)), uniform=t(uni),
                    out_ncommit=nc if outputs in ("all", "ncommit") else None,
                    out_commit_pos=cp if outputs == "all" else None, layout=layout)
    torch.cuda.synchronize()
    back = (lambda x: _rm(x, B, L)) if pm else (lambda x: x)
    return (back(tok_d.cpu().numpy()), back(msk_d.cpu().numpy()), bs_d.cpu().numpy(),
            fb.cpu().numpy(), nc.cpu().numpy(), cp.cpu().numpy().reshape(B, BL))


SHAPES = [
    # B, L, block_len   (B >= 4096 with block_len <= 64 takes the lane path)
    (5, 61, 7), (37, 300, 300), (4096, 40, 8), (5000, 64, 64), (4100, 33, 32),
    (4096, 100, 65), (4097, 1, 1),
    # lane path with 16-byte aligned rows and blocks <= 32 (wide loads)
    (4096, 32, 32), (4096, 64, 16), (8192, 96, 32), (4096, 48, 8),
]


PM_SHAPES = [
    # position-major: B % 4 == 0 with shared block starts takes the wide path
    (5, 61, 7), (6, 33, 32), (4096, 32, 32), (4096, 64, 16), (4100, 40, 8), (4099, 33, 32),
    (8, 100, 65), (4097, 1, 1), (1024, 48, 33),
]


@pytest.mark.parametrize("B,L,BL", SHAPES)
@pytest.mark.parametrize("rule", [0, 1, 2, 3, 4])
def test_select_matches_oracle(B, L, BL, rule):
    _check_against_oracle(B, L, BL, rule, _binding.FORK_LAYOUT_ROW_MAJOR)


@pytest.mark.parametrize("B,L,BL", PM_SHAPES)
@pytest.mark.parametrize("rule", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("shared_start", [False, True])
def test_select_position_major_matches_oracle(B, L, BL, rule, shared_start):
    """The position-major layout against the oracle (on the transposed
    state), with random block starts and with every sequence at the same
    block start (the wide path)."""
    _check_against_oracle(B, L, BL, rule, _binding.FORK_LAYOUT_POSITION_MAJOR, shared_start)


def _check_against_oracle(B, L, BL, rule, layout, shared_start=False):
    _need_gpu()
    conf, ent, am, tok, msk, bs, uni = _state(B, L, 1000, B * 31 + L + BL + rule)
    if shared_start:
        bs[:] = min(L - BL, 3)
    for tau in (0.3, 0.9):
        g = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, tau, rule, layout)
        o = oracle.select_ex(conf, am, tok, msk, bs, B, L, BL, float(np.float32(tau)), rule,
                             entropy=ent, uniform=uni)
        for k, (x, y) in enumerate(zip(g[:5], o)):
            assert np.array_equal(x, y), ("tokens", "mask", "block_start", "fallback", "ncommit")[k]
        # compacted commits: the positions the oracle unmasked, ascending
        for b in range(B):
            sl = slice(b * L, (b + 1) * L)
            done = np.nonzero(msk[sl] & ~o[1][sl])[0]
            assert np.array_equal(g[5][b, :done.size], done)
            assert np.all(g[5][b, done.size:] == -1)


@pytest.mark.parametrize("B,L,BL", [(4096, 32, 32), (4096, 64, 16), (8192, 48, 8),
                                    (4160, 64, 32)])
@pytest.mark.parametrize("rule", [0, 4, 1])
@pytest.mark.parametrize("outputs", ["all", "none"])
def test_row_major_whole_wave_blocks(B, L, BL, rule, outputs):
    """Row-major batches whose blocks start on multiples of 16 positions
    with 32 positions left in the row (the lane path's wide loads), every
    other wave with one sequence off that grid (its position-by-position
    path) and the last sequence idle, under the threshold, leftmost, random
    and highest-confidence rules, with and without the commit outputs.
    Against the oracle, bit for bit."""
    _need_gpu()
    conf, ent, am, tok, msk, bs, uni = _state(B, L, 1000, B + 7 * L + BL + rule)
    rng = np.random.default_rng(B + L + BL)
    bs[:] = rng.choice(np.arange(0, L - 32 + 1, 16), B)
    for w in range(1, B // 64, 2):
        bs[64 * w + 5] = min(bs[64 * w + 5] + 1, L)
    for tau in (0.3, 0.9):
        g = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, tau, rule, outputs=outputs)
        o = oracle.select_ex(conf, am, tok, msk, bs, B, L, BL, float(np.float32(tau)), rule,
                             entropy=ent, uniform=uni)
        n = 5 if outputs == "all" else 4
        for k, (x, y) in enumerate(zip(g[:n], o[:n])):
            assert np.array_equal(x, y), ("tokens", "mask", "block_start", "fallback", "ncommit")[k]
        if outputs == "all":
            for b in range(0, B, 97):
                sl = slice(b * L, (b + 1) * L)
                done = np.nonzero(msk[sl] & ~o[1][sl])[0]
                assert np.array_equal(g[5][b, :done.size], done)
                assert np.all(g[5][b, done.size:] == -1)


def test_lane_and_wave_paths_agree():
    """The first sequences of a large batch (lane path) and the same
    sequences run as a small batch (wave path) give identical results."""
    _need_gpu()
    B, L, BL = 4096, 64, 32
    conf, ent, am, tok, msk, bs, uni = _state(B, L, 500, 7)
    for rule in range(5):
        big = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, 0.5, rule)
        n = 64
        small = _run(conf[:n * L], ent[:n * L], am[:n * L], tok[:n * L], msk[:n * L], bs[:n],
                     uni[:n], n, L, BL, 0.5, rule)
        for x, y in zip(big, small):
            assert np.array_equal(x.reshape(-1)[:y.size], y.reshape(-1))


@pytest.mark.parametrize("B", [3, 4096])
def test_bad_block_start_reported_in_data_on_both_paths(B):
    _need_gpu()
    L, BL = 16, 4
    conf, ent, am, tok, msk, bs, uni = _state(B, L, 100, 3)
    msk[:] = 1
    bs[:] = 0
    bs[0], bs[1] = -1, L + 1
    bs[2] = L                           # nothing at or after the start: idle
    g = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, 0.5, 0)
    assert g[3][:3].tolist() == [-2, -2, -1]
    assert np.all(g[1][:3 * L] == 1) and np.all(g[4][:3] == 0) and np.all(g[5][:3] == -1)


@pytest.mark.parametrize("B", [1 << 16, 1 << 18])
@pytest.mark.parametrize("outputs", ["all", "none"])
def test_position_major_sweep_shape_matches_row_major(B, outputs):
    """The benchmark's sweep shape (blocks of 32 positions, one block per
    sequence, every sequence falling back), 2^16 sequences (one per lane)
    and 2^18 (four per lane): position-major and row-major give the same
    decisions, and every sequence commits its leftmost masked position."""
    _need_gpu()
    L, BL = 32, 32
    rng = np.random.default_rng(11)
    conf = (rng.random(B * L) * 0.03).astype(np.float32)
    am = rng.integers(0, 126464, B * L).astype(np.int32)
    tok = np.full(B * L, -1, np.int32)
    msk = np.ones(B * L, np.uint8)
    msk.reshape(B, L)[:, :5] = 0
    bs = np.zeros(B, np.int32)
    ent = np.zeros(B * L, np.float32)
    uni = np.zeros(B, np.float32)
    a = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, 0.9, 0, outputs=outputs)
    b = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, 0.9, 0,
             _binding.FORK_LAYOUT_POSITION_MAJOR, outputs=outputs)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    assert np.all(a[3] == 1)
    if outputs == "all":
        assert np.all(a[5][:, 0] == 5) and np.all(a[5][:, 1:] == -1)
    assert np.array_equal(a[0].reshape(B, L)[:, 5], am.reshape(B, L)[:, 5])
    assert np.all(a[1].reshape(B, L)[:, :6] == 0) and np.all(a[1].reshape(B, L)[:, 6:] == 1)


@pytest.mark.parametrize("B,L,BL", [((1 << 18), 40, 32), ((1 << 18) + 2, 33, 16),
                                    ((1 << 18), 20, 20)])
@pytest.mark.parametrize("rule", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("outputs", ["all", "ncommit", "none"])
def test_position_major_large_batches_match_row_major(B, L, BL, rule, outputs):
    """Batches large enough for four sequences per lane (and one not a
    multiple of four): random states, half of them sharing a block start,
    position-major against row-major (itself checked against the oracle).
    Without the commit positions, groups of four sequences that commit one
    position each, the same one, take the vector commit."""
    _need_gpu()
    conf, ent, am, tok, msk, bs, uni = _state(B, L, 1000, B + L + BL + rule)
    bs[: B // 2] = min(L - BL, 2)
    # a quarter of the sequences: one masked position, the same in each group
    # of four, so the vector commit runs for every rule
    q = B // 4
    msk.reshape(B, L)[:q] = 0
    msk.reshape(B, L)[:q, min(L - BL, 2) + 1] = 1
    for tau in (0.3, 0.9):
        a = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, tau, rule, outputs=outputs)
        b = _run(conf, ent, am, tok, msk, bs, uni, B, L, BL, tau, rule,
                 _binding.FORK_LAYOUT_POSITION_MAJOR, outputs=outputs)
        for k, (x, y) in enumerate(zip(a, b)):
            assert np.array_equal(x, y), k
        if outputs != "all":
            assert np.all(a[5] == -9) and (outputs == "ncommit" or np.all(a[4] == -9))
