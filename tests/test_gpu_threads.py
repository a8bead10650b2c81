"""Host-thread safety of the library-managed workspace: several threads call
fork_step and fork_logprob on one stream with different sizes, starting from
a released workspace so that the buffer grows while other threads' work is
queued.  Every result must equal, bit for bit, a sequential run of the same
call with a caller-provided workspace (the kernels are deterministic)."""
import threading

import pytest
import torch

from paper_2609_39859_amd import _binding, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")

# Sizes chosen so that each needs a larger workspace than the one before.
SHAPES = [
    dict(B=2, P=32, G=32, block_len=8, d=256, V=1024),
    dict(B=4, P=64, G=64, block_len=16, d=256, V=8192),
    dict(B=8, P=128, G=128, block_len=32, d=512, V=32000),
]


def _case(i, shape):
    cfg = synth.CONFIGS["mid"].with_(name="thread%d" % i, seed=101 + i, **shape)
    W = synth.weights(cfg).to(DEV)
    h = synth.hidden(cfg, 0).to(DEV)
    tok, msk, bs = synth.initial_state(cfg)
    g = torch.Generator().manual_seed(cfg.seed + 7)
    tgt = torch.randint(0, cfg.V, (cfg.M,), generator=g, dtype=torch.int64).to(torch.int32)
    return cfg, h, W, tok.to(DEV), msk.to(DEV), bs.to(DEV), tgt.to(DEV)


def _step(case, workspace=None):
    cfg, h, W, tok0, msk0, bs0, _ = case
    M, B = cfg.M, cfg.B
    tok, msk, bs = tok0.clone(), msk0.clone(), bs0.clone()
    f32 = dict(dtype=torch.float32, device=DEV)
    conf, ent, logp = (torch.empty(M, **f32) for _ in range(3))
    fb = torch.empty(B, dtype=torch.int32, device=DEV)
    _binding.fork_step_ex(h, W, tok, msk, bs, cfg.block_len, float(cfg.tau), conf, ent, logp, fb,
                          B=B, L=cfg.L, workspace=workspace)
    return [conf, ent, logp, fb, tok, msk, bs]


def _logprob(case, workspace=None):
    cfg, h, W, _, _, _, tgt = case
    q = torch.empty(cfg.M, dtype=torch.float32, device=DEV)
    _binding.logprob(h, W, tgt, q, workspace=workspace)
    return [q]


def _own_workspace(case, fn):
    cfg = case[0]
    n = (_binding.workspace_bytes(cfg.B, cfg.L, cfg.V) if fn is _step
         else _binding.logprob_workspace_bytes(cfg.M, cfg.V))
    return torch.empty(n + 256, dtype=torch.uint8, device=DEV)


def test_threads_share_managed_workspace():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(DEV)
    cases = [_case(i, s) for i, s in enumerate(SHAPES)]
    refs = {}
    for i, c in enumerate(cases):
        for fn in (_step, _logprob):
            ws = _own_workspace(c, fn)
            off = (-ws.data_ptr()) % 256
            refs[(i, fn.__name__)] = [t.clone() for t in fn(c, ws[off:])]
    torch.cuda.synchronize()
    _binding.release()

    results, errors = [], []
    lock = threading.Lock()
    start = threading.Barrier(len(cases))

    def worker(i):
        try:
            torch.cuda.set_device(DEV)
            start.wait()
            # largest case first on some threads, so growth happens while
            # smaller calls of other threads are queued
            order = (_step, _logprob) if i % 2 == 0 else (_logprob, _step)
            for rep in range(4):
                for fn in order:
                    out = fn(cases[(i + rep) % len(cases)])
                    with lock:
                        results.append(((i + rep) % len(cases), fn.__name__, out))
        except Exception as e:  # reported after join
            with lock:
                errors.append(repr(e))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    assert len(results) == len(cases) * 4 * 2
    for ci, name, out in results:
        ref = refs[(ci, name)]
        for k, (a, b) in enumerate(zip(out, ref)):
            assert torch.equal(a, b), "case %d %s output %d differs from the sequential run" % (ci, name, k)
    _binding.release()
