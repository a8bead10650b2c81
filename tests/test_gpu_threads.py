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


def test_streams_get_their_own_managed_workspace():
    """Two non-default streams (default priority) issue steps of different
    sizes concurrently on the managed workspace, with no synchronisation
    between them: each stream has its own buffer, so every result equals the
    sequential run with a caller workspace, bit for bit."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(DEV)
    cases = [_case(10 + i, s) for i, s in enumerate(SHAPES)]
    refs = []
    for c in cases:
        ws = _own_workspace(c, _step)
        off = (-ws.data_ptr()) % 256
        refs.append([t.clone() for t in _step(c, ws[off:])])
    torch.cuda.synchronize()
    _binding.release()
    streams = [torch.cuda.Stream(DEV), torch.cuda.Stream(DEV)]
    outs = {0: [], 1: []}
    for rep in range(3):
        for si, st in enumerate(streams):
            with torch.cuda.stream(st):
                # stream 0 walks the sizes upwards (its buffer grows while
                # its earlier steps are queued), stream 1 downwards
                ci = rep if si == 0 else len(cases) - 1 - rep
                outs[si].append((ci, _step(cases[ci])))
    torch.cuda.synchronize()
    for si in (0, 1):
        for ci, out in outs[si]:
            for k, (a, b) in enumerate(zip(out, refs[ci])):
                assert torch.equal(a, b), "stream %d case %d output %d differs" % (si, ci, k)
    _binding.release()


# the refused call enqueues nothing, so the captured graph is empty
@pytest.mark.filterwarnings("ignore:The CUDA Graph is empty")
def test_graph_capture_needs_a_caller_workspace():
    """A step captured into a graph without a workspace of its own is
    refused (FORK_EINVAL) before anything is enqueued; with a caller
    workspace it is captured, and each replay (eager state resets and
    synchronisations in between) gives the eager result."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(DEV)
    case = _case(20, SHAPES[1])
    cfg, h, W, tok0, msk0, bs0, _ = case
    ws = _own_workspace(case, _step)
    off = (-ws.data_ptr()) % 256
    ref = [t.clone() for t in _step(case, ws[off:])]
    torch.cuda.synchronize()
    M, B = cfg.M, cfg.B
    f32 = dict(dtype=torch.float32, device=DEV)
    conf, ent, logp = (torch.empty(M, **f32) for _ in range(3))
    fb = torch.empty(B, dtype=torch.int32, device=DEV)
    tok, msk, bs = tok0.clone(), msk0.clone(), bs0.clone()

    def step(workspace):
        _binding.fork_step_ex(h, W, tok, msk, bs, cfg.block_len, float(cfg.tau), conf, ent,
                              logp, fb, B=B, L=cfg.L, workspace=workspace)

    refused = []
    g0 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g0):
        try:
            step(None)
        except _binding.ForkError as e:
            refused.append(e)
    assert refused and refused[0].code == _binding.FORK_EINVAL, refused
    assert "captured" in str(refused[0])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(ws[off:])
    torch.cuda.synchronize()
    for _ in range(3):
        tok.copy_(tok0)
        msk.copy_(msk0)
        bs.copy_(bs0)
        for t in (conf, ent, logp):
            t.fill_(float("nan"))
        fb.fill_(-9)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip([conf, ent, logp, fb, tok, msk, bs], ref)):
            assert torch.equal(a, b), "replay output %d differs from the eager step" % k
