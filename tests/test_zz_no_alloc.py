"""fork_step_noalloc (the entry point for callers that cannot allocate
device memory) through the C ABI against fork_step_ex with a caller
workspace: the same kernels, so every output must agree bit for bit.  Calls
follow one another on one stream with shrinking inputs, so the second and
later calls find the static scratch holding the previous call's contents."""
import numpy as np
import pytest
import torch

from paper_2609_39859_amd import _binding, synth

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _inputs(cfg, step):
    W = synth.weights(cfg, device=DEV)
    h = synth.hidden(cfg, step, device=DEV, W=W if cfg.plant_peaks > 0 else None)
    tok, msk, bs = (x.to(DEV) for x in synth.initial_state(cfg))
    return W, h, tok, msk, bs


def _run(fn, cfg, W, h, tok0, msk0, bs0, **kw):
    """One step by `fn` on copies of the state; returns every output."""
    M, B, BL = cfg.M, cfg.B, cfg.block_len
    tok, msk, bs = tok0.clone(), msk0.clone(), bs0.clone()
    f32 = dict(dtype=torch.float32, device=DEV)
    i32 = dict(dtype=torch.int32, device=DEV)
    conf, ent, logp, lse = (torch.full((M,), float("nan"), **f32) for _ in range(4))
    am = torch.full((M,), -7, **i32)
    fb, nc = torch.full((B,), -9, **i32), torch.full((B,), -9, **i32)
    cp = torch.full((B * BL,), -9, **i32)
    print("no-alloc: %s %s B=%d L=%d d=%d V=%d %s" % (fn.__name__, cfg.name, B, cfg.L, cfg.d,
                                                        cfg.V, kw), flush=True)
    fn(h, W, tok, msk, bs, BL, cfg.tau, conf, ent, logp, fb, B=B, L=cfg.L, out_lse=lse,
       out_argmax=am, out_ncommit=nc, out_commit_pos=cp, **kw)
    torch.cuda.synchronize()
    return dict(conf=conf, entropy=ent, logp=logp, lse=lse, argmax=am, fallback=fb,
                ncommit=nc, commit_pos=cp, tokens=tok, mask=msk, block_start=bs)


def _with_workspace(cfg, **kw):
    nbytes = _binding.workspace_bytes(cfg.B, cfg.L, cfg.V)
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=DEV)
    off = (-buf.data_ptr()) % 256
    ws = buf[off:off + nbytes]

    def fork_step_ex(*a, **k):
        _binding.fork_step_ex(*a, workspace=ws, **k)
    return fork_step_ex


def _same(a, b, what):
    for k in a:
        x, y = a[k].cpu(), b[k].cpu()
        if x.dtype == torch.float32:
            x, y = x.view(torch.int32), y.view(torch.int32)
        assert torch.equal(x, y), "%s: %s differs from fork_step_ex" % (what, k)


# (config, options): each call smaller than the one before it
CALLS = [
    (synth.CONFIGS["mid"], {}),
    (synth.CONFIGS["grpo_small"], dict(rows_mode=_binding.FORK_ROWS_ACTIVE, temperature=0.8,
                                       seed=0x5EED, counter=3)),
    (synth.CONFIGS["tiny_peaked"], dict(rule=_binding.FORK_RULE_MAXCONF)),
]


def test_noalloc_matches_fork_step_ex_on_successive_calls():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(DEV)
    sizes = []
    for i, (cfg, kw) in enumerate(CALLS):
        W, h, tok, msk, bs = _inputs(cfg, i)
        got = _run(_binding.fork_step_noalloc, cfg, W, h, tok, msk, bs, **kw)
        ref = _run(_with_workspace(cfg), cfg, W, h, tok, msk, bs, **kw)
        _same(got, ref, "call %d (%s)" % (i, cfg.name))
        # the step did something: some position committed, statistics finite
        assert int((got["ncommit"] > 0).sum()) > 0
        assert bool(torch.isfinite(got["entropy"]).any())
        sizes.append(cfg.M * ((cfg.V + 255) // 256))
    assert sizes == sorted(sizes, reverse=True)


def test_noalloc_at_the_llada8b_shape():
    """The benchmark's shape (B*L = 4096, d = 4096, V = 126464) fits the
    scratch: bit-identical to fork_step_ex, twice in a row."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = synth.CONFIGS["llada8b"]
    W, h, tok, msk, bs = _inputs(cfg, 0)
    ref = _run(_with_workspace(cfg), cfg, W, h, tok, msk, bs)
    for rep in range(2):
        got = _run(_binding.fork_step_noalloc, cfg, W, h, tok, msk, bs)
        _same(got, ref, "llada8b call %d" % rep)
    assert torch.all(ref["fallback"] == 1)


def test_noalloc_rejects_what_does_not_fit():
    """Sizes beyond the scratch maximum and a caller workspace are refused
    before anything is enqueued, leaving the outputs untouched."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = synth.CONFIGS["mid"]
    W, h, tok, msk, bs = _inputs(cfg, 0)
    # 512 vocabulary tiles x 8192 positions x 16 B > 64 MiB
    big = cfg.with_(B=32, P=128, G=128)
    assert big.M * 125 * 16 <= _binding.FORK_NOALLOC_SCRATCH_BYTES  # fits at V = 32000 ...
    Vb = 131072
    Wb = torch.zeros(Vb, cfg.d, dtype=torch.bfloat16, device=DEV)
    hb = torch.zeros(big.M, cfg.d, dtype=torch.bfloat16, device=DEV)
    f32 = dict(dtype=torch.float32, device=DEV)
    conf, ent, logp = (torch.full((big.M,), 5.0, **f32) for _ in range(3))
    fb = torch.full((big.B,), -9, dtype=torch.int32, device=DEV)
    t = torch.zeros(big.M, dtype=torch.int32, device=DEV)
    m = torch.ones(big.M, dtype=torch.uint8, device=DEV)
    s = torch.full((big.B,), big.P, dtype=torch.int32, device=DEV)
    with pytest.raises(_binding.ForkError) as e:   # ... but not at V = 131072
        _binding.fork_step_noalloc(hb, Wb, t, m, s, big.block_len, 0.9, conf, ent, logp, fb,
                                   B=big.B, L=big.L)
    assert e.value.code == _binding.FORK_EUNSUPPORTED and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool(torch.all(conf == 5.0)) and bool(torch.all(fb == -9)) and bool(torch.all(m == 1))
    a = _binding._step_args(h, W, tok, msk, bs, cfg.block_len, cfg.tau, conf[:cfg.M],
                            ent[:cfg.M], logp[:cfg.M], fb[:cfg.B], cfg.B, cfg.L, None, None,
                            None, None, 0, None, None, None, None, 0, 0.0, 0, 0)
    a.workspace = Wb.data_ptr()
    a.workspace_bytes = 1 << 20
    import ctypes
    assert _binding.lib().fork_step_noalloc(ctypes.byref(a)) == _binding.FORK_EINVAL


def test_noalloc_under_graph_capture():
    """The callers it is for: a step captured into a HIP graph (after a first
    call on the device has looked up the scratch address).  Every replay,
    with eager state resets and synchronisations between them, gives the
    eager fork_step_ex result bit for bit."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(DEV)
    cfg = synth.CONFIGS["mid"]
    W, h, tok0, msk0, bs0 = _inputs(cfg, 2)
    ref = _run(_with_workspace(cfg), cfg, W, h, tok0, msk0, bs0)
    _run(_binding.fork_step_noalloc, cfg, W, h, tok0, msk0, bs0)  # first call on the device
    M, B, BL = cfg.M, cfg.B, cfg.block_len
    tok, msk, bs = tok0.clone(), msk0.clone(), bs0.clone()
    f32 = dict(dtype=torch.float32, device=DEV)
    i32 = dict(dtype=torch.int32, device=DEV)
    conf, ent, logp, lse = (torch.empty(M, **f32) for _ in range(4))
    am = torch.empty(M, **i32)
    fb, nc = torch.empty(B, **i32), torch.empty(B, **i32)
    cp = torch.empty(B * BL, **i32)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _binding.fork_step_noalloc(h, W, tok, msk, bs, BL, cfg.tau, conf, ent, logp, fb, B=B,
                                   L=cfg.L, out_lse=lse, out_argmax=am, out_ncommit=nc,
                                   out_commit_pos=cp)
    torch.cuda.synchronize()
    for rep in range(3):
        tok.copy_(tok0)
        msk.copy_(msk0)
        bs.copy_(bs0)
        for t in (conf, ent, logp, lse):
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = dict(conf=conf, entropy=ent, logp=logp, lse=lse, argmax=am, fallback=fb,
                   ncommit=nc, commit_pos=cp, tokens=tok, mask=msk, block_start=bs)
        _same(got, ref, "graph replay %d" % rep)
