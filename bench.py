"""Benchmark of the Fork-dLLM denoising step on one MI355X.

A step is one fork_step call (LM-head GEMM with the fused per-tile
statistics, the cross-tile merge, and the per-sequence selection) over one
batch of synthetic hidden states already resident in HBM.  The workload is
the LLaDA-8B-shaped configuration: B=8 sequences of L=512 positions
(256 prompt + 256 generation), block length 32, d=4096, V=126464, bf16
inputs with fp32 accumulation, threshold 0.9.

Prints ONE JSON line.  `value` is denoising steps per second; positions per
second (B*L rows through the LM head) is reported beside it.  `roofline`
covers the dominant kernel (the LM-head GEMM + statistics), timed with HIP
events recorded around that kernel alone on the stream it runs on.
`cpu_baseline` times the binary64 CPU oracle on a bounded sample of rows of
the same workload and scales it to steps per second.  `active_rows_mode`
times the same decode with the LM head restricted to each sequence's active
block (FORK_ROWS_ACTIVE), a separate, HBM-bound workload; `drawn_candidates`
times both modes with candidates drawn at sampling temperature 0.8;
`decode_loop` times whole decodes from the initial state until no position
is masked (NFE steps, committed tokens per second), on all rows and on the
active blocks' rows; `forkgrpo_likelihood` times one ForkGRPO batch of 4096 teacher-forced
log-probabilities plus its objective; `selection` gives the unmasking
rule's latency at the real shapes and its HBM bandwidth on a sweep of large
batches; `measured_peaks` gives this GPU's achievable MFMA and HBM rates
(probe kernels), and the rooflines also quote fractions of those.
`configs` times the other workloads of the benchmark definition (mid
B=4 L=256 d=1024 V=32000; rollout B=64 L=384; long B=2 L=2048 block 64),
each eagerly and as a captured HIP graph of the same steps; `cpu_baseline`
carries further legs (one thread and all threads, full steps of the tiny and
mid workloads, the host's CPU model); `context_unfused_torch` times the
same LLaDA-8B-shaped step done by unfused torch operations (library GEMM
writing the logits, then reductions and a tensor-level selection), for
context only.
"""
import argparse
import ctypes
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "denoising steps/sec and positions/sec at B·L×4096×126464; % MFMA bf16 peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_lmhead_llada8b.json")
LMHEAD_SRC = os.path.join(ROOT, "paper_2609_39859_amd", "csrc", "gemm_stats.hip")


def _hip():
    """The HIP runtime torch already loaded (same soname)."""
    lib = ctypes.CDLL("libamdhip64.so.7")
    lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipEventCreate.restype = ctypes.c_int
    lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
    lib.hipEventDestroy.restype = ctypes.c_int
    lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                        ctypes.c_void_p]
    lib.hipEventElapsedTime.restype = ctypes.c_int
    return lib


def _source_hash():
    with open(LMHEAD_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def _traffic_per_launch(kernel):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    runs, if they were taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256_16") != _source_hash():
        return None
    return t.get("kernels", {}).get(kernel, {}).get("hbm_bytes_per_launch")


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_threads():
    return int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0)) or 1


def cpu_baseline(cfg, W_dev, h_dev, target_s):
    """Time the oracle (as it is) on a bounded sample of rows of this
    workload; scale rows/s to steps/s (a step covers B*L rows)."""
    import numpy as np

    import oracle
    from paper_2609_39859_amd import synth
    Wb = synth.to_bits(W_dev)
    hb = synth.to_bits(h_dev)
    threads = _oracle_threads()
    orc = oracle.default()
    probe = np.arange(threads, dtype=np.int64)
    t0 = time.perf_counter()
    orc.row_stats(hb, Wb, probe, nthreads=threads)
    per_batch = time.perf_counter() - t0
    nb = max(1, int(target_s / max(per_batch, 1e-3)) - 1)
    rows = np.arange(threads, threads * (nb + 1), dtype=np.int64) % cfg.M
    t0 = time.perf_counter()
    st = orc.row_stats(hb, Wb, rows, nthreads=threads)
    dt = time.perf_counter() - t0
    assert np.all(np.isfinite(st["conf"]))
    rows_per_s = rows.size / dt
    # the same workload on one thread, a few rows
    rows1 = np.arange(4, dtype=np.int64)
    t0 = time.perf_counter()
    orc.row_stats(hb, Wb, rows1, nthreads=1)
    dt1 = time.perf_counter() - t0
    return {"value": rows_per_s / cfg.M, "unit": "steps/s", "cores": threads, "kind": "oracle",
            "sample": "%d of the %d rows of one step (binary64 logits over all %d vocabulary "
                      "entries + statistics), %.1f s on %d threads; value = rows/s / %d"
                      % (rows.size, cfg.M, cfg.V, dt, threads, cfg.M),
            "cpu_model": _cpu_model(), "host_cpus": len(os.sched_getaffinity(0)),
            "one_thread": {"value": rows1.size / dt1 / cfg.M, "unit": "steps/s",
                           "sample": "%d rows, %.1f s on 1 thread" % (rows1.size, dt1)}}


def cpu_legs():
    """Further oracle timings: whole steps (statistics of every row, then
    the selection) of the tiny and mid workloads on one thread and on all
    threads; the mid step on one thread is timed on a sample of rows and
    scaled (marked so)."""
    import numpy as np

    import oracle
    from paper_2609_39859_amd import synth
    threads = _oracle_threads()
    orc = oracle.default()
    out = {"cpu_model": _cpu_model(), "threads": threads, "legs": []}
    for name in ("tiny", "mid"):
        cfg = synth.CONFIGS[name]
        W = synth.to_bits(synth.weights(cfg))
        h = synth.to_bits(synth.hidden(cfg, 0))
        tok, msk, bs = (x.numpy() for x in synth.initial_state(cfg))
        lam = float(np.float32(cfg.tau))
        for nt in (1, threads):
            if name == "mid" and nt == 1:
                rows = np.arange(0, cfg.M, 16, dtype=np.int64)   # 64 of 1024 rows
                t0 = time.perf_counter()
                orc.row_stats(h, W, rows, nthreads=1)
                dt = (time.perf_counter() - t0) * cfg.M / rows.size
                how = "rows %d of %d timed, scaled to the whole step" % (rows.size, cfg.M)
            else:
                reps, t0 = 0, time.perf_counter()
                while True:
                    orc.step(h, W, tok, msk, bs, cfg.B, cfg.L, cfg.block_len, lam, nthreads=nt)
                    reps += 1
                    if time.perf_counter() - t0 > 0.5:
                        break
                dt = (time.perf_counter() - t0) / reps
                how = "%d whole steps" % reps
            out["legs"].append({"workload": name, "threads": nt, "s_per_step": dt,
                                "steps_per_s": 1.0 / dt, "how": how})
    return out


def grpo_likelihood(args, hip, W, h, dev):
    """One ForkGRPO likelihood batch: 16 prompts x 16 rollouts x 16 fallback
    steps = 4096 teacher-forced entries (hidden rows [4096, d], given tokens)
    through fork_logprob, then the clipped-surrogate objective over the
    batch.  LM-head time from HIP events around its launch."""
    import torch

    from paper_2609_39859_amd import _binding
    n_groups, G, per = 16, 16, 16
    R = n_groups * G
    n = R * per
    V, d = W.shape
    gen = torch.Generator(device=dev).manual_seed(0x6EED)
    toks = torch.randint(0, V, (n,), generator=gen, device=dev, dtype=torch.int32)
    hh = h[:n].contiguous()
    lp_new, lp_old = (torch.empty(n, device=dev) for _ in range(2))
    lp_old.copy_(-torch.rand(n, generator=gen, device=dev) * 8)
    rewards = (torch.rand(R, generator=gen, device=dev) < 0.5).float()
    offsets = torch.arange(0, n + 1, per, device=dev, dtype=torch.int32)
    gobj = torch.empty(n_groups, device=dev)
    skip = torch.empty(n_groups, dtype=torch.uint8, device=dev)
    J = torch.empty(1, device=dev)
    evs = []
    for _ in range(2 * args.steps):
        e = ctypes.c_void_p()
        assert hip.hipEventCreate(ctypes.byref(e)) == 0
        evs.append(e.value)

    def batch(i=None):
        _binding.logprob(hh, W, toks, lp_new,
                         events=None if i is None else (evs[2 * i], evs[2 * i + 1]))
        _binding.grpo_objective(rewards, offsets, lp_new, lp_old, G, 0.2, gobj, skip, J)

    print("bench: timing %d ForkGRPO likelihood batches" % args.steps, file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        batch()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.steps):
        batch(i)
    stop.record()
    torch.cuda.synchronize()
    assert math.isfinite(J.item())
    lm = []
    for i in range(args.steps):
        ms = ctypes.c_float()
        assert hip.hipEventElapsedTime(ctypes.byref(ms), evs[2 * i], evs[2 * i + 1]) == 0
        lm.append(ms.value)
    for e in evs:
        hip.hipEventDestroy(e)
    batch_ms = start.elapsed_time(stop) / args.steps
    lm_ms = sum(lm) / len(lm)
    tflops = 2.0 * n * d * V / (lm_ms * 1e-3) / 1e12
    return {"entries": n, "groups": n_groups, "G": G, "fallback_steps_per_rollout": per,
            "ms_per_batch": batch_ms, "lmhead_ms": lm_ms,
            "roofline": {"bound": "mfma", "achieved": tflops, "peak": PEAK_BF16_TFLOPS,
                         "unit": "TFLOP/s", "frac": tflops / PEAK_BF16_TFLOPS,
                         "kernel": "gemm_stats_bf16_target_kernel (teacher-forced LM head)"}}


SEL_BYTES_PER_SEQ = 4 + 32 + 32 * 4 + 4 + (4 + 1 + 4 + 4)
PROBE_LIB = os.path.join(ROOT, "paper_2609_39859_amd", "libforkprobe.so")


def measured_peaks(dev):
    """The achievable rates of this GPU: dense bf16 MFMA from a kernel that
    only issues independent MFMAs on register operands, HBM from a streaming
    copy of 2 x 1 GiB (read + write)."""
    import torch
    lib = ctypes.CDLL(PROBE_LIB)
    lib.fork_probe_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.fork_probe_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                    ctypes.c_void_p]
    lib.fork_probe_mfma_data.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                         ctypes.c_void_p]
    stream = torch.cuda.current_stream(dev).cuda_stream
    blocks, iters = 7904, 256      # the LM head's grid and K/16 at the LLaDA-8B shape
    flops = blocks * 8.0 * iters * 16 * 16384
    out = torch.empty(blocks * 512, device=dev)
    # operands drawn like the LM head's data: W_head N(0, 1/d) and hidden
    # rows N(0, 1) x RMS U[0.5, 2] (d = 4096), bf16
    nfrag = 1024
    gen = torch.Generator(device=dev).manual_seed(0xF00D)
    a_src = (torch.randn(nfrag * 16 * 64 * 8, generator=gen, device=dev) / 64.0).to(torch.bfloat16)
    b_src = (torch.randn(nfrag * 8 * 64 * 8, generator=gen, device=dev) *
             (0.5 + 1.5 * torch.rand(nfrag * 8 * 64 * 8, generator=gen, device=dev))
             ).to(torch.bfloat16)

    def const():
        assert lib.fork_probe_mfma(blocks, iters, out.data_ptr(), stream) == 0

    def data():
        assert lib.fork_probe_mfma_data(blocks, iters, a_src.data_ptr(), b_src.data_ptr(), nfrag,
                                        out.data_ptr(), stream) == 0

    # the GPU's power state settles over a few launches: time each probe in
    # five rounds of four launches, alternating the two, and keep the best
    best = {"const": 0.0, "data": 0.0}
    for fn in (const, data):
        fn()
    torch.cuda.synchronize()
    for _ in range(5):
        for name, fn in (("const", const), ("data", data)):
            start = torch.cuda.Event(enable_timing=True)
            stop = torch.cuda.Event(enable_timing=True)
            start.record()
            for _ in range(4):
                fn()
            stop.record()
            torch.cuda.synchronize()
            best[name] = max(best[name], flops * 4 / (start.elapsed_time(stop) * 1e-3) / 1e12)
    mfma, mfma_data = best["const"], best["data"]
    del a_src, b_src
    n = (1 << 30) // 16
    src = torch.ones(n * 16, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    assert lib.fork_probe_copy(src.data_ptr(), dst.data_ptr(), n, stream) == 0
    torch.cuda.synchronize()
    reps = 5
    start.record()
    for _ in range(reps):
        assert lib.fork_probe_copy(src.data_ptr(), dst.data_ptr(), n, stream) == 0
    stop.record()
    torch.cuda.synchronize()
    assert bool(dst[-1] == 1)
    hbm = 2.0 * (1 << 30) * reps / (start.elapsed_time(stop) * 1e-3) / 1e9
    del src, dst
    return {"mfma_bf16_TFLOP_s": mfma_data, "mfma_bf16_TFLOP_s_constant_operands": mfma,
            "hbm_copy_GB_s": hbm,
            "how": "MFMA: 7904 workgroups x 8 waves x 256 rounds of 16 independent "
                   "v_mfma_f32_16x16x32_bf16 (the LM-head kernel's instruction) on register "
                   "operands (the flops of one LM-head launch), operands alternating between two "
                   "sets of fragments loaded from random bf16 data drawn like W_head and the "
                   "hidden rows (the rate quoted), "
                   "and on one constant set (constant_operands); best of five rounds of four "
                   "launches, the two probes alternating; HBM: streaming copy of 1 GiB "
                   "(one 16-byte element per thread, nontemporal loads and stores), read + "
                   "write counted, 5 repetitions"}


def selection(args, dev):
    """The unmasking rule alone (fork_select).  At the real shapes it moves a
    few KB and is bound by launch latency: report its latency.  Its
    bandwidth is shown on a sweep of large batches (2^14..2^20 sequences,
    one block of 32 positions each, confidences at most 0.03 as at the
    LLaDA-8B shape, so every step is a fallback step committing one
    position): algorithmic bytes per sequence = block start, the block's 32
    mask bytes and 32 confidences read, the committed candidate read, and
    token, mask byte, fallback flag and block start written.  The timed
    launches cycle over enough distinct copies of the batch that the bytes
    one launch touches, summed over the copies, exceed twice the 256 MB
    last-level cache, so they come from HBM, not from the cache."""
    import torch

    from paper_2609_39859_amd import _binding
    out = {"latency_us": {}, "sweep": []}

    def make(B, L, seed):
        gen = torch.Generator(device=dev).manual_seed(seed)
        M = B * L
        return dict(conf=torch.rand(M, generator=gen, device=dev) * 0.03,
                    am=torch.randint(0, 126464, (M,), generator=gen, device=dev, dtype=torch.int32),
                    tok=torch.full((M,), -1, dtype=torch.int32, device=dev),
                    msk=torch.ones(M, dtype=torch.uint8, device=dev),
                    bs=torch.zeros(B, dtype=torch.int32, device=dev),
                    fb=torch.empty(B, dtype=torch.int32, device=dev))

    def run(B, L, BL, reps, warmup, nsets=1, layout=_binding.FORK_LAYOUT_ROW_MAJOR):
        sets = [make(B, L, B + L + k) for k in range(nsets)]
        pm = layout == _binding.FORK_LAYOUT_POSITION_MAJOR

        def launch(x):
            _binding.select(x["conf"], x["am"], x["tok"], x["msk"], x["bs"], BL, 0.9, x["fb"],
                            B=B, L=L, layout=layout)
        for k in range(warmup):
            launch(sets[k % nsets])
        torch.cuda.synchronize()
        # the timed launches replay as one HIP graph, so host launch
        # overhead does not separate them (the call allocates nothing)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for k in range(reps):
                launch(sets[k % nsets])
        torch.cuda.synchronize()
        graph.replay()  # untimed first replay
        torch.cuda.synchronize()
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        start.record()
        graph.replay()
        stop.record()
        torch.cuda.synchronize()
        # every launch committed one position of each sequence
        per_set = [warmup // nsets + (1 if k < warmup % nsets else 0) +
                   2 * (reps // nsets + (1 if k < reps % nsets else 0)) for k in range(nsets)]
        for x, n in zip(sets, per_set):
            assert int((x["fb"] == 1).sum().item()) == B
            m = x["msk"].view(L, B).t() if pm else x["msk"].view(B, L)
            assert int(m[:, :n].sum().item()) == 0
            assert int(m[:, n:].sum().item()) == B * (L - n)
        return start.elapsed_time(stop) * 1e3 / reps

    for name, B, L, BL in (("llada8b", 8, 512, 32), ("rollout", 64, 384, 32),
                           ("long", 2, 2048, 64)):
        out["latency_us"][name] = run(B, L, BL, 20, 3)
    for B in (1 << 14, 1 << 17, 1 << 20):
        # enough copies that the bytes one launch touches, summed over the
        # copies, exceed twice the last-level cache
        nsets = max(1, -(-(512 << 20) // (SEL_BYTES_PER_SEQ * B)))
        reps = max(20, nsets)
        assert 3 + 2 * -(-reps // nsets) < 32   # each copy keeps masked positions
        for layout, lname in ((_binding.FORK_LAYOUT_ROW_MAJOR, "row_major"),
                              (_binding.FORK_LAYOUT_POSITION_MAJOR, "position_major")):
            us = run(B, 32, 32, reps, 3, nsets, layout)
            gbs = SEL_BYTES_PER_SEQ * B / (us * 1e-6) / 1e9
            out["sweep"].append({"B": B, "L": 32, "block_len": 32, "layout": lname, "us": us,
                                 "GB_s": gbs, "frac_hbm": gbs / PEAK_HBM_GBS,
                                 "bytes_per_seq": SEL_BYTES_PER_SEQ, "batch_copies": nsets,
                                 "bytes_touched_cycled": nsets * SEL_BYTES_PER_SEQ * B})
    return out


def context_unfused_torch(cfg, W, h, state, dev, steps):
    """Context only: the same step done by unfused torch operations on the
    same GPU and inputs.  The library GEMM (torch's linear, hipBLASLt)
    writes the [B*L, V] logits; fp32 log-sum-exp, maximum and entropy follow
    as separate reductions; the selection is done with tensor operations
    over the sequences' active blocks.  Also times the library GEMM alone."""
    import torch
    import torch.nn.functional as F
    B, L, BL, M, V = cfg.B, cfg.L, cfg.block_len, cfg.M, cfg.V
    tok0, msk0, bs0 = (x.to(dev) for x in state)
    tok, msk, bs = tok0.clone(), msk0.clone(), bs0.clone()
    pos = torch.arange(L, device=dev)
    tau = float(cfg.tau)

    def gemm():
        return F.linear(h, W)

    def step():
        z = F.linear(h, W).float()
        lse = torch.logsumexp(z, dim=1)
        zmax, am = z.max(dim=1)
        p = torch.exp(z - lse[:, None])
        ent = lse - (p * z).sum(dim=1)
        conf = torch.exp(zmax - lse)
        logp = zmax - lse
        m2 = msk.view(B, L).bool()
        cand = m2 & (pos[None, :] >= bs[:, None])
        has = cand.any(dim=1)
        first = torch.where(has, cand.int().argmax(dim=1), torch.full_like(bs, L))
        s = bs + torch.div(first - bs, BL, rounding_mode="floor") * BL
        inblk = cand & (pos[None, :] >= s[:, None]) & (pos[None, :] < (s + BL)[:, None])
        passing = inblk & (conf.view(B, L) > tau)
        fb = ~passing.any(dim=1)
        commit = torch.where(fb[:, None], inblk & (pos[None, :] == first[:, None]), passing)
        tv = tok.view(B, L)
        tv[commit] = am.view(B, L).int()[commit]
        m2v = msk.view(B, L)
        m2v[commit] = 0
        bs.copy_(torch.where(has, s, bs))
        return ent, logp

    def timeit(fn, reps):
        fn()
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    gemm_ms = timeit(gemm, steps)
    step_ms = timeit(step, steps)
    # the torch step commits what the library commits (all-fallback here)
    assert bool((msk.view(B, L)[:, cfg.P:cfg.P + steps + 1] == 0).all())
    flops = 2.0 * M * cfg.d * V
    return {"library_gemm_ms": gemm_ms,
            "library_gemm_TFLOP_s": flops / (gemm_ms * 1e-3) / 1e12,
            "unfused_step_ms": step_ms, "unfused_steps_per_s": 1000.0 / step_ms,
            "how": "torch linear (hipBLASLt) bf16 logits [B*L, V], then fp32 logsumexp, max, "
                   "entropy and a tensor-level selection; %d steps" % steps}


# Figures the paper reports for its own setting (context for the numbers
# above, not measured here and not comparable to synthetic decodes, whose
# near-flat logits make every step a fallback step).
PAPER_CONTEXT = {
    "sampler_nfe": "Fork-dLLM needs 2-3x fewer model evaluations per sample than AR decoding "
                   "at matched pass@k; LLaDA-8B-Instruct, generation length 256, blocks of 32, "
                   "lambda = tau = 0.8: NFE 67.8 vs 227.9 (GSM8K), 92.3 vs 243.3 (MATH-500), "
                   "108.4 vs 242.3 (HumanEval), 75.8 vs 192.3 (MBPP) (Section 4.1; the appendix's "
                   "pass@k table for LLaDA-8B-Instruct)",
    "post_training_cost": "ForkGRPO with LoRA on 4 x H100 for 12 h (48 H100-hours) against the "
                          "JustGRPO checkpoint from full fine-tuning on 16 x H100 for 24 h "
                          "(384 H100-hours): 8x fewer H100-hours at comparable GSM8K accuracy "
                          "(Section 4.2)",
    "hardware": "NVIDIA H100 (the paper times nothing per step)",
}


class StepBench:
    """Decode steps of one workload on inputs resident in HBM: the
    weights, a few batches of hidden states used in turn, the decode state
    and the outputs."""

    def __init__(self, cfg, dev, hip, n_batches=4):
        import torch

        from paper_2609_39859_amd import synth
        self.cfg, self.dev, self.hip = cfg, dev, hip
        self.W = synth.weights(cfg, device=dev)
        self.hs = [synth.hidden(cfg, t, device=dev,
                                W=self.W if cfg.plant_peaks > 0 else None)
                   for t in range(n_batches)]
        self.state0 = synth.initial_state(cfg)
        self.tok, self.msk, self.bs = (x.to(dev) for x in self.state0)
        f32 = dict(dtype=torch.float32, device=dev)
        self.conf, self.ent, self.logp = (torch.empty(cfg.M, **f32) for _ in range(3))
        self.fb = torch.empty(cfg.B, dtype=torch.int32, device=dev)

    def reset(self):
        import torch
        for d, s in zip((self.tok, self.msk, self.bs), self.state0):
            d.copy_(s.to(self.dev))
        torch.cuda.synchronize()

    def step(self, i, events=None, rows_mode=0, temperature=0.0, workspace=None):
        from paper_2609_39859_amd import _binding
        c = self.cfg
        _binding.fork_step_ex(self.hs[i % len(self.hs)], self.W, self.tok, self.msk, self.bs,
                              c.block_len, c.tau, self.conf, self.ent, self.logp, self.fb,
                              B=c.B, L=c.L, events=events, rows_mode=rows_mode,
                              temperature=temperature, seed=0x5EED, counter=i,
                              workspace=workspace)

    def timed(self, rows_mode, steps, warmup, temperature=0.0):
        """Warm up, restart the decode, then time `steps` steps: total time
        from torch events on the current stream, LM-head time per step from
        HIP events the library records around that kernel on the same
        stream."""
        import torch
        hip = self.hip
        evs = []
        for _ in range(2 * steps):
            e = ctypes.c_void_p()
            assert hip.hipEventCreate(ctypes.byref(e)) == 0
            evs.append(e.value)
        for i in range(warmup):
            self.step(i, rows_mode=rows_mode, temperature=temperature)
        torch.cuda.synchronize()
        self.reset()
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        start.record()
        for i in range(steps):
            self.step(i, (evs[2 * i], evs[2 * i + 1]), rows_mode=rows_mode,
                      temperature=temperature)
        stop.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        lm = []
        for i in range(steps):
            ms = ctypes.c_float()
            assert hip.hipEventElapsedTime(ctypes.byref(ms), evs[2 * i], evs[2 * i + 1]) == 0
            lm.append(ms.value)
        for e in evs:
            hip.hipEventDestroy(e)
        return start.elapsed_time(stop), lm, wall

    def full_decode(self, rows_mode):
        """A whole decode from the initial state: steps until no position is
        masked.  An untimed pass counts the steps (NFE) and fallback steps,
        checking the mask after every step; the same NFE steps are then
        timed from the initial state, with no host check inside the timed
        region, and must end with every position unmasked.  Hidden states
        cycle through the preloaded batches."""
        import torch
        c = self.cfg
        self.reset()
        to_commit = int((self.msk != 0).sum())
        nfe = fallback = parallel = 0
        while bool((self.msk != 0).any()):
            self.step(nfe, rows_mode=rows_mode)
            fb = self.fb.cpu()
            fallback += int((fb == 1).sum())
            parallel += int((fb == 0).sum())
            nfe += 1
            # every step commits at least one position of each active sequence
            assert nfe <= to_commit, "decode did not finish"
        self.reset()
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        start.record()
        for i in range(nfe):
            self.step(i, rows_mode=rows_mode)
        stop.record()
        torch.cuda.synchronize()
        assert not bool((self.msk != 0).any())
        ms = start.elapsed_time(stop)
        self.reset()
        return {"nfe": nfe, "committed_tokens": to_commit, "ms": ms,
                "tokens_per_s": to_commit / (ms * 1e-3), "steps_per_s": nfe / (ms * 1e-3),
                "fallback_seq_steps": fallback, "parallel_seq_steps": parallel,
                "tokens_per_step": to_commit / nfe / c.B}

    def graph_timed(self, steps, rows_mode=0):
        """The same `steps` steps captured into one HIP graph (caller
        workspace) and replayed: the GPU's time per step without host
        launch gaps.  The replayed decode must end in the state the eager
        steps reach."""
        import torch

        from paper_2609_39859_amd import _binding
        c = self.cfg
        nbytes = _binding.workspace_bytes(c.B, c.L, c.V)
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.dev)
        off = (-buf.data_ptr()) % 256
        ws = buf[off:off + nbytes]
        self.reset()
        for i in range(steps):
            self.step(i, rows_mode=rows_mode, workspace=ws)
        torch.cuda.synchronize()
        want = (self.tok.clone(), self.msk.clone(), self.bs.clone())
        self.reset()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(steps):
                self.step(i, rows_mode=rows_mode, workspace=ws)
        ms = []
        for _ in range(2):
            self.reset()
            start = torch.cuda.Event(enable_timing=True)
            stop = torch.cuda.Event(enable_timing=True)
            start.record()
            graph.replay()
            stop.record()
            torch.cuda.synchronize()
            assert all(torch.equal(a, b) for a, b in zip((self.tok, self.msk, self.bs), want))
            ms.append(start.elapsed_time(stop) / steps)
        del graph
        return ms[-1]


def config_leg(name, args, dev, hip, cfg=None):
    """Eager and graph-replayed step times of one workload, all rows and
    active-block rows, with the LM head's fraction of the bf16 MFMA peak."""
    import torch

    from paper_2609_39859_amd import _binding, synth
    cfg = cfg or synth.CONFIGS[name]
    print("bench: workload %s B=%d L=%d d=%d V=%d" % (name, cfg.B, cfg.L, cfg.d, cfg.V),
          file=sys.stderr, flush=True)
    sb = StepBench(cfg, dev, hip)
    flops = 2.0 * cfg.M * cfg.d * cfg.V
    total, lm, _ = sb.timed(_binding.FORK_ROWS_ALL, args.steps, args.warmup)
    ms = total / args.steps
    lm_ms = sum(lm) / len(lm)
    g_ms = sb.graph_timed(args.steps)
    a_total, a_lm, _ = sb.timed(_binding.FORK_ROWS_ACTIVE, args.steps, args.warmup)
    a_g_ms = sb.graph_timed(args.steps, _binding.FORK_ROWS_ACTIVE)
    dec = {"active_rows": sb.full_decode(_binding.FORK_ROWS_ACTIVE)}
    if cfg.d * cfg.V <= (1 << 30) // 8:
        # small heads only: a whole decode on all rows stays within a second
        dec["all_rows"] = sb.full_decode(_binding.FORK_ROWS_ALL)
    tf = flops / (lm_ms * 1e-3) / 1e12
    out = {"workload": "B=%d, L=%d (prompt %d + gen %d), block_len %d, d=%d, V=%d, %s, tau=%g"
                       % (cfg.B, cfg.L, cfg.P, cfg.G, cfg.block_len, cfg.d, cfg.V, cfg.dtype,
                          cfg.tau),
           "ms_per_step": ms, "steps_per_s": 1000.0 / ms, "positions_per_s": 1000.0 / ms * cfg.M,
           "graph_ms_per_step": g_ms, "graph_steps_per_s": 1000.0 / g_ms,
           "lmhead_ms": lm_ms,
           "roofline": {"bound": "mfma", "achieved": tf, "peak": PEAK_BF16_TFLOPS,
                        "unit": "TFLOP/s", "frac": tf / PEAK_BF16_TFLOPS,
                        "kernel": "gemm_stats_bf16_kernel",
                        "algorithmic_flops_per_launch": flops},
           "step_mfma_frac_graph": flops / (g_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
           "step_ms_at_60pct_of_peak": flops / (0.6 * PEAK_BF16_TFLOPS * 1e12) * 1e3,
           "active_rows_mode": {"ms_per_step": a_total / args.steps,
                                "graph_ms_per_step": a_g_ms,
                                "lmhead_ms": sum(a_lm) / len(a_lm)},
           "decode_loop": dec}
    del sb
    torch.cuda.empty_cache()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="llada8b")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-active-rows", action="store_true",
                    help="skip the extra timing of the active-block-only LM head")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the whole-decode timings (committed tokens per second)")
    ap.add_argument("--no-drawn", action="store_true",
                    help="skip the extra timings with candidates drawn at temperature 0.8")
    ap.add_argument("--no-grpo", action="store_true",
                    help="skip the timing of the ForkGRPO likelihood batch")
    ap.add_argument("--no-selection", action="store_true",
                    help="skip the selection latency and bandwidth sweep")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measurement of the achievable MFMA and HBM rates")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the timings of the mid, rollout and long workloads")
    ap.add_argument("--no-context", action="store_true",
                    help="skip the unfused torch step (context only)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run a plain 1 GiB device copy (a known-size kernel for "
                         "scaling rocprofv3 FETCH_SIZE / WRITE_SIZE readings)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_39859_amd import _binding, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = synth.CONFIGS[args.config]
    B, L, BL, M, d, V = cfg.B, cfg.L, cfg.block_len, cfg.M, cfg.d, cfg.V
    print("bench: %s B=%d L=%d d=%d V=%d, generating inputs" % (cfg.name, B, L, d, V),
          file=sys.stderr, flush=True)

    if args.calibrate_copy:
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        print("bench: ran 3 copies of 1 GiB (read 1 GiB + write 1 GiB each)",
              file=sys.stderr, flush=True)

    hip = _hip()
    sb = StepBench(cfg, dev, hip)
    W, hs = sb.W, sb.hs

    print("bench: timing %d steps" % args.steps, file=sys.stderr, flush=True)
    total_ms, lm_ms, wall = sb.timed(_binding.FORK_ROWS_ALL, args.steps, args.warmup)

    ms_per_step = total_ms / args.steps
    steps_per_s = 1000.0 / ms_per_step
    lm_avg_ms = sum(lm_ms) / len(lm_ms)
    flops = 2.0 * M * d * V
    achieved_tflops = flops / (lm_avg_ms * 1e-3) / 1e12
    traffic = _traffic_per_launch("gemm_stats_bf16_kernel")

    out = {
        "metric": METRIC,
        "value": steps_per_s,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) hidden rows x RMS~U[0.5,2], W_head ~ N(0,1/d); no model weights)",
        "config": {"workload": "LLaDA-8B-shaped step: B=8, L=512 (prompt 256 + gen 256), block_len 32, "
                               "d=4096, V=126464, bf16, tau=0.9",
                   "B": B, "L": L, "block_len": BL, "d": d, "V": V, "tau": cfg.tau},
        "positions_per_s": steps_per_s * M,
        "mfma_frac_step": (flops / (ms_per_step * 1e-3) / 1e12) / PEAK_BF16_TFLOPS,
        "lmhead_ms": lm_avg_ms,
        "wall_s_timed": wall,
        "roofline": {"bound": "mfma", "achieved": achieved_tflops, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved_tflops / PEAK_BF16_TFLOPS,
                     "traffic": traffic,
                     "kernel": "gemm_stats_bf16_kernel (LM head + per-tile statistics)",
                     "algorithmic_flops_per_launch": flops},
        "cpu_baseline": None,
        "paper_context": PAPER_CONTEXT,
    }
    pk = None
    if not args.no_peaks:
        # right after the headline timing, so that the probes run in the same
        # thermal state as the timed LM-head launches
        print("bench: measuring achievable MFMA and HBM rates", file=sys.stderr, flush=True)
        pk = measured_peaks(dev)
        out["measured_peaks"] = pk
        rf = out["roofline"]
        rf["measured_peak"] = pk["mfma_bf16_TFLOP_s"]
        rf["frac_of_measured_peak"] = rf["achieved"] / pk["mfma_bf16_TFLOP_s"]
    out["graph_ms_per_step"] = sb.graph_timed(args.steps)
    if not args.no_active_rows:
        # The same workload with the LM head restricted to each sequence's
        # active block (B*block_len rows): W is read once per step and the
        # per-row work is small, so this mode is bounded by HBM bandwidth.
        print("bench: timing %d steps, active-block rows only" % args.steps, file=sys.stderr,
              flush=True)
        a_total, a_lm, _ = sb.timed(_binding.FORK_ROWS_ACTIVE, args.steps, args.warmup)
        sb.reset()
        Ma = B * BL
        a_ms = a_total / args.steps
        a_lm_ms = sum(a_lm) / len(a_lm)
        a_bytes = (V * d + Ma * d) * 2 + math.ceil(V / 256) * Ma * 16  # W, rows, partials
        a_gbs = a_bytes / (a_lm_ms * 1e-3) / 1e9
        out["active_rows_mode"] = {
            "rows_per_step": Ma, "ms_per_step": a_ms, "steps_per_s": 1000.0 / a_ms,
            "lmhead_ms": a_lm_ms,
            "graph_ms_per_step": sb.graph_timed(args.steps, _binding.FORK_ROWS_ACTIVE),
            "roofline": {"bound": "hbm", "achieved": a_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": a_gbs / PEAK_HBM_GBS,
                         "traffic": _traffic_per_launch("gemm_stats_bf16_rows_kernel"),
                         "kernel": "gemm_stats_bf16_rows_kernel (LM head on the active rows)",
                         "algorithmic_bytes_per_launch": a_bytes,
                         "mfma_frac": 2.0 * Ma * d * V / (a_lm_ms * 1e-3) / 1e12
                                      / PEAK_BF16_TFLOPS}}
        if pk:
            ar = out["active_rows_mode"]["roofline"]
            ar["measured_peak"] = pk["hbm_copy_GB_s"]
            ar["frac_of_measured_peak"] = ar["achieved"] / pk["hbm_copy_GB_s"]
    if not args.no_decode:
        print("bench: whole decodes (all rows, then active-block rows)", file=sys.stderr,
              flush=True)
        out["decode_loop"] = {"all_rows": sb.full_decode(_binding.FORK_ROWS_ALL),
                              "active_rows": sb.full_decode(_binding.FORK_ROWS_ACTIVE),
                              "hidden": "%d preloaded batches used in turn" % len(sb.hs)}
    if not args.no_drawn:
        # Candidates drawn at sampling temperature 0.8 (Gumbel-max over
        # Philox4x32-10 draws for the active blocks' positions).
        drawn = {"temperature": 0.8}
        for label, mode, kernel in (("all_rows", _binding.FORK_ROWS_ALL, "gemm_stats_bf16_draw_ilv_kernel"),
                                    ("active_rows", _binding.FORK_ROWS_ACTIVE,
                                     "gemm_stats_bf16_rows_draw_kernel")):
            print("bench: timing %d steps, drawn candidates, %s" % (args.steps, label),
                  file=sys.stderr, flush=True)
            d_total, d_lm, _ = sb.timed(mode, args.steps, args.warmup, temperature=0.8)
            sb.reset()
            drawn[label] = {"ms_per_step": d_total / args.steps,
                            "steps_per_s": 1000.0 * args.steps / d_total,
                            "lmhead_ms": sum(d_lm) / len(d_lm), "kernel": kernel}
        out["drawn_candidates"] = drawn
    if not args.no_grpo:
        out["forkgrpo_likelihood"] = grpo_likelihood(args, hip, W, hs[0], dev)
    if not args.no_context:
        print("bench: unfused torch step (context)", file=sys.stderr, flush=True)
        out["context_unfused_torch"] = context_unfused_torch(cfg, W, hs[0], sb.state0, dev,
                                                             min(args.steps, 10))
        torch.cuda.empty_cache()
    if not args.no_selection:
        print("bench: selection latency and bandwidth sweep", file=sys.stderr, flush=True)
        out["selection"] = selection(args, dev)
        torch.cuda.empty_cache()
        if pk:
            for x in out["selection"]["sweep"]:
                x["frac_of_measured_hbm"] = x["GB_s"] / pk["hbm_copy_GB_s"]
    if not args.no_configs:
        out["configs"] = {}
        for name in ("mid", "rollout", "long"):
            out["configs"][name] = config_leg(name, args, dev, hip)
        # One GPU's share of a vocabulary-sharded step over 8 GPUs: the
        # LLaDA-8B shape with V / 8 rows of W_head (the per-position partials
        # would then be all-gathered and merged on every GPU; that exchange
        # is not part of this single-GPU measurement).
        shard = synth.CONFIGS["llada8b"].with_(name="llada8b_vocab_shard_of_8", V=V // 8)
        leg = config_leg(shard.name, args, dev, hip, cfg=shard)
        leg["shards"] = 8
        out["configs"][shard.name] = leg
    if not args.no_cpu_baseline:
        print("bench: oracle CPU baseline (~%.0f s)" % args.cpu_seconds, file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(cfg, W, hs[0], args.cpu_seconds)
        print("bench: oracle CPU legs (tiny and mid whole steps)", file=sys.stderr, flush=True)
        out["cpu_baseline"]["legs"] = cpu_legs()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
