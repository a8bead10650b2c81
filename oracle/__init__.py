"""CPU oracle for one Fork-dLLM denoising step (binary64, plain C).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
CPU-baseline leg of the benchmark may import this package.  The product path
(the HIP library and its Python binding) never imports, links or calls it,
and the two share no code: this package holds its own C source and header and
reads nothing from the HIP sources.

Functions follow the paper (Fork-dLLM, Section 2 "Sampling in masked dLLMs",
Algorithm 2, Algorithm 1 for the differential tests, Section 3.2):

* ``row_stats`` -- per-position statistics of q^k(. | x_t): greedy candidate
  (lowest index of the maximum logit), confidence q(candidate), log q of the
  candidate, log-normaliser, entropy in nats and the top-2 logit gap.
* ``select`` -- the unmasking rule inside the active block (threshold set,
  then leftmost or highest-confidence fallback), applied to copies;
  ``select_ex`` adds the fallback ablations of Section 4.1 (lowest
  confidence, highest entropy, uniformly random masked position).
* ``step`` -- both, over every row.
* ``row_sample`` -- sampled candidates at a temperature tau > 0 (the draw
  x_0^k ~ q(. | x_t; tau) of Section 2, by the Gumbel-max property with
  Philox4x32-10 draws), with the untempered q and log q of the drawn token;
  ``philox``, ``exp_draw`` expose the generator.
* ``token_logprob``, ``grpo_objective``, ``top_entropy`` -- the ForkGRPO
  side of Section 3.2: teacher-forced log-probabilities of given tokens, the
  clipped surrogate averaged over each rollout's fallback steps with
  group-normalised advantages, and JustGRPO-Fast's highest-entropy
  positions.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fork_oracle.c")
_LIB = os.path.join(_HERE, "libforkoracle.so")

BF16 = 0
F32 = 1
RULE_LEFTMOST = 0
RULE_MAXCONF = 1
RULE_MINCONF = 2
RULE_MAXENT = 3
RULE_RANDOM = 4

def build(force: bool = True, src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc (plain C99 + OpenMP)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-I", _HERE, "-o", tmp, src, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _as_input(x: np.ndarray):
    """bf16 bits arrive as uint16/int16 arrays, binary32 as float32."""
    x = np.ascontiguousarray(x)
    if x.dtype in (np.uint16, np.int16):
        return x, BF16
    if x.dtype == np.float32:
        return x, F32
    raise TypeError("oracle inputs must be bf16 bits (uint16) or float32, got %s" % x.dtype)


class Oracle:
    """ctypes front end of one compiled copy of the oracle."""

    def __init__(self, libpath: str = _LIB):
        if libpath == _LIB and not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(libpath)
        P = ctypes.c_void_p
        lib.oracle_row_stats.restype = ctypes.c_int
        lib.oracle_row_stats.argtypes = [P, P, ctypes.c_int, ctypes.c_int64,
                                         ctypes.c_int64, P, ctypes.c_int64,
                                         P, P, P, P, P, P, ctypes.c_int]
        lib.oracle_select.restype = ctypes.c_int
        lib.oracle_select.argtypes = [ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_int32, P, P, ctypes.c_double,
                                      ctypes.c_int, P, P, P, P, P]
        lib.oracle_select_ex.restype = ctypes.c_int
        lib.oracle_select_ex.argtypes = [ctypes.c_int32, ctypes.c_int32,
                                         ctypes.c_int32, P, P, P, P,
                                         ctypes.c_double, ctypes.c_int,
                                         P, P, P, P, P]
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_philox4x32_10.argtypes = [P, P, P]
        lib.oracle_exp_draw.restype = ctypes.c_double
        lib.oracle_exp_draw.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64,
                                        ctypes.c_int64, P]
        lib.oracle_row_sample.restype = ctypes.c_int
        lib.oracle_row_sample.argtypes = [P, P, ctypes.c_int, ctypes.c_int64,
                                          ctypes.c_int64, P, ctypes.c_int64,
                                          ctypes.c_double, ctypes.c_uint64, ctypes.c_uint32,
                                          P, P, P, P, ctypes.c_int]
        lib.oracle_token_logprob.restype = ctypes.c_int
        lib.oracle_token_logprob.argtypes = [P, P, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                             ctypes.c_int64, P, P, ctypes.c_int64, P, P,
                                             ctypes.c_int]
        lib.oracle_grpo_objective.restype = ctypes.c_int
        lib.oracle_grpo_objective.argtypes = [ctypes.c_int32, ctypes.c_int32, P, P, P, P,
                                              ctypes.c_double, P, P, P, P, P, P, P]
        lib.oracle_top_entropy.restype = ctypes.c_int
        lib.oracle_top_entropy.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P, P]
        self.lib = lib

    def token_logprob(self, hidden, W, rows, tokens, nthreads: int = 0):
        """log q(tokens[e]) and the entropy at hidden row rows[e]."""
        h, dt_h = _as_input(hidden)
        w, dt_w = _as_input(W)
        if dt_h != dt_w:
            raise TypeError("hidden and W must share a dtype")
        M, d = h.shape
        V, d2 = w.shape
        if d != d2:
            raise ValueError("hidden is [M, %d] but W is [V, %d]" % (d, d2))
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64)).reshape(-1)
        tokens = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32)).reshape(-1)
        if rows.size != tokens.size:
            raise ValueError("rows and tokens differ in length")
        n = rows.size
        logp = np.empty(n, np.float64)
        ent = np.empty(n, np.float64)
        rc = self.lib.oracle_token_logprob(_ptr(h), _ptr(w), dt_h, M, d, V, _ptr(rows),
                                           _ptr(tokens), n, _ptr(logp), _ptr(ent), int(nthreads))
        if rc == -2:
            raise FloatingPointError("non-finite logit")
        if rc != 0:
            raise ValueError("oracle_token_logprob rejected its arguments (%d)" % rc)
        return {"logp": logp, "entropy": ent}

    def grpo_objective(self, rewards, offsets, lp_new, lp_old, G, eps):
        """ForkGRPO objective; rewards [n_groups * G], offsets [n_groups * G + 1]."""
        rewards = np.ascontiguousarray(rewards, dtype=np.float64).reshape(-1)
        offsets = np.ascontiguousarray(offsets, dtype=np.int32).reshape(-1)
        lp_new = np.ascontiguousarray(lp_new, dtype=np.float64).reshape(-1)
        lp_old = np.ascontiguousarray(lp_old, dtype=np.float64).reshape(-1)
        R = rewards.size
        if R % G or offsets.size != R + 1:
            raise ValueError("rewards must hold n_groups * G entries and offsets one more")
        ng = R // G
        n = lp_new.size
        out = {"adv": np.empty(R), "ratio": np.empty(n), "term": np.empty(n),
               "rollout_obj": np.empty(R), "group_obj": np.empty(ng),
               "skipped": np.empty(ng, np.uint8)}
        J = ctypes.c_double()
        rc = self.lib.oracle_grpo_objective(ng, int(G), _ptr(rewards), _ptr(offsets),
                                            _ptr(lp_new), _ptr(lp_old), float(eps),
                                            _ptr(out["adv"]), _ptr(out["ratio"]), _ptr(out["term"]),
                                            _ptr(out["rollout_obj"]), _ptr(out["group_obj"]),
                                            _ptr(out["skipped"]), ctypes.byref(J))
        if rc != 0:
            raise ValueError("oracle_grpo_objective rejected its arguments (%d)" % rc)
        out["J"] = J.value
        return out

    def top_entropy(self, entropy, k):
        """[R, Lg] entropies -> [R, Lg] uint8 selection of the k highest per row."""
        ent = np.ascontiguousarray(entropy, dtype=np.float64)
        if ent.ndim != 2:
            raise ValueError("entropy must be [R, Lg]")
        R, Lg = ent.shape
        sel = np.empty((R, Lg), np.uint8)
        rc = self.lib.oracle_top_entropy(R, Lg, int(k), _ptr(ent), _ptr(sel))
        if rc != 0:
            raise ValueError("oracle_top_entropy rejected its arguments (%d)" % rc)
        return sel

    def philox(self, ctr, key):
        """Philox4x32-10 of a 4-word counter under a 2-word key."""
        c = np.ascontiguousarray(ctr, dtype=np.uint32).reshape(4)
        k = np.ascontiguousarray(key, dtype=np.uint32).reshape(2)
        out = np.empty(4, np.uint32)
        self.lib.oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
        return out

    def exp_draw(self, seed, counter, row, v):
        """(E, U): the exponential draw of vocabulary entry v at position row
        and the uniform it comes from."""
        u = ctypes.c_double()
        e = self.lib.oracle_exp_draw(int(seed), int(counter), int(row), int(v), ctypes.byref(u))
        return e, u.value

    def row_sample(self, hidden, W, rows, tau, seed, counter, nthreads: int = 0):
        """Sampled candidates of ``rows``: dict with cand, conf, logp, keygap."""
        h, dt_h = _as_input(hidden)
        w, dt_w = _as_input(W)
        if dt_h != dt_w:
            raise TypeError("hidden and W must share a dtype")
        M, d = h.shape
        V, d2 = w.shape
        if d != d2:
            raise ValueError("hidden is [M, %d] but W is [V, %d]" % (d, d2))
        if rows is None:
            rows = np.arange(M, dtype=np.int64)
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64)).reshape(-1)
        if rows.size and (rows.min() < 0 or rows.max() >= M):
            raise IndexError("row index out of range")
        n = rows.size
        out = {k: np.empty(n, np.float64) for k in ("conf", "logp", "keygap")}
        out["cand"] = np.empty(n, np.int32)
        rc = self.lib.oracle_row_sample(_ptr(h), _ptr(w), dt_h, d, V, _ptr(rows), n,
                                        float(tau), int(seed), int(counter),
                                        _ptr(out["cand"]), _ptr(out["conf"]),
                                        _ptr(out["logp"]), _ptr(out["keygap"]), int(nthreads))
        if rc == -2:
            raise FloatingPointError("non-finite logit")
        if rc != 0:
            raise ValueError("oracle_row_sample rejected its arguments (%d)" % rc)
        return out

    def row_stats(self, hidden, W, rows=None, nthreads: int = 0):
        """Statistics of q(. | x_t) for ``rows`` of ``hidden`` ([M, d])
        against ``W`` ([V, d]); a dict of arrays indexed like ``rows``."""
        h, dt_h = _as_input(hidden)
        w, dt_w = _as_input(W)
        if dt_h != dt_w:
            raise TypeError("hidden and W must share a dtype")
        M, d = h.shape
        V, d2 = w.shape
        if d != d2:
            raise ValueError("hidden is [M, %d] but W is [V, %d]" % (d, d2))
        if rows is None:
            rows = np.arange(M, dtype=np.int64)
        rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64)).reshape(-1)
        if rows.size and (rows.min() < 0 or rows.max() >= M):
            raise IndexError("row index out of range")
        n = rows.size
        out = {k: np.empty(n, np.float64) for k in ("conf", "entropy", "logp", "lse", "gap")}
        out["argmax"] = np.empty(n, np.int32)
        rc = self.lib.oracle_row_stats(_ptr(h), _ptr(w), dt_h, d, V, _ptr(rows), n,
                                       _ptr(out["conf"]), _ptr(out["entropy"]),
                                       _ptr(out["logp"]), _ptr(out["lse"]),
                                       _ptr(out["argmax"]), _ptr(out["gap"]),
                                       int(nthreads))
        if rc == -2:
            raise FloatingPointError("non-finite logit")
        if rc != 0:
            raise ValueError("oracle_row_stats rejected its arguments (%d)" % rc)
        return out

    def select(self, conf, argmax_tok, tokens, mask, block_start, B, L,
               block_len, lam, rule=RULE_LEFTMOST):
        """Apply the unmasking rule; returns new (tokens, mask, block_start,
        fallback, ncommit) and leaves the inputs untouched."""
        conf = np.ascontiguousarray(conf, dtype=np.float64).reshape(-1)
        argmax_tok = np.ascontiguousarray(argmax_tok, dtype=np.int32).reshape(-1)
        tok = np.array(tokens, dtype=np.int32, copy=True).reshape(-1)
        msk = np.array(mask, dtype=np.uint8, copy=True).reshape(-1)
        bs = np.array(block_start, dtype=np.int32, copy=True).reshape(-1)
        if conf.size != B * L or argmax_tok.size != B * L or tok.size != B * L \
                or msk.size != B * L or bs.size != B:
            raise ValueError("array sizes do not match B=%d, L=%d" % (B, L))
        fb = np.empty(B, np.int32)
        nc = np.empty(B, np.int32)
        rc = self.lib.oracle_select(B, L, block_len, _ptr(conf), _ptr(argmax_tok),
                                    float(lam), int(rule), _ptr(tok), _ptr(msk),
                                    _ptr(bs), _ptr(fb), _ptr(nc))
        if rc != 0:
            raise ValueError("oracle_select rejected its arguments (%d)" % rc)
        return tok, msk, bs, fb, nc

    def select_ex(self, conf, argmax_tok, tokens, mask, block_start, B, L,
                  block_len, lam, rule=RULE_LEFTMOST, entropy=None, uniform=None):
        """select() with every fallback rule, including the Section 4.1
        ablations (entropy [B*L] for RULE_MAXENT, uniform [B] float32 in
        [0, 1) for RULE_RANDOM)."""
        conf = np.ascontiguousarray(conf, dtype=np.float64).reshape(-1)
        argmax_tok = np.ascontiguousarray(argmax_tok, dtype=np.int32).reshape(-1)
        tok = np.array(tokens, dtype=np.int32, copy=True).reshape(-1)
        msk = np.array(mask, dtype=np.uint8, copy=True).reshape(-1)
        bs = np.array(block_start, dtype=np.int32, copy=True).reshape(-1)
        if conf.size != B * L or argmax_tok.size != B * L or tok.size != B * L \
                or msk.size != B * L or bs.size != B:
            raise ValueError("array sizes do not match B=%d, L=%d" % (B, L))
        ent = None if entropy is None else np.ascontiguousarray(entropy, dtype=np.float64).reshape(-1)
        uni = None if uniform is None else np.ascontiguousarray(uniform, dtype=np.float32).reshape(-1)
        if ent is not None and ent.size != B * L:
            raise ValueError("entropy must have B*L entries")
        if uni is not None and uni.size != B:
            raise ValueError("uniform must have B entries")
        fb = np.empty(B, np.int32)
        nc = np.empty(B, np.int32)
        rc = self.lib.oracle_select_ex(B, L, block_len, _ptr(conf),
                                       None if ent is None else _ptr(ent),
                                       None if uni is None else _ptr(uni),
                                       _ptr(argmax_tok), float(lam), int(rule),
                                       _ptr(tok), _ptr(msk), _ptr(bs), _ptr(fb), _ptr(nc))
        if rc != 0:
            raise ValueError("oracle_select_ex rejected its arguments (%d)" % rc)
        return tok, msk, bs, fb, nc

    def step(self, hidden, W, tokens, mask, block_start, B, L, block_len, lam,
             rule=RULE_LEFTMOST, nthreads: int = 0):
        """One full step on every row: statistics, then selection."""
        st = self.row_stats(hidden, W, None, nthreads)
        tok, msk, bs, fb, nc = self.select(st["conf"], st["argmax"], tokens, mask,
                                           block_start, B, L, block_len, lam, rule)
        st.update(tokens=tok, mask=msk, block_start=bs, fallback=fb, ncommit=nc)
        return st


_default = None


def default() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def row_stats(*a, **k):
    return default().row_stats(*a, **k)


def select(*a, **k):
    return default().select(*a, **k)


def select_ex(*a, **k):
    return default().select_ex(*a, **k)


def step(*a, **k):
    return default().step(*a, **k)


def row_sample(*a, **k):
    return default().row_sample(*a, **k)


def philox(*a, **k):
    return default().philox(*a, **k)


def token_logprob(*a, **k):
    return default().token_logprob(*a, **k)


def grpo_objective(*a, **k):
    return default().grpo_objective(*a, **k)


def top_entropy(*a, **k):
    return default().top_entropy(*a, **k)


def exp_draw(*a, **k):
    return default().exp_draw(*a, **k)
