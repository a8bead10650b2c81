"""MI355X (gfx950) implementation of one Fork-dLLM denoising step.

The step (Fork-dLLM paper, Section 2 and Algorithm 2): the LM-head projection
of every position's final hidden state, the per-position statistics of the
resulting categorical (normaliser, confidence, entropy, greedy candidate and
its log-probability), then the unmasking rule inside each sequence's active
block -- commit every masked position whose confidence exceeds the threshold,
else only the leftmost masked position (a fallback step).

All of it runs in hand-written HIP kernels behind the C ABI declared in
``include/fork_step.h``; ``paper_2609_39859_amd.fork_step`` is a thin ctypes
binding over it.  ``synth`` holds the seeded input generators.
"""

__all__ = ["fork_step", "fork_step_ex", "workspace_bytes", "release", "version", "synth"]


def __getattr__(name):
    import importlib
    if name in ("fork_step", "fork_step_ex", "workspace_bytes", "release", "version", "lib"):
        return getattr(importlib.import_module("._binding", __name__), name)
    if name == "synth":
        return importlib.import_module(".synth", __name__)
    raise AttributeError(name)
