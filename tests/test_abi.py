"""The C-ABI library loads and exports every symbol its header declares, and
rejects bad arguments on the host before touching a GPU (no compute here)."""
import ctypes
import os
import re

import pytest

from paper_2609_39859_amd import _binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fork_step.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*(fork_[a-z_]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_entry_points():
    names = _declared_functions()
    for n in ("fork_step", "fork_step_ex", "fork_workspace_bytes", "fork_last_error",
              "fork_release", "fork_version"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_binding.LIB_PATH)
    for n in _declared_functions():
        assert hasattr(lib, n), "libforkstep.so does not export %s" % n


def test_exports_are_c_symbols():
    nm = os.popen("nm -D --defined-only %s" % _binding.LIB_PATH).read()
    for n in _declared_functions():
        assert re.search(r"\bT %s$" % n, nm, flags=re.M), n


def test_version_and_workspace_sizes():
    L = _binding.lib()
    assert L.fork_version() == 10100
    # per-tile partials (16 B per position per 256-entry vocabulary tile,
    # padded to 256 B) + candidates and active-row list (4 B per position each)
    # + the per-tile drawn candidates (as large as the partials)
    def expect(B, Lq, V):
        M = B * Lq
        nvt = (V + 255) // 256
        pad = lambda x: (x + 255) // 256 * 256
        return 2 * pad(nvt * M * 16) + pad(M * 4) + pad(M * 4)
    for B, Lq, V in [(1, 64, 1024), (4, 256, 32000), (8, 512, 126464), (3, 37, 1013)]:
        assert L.fork_workspace_bytes(B, Lq, V) == expect(B, Lq, V)
    assert L.fork_workspace_bytes(0, 5, 5) == 0
    assert L.fork_workspace_bytes(5, 5, -1) == 0
    assert L.fork_workspace_bytes(1 << 16, 1 << 16, 5) == 0


def _args(**kw):
    a = _binding.ForkStepArgs()
    good = dict(hidden=16, W_head=32, tokens=48, mask=64, block_start=80, block_len=4,
                tau=0.9, out_conf=96, out_entropy=112, out_logp=128, out_fallback=144,
                B=2, L=8, d=16, V=100, dtype=_binding.FORK_BF16, rule=0)
    good.update(kw)
    for k, v in good.items():
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("kw,code", [
    (dict(hidden=0), _binding.FORK_EINVAL),
    (dict(out_fallback=0), _binding.FORK_EINVAL),
    (dict(B=-1), _binding.FORK_EINVAL),
    (dict(V=-3), _binding.FORK_EINVAL),
    (dict(block_len=0), _binding.FORK_EINVAL),
    (dict(block_len=9), _binding.FORK_EINVAL),
    (dict(tau=float("nan")), _binding.FORK_EINVAL),
    (dict(tau=float("inf")), _binding.FORK_EINVAL),
    (dict(dtype=7), _binding.FORK_EINVAL),
    (dict(rule=5), _binding.FORK_EINVAL),
    (dict(rule=-1), _binding.FORK_EINVAL),
    (dict(rows_mode=2), _binding.FORK_EINVAL),
    (dict(sample_temperature=-0.5), _binding.FORK_EINVAL),
    (dict(sample_temperature=float("nan")), _binding.FORK_EINVAL),
    (dict(sample_temperature=float("inf")), _binding.FORK_EINVAL),
    (dict(rows_mode=1, B=64, L=2048, d=8192), _binding.FORK_EUNSUPPORTED),
    (dict(sample_temperature=1e-35), _binding.FORK_EINVAL),
    (dict(B=1 << 14, L=1 << 10, block_len=4, V=126464), _binding.FORK_EUNSUPPORTED),
    (dict(rule=4), _binding.FORK_EINVAL),          # random rule without uniforms
    (dict(d=12), _binding.FORK_EUNSUPPORTED),
    (dict(d=6, dtype=_binding.FORK_F32), _binding.FORK_EUNSUPPORTED),
    (dict(d=(1 << 20) + 8), _binding.FORK_EUNSUPPORTED),
    (dict(hidden=18), _binding.FORK_EINVAL),
    (dict(B=1 << 16, L=1 << 16), _binding.FORK_EINVAL),
    (dict(workspace=256, workspace_bytes=10), _binding.FORK_EINVAL),
    (dict(workspace=250, workspace_bytes=1 << 30), _binding.FORK_EINVAL),
])
def test_bad_arguments_rejected_on_host(kw, code):
    """Validation runs before any HIP call; the pointers here are never
    dereferenced."""
    L = _binding.lib()
    a = _args(**kw)
    assert L.fork_step_ex(ctypes.byref(a)) == code
    assert L.fork_last_error().decode() != ""


def test_empty_batch_is_a_no_op():
    """B == 0 returns before any HIP call, with every array pointer NULL; the
    scalar arguments are still checked."""
    L = _binding.lib()
    nulls = dict(hidden=0, W_head=0, tokens=0, mask=0, block_start=0, out_conf=0,
                 out_entropy=0, out_logp=0, out_fallback=0, B=0)
    assert L.fork_step_ex(ctypes.byref(_args(**nulls))) == _binding.FORK_OK
    assert L.fork_step_ex(ctypes.byref(_args(rule=4, **nulls))) == _binding.FORK_OK
    assert L.fork_step_ex(ctypes.byref(_args(tau=float("nan"), **nulls))) == _binding.FORK_EINVAL
    assert L.fork_step_ex(ctypes.byref(_args(block_len=9, **nulls))) == _binding.FORK_EINVAL
    assert L.fork_step(None, None, None, None, None, 4, 0.9, None, None, None, None,
                       0, 8, 16, 100, _binding.FORK_BF16, None) == _binding.FORK_OK
    sel_nulls = dict(conf=0, argmax=0, tokens=0, mask=0, block_start=0, out_fallback=0, B=0)
    assert L.fork_select(ctypes.byref(_sel_args(**sel_nulls))) == _binding.FORK_OK
    assert L.fork_select(ctypes.byref(_sel_args(rule=3, **sel_nulls))) == _binding.FORK_OK
    assert L.fork_select(ctypes.byref(_sel_args(rule=7, **sel_nulls))) == _binding.FORK_EINVAL


def test_null_args_struct():
    L = _binding.lib()
    assert L.fork_step_ex(None) == _binding.FORK_EINVAL


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(4, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        _binding.fork_step(x, x, None, None, None, 1, 0.5, None, None, None, None, B=1, L=4)


def test_grpo_entry_points_declared():
    names = _declared_functions()
    for n in ("fork_logprob", "fork_logprob_workspace_bytes", "fork_grpo_objective",
              "fork_top_entropy"):
        assert n in names


def test_logprob_workspace_sizes():
    L = _binding.lib()
    pad = lambda x: (x + 255) // 256 * 256
    for n, V in [(1, 1), (4096, 126464), (37, 1013)]:
        nvt = (V + 255) // 256
        assert L.fork_logprob_workspace_bytes(n, V) == pad(nvt * n * 16) + pad(n * 4)
    assert L.fork_logprob_workspace_bytes(-1, 5) == 0
    assert L.fork_logprob_workspace_bytes(5, 0) == 0


def _lp_args(**kw):
    a = _binding.ForkLogprobArgs()
    good = dict(hidden=16, W_head=32, rows=48, tokens=64, out_logp=80, n=4, M=8, d=16, V=100,
                dtype=_binding.FORK_BF16)
    good.update(kw)
    for k, v in good.items():
        assert hasattr(a, k)
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("kw,code", [
    (dict(hidden=0), _binding.FORK_EINVAL),
    (dict(tokens=0), _binding.FORK_EINVAL),
    (dict(out_logp=0), _binding.FORK_EINVAL),
    (dict(n=-1), _binding.FORK_EINVAL),
    (dict(M=0), _binding.FORK_EINVAL),
    (dict(V=0), _binding.FORK_EINVAL),
    (dict(dtype=3), _binding.FORK_EINVAL),
    (dict(rows=0, n=9), _binding.FORK_EINVAL),        # n > M without a row list
    (dict(d=12), _binding.FORK_EUNSUPPORTED),
    (dict(M=1 << 20, d=2048), _binding.FORK_EUNSUPPORTED),  # gathered rows past 2^31 bytes
    (dict(rows=0, n=1 << 24, M=1 << 24, V=126464), _binding.FORK_EUNSUPPORTED),  # grid
    (dict(hidden=18), _binding.FORK_EINVAL),
    (dict(workspace=256, workspace_bytes=10), _binding.FORK_EINVAL),
])
def test_logprob_bad_arguments_rejected_on_host(kw, code):
    L = _binding.lib()
    assert L.fork_logprob(ctypes.byref(_lp_args(**kw))) == code
    assert L.fork_last_error().decode() != ""


def test_logprob_zero_entries_is_a_no_op():
    L = _binding.lib()
    assert L.fork_logprob(ctypes.byref(_lp_args(n=0, tokens=0, out_logp=0))) == _binding.FORK_OK


def _grpo_args(**kw):
    a = _binding.ForkGrpoArgs()
    good = dict(n_groups=2, G=4, n=10, rewards=16, offsets=32, lp_new=48, lp_old=64, eps=0.2,
                out_group_obj=80, out_skipped=96, out_J=112)
    good.update(kw)
    for k, v in good.items():
        assert hasattr(a, k)
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("kw", [
    dict(G=0), dict(n_groups=-1), dict(n=-2), dict(G=1025), dict(eps=-0.1),
    dict(eps=float("nan")), dict(eps=float("inf")), dict(out_J=0), dict(rewards=0),
    dict(offsets=0), dict(out_group_obj=0), dict(out_skipped=0), dict(lp_new=0),
])
def test_grpo_bad_arguments_rejected_on_host(kw):
    L = _binding.lib()
    assert L.fork_grpo_objective(ctypes.byref(_grpo_args(**kw))) == _binding.FORK_EINVAL
    assert L.fork_last_error().decode() != ""


@pytest.mark.parametrize("R,Lg,k,ptr,code", [
    (2, 0, 0, 16, _binding.FORK_EINVAL), (-1, 8, 1, 16, _binding.FORK_EINVAL),
    (2, 8, 9, 16, _binding.FORK_EINVAL), (2, 8, -1, 16, _binding.FORK_EINVAL),
    (2, 8, 1, 0, _binding.FORK_EINVAL), (2, 16385, 1, 16, _binding.FORK_EUNSUPPORTED),
])
def test_top_entropy_bad_arguments_rejected_on_host(R, Lg, k, ptr, code):
    L = _binding.lib()
    assert L.fork_top_entropy(ptr, R, Lg, k, ptr, None) == code


def _sel_args(**kw):
    a = _binding.ForkSelectArgs()
    good = dict(conf=16, argmax=32, tokens=48, mask=64, block_start=80, out_fallback=96,
                B=2, L=8, block_len=4, tau=0.9, rule=0)
    good.update(kw)
    for k, v in good.items():
        assert hasattr(a, k)
        setattr(a, k, v)
    return a


@pytest.mark.parametrize("kw", [
    dict(layout=2), dict(layout=-1),
    dict(conf=0), dict(argmax=0), dict(tokens=0), dict(mask=0), dict(block_start=0),
    dict(out_fallback=0), dict(B=-1), dict(L=-1), dict(block_len=0), dict(block_len=9),
    dict(tau=float("nan")), dict(rule=5), dict(rule=4), dict(rule=3),
    dict(B=1 << 16, L=1 << 16),
])
def test_select_bad_arguments_rejected_on_host(kw):
    L = _binding.lib()
    assert L.fork_select(ctypes.byref(_sel_args(**kw))) == _binding.FORK_EINVAL
    assert L.fork_last_error().decode() != ""


def test_binding_fails_loudly_without_the_library(tmp_path):
    """No CPU or PyTorch fallback: with the library missing, the first call
    raises and says how to build it."""
    import subprocess
    import sys
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from paper_2609_39859_amd import _binding\n"
        "_binding.LIB_PATH = %r\n"
        "try:\n"
        "    _binding.lib()\n"
        "except RuntimeError as e:\n"
        "    assert 'not built' in str(e), e\n"
        "    print('raised')\n" % (ROOT, str(tmp_path / "absent.so")))
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0 and out.stdout.strip() == "raised", out.stderr


def test_workspace_registry_bookkeeping(tmp_path):
    """The library-managed workspace registry (paper_2609_39859_amd/csrc/
    workspace_registry.h), compiled for the host with a fake allocator:
    one buffer per (device, stream), geometric growth that retires the old
    allocation instead of freeing it under queued work, a failed allocation
    leaving the previous buffer, concurrent host threads, and release that
    synchronises every device before freeing."""
    import shutil
    import subprocess
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no host C++ compiler")
    exe = str(tmp_path / "registry_check")
    subprocess.run([gxx, "-std=c++17", "-O1", "-Wall", "-Wextra", "-Werror", "-pthread",
                    "-I", os.path.join(ROOT, "paper_2609_39859_amd", "csrc"),
                    os.path.join(ROOT, "tests", "native", "registry_check.cpp"), "-o", exe],
                   check=True)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    assert "registry ok" in r.stdout


@pytest.mark.parametrize("kw,code", [
    (dict(workspace=256, workspace_bytes=1 << 30), _binding.FORK_EINVAL),  # no caller workspace
    (dict(workspace_bytes=1), _binding.FORK_EINVAL),
    (dict(tau=float("nan")), _binding.FORK_EINVAL),                        # same validation
    # partials of 8192 positions x 512 vocabulary tiles = 64 MiB, + candidates
    (dict(B=16, L=512, block_len=32, V=131072), _binding.FORK_EUNSUPPORTED),
    # drawn candidates double the partials
    (dict(B=8, L=512, block_len=32, V=126464, sample_temperature=0.8, ), None),
    (dict(B=16, L=512, block_len=32, V=126464, sample_temperature=0.8), _binding.FORK_EUNSUPPORTED),
])
def test_noalloc_rejections_on_host(kw, code):
    """fork_step_noalloc refuses a caller workspace and sizes beyond its
    static scratch before any HIP call (the pointers are never used)."""
    L = _binding.lib()
    if code is None:
        # fits: the scratch size check passes (the LLaDA-8B shape with drawn
        # candidates needs 2 x 32.4 MB of partials + 32 KB)
        assert L.fork_workspace_bytes(8, 512, 126464) <= _binding.FORK_NOALLOC_SCRATCH_BYTES
        return
    assert L.fork_step_noalloc(ctypes.byref(_args(**kw))) == code
    msg = L.fork_last_error().decode()
    assert msg != ""
    if code == _binding.FORK_EUNSUPPORTED:
        assert "scratch" in msg


def test_noalloc_empty_batch_is_a_no_op():
    L = _binding.lib()
    nulls = dict(hidden=0, W_head=0, tokens=0, mask=0, block_start=0, out_conf=0,
                 out_entropy=0, out_logp=0, out_fallback=0, B=0)
    assert L.fork_step_noalloc(ctypes.byref(_args(**nulls))) == _binding.FORK_OK


def test_plain_c_caller(tmp_path):
    """tests/native/abi_c_caller.c: the public header compiles as C99
    (-pedantic), the library links from C, and host-side validation answers
    through fork_step_ex / fork_last_error without a GPU."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no host C compiler")
    exe = str(tmp_path / "abi_c_caller")
    lib_dir = os.path.dirname(_binding.LIB_PATH)
    subprocess.run([gcc, "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror",
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "native", "abi_c_caller.c"), "-L", lib_dir,
                    "-lforkstep", "-Wl,-rpath," + lib_dir, "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 0, (r.returncode, r.stderr)
    assert "c abi ok" in r.stdout
