"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
rejects bad arguments on the host before touching a device.  No kernel runs
here (none of these calls gets past argument validation)."""
import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))
LIB = os.path.join(ROOT, "paper_2512_22737_amd", "libwedlm.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB),
                                reason="libwedlm.so not built")


def declared_symbols():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wedlm_\w+)\s*\(", text)))


def test_header_declares_the_four_calls():
    syms = declared_symbols()
    for name in ["wedlm_reorder", "wedlm_window_attn", "wedlm_score",
                 "wedlm_commit"]:
        assert name in syms


def test_every_declared_symbol_is_exported():
    import torch  # noqa: F401  (same runtime as the GPU path)
    lib = ctypes.CDLL(LIB)
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_binding_names_match_header():
    from paper_2512_22737_amd import wedlm
    assert sorted(wedlm.EXPORTED) == declared_symbols()
    for name in declared_symbols():
        assert callable(getattr(wedlm, name))


def _lib():
    from paper_2512_22737_amd import wedlm
    return wedlm.lib()


def test_version_and_strerror():
    lib = _lib()
    assert lib.wedlm_version() >= 100
    assert lib.wedlm_strerror(0) == b"ok"
    assert b"workspace" in lib.wedlm_strerror(-3)
    assert lib.wedlm_strerror(12345) == b"unknown error code"


def _fake():
    # a non-null address that is never dereferenced: validation fails first
    return ctypes.c_void_p(0x1000)


def test_reorder_rejects_bad_arguments():
    lib = _lib()
    f = _fake()
    # `args` is valid and is never passed as is: only the broken variants
    # below are called, and each fails validation before any launch
    args = [f, f, f, 1, 16, 4, 2, 64, 1e6] + [f] * 7 + [None]
    bad = list(args)
    bad[0] = None
    assert lib.wedlm_reorder(*bad) == -1           # null pointer
    bad = list(args)
    bad[4] = 65
    assert lib.wedlm_reorder(*bad) == -2           # W > 64
    bad = list(args)
    bad[7] = 96
    assert lib.wedlm_reorder(*bad) == -2           # D not in {64, 128}
    bad = list(args)
    bad[5] = 5
    assert lib.wedlm_reorder(*bad) == -2           # Hq % Hkv != 0
    bad = list(args)
    bad[8] = 0.5
    assert lib.wedlm_reorder(*bad) == -1           # theta <= 1


def test_attn_workspace_plan():
    lib = _lib()
    ws = lib.wedlm_window_attn_workspace_size
    # a single split needs no workspace
    assert ws(1, 16, 4, 2, 64, 256) == 0
    # the long-prefix shape splits the prefix and needs partials
    n = ws(8, 64, 32, 8, 128, 32768)
    assert n > 0 and n % 4 == 0
    # invalid shapes report 0
    assert ws(1, 65, 32, 8, 128, 100) == 0
    assert ws(1, 16, 32, 8, 96, 100) == 0


def test_attn_rejects_small_workspace():
    lib = _lib()
    f = _fake()
    need = lib.wedlm_window_attn_workspace_size(8, 64, 32, 8, 128, 32768)
    code = lib.wedlm_window_attn(f, f, f, f, f, 100, f, 2100, f, 8, 64, 32, 8,
                                 128, 32768, 0.088, f, None, None, f,
                                 need - 1, None)
    assert code == -3
    code = lib.wedlm_window_attn(f, f, f, f, f, 100, f, 2100, f, 8, 64, 32, 8,
                                 128, 32768, -1.0, f, None, None, f, need,
                                 None)
    assert code == -1                              # bad softmax scale


def test_score_rejects_bad_arguments():
    lib = _lib()
    f = _fake()
    assert lib.wedlm_score(f, 100, f, 1, 16, 100, 0.0, f, f, None, None, 0,
                           None) == -1             # temperature 0
    assert lib.wedlm_score(f, 99, f, 1, 16, 100, 0.1, f, f, None, None, 0,
                           None) == -2             # row stride < V
    need = lib.wedlm_score_workspace_size(1, 32, 151936)
    assert need > 0
    assert lib.wedlm_score(f, 151936, f, 1, 32, 151936, 0.1, f, f, None, f,
                           need - 1, None) == -3


def test_commit_rejects_bad_arguments():
    lib = _lib()
    f = _fake()
    args = [f, f, f, f, 0.9, 0.01, f, f, f, f, 100, f, 10, 1, 16, 2, 64,
            f, f, f, f, f, None]
    bad = list(args)
    bad[4] = float("nan")
    assert lib.wedlm_commit(*bad) == -1
    bad = list(args)
    bad[14] = 0
    assert lib.wedlm_commit(*bad) == -2
    bad = list(args)
    bad[21] = None
    assert lib.wedlm_commit(*bad) == -1            # status is required


def test_reorder_gather_outputs_all_or_none():
    lib = _lib()
    f = _fake()
    # indices only needs qkv_in and the three outputs all NULL; a mix fails
    args = [f, f, None, 1, 16, 4, 2, 64, 1e6] + [f] * 4 + [f, None, None,
                                                          None]
    assert lib.wedlm_reorder(*args) == -1


def _cfg(**kw):
    from paper_2512_22737_amd import wedlm
    d = dict(L=2, Hd=256, Hq=4, Hkv=2, D=64, I=512, V=1000, mask_token=999)
    d.update(kw)
    return wedlm.model_config(**d)


def test_model_workspace_and_config_checks():
    lib = _lib()
    ws = lib.wedlm_model_workspace_size
    good = _cfg()
    n = ws(ctypes.byref(good), 2, 16, 300)
    assert n > 0 and n % 256 == 0
    # hidden not a multiple of 256, bad head dim, mask token outside V, W > 64
    for bad in (_cfg(Hd=320), _cfg(D=96), _cfg(mask_token=1000),
                _cfg(Hq=5)):
        assert ws(ctypes.byref(bad), 2, 16, 300) == 0
    assert ws(ctypes.byref(good), 2, 65, 300) == 0
    assert ws(None, 2, 16, 300) == 0


def test_linear_and_small_kernels_reject_bad_arguments():
    lib = _lib()
    f = _fake()
    lin = lambda *a: lib.wedlm_linear(*a, None, 0, None)
    assert lin(f, f, 4, 48, 256, 0, f, 48) == -2      # N % 32
    assert lin(f, f, 4, 64, 200, 0, f, 64) == -2      # K % 64
    assert lin(f, f, 4, 64, 256, 3, f, 64) == -1      # epilogue
    assert lin(f, f, 4, 64, 256, 0, f, 32) == -2      # ldo < N
    assert lin(None, f, 4, 64, 256, 0, f, 64) == -1
    # N = 4096 at 32 rows splits K over workgroups: a workspace is needed
    need = lib.wedlm_linear_workspace_size(32, 4096, 4096, 1)
    assert need > 0
    assert lin(f, f, 32, 4096, 4096, 1, f, 4096) == -3
    assert lib.wedlm_linear(f, f, 32, 4096, 4096, 1, f, 4096, f, need - 1,
                            None) == -3
    assert lib.wedlm_linear_workspace_size(32, 48, 256, 0) == 0
    assert lib.wedlm_rmsnorm(f, f, 4, 256, 0.0, f, None) == -1       # eps
    assert lib.wedlm_rmsnorm(f, f, 4, 254, 1e-6, f, None) == -2
    assert lib.wedlm_embed(f, 4, 1000, f, 1000, 256, f, None) == -2  # mask id
    assert lib.wedlm_qk_norm_rope(f, f, f, f, 4, 4, 2, 96, 1e6, 1e-6, f, f,
                                  f, None) == -2
    assert lib.wedlm_qk_norm_rope(f, f, f, f, 4, 4, 2, 64, 1.0, 1e-6, f, f,
                                  f, None) == -1


def test_model_forward_and_commit_layers_reject_bad_arguments():
    from paper_2512_22737_amd import wedlm
    lib = _lib()
    f = _fake()
    cfg = _cfg()
    w = wedlm.ModelWeights(*([0x1000] * len(wedlm.WEIGHT_NAMES)))
    need = lib.wedlm_model_workspace_size(ctypes.byref(cfg), 2, 16, 300)
    args = [ctypes.byref(cfg), ctypes.byref(w), f, f, 2, 16, f, f, 100, f, 20,
            300, 0.1] + [f] * 4 + [f, f, f, f, None, f, f, need, None]
    bad = list(args)
    bad[-2] = need - 1
    assert lib.wedlm_model_forward(*bad) == -3
    bad = list(args)
    bad[12] = 0.0
    assert lib.wedlm_model_forward(*bad) == -1     # temperature
    w0 = wedlm.ModelWeights(*([0x1000] * (len(wedlm.WEIGHT_NAMES) - 1) + [0]))
    bad = list(args)
    bad[1] = ctypes.byref(w0)
    assert lib.wedlm_model_forward(*bad) == -1     # lm_head missing
    cargs = [f, f, f, f, 0.9, 0.01, f, f, f, f, 100, f, 10, 2, 16, 2, 64, 2,
             f, f, f, f, f, 0, None]
    bad = list(cargs)
    bad[17] = 0
    assert lib.wedlm_commit_layers(*bad) == -2     # no layers
    bad = list(cargs)
    bad[23] = 7
    assert lib.wedlm_commit_layers(*bad) == -1     # unknown rule
