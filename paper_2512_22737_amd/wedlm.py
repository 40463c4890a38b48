"""Thin Python binding of libwedlm.so (include/wedlm.h).

Argument marshalling only: each function checks the tensors it is handed
(device, dtype, contiguity, shape), reads the sizes off them and calls the C
entry point of the same name on torch's current HIP stream.  Every step of
the computation runs in the library's HIP kernels; there is no fallback.
torch is imported first so that the library binds to the HIP runtime torch
already loaded (one runtime, one set of streams and pointers).
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwedlm.so")

WEDLM_OK = 0
MASK_TOKEN = -1
PAGE_SIZE = 16
MAX_WINDOW = 64
SEQ_CAPACITY, SEQ_BAD_PAGE, SEQ_BAD_LEN = 1, 2, 4

_lib = None


class WedlmError(RuntimeError):
    pass


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise WedlmError(
            f"{LIB_PATH} is missing: build it with "
            "`python -m paper_2512_22737_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F, D_, SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                              ctypes.c_float, ctypes.c_double, ctypes.c_size_t)
    lib.wedlm_reorder.argtypes = [P, P, P, I32, I32, I32, I32, I32, D_, P, P,
                                  P, P, P, P, P, P]
    lib.wedlm_reorder.restype = ctypes.c_int
    lib.wedlm_window_attn_workspace_size.argtypes = [I32] * 6
    lib.wedlm_window_attn_workspace_size.restype = SZ
    lib.wedlm_window_attn.argtypes = [P, P, P, P, P, I64, P, I32, P, I32, I32,
                                      I32, I32, I32, I32, F, P, P, P, P, SZ,
                                      P]
    lib.wedlm_window_attn.restype = ctypes.c_int
    lib.wedlm_score_workspace_size.argtypes = [I32, I32, I32]
    lib.wedlm_score_workspace_size.restype = SZ
    lib.wedlm_score.argtypes = [P, I64, P, I32, I32, I32, D_, P, P, P, P, SZ,
                                P]
    lib.wedlm_score.restype = ctypes.c_int
    lib.wedlm_commit.argtypes = [P, P, P, P, D_, D_, P, P, P, P, I64, P, I32,
                                 I32, I32, I32, I32, P, P, P, P, P, P]
    lib.wedlm_commit.restype = ctypes.c_int
    lib.wedlm_commit_rule.argtypes = [P, P, P, P, D_, D_, P, P, P, P, I64, P,
                                      I32, I32, I32, I32, I32, P, P, P, P, P,
                                      I32, P]
    lib.wedlm_commit_rule.restype = ctypes.c_int
    lib.wedlm_lm_head_score_workspace_size.argtypes = [I32, I32, I32]
    lib.wedlm_lm_head_score_workspace_size.restype = SZ
    lib.wedlm_lm_head_score.argtypes = [P, P, I32, I32, I32, D_, P, P, P, P,
                                        SZ, P]
    lib.wedlm_lm_head_score.restype = ctypes.c_int
    lib.wedlm_strerror.argtypes = [ctypes.c_int]
    lib.wedlm_strerror.restype = ctypes.c_char_p
    lib.wedlm_version.argtypes = []
    lib.wedlm_version.restype = ctypes.c_int
    _lib = lib
    return lib


def lib():
    return _load()


EXPORTED = ["wedlm_reorder", "wedlm_window_attn_workspace_size",
            "wedlm_window_attn", "wedlm_score_workspace_size", "wedlm_score",
            "wedlm_commit", "wedlm_commit_rule",
            "wedlm_lm_head_score_workspace_size", "wedlm_lm_head_score",
            "wedlm_strerror", "wedlm_version"]

# decoding rules of wedlm_commit_rule (include/wedlm.h)
RULE_STREAMING, RULE_BLOCK, RULE_ONE_TOKEN = 0, 1, 2
RULES = {"stream": RULE_STREAMING, "block": RULE_BLOCK, "one": RULE_ONE_TOKEN}


def _check(code: int, what: str):
    if code != WEDLM_OK:
        msg = _load().wedlm_strerror(code).decode()
        raise WedlmError(f"{what} failed: {msg} ({code})")


_BF16 = (torch.bfloat16, torch.int16, torch.uint16)


def _t(x: Optional[torch.Tensor], name: str, dtypes, shape=None,
       allow_none=False):
    if x is None:
        if allow_none:
            return None
        raise WedlmError(f"{name} is required")
    if not x.is_cuda:
        raise WedlmError(f"{name} must be a device tensor")
    if x.dtype not in dtypes:
        raise WedlmError(f"{name}: dtype {x.dtype} not in {dtypes}")
    if not x.is_contiguous():
        raise WedlmError(f"{name} must be contiguous")
    if shape is not None and tuple(x.shape) != tuple(shape):
        raise WedlmError(f"{name}: shape {tuple(x.shape)} != {tuple(shape)}")
    return x.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def wedlm_version() -> int:
    return _load().wedlm_version()


def wedlm_strerror(code: int) -> str:
    return _load().wedlm_strerror(code).decode()


def wedlm_reorder(win_tok, win_start, qkv_in, Hq: int, Hkv: int,
                  rope_theta: float, perm, pos_ids, tok_phys, n_obs, q_phys,
                  k_phys, v_phys) -> None:
    B, W = win_tok.shape
    D = qkv_in.shape[-1]
    i32 = (torch.int32,)
    code = _load().wedlm_reorder(
        _t(win_tok, "win_tok", i32, (B, W)),
        _t(win_start, "win_start", i32, (B,)),
        _t(qkv_in, "qkv_in", _BF16, (B, W, Hq + 2 * Hkv, D)),
        B, W, Hq, Hkv, D, float(rope_theta),
        _t(perm, "perm", i32, (B, W)), _t(pos_ids, "pos_ids", i32, (B, W)),
        _t(tok_phys, "tok_phys", i32, (B, W)), _t(n_obs, "n_obs", i32, (B,)),
        _t(q_phys, "q_phys", _BF16, (B, W, Hq, D)),
        _t(k_phys, "k_phys", _BF16, (B, W, Hkv, D)),
        _t(v_phys, "v_phys", _BF16, (B, W, Hkv, D)), _stream())
    _check(code, "wedlm_reorder")


def wedlm_window_attn_workspace_size(B, W, Hq, Hkv, D, max_prefix_len) -> int:
    return int(_load().wedlm_window_attn_workspace_size(
        B, W, Hq, Hkv, D, max_prefix_len))


def wedlm_window_attn(q_phys, k_phys, v_phys, k_cache, v_cache, block_table,
                      prefix_len, max_prefix_len: int, out, lse=None,
                      status=None, workspace=None,
                      softmax_scale: Optional[float] = None) -> None:
    B, W, Hq, D = q_phys.shape
    Hkv = k_phys.shape[2]
    P = k_cache.shape[0]
    maxp = block_table.shape[1]
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    ws_need = wedlm_window_attn_workspace_size(B, W, Hq, Hkv, D,
                                               max_prefix_len)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        if not workspace.is_cuda or not workspace.is_contiguous():
            raise WedlmError("workspace must be a contiguous device tensor")
        ws_ptr = workspace.data_ptr()
        ws_bytes = workspace.numel() * workspace.element_size()
    elif ws_need:
        raise WedlmError(f"workspace of {ws_need} bytes required")
    i32 = (torch.int32,)
    code = _load().wedlm_window_attn(
        _t(q_phys, "q_phys", _BF16), _t(k_phys, "k_phys", _BF16, (B, W, Hkv, D)),
        _t(v_phys, "v_phys", _BF16, (B, W, Hkv, D)),
        _t(k_cache, "k_cache", _BF16, (P, Hkv, PAGE_SIZE, D)),
        _t(v_cache, "v_cache", _BF16, (P, Hkv, D, PAGE_SIZE)), P,
        _t(block_table, "block_table", i32, (B, maxp)), maxp,
        _t(prefix_len, "prefix_len", i32, (B,)), B, W, Hq, Hkv, D,
        int(max_prefix_len), float(softmax_scale),
        _t(out, "out", _BF16, (B, W, Hq, D)),
        _t(lse, "lse", (torch.float32,), (B, W, Hq), allow_none=True),
        _t(status, "status", i32, (B,), allow_none=True), ws_ptr, ws_bytes,
        _stream())
    _check(code, "wedlm_window_attn")


def wedlm_score_workspace_size(B, W, V) -> int:
    return int(_load().wedlm_score_workspace_size(B, W, V))


def wedlm_score(logits, n_obs, temperature: float, argmax, entropy,
                pmax=None, workspace=None, V: Optional[int] = None) -> None:
    """logits: [B, W, row_stride] fp32 (row_stride >= V); V defaults to the
    last dimension."""
    B, W, stride = logits.shape
    V = stride if V is None else V
    need = wedlm_score_workspace_size(B, W, V)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        ws_ptr = workspace.data_ptr()
        ws_bytes = workspace.numel() * workspace.element_size()
    elif need:
        raise WedlmError(f"workspace of {need} bytes required")
    i32, f32 = (torch.int32,), (torch.float32,)
    code = _load().wedlm_score(
        _t(logits, "logits", f32), stride, _t(n_obs, "n_obs", i32, (B,)),
        B, W, V, float(temperature), _t(argmax, "argmax", i32, (B, W)),
        _t(entropy, "entropy", f32, (B, W)),
        _t(pmax, "pmax", f32, (B, W), allow_none=True), ws_ptr, ws_bytes,
        _stream())
    _check(code, "wedlm_score")


def wedlm_lm_head_score_workspace_size(R, Hd, V) -> int:
    return int(_load().wedlm_lm_head_score_workspace_size(R, Hd, V))


def wedlm_lm_head_score(hidden, w_vocab, temperature: float, argmax, entropy,
                        pmax=None, workspace=None) -> None:
    """hidden [R, Hd] bf16, w_vocab [V, Hd] bf16 -> argmax [R] int32,
    entropy [R] fp32, pmax [R] fp32 (optional).  A workspace of at least
    wedlm_lm_head_score_workspace_size(R, Hd, V) bytes is allocated here if
    none is given."""
    R, Hd = hidden.shape
    V = w_vocab.shape[0]
    need = wedlm_lm_head_score_workspace_size(R, Hd, V)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=hidden.device)
    ws_ptr = None if workspace is None else workspace.data_ptr()
    ws_bytes = 0 if workspace is None else workspace.numel()
    code = _load().wedlm_lm_head_score(
        _t(hidden, "hidden", _BF16, (R, Hd)),
        _t(w_vocab, "w_vocab", _BF16, (V, Hd)), R, Hd, V, float(temperature),
        _t(argmax, "argmax", (torch.int32,), (R,)),
        _t(entropy, "entropy", (torch.float32,), (R,)),
        _t(pmax, "pmax", (torch.float32,), (R,), allow_none=True),
        ws_ptr, ws_bytes, _stream())
    _check(code, "wedlm_lm_head_score")


def _commit_args(win_tok, win_start, argmax, entropy, tau, lam, k_phys,
                 v_phys, k_cache, v_cache, block_table, n_commit,
                 committed_tok, committed_slot, selected, status):
    B, W = win_tok.shape
    Hkv, D = k_phys.shape[2], k_phys.shape[3]
    P = k_cache.shape[0]
    maxp = block_table.shape[1]
    i32 = (torch.int32,)
    return [
        _t(win_tok, "win_tok", i32, (B, W)), _t(win_start, "win_start", i32, (B,)),
        _t(argmax, "argmax", i32, (B, W)),
        _t(entropy, "entropy", (torch.float32,), (B, W)), float(tau),
        float(lam), _t(k_phys, "k_phys", _BF16, (B, W, Hkv, D)),
        _t(v_phys, "v_phys", _BF16, (B, W, Hkv, D)),
        _t(k_cache, "k_cache", _BF16, (P, Hkv, PAGE_SIZE, D)),
        _t(v_cache, "v_cache", _BF16, (P, Hkv, D, PAGE_SIZE)), P,
        _t(block_table, "block_table", i32, (B, maxp)), maxp, B, W, Hkv, D,
        _t(n_commit, "n_commit", i32, (B,)),
        _t(committed_tok, "committed_tok", i32, (B, W)),
        _t(committed_slot, "committed_slot", i32, (B, W)),
        _t(selected, "selected", (torch.uint8,), (B, W)),
        _t(status, "status", i32, (B,))]


def wedlm_commit(win_tok, win_start, argmax, entropy, tau: float, lam: float,
                 k_phys, v_phys, k_cache, v_cache, block_table, n_commit,
                 committed_tok, committed_slot, selected, status) -> None:
    args = _commit_args(win_tok, win_start, argmax, entropy, tau, lam, k_phys,
                        v_phys, k_cache, v_cache, block_table, n_commit,
                        committed_tok, committed_slot, selected, status)
    _check(_load().wedlm_commit(*args, _stream()), "wedlm_commit")


def wedlm_commit_rule(win_tok, win_start, argmax, entropy, tau: float,
                      lam: float, k_phys, v_phys, k_cache, v_cache,
                      block_table, n_commit, committed_tok, committed_slot,
                      selected, status, rule: int) -> None:
    args = _commit_args(win_tok, win_start, argmax, entropy, tau, lam, k_phys,
                        v_phys, k_cache, v_cache, block_table, n_commit,
                        committed_tok, committed_slot, selected, status)
    _check(_load().wedlm_commit_rule(*args, int(rule), _stream()),
           "wedlm_commit_rule")


class DecodeStep:
    """Device buffers for one batch and the four calls of one decode step.

    state: win_tok [B,W] int32, win_start [B] int32, k_cache/v_cache pages,
    block_table.  Per-step inputs: qkv_in [B,W,Hq+2Hkv,D] bf16 and logits
    [B,W,V] fp32 (physical row order)."""

    def __init__(self, B, W, Hq, Hkv, D, V, max_prefix_len, theta=1e6,
                 tau=0.9, lam=0.01, temperature=0.1, device="cuda",
                 rule="stream"):
        self.B, self.W, self.Hq, self.Hkv, self.D, self.V = B, W, Hq, Hkv, D, V
        self.rule = RULES[rule]
        self.theta, self.tau, self.lam, self.temperature = (theta, tau, lam,
                                                            temperature)
        self.max_prefix_len = int(max_prefix_len)
        dev = torch.device(device)
        i32 = dict(dtype=torch.int32, device=dev)
        bf = dict(dtype=torch.bfloat16, device=dev)
        self.perm = torch.empty(B, W, **i32)
        self.pos_ids = torch.empty(B, W, **i32)
        self.tok_phys = torch.empty(B, W, **i32)
        self.n_obs = torch.empty(B, **i32)
        self.q_phys = torch.empty(B, W, Hq, D, **bf)
        self.k_phys = torch.empty(B, W, Hkv, D, **bf)
        self.v_phys = torch.empty(B, W, Hkv, D, **bf)
        self.out = torch.empty(B, W, Hq, D, **bf)
        self.lse = torch.empty(B, W, Hq, dtype=torch.float32, device=dev)
        self.attn_status = torch.zeros(B, **i32)
        self.argmax = torch.full((B, W), -1, **i32)
        self.entropy = torch.full((B, W), float("nan"), dtype=torch.float32,
                                  device=dev)
        self.pmax = torch.full((B, W), float("nan"), dtype=torch.float32,
                               device=dev)
        self.n_commit = torch.empty(B, **i32)
        self.committed_tok = torch.empty(B, W, **i32)
        self.committed_slot = torch.empty(B, W, **i32)
        self.selected = torch.empty(B, W, dtype=torch.uint8, device=dev)
        self.status = torch.empty(B, **i32)
        self.set_max_prefix(self.max_prefix_len)
        nsw = wedlm_score_workspace_size(B, W, V)
        self.score_ws = torch.empty(max(nsw, 1), dtype=torch.uint8, device=dev)

    def set_max_prefix(self, max_prefix_len: int):
        self.max_prefix_len = int(max_prefix_len)
        n = wedlm_window_attn_workspace_size(self.B, self.W, self.Hq, self.Hkv,
                                             self.D, self.max_prefix_len)
        cur = getattr(self, "attn_ws", None)
        if cur is None or cur.numel() < n:
            self.attn_ws = torch.empty(max(n, 1), dtype=torch.uint8,
                                       device=self.perm.device)

    def reorder(self, win_tok, win_start, qkv_in):
        wedlm_reorder(win_tok, win_start, qkv_in, self.Hq, self.Hkv,
                      self.theta, self.perm, self.pos_ids, self.tok_phys,
                      self.n_obs, self.q_phys, self.k_phys, self.v_phys)

    def attn(self, k_cache, v_cache, block_table, win_start):
        wedlm_window_attn(self.q_phys, self.k_phys, self.v_phys, k_cache,
                          v_cache, block_table, win_start,
                          self.max_prefix_len, self.out, self.lse,
                          self.attn_status, self.attn_ws)

    def score(self, logits):
        wedlm_score(logits, self.n_obs, self.temperature, self.argmax,
                    self.entropy, self.pmax, self.score_ws, V=self.V)

    def commit(self, win_tok, win_start, k_cache, v_cache, block_table):
        args = (win_tok, win_start, self.argmax, self.entropy, self.tau,
                self.lam, self.k_phys, self.v_phys, k_cache, v_cache,
                block_table, self.n_commit, self.committed_tok,
                self.committed_slot, self.selected, self.status)
        if self.rule == RULE_STREAMING:
            wedlm_commit(*args)
        else:
            wedlm_commit_rule(*args, self.rule)

    def __call__(self, win_tok, win_start, qkv_in, logits, k_cache, v_cache,
                 block_table):
        self.reorder(win_tok, win_start, qkv_in)
        self.attn(k_cache, v_cache, block_table, win_start)
        self.score(logits)
        self.commit(win_tok, win_start, k_cache, v_cache, block_table)
