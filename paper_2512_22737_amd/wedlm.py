"""Thin Python binding of libwedlm.so (include/wedlm.h, include/wedlm_model.h,
include/wedlm_train.h).

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
    lib.wedlm_window_attn_noalloc.argtypes = [P, P, P, P, P, I64, P, I32, P,
                                              I32, I32, I32, I32, I32, I32, F,
                                              P, P, P, P]
    lib.wedlm_window_attn_noalloc.restype = ctypes.c_int
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
    lib.wedlm_embed.argtypes = [P, I32, I32, P, I32, I32, P, P]
    lib.wedlm_embed.restype = ctypes.c_int
    lib.wedlm_rmsnorm.argtypes = [P, P, I32, I32, F, P, P]
    lib.wedlm_rmsnorm.restype = ctypes.c_int
    lib.wedlm_pack_weights.argtypes = [P, I64, I32, P, P]
    lib.wedlm_pack_weights.restype = ctypes.c_int
    lib.wedlm_linear_workspace_size.argtypes = [I32, I32, I32, I32]
    lib.wedlm_linear_workspace_size.restype = SZ
    lib.wedlm_linear.argtypes = [P, P, I32, I32, I32, I32, P, I32, P, SZ, P]
    lib.wedlm_linear.restype = ctypes.c_int
    lib.wedlm_qk_norm_rope.argtypes = [P, P, P, P, I32, I32, I32, I32, D_, F,
                                       P, P, P, P]
    lib.wedlm_qk_norm_rope.restype = ctypes.c_int
    lib.wedlm_model_workspace_size.argtypes = [P, I32, I32, I32]
    lib.wedlm_model_workspace_size.restype = SZ
    lib.wedlm_model_forward.argtypes = [P, P, P, P, I32, I32, P, P, I64, P,
                                        I32, I32, D_, P, P, P, P, P, P, P, P,
                                        P, P, P, SZ, P]
    lib.wedlm_model_forward.restype = ctypes.c_int
    lib.wedlm_commit_layers.argtypes = [P, P, P, P, D_, D_, P, P, P, P, I64,
                                        P, I32, I32, I32, I32, I32, I32, P, P,
                                        P, P, P, I32, P]
    lib.wedlm_commit_layers.restype = ctypes.c_int
    lib.wedlm_dual_stream_attn_workspace_size.argtypes = [I32] * 6
    lib.wedlm_dual_stream_attn_workspace_size.restype = SZ
    lib.wedlm_dual_stream_attn.argtypes = [P, P, P, I32, I32, I32, I32, I32,
                                           I32, F, P, P, P, SZ, P]
    lib.wedlm_dual_stream_attn.restype = ctypes.c_int
    lib.wedlm_strerror.argtypes = [ctypes.c_int]
    lib.wedlm_strerror.restype = ctypes.c_char_p
    lib.wedlm_version.argtypes = []
    lib.wedlm_version.restype = ctypes.c_int
    _lib = lib
    return lib


def lib():
    return _load()


EXPORTED = ["wedlm_reorder", "wedlm_window_attn_workspace_size",
            "wedlm_window_attn", "wedlm_window_attn_noalloc",
            "wedlm_score_workspace_size", "wedlm_score",
            "wedlm_commit", "wedlm_commit_rule",
            "wedlm_lm_head_score_workspace_size", "wedlm_lm_head_score",
            "wedlm_strerror", "wedlm_version", "wedlm_embed", "wedlm_rmsnorm",
            "wedlm_linear", "wedlm_linear_workspace_size",
            "wedlm_pack_weights", "wedlm_qk_norm_rope",
            "wedlm_model_workspace_size",
            "wedlm_model_forward", "wedlm_commit_layers",
            "wedlm_dual_stream_attn_workspace_size", "wedlm_dual_stream_attn"]

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
                  k_phys, v_phys, D: Optional[int] = None) -> None:
    """qkv_in, q_phys, k_phys, v_phys all None: indices only (D then sizes
    the argument check alone)."""
    B, W = win_tok.shape
    none = qkv_in is None
    D = (D or 128) if none else qkv_in.shape[-1]
    i32 = (torch.int32,)
    code = _load().wedlm_reorder(
        _t(win_tok, "win_tok", i32, (B, W)),
        _t(win_start, "win_start", i32, (B,)),
        _t(qkv_in, "qkv_in", _BF16, (B, W, Hq + 2 * Hkv, D), allow_none=none),
        B, W, Hq, Hkv, D, float(rope_theta),
        _t(perm, "perm", i32, (B, W)), _t(pos_ids, "pos_ids", i32, (B, W)),
        _t(tok_phys, "tok_phys", i32, (B, W)), _t(n_obs, "n_obs", i32, (B,)),
        _t(q_phys, "q_phys", _BF16, (B, W, Hq, D), allow_none=none),
        _t(k_phys, "k_phys", _BF16, (B, W, Hkv, D), allow_none=none),
        _t(v_phys, "v_phys", _BF16, (B, W, Hkv, D), allow_none=none),
        _stream())
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


def wedlm_window_attn_noalloc(q_phys, k_phys, v_phys, k_cache, v_cache,
                              block_table, prefix_len, max_prefix_len: int,
                              out, lse=None, status=None,
                              softmax_scale: Optional[float] = None) -> None:
    """wedlm_window_attn with the library's own scratch array in place of a
    workspace (include/wedlm.h); nothing is allocated."""
    B, W, Hq, D = q_phys.shape
    Hkv = k_phys.shape[2]
    P = k_cache.shape[0]
    maxp = block_table.shape[1]
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    i32 = (torch.int32,)
    code = _load().wedlm_window_attn_noalloc(
        _t(q_phys, "q_phys", _BF16), _t(k_phys, "k_phys", _BF16, (B, W, Hkv, D)),
        _t(v_phys, "v_phys", _BF16, (B, W, Hkv, D)),
        _t(k_cache, "k_cache", _BF16, (P, Hkv, PAGE_SIZE, D)),
        _t(v_cache, "v_cache", _BF16, (P, Hkv, D, PAGE_SIZE)), P,
        _t(block_table, "block_table", i32, (B, maxp)), maxp,
        _t(prefix_len, "prefix_len", i32, (B,)), B, W, Hq, Hkv, D,
        int(max_prefix_len), float(softmax_scale),
        _t(out, "out", _BF16, (B, W, Hq, D)),
        _t(lse, "lse", (torch.float32,), (B, W, Hq), allow_none=True),
        _t(status, "status", i32, (B,), allow_none=True), _stream())
    _check(code, "wedlm_window_attn_noalloc")


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


# ---------------------------------------------------------------------------
# the decoder around the step (include/wedlm_model.h)
# ---------------------------------------------------------------------------

EPI_STORE_BF16, EPI_ADD_F32, EPI_SWIGLU = 0, 1, 2


class ModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("mask_token", ctypes.c_int32),
                ("rope_theta", ctypes.c_double), ("rms_eps", ctypes.c_float)]


WEIGHT_NAMES = ("embed", "attn_norm", "w_qkv", "q_norm", "k_norm", "w_o",
                "mlp_norm", "w_gate_up", "w_down", "final_norm", "lm_head")


class ModelWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_NAMES]


def model_config(L, Hd, Hq, Hkv, D, I, V, mask_token, theta=1e6, eps=1e-6):
    return ModelConfig(L, Hd, Hq, Hkv, D, I, V, mask_token, float(theta),
                       float(eps))


def weight_shapes(cfg: ModelConfig):
    L, Hd, Hq, Hkv = cfg.n_layers, cfg.hidden, cfg.n_heads, cfg.n_kv_heads
    D, I, V = cfg.head_dim, cfg.inter, cfg.vocab
    return {"embed": (V, Hd), "attn_norm": (L, Hd),
            "w_qkv": (L, (Hq + 2 * Hkv) * D, Hd), "q_norm": (L, D),
            "k_norm": (L, D), "w_o": (L, Hd, Hq * D), "mlp_norm": (L, Hd),
            "w_gate_up": (L, 2 * I, Hd), "w_down": (L, Hd, I),
            "final_norm": (Hd,), "lm_head": (V, Hd)}


def model_weights(cfg: ModelConfig, tensors: dict) -> ModelWeights:
    """Check the weight tensors against the config and point the struct at
    them (the caller keeps the tensors alive)."""
    shapes = weight_shapes(cfg)
    return ModelWeights(*[_t(tensors[n], n, _BF16, shapes[n])
                          for n in WEIGHT_NAMES])


def wedlm_embed(tok, mask_token: int, table, x) -> None:
    M = tok.numel()
    V, Hd = table.shape
    code = _load().wedlm_embed(
        _t(tok, "tok", (torch.int32,)), M, int(mask_token),
        _t(table, "table", _BF16), V, Hd,
        _t(x, "x", (torch.float32,), (M, Hd)), _stream())
    _check(code, "wedlm_embed")


def wedlm_rmsnorm(x, gain, eps: float, y) -> None:
    M, Hd = x.shape
    code = _load().wedlm_rmsnorm(
        _t(x, "x", (torch.float32,)), _t(gain, "gain", _BF16, (Hd,)), M, Hd,
        float(eps), _t(y, "y", _BF16, (M, Hd)), _stream())
    _check(code, "wedlm_rmsnorm")


def wedlm_pack_weights(w, packed) -> None:
    """Row-major w [rows, K] -> the packed MFMA-tile layout (same shape)."""
    rows, K = w.shape
    code = _load().wedlm_pack_weights(
        _t(w, "w", _BF16), rows, K, _t(packed, "packed", _BF16, (rows, K)),
        _stream())
    _check(code, "wedlm_pack_weights")


def pack(w):
    """A packed copy of a row-major weight matrix (or a stack of them, each
    matrix packed on its own)."""
    out = torch.empty_like(w)
    if w.dim() == 2:
        wedlm_pack_weights(w, out)
    else:
        for i in range(w.shape[0]):
            wedlm_pack_weights(w[i], out[i])
    return out


PACKED = ("w_qkv", "w_o", "w_gate_up", "w_down")


def wedlm_linear_workspace_size(M, N, K, epilogue) -> int:
    return int(_load().wedlm_linear_workspace_size(M, N, K, epilogue))


def wedlm_linear(x, w, epilogue: int, out, workspace=None) -> None:
    """out = x w^T with the epilogue of include/wedlm_model.h; x [M, K],
    w [rows, K] packed (pack()), rows = 2N for SwiGLU; out [M, ldo] with
    ldo >= N.  A workspace is allocated here if one is needed and none is
    given."""
    M, K = x.shape
    rows = w.shape[0]
    N = rows // 2 if epilogue == EPI_SWIGLU else rows
    odt = (torch.float32,) if epilogue == EPI_ADD_F32 else _BF16
    if out.dim() != 2 or out.shape[0] != M:
        raise WedlmError(f"out: shape {tuple(out.shape)} is not [{M}, >= {N}]")
    need = wedlm_linear_workspace_size(M, N, K, epilogue)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    code = _load().wedlm_linear(
        _t(x, "x", _BF16), _t(w, "w", _BF16, (rows, K)), M, N, K,
        int(epilogue), _t(out, "out", odt), out.shape[1],
        None if workspace is None else workspace.data_ptr(),
        0 if workspace is None else workspace.numel(), _stream())
    _check(code, "wedlm_linear")


def wedlm_qk_norm_rope(qkv, q_gain, k_gain, pos_ids, Hq: int, Hkv: int,
                       rope_theta: float, eps: float, q_out, k_out,
                       v_out) -> None:
    M = qkv.shape[0]
    D = q_gain.shape[0]
    i32 = (torch.int32,)
    code = _load().wedlm_qk_norm_rope(
        _t(qkv, "qkv", _BF16, (M, (Hq + 2 * Hkv) * D)),
        _t(q_gain, "q_gain", _BF16, (D,)), _t(k_gain, "k_gain", _BF16, (D,)),
        _t(pos_ids, "pos_ids", i32), M, Hq, Hkv, D, float(rope_theta),
        float(eps), _t(q_out, "q_out", _BF16), _t(k_out, "k_out", _BF16),
        _t(v_out, "v_out", _BF16), _stream())
    _check(code, "wedlm_qk_norm_rope")


def wedlm_model_workspace_size(cfg: ModelConfig, B: int, W: int,
                               max_prefix_len: int) -> int:
    return int(_load().wedlm_model_workspace_size(ctypes.byref(cfg), B, W,
                                                  max_prefix_len))


def wedlm_model_forward(cfg: ModelConfig, weights: ModelWeights, win_tok,
                        win_start, k_cache, v_cache, block_table,
                        max_prefix_len: int, temperature: float, perm,
                        pos_ids, tok_phys, n_obs, k_win, v_win, argmax,
                        entropy, pmax, status, workspace) -> None:
    B, W = win_tok.shape
    L, Hkv, D = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
    P = k_cache.shape[1]
    maxp = block_table.shape[1]
    i32, f32 = (torch.int32,), (torch.float32,)
    code = _load().wedlm_model_forward(
        ctypes.byref(cfg), ctypes.byref(weights),
        _t(win_tok, "win_tok", i32, (B, W)),
        _t(win_start, "win_start", i32, (B,)), B, W,
        _t(k_cache, "k_cache", _BF16, (L, P, Hkv, PAGE_SIZE, D)),
        _t(v_cache, "v_cache", _BF16, (L, P, Hkv, D, PAGE_SIZE)), P,
        _t(block_table, "block_table", i32, (B, maxp)), maxp,
        int(max_prefix_len), float(temperature),
        _t(perm, "perm", i32, (B, W)), _t(pos_ids, "pos_ids", i32, (B, W)),
        _t(tok_phys, "tok_phys", i32, (B, W)), _t(n_obs, "n_obs", i32, (B,)),
        _t(k_win, "k_win", _BF16, (L, B, W, Hkv, D)),
        _t(v_win, "v_win", _BF16, (L, B, W, Hkv, D)),
        _t(argmax, "argmax", i32, (B, W)), _t(entropy, "entropy", f32, (B, W)),
        _t(pmax, "pmax", f32, (B, W), allow_none=True),
        _t(status, "status", i32, (B,)), _t(workspace, "workspace",
                                            (torch.uint8,)),
        workspace.numel(), _stream())
    _check(code, "wedlm_model_forward")


def wedlm_commit_layers(win_tok, win_start, argmax, entropy, tau: float,
                        lam: float, k_win, v_win, k_cache, v_cache,
                        block_table, n_commit, committed_tok, committed_slot,
                        selected, status, rule: int = RULE_STREAMING) -> None:
    B, W = win_tok.shape
    L, _, _, Hkv, D = k_win.shape
    P = k_cache.shape[1]
    maxp = block_table.shape[1]
    i32 = (torch.int32,)
    code = _load().wedlm_commit_layers(
        _t(win_tok, "win_tok", i32, (B, W)),
        _t(win_start, "win_start", i32, (B,)),
        _t(argmax, "argmax", i32, (B, W)),
        _t(entropy, "entropy", (torch.float32,), (B, W)), float(tau),
        float(lam), _t(k_win, "k_win", _BF16, (L, B, W, Hkv, D)),
        _t(v_win, "v_win", _BF16, (L, B, W, Hkv, D)),
        _t(k_cache, "k_cache", _BF16, (L, P, Hkv, PAGE_SIZE, D)),
        _t(v_cache, "v_cache", _BF16, (L, P, Hkv, D, PAGE_SIZE)), P,
        _t(block_table, "block_table", i32, (B, maxp)), maxp, B, W, Hkv, D, L,
        _t(n_commit, "n_commit", i32, (B,)),
        _t(committed_tok, "committed_tok", i32, (B, W)),
        _t(committed_slot, "committed_slot", i32, (B, W)),
        _t(selected, "selected", (torch.uint8,), (B, W)),
        _t(status, "status", i32, (B,)), int(rule), _stream())
    _check(code, "wedlm_commit_layers")


class Decoder:
    """A decoder's device state for B sequences and the two calls of one
    streaming step (wedlm_model_forward, wedlm_commit_layers).

    weights: dict of bf16 device tensors (WEIGHT_NAMES, weight_shapes()),
    all row-major unless packed=True says the projections (PACKED) are
    already in the layout of wedlm_pack_weights; row-major ones are packed
    here into copies.
    Caches: [L, num_pages, ...]; each sequence owns the pages its block-table
    row lists.  The window state (win_tok, win_start) lives here and is
    updated in place by step()."""

    def __init__(self, cfg: ModelConfig, weights: dict, B: int, W: int,
                 num_pages: int, block_table, max_prefix_len: int,
                 tau=0.9, lam=0.01, temperature=0.1, rule="stream",
                 device="cuda", packed=False):
        self.cfg, self.B, self.W = cfg, B, W
        if not packed:
            weights = dict(weights)
            for n in PACKED:
                weights[n] = pack(weights[n])
        self.tensors = weights
        self.weights = model_weights(cfg, weights)
        self.tau, self.lam, self.temperature = tau, lam, temperature
        self.rule = RULES[rule]
        self.max_prefix_len = int(max_prefix_len)
        dev = torch.device(device)
        L, Hkv, D = cfg.n_layers, cfg.n_kv_heads, cfg.head_dim
        i32 = dict(dtype=torch.int32, device=dev)
        bf = dict(dtype=torch.bfloat16, device=dev)
        self.k_cache = torch.zeros(L, num_pages, Hkv, PAGE_SIZE, D, **bf)
        self.v_cache = torch.zeros(L, num_pages, Hkv, D, PAGE_SIZE, **bf)
        self.block_table = block_table
        self.win_tok = torch.full((B, W), MASK_TOKEN, **i32)
        self.win_start = torch.zeros(B, **i32)
        self.perm = torch.empty(B, W, **i32)
        self.pos_ids = torch.empty(B, W, **i32)
        self.tok_phys = torch.empty(B, W, **i32)
        self.n_obs = torch.empty(B, **i32)
        self.k_win = torch.empty(L, B, W, Hkv, D, **bf)
        self.v_win = torch.empty(L, B, W, Hkv, D, **bf)
        self.argmax = torch.empty(B, W, **i32)
        self.entropy = torch.empty(B, W, dtype=torch.float32, device=dev)
        self.pmax = torch.empty(B, W, dtype=torch.float32, device=dev)
        self.attn_status = torch.zeros(B, **i32)
        self.n_commit = torch.empty(B, **i32)
        self.committed_tok = torch.empty(B, W, **i32)
        self.committed_slot = torch.empty(B, W, **i32)
        self.selected = torch.empty(B, W, dtype=torch.uint8, device=dev)
        self.status = torch.zeros(B, **i32)
        n = wedlm_model_workspace_size(cfg, B, W, self.max_prefix_len)
        if n == 0:
            raise WedlmError("invalid decoder configuration")
        self.workspace = torch.empty(n, dtype=torch.uint8, device=dev)

    def forward(self):
        wedlm_model_forward(
            self.cfg, self.weights, self.win_tok, self.win_start,
            self.k_cache, self.v_cache, self.block_table,
            self.max_prefix_len, self.temperature, self.perm, self.pos_ids,
            self.tok_phys, self.n_obs, self.k_win, self.v_win, self.argmax,
            self.entropy, self.pmax, self.attn_status, self.workspace)

    def commit(self):
        wedlm_commit_layers(
            self.win_tok, self.win_start, self.argmax, self.entropy,
            self.tau, self.lam, self.k_win, self.v_win, self.k_cache,
            self.v_cache, self.block_table, self.n_commit,
            self.committed_tok, self.committed_slot, self.selected,
            self.status, self.rule)

    def step(self):
        self.forward()
        self.commit()


# ---------------------------------------------------------------------------
# training-time attention (include/wedlm_train.h)
# ---------------------------------------------------------------------------

def wedlm_dual_stream_attn_workspace_size(n_seq, L, block, Hq, Hkv, D) -> int:
    return int(_load().wedlm_dual_stream_attn_workspace_size(
        n_seq, L, block, Hq, Hkv, D))


def wedlm_dual_stream_attn(q, k, v, block: int, out, lse=None, workspace=None,
                           softmax_scale: Optional[float] = None) -> None:
    """q [n_seq, 2L, Hq, D], k, v [n_seq, 2L, Hkv, D] bf16 in the physical
    layout of include/wedlm_train.h -> out [n_seq, 2L, Hq, D] bf16, lse
    [n_seq, 2L, Hq] fp32 (optional).  A workspace is allocated here if none
    is given."""
    n_seq, L2, Hq, D = q.shape
    Hkv = k.shape[2]
    L = L2 // 2
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    need = wedlm_dual_stream_attn_workspace_size(n_seq, L, block, Hq, Hkv, D)
    if need == 0:
        raise WedlmError("unsupported dual-stream shape")
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    code = _load().wedlm_dual_stream_attn(
        _t(q, "q", _BF16, (n_seq, 2 * L, Hq, D)),
        _t(k, "k", _BF16, (n_seq, 2 * L, Hkv, D)),
        _t(v, "v", _BF16, (n_seq, 2 * L, Hkv, D)), n_seq, L, int(block), Hq,
        Hkv, D, float(softmax_scale), _t(out, "out", _BF16, (n_seq, 2 * L, Hq, D)),
        _t(lse, "lse", (torch.float32,), (n_seq, 2 * L, Hq), allow_none=True),
        _t(workspace, "workspace", (torch.uint8,)), workspace.numel(),
        _stream())
    _check(code, "wedlm_dual_stream_attn")
