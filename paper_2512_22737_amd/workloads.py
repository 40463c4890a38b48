"""Seeded synthetic inputs for the WeDLM streaming parallel-decode step.

This module only draws random numbers and lays them out in the buffers the
step consumes.  It holds none of the method's arithmetic: no reordering, no
RoPE, no attention, no entropy, no selection.  Both the HIP path and the CPU
oracle take their inputs from here, so the same bytes reach both.

Workloads (the paper measures on GSM8K/MATH prompts with trained 7B/8B
weights; these synthetic tensors stand in for them with Qwen3-8B shapes):

  tiny            B=1,  prefix 256 (contiguous), W=16, Hq=4,  Hkv=2, D=64,
                  V=1024, 8 observed slots, +8 spike on 50% of rows
  qwen3_8b_layer  B=1,  prefix 2048 (contiguous), W=32, Hq=32, Hkv=8, D=128,
                  V=151936, observed fraction 0.5, +10 spike on 60% of rows
  ragged64        B=64, prefix ~ U[512,4096] (paged), W=32, 32/8 heads, D=128,
                  observed fraction ~ U[0,0.75] per sequence, +10 spike, 60%
  long_prefix     B=8,  prefix 32768 (paged), W=64, 32/8 heads, D=128,
                  observed fraction 0.25, +6 spike on 30% of rows
  stream512       B=16, starting prefix 1024 (paged), W=32, 32/8 heads,
                  D=128, 512 steps, window starts all-mask, fresh Q/K/V and
                  logits each step, +12 spike on 90% of rows

Random streams: numpy PCG64 seeded with SeedSequence([seed, config_id, step,
part]).  Every value is N(0,1) (bf16-rounded for Q/K/V and the prefix cache,
fp32 for logits); token ids are uniform in [0, V).

Buffer layouts (the C-ABI header documents the same ones):
  win_tok      [B, W]              int32, -1 marks a mask slot
  win_start    [B]                 int32, committed prefix length c
  qkv_in       [B, W, Hq+2Hkv, D]  bf16 bits (uint16), logical slot order
  k_cache      [P, Hkv, 16, D]     bf16 bits, one 16-token page per P index
  v_cache      [P, Hkv, D, 16]     bf16 bits, the page's V stored transposed
  block_table  [B, max_pages]      int32 page ids, -1 where unused
  logits       [B, W, V]           fp32, physical (reordered) row order

Cache slots that hold no committed token are filled with bf16 NaN, and
logits rows of observed (filled) slots are NaN: a kernel that reads either
poisons its output, which the parity tests would see.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

PAGE = 16
MASK = -1
BF16_NAN = np.uint16(0x7FC0)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cid: int                 # config id used in the seed key
    B: int
    W: int
    Hq: int
    Hkv: int
    D: int
    V: int
    prefix: int              # fixed prefix length (or lower bound if ragged)
    prefix_hi: int = 0       # >0: ragged prefix ~ U[prefix, prefix_hi]
    paged: bool = True       # False: identity block table (contiguous cache)
    obs_frac: float = 0.5    # observed fraction of the window
    obs_frac_hi: float = -1  # >=0: per-sequence fraction ~ U[obs_frac, hi]
    spike: float = 8.0
    spike_prob: float = 0.5
    steps: int = 1           # >1: streaming loop, window starts all-mask
    theta: float = 1e6       # RoPE base
    tau: float = 0.9         # entropy threshold
    lam: float = 0.01        # distance penalty
    temp: float = 0.1        # temperature inside the entropy's softmax
    logit_pool: int = 0      # >0: logits rows drawn from a pool (streaming)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def heads(self) -> int:
        return self.Hq + 2 * self.Hkv

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 1, B=1, W=16, Hq=4, Hkv=2, D=64, V=1024,
                     prefix=256, paged=False, obs_frac=0.5,
                     spike=8.0, spike_prob=0.5),
    "qwen3_8b_layer": Workload("qwen3_8b_layer", 2, B=1, W=32, Hq=32, Hkv=8,
                               D=128, V=151936, prefix=2048, paged=False,
                               obs_frac=0.5, spike=10.0, spike_prob=0.6),
    "ragged64": Workload("ragged64", 3, B=64, W=32, Hq=32, Hkv=8, D=128,
                         V=151936, prefix=512, prefix_hi=4096,
                         obs_frac=0.0, obs_frac_hi=0.75,
                         spike=10.0, spike_prob=0.6),
    "long_prefix": Workload("long_prefix", 4, B=8, W=64, Hq=32, Hkv=8, D=128,
                            V=151936, prefix=32768, obs_frac=0.25,
                            spike=6.0, spike_prob=0.3),
    "stream512": Workload("stream512", 5, B=16, W=32, Hq=32, Hkv=8, D=128,
                          V=151936, prefix=1024, steps=512, obs_frac=0.0,
                          spike=12.0, spike_prob=0.9, logit_pool=256),
}


def rng_for(seed: int, cid: int, step: int, part: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([seed, cid, step, part])))


# parts of the seed key
_P_PREFIX_LEN, _P_WINDOW, _P_QKV, _P_TABLE, _P_LOGITS, _P_POOL, _P_KV = range(7)
_P_DECISION = 7
_P_MODEL, _P_PROMPT = 8, 9


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest even) and return the bit pattern."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    out = (r >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def _normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def prefix_lengths(wl: Workload, seed: int = 0) -> np.ndarray:
    if wl.prefix_hi > 0:
        rng = rng_for(seed, wl.cid, 0, _P_PREFIX_LEN)
        return rng.integers(wl.prefix, wl.prefix_hi, size=wl.B,
                            endpoint=True).astype(np.int32)
    return np.full(wl.B, wl.prefix, dtype=np.int32)


def pages_needed(wl: Workload, c: int, extra: int = 0) -> int:
    """Pages a sequence with prefix c needs for the whole run: its prefix,
    every token the run can commit (at most W per step), one window, and
    `extra` more positions."""
    span = wl.steps * wl.W + wl.W if wl.steps > 1 else wl.W
    return -(-(c + span + extra) // PAGE)


def block_table(wl: Workload, c: np.ndarray, seed: int = 0, extra: int = 0):
    """Per-sequence page lists.  Paged workloads take a seeded random
    permutation of all page ids; contiguous ones take pages in order."""
    npg = np.array([pages_needed(wl, int(x), extra) for x in c],
                   dtype=np.int64)
    total = int(npg.sum())
    if wl.paged:
        ids = rng_for(seed, wl.cid, 0, _P_TABLE).permutation(total)
    else:
        ids = np.arange(total)
    maxp = int(npg.max())
    bt = np.full((wl.B, maxp), -1, dtype=np.int32)
    off = 0
    for b in range(wl.B):
        bt[b, :npg[b]] = ids[off:off + npg[b]]
        off += npg[b]
    return bt, total


def initial_window(wl: Workload, seed: int = 0, step: int = 0) -> np.ndarray:
    """Window tokens: exactly round(f*W) observed slots at seeded random
    window indices, token ids uniform in [0, V); -1 elsewhere.  Streaming
    workloads start from an all-mask window."""
    win = np.full((wl.B, wl.W), MASK, dtype=np.int32)
    if wl.steps > 1:
        return win
    rng = rng_for(seed, wl.cid, step, _P_WINDOW)
    for b in range(wl.B):
        f = wl.obs_frac
        if wl.obs_frac_hi >= 0:
            f = rng.uniform(wl.obs_frac, wl.obs_frac_hi)
        n_o = int(round(f * wl.W))
        slots = rng.choice(wl.W, size=n_o, replace=False)
        win[b, slots] = rng.integers(0, wl.V, size=n_o)
    return win


def qkv(wl: Workload, seed: int = 0, step: int = 0) -> np.ndarray:
    rng = rng_for(seed, wl.cid, step, _P_QKV)
    return _normal_bf16(rng, (wl.B, wl.W, wl.heads, wl.D))


def prefix_kv(wl: Workload, b: int, c: int, seed: int = 0):
    """Logical prefix K (post-RoPE, as a cache holds it) and V of sequence b,
    each [c, Hkv, D] bf16 bits."""
    rng = rng_for(seed, wl.cid, b, _P_KV)
    k = _normal_bf16(rng, (c, wl.Hkv, wl.D))
    v = _normal_bf16(rng, (c, wl.Hkv, wl.D))
    return k, v


def pack_pages(wl: Workload, c: np.ndarray, bt: np.ndarray, total: int,
               seed: int = 0):
    """Scatter each sequence's logical prefix into 16-token pages.
    K pages are [Hkv, 16, D]; V pages are [Hkv, D, 16] (transposed).
    Sequences are drawn and scattered in parallel threads (each has its own
    random stream and its own pages, so the result does not depend on the
    threading)."""
    from concurrent.futures import ThreadPoolExecutor
    kc = np.empty((total, wl.Hkv, PAGE, wl.D), dtype=np.uint16)
    vc = np.empty((total, wl.Hkv, wl.D, PAGE), dtype=np.uint16)
    kc.fill(BF16_NAN)
    vc.fill(BF16_NAN)

    def one(b):
        cb = int(c[b])
        if cb == 0:
            return
        k, v = prefix_kv(wl, b, cb, seed)
        full = cb // PAGE
        pg = bt[b, :full]
        if full:
            kk = k[:full * PAGE].reshape(full, PAGE, wl.Hkv, wl.D)
            vv = v[:full * PAGE].reshape(full, PAGE, wl.Hkv, wl.D)
            kc[pg] = kk.transpose(0, 2, 1, 3)
            vc[pg] = vv.transpose(0, 2, 3, 1)
        rem = cb - full * PAGE
        if rem:
            p = bt[b, full]
            kc[p, :, :rem, :] = k[full * PAGE:].transpose(1, 0, 2)
            vc[p, :, :, :rem] = v[full * PAGE:].transpose(1, 2, 0)

    with ThreadPoolExecutor(max_workers=min(16, max(1, wl.B))) as ex:
        list(ex.map(one, range(wl.B)))
    return kc, vc


def _logit_pool(wl: Workload, seed: int) -> np.ndarray:
    rng = rng_for(seed, wl.cid, 0, _P_POOL)
    return rng.standard_normal((wl.logit_pool, wl.V), dtype=np.float32)


def logit_row_params(wl: Workload, seed: int, step: int):
    """Per physical row: (pool index, cyclic shift, spiked?, spike token).
    Without a pool the first two are unused."""
    rng = rng_for(seed, wl.cid, step, _P_LOGITS)
    n = wl.B * wl.W
    idx = rng.integers(0, max(wl.logit_pool, 1), size=n)
    shift = rng.integers(0, wl.V, size=n)
    spiked = rng.random(n) < wl.spike_prob
    tok = rng.integers(0, wl.V, size=n)
    return idx, shift, spiked, tok


def logits(wl: Workload, n_obs: Optional[np.ndarray], seed: int = 0,
           step: int = 0, pool: Optional[np.ndarray] = None) -> np.ndarray:
    """fp32 logits [B, W, V] in physical row order: N(0,1) plus +spike on a
    uniform random token in a seeded fraction of rows.  Rows below n_obs[b]
    (observed slots after reordering) are NaN: the step never reads them.
    Streaming workloads build each row as a cyclic shift of a row of a
    seeded N(0,1) pool, which keeps each row N(0,1) at a fraction of the
    cost; the per-row draws are the same either way."""
    idx, shift, spiked, tok = logit_row_params(wl, seed, step)
    out = np.empty((wl.B, wl.W, wl.V), dtype=np.float32)
    flat = out.reshape(wl.B * wl.W, wl.V)
    if wl.logit_pool:
        if pool is None:
            pool = _logit_pool(wl, seed)
        for r in range(wl.B * wl.W):
            flat[r] = np.roll(pool[idx[r]], shift[r])
    else:
        rng = rng_for(seed, wl.cid, step, _P_LOGITS + 100)
        for b in range(wl.B):
            lo = 0 if n_obs is None else int(n_obs[b])
            flat[b * wl.W:b * wl.W + lo] = np.nan
            if wl.W - lo:
                flat[b * wl.W + lo:(b + 1) * wl.W] = rng.standard_normal(
                    (wl.W - lo, wl.V), dtype=np.float32)
    rows = np.nonzero(spiked)[0]
    flat[rows, tok[rows]] += np.float32(wl.spike)
    if wl.logit_pool and n_obs is not None:
        for b in range(wl.B):
            flat[b * wl.W:b * wl.W + int(n_obs[b])] = np.nan
    return out


def logit_pool(wl: Workload, seed: int = 0) -> np.ndarray:
    return _logit_pool(wl, seed)


def logits_torch(wl: Workload, pool_dev, seed: int, step: int):
    """Streaming workloads: the same rows as `logits(..., n_obs=None)`, built
    on the device from a device copy of the pool (gather + add only)."""
    import torch
    idx, shift, spiked, tok = logit_row_params(wl, seed, step)
    dev = pool_dev.device
    n = wl.B * wl.W
    ar = torch.arange(wl.V, device=dev, dtype=torch.int64)
    sh = torch.as_tensor(shift, device=dev, dtype=torch.int64)
    col = (ar[None, :] - sh[:, None]) % wl.V
    rows = pool_dev[torch.as_tensor(idx, device=dev, dtype=torch.int64)]
    out = torch.gather(rows, 1, col)
    sp = np.nonzero(spiked)[0]
    if len(sp):
        r = torch.as_tensor(sp, device=dev, dtype=torch.int64)
        t = torch.as_tensor(tok[sp], device=dev, dtype=torch.int64)
        out[r, t] += wl.spike
    return out.view(wl.B, wl.W, wl.V)


def step_inputs(wl: Workload, seed: int = 0, step: int = 0,
                with_cache: bool = True, extra_positions: int = 0,
                nan_observed_rows: bool = True) -> dict:
    """Everything one single step consumes, as numpy arrays.
    extra_positions: more block-table room per sequence (repeated steps).
    nan_observed_rows=False draws logits for every row."""
    c = prefix_lengths(wl, seed)
    win = initial_window(wl, seed, step)
    n_obs = (win != MASK).sum(axis=1).astype(np.int32)
    bt, total = block_table(wl, c, seed, extra_positions)
    d = dict(win_tok=win, win_start=c.copy(), qkv_in=qkv(wl, seed, step),
             block_table=bt, num_pages=total, n_obs_gen=n_obs)
    if with_cache:
        d["k_cache"], d["v_cache"] = pack_pages(wl, c, bt, total, seed)
    if wl.steps == 1:
        d["logits"] = logits(wl, n_obs if nan_observed_rows else None, seed,
                             step)
    return d


def decision_inputs(B: int, W: int, Hkv: int, D: int, seed: int, step: int,
                    quantum: float = 0.0625, levels: int = 24,
                    p_zero: float = 0.3):
    """Synthetic per-physical-row inputs of the commit step alone: entropy
    [B, W] fp32 on a grid of `quantum` (so equal values, and sums with a
    binary lambda, are exact on every side), a share `p_zero` of rows at
    entropy 0, argmax [B, W] int32 and window K/V rows [B, W, Hkv, D] bf16
    bits.  Stream of steps keyed by `step`; cid 100 keeps it apart from the
    workloads' own streams."""
    rng = rng_for(seed, 100, step, _P_DECISION)
    h = rng.integers(0, levels, size=(B, W)).astype(np.float64) * quantum
    h[rng.random((B, W)) < p_zero] = 0.0
    tok = rng.integers(0, 1 << 20, size=(B, W)).astype(np.int32)
    k = _normal_bf16(rng, (B, W, Hkv, D))
    v = _normal_bf16(rng, (B, W, Hkv, D))
    return h.astype(np.float32), tok, k, v


def lm_head_inputs(R: int, Hd: int, V: int, seed: int = 0,
                   kind: str = "normal", spike_frac: float = 0.5,
                   spike: float = 1.5):
    """Inputs of the fused output layer + score: hidden [R, Hd] and the
    vocabulary matrix W [V, Hd] (one row per token), bf16 bits.

    kind "normal": hidden ~ N(0, 1) and W ~ N(0, 1/Hd), so logits are about
    N(0, 1); a share `spike_frac` of the rows gets hidden += spike * W[t] /
    |W[t]|^2 for a random token t, lifting that logit by about `spike`.
    kind "exact": small integers times powers of two (hidden in {-1,0,1}/8,
    W in {-3..3}/32), so every product and every partial sum of a row is a
    multiple of 2^-8 below 2^6 in magnitude: exact in fp32 in any order."""
    rng = rng_for(seed, 200, 0, _P_DECISION)
    if kind == "exact":
        h = rng.integers(-1, 2, size=(R, Hd)).astype(np.float32) / 8.0
        w = rng.integers(-3, 4, size=(V, Hd)).astype(np.float32) / 32.0
        return f32_to_bf16_bits(h), f32_to_bf16_bits(w)
    w = (rng.standard_normal((V, Hd), dtype=np.float32) /
         np.float32(np.sqrt(Hd)))
    wb = f32_to_bf16_bits(w)
    h = rng.standard_normal((R, Hd), dtype=np.float32)
    sp = np.nonzero(rng.random(R) < spike_frac)[0]
    toks = rng.integers(0, V, size=len(sp))
    for r, t in zip(sp, toks):
        wt = (wb[t].astype(np.uint32) << 16).view(np.float32)
        h[r] += np.float32(spike) * wt / np.float32((wt.astype(np.float64) ** 2).sum())
    return f32_to_bf16_bits(h), wb


# --------------------------------------------------------------------------
# decoder weights around the step (a Qwen3-shaped backbone, random init)
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    cid: int
    L: int                   # decoder layers
    Hd: int                  # hidden size
    Hq: int
    Hkv: int
    D: int
    I: int                   # MLP inner size
    V: int
    theta: float = 1e6
    eps: float = 1e-6        # RMSNorm epsilon
    mask_id: int = -1        # vocabulary row of [M]; -1: the last row

    @property
    def mask_row(self) -> int:
        return self.V - 1 if self.mask_id < 0 else self.mask_id

    @property
    def qkv_rows(self) -> int:
        return (self.Hq + 2 * self.Hkv) * self.D


MODEL_SHAPES: Dict[str, ModelShape] = {
    "tiny2": ModelShape("tiny2", 300, L=2, Hd=256, Hq=4, Hkv=2, D=64, I=512,
                        V=1000),
    "qwen3_8b": ModelShape("qwen3_8b", 301, L=36, Hd=4096, Hq=32, Hkv=8,
                           D=128, I=12288, V=151936),
}

MODEL_TENSORS = ("embed", "attn_norm", "w_qkv", "q_norm", "k_norm", "w_o",
                 "mlp_norm", "w_gate_up", "w_down", "final_norm", "lm_head")


def model_tensor_shapes(ms: ModelShape, layers: Optional[int] = None):
    L = ms.L if layers is None else layers
    return {
        "embed": (ms.V, ms.Hd), "attn_norm": (L, ms.Hd),
        "w_qkv": (L, ms.qkv_rows, ms.Hd), "q_norm": (L, ms.D),
        "k_norm": (L, ms.D), "w_o": (L, ms.Hd, ms.Hq * ms.D),
        "mlp_norm": (L, ms.Hd), "w_gate_up": (L, 2 * ms.I, ms.Hd),
        "w_down": (L, ms.Hd, ms.I), "final_norm": (ms.Hd,),
        "lm_head": (ms.V, ms.Hd)}


def model_weights(ms: ModelShape, seed: int = 0,
                  layers: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Random weights of the decoder, bf16 bits.  Projections ~ N(0, 1/fan_in)
    (activations keep unit scale), norm gains 1 + N(0, 0.1^2), embeddings
    N(0, 1), output layer N(0, 1/Hd).  Layouts: every projection is [out,
    in] (one row per output feature); w_gate_up holds the gate rows, then
    the up rows."""
    out = {}
    for i, (name, shape) in enumerate(model_tensor_shapes(ms, layers).items()):
        rng = rng_for(seed, ms.cid, i, _P_MODEL)
        x = rng.standard_normal(shape, dtype=np.float32)
        if name.endswith("norm"):
            x = np.float32(1.0) + np.float32(0.1) * x
        elif name != "embed":
            x /= np.float32(np.sqrt(shape[-1]))
        out[name] = f32_to_bf16_bits(x)
    return out


def model_prompt(ms: ModelShape, B: int, c: int, seed: int = 0) -> np.ndarray:
    """Prompt token ids [B, c], uniform over the vocabulary minus [M]."""
    rng = rng_for(seed, ms.cid, 0, _P_PROMPT)
    t = rng.integers(0, ms.V - 1, size=(B, c)).astype(np.int32)
    t[t >= ms.mask_row] += 1
    return t


def gather_prefix(k_cache: np.ndarray, v_cache: np.ndarray, bt: np.ndarray,
                  b: int, c: int):
    """Read sequence b's first c cache positions back into logical order,
    [c, Hkv, D] each (bf16 bits).  Layout plumbing only."""
    pos = np.arange(c)
    pg = bt[b, pos // PAGE]
    off = pos % PAGE
    k = k_cache[pg, :, off, :]                       # [c, Hkv, D]
    v = v_cache[pg, :, :, off]                       # [c, Hkv, D]
    return k, v
