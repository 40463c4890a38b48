"""Plain fp64 CPU oracle of the decoder forward that produces the step's
queries, keys, values and logits.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never imports it.

WeDLM-8B starts from Qwen3-8B and keeps its architecture (Sec. 6.1); the
paper changes the attention pattern and the positions (Sec. 4), not the
layers.  The layer is therefore the public Qwen3 decoder layer, written
here from its definition:

  x      = E[token]                                   (embedding row)
  per layer l:
    a    = RMSNorm(x) * g_attn
    q, k, v = a W_q^T, a W_k^T, a W_v^T               (no biases)
    q, k = RMSNorm over each head's D values * g_q / g_k
    q, k = RoPE at the token's logical position (Eq. 2)
    o    = softmax(q k^T / sqrt(D) + mask) v          (GQA: head h reads kv
                                                       head h // (Hq/Hkv))
    x    = x + o W_o^T
    m    = RMSNorm(x) * g_mlp
    x    = x + (silu(m W_gate^T) * (m W_up^T)) W_down^T
  h      = RMSNorm(x) * g_final,  logits = h W_vocab^T
  RMSNorm(x) = x / sqrt(mean(x^2) + eps)

The forward is computed WITHOUT a cache and WITHOUT reordering: the whole
sequence (committed prefix, then the window in logical order, masks as the
[M] embedding) goes through every layer at once, and the attention mask is
the logical visibility rule of Sec. 3.2 / Sec. 4.1 (prefix causal; observed
window slots see the prefix and earlier observed slots; masks see the
prefix, every observed slot and earlier masks).  Sec. 5.2's argument that
the committed prefix's keys and values do not depend on the window is then
something the tests check rather than something the oracle assumes.

Readings (listed with their reasons in the design notes):
  * Qwen3's layer as above, RMSNorm eps 1e-6, RoPE base 1e6 "rotate half".
  * [M] is one row of the embedding matrix (the last row unless given).
  * Every window row is scored (the step only reads the masked ones).
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Sequence

import numpy as np

from . import wedlm_oracle as O


def decode(bits: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """bf16 bit arrays -> fp64 arrays, same keys."""
    return {k: O.bf16_to_f64(np.asarray(v)) for k, v in bits.items()}


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x); sigmoid(x) = 1 / (1 + e^-|x|) for x >= 0 and
    e^-|x| / (1 + e^-|x|) below, so no exponential overflows."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, x / (1.0 + e), x * e / (1.0 + e))


def logical_visibility(c: int, win_tok: Sequence[int]) -> np.ndarray:
    """vis[i, j]: may position i attend to position j, for the sequence of c
    committed tokens followed by the W window slots in logical order."""
    W = len(win_tok)
    n = c + W
    vis = np.zeros((n, n), dtype=bool)
    for i in range(n):
        for j in range(n):
            if j < c:
                vis[i, j] = j <= i          # prefix keys: causal
            elif i < c:
                vis[i, j] = False           # prefix never sees the window
            else:
                vis[i, j] = O.visible(win_tok, i - c, j - c)
    return vis


def forward(ms, w: Dict[str, np.ndarray], tokens: Sequence[int],
            pos: Sequence[int], vis: np.ndarray, layers: Optional[int] = None):
    """The decoder over one sequence of tokens with explicit positions and
    visibility.  w: fp64 weights (decode()).  Returns the final normalised
    hidden states [n, Hd], and per layer the rotated keys and the values
    [L, n, Hkv, D]."""
    L = ms.L if layers is None else layers
    n = len(tokens)
    Hq, Hkv, D, I = ms.Hq, ms.Hkv, ms.D, ms.I
    G = Hq // Hkv
    x = w["embed"][np.asarray(tokens)].copy()
    ks = np.zeros((L, n, Hkv, D))
    vs = np.zeros((L, n, Hkv, D))
    scale = 1.0 / math.sqrt(D)
    for l in range(L):
        a = rmsnorm(x, w["attn_norm"][l], ms.eps)
        qkv = a @ w["w_qkv"][l].T
        q = qkv[:, :Hq * D].reshape(n, Hq, D)
        k = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(n, Hkv, D)
        v = qkv[:, (Hq + Hkv) * D:].reshape(n, Hkv, D)
        q = rmsnorm(q, w["q_norm"][l], ms.eps)
        k = rmsnorm(k, w["k_norm"][l], ms.eps)
        for t in range(n):
            q[t] = O.rope(q[t], pos[t], ms.theta)
            k[t] = O.rope(k[t], pos[t], ms.theta)
        ks[l], vs[l] = k, v
        o = np.zeros((n, Hq, D))
        for h in range(Hq):
            s = (q[:, h, :] @ k[:, h // G, :].T) * scale
            s = np.where(vis, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            o[:, h, :] = p @ v[:, h // G, :]
        x = x + o.reshape(n, Hq * D) @ w["w_o"][l].T
        m = rmsnorm(x, w["mlp_norm"][l], ms.eps)
        gu = m @ w["w_gate_up"][l].T
        x = x + (silu(gu[:, :I]) * gu[:, I:]) @ w["w_down"][l].T
    return rmsnorm(x, w["final_norm"], ms.eps), ks, vs


def window_forward(ms, w: Dict[str, np.ndarray], prefix: Sequence[int],
                   win_tok: Sequence[int], layers: Optional[int] = None):
    """Committed prefix + window (logical order, masks as the [M] row),
    positions 0..c+W-1, logical visibility.  Returns the final hidden states
    of the window slots [W, Hd] (logical order) and the keys / values of all
    c+W positions [L, c+W, Hkv, D]."""
    c = len(prefix)
    toks = [int(t) for t in prefix] + [
        int(t) if t != O.MASK else ms.mask_row for t in win_tok]
    vis = logical_visibility(c, win_tok)
    h, ks, vs = forward(ms, w, toks, list(range(c + len(win_tok))), vis,
                        layers)
    return h[c:], ks, vs


def window_scores(ms, w: Dict[str, np.ndarray], prefix: Sequence[int],
                  win_tok: Sequence[int], temperature: float,
                  layers: Optional[int] = None):
    """Logits of every window slot (h W_vocab^T) and their scores, indexed by
    PHYSICAL row (the order of Eq. 5/6, which the step's outputs use).
    Returns dict(perm, n_obs, logits [W, V] physical, tok, H, pmax [W]),
    plus the window's keys / values in logical order."""
    h, ks, vs = window_forward(ms, w, prefix, win_tok, layers)
    perm, _, _, n_obs = O.reorder(list(win_tok), len(prefix))
    logits = h[perm] @ w["lm_head"].T
    sc = [O.score_row(r, temperature, as_f32=False) for r in logits]
    return dict(perm=perm, n_obs=n_obs, logits=logits,
                tok=np.array([s[0] for s in sc], dtype=np.int64),
                H=np.array([s[1] for s in sc]),
                pmax=np.array([s[2] for s in sc]), k=ks, v=vs)
