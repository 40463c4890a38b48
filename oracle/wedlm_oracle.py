"""Plain fp64 CPU oracle of WeDLM's streaming parallel-decode step.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never imports it; the two meet only through the arrays
the seeded input generator produces.

What it computes, following WeDLM (arXiv 2512.22737):

  reorder      Topological reordering, Eq. (5) and Eq. (6): observed slots
               first, masks last, each group in ascending logical order; the
               logical position ids travel with the tokens.
  rope         Rotary embedding at the supplied logical positions, the
               decoupled positional representation of Eq. (2) (Sec. 2.2).
  window_attn  One causal forward of the reordered window over the cached
               prefix (Sec. 4.1 "Context Awareness under Causal Masking",
               Algorithm 1 Forward): physical row i sees every cached prefix
               position and window rows 0..i.
  visible      The logical visibility rule the reordering realises
               (Sec. 3.2 design principles (i) and (ii)), written
               independently of the physical causal mask.
  score        Entropy of the predicted distribution at each mask slot
               (Sec. 5.2, the quantity inside Eq. (11)) plus the greedy token.
  commit       Algorithm 1 commit / SelectByEntropy / Sample / refill steps,
               with the distance-adjusted entropy of Eq. (11); also the two
               decoding rules the paper compares against: block-wise
               stop-and-wait commit (Fig. 3, Sec. 6.4) and one token per
               step (Sec. 6.2).
  stream       Algorithm 1's loop over many steps.
  lm_head_score  The logits of the forward's output layer (hidden states
               times the vocabulary matrix) scored as above, for the fused
               LM-head kernel.
  dual_stream_*  The training-time attention of Sec. 4.2: a clean memory
               stream followed by the block-wise reordered prediction
               stream, with the block attention pattern written out as a
               dense mask (masked_attention).

Readings where the paper is silent or loose (each is listed with its reason
in the design notes of the repository):
  * Commit count: the leftmost contiguous run of filled slots in logical
    window order (Sec. 5.2 text and the commit comment of Algorithm 1); after
    the stable reordering these are exactly physical rows 0..n-1.
  * The causal mask includes the diagonal (a row sees itself).
  * Entropy in nats of softmax(logits / T); T defaults to 0.1, the paper's
    decoding temperature (Sec. 6.2).
  * d_i = window index of slot i minus window index of the leftmost mask.
  * Selection is the strict test H_i < tau - lambda * d_i, evaluated in
    fp64 on the entropy rounded to fp32 (the precision the kernel stores).
  * If no mask passes and at least one mask exists, the single mask with the
    smallest adjusted entropy H_i + lambda * d_i is filled (ties: leftmost),
    the paper's one-token-per-step rule (Sec. 6.2); without it the loop can
    stall.
  * Sample is greedy: argmax of the raw fp32 logits, ties to the lowest id.
  * RoPE pairs dimension i with i + D/2 ("rotate half"), frequency
    theta^(-2i/D); positions are 0-based, the window starting at c.
  * Softmax scale 1/sqrt(D); query head h reads kv head h // (Hq/Hkv).
  * Block-wise rule: the block is the W-slot window.  Selection is the same
    as streaming, but nothing is committed while any slot of the block is a
    mask; the step that sees the whole block filled commits all W slots and
    the window refills with W masks (Fig. 3 "stop-and-wait", Sec. 6.4).
  * Dual-stream attention: the memory stream is causal over itself (it is
    the clean sequence); block k of the prediction stream sees memory
    positions < kB and its own reordered block causally, itself included;
    both streams carry the logical positions 0..L-1 (Eq. 8).
  * One-token rule: exactly one mask per step, the one with the smallest
    H_i + lambda * d_i (ties: leftmost), whatever tau; commit as in
    streaming (Sec. 6.2's unified step-wise scheme).

Numbers are fp64 throughout, computed from the bf16-decoded inputs.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

MASK = -1
PAGE = 16


# --------------------------------------------------------------------------
# data decoding
# --------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode bf16 bit patterns (uint16) to fp64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Eq. (5)/(6): topological reordering
# --------------------------------------------------------------------------

def reorder(win_tok: Sequence[int], c: int):
    """Topological reordering of one window (Eq. 5 and Eq. 6).

    win_tok: W token ids in logical slot order, MASK (-1) for [M].
    c:       committed prefix length; slot s has logical position c + s.
    Returns perm (physical row -> logical slot), pos (logical position of
    each physical row), tok_phys (token of each physical row) and n_obs.
    """
    W = len(win_tok)
    observed = [s for s in range(W) if win_tok[s] != MASK]
    masked = [s for s in range(W) if win_tok[s] == MASK]
    perm = observed + masked
    pos = [c + s for s in perm]
    tok_phys = [int(win_tok[s]) for s in perm]
    return perm, pos, tok_phys, len(observed)


# --------------------------------------------------------------------------
# Eq. (2): rotary embedding at logical positions
# --------------------------------------------------------------------------

def rope(x: np.ndarray, pos: float, theta: float) -> np.ndarray:
    """Rotate the last axis (length D) of x at logical position `pos`.
    Dimension i pairs with i + D/2 at angle pos * theta^(-2i/D)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    out = np.empty_like(x)
    for i in range(half):
        ang = pos * theta ** (-2.0 * i / D)
        cs, sn = math.cos(ang), math.sin(ang)
        a, b = x[..., i], x[..., i + half]
        out[..., i] = a * cs - b * sn
        out[..., i + half] = b * cs + a * sn
    return out


# --------------------------------------------------------------------------
# Sec. 3.2 / Sec. 4.1: who may see whom
# --------------------------------------------------------------------------

def visible(win_tok: Sequence[int], q_slot: int, k_slot: int) -> bool:
    """Logical visibility between two window slots, stated from the design
    principles rather than from the physical mask: an observed key is seen
    by every masked query (principle (i)); masks see earlier masks in
    ascending order (principle (ii) with the order of Eq. 6); observed
    tokens see earlier-or-equal observed tokens (causal LM); an observed
    query never sees a mask.  A slot always sees itself."""
    q_obs = win_tok[q_slot] != MASK
    k_obs = win_tok[k_slot] != MASK
    if k_obs and not q_obs:
        return True
    if k_obs and q_obs:
        return k_slot <= q_slot
    if not k_obs and not q_obs:
        return k_slot <= q_slot
    return False


def physical_causal_visible(win_tok: Sequence[int], c: int, q_slot: int,
                            k_slot: int) -> bool:
    """Visibility induced by the plain causal mask on the reordered window:
    physical row of k <= physical row of q."""
    perm, _, _, _ = reorder(win_tok, c)
    phys = {s: i for i, s in enumerate(perm)}
    return phys[k_slot] <= phys[q_slot]


# --------------------------------------------------------------------------
# Forward: causal attention of the reordered window over the cache
# --------------------------------------------------------------------------

def window_attn(q: np.ndarray, k_win: np.ndarray, v_win: np.ndarray,
                k_pre: np.ndarray, v_pre: np.ndarray,
                rows: Optional[Sequence[int]] = None,
                heads: Optional[Sequence[int]] = None):
    """Attention of one sequence's reordered window.

    q:      [W, Hq, D]  RoPE'd queries, physical order
    k_win:  [W, Hkv, D] RoPE'd window keys, physical order
    v_win:  [W, Hkv, D] window values, physical order
    k_pre:  [c, Hkv, D] cached prefix keys (already rotated), logical order
    v_pre:  [c, Hkv, D] cached prefix values
    Physical row i attends to all c prefix positions and window rows 0..i.
    Returns out [len(rows), len(heads), D] and lse (natural log) of the same
    leading shape.
    """
    W, Hq, D = q.shape
    Hkv = k_win.shape[1]
    G = Hq // Hkv
    c = k_pre.shape[0]
    rows = list(range(W)) if rows is None else list(rows)
    heads = list(range(Hq)) if heads is None else list(heads)
    scale = 1.0 / math.sqrt(D)
    out = np.zeros((len(rows), len(heads), D))
    lse = np.zeros((len(rows), len(heads)))
    for hi, h in enumerate(heads):
        g = h // G
        keys = np.concatenate([k_pre[:, g, :], k_win[:, g, :]], axis=0)
        vals = np.concatenate([v_pre[:, g, :], v_win[:, g, :]], axis=0)
        for ri, i in enumerate(rows):
            n_ctx = c + i + 1                      # prefix + window rows 0..i
            s = keys[:n_ctx] @ q[i, h, :] * scale
            m = s.max()
            w = np.exp(s - m)
            z = w.sum()
            out[ri, hi] = (w / z) @ vals[:n_ctx]
            lse[ri, hi] = m + math.log(z)
    return out, lse


# --------------------------------------------------------------------------
# Sec. 5.2: entropy of a mask slot's predicted distribution, greedy token
# --------------------------------------------------------------------------

def score_row(logit_row: np.ndarray, temperature: float,
              as_f32: bool = True):
    """Greedy token, entropy H (nats) and top probability of
    p = softmax(logits / T).

    H = -sum_v p_v log p_v, with log p_v = z_v - log Z written out so that
    nothing cancels: z_v = (l_v - l_max) / T and log Z = log1p(sum over
    v != argmax of e^{z_v}).  The logits are taken as fp32 (what wedlm_score
    reads) unless as_f32 is False."""
    x = np.asarray(logit_row, dtype=np.float32 if as_f32 else np.float64)
    tok = int(np.argmax(x))                        # first maximum
    x = x.astype(np.float64)
    z = (x - x[tok]) / temperature
    rest = np.delete(z, tok)
    log_z = math.log1p(float(np.exp(rest).sum()))
    logp = z - log_z
    p = np.exp(logp)
    H = float(-(p * logp).sum())
    return tok, H, math.exp(-log_z)


def score(logits: np.ndarray, n_obs: int, temperature: float):
    """Score the masked physical rows n_obs..W-1 of one sequence.
    Returns argmax [W] int, entropy [W], pmax [W]; observed rows are -1/NaN.
    """
    W = logits.shape[0]
    tok = np.full(W, -1, dtype=np.int64)
    H = np.full(W, np.nan)
    pm = np.full(W, np.nan)
    for i in range(n_obs, W):
        tok[i], H[i], pm[i] = score_row(logits[i], temperature)
    return tok, H, pm


# --------------------------------------------------------------------------
# Algorithm 1: commit, SelectByEntropy (Eq. 11), Sample, refill
# --------------------------------------------------------------------------

def lm_head_score(hidden_bits: np.ndarray, w_bits: np.ndarray,
                  temperature: float, rows: Optional[Sequence[int]] = None,
                  chunk: int = 8192):
    """Output layer plus score: logits[r, v] = sum_k hidden[r, k] * W[v, k]
    exactly in fp64 from the bf16-decoded inputs (hidden [R, Hd], W [V, Hd],
    the output layer's weight as stored, one row per token), then the
    greedy token, entropy and top probability of softmax(logits / T) of
    each row, on the fp64 logits.  `rows` limits the work to sampled rows;
    the vocabulary is processed in chunks to bound memory.
    Returns (tok [n], H [n], p_max [n]) for the rows in order."""
    h = bf16_to_f64(np.asarray(hidden_bits))
    rr = list(range(h.shape[0])) if rows is None else list(rows)
    hs = h[rr]
    V = w_bits.shape[0]
    logits = np.empty((len(rr), V))
    for v0 in range(0, V, chunk):
        w = bf16_to_f64(np.asarray(w_bits[v0:v0 + chunk]))
        logits[:, v0:v0 + w.shape[0]] = hs @ w.T
    out = [score_row(row, temperature, as_f32=False) for row in logits]
    tok = np.array([o[0] for o in out], dtype=np.int64)
    H = np.array([o[1] for o in out])
    pm = np.array([o[2] for o in out])
    return tok, H, pm


def slot_of(block_table_row: Sequence[int], pos: int) -> int:
    """Cache slot of logical position `pos` in 16-token pages."""
    return int(block_table_row[pos // PAGE]) * PAGE + pos % PAGE


RULES = ("stream", "block", "one")


def commit(win_tok: Sequence[int], c: int, entropy_phys: Sequence[float],
           argmax_phys: Sequence[int], tau: float, lam: float,
           block_table_row: Optional[Sequence[int]] = None,
           rule: str = "stream"):
    """One commit/select/fill/refill step on one window (Algorithm 1).

    entropy_phys / argmax_phys are indexed by physical row (the reordered
    order in which the forward produced them).  The entropy used in the
    decision should already be in the precision of the caller's choice.
    rule: "stream" (Algorithm 1), "block" (block-wise stop-and-wait commit
    of the whole window, Fig. 3 / Sec. 6.4) or "one" (one token per step,
    Sec. 6.2).
    Returns a dict with n, committed tokens, committed slots, the selection
    (logical slot -> 1 threshold / 2 smallest adjusted entropy), the new
    window and c.
    """
    if rule not in RULES:
        raise ValueError(f"unknown decoding rule {rule!r}")
    W = len(win_tok)
    win = [int(t) for t in win_tok]
    perm, _, _, n_obs = reorder(win, c)
    phys = {s: i for i, s in enumerate(perm)}

    # commit: the leading run of filled slots, in logical order; the block
    # rule commits only a window with no mask left, all W slots at once
    n = 0
    while n < W and win[n] != MASK:
        n += 1
    if rule == "block" and n < W:
        n = 0
    committed = win[:n]
    slots = ([slot_of(block_table_row, c + j) for j in range(n)]
             if block_table_row is not None else [])

    # SelectByEntropy with the distance-adjusted entropy of Eq. (11)
    masks = [s for s in range(W) if win[s] == MASK]
    selected = [0] * W
    if masks:
        s0 = masks[0]
        for s in masks:
            d = s - s0
            if rule != "one" and float(entropy_phys[phys[s]]) < tau - lam * d:
                selected[s] = 1
        if not any(selected):
            best, best_key = None, None
            for s in masks:
                key = float(entropy_phys[phys[s]]) + lam * (s - s0)
                if best is None or key < best_key:
                    best, best_key = s, key
            selected[best] = 2
    # Sample (greedy) into the selected masks
    filled = list(win)
    for s in masks:
        if selected[s]:
            filled[s] = int(argmax_phys[phys[s]])
    # drop the committed run, refill with masks
    new_win = filled[n:] + [MASK] * n
    return dict(n=n, committed=committed, slots=slots, selected=selected,
                win=new_win, c=c + n, perm=perm, n_obs=n_obs)


# --------------------------------------------------------------------------
# one step / many steps
# --------------------------------------------------------------------------

def rope_window(qkv_in_bits: np.ndarray, perm: Sequence[int],
                pos: Sequence[int], Hq: int, Hkv: int, theta: float):
    """Gather one sequence's window rows into physical order and rotate Q
    and K at their logical positions.  qkv_in is [W, Hq+2Hkv, D] (bf16 bits,
    logical order); perm/pos may list only the first physical rows.
    Returns q [n,Hq,D], k [n,Hkv,D], v [n,Hkv,D] fp64, n = len(perm)."""
    x = bf16_to_f64(qkv_in_bits)
    D = x.shape[-1]
    W = len(perm)
    q = np.empty((W, Hq, D))
    k = np.empty((W, Hkv, D))
    v = np.empty((W, Hkv, D))
    for i, s in enumerate(perm):
        q[i] = rope(x[s, :Hq], pos[i], theta)
        k[i] = rope(x[s, Hq:Hq + Hkv], pos[i], theta)
        v[i] = x[s, Hq + Hkv:]
    return q, k, v


def to_f32_decision(h: np.ndarray) -> np.ndarray:
    """Entropy as the decision sees it: rounded to fp32, compared in fp64."""
    return np.asarray(h, dtype=np.float64).astype(np.float32).astype(np.float64)


def stream(win0: np.ndarray, c0: np.ndarray, steps: int,
           inputs_for_step: Callable[[int], dict], Hq: int, Hkv: int,
           theta: float, tau: float, lam: float, temperature: float,
           block_table: np.ndarray,
           prefix_kv: Optional[Callable[[int], tuple]] = None,
           attn_steps: Sequence[int] = (),
           logits_row: Optional[Callable[[int, int, int], np.ndarray]] = None,
           progress: Optional[Callable[[int], None]] = None,
           rule: str = "stream"):
    """Algorithm 1's loop for a batch of independent sequences.

    inputs_for_step(t) returns {"qkv_in": [B,W,Hq+2Hkv,D] bf16 bits} and,
    unless `logits_row` is given, {"logits": [B,W,V] fp32}.
    logits_row(t, b, i) may instead return one physical row on demand.
    prefix_kv(b) returns the initial cached (k, v) of sequence b as bf16
    bits [c0, Hkv, D]; it is needed only when attention is evaluated
    (steps listed in attn_steps).  The oracle's cache keeps appended rows
    in fp64; rows are rotated only where they are used (attention steps, and
    committed rows while a cache is kept).
    Returns per-sequence committed tokens and slots, per-step n and c, final
    window/c, and attention outputs for the requested steps.
    """
    B, W = win0.shape
    win = [list(map(int, win0[b])) for b in range(B)]
    c = [int(x) for x in c0]
    toks: List[List[int]] = [[] for _ in range(B)]
    slots: List[List[int]] = [[] for _ in range(B)]
    n_hist = np.zeros((steps, B), dtype=np.int64)
    c_hist = np.zeros((steps, B), dtype=np.int64)
    sel_hist = []
    attn: Dict[int, list] = {}
    keep_cache = len(attn_steps) > 0
    cache_k: List[list] = [[] for _ in range(B)]
    cache_v: List[list] = [[] for _ in range(B)]
    if keep_cache:
        for b in range(B):
            kb, vb = prefix_kv(b)
            cache_k[b] = [bf16_to_f64(kb)]
            cache_v[b] = [bf16_to_f64(vb)]
    last_attn = max(attn_steps) if keep_cache else -1
    for t in range(steps):
        inp = inputs_for_step(t)
        outs_t = []
        sel_t = []
        for b in range(B):
            c_hist[t, b] = c[b]
            perm, pos, _, n_obs = reorder(win[b], c[b])
            if t in attn_steps:
                q, k, v = rope_window(inp["qkv_in"][b], perm, pos, Hq, Hkv,
                                      theta)
                kp = np.concatenate(cache_k[b], axis=0)
                vp = np.concatenate(cache_v[b], axis=0)
                outs_t.append(window_attn(q, k, v, kp, vp)[0])
            H = np.full(W, np.nan)
            tok = np.full(W, -1, dtype=np.int64)
            for i in range(n_obs, W):
                row = (logits_row(t, b, i) if logits_row is not None
                       else inp["logits"][b, i])
                tok[i], H[i], _ = score_row(row, temperature)
            r = commit(win[b], c[b], to_f32_decision(H), tok, tau, lam,
                       block_table[b], rule=rule)
            toks[b] += r["committed"]
            slots[b] += r["slots"]
            n_hist[t, b] = r["n"]
            sel_t.append(r["selected"])
            n = r["n"]
            if keep_cache and n and t < last_attn:
                # committed rows are physical rows 0..n-1 = logical slots
                # 0..n-1, at positions c..c+n-1
                _, kn, vn = rope_window(inp["qkv_in"][b], perm[:n], pos[:n],
                                        Hq, Hkv, theta)
                cache_k[b].append(kn)
                cache_v[b].append(vn)
            win[b], c[b] = r["win"], r["c"]
        sel_hist.append(sel_t)
        if t in attn_steps:
            attn[t] = outs_t
        if progress is not None:
            progress(t)
    return dict(tokens=toks, slots=slots, n=n_hist, c_hist=c_hist,
                win=np.array(win), c=np.array(c), attn=attn,
                selected=sel_hist)


def p_cache(n_hist: np.ndarray, W: int) -> float:
    """Eq. (4): tokens that became committed per token instance forwarded
    (each step forwards W window tokens per sequence)."""
    steps, B = n_hist.shape
    return float(n_hist.sum()) / float(steps * B * W)


# --------------------------------------------------------------------------
# Sec. 4.2: dual-stream masking (training forward of the attention)
# --------------------------------------------------------------------------

def dual_stream_order(L: int, B: int, masked):
    """Physical layout of Eq. (7)'s input: the memory stream (logical
    positions 0..L-1 in order), then the prediction stream cut into blocks of
    B, each block reordered as in Sec. 4.1 (its observed positions first,
    then its masked ones, each group ascending).  masked: set of masked
    logical positions of the prediction stream.  Returns a list of
    (stream, logical position, masked) per physical row, stream 0 = memory,
    1 = prediction."""
    rows = [(0, p, False) for p in range(L)]
    for b0 in range(0, L, B):
        blk = list(range(b0, min(b0 + B, L)))
        obs = [p for p in blk if p not in masked]
        msk = [p for p in blk if p in masked]
        rows += [(1, p, False) for p in obs] + [(1, p, True) for p in msk]
    return rows


def dual_stream_visible(L: int, B: int, masked):
    """vis[i, j] for the physical rows of dual_stream_order, written from the
    attention pattern of Sec. 4.2: a memory token sees earlier-or-equal
    memory tokens (the clean causal stream); a prediction token in block k
    sees the memory tokens whose logical positions precede block k and the
    tokens of its own reordered block that physically precede it (itself
    included); nothing else."""
    rows = dual_stream_order(L, B, masked)
    n = len(rows)
    vis = np.zeros((n, n), dtype=bool)
    for i, (si, pi, _) in enumerate(rows):
        ki = pi // B
        for j, (sj, pj, _) in enumerate(rows):
            if si == 0:
                vis[i, j] = sj == 0 and pj <= pi
            elif sj == 0:
                vis[i, j] = pj < ki * B
            else:
                vis[i, j] = pj // B == ki and j <= i
    return vis


def masked_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     vis: np.ndarray):
    """softmax(q k^T / sqrt(D) restricted to vis) v for every row and head.
    q [n, Hq, D], k and v [n, Hkv, D] (rotated q and k), GQA h -> h // G.
    Returns out [n, Hq, D] and lse [n, Hq] (natural log)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, Hq, D = q.shape
    G = Hq // k.shape[1]
    out = np.zeros((n, Hq, D))
    lse = np.zeros((n, Hq))
    for h in range(Hq):
        s = (q[:, h] @ k[:, h // G].T) / math.sqrt(D)
        s = np.where(vis, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        p = np.exp(s - m)
        z = p.sum(axis=1, keepdims=True)
        out[:, h] = (p / z) @ v[:, h // G]
        lse[:, h] = (m + np.log(z))[:, 0]
    return out, lse
