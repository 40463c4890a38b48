"""Pins of the fp64 oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: a
hand-worked example of the paper's equations or algorithm (tests/golden/),
a library routine that the step reduces to in a special case, a closed form,
an invariant, or brute force.  None of them uses the HIP library.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# Eq. (5)/(6) reordering
# --------------------------------------------------------------------------

def test_reorder_hand_worked_eq5_eq6():
    g = _golden("reorder_eq5_eq6.json")
    for case in g["cases"]:
        perm, pos, tok, n_obs = O.reorder(case["win_tok"], case["c"])
        assert perm == case["perm"]
        assert pos == case["pos"]
        assert tok == case["tok_phys"]
        assert n_obs == case["n_obs"]


@pytest.mark.parametrize("W", [1, 2, 5, 8, 12])
def test_reorder_is_stable_partition_exhaustive(W):
    """Eq. (5)/(6) is a stable sort of the slots by the key 'is a mask';
    Python's sorted() is stable, so it is an independent statement of it."""
    for bits in range(1 << W):
        win = [(-1 if (bits >> s) & 1 else 100 + s) for s in range(W)]
        perm, pos, tok, n_obs = O.reorder(win, 37)
        ref = sorted(range(W), key=lambda s: win[s] == -1)
        assert perm == ref
        assert pos == [37 + s for s in ref]
        assert tok == [win[s] for s in ref]
        assert n_obs == W - bin(bits).count("1")


# --------------------------------------------------------------------------
# Sec. 3.2 / 4.1: the physical causal mask realises the design principles
# --------------------------------------------------------------------------

@pytest.mark.parametrize("W", [1, 3, 6, 10])
def test_physical_causal_equals_logical_visibility(W):
    """Conjugating the causal mask by the reordering gives exactly the
    visibility of principles (i) and (ii) with the order of Eq. (6)."""
    for bits in range(1 << W):
        win = [(-1 if (bits >> s) & 1 else 5) for s in range(W)]
        perm, _, _, _ = O.reorder(win, 0)
        P = np.zeros((W, W), dtype=np.int64)
        for i, s in enumerate(perm):
            P[i, s] = 1                      # physical i <- logical s
        causal = np.tril(np.ones((W, W), dtype=np.int64))
        logical = P.T @ causal @ P           # [q_slot, k_slot]
        for q in range(W):
            for k in range(W):
                assert bool(logical[q, k]) == O.visible(win, q, k)
                assert O.physical_causal_visible(win, 0, q, k) == \
                    O.visible(win, q, k)


def test_every_mask_sees_every_observed_token():
    """Principle (i) of Sec. 3.2 stated directly."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        W = int(rng.integers(1, 20))
        win = [int(x) for x in np.where(rng.random(W) < 0.5, -1, 9)]
        for q in range(W):
            if win[q] != -1:
                continue
            for k in range(W):
                if win[k] != -1:
                    assert O.visible(win, q, k)


# --------------------------------------------------------------------------
# Eq. (2): rotary embedding at logical positions
# --------------------------------------------------------------------------

def test_rope_matches_complex_rotation():
    """Half-split RoPE is multiplication of z_i = x_i + i x_{i+D/2} by
    exp(i * pos * theta^(-2i/D))."""
    rng = np.random.default_rng(0)
    D, theta = 16, 1e6
    x = rng.standard_normal(D)
    for pos in [0, 1, 7, 1000, 40000]:
        z = x[:D // 2] + 1j * x[D // 2:]
        w = theta ** (-2.0 * np.arange(D // 2) / D)
        zr = z * np.exp(1j * pos * w)
        ref = np.concatenate([zr.real, zr.imag])
        np.testing.assert_allclose(O.rope(x, pos, theta), ref, rtol=0,
                                   atol=1e-12)


def test_rope_relative_position_property():
    """Scores depend on logical offsets only (the property Eq. 2 relies on)."""
    rng = np.random.default_rng(1)
    D, theta = 64, 1e6
    q, k = rng.standard_normal(D), rng.standard_normal(D)
    a = O.rope(q, 50, theta) @ O.rope(k, 20, theta)
    b = O.rope(q, 50 + 12345, theta) @ O.rope(k, 20 + 12345, theta)
    assert abs(a - b) < 1e-9
    assert np.allclose(O.rope(q, 0, theta), q)
    # two-dimensional case: a plain rotation by `pos` radians
    v = np.array([1.0, 0.0])
    np.testing.assert_allclose(O.rope(v, 0.5, theta), [math.cos(0.5),
                                                       math.sin(0.5)])


# --------------------------------------------------------------------------
# Forward: attention of the reordered window over the cache
# --------------------------------------------------------------------------

def _naive_logical_attention(win, c, x_log, k_pre, v_pre, Hq, Hkv, theta):
    """Attention computed in LOGICAL order with the explicit visibility rule:
    every window slot rotated at its own logical position c + s, the prefix
    always visible, window keys visible per O.visible.  Returns [W, Hq, D]
    in logical slot order."""
    W, _, D = x_log.shape
    G = Hq // Hkv
    out = np.zeros((W, Hq, D))
    qs = np.stack([O.rope(x_log[s, :Hq], c + s, theta) for s in range(W)])
    ks = np.stack([O.rope(x_log[s, Hq:Hq + Hkv], c + s, theta)
                   for s in range(W)])
    vs = x_log[:, Hq + Hkv:]
    for h in range(Hq):
        g = h // G
        for qs_ in range(W):
            keys = [k_pre[j, g] for j in range(k_pre.shape[0])]
            vals = [v_pre[j, g] for j in range(k_pre.shape[0])]
            for ks_ in range(W):
                if O.visible(win, qs_, ks_):
                    keys.append(ks[ks_, g])
                    vals.append(vs[ks_, g])
            K = np.array(keys)
            V = np.array(vals)
            s = K @ qs[qs_, h] / math.sqrt(D)
            p = np.exp(s - s.max())
            out[qs_, h] = (p / p.sum()) @ V
    return out


def _bits(rng, shape):
    x = rng.standard_normal(shape).astype(np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)   # truncation is fine


@pytest.mark.parametrize("W,c", [(1, 5), (4, 0), (5, 9), (8, 3)])
def test_attention_equals_logical_order_bruteforce(W, c):
    """For every fill pattern, the oracle's physical-order causal attention
    equals attention in logical order with the explicit visibility rule."""
    rng = np.random.default_rng(W * 100 + c)
    Hq, Hkv, D, theta = 4, 2, 8, 1e4
    k_pre = rng.standard_normal((c, Hkv, D))
    v_pre = rng.standard_normal((c, Hkv, D))
    patterns = range(1 << W) if W <= 5 else rng.integers(0, 1 << W, 12)
    for bits in patterns:
        win = [(-1 if (int(bits) >> s) & 1 else 7) for s in range(W)]
        xb = _bits(rng, (W, Hq + 2 * Hkv, D))
        x_log = O.bf16_to_f64(xb)
        perm, pos, _, _ = O.reorder(win, c)
        q, k, v = O.rope_window(xb, perm, pos, Hq, Hkv, theta)
        out_phys, _ = O.window_attn(q, k, v, k_pre, v_pre)
        ref = _naive_logical_attention(win, c, x_log, k_pre, v_pre, Hq, Hkv,
                                       theta)
        for i, s in enumerate(perm):
            np.testing.assert_allclose(out_phys[i], ref[s], rtol=0,
                                       atol=1e-12)


def test_attention_matches_torch_sdpa_fp64():
    """Textbook comparator: torch's scaled_dot_product_attention in fp64 on
    the CPU with an explicit boolean mask (prefix all visible, causal on the
    window including the diagonal), GQA by repeating kv heads."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(11)
    W, c, Hq, Hkv, D = 7, 13, 6, 2, 16
    q = rng.standard_normal((W, Hq, D))
    kw = rng.standard_normal((W, Hkv, D))
    vw = rng.standard_normal((W, Hkv, D))
    kp = rng.standard_normal((c, Hkv, D))
    vp = rng.standard_normal((c, Hkv, D))
    out, lse = O.window_attn(q, kw, vw, kp, vp)
    G = Hq // Hkv
    K = np.concatenate([kp, kw], 0).repeat(G, axis=1)      # [c+W, Hq, D]
    V = np.concatenate([vp, vw], 0).repeat(G, axis=1)
    mask = np.zeros((W, c + W), dtype=bool)
    mask[:, :c] = True
    mask[:, c:] = np.tril(np.ones((W, W), dtype=bool))
    tq = torch.tensor(q).permute(1, 0, 2)
    tk = torch.tensor(K).permute(1, 0, 2)
    tv = torch.tensor(V).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=torch.tensor(mask)).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    # lse against a direct logsumexp
    s = np.einsum("whd,khd->whk", q, K) / math.sqrt(D)
    s = np.where(mask[:, None, :], s, -np.inf)
    ref_lse = np.log(np.exp(s - s.max(-1, keepdims=True)).sum(-1)) + \
        s.max(-1)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    Hq, Hkv, D = 2, 1, 8
    # c = 0, row 0 sees only itself: output is its own value row
    q = rng.standard_normal((3, Hq, D))
    kw = rng.standard_normal((3, Hkv, D))
    vw = rng.standard_normal((3, Hkv, D))
    e = np.zeros((0, Hkv, D))
    out, lse = O.window_attn(q, kw, vw, e, e)
    np.testing.assert_allclose(out[0, 0], vw[0, 0], atol=1e-14)
    np.testing.assert_allclose(out[0, 1], vw[0, 0], atol=1e-14)
    np.testing.assert_allclose(lse[0, 0], q[0, 0] @ kw[0, 0] / math.sqrt(D))
    # constant values give that constant whatever the scores
    vconst = np.ones((3, Hkv, D)) * 2.5
    kp = rng.standard_normal((4, Hkv, D))
    out, _ = O.window_attn(q, kw, vconst, kp, np.ones((4, Hkv, D)) * 2.5)
    np.testing.assert_allclose(out, 2.5, atol=1e-13)
    # zero queries give the plain mean of the visible values
    vp = rng.standard_normal((4, Hkv, D))
    out, _ = O.window_attn(np.zeros_like(q), kw, vw, kp, vp)
    np.testing.assert_allclose(
        out[2, 0], np.concatenate([vp[:, 0], vw[:3, 0]]).mean(0), atol=1e-13)


def test_attention_position_shift_invariance():
    """Shifting c shifts every logical position; with rotated prefix keys
    rotated consistently, scores (hence outputs) are unchanged."""
    rng = np.random.default_rng(8)
    W, c, Hq, Hkv, D, theta = 5, 6, 2, 1, 8, 1e4
    win = [3, -1, 4, -1, -1]
    xb = _bits(rng, (W, Hq + 2 * Hkv, D))
    raw_k = rng.standard_normal((c, Hkv, D))
    vp = rng.standard_normal((c, Hkv, D))
    outs = []
    for shift in [0, 1000]:
        kp = np.stack([O.rope(raw_k[j], shift + j, theta) for j in range(c)])
        perm, pos, _, _ = O.reorder(win, c + shift)
        q, k, v = O.rope_window(xb, perm, pos, Hq, Hkv, theta)
        outs.append(O.window_attn(q, k, v, kp, vp)[0])
    np.testing.assert_allclose(outs[0], outs[1], atol=1e-10)


# --------------------------------------------------------------------------
# Sec. 5.2 entropy
# --------------------------------------------------------------------------

def test_entropy_uniform_is_log_v():
    for V in [1, 2, 1024, 151936]:
        tok, H, pm = O.score_row(np.zeros(V, dtype=np.float32), 0.1)
        assert tok == 0
        assert abs(H - math.log(V)) < 1e-12 * max(1.0, math.log(V))
        assert abs(pm - 1.0 / V) < 1e-15


def test_entropy_k_way_tie_is_log_k():
    V = 4096
    for k in [2, 3, 17]:
        x = np.full(V, -1e30, dtype=np.float32)
        idx = np.random.default_rng(k).choice(V, k, replace=False)
        x[idx] = 1.5
        tok, H, pm = O.score_row(x, 1.0)
        assert tok == int(idx.min())                # lowest id on ties
        assert abs(H - math.log(k)) < 1e-14
        assert abs(pm - 1.0 / k) < 1e-15


@pytest.mark.parametrize("delta,V,T", [(8.0, 1024, 1.0), (10.0, 151936, 1.0),
                                      (2.0, 50, 0.5), (0.25, 7, 1.0)])
def test_entropy_single_spike_closed_form(delta, V, T):
    """One logit at delta, V-1 at zero: with a = delta/T and
    Z = e^a + V - 1, H = ln Z - a e^a / Z and p_max = e^a / Z."""
    import mpmath as mp
    mp.mp.dps = 40
    x = np.zeros(V, dtype=np.float32)
    x[V // 3] = delta
    tok, H, pm = O.score_row(x, T)
    a = mp.mpf(delta) / T
    Z = mp.e ** a + (V - 1)
    assert tok == V // 3
    assert abs(H - float(mp.log(Z) - a * mp.e ** a / Z)) <= 1e-13 * float(
        mp.log(Z))
    assert abs(pm - float(mp.e ** a / Z)) <= 1e-15


def test_entropy_extreme_peak_against_mpmath():
    """At T = 0.1 with a large spike, H is ~1e-20 or smaller; the oracle must
    keep its relative accuracy (a naive fp64 -sum p log p loses it)."""
    import mpmath as mp
    # p_max = 1 - O(1e-55): log(p_max) needs more than 55 digits
    mp.mp.dps = 150
    rng = np.random.default_rng(2)
    for trial in range(6):
        V = 64
        x = rng.standard_normal(V).astype(np.float32)
        x[trial] += np.float32(6.0 + 2 * trial)
        T = 0.1
        tok, H, pm = O.score_row(x, T)
        xs = [mp.mpf(float(v)) / mp.mpf(T) for v in x]
        m = max(xs)
        es = [mp.exp(v - m) for v in xs]
        Z = mp.fsum(es)
        ps = [e / Z for e in es]
        Hm = -mp.fsum([p * mp.log(p) for p in ps])
        assert abs(H - float(Hm)) <= 1e-12 * float(Hm) + 1e-300
        assert abs(pm - float(max(ps))) <= 1e-15


def test_entropy_matches_torch_categorical():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(4)
    for T in [1.0, 0.5, 0.1]:
        x = rng.standard_normal(5000).astype(np.float32)
        tok, H, pm = O.score_row(x, T)
        ref = torch.distributions.Categorical(
            logits=torch.tensor(x, dtype=torch.float64) / T).entropy().item()
        assert abs(H - ref) <= 1e-12 * ref
        assert tok == int(np.argmax(x))


def test_score_skips_observed_rows():
    x = np.random.default_rng(0).standard_normal((4, 32)).astype(np.float32)
    x[:2] = np.nan
    tok, H, pm = O.score(x, 2, 1.0)
    assert list(tok[:2]) == [-1, -1] and np.isnan(H[:2]).all()
    assert np.isfinite(H[2:]).all()


# --------------------------------------------------------------------------
# Algorithm 1: commit / select / refill
# --------------------------------------------------------------------------

def test_commit_hand_worked_trace():
    g = _golden("commit_trace_alg1.json")
    win, c = g["W"] * [-1], g["c0"]
    y, ys = [], []
    for st in g["steps"]:
        assert win == st["win"] and c == st["c"]
        H = [np.nan if h is None else h for h in st["H"]]
        tok = [-1 if t is None else t for t in st["tok"]]
        r = O.commit(win, c, H, tok, g["tau"], g["lam"], g["block_table"])
        assert r["n"] == st["n"]
        assert r["committed"] == st["committed"]
        assert r["slots"] == st["slots"]
        assert r["selected"] == st["selected"]
        assert r["win"] == st["win_after"]
        assert r["c"] == st["c_after"]
        y += r["committed"]
        ys += r["slots"]
        win, c = r["win"], r["c"]
    assert y == g["y"] and ys == g["y_slots"]


@pytest.mark.parametrize("rule", ["block", "one"])
def test_commit_rules_hand_worked_traces(rule):
    """Block-wise stop-and-wait (Fig. 3, Sec. 6.4) and one token per step
    (Sec. 6.2), traced by hand from the same first step as the streaming
    trace."""
    g = _golden("commit_trace_rules.json")
    tr = g["rules"][rule]
    win, c = g["W"] * [-1], g["c0"]
    y, ys = [], []
    for st in tr["steps"]:
        assert win == st["win"] and c == st["c"]
        H = [np.nan if h is None else h for h in st["H"]]
        tok = [-1 if t is None else t for t in st["tok"]]
        r = O.commit(win, c, H, tok, g["tau"], g["lam"], g["block_table"],
                     rule=rule)
        assert r["n"] == st["n"]
        assert r["committed"] == st["committed"]
        assert r["slots"] == st["slots"]
        assert r["selected"] == st["selected"]
        assert r["win"] == st["win_after"]
        assert r["c"] == st["c_after"]
        y += r["committed"]
        ys += r["slots"]
        win, c = r["win"], r["c"]
    assert y == tr["y"] and ys == tr["y_slots"]


def test_unknown_rule_is_rejected():
    with pytest.raises(ValueError):
        O.commit([-1, -1], 0, [0.1, 0.1], [1, 2], 0.9, 0.1, rule="blocks")


def test_threshold_boundary_is_strict():
    """lambda = 0.1, d = 9: tau - lambda*d is exactly 0.0 in fp64, so a slot
    with H = 0 at distance 9 does not pass the strict test of Eq. (11)."""
    assert 0.9 - 0.1 * 9 == 0.0
    W = 10
    win = [-1] * W
    H = [5.0] * 9 + [0.0]
    r = O.commit(win, 0, H, list(range(W)), 0.9, 0.1)
    # not by the threshold (that would be 1): nothing passes, and the
    # fallback's argmin of H + lambda*d (0 + 0.9 at slot 9 against 5.0
    # elsewhere) fills it instead
    assert r["selected"] == [0] * 9 + [2]
    # one step closer (d = 8) the same entropy passes the threshold
    H8 = [5.0] * 8 + [0.0, 5.0]
    r = O.commit(win, 0, H8, list(range(W)), 0.9, 0.1)
    assert r["selected"] == [0] * 8 + [1, 0]


def test_fallback_ties_go_left():
    r = O.commit([-1, -1, -1], 0, [1.0, 0.9, 0.8], [5, 6, 7], 0.5, 0.1)
    # keys 1.0, 1.0, 1.0 (0.9 + 0.1, 0.8 + 0.2 in fp64): ties -> leftmost?
    keys = [1.0 + 0.1 * 0, 0.9 + 0.1 * 1, 0.8 + 0.1 * 2]
    best = min(range(3), key=lambda s: (keys[s], s))
    assert r["selected"][best] == 2 and sum(map(bool, r["selected"])) == 1


def _const_stream(W, steps, H_value, tau, lam, c0=7, rule="stream"):
    """Stream in which every masked row has the given entropy."""
    win, c = [-1] * W, c0
    ns, toks, fills = [], [], {}
    for t in range(steps):
        perm, _, _, n_obs = O.reorder(win, c)
        H = [H_value] * W
        tok = [1000 * t + i for i in range(W)]
        r = O.commit(win, c, H, tok, tau, lam, list(range(100)), rule=rule)
        ns.append(r["n"])
        toks.append(r["committed"])
        win, c = r["win"], r["c"]
    return ns, toks, c


def test_all_select_regime_closed_form():
    """Every mask has H = 0 < tau and lambda = 0: a step fills the whole
    window, the next commits all W, and so on; p_cache is exactly 1/2."""
    W, steps = 8, 10
    ns, _, c = _const_stream(W, steps, 0.0, 0.5, 0.0)
    assert ns == [0, W] * (steps // 2)
    assert c == 7 + W * steps // 2
    assert O.p_cache(np.array(ns)[:, None], W) == 0.5


def test_fallback_only_regime_is_autoregressive():
    """tau <= 0: no mask passes the threshold; with a large lambda the
    fallback fills the leftmost mask, so from the second step on exactly
    one token is committed per step, as in autoregressive decoding."""
    W, steps = 6, 12
    ns, toks, c = _const_stream(W, steps, 0.3, 0.0, 10.0)
    assert ns == [0] + [1] * (steps - 1)
    assert c == 7 + steps - 1


def test_block_rule_closed_forms():
    """Block-wise rule.  All masks pass: one step fills the block, the next
    commits it, as in streaming (p_cache 1/2).  One fill per step (tau <= 0,
    leftmost by a large lambda): a block takes W fill steps and one commit
    step, so p_cache = W / ((W + 1) W) = 1 / (W + 1), against streaming's
    (steps - 1) / (steps W) in the same regime."""
    W, steps = 8, 10
    ns, _, c = _const_stream(W, steps, 0.0, 0.5, 0.0, rule="block")
    assert ns == [0, W] * (steps // 2)
    W, blocks = 5, 4
    steps = blocks * (W + 1)
    ns, toks, c = _const_stream(W, steps, 0.3, 0.0, 10.0, rule="block")
    assert ns == ([0] * W + [W]) * blocks
    assert c == 7 + W * blocks
    assert O.p_cache(np.array(ns)[:, None], W) == pytest.approx(1 / (W + 1))
    ns_s, _, _ = _const_stream(W, steps, 0.3, 0.0, 10.0)
    assert O.p_cache(np.array(ns_s)[:, None], W) == \
        pytest.approx((steps - 1) / (steps * W))


def test_one_token_rule_is_autoregressive_whatever_tau():
    """One token per step: even when every mask would pass the threshold
    (tau = 10), exactly one mask is filled per step; with equal entropies
    and lambda > 0 it is the leftmost, so from the second step on one token
    is committed per step."""
    W, steps = 6, 12
    for tau in (10.0, 0.9, -1.0):
        ns, toks, c = _const_stream(W, steps, 0.3, tau, 0.1, rule="one")
        assert ns == [0] + [1] * (steps - 1)
        # the token committed at step t + 1 was filled at step t: physical
        # row 0 at step 0 (all masks), row 1 (the leftmost mask, behind one
        # filled slot) afterwards
        assert [t[0] for t in toks[1:]] == \
            [0] + [1000 * t + 1 for t in range(1, steps - 1)]


def test_slot_formula():
    bt = [9, 4, 0, 7]
    assert [O.slot_of(bt, p) for p in [0, 15, 16, 31, 32, 63]] == \
        [144, 159, 64, 79, 0, 127]


def _random_stream(seed, B=3, W=8, steps=40, V=50):
    rng = np.random.default_rng(seed)
    Hq, Hkv, D = 2, 1, 4

    def inputs(t):
        x = rng.standard_normal((B, W, V)).astype(np.float32)
        spike = rng.random((B, W)) < 0.5
        x[spike, rng.integers(0, V)] += 8.0
        q = (rng.standard_normal((B, W, Hq + 2 * Hkv, D)).astype(np.float32)
             .view(np.uint32) >> 16).astype(np.uint16)
        return {"qkv_in": q, "logits": x}

    bt = np.arange(B * 40).reshape(B, 40)
    return O.stream(np.full((B, W), -1), np.array([5, 0, 31]), steps, inputs,
                    Hq, Hkv, 1e4, 0.9, 0.05, 0.1, bt)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stream_invariants(seed):
    """Sec. 5.1 requirements as invariants: c never decreases, the window
    keeps W slots, committed tokens only grow left to right, the cache holds
    exactly c positions (slots = one per committed token), and p_cache <= 1/2
    because every committed token was forwarded once as [M] and once filled.
    """
    B, W, steps = 3, 8, 40
    r = _random_stream(seed, B, W, steps)
    assert r["win"].shape == (B, W)
    for b in range(B):
        assert len(r["tokens"][b]) == r["n"][:, b].sum()
        assert r["c"][b] == [5, 0, 31][b] + r["n"][:, b].sum()
        assert len(r["slots"][b]) == len(r["tokens"][b])
        assert len(set(r["slots"][b])) == len(r["slots"][b])
    assert (r["n"] >= 0).all()
    assert O.p_cache(r["n"], W) <= 0.5


def test_committed_token_was_filled_in_an_earlier_step():
    """A token enters y only in a step after the one that filled it: trace
    each sequence's window and check that tokens committed at step t were
    already in the window before step t's selection."""
    rng = np.random.default_rng(9)
    W = 6
    win, c = [-1] * W, 0
    for t in range(60):
        before = list(win)
        H = list(rng.random(W) * 2)
        tok = list(rng.integers(0, 100, W))
        r = O.commit(win, c, H, tok, 0.9, 0.05)
        assert r["committed"] == before[:r["n"]]
        assert all(x != -1 for x in r["committed"])
        win, c = r["win"], r["c"]
        assert len(win) == W


def test_stream_batch_independence():
    """Sequences in a batch never interact: the batched stream equals each
    sequence run on its own."""
    r = _random_stream(5, B=3)
    assert len(r["tokens"]) == 3
    # rerun the same per-step draws sequence by sequence
    rng = np.random.default_rng(5)
    B, W, V, steps = 3, 8, 50, 40
    draws = []
    for t in range(steps):
        x = rng.standard_normal((B, W, V)).astype(np.float32)
        spike = rng.random((B, W)) < 0.5
        x[spike, rng.integers(0, V)] += 8.0
        rng.standard_normal((B, W, 4, 4))
        draws.append(x)
    for b in range(B):
        win, c = [-1] * W, [5, 0, 31][b]
        toks = []
        for t in range(steps):
            perm, _, _, n_obs = O.reorder(win, c)
            tk, H, _ = O.score(draws[t][b], n_obs, 0.1)
            rr = O.commit(win, c, O.to_f32_decision(H), tk, 0.9, 0.05)
            toks += rr["committed"]
            win, c = rr["win"], rr["c"]
        assert toks == r["tokens"][b]


# --------------------------------------------------------------------------
# output layer + score (the fused LM-head kernel's definition)
# --------------------------------------------------------------------------

def _bf16(x):
    return WL.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def test_lm_head_zero_hidden_is_uniform():
    """hidden = 0: every logit is 0, so the distribution is uniform over V:
    H = ln V, p_max = 1/V, token 0 (the first maximum)."""
    V, Hd = 37, 16
    rng = np.random.default_rng(0)
    tok, H, pm = O.lm_head_score(_bf16(np.zeros((2, Hd))),
                                 _bf16(rng.standard_normal((V, Hd))), 0.1)
    assert list(tok) == [0, 0]
    assert np.allclose(H, math.log(V), rtol=1e-12)
    assert np.allclose(pm, 1.0 / V, rtol=1e-12)


def test_lm_head_one_hot_vocabulary_selects_hidden_entries():
    """W = identity rows (V <= Hd): logits are the hidden entries 0..V-1, so
    the result is the score of those numbers."""
    V, Hd = 12, 16
    rng = np.random.default_rng(1)
    h = _bf16(rng.standard_normal((3, Hd)))
    tok, H, pm = O.lm_head_score(h, _bf16(np.eye(V, Hd)), 0.5)
    x = O.bf16_to_f64(h)[:, :V]
    for r in range(3):
        t2, H2, p2 = O.score_row(x[r], 0.5, as_f32=False)
        assert tok[r] == int(np.argmax(x[r])) == t2
        assert H[r] == pytest.approx(H2, rel=1e-13)
        assert pm[r] == pytest.approx(p2, rel=1e-13)


def test_lm_head_exact_inputs_against_integer_dot_products():
    """The "exact" recipe: hidden*8 and W*32 are small integers, so every
    logit*256 is an integer; Python integer dot products (no floating point)
    give the logits, and ties between equal logits go to the lower id."""
    R, Hd, V = 5, 64, 300
    hb, wb = WL.lm_head_inputs(R, Hd, V, seed=3, kind="exact")
    hi = np.rint(O.bf16_to_f64(hb) * 8).astype(np.int64)
    wi = np.rint(O.bf16_to_f64(wb) * 32).astype(np.int64)
    tok, H, pm = O.lm_head_score(hb, wb, 0.1, chunk=37)
    for r in range(R):
        lg = [sum(int(a) * int(b) for a, b in zip(hi[r], wi[v]))
              for v in range(V)]
        best = max(lg)
        assert tok[r] == lg.index(best)
        t2, H2, p2 = O.score_row(np.array(lg, dtype=np.float64) / 256.0, 0.1,
                                 as_f32=False)
        assert H[r] == pytest.approx(H2, rel=1e-13, abs=1e-300)
        assert pm[r] == pytest.approx(p2, rel=1e-13)


def test_lm_head_rows_and_chunks_do_not_change_results():
    R, Hd, V = 6, 32, 101
    hb, wb = WL.lm_head_inputs(R, Hd, V, seed=4)
    full = O.lm_head_score(hb, wb, 0.1)
    part = O.lm_head_score(hb, wb, 0.1, rows=[4, 1], chunk=10)
    assert list(part[0]) == [full[0][4], full[0][1]]
    assert np.array_equal(part[1], full[1][[4, 1]])


def test_lm_head_spiked_rows_pick_their_token():
    """The "normal" recipe lifts one logit of a spiked row by about the
    spike; with a large spike that token is the greedy one."""
    R, Hd, V = 8, 256, 500
    hb, wb = WL.lm_head_inputs(R, Hd, V, seed=5, spike_frac=1.0, spike=30.0)
    tok, H, pm = O.lm_head_score(hb, wb, 0.1)
    # the spiked token wins by a wide margin: p_max near 1
    assert (pm > 0.99).all()
