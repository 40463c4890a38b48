"""GPU parity of the decoder around the step (include/wedlm_model.h) against
the fp64 oracle (oracle/model_oracle.py).

Kernel by kernel, on the same bf16 inputs:
  * wedlm_embed bit-exact (bf16 -> fp32 is exact);
  * wedlm_rmsnorm within one bf16 rounding of the fp64 value (plus fp32
    noise);
  * wedlm_qk_norm_rope within one bf16 rounding of each rotated pair;
  * wedlm_linear within the fp32 summation bound K * 2^-24 * sum|x w| (plus
    the output's bf16 rounding), for every epilogue and for row counts that
    cover one, two and four 32-row blocks, ragged tails and several row
    groups.

Whole decoder (`tiny2`: 2 layers, hidden 256, 4/2 heads of 64, MLP 512,
vocabulary 1000): a prefill of the prompt through the window path itself
(all-filled windows), then streaming steps.  At every step the oracle runs
the full-sequence forward from the GPU's own state (committed tokens and
window), with no cache and no reordering, so errors do not compound.  The
step's scores are compared at T = 1 (entropy within 0.03 nats; greedy
tokens equal wherever the oracle's top two logits are more than 0.05
apart: the hidden states carry a few bf16 roundings per layer, about 0.4%
of a logit of unit scale after two layers).  The commit is checked
bit-exactly against the oracle's commit fed the GPU's own scores, and at
the end every committed cache row against the oracle's keys and values.
A step captured in a HIP graph and replayed gives the same bits as eager
steps.
"""
import math

import numpy as np
import pytest
import torch

from oracle import model_oracle as MO
from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL

pytestmark = pytest.mark.gpu

DEV = "cuda"


def W_():
    from paper_2512_22737_amd import wedlm
    return wedlm


def _bf(a):
    return (torch.from_numpy(np.ascontiguousarray(a)).view(torch.int16)
            .to(DEV).view(torch.bfloat16))


def _f64(t):
    return t.float().cpu().double().numpy()


def _rand_bf16(rng, shape, scale=1.0):
    return WL.f32_to_bf16_bits(
        (rng.standard_normal(shape) * scale).astype(np.float32))


# ---------------------------------------------------------------------------
# kernels
# ---------------------------------------------------------------------------

def test_embed_exact():
    w = W_()
    rng = np.random.default_rng(1)
    table = _rand_bf16(rng, (50, 256))
    tok = np.array([3, -1, 49, 0, 7, -1, 60], dtype=np.int32)  # 60 >= V
    x = torch.empty(len(tok), 256, dtype=torch.float32, device=DEV)
    w.wedlm_embed(torch.from_numpy(tok).to(DEV), 10, _bf(table), x)
    torch.cuda.synchronize()
    ids = np.where((tok < 0) | (tok >= 50), 10, tok)
    ref = O.bf16_to_f64(table[ids])
    assert np.array_equal(x.cpu().double().numpy(), ref)


# Hd up to 8192 in registers (1, 2, 4 or 8 float4 chunks per thread, the
# last one partly masked at 1000), longer rows through the chunk loop
@pytest.mark.parametrize("M,Hd", [(1, 256), (7, 4096), (33, 1000), (3, 8192),
                                  (2, 2048), (2, 12288)])
def test_rmsnorm(M, Hd):
    w = W_()
    rng = np.random.default_rng(M)
    x = (rng.standard_normal((M, Hd)) * 3).astype(np.float32)
    g = _rand_bf16(rng, (Hd,), 0.1)
    g = WL.f32_to_bf16_bits(1.0 + O.bf16_to_f64(g).astype(np.float32))
    y = torch.empty(M, Hd, dtype=torch.bfloat16, device=DEV)
    w.wedlm_rmsnorm(torch.from_numpy(x).to(DEV), _bf(g), 1e-6, y)
    torch.cuda.synchronize()
    ref = MO.rmsnorm(x.astype(np.float64), O.bf16_to_f64(g), 1e-6)
    err = np.abs(_f64(y) - ref)
    assert (err <= 2.0 ** -8 * np.abs(ref) + 1e-6).all(), err.max()


# one round of q/k items, two rounds, and three with more than 256 pieces of
# v (the first round of each is loaded before the rotation table)
@pytest.mark.parametrize("M,Hq,Hkv,D", [(5, 4, 2, 64), (33, 32, 8, 128),
                                        (2, 64, 32, 128)])
def test_qk_norm_rope(M, Hq, Hkv, D):
    w = W_()
    rng = np.random.default_rng(D + M)
    qkv = _rand_bf16(rng, (M, (Hq + 2 * Hkv) * D), 2.0)
    gq = WL.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(D).astype(np.float32))
    gk = WL.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(D).astype(np.float32))
    pos = rng.integers(0, 40000, size=M).astype(np.int32)
    q = torch.empty(M, Hq, D, dtype=torch.bfloat16, device=DEV)
    k = torch.empty(M, Hkv, D, dtype=torch.bfloat16, device=DEV)
    v = torch.empty(M, Hkv, D, dtype=torch.bfloat16, device=DEV)
    w.wedlm_qk_norm_rope(_bf(qkv), _bf(gq), _bf(gk),
                         torch.from_numpy(pos).to(DEV), Hq, Hkv, 1e6, 1e-6,
                         q, k, v)
    torch.cuda.synchronize()
    x = O.bf16_to_f64(qkv).reshape(M, Hq + 2 * Hkv, D)
    nq = MO.rmsnorm(x[:, :Hq], O.bf16_to_f64(gq), 1e-6)
    nk = MO.rmsnorm(x[:, Hq:Hq + Hkv], O.bf16_to_f64(gk), 1e-6)
    half = D // 2
    for got, n in ((q, nq), (k, nk)):
        g = _f64(got)
        ref = np.stack([O.rope(n[t], float(pos[t]), 1e6) for t in range(M)])
        # a rotated pair's error: its bf16 rounding plus fp32 noise
        mag = np.abs(n[..., :half]) + np.abs(n[..., half:])
        mag = np.concatenate([mag, mag], axis=-1)
        err = np.abs(g - ref)
        assert (err <= 2.0 ** -8 * mag + 1e-5).all(), err.max()
    assert np.array_equal(v.cpu().view(torch.int16).numpy().view(np.uint16),
                          qkv.reshape(M, Hq + 2 * Hkv, D)[:, Hq + Hkv:])


def test_pack_layout_exact():
    """The packed tile layout of include/wedlm_model.h, element by element."""
    w = W_()
    rows, K = 96, 192
    src = np.arange(rows * K, dtype=np.uint16).reshape(rows, K)
    got = w.pack(_bf(src)).cpu().view(torch.int16).numpy().view(np.uint16)
    got = got.reshape(-1)
    S = K // 64
    for r in range(rows // 32):
        for s in range(S):
            base = (r * S + s) * 2048
            for j in range(4):
                for l in range(64):
                    k0 = 64 * s + 32 * (l // 32) + 8 * j
                    e = base + (j * 64 + l) * 8
                    assert np.array_equal(got[e:e + 8],
                                          src[32 * r + l % 32, k0:k0 + 8])


LINEAR_CASES = [
    # M, N, K
    (1, 32, 64), (5, 96, 256), (32, 256, 4096), (33, 64, 512),
    (64, 128, 1024), (100, 64, 320), (200, 96, 256), (300, 32, 640),
]


@pytest.mark.parametrize("M,N,K", LINEAR_CASES)
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_linear(M, N, K, epi):
    w = W_()
    rng = np.random.default_rng(M * 7 + N + K + epi)
    x = _rand_bf16(rng, (M, K))
    rows = 2 * N if epi == 2 else N
    wt = _rand_bf16(rng, (rows, K), 1.0 / math.sqrt(K))
    xf, wf = O.bf16_to_f64(x), O.bf16_to_f64(wt)
    prod = xf @ wf.T                                    # [M, rows]
    bound = K * 2.0 ** -24 * (np.abs(xf) @ np.abs(wf).T)
    ldo = N + 32 if epi == 1 else N                     # a padded row once
    if epi == 1:
        base = rng.standard_normal((M, ldo)).astype(np.float32)
        out = torch.from_numpy(base.copy()).to(DEV)
    else:
        out = torch.full((M, ldo), float("nan"), dtype=torch.bfloat16,
                         device=DEV)
    w.wedlm_linear(_bf(x), w.pack(_bf(wt)), epi, out)
    torch.cuda.synchronize()
    got = _f64(out)
    if epi == 0:
        err = np.abs(got - prod)
        assert (err <= 2.0 ** -8 * np.abs(prod) + bound + 1e-30).all(), err.max()
    elif epi == 1:
        ref = base[:, :N].astype(np.float64) + prod
        err = np.abs(got[:, :N] - ref)
        assert (err <= bound + 2.0 ** -23 * np.abs(ref)).all(), err.max()
        assert np.array_equal(got[:, N:], base[:, N:])      # untouched
    else:
        g, u = prod[:, :N], prod[:, N:]
        ref = MO.silu(g) * u
        eg, eu = bound[:, :N], bound[:, N:]
        # |d silu / dg| <= 1.1; silu(g) error 1e-6 relative (fp32 exp)
        tol = (2.0 ** -8 * np.abs(ref) + 1.1 * eg * np.abs(u) +
               np.abs(MO.silu(g)) * eu + 1e-6 * np.abs(ref) + 1e-30)
        err = np.abs(got - ref)
        assert (err <= tol).all(), err.max()


def test_linear_split_workspace_reuse():
    """Products that split K over workgroups (residual add at N = 4096) share
    one workspace back to back with products that do not."""
    w = W_()
    rng = np.random.default_rng(11)
    need = max(w.wedlm_linear_workspace_size(32, 4096, 4096, 1),
               w.wedlm_linear_workspace_size(32, 256, 4096, 0))
    ws = torch.zeros(need, dtype=torch.uint8, device=DEV)
    for (N, epi) in ((4096, 1), (256, 0), (4096, 1)):
        x = _rand_bf16(rng, (32, 4096))
        wt = _rand_bf16(rng, (N, 4096), 1 / 64)
        out = (torch.zeros(32, N, dtype=torch.float32, device=DEV) if epi
               else torch.empty(32, N, dtype=torch.bfloat16, device=DEV))
        w.wedlm_linear(_bf(x), w.pack(_bf(wt)), epi, out, workspace=ws)
        torch.cuda.synchronize()
        prod = O.bf16_to_f64(x) @ O.bf16_to_f64(wt).T
        bound = 4096 * 2.0 ** -24 * (np.abs(O.bf16_to_f64(x)) @
                                     np.abs(O.bf16_to_f64(wt)).T)
        err = np.abs(_f64(out) - prod)
        assert (err <= 2.0 ** -8 * np.abs(prod) * (epi == 0) + bound +
                1e-30).all()


# ---------------------------------------------------------------------------
# the whole decoder
# ---------------------------------------------------------------------------

MS = WL.MODEL_SHAPES["tiny2"]


def _decoder(ms, wbits, B, W, pages_per_seq, T, seed=0):
    w = W_()
    cfg = w.model_config(ms.L, ms.Hd, ms.Hq, ms.Hkv, ms.D, ms.I, ms.V,
                         ms.mask_row, ms.theta, ms.eps)
    tens = {k: _bf(v) for k, v in wbits.items()}
    rng = np.random.default_rng(seed)
    total = B * pages_per_seq
    bt = rng.permutation(total).astype(np.int32).reshape(B, pages_per_seq)
    dec = w.Decoder(cfg, tens, B, W, total, torch.from_numpy(bt).to(DEV),
                    max_prefix_len=pages_per_seq * 16, temperature=T)
    return dec, bt


def _prefill(dec, prompt):
    """Prompt through all-filled windows: each step commits W tokens."""
    B, c0 = prompt.shape
    W = dec.W
    assert c0 % W == 0
    for k in range(c0 // W):
        dec.win_tok.copy_(torch.from_numpy(prompt[:, k * W:(k + 1) * W]))
        dec.step()
        torch.cuda.synchronize()
        assert (dec.n_commit.cpu().numpy() == W).all()
        assert np.array_equal(dec.committed_tok.cpu().numpy(),
                              prompt[:, k * W:(k + 1) * W])
    assert (dec.win_start.cpu().numpy() == c0).all()
    assert (dec.win_tok.cpu().numpy() == O.MASK).all()


@pytest.mark.parametrize("B,W", [(2, 16), (3, 12), (17, 16)])
def test_decoder_streaming_steps_against_oracle(B, W):
    """(2, 16): 32 window rows, one row tile; (3, 12): 36 rows, a ragged
    second tile in the packed activations; (17, 16): 272 rows, the 2-D tiled
    products (three row tiles of 128, the last mostly empty)."""
    c0, steps, T = 2 * W, 6, 1.0
    wbits = WL.model_weights(MS, seed=0)
    wf = MO.decode(wbits)
    dec, bt = _decoder(MS, wbits, B, W, pages_per_seq=12, T=T)
    prompt = WL.model_prompt(MS, B, c0, seed=3)
    _prefill(dec, prompt)
    y = [list(prompt[b]) for b in range(B)]
    tau, lam = dec.tau, dec.lam
    worst_h, compared = 0.0, 0
    for t in range(steps):
        win = dec.win_tok.cpu().numpy().copy()
        c = dec.win_start.cpu().numpy().copy()
        dec.forward()
        torch.cuda.synchronize()
        am = dec.argmax.cpu().numpy()
        H = dec.entropy.cpu().numpy()
        kw = _f64(dec.k_win)                        # [L, B, W, Hkv, D]
        for b in range(B):
            assert c[b] == len(y[b])
            r = MO.window_scores(MS, wf, y[b], list(win[b]), T)
            n_obs = r["n_obs"]
            assert int(dec.n_obs[b]) == n_obs
            assert list(dec.perm[b].cpu().numpy()) == list(r["perm"])
            for i in range(n_obs, W):
                lg = np.sort(r["logits"][i])
                worst_h = max(worst_h, abs(H[b, i] - r["H"][i]))
                assert abs(H[b, i] - r["H"][i]) < 0.03, (t, b, i)
                if lg[-1] - lg[-2] > 0.05:
                    assert am[b, i] == r["tok"][i], (t, b, i)
                    compared += 1
            # keys of the window rows (physical order) vs the oracle's
            kref = r["k"][:, c[b] + np.asarray(r["perm"])]
            scale = np.abs(kref).max()
            assert np.abs(kw[:, b] - kref).max() < 0.02 * scale, (t, b)
        # the commit on the GPU's own scores equals the oracle's commit
        exp = [O.commit(list(win[b]), int(c[b]), list(H[b].astype(np.float64)),
                        list(am[b]), tau, lam, list(bt[b])) for b in range(B)]
        dec.commit()
        torch.cuda.synchronize()
        for b in range(B):
            e = exp[b]
            assert int(dec.n_commit[b]) == e["n"]
            assert list(dec.win_tok[b].cpu().numpy()) == e["win"]
            assert int(dec.win_start[b]) == e["c"]
            y[b] += e["committed"]
    assert compared > 20
    # every committed cache row against the oracle's causal keys / values
    kc = dec.k_cache.cpu().view(torch.int16).numpy().view(np.uint16)
    vc = dec.v_cache.cpu().view(torch.int16).numpy().view(np.uint16)
    for b in range(B):
        n = len(y[b])
        _, ks, vs = MO.forward(MS, wf, y[b], list(range(n)),
                               np.tril(np.ones((n, n), dtype=bool)))
        for l in range(MS.L):
            kg, vg = WL.gather_prefix(kc[l], vc[l], bt, b, n)
            kg, vg = O.bf16_to_f64(kg), O.bf16_to_f64(vg)
            assert np.abs(kg - ks[l]).max() < 0.02 * np.abs(ks[l]).max()
            assert np.abs(vg - vs[l]).max() < 0.02 * np.abs(vs[l]).max()


def test_decoder_graph_replay_matches_eager():
    """One step (forward + commit) captured in a HIP graph: replays from the
    same start state give exactly the eager steps' outputs."""
    B, W, c0, steps = 2, 16, 32, 4
    wbits = WL.model_weights(MS, seed=1)
    prompt = WL.model_prompt(MS, B, c0, seed=4)
    runs = []
    for mode in ("eager", "graph"):
        dec, _ = _decoder(MS, wbits, B, W, pages_per_seq=10, T=0.1, seed=2)
        _prefill(dec, prompt)
        hist = []
        if mode == "graph":
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            # warm the launch path on the side stream, then restore the
            # state it consumed before capturing
            save = (dec.win_tok.clone(), dec.win_start.clone(),
                    dec.k_cache.clone(), dec.v_cache.clone())
            with torch.cuda.stream(s):
                dec.step()
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            for dst, src in zip((dec.win_tok, dec.win_start, dec.k_cache,
                                 dec.v_cache), save):
                dst.copy_(src)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                dec.step()
            torch.cuda.synchronize()
        for t in range(steps):
            if mode == "graph":
                g.replay()
            else:
                dec.step()
            torch.cuda.synchronize()
            hist.append((dec.win_tok.cpu().numpy().copy(),
                         dec.win_start.cpu().numpy().copy(),
                         dec.entropy.cpu().numpy().copy(),
                         dec.committed_tok.cpu().numpy().copy()))
        runs.append((hist, dec.k_cache.cpu().clone(), dec.v_cache.cpu().clone()))
    (h0, k0, v0), (h1, k1, v1) = runs
    for a, b in zip(h0, h1):
        for x, y in zip(a, b):
            assert np.array_equal(x, y, equal_nan=True)
    assert torch.equal(k0.view(torch.int16), k1.view(torch.int16))
    assert torch.equal(v0.view(torch.int16), v1.view(torch.int16))


@pytest.mark.parametrize("B,W", [(2, 32), (8, 32), (16, 32), (13, 31)])
def test_qwen3_shaped_layer_against_oracle(B, W):
    """One layer at the Qwen3-8B sizes (hidden 4096, 32/8 heads of 128, MLP
    12288; vocabulary cut to 4096), B sequences of W slots: 64 rows (the
    split-K products, the RMSNorms summing split partials), 256 rows (the
    2-D tiled products, o's input packed, residual-add products split over
    8 workgroups), 512 rows (the gate/up product in 256-token tiles) or 403
    rows (those tiles with a partly filled last row tile and a partly used
    second group of 256 tokens).  Prefill of 2W prompt tokens, then two
    streaming steps checked against the full-sequence oracle as in the tiny
    decoder test."""
    ms = WL.ModelShape("qwen3_8b_1l_v4k", 302, L=1, Hd=4096, Hq=32, Hkv=8,
                       D=128, I=12288, V=4096)
    c0, T = 2 * W, 1.0                  # prompt of two all-filled windows
    wbits = WL.model_weights(ms, seed=0)
    wf = MO.decode(wbits)
    dec, bt = _decoder(ms, wbits, B, W, pages_per_seq=10, T=T)
    prompt = WL.model_prompt(ms, B, c0, seed=5)
    _prefill(dec, prompt)
    y = [list(prompt[b]) for b in range(B)]
    compared = 0
    for t in range(2):
        win = dec.win_tok.cpu().numpy().copy()
        c = dec.win_start.cpu().numpy().copy()
        dec.forward()
        torch.cuda.synchronize()
        am = dec.argmax.cpu().numpy()
        H = dec.entropy.cpu().numpy()
        kw = _f64(dec.k_win)
        for b in range(B):
            r = MO.window_scores(ms, wf, y[b], list(win[b]), T)
            for i in range(r["n_obs"], W):
                lg = np.sort(r["logits"][i])
                assert abs(H[b, i] - r["H"][i]) < 0.03, (t, b, i)
                if lg[-1] - lg[-2] > 0.05:
                    assert am[b, i] == r["tok"][i], (t, b, i)
                    compared += 1
            kref = r["k"][:, c[b] + np.asarray(r["perm"])]
            assert np.abs(kw[:, b] - kref).max() < 0.02 * np.abs(kref).max()
        exp = [O.commit(list(win[b]), int(c[b]), list(H[b].astype(np.float64)),
                        list(am[b]), dec.tau, dec.lam, list(bt[b]))
               for b in range(B)]
        dec.commit()
        torch.cuda.synchronize()
        for b in range(B):
            assert int(dec.n_commit[b]) == exp[b]["n"]
            assert list(dec.win_tok[b].cpu().numpy()) == exp[b]["win"]
            y[b] += exp[b]["committed"]
    assert compared > 10
