"""CPU pins of the dual-stream attention oracle (Sec. 4.2).

* masked_attention under a causal mask equals torch's scaled-dot-product
  attention with is_causal in fp64 (a library routine);
* the memory stream's rows are exactly that causal attention;
* block k of the prediction stream equals the inference-time window step
  (window_attn, written separately for the decode path) with the memory
  tokens of the earlier blocks as the cached prefix and the reordered block
  as the window: the paper's claim that dual-stream training simulates
  prefix-conditioned decoding, as an identity between the two oracles;
* the first block sees no memory, and with one block covering the whole
  sequence the prediction stream never reads the memory stream;
* the reordered block puts observed positions first (Eq. 5/6 per block).
"""
import numpy as np
import pytest
import torch

from oracle import wedlm_oracle as O


def _qkv(n, Hq, Hkv, D, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((n, Hq, D)), rng.standard_normal((n, Hkv, D)),
            rng.standard_normal((n, Hkv, D)))


def _masked(L, B, seed, frac=0.5):
    rng = np.random.default_rng(seed)
    return {p for p in range(L) if rng.random() < frac}


def test_masked_attention_causal_is_sdpa():
    n, Hq, Hkv, D = 24, 4, 2, 16
    q, k, v = _qkv(n, Hq, Hkv, D, 1)
    out, _ = O.masked_attention(q, k, v, np.tril(np.ones((n, n), dtype=bool)))
    G = Hq // Hkv
    t = lambda a: torch.from_numpy(a).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(np.repeat(k, G, axis=1)), t(np.repeat(v, G, axis=1)),
        is_causal=True)[0].permute(1, 0, 2).numpy()
    assert np.abs(out - ref).max() < 1e-12


@pytest.mark.parametrize("L,B", [(24, 8), (32, 32), (40, 16)])
def test_dual_stream_blocks_equal_window_steps(L, B):
    Hq, Hkv, D = 4, 2, 16
    masked = _masked(L, B, L + B)
    rows = O.dual_stream_order(L, B, masked)
    vis = O.dual_stream_visible(L, B, masked)
    q, k, v = _qkv(2 * L, Hq, Hkv, D, 7)
    out, lse = O.masked_attention(q, k, v, vis)
    # memory rows: plain causal attention over the memory stream
    mout, mlse = O.masked_attention(q[:L], k[:L], v[:L],
                                    np.tril(np.ones((L, L), dtype=bool)))
    assert np.abs(out[:L] - mout).max() < 1e-12
    # prediction block k: the decode step with the memory of blocks < k
    for b0 in range(0, L, B):
        r0 = L + b0
        r1 = L + min(b0 + B, L)
        wout, wlse = O.window_attn(q[r0:r1], k[r0:r1], v[r0:r1], k[:b0],
                                   v[:b0])
        assert np.abs(out[r0:r1] - wout).max() < 1e-12
        assert np.abs(lse[r0:r1] - wlse).max() < 1e-12
        # the reordered block: observed positions first, each group in order
        blk = [p for (_, p, _) in rows[r0:r1]]
        obs = [p for p in range(b0, min(b0 + B, L)) if p not in masked]
        assert blk[:len(obs)] == obs
        assert sorted(blk) == list(range(b0, min(b0 + B, L)))


def test_dual_stream_visibility_structure():
    L, B = 12, 4
    masked = {1, 2, 6, 9, 10, 11}
    vis = O.dual_stream_visible(L, B, masked)
    rows = O.dual_stream_order(L, B, masked)
    # memory never reads the prediction stream; block 0 reads no memory
    assert not vis[:L, L:].any()
    assert not vis[L:L + B, :L].any()
    # one block over the whole sequence: no memory at all
    assert not O.dual_stream_visible(L, L, masked)[L:, :L].any()
    # a prediction token never reads another block of the prediction stream
    for i in range(L, 2 * L):
        for j in range(L, 2 * L):
            if rows[i][1] // B != rows[j][1] // B:
                assert not vis[i, j]
    # block 2 (positions 8..11) reads exactly memory positions 0..7
    assert (vis[L + 2 * B:, :8]).all() and not vis[L + 2 * B:, 8:L].any()
