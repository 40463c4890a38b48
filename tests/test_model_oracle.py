"""CPU pins of the decoder oracle (oracle/model_oracle.py).

The decoder layer is pinned to an independent implementation: the Qwen3
model of the installed `transformers` package, run in float64 with the same
weights (it keeps RMSNorm and the rotary tables in float32, hence the 1e-5
tolerance; a wrong norm placement, head mapping or gate/up order moves the
logits by O(1)).  The same model with a 4-D additive mask built from the
logical visibility rule pins the window forward.  Sec. 5.2's cache argument
is checked as a property of the oracle: the prefix's keys and values, and
those of the leftmost filled run, do not depend on the rest of the window.
"""
import numpy as np
import pytest
import torch

from oracle import model_oracle as MO
from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL

MS = WL.MODEL_SHAPES["tiny2"]


@pytest.fixture(scope="module")
def weights():
    return MO.decode(WL.model_weights(MS, seed=0))


def _hf_model(w):
    transformers = pytest.importorskip("transformers")
    cfg = transformers.Qwen3Config(
        vocab_size=MS.V, hidden_size=MS.Hd, intermediate_size=MS.I,
        num_hidden_layers=MS.L, num_attention_heads=MS.Hq,
        num_key_value_heads=MS.Hkv, head_dim=MS.D, rope_theta=MS.theta,
        rms_norm_eps=MS.eps, tie_word_embeddings=False,
        attn_implementation="eager")
    m = transformers.Qwen3ForCausalLM(cfg).double().eval()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    Hq, Hkv, D, I = MS.Hq, MS.Hkv, MS.D, MS.I
    sd = {"model.embed_tokens.weight": t(w["embed"]),
          "lm_head.weight": t(w["lm_head"]),
          "model.norm.weight": t(w["final_norm"])}
    for l in range(MS.L):
        p = f"model.layers.{l}."
        qkv = w["w_qkv"][l]
        sd.update({
            p + "input_layernorm.weight": t(w["attn_norm"][l]),
            p + "post_attention_layernorm.weight": t(w["mlp_norm"][l]),
            p + "self_attn.q_proj.weight": t(qkv[:Hq * D]),
            p + "self_attn.k_proj.weight": t(qkv[Hq * D:(Hq + Hkv) * D]),
            p + "self_attn.v_proj.weight": t(qkv[(Hq + Hkv) * D:]),
            p + "self_attn.o_proj.weight": t(w["w_o"][l]),
            p + "self_attn.q_norm.weight": t(w["q_norm"][l]),
            p + "self_attn.k_norm.weight": t(w["k_norm"][l]),
            p + "mlp.gate_proj.weight": t(w["w_gate_up"][l][:I]),
            p + "mlp.up_proj.weight": t(w["w_gate_up"][l][I:]),
            p + "mlp.down_proj.weight": t(w["w_down"][l])})
    m.load_state_dict(sd, strict=True)
    return m


def test_decoder_matches_transformers_causal(weights):
    """All positions observed: the plain causal LM."""
    m = _hf_model(weights)
    n = 40
    toks = WL.model_prompt(MS, 1, n, seed=1)[0]
    with torch.no_grad():
        ref = m(input_ids=torch.from_numpy(toks[None].astype(np.int64))
                ).logits[0].numpy()
    h, _, _ = MO.forward(MS, weights, toks, list(range(n)),
                         np.tril(np.ones((n, n), dtype=bool)))
    got = h @ weights["lm_head"].T
    assert np.abs(got - ref).max() < 1e-5 * max(1.0, np.abs(ref).max())


def test_window_forward_matches_transformers_visibility_mask(weights):
    """A window with masks: the same model under a 4-D additive mask built
    from the logical visibility rule, masks fed as the [M] row."""
    m = _hf_model(weights)
    c, W = 24, 16
    toks = WL.model_prompt(MS, 1, c + W, seed=2)[0]
    win = [int(x) for x in toks[c:]]
    for s in (1, 2, 5, 9, 10, 15):
        win[s] = O.MASK
    vis = MO.logical_visibility(c, win)
    ids = [int(x) for x in toks[:c]] + [x if x != O.MASK else MS.mask_row
                                        for x in win]
    mask4 = torch.where(torch.from_numpy(vis), 0.0,
                        float("-inf")).double()[None, None]
    with torch.no_grad():
        ref = m(input_ids=torch.tensor([ids]), attention_mask=mask4,
                position_ids=torch.arange(c + W)[None]).logits[0].numpy()
    hw, _, _ = MO.window_forward(MS, weights, toks[:c], win)
    got = hw @ weights["lm_head"].T
    assert np.abs(got - ref[c:]).max() < 1e-5 * max(1.0, np.abs(ref).max())


def test_rmsnorm_and_silu_against_torch():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((7, 96)) * 3.0
    g = 1.0 + 0.1 * rng.standard_normal(96)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,),
                                       torch.from_numpy(g), eps=1e-6).numpy()
    assert np.abs(MO.rmsnorm(x, g, 1e-6) - ref).max() < 1e-13
    # a constant row c normalises to g * c / sqrt(c^2 + eps)
    row = np.full(96, -2.5)
    assert np.allclose(MO.rmsnorm(row, g, 1e-6),
                       g * -2.5 / np.sqrt(6.25 + 1e-6), rtol=1e-15)
    y = rng.standard_normal(1000) * 20.0
    assert np.abs(MO.silu(y) - torch.nn.functional.silu(
        torch.from_numpy(y)).numpy()).max() < 1e-12
    assert MO.silu(np.array([0.0]))[0] == 0.0
    assert MO.silu(np.array([-1e4]))[0] == 0.0


def test_zero_output_projections_leave_the_embedding(weights):
    """With W_o = W_down = 0 every residual branch adds zero: the final
    hidden state is RMSNorm(E[token]) * g_final."""
    w = dict(weights)
    w["w_o"] = np.zeros_like(w["w_o"])
    w["w_down"] = np.zeros_like(w["w_down"])
    toks = WL.model_prompt(MS, 1, 9, seed=4)[0]
    h, _, _ = MO.forward(MS, w, toks, list(range(9)),
                         np.tril(np.ones((9, 9), dtype=bool)))
    ref = MO.rmsnorm(w["embed"][toks], w["final_norm"], MS.eps)
    assert np.abs(h - ref).max() < 1e-12


def test_cache_validity_of_prefix_and_leftmost_run(weights):
    """Sec. 5.2: keys/values of the committed prefix and of the leftmost
    filled run equal those of a causal forward over those tokens alone,
    whatever else the window holds; a filled slot after a mask is not
    cache-valid in general (it would see a different context once the
    mask is filled)."""
    c, W = 20, 12
    toks = WL.model_prompt(MS, 1, c + W, seed=5)[0]
    win = [int(x) for x in toks[c:]]
    for s in (4, 7, 8):
        win[s] = O.MASK
    n = 4                                        # leftmost filled run
    _, ks, vs = MO.window_forward(MS, weights, toks[:c], win)
    run = list(toks[:c + n])
    _, ks0, vs0 = MO.forward(MS, weights, run, list(range(c + n)),
                             np.tril(np.ones((c + n, c + n), dtype=bool)))
    assert np.abs(ks[:, :c + n] - ks0).max() < 1e-10
    assert np.abs(vs[:, :c + n] - vs0).max() < 1e-10
    # the filled slot at window index 5 sits after a mask; with the mask
    # filled by some token its key changes
    win2 = list(win)
    win2[4] = 7
    _, ks2, _ = MO.window_forward(MS, weights, toks[:c], win2)
    assert np.abs(ks2[:, c + 5] - ks[:, c + 5]).max() > 1e-3


def test_window_scores_physical_order(weights):
    """Scores come back in the physical order of Eq. 5/6: row i is logical
    slot perm[i]."""
    c, W = 10, 8
    toks = WL.model_prompt(MS, 1, c + W, seed=6)[0]
    win = [int(x) for x in toks[c:]]
    win[1] = win[3] = win[6] = O.MASK
    r = MO.window_scores(MS, weights, toks[:c], win, temperature=0.1)
    perm, _, _, n_obs = O.reorder(win, c)
    assert list(r["perm"]) == list(perm) and r["n_obs"] == n_obs == 5
    hw, _, _ = MO.window_forward(MS, weights, toks[:c], win)
    lg = hw[perm[6]] @ weights["lm_head"].T
    assert np.abs(r["logits"][6] - lg).max() < 1e-12
    assert r["tok"][6] == int(np.argmax(lg))
