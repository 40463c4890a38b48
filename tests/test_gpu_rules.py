"""GPU parity of the decoding rules of wedlm_commit_rule: block-wise
stop-and-wait commit (Fig. 3, Sec. 6.4) and one token per step (Sec. 6.2),
against the fp64 oracle's commit under the same rule.

* Whole decode steps (reorder, attention, score, commit) on seeded
  workloads, with the edge windows (every slot filled: the block rule
  commits all W; every slot a mask).
* The commit step alone over a 48-step stream per rule, driven by seeded
  decision inputs (entropy on a 1/16 grid with many exact zeros, so ties and
  exact threshold equalities occur, greedy tokens, window K/V rows): both
  sides evolve their own windows from the same inputs, and every step is
  compared bit-exactly (commit count, committed tokens and slots, selection,
  window, prefix length), with the appended cache rows checked at the end.
"""
import numpy as np
import pytest

from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL
from tests import parity_lib as PL

pytestmark = pytest.mark.gpu

RULES = ["block", "one"]


def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("rule", RULES)
def test_rule_decode_step(rule):
    _gpu()
    wl = WL.Workload("rules_step", 70, B=6, W=16, Hq=4, Hkv=2, D=64, V=700,
                     prefix=20, prefix_hi=300, obs_frac=0.0, obs_frac_hi=0.8,
                     spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    d["win_tok"][1] = np.arange(16) + 5          # every slot filled
    d["win_tok"][2] = -1                          # every slot a mask
    n_obs = (d["win_tok"] != -1).sum(1)
    d["logits"] = WL.logits(wl, n_obs, 0, 0)
    PL.log(f"case rule step {rule}: B={wl.B} W={wl.W}")
    g, _, dev = PL.run_gpu_step(wl, d, rule=rule)
    o = PL.oracle_step(wl, d, attn_seqs=range(wl.B), rule=rule)
    PL.check_reorder(wl, g, o)
    PL.check_attention(wl, g, o, range(wl.B))
    PL.check_score(wl, d, g, o)
    PL.check_commit(wl, d, g, o)
    PL.check_append(wl, dev, g, o)
    if rule == "block":
        assert int(g["n_commit"][1]) == wl.W
        assert (g["win_tok"][1] == -1).all()
    else:
        assert int((g["selected"][2] != 0).sum()) == 1


@pytest.mark.parametrize("rule", ["stream"] + RULES)
@pytest.mark.parametrize("W,lam", [(7, 0.125), (32, 0.1), (64, 0.0625)])
def test_rule_commit_stream(rule, W, lam):
    torch = _gpu()
    from paper_2512_22737_amd import wedlm
    B, Hkv, D, steps, tau = 24, 2, 64, 48, 0.75
    seed = 3
    rng = np.random.default_rng(1234 + W)
    c0 = rng.integers(0, 200, size=B).astype(np.int32)
    maxp = (int(c0.max()) + steps * W + W) // WL.PAGE + 2
    num_pages = B * maxp
    bt = rng.permutation(num_pages).reshape(B, maxp).astype(np.int32)
    win0 = np.full((B, W), -1, dtype=np.int32)
    win0[: B // 2] = np.where(rng.random((B // 2, W)) < 0.4,
                              rng.integers(0, 999, (B // 2, W)), -1)
    PL.log(f"case commit stream rule={rule} W={W} lam={lam}: B={B} "
           f"steps={steps}")

    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    win_d, c_d, bt_d = dev(win0), dev(c0), dev(bt)
    kc = torch.zeros(num_pages, Hkv, WL.PAGE, D, dtype=torch.bfloat16,
                     device="cuda")
    vc = torch.zeros(num_pages, Hkv, D, WL.PAGE, dtype=torch.bfloat16,
                     device="cuda")
    outs = dict(n=torch.empty(B, dtype=torch.int32, device="cuda"),
                tok=torch.empty(B, W, dtype=torch.int32, device="cuda"),
                slot=torch.empty(B, W, dtype=torch.int32, device="cuda"),
                sel=torch.empty(B, W, dtype=torch.uint8, device="cuda"),
                st=torch.empty(B, dtype=torch.int32, device="cuda"))
    win = [list(map(int, win0[b])) for b in range(B)]
    c = [int(x) for x in c0]
    last_rows = {}
    for t in range(steps):
        h, tok, k, v = WL.decision_inputs(B, W, Hkv, D, seed, t)
        kd = dev(k).view(torch.int16).view(torch.bfloat16)
        vd = dev(v).view(torch.int16).view(torch.bfloat16)
        wedlm.wedlm_commit_rule(win_d, c_d, dev(tok), dev(h), tau, lam, kd,
                                vd, kc, vc, bt_d, outs["n"], outs["tok"],
                                outs["slot"], outs["sel"], outs["st"],
                                wedlm.RULES[rule])
        g = {k2: v2.cpu().numpy() for k2, v2 in outs.items()}
        gw, gc = win_d.cpu().numpy(), c_d.cpu().numpy()
        assert (g["st"] == 0).all(), t
        for b in range(B):
            r = O.commit(win[b], c[b], h[b].astype(np.float64), tok[b], tau,
                         lam, bt[b], rule=rule)
            n = r["n"]
            assert int(g["n"][b]) == n, (t, b)
            assert list(g["tok"][b][:n]) == r["committed"], (t, b)
            assert list(g["slot"][b][:n]) == r["slots"], (t, b)
            assert list(g["sel"][b]) == r["selected"], (t, b)
            assert list(gw[b]) == r["win"], (t, b)
            assert int(gc[b]) == r["c"], (t, b)
            if rule == "one" and any(x == -1 for x in win[b]):
                assert sum(map(bool, r["selected"])) == 1
            if rule == "block":
                assert n in (0, W)
            for j, slot in enumerate(r["slots"]):
                last_rows[slot] = (k[b, j], v[b, j])
            win[b], c[b] = r["win"], r["c"]
    # every appended row holds the K/V of the step that committed it
    kh = PL.bf16_bits(kc)
    vh = PL.bf16_bits(vc)
    assert last_rows, "nothing was committed"
    for slot, (kr, vr) in last_rows.items():
        pg, row = slot // WL.PAGE, slot % WL.PAGE
        assert (kh[pg, :, row, :] == kr).all(), slot
        assert (vh[pg, :, :, row] == vr).all(), slot
    PL.log(f"  {steps} steps bit-exact, {len(last_rows)} appended rows, "
           f"p_cache {sum(c[b] - int(c0[b]) for b in range(B)) / (steps * B * W):.3f}")


def test_rule_argument_is_checked():
    torch = _gpu()
    from paper_2512_22737_amd import wedlm
    B, W, Hkv, D = 1, 4, 1, 64
    z = lambda *s, dt=torch.int32: torch.zeros(*s, dtype=dt, device="cuda")
    args = [z(B, W), z(B), z(B, W), z(B, W, dt=torch.float32), 0.9, 0.1,
            z(B, W, Hkv, D, dt=torch.bfloat16), z(B, W, Hkv, D, dt=torch.bfloat16),
            z(2, Hkv, 16, D, dt=torch.bfloat16), z(2, Hkv, D, 16, dt=torch.bfloat16),
            z(B, 2), z(B), z(B, W), z(B, W), z(B, W, dt=torch.uint8), z(B)]
    with pytest.raises(wedlm.WedlmError):
        wedlm.wedlm_commit_rule(*args, 3)
