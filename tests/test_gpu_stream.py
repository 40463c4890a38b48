"""GPU parity of Algorithm 1's loop: the 512-step streaming workload
(16 sequences, starting prefix 1024, W=32, Hq/Hkv=32/8, D=128, V=151936,
all-mask start, +12 spike on 90% of rows) run through the C ABI, step after
step, against the oracle's stream stored in tests/golden/stream512.json
(written by tests/golden/make_stream512.py, which calls only the oracle).

Bit-exact: the commit count of every step of every sequence, the committed
token stream and the cache slots (both by sha256, the slots also re-derived
from the block table), the window and prefix length before the snapshot
steps, the final window.  Attention at sampled steps and sequences against
the oracle, whose cache is rebuilt from the stored commit counts and the
seeded inputs; the appended V rows of the sampled sequences bit-exact.
"""
import hashlib
import json
import os

import numpy as np
import pytest

from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL
from tests import parity_lib as PL

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "stream512.json")
ATTN_STEPS = (1, 255, 511)
ATTN_SEQS = (0, 9)
ATTN_ROWS = (0, 5, 17, 31)
SEED = 0


def _sha(a) -> str:
    return hashlib.sha256(np.asarray(a, dtype="<i4").tobytes()).hexdigest()


def test_stream512_against_oracle_stream():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_22737_amd import wedlm
    wedlm.lib()
    gold = json.load(open(GOLDEN))
    wl = WL.WORKLOADS["stream512"]
    assert gold["steps"] == wl.steps and gold["B"] == wl.B
    B, W, steps = wl.B, wl.W, wl.steps

    PL.log(f"case stream512: B={B} W={W} steps={steps}")
    d = WL.step_inputs(wl, seed=SEED)
    dev = PL.to_dev(d)
    pool = torch.from_numpy(WL.logit_pool(wl, SEED)).to("cuda")
    c0 = d["win_start"].copy()
    step = wedlm.DecodeStep(B, W, wl.Hq, wl.Hkv, wl.D, wl.V,
                            int(c0.max()) + steps * W, theta=wl.theta,
                            tau=wl.tau, lam=wl.lam, temperature=wl.temp)

    n_hist = np.zeros((steps, B), dtype=np.int64)
    toks = [[] for _ in range(B)]
    slots = [[] for _ in range(B)]
    keep = {b: [] for b in ATTN_SEQS}     # committed qkv rows per step
    attn_got, qkv_at = {}, {}
    snaps = set(int(s) for s in gold["snapshots"])
    for t in range(steps):
        qkv_np = d["qkv_in"] if t == 0 else WL.qkv(wl, SEED, t)
        qkv = PL.to_dev({"q": qkv_np})["q"]
        logits = WL.logits_torch(wl, pool, SEED, t)
        if t in snaps:
            win_now = dev["win_tok"].cpu().numpy()
            c_now = dev["win_start"].cpu().numpy()
            for b in range(B):
                s = gold["sequences"][b]["snapshots"][str(t)]
                assert list(win_now[b]) == s["win"], (t, b)
                assert int(c_now[b]) == s["c"], (t, b)
        step(dev["win_tok"], dev["win_start"], qkv, logits, dev["k_cache"],
             dev["v_cache"], dev["block_table"])
        n = step.n_commit.cpu().numpy()
        assert (step.status.cpu().numpy() == 0).all(), t
        ct = step.committed_tok.cpu().numpy()
        cs = step.committed_slot.cpu().numpy()
        n_hist[t] = n
        for b in range(B):
            toks[b] += list(ct[b, :n[b]])
            slots[b] += list(cs[b, :n[b]])
            assert int(n[b]) == gold["sequences"][b]["n"][t], (t, b)
        for b in ATTN_SEQS:
            keep[b].append(qkv_np[b, :gold["sequences"][b]["n"][t]].copy())
        if t in ATTN_STEPS:
            attn_got[t] = PL.bf16_bits(step.out)[list(ATTN_SEQS)]
            qkv_at[t] = qkv_np[list(ATTN_SEQS)].copy()
        if t % 64 == 63:
            PL.log(f"  step {t + 1}/{steps}: committed "
                   f"{sum(len(x) for x in toks)} tokens")

    win_end = dev["win_tok"].cpu().numpy()
    c_end = dev["win_start"].cpu().numpy()
    bt = d["block_table"]
    for b in range(B):
        g = gold["sequences"][b]
        assert len(toks[b]) == g["n_tokens"], b
        assert toks[b][:64] == g["tokens_head"], b
        assert _sha(toks[b]) == g["tokens_sha256"], b
        assert _sha(slots[b]) == g["slots_sha256"], b
        assert slots[b] == [O.slot_of(bt[b], int(c0[b]) + j)
                            for j in range(len(slots[b]))], b
        assert list(win_end[b]) == g["final_win"], b
        assert int(c_end[b]) == g["final_c"], b
    PL.log(f"  stream: {steps} steps, p_cache "
           f"{O.p_cache(n_hist, W):.4f} (oracle {gold['p_cache']:.4f})")

    # attention at sampled steps, against the oracle on its own cache
    kc = PL.bf16_bits(dev["k_cache"])
    vc = PL.bf16_bits(dev["v_cache"])
    for j, b in enumerate(ATTN_SEQS):
        g = gold["sequences"][b]
        kp, vp = WL.prefix_kv(wl, b, int(c0[b]), SEED)
        cache_k = [O.bf16_to_f64(kp)]
        cache_v = [O.bf16_to_f64(vp)]
        c = int(c0[b])
        for t in range(steps):
            if t in ATTN_STEPS:
                s = g["snapshots"][str(t)]
                assert s["c"] == c
                perm, pos, _, _ = O.reorder(s["win"], c)
                q, k, v = O.rope_window(qkv_at[t][j], perm, pos, wl.Hq,
                                        wl.Hkv, wl.theta)
                ref, _ = O.window_attn(q, k, v, np.concatenate(cache_k),
                                       np.concatenate(cache_v),
                                       rows=ATTN_ROWS)
                got = O.bf16_to_f64(attn_got[t][j])[list(ATTN_ROWS)]
                err = np.abs(got - ref)
                rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
                PL.log(f"  attention seq {b} step {t} (c={c}): max abs "
                       f"{err.max():.2e}, rel {rel:.2e}")
                assert err.max() <= PL.ATTN_MAX_ABS
                assert rel <= PL.ATTN_REL_NORM
            n = g["n"][t]
            if n:
                # committed rows: logical slots 0..n-1 at positions c..
                _, kn, vn = O.rope_window(keep[b][t], list(range(n)),
                                          [c + i for i in range(n)], wl.Hq,
                                          wl.Hkv, wl.theta)
                cache_k.append(kn)
                cache_v.append(vn)
                # appended V is the window's V, bit-exact, in its slots
                for i in range(n):
                    slot = O.slot_of(bt[b], c + i)
                    got_v = O.bf16_to_f64(vc[slot // WL.PAGE, :, :,
                                             slot % WL.PAGE])
                    assert (got_v == vn[i]).all(), (b, t, i)
                    got_k = O.bf16_to_f64(kc[slot // WL.PAGE, :,
                                             slot % WL.PAGE, :])
                    assert (np.abs(got_k - kn[i]) <=
                            np.abs(kn[i]) * 2 ** -7 + 1e-30).all()
            c += n

