"""Shared helpers of the GPU parity tests: run one decode step through the
C ABI and the same step through the fp64 oracle, on the same seeded inputs,
and compare them."""
from __future__ import annotations

import math
import sys
from typing import Dict, List, Optional, Sequence

import numpy as np

from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL

ATTN_MAX_ABS = 2e-2      # max |o - r| over compared elements
ATTN_REL_NORM = 1e-2     # ||o - r|| / ||r|| over compared elements
H_REL, H_ABS = 1e-5, 1e-12
NEAR = 1e-6              # near-tie / near-threshold band, reported apart


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(d: dict):
    import torch
    out = {}
    for k, v in d.items():
        if not isinstance(v, np.ndarray):
            out[k] = v
            continue
        t = torch.from_numpy(np.ascontiguousarray(v))
        if v.dtype == np.uint16:
            t = t.view(torch.int16).view(torch.bfloat16)
        out[k] = t.cuda()
    return out


def bf16_bits(t) -> np.ndarray:
    import torch
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def run_gpu_step(wl: WL.Workload, d: dict, max_prefix: Optional[int] = None,
                 rule: str = "stream"):
    """One decode step through the C ABI (under the decoding rule `rule`).
    Returns host copies of every output plus the device state for further
    steps."""
    import torch
    from paper_2512_22737_amd import wedlm
    dev = to_dev(d)
    c = d["win_start"]
    mp = int(c.max()) if max_prefix is None else max_prefix
    step = wedlm.DecodeStep(wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, wl.V, mp,
                            theta=wl.theta, tau=wl.tau, lam=wl.lam,
                            temperature=wl.temp, rule=rule)
    step(dev["win_tok"], dev["win_start"], dev["qkv_in"], dev["logits"],
         dev["k_cache"], dev["v_cache"], dev["block_table"])
    torch.cuda.synchronize()
    r = dict(
        perm=step.perm.cpu().numpy(), pos_ids=step.pos_ids.cpu().numpy(),
        tok_phys=step.tok_phys.cpu().numpy(), n_obs=step.n_obs.cpu().numpy(),
        q_phys=bf16_bits(step.q_phys), k_phys=bf16_bits(step.k_phys),
        v_phys=bf16_bits(step.v_phys),
        out=step.out.float().cpu().numpy().astype(np.float64),
        lse=step.lse.cpu().numpy().astype(np.float64),
        attn_status=step.attn_status.cpu().numpy(),
        argmax=step.argmax.cpu().numpy(),
        entropy=step.entropy.cpu().numpy(), pmax=step.pmax.cpu().numpy(),
        n_commit=step.n_commit.cpu().numpy(),
        committed_tok=step.committed_tok.cpu().numpy(),
        committed_slot=step.committed_slot.cpu().numpy(),
        selected=step.selected.cpu().numpy(), status=step.status.cpu().numpy(),
        win_tok=dev["win_tok"].cpu().numpy(),
        win_start=dev["win_start"].cpu().numpy(),
    )
    return r, step, dev


def oracle_step(wl: WL.Workload, d: dict, attn_seqs: Sequence[int] = (),
                rows=None, heads=None, rule: str = "stream"):
    """The oracle's view of the same step.  Attention is evaluated for the
    listed sequences (all rows/heads unless sampled)."""
    res = []
    for b in range(wl.B):
        win = list(map(int, d["win_tok"][b]))
        c = int(d["win_start"][b])
        perm, pos, tok_phys, n_obs = O.reorder(win, c)
        q, k, v = O.rope_window(d["qkv_in"][b], perm, pos, wl.Hq, wl.Hkv,
                                wl.theta)
        e = dict(perm=perm, pos=pos, tok_phys=tok_phys, n_obs=n_obs, q=q, k=k,
                 v=v)
        if b in attn_seqs:
            kb, vb = WL.gather_prefix(d["k_cache"], d["v_cache"],
                                      d["block_table"], b, c)
            rr = list(range(wl.W)) if rows is None else rows(b, n_obs)
            hh = list(range(wl.Hq)) if heads is None else heads(b)
            o, l = O.window_attn(q, k, v, O.bf16_to_f64(kb),
                                 O.bf16_to_f64(vb), rr, hh)
            e.update(attn_rows=rr, attn_heads=hh, attn=o, lse=l)
        tok, H, pm = O.score(d["logits"][b], n_obs, wl.temp)
        e.update(argmax=tok, entropy=H, pmax=pm)
        cm = O.commit(win, c, O.to_f32_decision(H), tok, wl.tau, wl.lam,
                      d["block_table"][b], rule=rule)
        e["commit"] = cm
        res.append(e)
    return res


def check_reorder(wl, g, o):
    for b in range(wl.B):
        assert list(g["perm"][b]) == o[b]["perm"], b
        assert list(g["pos_ids"][b]) == o[b]["pos"], b
        assert list(g["tok_phys"][b]) == o[b]["tok_phys"], b
        assert int(g["n_obs"][b]) == o[b]["n_obs"], b
        # rotated Q/K within one bf16 ulp of the fp64 rotation, V exact
        for name, ref in (("q_phys", o[b]["q"]), ("k_phys", o[b]["k"])):
            got = O.bf16_to_f64(g[name][b])
            ulp = np.abs(ref) * 2.0 ** -7 + 1e-30
            assert (np.abs(got - ref) <= ulp).all(), (name, b)
        assert (O.bf16_to_f64(g["v_phys"][b]) == o[b]["v"]).all(), b


def check_attention(wl, g, o, seqs, lse_bound=None):
    """lse_bound(b): per (row, head) bound on |lse - lse_ref| (default
    2e-2 everywhere)."""
    worst_abs, num, den, n = 0.0, 0.0, 0.0, 0
    for b in seqs:
        rr, hh = o[b]["attn_rows"], o[b]["attn_heads"]
        got = g["out"][b][np.ix_(rr, hh)]
        ref = o[b]["attn"]
        err = np.abs(got - ref)
        worst_abs = max(worst_abs, float(err.max()))
        num += float((err ** 2).sum())
        den += float((ref ** 2).sum())
        n += err.size
        glse = g["lse"][b][np.ix_(rr, hh)]
        bound = 2e-2 if lse_bound is None else lse_bound(b)
        assert (np.abs(glse - o[b]["lse"]) < bound).all(), b
        assert int(g["attn_status"][b]) == 0, b
    rel = math.sqrt(num / max(den, 1e-300))
    log(f"  attention: {n} values, max abs {worst_abs:.3e}, rel norm {rel:.3e}")
    assert worst_abs <= ATTN_MAX_ABS
    assert rel <= ATTN_REL_NORM
    return worst_abs, rel


def check_score(wl, d, g, o):
    near_tie = 0
    worst = 0.0
    for b in range(wl.B):
        n_obs = o[b]["n_obs"]
        for i in range(n_obs, wl.W):
            assert int(g["argmax"][b, i]) == int(o[b]["argmax"][i]), (b, i)
            top2 = np.partition(d["logits"][b, i], -2)[-2:]
            near_tie += int(abs(float(top2[1]) - float(top2[0])) < NEAR)
            Hr = o[b]["entropy"][i]
            Hg = float(g["entropy"][b, i])
            err = abs(Hg - Hr)
            assert err <= H_REL * abs(Hr) + H_ABS, (b, i, Hg, Hr)
            worst = max(worst, err / max(abs(Hr), 1e-300))
            pr = o[b]["pmax"][i]
            assert abs(float(g["pmax"][b, i]) - pr) <= H_REL * pr, (b, i)
    log(f"  score: worst entropy rel err {worst:.3e}, near ties {near_tie}")
    return worst


def near_threshold(wl, o_b) -> bool:
    """True if a mask slot's decision sits within NEAR of its threshold or of
    another mask's fallback key (such rows are reported, not failed)."""
    cm = o_b["commit"]
    perm = o_b["perm"]
    phys = {s: i for i, s in enumerate(perm)}
    masks = [s for s, i in phys.items() if i >= o_b["n_obs"]]
    if not masks:
        return False
    s0 = min(masks)
    keys = []
    for s in masks:
        H = float(o_b["entropy"][phys[s]])
        d = s - s0
        if abs(H - (wl.tau - wl.lam * d)) < NEAR:
            return True
        keys.append(H + wl.lam * d)
    keys.sort()
    return len(keys) > 1 and keys[1] - keys[0] < NEAR


def check_commit(wl, d, g, o):
    """Commit count, committed tokens and slots, status and the new prefix
    length depend on no entropy and are always compared bit-exactly.  The
    selection and the refilled window are compared bit-exactly too, except
    on sequences whose decision sits within NEAR of a threshold, which are
    counted and reported."""
    near = 0
    for b in range(wl.B):
        cm = o[b]["commit"]
        assert int(g["status"][b]) == 0, b
        assert int(g["n_commit"][b]) == cm["n"], b
        n = cm["n"]
        assert list(g["committed_tok"][b][:n]) == cm["committed"], b
        assert list(g["committed_slot"][b][:n]) == cm["slots"], b
        assert (g["committed_tok"][b][n:] == -1).all()
        assert int(g["win_start"][b]) == cm["c"], b
        same = (list(g["selected"][b]) == cm["selected"] and
                list(g["win_tok"][b]) == cm["win"])
        if not same and near_threshold(wl, o[b]):
            near += 1
            continue
        assert list(g["selected"][b]) == cm["selected"], b
        assert list(g["win_tok"][b]) == cm["win"], b
    log(f"  commit: {wl.B} sequences, near-threshold mismatches {near}")
    return near


def check_append(wl, step_dev, g, o):
    """Committed rows now sit in the cache: V bit-exact, K within 1 ulp of
    the fp64 rotation."""
    import torch
    kc = bf16_bits(step_dev["k_cache"])
    vc = bf16_bits(step_dev["v_cache"])
    for b in range(wl.B):
        cm = o[b]["commit"]
        for j, slot in enumerate(cm["slots"]):
            pg, row = slot // WL.PAGE, slot % WL.PAGE
            kref = o[b]["k"][j]                        # [Hkv, D]
            kgot = O.bf16_to_f64(kc[pg, :, row, :])
            assert (np.abs(kgot - kref) <= np.abs(kref) * 2 ** -7 + 1e-30).all()
            vgot = O.bf16_to_f64(vc[pg, :, :, row])
            assert (vgot == o[b]["v"][j]).all()
