"""GPU parity: the HIP library through its C ABI against the fp64 oracle, on
the same seeded inputs.

Integer outputs (permutation, positions, tokens, argmax, selections, commit
counts, slots, the new window) are compared bit-exactly; rows whose decision
sits within 1e-6 of a threshold are counted and reported apart.  Attention:
max |o - r| <= 2e-2 and ||o - r|| / ||r|| <= 1e-2 against the fp64 oracle on
the bf16 inputs.  Entropy: |H - H_ref| <= 1e-5 |H_ref| + 1e-12.
"""
import numpy as np
import pytest

from paper_2512_22737_amd import workloads as WL
from tests import parity_lib as PL

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2512_22737_amd import wedlm
    wedlm.lib()     # raises if the HIP library is missing


def _full_check(wl, d, attn_seqs=None, rows=None, heads=None):
    PL.log(f"case {wl.name}: B={wl.B} W={wl.W} Hq={wl.Hq} Hkv={wl.Hkv} "
           f"D={wl.D} V={wl.V} c={list(d['win_start'][:4])}")
    g, step, dev = PL.run_gpu_step(wl, d)
    seqs = list(range(wl.B)) if attn_seqs is None else attn_seqs
    o = PL.oracle_step(wl, d, seqs, rows, heads)
    PL.check_reorder(wl, g, o)
    PL.check_attention(wl, g, o, seqs)
    PL.check_score(wl, d, g, o)
    PL.check_commit(wl, d, g, o)
    PL.check_append(wl, dev, g, o)
    return g, o


def test_tiny_step():
    wl = WL.WORKLOADS["tiny"]
    _full_check(wl, WL.step_inputs(wl, seed=0))


@pytest.mark.parametrize("seed", [1, 2])
def test_tiny_step_more_seeds(seed):
    wl = WL.WORKLOADS["tiny"]
    _full_check(wl, WL.step_inputs(wl, seed=seed))


SMALL = [
    # name, W, Hq, Hkv, D, prefix range, obs fraction range, V
    ("w1_d128_g4", 1, 8, 2, 128, (0, 40), (0.0, 1.0), 500),
    ("w16_d64_g1", 16, 4, 4, 64, (17, 300), (0.0, 0.9), 777),
    ("w33_d128_g8", 33, 16, 2, 128, (1, 129), (0.2, 0.6), 1000),
    ("w64_d128_g4", 64, 8, 2, 128, (200, 700), (0.0, 0.75), 2048),
    ("w64_d64_g2", 64, 4, 2, 64, (0, 31), (0.5, 1.0), 333),
    ("w7_d128_g2_long", 7, 4, 2, 128, (3000, 9000), (0.0, 0.5), 4096),
    # eight waves at D = 64 (256 query rows per kv head), and two query
    # blocks per kv head at D = 64 (384 rows)
    ("w64_d64_g4", 64, 8, 2, 64, (100, 900), (0.1, 0.6), 1500),
    ("w48_d64_g8", 48, 16, 2, 64, (40, 600), (0.0, 0.5), 640),
    # 96 heads of 128: three rounds of rotation items per row in the
    # reorder, two of value pieces
    ("w8_d128_h96", 8, 64, 32, 128, (0, 100), (0.0, 0.8), 300),
]


@pytest.mark.parametrize("name,W,Hq,Hkv,D,pr,fr,V", SMALL)
def test_small_shapes(name, W, Hq, Hkv, D, pr, fr, V):
    wl = WL.Workload(name, 50 + SMALL.index(
        next(s for s in SMALL if s[0] == name)), B=5, W=W, Hq=Hq, Hkv=Hkv,
        D=D, V=V, prefix=pr[0], prefix_hi=pr[1], obs_frac=fr[0],
        obs_frac_hi=fr[1], spike=9.0, spike_prob=0.5)
    _full_check(wl, WL.step_inputs(wl, seed=0))


def test_eight_wave_tile_counts():
    """256 query rows per kv head at D = 128 (eight waves, two per SIMD):
    every count of full 32-key prefix tiles from 0 to 10 in one split,
    with and without a partial last tile, so that both wave halves' barrier
    schedules and the loop's remainder path meet every case."""
    wl = WL.Workload("w64_g4_tiles", 70, B=14, W=64, Hq=8, Hkv=2, D=128,
                     V=600, prefix=330, prefix_hi=330, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    # the block tables cover 330 + W positions; shorter prefixes use a part
    d["win_start"][:] = [0, 31, 32, 64, 95, 96, 128, 161, 192, 224, 256,
                         288, 320, 330]
    _full_check(wl, d)


def test_four_wave_two_per_cu_tile_counts():
    """128 query rows per kv head on a grid of 512 workgroups (64 sequences
    x 8 kv heads): the four-wave kernel that runs two workgroups per CU,
    with its four-slot ring and a barrier after every tile.  Prefixes give
    every count of full tiles from 0 to 10, with and without a partial
    tile; attention checked on those sequences."""
    wl = WL.Workload("w16_g8_two", 72, B=64, W=16, Hq=64, Hkv=8, D=64,
                     V=300, prefix=330, prefix_hi=330, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    lens = [0, 31, 32, 64, 95, 96, 128, 161, 192, 224, 256, 288, 320, 330]
    d["win_start"][:len(lens)] = lens
    _full_check(wl, d, list(range(len(lens))) + [40, 63])


def _lift_scores_from(wl, d, start, alpha):
    """Scores that jump far above the first tile's: coordinate j = D/2 - 1 of
    every query is set to 4 (its RoPE pair turns by under 0.01 rad at these
    positions, so it stays near 4 after rotation), and alpha is added to
    that coordinate of the cached keys of every prefix position >= start
    (bf16).  Every query then scores those keys about 4 * alpha / sqrt(D)
    higher, in common, while the spread among them stays that of the
    original keys: the softmax is well conditioned, however large alpha."""
    j = wl.D // 2 - 1
    qkv = d["qkv_in"]
    qkv[:, :, :wl.Hq, j] = WL.f32_to_bf16_bits(np.float32(4.0))
    k = d["k_cache"]
    bt = d["block_table"]
    for b in range(bt.shape[0]):
        c = int(d["win_start"][b])
        for pos in range(start - start % WL.PAGE, c, WL.PAGE):
            pg = int(bt[b, pos // WL.PAGE])
            lo = max(start - pos, 0)
            f = (k[pg, :, lo:, j].astype(np.uint32) << 16).view(np.float32)
            k[pg, :, lo:, j] = WL.f32_to_bf16_bits(f + np.float32(alpha))


def _grow_check(wl, d, seqs, rows=None, heads=None):
    """A full step check whose lse bound follows from the inputs: the kernel
    scores with queries rounded to bf16 twice (the rotation's output, then
    the pre-scaled copy), each rounding at most 2^-8 relative (half an ulp
    at the bottom of a binade), so its scores and lse are within
    2^-7 * max_k sum_i |q_i k_i| / sqrt(D) of the oracle's (lse moves by at
    most the largest score change)."""
    PL.log(f"case {wl.name}: B={wl.B} W={wl.W} Hq={wl.Hq} Hkv={wl.Hkv} "
           f"D={wl.D} c={list(d['win_start'][:4])}")
    g, step, dev = PL.run_gpu_step(wl, d)
    o = PL.oracle_step(wl, d, seqs, rows, heads)

    def lse_bound(b):
        from oracle import wedlm_oracle as O
        c = int(d["win_start"][b])
        kp, _ = WL.gather_prefix(d["k_cache"], d["v_cache"], d["block_table"],
                                 b, c)
        keys = np.concatenate([O.bf16_to_f64(kp), o[b]["k"]], axis=0)
        q = o[b]["q"]
        rr, hh = o[b]["attn_rows"], o[b]["attn_heads"]
        out = np.zeros((len(rr), len(hh)))
        for hi, h in enumerate(hh):
            ak = np.abs(keys[:, h // wl.G, :])
            for ri, i in enumerate(rr):
                m = (ak[:c + i + 1] @ np.abs(q[i, h])).max()
                out[ri, hi] = 2e-2 + 2.0 ** -7 * m / np.sqrt(wl.D)
        return out

    PL.check_reorder(wl, g, o)
    PL.check_attention(wl, g, o, seqs, lse_bound)
    PL.check_score(wl, d, g, o)
    PL.check_commit(wl, d, g, o)
    PL.check_append(wl, dev, g, o)


@pytest.mark.parametrize("alpha", [200.0, 2000.0])
def test_scores_growing_past_first_tile(alpha):
    """Keys of prefix positions from 64 on lifted by about 70 nats (alpha
    200: past the 64 log2 units the running sum tolerates) or 700 nats
    (alpha 2000: 2^s overflows fp32) above the first two tiles: the kernel
    must raise the reference max, rescale, and shift the in-flight next
    tile.  Sequences of 600-1200 positions split four ways, so one split
    meets the jump inside its range and the others start above it."""
    wl = WL.Workload(f"grow{int(alpha)}", 73, B=3, W=16, Hq=8, Hkv=2, D=128,
                     V=400, prefix=600, prefix_hi=1200, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    _lift_scores_from(wl, d, 64, alpha)
    _grow_check(wl, d, list(range(wl.B)))


def test_scores_growing_two_per_cu():
    """The same jump on the four-wave two-per-CU kernel (128 query rows per
    kv head, 512 workgroups), whose exponent arguments subtract the
    reference max per score instead of seeding the MFMA accumulators."""
    wl = WL.Workload("grow_two", 74, B=64, W=32, Hq=32, Hkv=8, D=128,
                     V=300, prefix=200, prefix_hi=330, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    _lift_scores_from(wl, d, 64, 2000.0)
    _grow_check(wl, d, [0, 1, 33, 63], lambda b, n: _sample_rows(b, n, wl.W),
                lambda b: sorted({0, 3, 4, 31, (5 * b) % 32}))


def test_two_per_cu_with_prefix_splits():
    """128 query rows per kv head on a grid of 128 (sequence, kv head)
    pairs, with a prefix bound long enough to split four ways: the
    four-wave kernel that runs two per CU over 512 workgroups.  Each
    sequence splits its own prefix (0 to 4 splits in use: empty, short and
    long prefixes); attention checked on sampled rows and heads."""
    wl = WL.Workload("two_split", 75, B=16, W=32, Hq=32, Hkv=8, D=128, V=300,
                     prefix=4200, prefix_hi=4200, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    # the block tables and caches cover 4200 + W positions; shorter
    # prefixes use a part
    d["win_start"][:] = [0, 40, 255, 4200, 3000, 1000, 511, 2047, 256, 4100,
                         17, 700, 1500, 2600, 3900, 4199]
    _full_check(wl, d, [0, 1, 2, 3, 9], lambda b, n: _sample_rows(b, n, wl.W),
                lambda b: sorted({0, 3, 4, 31, (5 * b) % 32}))


def test_prefix_bound_far_above_the_prefixes():
    """max_prefix_len four times the longest prefix (a serving loop sizes
    its buffers for the whole run): the splits follow each sequence's own
    prefix, and the results are those of a tight bound."""
    wl = WL.Workload("slack", 76, B=6, W=64, Hq=8, Hkv=2, D=128, V=500,
                     prefix=300, prefix_hi=3000, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0, extra_positions=9000)
    mp = 4 * int(d["win_start"].max())
    PL.log(f"case slack: max_prefix {mp}")
    g, step, dev = PL.run_gpu_step(wl, d, max_prefix=mp)
    o = PL.oracle_step(wl, d, list(range(wl.B)))
    PL.check_reorder(wl, g, o)
    PL.check_attention(wl, g, o, list(range(wl.B)))
    PL.check_score(wl, d, g, o)
    PL.check_commit(wl, d, g, o)


@pytest.mark.parametrize("D,Hq,Hkv,W,prefix,lo", [
    (128, 32, 8, 32, 3000, 2000),   # 11 split slots: two slot groups
    (128, 16, 4, 32, 9000, 6000),   # 22 slots: four slot groups
    (128, 8, 2, 32, 9000, 300),     # 35 slots: four groups of up to nine
    (64, 2, 1, 16, 9000, 300),      # 35 slots: eight slot groups
])
def test_combine_slot_groups(D, Hq, Hkv, W, prefix, lo):
    """Prefixes split more than eight ways: the combine spreads a row's
    split slots over 2, 4 or 8 groups of lanes of one wave, each loading
    its slots at once, and joins their max and sums by lane exchanges.
    Sequences of one call use different numbers of splits."""
    wl = WL.Workload("slots", 77 + D + prefix, B=3, W=W, Hq=Hq, Hkv=Hkv, D=D,
                     V=400, prefix=prefix, prefix_hi=prefix, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    # the block tables and caches cover prefix + W positions; the shorter
    # prefixes use a part
    d["win_start"][1:] = [lo, (lo + prefix) // 2 + 5]
    _full_check(wl, d, [0, 1, 2], lambda b, n: _sample_rows(b, n, wl.W),
                lambda b: sorted({0, Hq - 1, (5 * b) % Hq}))


def test_prefix_beyond_one_split_of_pages():
    """A prefix longer than one split's staged page ids (2048 pages, 32,768
    positions) on a grid that already fills the CUs (16 sequences x 16 kv
    heads = 256 workgroups): the plan must still split it (two splits of
    516 tiles) and merge them.  Attention checked on sampled sequences,
    rows and heads."""
    wl = WL.Workload("split_pages", 71, B=16, W=16, Hq=16, Hkv=16, D=64,
                     V=500, prefix=33000, prefix_hi=33000, obs_frac=0.0,
                     obs_frac_hi=0.75, spike=9.0, spike_prob=0.5)
    d = WL.step_inputs(wl, seed=0)
    _full_check(wl, d, [0, 9, 15], lambda b, n: _sample_rows(b, n, wl.W),
                lambda b: sorted({0, 6, 15, (3 * b) % 16}))


def test_all_masks_and_all_filled():
    wl = WL.Workload("edge", 60, B=4, W=16, Hq=4, Hkv=2, D=64, V=300,
                     prefix=0, prefix_hi=50, obs_frac=0.0, spike=9.0)
    d = WL.step_inputs(wl, seed=0)
    d["win_tok"][1] = np.arange(16) + 5          # every slot filled
    d["win_tok"][2] = -1                          # every slot a mask
    d["win_tok"][3, :] = -1
    d["win_tok"][3, 5] = 77                       # one filled slot, not first
    n_obs = (d["win_tok"] != -1).sum(1)
    d["logits"] = WL.logits(wl, n_obs, 0, 0)
    _full_check(wl, d)


def test_qwen3_8b_layer_step():
    wl = WL.WORKLOADS["qwen3_8b_layer"]
    _full_check(wl, WL.step_inputs(wl, seed=0))


def _sample_rows(b, n_obs, W=32):
    rows = {0, max(n_obs - 1, 0), min(n_obs, W - 1), W - 1, (7 * b + 3) % W}
    return sorted(rows)


def test_ragged64_step_sampled():
    wl = WL.WORKLOADS["ragged64"]
    d = WL.step_inputs(wl, seed=0)
    seqs = [0, 1, 17, 40, 63]
    _full_check(wl, d, seqs, lambda b, n: _sample_rows(b, n, wl.W),
                lambda b: sorted({0, 3, 4, 31, (5 * b) % 32}))


def test_long_prefix_step_sampled():
    wl = WL.WORKLOADS["long_prefix"]
    d = WL.step_inputs(wl, seed=0)
    seqs = [0, 5, 7]
    _full_check(wl, d, seqs, lambda b, n: _sample_rows(b, n, wl.W),
                lambda b: sorted({0, 7, 8, 31}))


def test_capacity_error_leaves_state():
    """A block table without a page for a committed position: the commit is
    a no-op for that sequence and status says why; others proceed."""
    import torch
    wl = WL.Workload("cap", 61, B=2, W=8, Hq=2, Hkv=1, D=64, V=100,
                     prefix=16, obs_frac=0.5, spike=9.0)
    d = WL.step_inputs(wl, seed=0)
    d["win_tok"][:, :3] = [1, 2, 3]               # leading run of 3
    n_obs = (d["win_tok"] != -1).sum(1)
    d["logits"] = WL.logits(wl, n_obs, 0, 0)
    d["block_table"] = d["block_table"][:, :1].copy()   # only page 0
    g, step, dev = PL.run_gpu_step(wl, d)
    assert list(g["status"]) == [1, 1]            # WEDLM_SEQ_CAPACITY
    assert list(g["n_commit"]) == [0, 0]
    assert (g["win_tok"] == d["win_tok"]).all()
    assert (g["win_start"] == d["win_start"]).all()
    torch.cuda.synchronize()


@pytest.mark.parametrize("lam,temp", [(0.1, 0.1), (0.01, 1.0)])
def test_secondary_readings(lam, temp):
    """The paper's default lambda = 0.1, and the entropy at T = 1 (where the
    threshold almost never passes and the fallback fills one mask)."""
    for name in ("tiny", "qwen3_8b_layer"):
        wl = WL.WORKLOADS[name].replace(lam=lam, temp=temp)
        _full_check(wl, WL.step_inputs(wl, seed=3))


def test_attention_workspace_reuse():
    """One workspace, three calls with shrinking prefixes (so the number of
    prefix splits per sequence changes between calls): partials a longer
    call left in the workspace must not leak into a shorter one."""
    import torch
    from oracle import wedlm_oracle as O
    from paper_2512_22737_amd import wedlm
    wl = WL.Workload("reuse", 62, B=3, W=24, Hq=8, Hkv=2, D=128, V=300,
                     prefix=2000, prefix_hi=6000, obs_frac=0.3,
                     obs_frac_hi=0.6, spike=9.0)
    d = WL.step_inputs(wl, seed=0)
    dev = PL.to_dev(d)
    c_full = d["win_start"].copy()
    step = wedlm.DecodeStep(wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, wl.V,
                            int(c_full.max()))
    for frac in (1.0, 0.5, 0.1):
        c = (c_full * frac).astype(np.int32)
        c_dev = torch.from_numpy(c).cuda()
        step.reorder(dev["win_tok"], c_dev, dev["qkv_in"])
        step.attn(dev["k_cache"], dev["v_cache"], dev["block_table"], c_dev)
        got = step.out.float().cpu().numpy().astype(np.float64)
        assert (step.attn_status.cpu().numpy() == 0).all()
        for b in range(wl.B):
            perm, pos, _, _ = O.reorder(list(d["win_tok"][b]), int(c[b]))
            q, k, v = O.rope_window(d["qkv_in"][b], perm, pos, wl.Hq, wl.Hkv,
                                    wl.theta)
            kp, vp = WL.gather_prefix(d["k_cache"], d["v_cache"],
                                      d["block_table"], b, int(c[b]))
            ref, _ = O.window_attn(q, k, v, O.bf16_to_f64(kp),
                                   O.bf16_to_f64(vp))
            err = np.abs(got[b] - ref)
            rel = np.linalg.norm(got[b] - ref) / np.linalg.norm(ref)
            PL.log(f"  reuse frac {frac} seq {b} c={int(c[b])}: max abs "
                   f"{err.max():.2e} rel {rel:.2e}")
            assert err.max() <= PL.ATTN_MAX_ABS and rel <= PL.ATTN_REL_NORM


def test_attention_workspace_shared_by_shapes():
    """One workspace, filled with random bytes first, serves calls of two
    shapes in turn (their split plans place the partials and the (m, l)
    pairs at different offsets, so each call's slots sit on bytes the other
    shape wrote), three times over; every output is checked against the
    oracle.  The combine reads only the slots of the splits a sequence
    uses, which that call's main kernel has written; bytes left by another
    call or shape must never enter a result."""
    import torch
    from oracle import wedlm_oracle as O
    from paper_2512_22737_amd import wedlm
    shapes = [
        WL.Workload("share_a", 63, B=3, W=48, Hq=8, Hkv=2, D=128, V=300,
                    prefix=3000, prefix_hi=9000, obs_frac=0.3,
                    obs_frac_hi=0.6, spike=9.0),
        WL.Workload("share_b", 64, B=5, W=16, Hq=4, Hkv=2, D=128, V=300,
                    prefix=800, prefix_hi=2500, obs_frac=0.3,
                    obs_frac_hi=0.6, spike=9.0),
    ]
    runs = []
    need = 0
    for wl in shapes:
        d = WL.step_inputs(wl, seed=1)
        mp = int(d["win_start"].max())
        need = max(need, wedlm.wedlm_window_attn_workspace_size(
            wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, mp))
        step = wedlm.DecodeStep(wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, wl.V, mp)
        runs.append((wl, d, PL.to_dev(d), step, mp))
    assert need > 0
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    ws = torch.randint(0, 256, (need,), dtype=torch.uint8, device="cuda",
                       generator=g)
    refs = {}
    for rnd in range(3):
        for wl, d, dev, step, mp in runs:
            PL.log(f"case {wl.name} round {rnd}")
            step.reorder(dev["win_tok"], dev["win_start"], dev["qkv_in"])
            out = torch.full_like(step.out, float("nan"))
            status = torch.zeros_like(step.attn_status)
            wedlm.wedlm_window_attn(step.q_phys, step.k_phys, step.v_phys,
                                    dev["k_cache"], dev["v_cache"],
                                    dev["block_table"], dev["win_start"], mp,
                                    out, status=status, workspace=ws)
            torch.cuda.synchronize()
            assert (status.cpu().numpy() == 0).all()
            got = out.float().cpu().numpy().astype(np.float64)
            for b in range(wl.B):
                key = (wl.name, b)
                if key not in refs:
                    c = int(d["win_start"][b])
                    perm, pos, _, _ = O.reorder(list(d["win_tok"][b]), c)
                    q, k, v = O.rope_window(d["qkv_in"][b], perm, pos, wl.Hq,
                                            wl.Hkv, wl.theta)
                    kp, vp = WL.gather_prefix(d["k_cache"], d["v_cache"],
                                              d["block_table"], b, c)
                    refs[key], _ = O.window_attn(q, k, v, O.bf16_to_f64(kp),
                                                 O.bf16_to_f64(vp))
                ref = refs[key]
                err = np.abs(got[b] - ref)
                rel = np.linalg.norm(got[b] - ref) / np.linalg.norm(ref)
                assert err.max() <= PL.ATTN_MAX_ABS and rel <= PL.ATTN_REL_NORM, \
                    (wl.name, rnd, b, float(err.max()), float(rel))


def test_attention_status_bits():
    """Device-side checks of wedlm_window_attn: a prefix longer than
    max_prefix_len is reported (WEDLM_SEQ_BAD_LEN) and that sequence is
    skipped; a page id outside the cache is reported (WEDLM_SEQ_BAD_PAGE)
    and read as page 0 (in bounds).  The other sequences are unaffected."""
    import torch
    from oracle import wedlm_oracle as O
    from paper_2512_22737_amd import wedlm
    wl = WL.Workload("status", 63, B=3, W=16, Hq=8, Hkv=2, D=128, V=300,
                     prefix=300, prefix_hi=700, obs_frac=0.4, spike=9.0)
    d = WL.step_inputs(wl, seed=1)
    dev = PL.to_dev(d)
    c = d["win_start"].copy()
    max_prefix = int(c.max())
    step = wedlm.DecodeStep(wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, wl.V, max_prefix)
    bad_c = c.copy()
    bad_c[1] = max_prefix + 17                        # longer than the bound
    bt = d["block_table"].copy()
    bt[2, 3] = -1                                     # a hole inside c[2]
    assert c[2] > 4 * WL.PAGE
    c_dev = torch.from_numpy(bad_c).cuda()
    bt_dev = torch.from_numpy(bt).cuda()
    step.reorder(dev["win_tok"], c_dev, dev["qkv_in"])
    step.out.fill_(0)
    step.attn_status.zero_()
    step.attn(dev["k_cache"], dev["v_cache"], bt_dev, c_dev)
    st = step.attn_status.cpu().numpy()
    assert st[0] == 0
    assert st[1] & wedlm.SEQ_BAD_LEN
    assert st[2] & wedlm.SEQ_BAD_PAGE
    out = step.out.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(out[2]).all()                  # page 0 read instead
    b = 0
    perm, pos, _, _ = O.reorder(list(d["win_tok"][b]), int(c[b]))
    q, k, v = O.rope_window(d["qkv_in"][b], perm, pos, wl.Hq, wl.Hkv,
                            wl.theta)
    kp, vp = WL.gather_prefix(d["k_cache"], d["v_cache"], d["block_table"],
                              b, int(c[b]))
    ref, _ = O.window_attn(q, k, v, O.bf16_to_f64(kp), O.bf16_to_f64(vp))
    err = np.abs(out[b] - ref)
    assert err.max() <= PL.ATTN_MAX_ABS
    assert np.linalg.norm(out[b] - ref) / np.linalg.norm(ref) <= PL.ATTN_REL_NORM
