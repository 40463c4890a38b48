"""The seeded input generator: determinism, layouts and the stated recipe."""
import numpy as np
import pytest

from paper_2512_22737_amd import workloads as WL


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    x[:4] = [1.0, -0.0, 3.0e38, 1e-40]
    ours = WL.f32_to_bf16_bits(x)
    ref = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy()
    assert (ours == ref.view(np.uint16)).all()


def test_tiny_inputs_deterministic_and_shaped():
    wl = WL.WORKLOADS["tiny"]
    a = WL.step_inputs(wl, seed=0)
    b = WL.step_inputs(wl, seed=0)
    for k in ["win_tok", "win_start", "qkv_in", "block_table", "k_cache",
              "v_cache"]:
        assert (a[k] == b[k]).all(), k
    assert np.array_equal(a["logits"], b["logits"], equal_nan=True)
    assert a["win_tok"].shape == (1, 16)
    assert (a["win_tok"] != -1).sum() == 8              # 8 observed slots
    assert a["qkv_in"].shape == (1, 16, 4 + 4, 64)
    assert a["logits"].shape == (1, 16, 1024)
    assert np.isnan(a["logits"][0, :8]).all()           # observed rows
    assert np.isfinite(a["logits"][0, 8:]).all()
    # contiguous prefix: identity block table
    assert list(a["block_table"][0]) == list(range(a["block_table"].shape[1]))
    c = WL.step_inputs(wl, seed=1)
    assert not (c["qkv_in"] == a["qkv_in"]).all()


def test_pages_round_trip():
    wl = WL.WORKLOADS["ragged64"].replace(B=3, prefix=20, prefix_hi=70,
                                          V=64)
    d = WL.step_inputs(wl, seed=0)
    c = d["win_start"]
    for b in range(3):
        k, v = WL.gather_prefix(d["k_cache"], d["v_cache"], d["block_table"],
                                b, int(c[b]))
        k0, v0 = WL.prefix_kv(wl, b, int(c[b]), 0)
        assert (k == k0).all() and (v == v0).all()
    # every page id used exactly once, unused table entries are -1
    bt = d["block_table"]
    used = bt[bt >= 0]
    assert sorted(used.tolist()) == list(range(d["num_pages"]))
    # slots past the prefix hold NaN
    b = 0
    pos = int(c[b])
    pg = bt[b, pos // 16]
    assert d["k_cache"][pg, 0, pos % 16, 0] == WL.BF16_NAN


def test_spike_recipe():
    wl = WL.WORKLOADS["qwen3_8b_layer"].replace(V=4096)
    d = WL.step_inputs(wl, seed=0, with_cache=False)
    lg = d["logits"][0, 16:]
    top = np.sort(lg, axis=1)[:, -1]
    assert ((top > 7.0).mean() > 0.3)                    # spiked rows exist
    assert lg.std() < 1.2


def test_stream_pool_logits_device_and_host_agree():
    torch = pytest.importorskip("torch")
    wl = WL.WORKLOADS["stream512"].replace(B=2, W=4, V=300, logit_pool=5)
    pool = WL.logit_pool(wl, 0)
    host = WL.logits(wl, None, 0, 3, pool=pool)
    dev = WL.logits_torch(wl, torch.tensor(pool), 0, 3).numpy()
    assert np.array_equal(host, dev)
