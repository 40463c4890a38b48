"""bench.py's roofline arithmetic, on the CPU: the algorithmic bytes of an
attention launch and of a whole step, written out from their definitions
(every cached K/V position once, the window's Q/K/V once, O and lse once,
each masked row's logits once, the appended rows read and written), and the
gate that only reports counter traffic taken on the current kernel source."""
import hashlib
import os

import numpy as np
import pytest

import bench
from paper_2512_22737_amd import workloads as WL


def test_attention_bytes_long_prefix():
    wl = WL.WORKLOADS["long_prefix"]
    c = np.full(wl.B, 32768)
    kv = 8 * 32768 * 8 * 128 * 2 * 2          # B * c * Hkv * D * (K,V) * bf16
    q_kv = 8 * 64 * (32 + 16) * 128 * 2       # window Q, K, V
    out = 8 * 64 * 32 * (128 * 2 + 4)         # O bf16 + lse fp32
    assert bench.attn_bytes(wl, c) == kv + q_kv + out == 1084293120


def test_step_bytes_adds_reorder_logits_and_append():
    wl = WL.WORKLOADS["long_prefix"]
    c = np.full(wl.B, 32768)
    n_masked, n_commit_rows = 384, 7
    qkv = 8 * 64 * 48 * 128 * 2
    want = (2 * qkv + bench.attn_bytes(wl, c) + 4 * wl.V * n_masked +
            2 * 2 * 2 * wl.Hkv * wl.D * n_commit_rows)
    assert bench.step_bytes(wl, c, n_masked, n_commit_rows) == want


def test_traffic_is_reported_only_for_the_current_source(tmp_path, monkeypatch):
    src = tmp_path / "window_attn.hip"
    src.write_bytes(b"kernel v1")
    sha = hashlib.sha256(b"kernel v1").hexdigest()
    prof = tmp_path / "window_attn_{wl}_traffic.txt"
    (tmp_path / "window_attn_w_traffic.txt").write_text(
        "# header: ignored\nsource_sha256: %s\ntraffic_bytes_per_launch: 123\n"
        % sha)
    monkeypatch.setattr(bench, "ATTN_SRC", str(src))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(prof))
    assert bench.read_traffic("w") == 123.0
    src.write_bytes(b"kernel v2")              # the kernel changed since
    assert bench.read_traffic("w") is None
    assert bench.read_traffic("other") is None


def test_committed_traffic_file_matches_the_kernel():
    """The committed long_prefix traffic summary was taken on the current
    attention source (else bench.py reports traffic null)."""
    assert bench.read_traffic("long_prefix") is not None


def test_gpus_above_one_exit_with_a_message(monkeypatch, capsys):
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        bench.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err
