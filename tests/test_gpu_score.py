"""GPU parity of wedlm_score on its own (Sec. 5.2, the H of Eq. (11))
against the fp64 oracle's score_row, for the ways the work is split.

With fewer than 768 window rows the kernel counts the masked rows of the
call on the device and splits each into vocabulary chunks so that about
768 workgroups stream; the cases below vary that count (none, one, a few,
most), the number of sequences (the masked-row list is found by a scan in
groups of 64 sequences: 1, 4 and 300 sequences), the vocabulary (one chunk
or many; a length that is not a multiple of 4), the row stride (16-byte
aligned or not) and n_obs outside [0, W] (clamped).  With 768 rows or more
every row is its own workgroup.  Greedy tokens must match exactly (the
logits are drawn without ties at the top), entropy and top probability
within the 1e-5 relative bar; observed rows' outputs stay untouched.
"""
import numpy as np
import pytest

from oracle import wedlm_oracle as O
from tests import parity_lib as PL

pytestmark = pytest.mark.gpu


def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _logits(rng, B, W, V, stride):
    x = np.full((B, W, stride), np.float32(-1e30), dtype=np.float32)
    body = rng.standard_normal((B, W, V)).astype(np.float32) * 3.0
    # a few peaked rows (entropy far below 1) among the ordinary ones
    peak = rng.random((B, W)) < 0.2
    top = rng.integers(0, V, size=(B, W))
    bb, ww = np.nonzero(peak)
    body[bb, ww, top[bb, ww]] += 40.0
    x[:, :, :V] = body
    return x


@pytest.mark.parametrize("B,W,V,stride,obs", [
    (4, 64, 151936, 151936, [64, 0, 63, 10]),     # 119 masked rows
    (1, 32, 151936, 151936, [31]),                # one masked row
    (2, 8, 40000, 40000, [8, 8]),                 # none masked
    (300, 1, 40001, 40004, None),                 # 300 sequences, W = 1
    (16, 32, 20001, 20003, None),                 # 512 rows: one workgroup each, unaligned rows
    (73, 7, 20001, 20001, None),                  # 511 rows: chunked, two chunks at most
    (3, 16, 5000, 5000, [-4, 20, 7]),             # one chunk per row; n_obs clamped
    (800, 1, 3000, 3000, None),                   # 800 rows: one workgroup each
])
def test_score_chunking(B, W, V, stride, obs):
    torch = _gpu()
    from paper_2512_22737_amd import wedlm
    PL.log(f"case score B={B} W={W} V={V} stride={stride}")
    rng = np.random.default_rng(B * 1000 + W + V)
    x = _logits(rng, B, W, V, stride)
    if obs is None:
        obs = rng.integers(-1, W + 2, size=B)
    n_obs = np.asarray(obs, dtype=np.int32)
    T = 0.1
    dev = torch.device("cuda")
    lg = torch.from_numpy(x).to(dev)
    am = torch.full((B, W), -7, dtype=torch.int32, device=dev)
    H = torch.full((B, W), -1.0, dtype=torch.float32, device=dev)
    pm = torch.full((B, W), -1.0, dtype=torch.float32, device=dev)
    need = wedlm.wedlm_score_workspace_size(B, W, V)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    wedlm.wedlm_score(lg, torch.from_numpy(n_obs).to(dev), T, am, H, pm,
                      workspace=ws, V=V)
    torch.cuda.synchronize()
    am, H, pm = am.cpu().numpy(), H.cpu().numpy(), pm.cpu().numpy()
    masked = 0
    for b in range(B):
        no = int(min(max(int(n_obs[b]), 0), W))
        for i in range(W):
            if i < no:
                assert am[b, i] == -7 and H[b, i] == -1.0 and pm[b, i] == -1.0
                continue
            masked += 1
            tok, Hr, pr = O.score_row(x[b, i, :V], T)
            assert int(am[b, i]) == tok, (b, i)
            assert abs(float(H[b, i]) - Hr) <= PL.H_REL * abs(Hr) + PL.H_ABS, \
                (b, i, float(H[b, i]), Hr)
            assert abs(float(pm[b, i]) - pr) <= PL.H_REL * pr, (b, i)
    PL.log(f"  {masked} masked rows checked")
