"""GPU parity of wedlm_lm_head_score (output layer fused with the score of
each row) against the fp64 oracle.

* "exact" inputs (small integers times powers of two): every product and
  partial sum is exact in fp32 in any order, so the kernel's logits equal
  the oracle's exactly.  Greedy token bit-exact (ties included), entropy and
  top probability within the score's tolerance.  Shapes cover one and
  several 32-row blocks per vocabulary stream, streams shorter than a
  block, ragged row tails, one to four 32-row blocks of hidden rows per
  wave, and several row groups.
* "normal" inputs (N(0,1) hidden, N(0,1/Hd) weights, spiked rows) at the
  Qwen3-8B output-layer shape (Hd 4096, V 151936) on sampled rows: fp32
  accumulation over 4096 products.  Per row the logit error is bounded by
  Hd * 2^-24 * max_v sum_k |h_k w_vk| (recursive fp32 summation), the
  entropy error by 2 H max|dz| + 1e-12 with dz = dlogit / T; the greedy
  token must match wherever the top two logits differ by more than twice
  the logit bound.
"""
import math

import numpy as np
import pytest

from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL
from tests import parity_lib as PL

pytestmark = pytest.mark.gpu


def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _run(hb, wb, T):
    torch = _gpu()
    from paper_2512_22737_amd import wedlm
    dev = lambda a: (torch.from_numpy(np.ascontiguousarray(a)).cuda()
                     .view(torch.int16).view(torch.bfloat16))
    h, w = dev(hb), dev(wb)
    R = hb.shape[0]
    am = torch.full((R,), -7, dtype=torch.int32, device="cuda")
    H = torch.full((R,), float("nan"), dtype=torch.float32, device="cuda")
    pm = torch.full((R,), float("nan"), dtype=torch.float32, device="cuda")
    wedlm.wedlm_lm_head_score(h, w, T, am, H, pm)
    torch.cuda.synchronize()
    return am.cpu().numpy(), H.cpu().numpy().astype(np.float64), \
        pm.cpu().numpy().astype(np.float64)


EXACT = [
    # R, Hd, V
    (1, 256, 7),         # one pipeline group of k steps, fewer tokens than lanes
    (5, 256, 256),       # one 32-row block per stream at most
    (32, 256, 1000),     # one row block, ragged vocabulary ranges
    (40, 512, 513),      # two row blocks, ragged rows
    (96, 256, 2047),     # three row blocks
    (97, 256, 1000),     # one 128-row group in two row waves of two blocks
                         # (two vocabulary blocks per wave), 31 padded rows
    (128, 512, 3001),    # one full 128-row group
    (160, 512, 1500),    # one 256-row group in four row waves, ragged
    (200, 768, 1500),    # one 256-row group, ragged
    (300, 512, 2000),    # one 384-row group (four row waves, two vocabulary
                         # blocks per wave), ragged rows
    (384, 256, 1111),    # one full 384-row group, vocabulary ranges ending
                         # inside a 64-row block
    (448, 256, 1200),    # one 512-row group (LDS-destination loads), ragged
    (512, 512, 3001),    # one full 512-row group
    (513, 256, 999),     # two 512-row groups, the second of one row
    (800, 256, 777),     # two 512-row groups, the second ragged
    (17, 1024, 40000),   # several 32-row blocks per stream
    # k split over the waves (R <= 32, Hd 2048 / 4096)
    (7, 2048, 33),       # two blocks, the second with one row
    (1, 4096, 100),      # fewer blocks than workgroups
    (16, 2048, 20000),   # four k steps per wave, runs of two or three blocks
    (32, 4096, 9001),    # eight k steps per wave, ragged last block
]


@pytest.mark.parametrize("R,Hd,V", EXACT)
@pytest.mark.parametrize("T", [0.1, 1.0])
def test_lm_head_exact(R, Hd, V, T):
    PL.log(f"case lm_head exact R={R} Hd={Hd} V={V} T={T}")
    hb, wb = WL.lm_head_inputs(R, Hd, V, seed=R + V, kind="exact")
    tok, H, pm = O.lm_head_score(hb, wb, T)
    gt, gH, gp = _run(hb, wb, T)
    assert (gt == tok).all(), np.nonzero(gt != tok)
    err = np.abs(gH - H)
    assert (err <= PL.H_REL * np.abs(H) + PL.H_ABS).all(), err.max()
    assert (np.abs(gp - pm) <= PL.H_REL * pm).all()
    PL.log(f"  tokens exact, worst entropy rel err "
           f"{(err / np.maximum(np.abs(H), 1e-300)).max():.2e}")


@pytest.mark.parametrize("R", [16, 32, 384])
def test_lm_head_qwen3_shape_sampled(R):
    Hd, V, T = 4096, 151936, 0.1
    PL.log(f"case lm_head normal R={R} Hd={Hd} V={V} (sampled rows)")
    hb, wb = WL.lm_head_inputs(R, Hd, V, seed=11)
    gt, gH, gp = _run(hb, wb, T)
    rows = sorted({r for r in (0, 1, 15, 31, 63, 127, 128, 200, 255, 256, 383)
                   if r < R})
    tok, H, pm = O.lm_head_score(hb, wb, T, rows=rows)
    # logit error bound per row: Hd * 2^-24 * max_v sum_k |h_k w_vk|
    h = np.abs(O.bf16_to_f64(hb[rows]))
    bound = np.zeros(len(rows))
    for v0 in range(0, V, 8192):
        w = np.abs(O.bf16_to_f64(wb[v0:v0 + 8192]))
        bound = np.maximum(bound, (h @ w.T).max(axis=1))
    dl = Hd * 2.0 ** -24 * bound
    dz = dl / T
    worst_rel = 0.0
    for j, r in enumerate(rows):
        tol = 2 * H[j] * dz[j] + 1e-12
        assert abs(gH[r] - H[j]) <= tol, (r, gH[r], H[j], tol)
        worst_rel = max(worst_rel, abs(gH[r] - H[j]) / max(H[j], 1e-300))
        assert abs(gp[r] - pm[j]) <= pm[j] * (math.expm1(2 * dz[j]) + 1e-6)
        # the greedy token, wherever the top two logits are apart
        lg = O.bf16_to_f64(hb[r]) @ O.bf16_to_f64(wb[[gt[r], tok[j]]]).T
        if gt[r] != tok[j]:
            assert abs(lg[0] - lg[1]) <= 2 * dl[j], (r, gt[r], tok[j])
    PL.log(f"  {len(rows)} rows: worst entropy rel err {worst_rel:.2e} "
           f"(bound {2 * dz.max():.1e}), tokens equal "
           f"{int((gt[rows] == tok).sum())}/{len(rows)}")


def test_lm_head_argument_checks():
    torch = _gpu()
    from paper_2512_22737_amd import wedlm
    bf = dict(dtype=torch.bfloat16, device="cuda")
    am = torch.empty(2, dtype=torch.int32, device="cuda")
    H = torch.empty(2, dtype=torch.float32, device="cuda")
    for Hd in (96, 320):                       # Hd not a multiple of 256
        with pytest.raises(wedlm.WedlmError):
            wedlm.wedlm_lm_head_score(torch.zeros(2, Hd, **bf),
                                      torch.zeros(10, Hd, **bf), 0.1, am, H)
    with pytest.raises(wedlm.WedlmError):       # temperature
        wedlm.wedlm_lm_head_score(torch.zeros(2, 256, **bf),
                                  torch.zeros(10, 256, **bf), 0.0, am, H)
