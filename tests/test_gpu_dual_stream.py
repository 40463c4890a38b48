"""GPU parity of wedlm_dual_stream_attn (include/wedlm_train.h) against the
oracle's dense block mask (Sec. 4.2), within the attention bar of the
decode step (max-abs 2e-2 and 1e-2 relative to the output scale; lse within
1e-3): one and two sequences, blocks of 8, 16, 32 (paired windows) and 64
(one window per block), the decode step's head shapes, the Qwen3-8B heads,
8 query heads per kv head (two query blocks per paired window), and 32
pairs of one kv head whose prefixes split three ways (the combine kernel in
the paired layout)."""
import math

import numpy as np
import pytest
import torch

from oracle import wedlm_oracle as O
from paper_2512_22737_amd import workloads as WL

pytestmark = pytest.mark.gpu


def _bf16(rng, shape):
    return WL.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def _dev(a):
    return (torch.from_numpy(np.ascontiguousarray(a)).view(torch.int16)
            .cuda().view(torch.bfloat16))


# blocks of up to 32 run paired (memory block k and prediction block k in one
# window of 2B rows, each half masked from the other's block); 64 one block
# per window
@pytest.mark.parametrize("n_seq,L,B,Hq,Hkv,D", [
    (1, 64, 16, 4, 2, 64), (2, 128, 32, 8, 2, 128), (1, 256, 32, 32, 8, 128),
    (1, 96, 32, 4, 4, 64), (2, 64, 8, 8, 2, 64), (1, 192, 64, 8, 2, 128),
    (1, 128, 32, 16, 2, 64), (1, 1024, 32, 4, 1, 64)])
def test_dual_stream_attention(n_seq, L, B, Hq, Hkv, D):
    from paper_2512_22737_amd import wedlm
    rng = np.random.default_rng(L + B + Hq)
    q = _bf16(rng, (n_seq, 2 * L, Hq, D))
    k = _bf16(rng, (n_seq, 2 * L, Hkv, D))
    v = _bf16(rng, (n_seq, 2 * L, Hkv, D))
    out = torch.full((n_seq, 2 * L, Hq, D), float("nan"), dtype=torch.bfloat16,
                     device="cuda")
    lse = torch.full((n_seq, 2 * L, Hq), float("nan"), device="cuda")
    wedlm.wedlm_dual_stream_attn(_dev(q), _dev(k), _dev(v), B, out, lse)
    torch.cuda.synchronize()
    got = out.float().cpu().double().numpy()
    gl = lse.cpu().double().numpy()
    for s in range(n_seq):
        masked = {p for p in range(L) if rng.random() < 0.5}
        vis = O.dual_stream_visible(L, B, masked)
        ref, rl = O.masked_attention(O.bf16_to_f64(q[s]), O.bf16_to_f64(k[s]),
                                     O.bf16_to_f64(v[s]), vis)
        err = np.abs(got[s] - ref)
        assert err.max() < 2e-2, err.max()
        assert err.max() < 1e-2 * max(1.0, np.abs(ref).max())
        assert np.abs(gl[s] - rl).max() < 1e-3


def test_dual_stream_rejects_bad_shapes():
    from paper_2512_22737_amd import wedlm
    lib = wedlm.lib()
    ws = lib.wedlm_dual_stream_attn_workspace_size
    assert ws(1, 100, 32, 4, 2, 64) == 0          # L not a multiple of B
    assert ws(1, 128, 96, 4, 2, 64) == 0          # block > 64
    assert ws(1, 128, 32, 4, 2, 96) == 0          # D
    assert ws(1, 128, 32, 4, 2, 64) > 0
