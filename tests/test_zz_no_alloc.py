"""wedlm_window_attn_noalloc (include/wedlm.h) through the C ABI against
wedlm_window_attn with a caller-owned workspace, on the same seeded inputs:
two calls in a row, the second on a smaller batch with shorter prefixes
(fewer prefix splits, so the scratch array still holds the first call's
partials where the second call does not write).  Both calls must need a
workspace (several prefix splits), and the outputs and lse must be
bit-identical (the two entry points run the same kernels on the same plan).
The first pair is also checked against the fp64 oracle on one sequence."""
import ctypes

import numpy as np
import pytest

from paper_2512_22737_amd import workloads as WL
from tests import parity_lib as PL

pytestmark = pytest.mark.gpu


def _case(wl, d, lib):
    import torch
    from paper_2512_22737_amd import wedlm
    dev = PL.to_dev(d)
    c = d["win_start"]
    mp = int(c.max())
    step = wedlm.DecodeStep(wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, wl.V, mp)
    need = wedlm.wedlm_window_attn_workspace_size(wl.B, wl.W, wl.Hq, wl.Hkv,
                                                  wl.D, mp)
    assert need > 0, "the case must use split-K partials"
    step.reorder(dev["win_tok"], dev["win_start"], dev["qkv_in"])
    outs = []
    for noalloc in (False, True):
        out = torch.full_like(step.out, float("nan"))
        lse = torch.full_like(step.lse, float("nan"))
        status = torch.zeros_like(step.attn_status)
        P = dev["k_cache"].shape[0]
        common = [step.q_phys.data_ptr(), step.k_phys.data_ptr(),
                  step.v_phys.data_ptr(), dev["k_cache"].data_ptr(),
                  dev["v_cache"].data_ptr(), P, dev["block_table"].data_ptr(),
                  dev["block_table"].shape[1], dev["win_start"].data_ptr(),
                  wl.B, wl.W, wl.Hq, wl.Hkv, wl.D, mp,
                  ctypes.c_float(1.0 / np.sqrt(wl.D)), out.data_ptr(),
                  lse.data_ptr(), status.data_ptr()]
        stream = torch.cuda.current_stream().cuda_stream
        if noalloc:
            code = lib.wedlm_window_attn_noalloc(*common, stream)
        else:
            ws = torch.empty(need, dtype=torch.uint8, device="cuda")
            code = lib.wedlm_window_attn(*common, ws.data_ptr(), need, stream)
        assert code == 0, code
        torch.cuda.synchronize()
        assert (status.cpu().numpy() == 0).all()
        outs.append((PL.bf16_bits(out), lse.cpu().numpy()))
    (oa, la), (ob, lb) = outs
    assert np.array_equal(oa, ob)
    assert np.array_equal(la.view(np.uint32), lb.view(np.uint32))
    return step, oa


def test_noalloc_matches_workspace_entry_point_twice():
    import torch
    from oracle import wedlm_oracle as O
    from paper_2512_22737_amd import wedlm
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = wedlm.lib()
    big = WL.Workload("noalloc_a", 80, B=3, W=64, Hq=8, Hkv=2, D=128, V=300,
                      prefix=2500, prefix_hi=4000, obs_frac=0.0,
                      obs_frac_hi=0.75, spike=9.0)
    small = WL.Workload("noalloc_b", 81, B=2, W=32, Hq=8, Hkv=2, D=128, V=300,
                        prefix=700, prefix_hi=1500, obs_frac=0.0,
                        obs_frac_hi=0.75, spike=9.0)
    PL.log("case noalloc: B=3 W=64 prefixes 2500-4000, then B=2 W=32 "
           "prefixes 700-1500")
    d = WL.step_inputs(big, seed=0)
    step, out = _case(big, d, lib)
    # the first call against the oracle on sequence 0
    b = 0
    perm, pos, _, _ = O.reorder(list(d["win_tok"][b]), int(d["win_start"][b]))
    q, k, v = O.rope_window(d["qkv_in"][b], perm, pos, big.Hq, big.Hkv,
                            big.theta)
    kp, vp = WL.gather_prefix(d["k_cache"], d["v_cache"], d["block_table"], b,
                              int(d["win_start"][b]))
    ref, _ = O.window_attn(q, k, v, O.bf16_to_f64(kp), O.bf16_to_f64(vp))
    got = O.bf16_to_f64(out[b])
    assert np.abs(got - ref).max() <= PL.ATTN_MAX_ABS
    assert (np.linalg.norm(got - ref) / np.linalg.norm(ref)
            <= PL.ATTN_REL_NORM)
    _case(small, WL.step_inputs(small, seed=1), lib)


def test_noalloc_rejects_a_plan_beyond_the_scratch():
    """A prefix so long that the split-K partials exceed the fixed array:
    refused on the host, before anything is enqueued."""
    from paper_2512_22737_amd import wedlm
    lib = wedlm.lib()
    f = ctypes.c_void_p(0x1000)      # never dereferenced: the call fails first
    need = wedlm.wedlm_window_attn_workspace_size(8, 64, 32, 8, 128, 10 ** 7)
    assert need > (64 << 20)
    code = lib.wedlm_window_attn_noalloc(
        f, f, f, f, f, 1 << 20, f, 700000, f, 8, 64, 32, 8, 128, 10 ** 7,
        ctypes.c_float(0.088), f, None, None, None)
    assert code == -6        # WEDLM_E_SCRATCH
