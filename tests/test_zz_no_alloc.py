"""The entry point that allocates nothing, ptf_calibrate_noalloc, against
ptf_calibrate with a caller-owned workspace (the same kernels): scale, zero
point and every alpha bit for bit, on two calls in a row, the second smaller
than the first (the fixed scratch keeps the first call's contents), through
the C ABI."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


def test_noalloc_calibration_matches_workspace_call():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2111_13824_amd as fq
    for T, C, outliers, seed in ((12608, 768, 8, 2), (333, 150, 2, 5)):
        print("CASE noalloc calibrate", T, C, flush=True)
        x = torch.from_numpy(W.ln_inputs(T, C, seed=seed, outliers=outliers)["x_float"]
                             .astype(np.float32)).to("cuda:0")
        s1, zp1, a1 = fq.ptf_calibrate(x, 8, 3)
        s2 = torch.full((1,), float("nan"), dtype=torch.float64, device="cuda:0")
        zp2 = torch.full((1,), 77, dtype=torch.int32, device="cuda:0")
        a2 = torch.full((C,), 0xEE, dtype=torch.uint8, device="cuda:0")
        fq.ptf_calibrate_noalloc(x, 8, 3, s=s2, zp=zp2, alpha=a2)
        torch.cuda.synchronize()
        assert s2.cpu().numpy()[0] == s1.cpu().numpy()[0]
        assert zp2.cpu().numpy()[0] == zp1.cpu().numpy()[0]
        assert np.array_equal(a2.cpu().numpy(), a1.cpu().numpy())
    with pytest.raises(fq.FqError) as ei:
        big = torch.zeros((200000, 768), dtype=torch.float32, device="cuda:0")
        fq.ptf_calibrate_noalloc(big, 8, 3)
    assert ei.value.status == fq.binding.FQ_ERR_SCRATCH
