"""Two resident WTV calls issued at once on two streams of one device with
AAL_FLAG_COOPERATIVE: each grid fills the device, and the runtime's
cooperative launch places each whole grid before it starts, so both calls
finish with the results of a lone call (a finite loss, the same bits)."""
import math

import pytest
import torch

pytestmark = pytest.mark.gpu


def test_cooperative_calls_on_two_streams():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_24150_amd as A
    from paper_2609_24150_amd.inputs import make_logits
    dev = torch.device("cuda:0")
    zd, zt = make_logits("c2", (64, 7, 128256), torch.bfloat16, seed=41, device="cpu")
    zd, zt = zd.to(dev), zt.to(dev)
    ref = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    s1.wait_stream(torch.cuda.current_stream(dev))
    s2.wait_stream(torch.cuda.current_stream(dev))
    outs = []
    for _ in range(3):
        with torch.cuda.stream(s1):
            outs.append(A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0, flags=A.AAL_FLAG_COOPERATIVE, stream=s1))
        with torch.cuda.stream(s2):
            outs.append(A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0, flags=A.AAL_FLAG_COOPERATIVE, stream=s2))
    torch.cuda.synchronize()
    for r in outs:
        assert math.isfinite(r["loss"].item())
        for k in ("loss", "E", "accept", "grad"):
            assert torch.equal(r[k].view(torch.uint8), ref[k].view(torch.uint8)), k
