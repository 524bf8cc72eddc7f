"""The resident kernels' time-out path, forced from the host: with the
environment variable AAL_TEST_PRESET_TIMEOUT=1 the kernels start with their
error word set, as a poll time-out leaves it, so every bounded wait ends at
once, the kernel drains and the loss must read NaN.  The next call without
the variable must give the results of a call before it, bit for bit (the path
leaves nothing behind), and the streaming schedule, which has no such wait,
is unaffected."""
import math

import pytest
import torch

pytestmark = pytest.mark.gpu

BF16 = torch.bfloat16


@pytest.fixture(scope="module")
def A():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_24150_amd as lib
    return lib


def test_forced_timeout_gives_nan_then_recovers(A, monkeypatch):
    from paper_2609_24150_amd.inputs import make_logits
    dev = torch.device("cuda:0")
    N, K, V = 20, 7, 128256
    zd, zt = make_logits("c2", (N, K, V), BF16, seed=17, device="cpu")
    zd, zt = zd.to(dev), zt.to(dev)
    sd, st = zd.view(K, N, V), zt.view(K, N, V)
    calls = {
        "wtv": lambda: A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0),
        "eal": lambda: A.aal_eal_fwd_bwd(zd, zt, 1.0),
        "kl+0.1eal": lambda: A.aal_loss_fwd_bwd(zd, zt, K, weights=(0.0, 0.1, 1.0, 0.0)),
        "sliding": lambda: A.aal_loss_fwd_bwd(sd, st, K, weights=(1.0, 0.0, 0.0, 0.0),
                                              layout=A.AAL_LAYOUT_SEQUENCES),
    }
    ref = {k: f() for k, f in calls.items()}
    torch.cuda.synchronize()
    for k, r in ref.items():
        assert math.isfinite(r["loss"].item()), k
    monkeypatch.setenv("AAL_TEST_PRESET_TIMEOUT", "1")
    for k, f in calls.items():
        r = f()
        torch.cuda.synchronize()
        assert math.isnan(r["loss"].item()), k
    s = A.aal_wtv_fwd_bwd(zd, zt, 1.0, 1.0, flags=A.AAL_FLAG_STREAMING)
    torch.cuda.synchronize()
    assert math.isfinite(s["loss"].item())
    monkeypatch.delenv("AAL_TEST_PRESET_TIMEOUT")
    for k, f in calls.items():
        r = f()
        torch.cuda.synchronize()
        for name, v in ref[k].items():
            if v is not None:
                assert torch.equal(r[name].view(torch.uint8), v.view(torch.uint8)), (k, name)
