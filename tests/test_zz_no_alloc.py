"""The allocation-free WTV entry point (static device scratch) against the
ordinary one with a caller workspace: same kernels, so the outputs must agree
to the tolerances of tests/parity.py (and here they agree bit for bit), over
two calls in a row whose second input is smaller, through the C ABI."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

BF16, F32 = torch.bfloat16, torch.float32


def _codes(lib, t):
    return lib.AAL_BF16 if t == BF16 else lib.AAL_F32


def _run(lib, zd, zt, Td, Tt, noalloc):
    """One call through the C ABI with preallocated outputs."""
    N, K, V = zd.shape
    dev = zd.device
    out = {"loss": torch.full((1,), float("nan"), device=dev), "E": torch.full((N,), -1.0, device=dev),
           "accept": torch.full((N, K), -1.0, device=dev), "grad": torch.full((N, K, V), 7.0, dtype=zd.dtype, device=dev)}
    s = torch.cuda.current_stream(dev).cuda_stream
    L = lib.lib()
    head = (zd.data_ptr(), zt.data_ptr(), _codes(lib, zd.dtype), N, K, V, Td, Tt, out["loss"].data_ptr(),
            out["E"].data_ptr(), out["accept"].data_ptr(), out["grad"].data_ptr(), _codes(lib, zd.dtype), None)
    if noalloc:
        st = L.aal_wtv_fwd_bwd_noalloc(*head, s)
    else:
        ws = torch.empty(L.aal_workspace_bytes(N * K, N), dtype=torch.uint8, device=dev)
        st = L.aal_wtv_fwd_bwd(*head, ws.data_ptr(), ws.numel(), s)
    lib.check(st, "noalloc" if noalloc else "aal_wtv_fwd_bwd")
    torch.cuda.synchronize()
    return out


def _same(a, b):
    for k in ("loss", "E", "accept"):
        assert torch.equal(a[k], b[k]), k
    assert torch.equal(a["grad"].view(torch.uint8), b["grad"].view(torch.uint8)), "grad"


def test_noalloc_matches_workspace_call_twice_then_smaller():
    import paper_2609_24150_amd._lib as lib
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_24150_amd.inputs import make_logits
    dev = torch.device("cuda:0")
    # first call: c2's rows at 40 windows (the resident kernel, bf16)
    zd, zt = make_logits("c2", (40, 7, 128256), BF16, seed=3, device="cpu")
    zd, zt = zd.to(dev), zt.to(dev)
    ref = _run(lib, zd, zt, 1.0, 1.0, False)
    got = _run(lib, zd, zt, 1.0, 1.0, True)
    _same(got, ref)
    assert np.isfinite(got["loss"].item())
    # second call, smaller and of another shape: fp32, V not a multiple of the
    # 16-byte vector, so the streaming schedule (per-row records in the scratch)
    zd2, zt2 = make_logits("c1", (5, 3, 4099), F32, seed=4, device="cpu")
    zd2, zt2 = zd2.to(dev), zt2.to(dev)
    ref2 = _run(lib, zd2, zt2, 0.7, 0.9, False)
    got2 = _run(lib, zd2, zt2, 0.7, 0.9, True)
    _same(got2, ref2)
    # third: the first shape again after the array held the smaller call's data
    got3 = _run(lib, zd, zt, 1.0, 1.0, True)
    _same(got3, ref)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    import paper_2609_24150_amd._lib as lib
    L = lib.lib()
    # 1,000,000 rows need 32 MB of row records plus the fixed region: too large
    st = L.aal_wtv_fwd_bwd_noalloc(16, 16, 0, 1000000, 1, 8, 1.0, 1.0, 16, None, None, None, 0, None, None)
    assert st == lib.AAL_ERR_WORKSPACE
    assert b"static scratch" in L.aal_last_error()
    st = L.aal_wtv_fwd_bwd_noalloc(16, 16, 0, 0, 1, 8, 1.0, 1.0, 16, None, None, None, 0, None, None)
    assert st == lib.AAL_ERR_ARG
