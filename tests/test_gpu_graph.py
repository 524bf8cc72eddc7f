"""The loss calls captured into a HIP graph (through torch.cuda.graph): the
resident schedule launches ordinary kernels (slot clear, the persistent loss
kernel, the loss reduction; no memset nodes), so a captured call replays.
Each replay follows eager work (the inputs are rewritten between replays)
and is checked bit for bit against an eager call on the same inputs."""
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


def _logits(recipe, shape, seed, dev):
    from paper_2609_24150_amd.inputs import make_logits
    zd, zt = make_logits(recipe, shape, BF16, seed=seed, device="cpu")
    return zd.to(dev), zt.to(dev)


def _same(got, ref, what):
    for k, v in ref.items():
        if v is None:
            continue
        a, b = got[k], v
        if a.dtype == BF16:
            a, b = a.view(torch.int16), b.view(torch.int16)
        assert torch.equal(a, b), (what, k)


def test_captured_calls_replay_bitwise(A):
    from paper_2609_24150_amd import api
    dev = torch.device("cuda:0")
    N, K, V = 40, 7, 128256
    inputs = [_logits("c2", (N, K, V), s, dev) for s in (21, 22)]
    seq = [(zd.view(K, N, V).contiguous(), zt.view(K, N, V).contiguous()) for zd, zt in inputs]
    from paper_2609_24150_amd import _lib

    def noalloc(d, t, ws):
        # the allocation-free entry point (its static scratch instead of ws)
        out = {"loss": torch.empty(1, device=dev), "E": torch.empty(N, device=dev),
               "accept": torch.empty(N, K, device=dev), "grad": torch.empty(N, K, V, dtype=BF16, device=dev)}
        st = _lib.lib().aal_wtv_fwd_bwd_noalloc(
            d.data_ptr(), t.data_ptr(), _lib.AAL_BF16, N, K, V, 0.8, 1.2, out["loss"].data_ptr(),
            out["E"].data_ptr(), out["accept"].data_ptr(), out["grad"].data_ptr(), _lib.AAL_BF16, None,
            torch.cuda.current_stream(dev).cuda_stream)
        _lib.check(st, "aal_wtv_fwd_bwd_noalloc")
        return out

    calls = {
        "wtv": lambda d, t, ws: A.aal_wtv_fwd_bwd(d, t, 1.0, 1.0, ws=ws),
        "eal": lambda d, t, ws: A.aal_eal_fwd_bwd(d, t, 0.9, ws=ws),
        "noalloc": noalloc,
    }
    ws = {k: api.workspace(N * K, N, dev) for k in calls}
    lws = torch.empty(A.aal_loss_workspace_bytes(A.AAL_LAYOUT_SEQUENCES, K, N, K), dtype=torch.uint8, device=dev)

    def sliding(d, t):
        return A.aal_loss_fwd_bwd(d, t, K, weights=(1.0, 0.0, 0.0, 0.0), layout=A.AAL_LAYOUT_SEQUENCES, ws=lws)

    # eager references for both input sets
    ref = [{k: f(zd, zt, ws[k]) for k, f in calls.items()} for zd, zt in inputs]
    sref = [sliding(d, t) for d, t in seq]
    torch.cuda.synchronize()
    # the graph's own input buffers
    xd, xt = inputs[0][0].clone(), inputs[0][1].clone()
    sd, st = seq[0][0].clone(), seq[0][1].clone()
    side = torch.cuda.Stream(dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):  # a warm-up call off the capture
        for k, f in calls.items():
            f(xd, xt, ws[k])
        sliding(sd, st)
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = {k: f(xd, xt, ws[k]) for k, f in calls.items()}
        sout = sliding(sd, st)
    for i in (1, 0, 1, 1):
        # eager work between the replays: the inputs are rewritten
        xd.copy_(inputs[i][0])
        xt.copy_(inputs[i][1])
        sd.copy_(seq[i][0])
        st.copy_(seq[i][1])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in calls:
            _same(out[k], ref[i][k], f"{k} replay with inputs {i}")
        _same(sout, sref[i], f"sliding replay with inputs {i}")
