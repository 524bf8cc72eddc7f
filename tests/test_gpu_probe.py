"""The streaming probe behind the bench's practical ceilings (a measurement
aid, not part of the method): its sums and its flag, through the C ABI."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def A():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_24150_amd as A
    return A


# 16-byte vectors: one, a ragged count past the grid's tiles, several tiles
@pytest.mark.parametrize("nvec", [1, 1000, 4 * 256 * 2048 + 37])
@pytest.mark.parametrize("n_src", [1, 2, 3])
def test_probe_sums(A, nvec, n_src):
    g = torch.Generator().manual_seed(nvec + n_src)
    srcs = [torch.randint(-2**31, 2**31 - 1, (nvec * 4,), generator=g, dtype=torch.int64) for _ in range(n_src)]
    want = sum(srcs) & 0xFFFFFFFF
    want = torch.where(want >= 2**31, want - 2**32, want).to(torch.int32)
    dev = [s.to(torch.int32).cuda() for s in srcs]
    dst = torch.full_like(dev[0], 7)
    A.aal_stream_probe(dev, dst)
    torch.cuda.synchronize()
    assert torch.equal(dst.cpu(), want)


def test_probe_flag(A):
    a = torch.ones(4096, dtype=torch.int32, device="cuda")
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    A.aal_stream_probe([a, a], flag=flag)
    torch.cuda.synchronize()
    assert flag.item() == 0
    b = torch.zeros_like(a)
    b[100:104] = -1  # one 16-byte vector of all-ones words
    A.aal_stream_probe([b], flag=flag)
    torch.cuda.synchronize()
    assert flag.item() == 1
