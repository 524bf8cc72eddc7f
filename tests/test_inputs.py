"""The seeded input recipes (host logic, CPU): the statistics each workload's
recipe states, reproducibility, and the uniforms' range."""
import math

import pytest
import torch

from paper_2609_24150_amd.inputs import CONFIGS, RECIPES, make_logits, make_uniforms


def _fit(zd, zt):
    """Least-squares slope and residual std of z_d on z_t, pooled over rows."""
    x, y = zt.double().flatten(), zd.double().flatten()
    slope = float(((x - x.mean()) * (y - y.mean())).sum() / ((x - x.mean()) ** 2).sum())
    resid = y - slope * x
    return slope, float(resid.std())


@pytest.mark.parametrize("recipe", ["c1", "c4"])
def test_plain_recipes(recipe):
    r = RECIPES[recipe]
    zd, zt = make_logits(recipe, (16, 4, 2048), torch.float32, seed=5, device="cpu")
    assert zd.shape == zt.shape == (16, 4, 2048) and zd.dtype == torch.float32
    assert abs(float(zt.double().std()) - r["sigma_t"]) < 0.02 * r["sigma_t"]
    slope, sd = _fit(zd, zt)
    assert abs(slope - r["alpha"]) < 0.01 and abs(sd - r["sigma_d"]) < 0.02 * r["sigma_d"]


def test_peaked_recipe_c2():
    r = RECIPES["c2"]
    V = 4096
    zd, zt = make_logits("c2", (32, V), torch.float32, seed=6, device="cpu")
    # the peaks add peaks * bump / V to a row's mean; entries above bump - 1:
    # peaks * P(N(bump, s^2) > bump - 1) + (V - peaks) * P(N(0, s^2) > bump - 1)
    assert abs(float(zt.double().mean()) - r["peaks"] * r["bump"] / V) < 0.03
    thr, sg = r["bump"] - 1.0, r["sigma_t"]
    tail = lambda x: 0.5 * math.erfc(x / (sg * math.sqrt(2.0)))  # noqa: E731
    want = r["peaks"] * tail(thr - r["bump"]) + (V - r["peaks"]) * tail(thr)
    far = (zt > thr).sum(dim=1).double()
    assert abs(float(far.mean()) - want) < 0.1 * want
    slope, _ = _fit(zd, zt)
    assert abs(slope - r["alpha"]) < 0.02


def test_shifted_rows_c3():
    """On 10% of the rows the draft's bumps leave the target's peaks."""
    r = RECIPES["c3"]
    rows, V = 200, 4096
    zd, zt = make_logits("c3", (rows, V), torch.float32, seed=7, device="cpu")
    pk = zt.topk(r["peaks"], dim=1).indices
    # draft mass at the target's peaks relative to the row: high on ordinary
    # rows (alpha * bump above the rest), absent on the shifted ones
    at_peaks = zd.gather(1, pk).mean(dim=1) - zd.mean(dim=1)
    shifted = at_peaks < 0.5 * r["alpha"] * r["bump"]
    assert abs(int(shifted.sum()) - round(r["shift_frac"] * rows)) <= 2  # a statistical split
    # the shifted rows' bumps sit on as many other tokens
    top_d = zd[shifted].topk(r["peaks"], dim=1).values.mean() - zd[shifted].mean()
    assert float(top_d) > 0.5 * r["alpha"] * r["bump"]


def test_bf16_is_rounded_fp32_and_reproducible():
    a = make_logits("c2", (3, 7, 1000), torch.bfloat16, seed=11, device="cpu")
    b = make_logits("c2", (3, 7, 1000), torch.bfloat16, seed=11, device="cpu")
    f = make_logits("c2", (3, 7, 1000), torch.float32, seed=11, device="cpu")
    c = make_logits("c2", (3, 7, 1000), torch.bfloat16, seed=12, device="cpu")
    for x, y, z in zip(a, b, f):
        assert torch.equal(x, y)
        assert torch.equal(x, z.to(torch.bfloat16))
    assert not torch.equal(a[0], c[0])


def test_uniforms():
    u1, u2 = make_uniforms((4, 8, 7), seed=3, device="cpu")
    for u in (u1, u2):
        assert u.shape == (4, 8, 7) and u.dtype == torch.float32
        assert float(u.min()) >= 0.0 and float(u.max()) < 1.0
    assert not torch.equal(u1, u2)
    v1, _ = make_uniforms((4, 8, 7), seed=3, device="cpu")
    assert torch.equal(u1, v1)


def test_configs_name_the_workload_sizes():
    assert (CONFIGS["c2"]["N"], CONFIGS["c2"]["K"], CONFIGS["c2"]["V"]) == (2048, 7, 128256)
    assert (CONFIGS["c3"]["N"], CONFIGS["c3"]["K"], CONFIGS["c3"]["V"]) == (4096, 5, 151936)
    assert (CONFIGS["c4"]["N"], CONFIGS["c4"]["K"], CONFIGS["c4"]["V"]) == (16384, 16, 32000)
    assert (CONFIGS["c5"]["P"], CONFIGS["c5"]["G"], CONFIGS["c5"]["K"]) == (256, 8, 7)
    assert CONFIGS["c1"]["dtype"] == torch.float32 and CONFIGS["c4"]["dtype"] == torch.float32
