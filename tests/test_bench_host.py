"""Host logic of bench.py (CPU): the committed counter profile is used only
while the kernel sources hash to the profiled version, and the ALU roofline
follows from the counters by its stated arithmetic."""
import os

import bench


def test_profile_fields_follow_the_kernel_sources(tmp_path, monkeypatch):
    f = bench.profile_fields("c2")
    assert f, "the committed profile matches the committed kernel sources"
    for k in ("traffic_bytes_per_launch", "valu_instructions_per_launch", "valu_active_quad_cycles_per_launch"):
        assert float(f[k]) > 0, k
    assert bench.profile_fields("c4") == {}  # the profile covers the c2 workload only
    # a kernel source that differs from the profiled one: no fields
    src = tmp_path / "k.hip"
    src.write_text(open(os.path.join(bench.ROOT, bench.KERNEL_SOURCES[0])).read() + "\n// changed\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(src)] + bench.KERNEL_SOURCES[1:])
    assert bench.profile_fields("c2") == {}


def test_alu_roofline_arithmetic():
    # 1e9 wave instructions at 4.5 cycles each: 4.5e9 SIMD cycles over 1024 SIMDs at 2.4 GHz
    f = {"valu_instructions_per_launch": "1e9", "valu_active_quad_cycles_per_launch": str(4.5e9 / 4)}
    r = bench.alu_roofline(f, ms=2.5, alg_bytes=11e9)
    floor_s = 4.5e9 / 1024 / 2.4e9
    assert abs(r["floor_ms"] - floor_s * 1e3) < 1e-9
    assert abs(r["cycles_per_instruction"] - 4.5) < 1e-12
    assert abs(r["frac"] - floor_s / 2.5e-3) < 1e-12  # issue rate over the peak rate of this mix
    assert abs(r["hbm_frac_at_alu_floor"] - 11e9 / floor_s / 8e12) < 1e-12
    assert bench.alu_roofline({}, 2.5, 11e9) is None
