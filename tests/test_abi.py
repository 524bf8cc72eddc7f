"""CPU checks of the C ABI: the library loads, exports every function that
include/aal.h declares, and rejects invalid arguments before touching a GPU.
No call here reaches a kernel launch."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aal.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(aal_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2609_24150_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libaal.so is not built (run __graft_entry__.build())")
    return _lib


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("aal_eal_fwd_bwd", "aal_wtv_fwd_bwd", "aal_sim_accept_grpo", "aal_workspace_bytes",
              "aal_loss_fwd_bwd", "aal_loss_workspace_bytes", "aal_grpo_fwd_bwd", "aal_grpo_workspace_bytes",
              "aal_status_string", "aal_last_error", "aal_version", "aal_vp_row_partials", "aal_vp_merge_rows",
              "aal_vp_accept_partials", "aal_vp_window_scan", "aal_vp_sequence_scan", "aal_vp_grad",
              "aal_eal_fwd_bwd_ex", "aal_wtv_fwd_bwd_ex", "aal_sim_accept_grpo_ex"):
        assert n in names


# The six calls of the boundary with their exact C types: each line assigns the
# declared function to a pointer of the stated type, and the C compiler
# rejects any mismatch (-Werror).  The `_ex` calls add the schedule flags (and
# the simulation's per-position accept output) beside these, unchanged.
BOUNDARY_SIGNATURES = '''
size_t (*f_ws)(int64_t, int64_t) = aal_workspace_bytes;
const char* (*f_ss)(aal_status_t) = aal_status_string;
const char* (*f_le)(void) = aal_last_error;
aal_status_t (*f_eal)(const void*, const void*, aal_dtype_t, int64_t, int32_t, int32_t, float,
                      float*, float*, float*, int32_t*, void*, aal_dtype_t, const float*,
                      void*, size_t, hipStream_t) = aal_eal_fwd_bwd;
aal_status_t (*f_wtv)(const void*, const void*, aal_dtype_t, int64_t, int32_t, int32_t, float, float,
                      float*, float*, float*, void*, aal_dtype_t, const float*,
                      void*, size_t, hipStream_t) = aal_wtv_fwd_bwd;
aal_status_t (*f_sim)(const void*, const void*, aal_dtype_t, int32_t, int32_t, int32_t, int32_t, float,
                      const float*, const float*, int32_t*, int32_t*, float*, float, int32_t, float,
                      void*, size_t, hipStream_t) = aal_sim_accept_grpo;
_Static_assert(AAL_BF16 == 0 && AAL_F32 == 1, "dtype codes");
_Static_assert(AAL_FLAG_STREAMING == 1u && AAL_FLAG_COOPERATIVE == 2u, "flag bits");
_Static_assert(AAL_OK == 0 && AAL_ERR_ARG == 1 && AAL_ERR_DTYPE == 2 && AAL_ERR_ALIGN == 3 &&
               AAL_ERR_WORKSPACE == 4 && AAL_ERR_HIP == 5, "status codes");
'''


def test_boundary_signatures_are_exact(tmp_path):
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "boundary.c"
    src.write_text('#include "aal.h"\n' + BOUNDARY_SIGNATURES)
    r = subprocess.run([cc, "-std=c11", "-Werror", "-Wall", "-fsyntax-only", f"-I{os.path.join(ROOT, 'include')}",
                        str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    # the header still compiles after HIP's own declaration of hipStream_t (C++)
    cxx = shutil.which("g++")
    if cxx:
        src2 = tmp_path / "twice.cc"
        src2.write_text('typedef struct ihipStream_t* hipStream_t;\n#include "aal.h"\nint main() { return 0; }\n')
        r = subprocess.run([cxx, "-std=c++17", "-Werror", "-fsyntax-only", f"-I{os.path.join(ROOT, 'include')}",
                            str(src2)], capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_library_exports_every_declared_symbol(lib):
    h = C.CDLL(lib.LIB_PATH)
    for n in declared_functions():
        assert hasattr(h, n), f"{n} not exported"
    assert set(lib._SIGNATURES) == set(declared_functions())


def test_status_strings_and_version(lib):
    L = lib.lib()
    assert L.aal_version() >= 100
    for s in range(6):
        assert L.aal_status_string(s).decode().startswith("AAL_")
    assert L.aal_status_string(99) == b"unknown status"


def test_workspace_bytes(lib):
    L = lib.lib()
    a = L.aal_workspace_bytes(14336, 2048)
    b = L.aal_workspace_bytes(28672, 2048)
    assert b > a > 0 and a % 256 == 0
    assert L.aal_workspace_bytes(-1, 3) == 0


def _eal(L, **kw):
    args = dict(zd=16, zt=16, dt=0, N=2, K=3, V=8, T=1.0, loss=16, grad=None, gdt=0, ws=256, wsb=1 << 30)
    args.update(kw)
    return L.aal_eal_fwd_bwd(args["zd"], args["zt"], args["dt"], args["N"], args["K"], args["V"], args["T"],
                             args["loss"], None, None, None, args["grad"], args["gdt"], None, args["ws"],
                             args["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(zd=None), 1), (dict(loss=None), 1), (dict(N=0), 1), (dict(K=0), 1), (dict(K=65), 1),
    (dict(V=0), 1), (dict(T=0.0), 1), (dict(T=-1.0), 1), (dict(T=float("nan")), 1), (dict(T=float("inf")), 1),
    (dict(T=1e-45), 1), (dict(dt=7), 2), (dict(grad=16, gdt=9), 2), (dict(zd=18), 3), (dict(grad=24), 3),
    (dict(ws=None), 4), (dict(ws=128), 3), (dict(wsb=100), 4), (dict(N=1 << 30, K=4), 1),
])
def test_eal_validation(lib, kw, code):
    L = lib.lib()
    assert _eal(L, **kw) == code
    assert L.aal_last_error().decode() != ""


def test_wtv_and_sim_validation(lib):
    L = lib.lib()
    st = L.aal_wtv_fwd_bwd(16, 16, 0, 2, 3, 8, 1.0, 0.0, 16, None, None, None, 0, None, 256, 1 << 30, None)
    assert st == 1 and b"temp_target" in L.aal_last_error()
    st = L.aal_wtv_fwd_bwd_ex(16, 16, 0, 2, 3, 8, 1.0, 1.0, 16, None, None, None, 0, None, 4, 256, 1 << 30, None)
    assert st == 1 and b"flags" in L.aal_last_error()
    st = L.aal_eal_fwd_bwd_ex(16, 16, 0, 2, 3, 8, 1.0, 16, None, None, None, None, 0, None, 4, 256, 1 << 30, None)
    assert st == 1 and b"flags" in L.aal_last_error()
    st = L.aal_eal_fwd_bwd_ex(16, 16, 0, 0, 3, 8, 1.0, 16, None, None, None, None, 0, None, 1, 256, 1 << 30, None)
    assert st == 1 and b"N must" in L.aal_last_error()

    def sim(**kw):
        a = dict(P=2, G=4, K=3, V=10, T=1.0, u1=16, rew=16, eps=1e-6, ddof=0, ws=256, wsb=1 << 30)
        a.update(kw)
        return L.aal_sim_accept_grpo(16, 16, 0, a["P"], a["G"], a["K"], a["V"], a["T"], a["u1"], 16, None,
                                     a["rew"], 16, a["eps"], a["ddof"], 0.0, a["ws"], a["wsb"], None)
    assert sim(u1=None) == 1
    assert sim(rew=None) == 1
    assert sim(G=1, ddof=1) == 1
    assert sim(V=(1 << 21) + 1) == 1
    assert sim(T=float("nan")) == 1
    assert sim(eps=-1.0) == 1
    assert sim(wsb=8) == 4
    assert sim(ws=8) == 3
    st = L.aal_sim_accept_grpo_ex(16, 16, 0, 2, 4, 3, 10, 1.0, None, 16, None, None, 16, 16, 1e-6, 0, 0.0, 256,
                                  1 << 30, None)
    assert st == 1 and b"u1" in L.aal_last_error()


def test_loss_workspace_bytes(lib):
    L = lib.lib()
    a = L.aal_loss_workspace_bytes(0, 2048, 0, 7)
    b = L.aal_loss_workspace_bytes(1, 4, 2048, 7)
    assert a > 0 and b > 0 and a % 256 == 0 and b % 256 == 0
    assert L.aal_loss_workspace_bytes(1, 2, 0, 7) == 0
    assert L.aal_loss_workspace_bytes(5, 2, 8, 7) == 0
    assert L.aal_loss_workspace_bytes(0, 0, 0, 7) == 0


def _loss(L, lib, **kw):
    a = dict(zd=16, zt=16, lab=None, dt=0, lay=1, B=2, S=9, K=3, V=8, Td=1.0, Tt=1.0, w=(1.0, 0.0, 0.0, 0.0),
             loss=16, grad=None, gdt=0, flags=0, ws=256, wsb=1 << 30)
    a.update(kw)
    return L.aal_loss_fwd_bwd(a["zd"], a["zt"], a["lab"], a["dt"], a["lay"], a["B"], a["S"], a["K"], a["V"],
                              a["Td"], a["Tt"], lib.LossWeights(*a["w"]), a["loss"], None, None, None, None, None,
                              None, a["grad"], a["gdt"], None, a["flags"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(lay=3), 1), (dict(B=0), 1), (dict(K=0), 1), (dict(K=65), 1), (dict(V=0), 1), (dict(S=0), 1),
    (dict(Td=0.0), 1), (dict(Tt=float("nan")), 1), (dict(w=(float("inf"), 0, 0, 0)), 1),
    (dict(zd=None), 1), (dict(zt=None), 1), (dict(zt=None, w=(0, 1.0, 0, 0)), 1), (dict(loss=None), 1),
    (dict(dt=5), 2), (dict(grad=16, gdt=7), 2), (dict(zd=20), 3), (dict(grad=40), 3),
    (dict(ws=None), 4), (dict(ws=64), 3), (dict(wsb=1000), 4), (dict(B=1 << 30, S=4), 1), (dict(flags=4), 1),
])
def test_loss_validation(lib, kw, code):
    L = lib.lib()
    assert _loss(L, lib, **kw) == code
    assert L.aal_last_error().decode() != ""


def test_grpo_workspace_bytes(lib):
    L = lib.lib()
    assert L.aal_grpo_workspace_bytes(0, 64, 0, 0, 8, 7) > 0
    assert L.aal_grpo_workspace_bytes(1, 4, 2048, 4, 8, 7) > 0
    assert L.aal_grpo_workspace_bytes(1, 4, 2048, 0, 8, 7) == 0
    assert L.aal_grpo_workspace_bytes(0, 0, 0, 0, 8, 7) == 0


def _grpo(L, lib, **kw):
    a = dict(zth=16, zrf=16, zt=16, lab=None, dt=0, lay=1, B=2, S=20, G=2, m=4, K=3, V=8, anc=16, T=1.0,
             prm=(1e-6, 0.0, 0.2, 0.0, float("inf")), loss=16, grad=None, gdt=0, ws=256, wsb=1 << 30)
    a.update(kw)
    return L.aal_grpo_fwd_bwd(a["zth"], a["zrf"], a["zt"], a["lab"], a["dt"], a["lay"], a["B"], a["S"], a["G"],
                              a["m"], a["K"], a["V"], a["anc"], a["T"], lib.GrpoParams(*a["prm"]), a["loss"],
                              None, None, None, None, a["grad"], a["gdt"], None, a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(lay=4), 1), (dict(B=0), 1), (dict(K=0), 1), (dict(K=65), 1), (dict(m=0), 1), (dict(m=65), 1),
    (dict(V=0), 1), (dict(G=0), 1), (dict(S=5), 1), (dict(anc=None), 1), (dict(zth=None), 1),
    (dict(zt=None), 1), (dict(loss=None), 1), (dict(T=0.0), 1),
    (dict(prm=(-1.0, 0.0, 0.2, 0.0, 1.0)), 1), (dict(prm=(0.0, float("nan"), 0.2, 0.0, 1.0)), 1),
    (dict(prm=(0.0, 0.0, -0.1, 0.0, 1.0)), 1), (dict(prm=(0.0, 0.0, 0.2, 2.0, 1.0)), 1),
    (dict(prm=(0.0, 0.0, 0.2, 0.0, float("nan"))), 1), (dict(dt=3), 2), (dict(grad=16, gdt=3), 2),
    (dict(zrf=24), 3), (dict(grad=8), 3), (dict(ws=None), 4), (dict(ws=32), 3), (dict(wsb=64), 4),
])
def test_grpo_validation(lib, kw, code):
    L = lib.lib()
    assert _grpo(L, lib, **kw) == code
    assert L.aal_last_error().decode() != ""


def test_vp_validation(lib):
    """Every case fails validation, so no kernel is launched."""
    L = lib.lib()
    P = L.aal_vp_row_partials

    def part(zd=16, zt=16, lab=None, dt=0, rows=2, vs=8, v0=0, vtot=None, mode=0, td=1.0, tt=1.0, parts=16):
        vtot = v0 + vs if vtot is None else vtot
        return P(zd, zt, lab, dt, rows, vs, v0, vtot, mode, td, tt, parts, None)

    for kw, code in [(dict(rows=0), 1), (dict(vs=0), 1), (dict(v0=-1), 1), (dict(v0=(1 << 31) - 4), 1),
                     (dict(dt=5), 2), (dict(zd=18), 3), (dict(zt=None), 1), (dict(mode=9), 1),
                     (dict(mode=1, tt=0.0), 1), (dict(td=float("nan")), 1), (dict(parts=None), 1),
                     (dict(parts=18), 3), (dict(rows=1 << 60), 1), (dict(lab=16, mode=1), 1),
                     (dict(lab=18), 3), (dict(lab=16, zd=None), 1), (dict(v0=8, vtot=15), 1),
                     (dict(vtot=0), 1)]:
        assert part(**kw) == code, kw
        assert L.aal_last_error().decode() != ""
    M = L.aal_vp_merge_rows
    assert M(16, 0, 4, 0, 1.0, 1.0, 16, None) == 1
    assert M(16, 2, 0, 0, 1.0, 1.0, 16, None) == 1
    assert M(None, 2, 4, 0, 1.0, 1.0, 16, None) == 1
    assert M(16, 2, 4, 1, 1.0, -1.0, 16, None) == 1
    assert M(16, 2, 4, 3, 1.0, 1.0, 16, None) == 1
    Acc = L.aal_vp_accept_partials
    assert Acc(16, 16, 0, 2, 8, 1.0, 1.0, None, 16, None) == 1
    assert Acc(16, None, 0, 2, 8, 1.0, 1.0, 16, 16, None) == 1
    S = L.aal_vp_window_scan
    assert S(16, None, 1, 2, 3, 1, 1.0, None, 16, 16, None, None, None) == 1   # WTV needs acc_all
    assert S(16, 16, 1, 2, 65, 0, 1.0, None, 16, 16, None, None, None) == 1
    assert S(16, 16, 1, 0, 3, 0, 1.0, None, 16, 16, None, None, None) == 1
    assert S(16, 16, 1, 2, 3, 0, 1.0, None, None, 16, None, None, None) == 1
    assert S(16, 16, 1, 2, 3, 0, 1.0, None, 16, None, None, None, None) == 1
    assert S(16, 16, 1, 2, 3, 0, 0.0, None, 16, 16, None, None, None) == 1
    Q = L.aal_vp_sequence_scan
    assert Q(16, 16, 1, 2, 5, 7, 0, 1.0, None, 16, 16, None, None, None) == 1   # S < K
    assert Q(16, 16, 1, 0, 8, 7, 0, 1.0, None, 16, 16, None, None, None) == 1   # B = 0
    assert Q(16, None, 1, 2, 8, 7, 1, 1.0, None, 16, 16, None, None, None) == 1  # WTV needs acc_all
    assert Q(16, 16, 1, 2, 8, 65, 0, 1.0, None, 16, 16, None, None, None) == 1
    assert Q(16, 16, 1, 2, 8, 7, 0, 1.0, None, 16, None, None, None, None) == 1
    assert Q(16, 16, 1, 2, 8, 7, 5, 1.0, None, 16, 16, None, None, None) == 1
    G = L.aal_vp_grad
    assert G(16, 16, 0, 2, 8, 0, 1, 1.0, 1.0, 16, None, 0, None) == 1
    assert G(16, 16, 0, 2, 8, 0, 1, 1.0, 1.0, 16, 16, 9, None) == 2
    assert G(16, 16, 0, 2, 8, 0, 1, 1.0, 1.0, 16, 24, 0, None) == 3
    assert G(16, None, 0, 2, 8, 0, 1, 1.0, 1.0, 16, 16, 0, None) == 1   # WTV reads the target


def test_vp_record_layouts_match_the_binding(tmp_path, lib):
    """The record sizes the Python binding allocates equal the C struct sizes."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "layout.c"
    src.write_text(
        '#include "aal.h"\n'
        f"_Static_assert(sizeof(aal_vp_part_t) == {lib.VP_PART_BYTES}, \"part\");\n"
        f"_Static_assert(sizeof(aal_vp_acc_t) == {lib.VP_ACC_BYTES}, \"acc\");\n"
        f"_Static_assert(sizeof(aal_vp_row_t) == {lib.VP_ROW_BYTES}, \"row\");\n"
        f"_Static_assert(AAL_VP_EAL == {lib.AAL_VP_EAL} && AAL_VP_WTV == {lib.AAL_VP_WTV}, \"modes\");\n")
    r = subprocess.run([cc, "-std=c11", "-fsyntax-only", f"-I{os.path.join(ROOT, 'include')}", str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_binding_flag_values_match_the_header(lib):
    # the header's values are checked by the C compiler in the signature test
    assert lib.AAL_FLAG_STREAMING == 1 and lib.AAL_FLAG_COOPERATIVE == 2
