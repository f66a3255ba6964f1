"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments before touching a GPU."""

import ctypes
import os
import re

import pytest

from paper_2608_09307_amd import linsimp as L

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")


def _declared(header):
    text = open(os.path.join(INCLUDE, header)).read()
    decl = r"^(?:int|size_t|const char\*)\s+(linsimp_[a-z_]+)\s*\("
    return sorted(set(re.findall(decl, text, flags=re.MULTILINE)))


def test_library_exports_every_declared_symbol():
    lib = L.lib()
    assert sorted(os.listdir(INCLUDE)) == ["linsimp.h", "linsimp_bank.h", "linsimp_head.h"]
    for header, exports in (("linsimp.h", L.EXPORTS), ("linsimp_head.h", L.HEAD_EXPORTS),
                            ("linsimp_bank.h", L.BANK_EXPORTS)):
        names = _declared(header)
        assert set(names) == set(exports), header
        for name in names:
            assert hasattr(lib, name), name
    assert lib.linsimp_version() == 103


def test_head_sizes_and_argument_errors():
    lib = L.lib()
    d = L.make_dims(2, 16, 16384, 128, 128, 128, 64, L.BF16)
    saved = lib.linsimp_head_saved_size(ctypes.byref(d))
    # q', k', r' and o~ in bf16, 2 + 1 floats per row
    rows = 2 * 16 * 16384
    assert saved == rows * (3 * 128 + 128) * 2 + rows * 12
    assert lib.linsimp_head_workspace_size(ctypes.byref(d), 1) > L.workspace_size(d, True)
    bad = L.make_dims(1, 1, 64, 48, 48, 32, 8, L.BF16)
    assert lib.linsimp_head_saved_size(ctypes.byref(bad)) == 0
    vp = ctypes.c_void_p
    good = [4096 * (i + 1) for i in range(10)]
    dd = L.make_dims(1, 1, 64, 32, 32, 32, 8, L.F32)
    o = L.head_opts(7)
    rc = lib.linsimp_head_fwd(ctypes.byref(dd), ctypes.byref(o), *[vp(p) for p in good],
                              1 << 20, vp(1 << 20), 1 << 20, vp(0))
    assert rc == -1 and b"gate" in lib.linsimp_last_error()
    o = L.head_opts(L.GATE_HEAD)
    rc = lib.linsimp_head_fwd(ctypes.byref(dd), ctypes.byref(o), *[vp(p) for p in good],
                              16, vp(1 << 20), 1 << 20, vp(0))
    assert rc == -3 and b"saved" in lib.linsimp_last_error()


def test_workspace_size_and_unsupported_shapes():
    d = L.make_dims(2, 16, 16384, 128, 128, 128, 64, L.BF16)
    fw, bw = L.workspace_size(d, False), L.workspace_size(d, True)
    assert 0 < fw < bw
    # windows up to 128 under the launch rule w * min(m, 128) <= 8192
    for ok in (L.make_dims(1, 1, 256, 128, 128, 64, 128, L.BF16), L.make_dims(1, 1, 256, 64, 64, 64, 96, L.F32),
               L.make_dims(1, 1, 256, 32, 32, 64, 128, L.F32), L.make_dims(1, 1, 256, 64, 64, 128, 64, L.BF16)):
        assert L.workspace_size(ok, True) > 0
    for bad in (L.make_dims(1, 1, 256, 48, 48, 32, 64, L.BF16),     # D not supported
                L.make_dims(1, 1, 256, 32, 32, 32, 129, L.BF16),    # w > 128
                L.make_dims(1, 1, 256, 128, 128, 128, 65, L.BF16),  # w * m > 8192
                L.make_dims(1, 1, 256, 64, 64, 64, 97, L.F32),      # f32 D = m = 64 stops at w = 96
                L.make_dims(1, 1, 256, 128, 128, 128, 64, L.F32),   # f32 only up to 64
                L.make_dims(1, 1, 0, 32, 32, 32, 64, L.BF16),       # n = 0
                L.make_dims(1, 1, 8, 32, 32, 32, 64, 7),            # bad dtype
                L.make_dims(256, 256, 64, 32, 32, 32, 64, L.BF16),  # B*H above the grid's y limit
                L.make_dims(1, 3, 1 << 30, 32, 32, 32, 64, L.BF16)):  # B*H*n above 2^31
        assert L.workspace_size(bad, False) == 0
        assert L.lib().linsimp_last_error()


def _call_fwd(d, ptrs, ws, nbytes):
    lib = L.lib()
    vp = ctypes.c_void_p
    return lib.linsimp_fwd(ctypes.byref(d), *[vp(p) for p in ptrs], vp(ws), nbytes, vp(0))


def test_argument_errors_are_reported_not_raised():
    d = L.make_dims(1, 1, 64, 32, 32, 32, 8, L.F32)
    good = [4096 * (i + 1) for i in range(8)]
    need = L.workspace_size(d, False)
    # NULL q
    assert _call_fwd(d, [0] + good[1:], 1 << 20, need) == -1
    assert b"NULL" in L.lib().linsimp_last_error()
    # misaligned k
    assert _call_fwd(d, [good[0], good[1] + 4] + good[2:], 1 << 20, need) == -1
    # workspace too small / misaligned
    assert _call_fwd(d, good, 1 << 20, need - 1) == -3
    assert _call_fwd(d, good, (1 << 20) + 16, need) == -3
    # unsupported shape
    d2 = L.make_dims(1, 1, 64, 96, 96, 32, 8, L.F32)
    assert _call_fwd(d2, good, 1 << 20, 1 << 30) == -2
    # decode: bad window
    lib = L.lib()
    vp = ctypes.c_void_p
    rc = lib.linsimp_decode_step(4, 2, 32, 32, 32, 0, L.BF16, 1e-30,
                                 *[vp(4096 * (i + 1)) for i in range(13)], vp(0))
    assert rc == -1


def test_reuse_flag_without_a_matching_forward_is_refused():
    """LINSIMP_BWD_REUSE_STATES is accepted only for a workspace a forward with
    the same dims, k, v and omega left its states in (a host-side record); a
    workspace no forward has used is refused before anything is launched."""
    lib = L.lib()
    vp = ctypes.c_void_p
    d = L.make_dims(1, 1, 64, 32, 32, 32, 8, L.F32)
    need = L.workspace_size(d, True)
    ptrs = [vp(4096 * (i + 1)) for i in range(14)]
    rc = lib.linsimp_bwd_ex(ctypes.byref(d), *ptrs, L.BWD_REUSE_STATES, vp(1 << 24), need, vp(0))
    assert rc == -1 and b"no forward" in lib.linsimp_last_error()
    # the head entry point checks the same record
    o = L.head_opts(L.GATE_HEAD)
    hw = lib.linsimp_head_workspace_size(ctypes.byref(d), 1)
    hp = [vp(4096 * (i + 1)) for i in range(17)]
    hp[10] = vp(1 << 22)                         # saved: 256-byte aligned
    rc = lib.linsimp_head_bwd_ex(ctypes.byref(d), ctypes.byref(o), *hp, L.BWD_REUSE_STATES,
                                 vp(1 << 24), hw, vp(0))
    assert rc == -1 and b"no forward" in lib.linsimp_last_error()


def test_decode_grid_bound_is_an_error():
    """One workgroup per (sequence, head): S*H above 2^24 - 1 is refused
    (LINSIMP_E_UNSUPPORTED) before any launch."""
    lib = L.lib()
    vp = ctypes.c_void_p
    ptrs = [vp(4096 * (i + 1)) for i in range(13)]
    rc = lib.linsimp_decode_step(1 << 20, 16, 32, 32, 32, 8, L.BF16, 1e-30, *ptrs, vp(0))
    assert rc == -2 and b"at most" in lib.linsimp_last_error()
    rc = lib.linsimp_decode_chunk(1 << 20, 16, 2, 32, 32, 32, 8, L.BF16, 1e-30, *ptrs, vp(0))
    assert rc == -2


def test_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 1, 8, 32)
    om = torch.zeros(1, 32, 32)
    with pytest.raises((ValueError, RuntimeError)):
        L.fwd(x, x, x, x, x, om, 4, workspace=torch.zeros(1 << 16, dtype=torch.uint8))


def test_feature_bank_argument_errors():
    lib = L.lib()
    vp = ctypes.c_void_p
    ok = [vp(4096 * (i + 1)) for i in range(3)]
    assert lib.linsimp_feature_bank(1, 64, 48, *ok, 1, vp(0)) == -2
    assert lib.linsimp_feature_bank(1, 0, 64, *ok, 1, vp(0)) == -1
    assert lib.linsimp_feature_bank(1, 64, 64, *ok, 2, vp(0)) == -1
    assert lib.linsimp_feature_bank(1, 64, 64, vp(0), ok[1], ok[2], 1, vp(0)) == -1
    assert lib.linsimp_feature_bank(70000, 64, 64, *ok, 1, vp(0)) == -2


def test_binding_checks_shapes_and_dtypes_before_the_call():
    """The C ABI takes bare pointers; the binding refuses tensors whose shape
    or dtype disagrees with the others before any pointer is passed."""
    import torch
    B, H, n, D = 1, 2, 8, 32
    x = {nm: torch.zeros(B, H, n, D) for nm in ("q", "k", "v", "r", "u")}
    om = torch.zeros(H, 32, D)
    bad_k = torch.zeros(B, H, n - 1, D)
    with pytest.raises(ValueError, match="k has shape"):
        L.fwd(x["q"], bad_k, x["v"], x["r"], x["u"], om, 8)
    with pytest.raises(TypeError, match="omega has dtype"):
        L.fwd(x["q"], x["k"], x["v"], x["r"], x["u"], om.double(), 8)
    with pytest.raises(ValueError, match="dout has shape"):
        L.bwd(*(x[nm] for nm in ("q", "k", "v", "r", "u")), om, 8, x["v"], torch.zeros(B, H, n, 2),
              torch.zeros(B, H, n, D + 1))
    st = {"M": torch.zeros(B, H, 32, D), "a": torch.zeros(B, H, 32), "rho": torch.zeros(B, H),
          "ring_r": torch.zeros(B, H, 8, D), "ring_u": torch.zeros(B, H, 7, D),
          "pos": torch.zeros(B, dtype=torch.int64)}
    tok = {nm: torch.zeros(B, H, D) for nm in ("q", "k", "v", "r", "u")}
    with pytest.raises(ValueError, match="ring_u has shape"):
        L.decode_step(st, *(tok[nm] for nm in ("q", "k", "v", "r", "u")), om, 8)
    with pytest.raises(ValueError, match="gate has shape"):
        L.head_fwd(*(x[nm] for nm in ("q", "k", "v", "r", "u")), om, 8, torch.zeros(H),
                   torch.zeros(H + 1))


def test_plain_c_client_links_and_runs(tmp_path):
    """The headers and the library are usable from C with no Python or torch:
    a C client is compiled with gcc against include/, linked with
    liblinsimp.so and run (calls that need no GPU)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    libdir = os.path.dirname(L.lib_path())
    exe = str(tmp_path / "abi_smoke")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(root, "include"),
                    os.path.join(root, "tests", "c", "abi_smoke.c"), "-L", libdir, "-llinsimp",
                    "-Wl,-rpath," + libdir, "-o", exe], check=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "0 failure(s)" in res.stdout
