"""Host-only checks of the C ABI: the library loads, exports every declared
entry point, and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2606_29563_amd import kvec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvec.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:kvec_status|const char\*|int32_t)\s+(kvec_\w+)\s*\(", src, re.M)))


def test_header_declares_expected_calls():
    assert _declared() == sorted(kvec.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = kvec.load()
    for name in _declared():
        assert hasattr(lib, name), name


def test_library_is_gfx950():
    data = open(kvec.LIB_PATH, "rb").read()
    assert b"gfx950" in data


def _cfg(**kw):
    base = dict(batch=1, n_layers=32, n_kv_heads=8, n_q_heads=32, head_dim=128, seq_len=32768,
                window=32, window_ext=64, budget=1024, pool_kernel=7, n_adjust_heads=3, lam=1.0,
                beta=0.25, dtype=kvec.KVEC_BF16)
    base.update(kw)
    return kvec.Config(**base)


def _ws_status(cfg):
    out = ctypes.c_size_t(0)
    c = cfg.c()
    return kvec.load().kvec_workspace_size(ctypes.byref(c), ctypes.byref(out)), out.value


def test_workspace_size_positive_and_monotone():
    s1, b1 = _ws_status(_cfg(seq_len=4096, budget=128))
    s2, b2 = _ws_status(_cfg())
    assert s1 == kvec.KVEC_OK and s2 == kvec.KVEC_OK
    assert 0 < b1 < b2
    assert kvec.kvec_workspace_size(_cfg()) == b2


@pytest.mark.parametrize("over,code", [
    (dict(batch=0), kvec.KVEC_ERR_INVALID),
    (dict(n_layers=0), kvec.KVEC_ERR_INVALID),
    (dict(n_layers=256), kvec.KVEC_ERR_INVALID),
    (dict(n_q_heads=30), kvec.KVEC_ERR_INVALID),
    (dict(window=0), kvec.KVEC_ERR_INVALID),
    (dict(window=40000), kvec.KVEC_ERR_INVALID),
    (dict(window_ext=16), kvec.KVEC_ERR_INVALID),
    (dict(budget=16), kvec.KVEC_ERR_INVALID),
    (dict(pool_kernel=6), kvec.KVEC_ERR_INVALID),
    (dict(pool_kernel=0), kvec.KVEC_ERR_INVALID),
    (dict(n_adjust_heads=-1), kvec.KVEC_ERR_INVALID),
    (dict(n_adjust_heads=9), kvec.KVEC_ERR_INVALID),
    (dict(lam=-1.0), kvec.KVEC_ERR_INVALID),
    (dict(lam=float("nan")), kvec.KVEC_ERR_INVALID),
    (dict(beta=1.5), kvec.KVEC_ERR_INVALID),
    (dict(dtype=7), kvec.KVEC_ERR_INVALID),
    (dict(head_criterion=2), kvec.KVEC_ERR_INVALID),
    (dict(head_criterion=-1), kvec.KVEC_ERR_INVALID),
    (dict(head_dim=96), kvec.KVEC_ERR_UNSUPPORTED),
    (dict(n_q_heads=72), kvec.KVEC_ERR_UNSUPPORTED),        # G = 9
    (dict(n_kv_heads=16, n_q_heads=32), kvec.KVEC_ERR_UNSUPPORTED),
    (dict(n_kv_heads=3, n_q_heads=12), kvec.KVEC_ERR_UNSUPPORTED),
    (dict(seq_len=300000), kvec.KVEC_ERR_UNSUPPORTED),
    (dict(pool_kernel=65), kvec.KVEC_ERR_UNSUPPORTED),
])
def test_config_validation(over, code):
    st, _ = _ws_status(_cfg(**over))
    assert st == code


def test_entry_points_reject_before_launch():
    lib = kvec.load()
    c = _cfg().c()
    st3 = (ctypes.c_int64 * 3)(32 * 64 * 128, 64 * 128, 128)
    ks3 = (ctypes.c_int64 * 3)(8 * 32768 * 128, 32768 * 128, 128)
    fake = ctypes.c_void_p(1 << 20)          # aligned, never dereferenced
    # null outputs
    assert lib.kvec_score(ctypes.byref(c), fake, st3, fake, ks3, None, fake, fake, fake, 1 << 40,
                          None) == kvec.KVEC_ERR_INVALID
    # misaligned input
    assert lib.kvec_score(ctypes.byref(c), ctypes.c_void_p((1 << 20) + 2), st3, fake, ks3, fake,
                          fake, fake, fake, 1 << 40, None) == kvec.KVEC_ERR_INVALID
    # stride not a multiple of 16 bytes
    bad = (ctypes.c_int64 * 3)(8 * 32768 * 128, 32768 * 128, 127)
    assert lib.kvec_score(ctypes.byref(c), fake, st3, fake, bad, fake, fake, fake, fake, 1 << 40,
                          None) == kvec.KVEC_ERR_INVALID
    # workspace too small
    assert lib.kvec_score(ctypes.byref(c), fake, st3, fake, ks3, fake, fake, fake, fake, 16,
                          None) == kvec.KVEC_ERR_WORKSPACE
    # layer out of range
    assert lib.kvec_select_cover(ctypes.byref(c), 32, fake, fake, fake, fake, fake, None, fake,
                                 1 << 40, None) == kvec.KVEC_ERR_INVALID
    assert lib.kvec_select_cover(ctypes.byref(c), -1, fake, fake, fake, fake, fake, None, fake,
                                 1 << 40, None) == kvec.KVEC_ERR_INVALID
    assert lib.kvec_select_cover(ctypes.byref(c), 0, fake, fake, fake, fake, fake, None, fake, 16,
                                 None) == kvec.KVEC_ERR_WORKSPACE
    assert lib.kvec_coverage(ctypes.byref(c), fake, 32, fake, None) == kvec.KVEC_ERR_INVALID
    assert lib.kvec_compact(ctypes.byref(c), fake, ks3, None, ks3, fake, fake, fake,
                            None) == kvec.KVEC_ERR_INVALID
    # caller-supplied row normalisers: null, misaligned, negative stride
    ls2 = (ctypes.c_int64 * 2)(32 * 64, 64)
    for lse, ls in ((None, ls2), (ctypes.c_void_p((1 << 20) + 2), ls2),
                    (fake, (ctypes.c_int64 * 2)(-1, 64))):
        assert lib.kvec_score_lse(ctypes.byref(c), fake, st3, lse, ls, fake, ks3, fake, fake, fake,
                                  fake, 1 << 40, None) == kvec.KVEC_ERR_INVALID
    assert lib.kvec_score_lse(ctypes.byref(c), fake, st3, fake, ls2, fake, ks3, fake, fake, fake,
                              fake, 16, None) == kvec.KVEC_ERR_WORKSPACE
    vs3 = ks3
    assert lib.kvec_evict_layer_lse(ctypes.byref(c), 0, fake, st3, None, ls2, fake, ks3, fake, vs3,
                                    fake, fake, fake, fake, fake, 1 << 40,
                                    None) == kvec.KVEC_ERR_INVALID
    assert lib.kvec_evict_layer_lse(ctypes.byref(c), 32, fake, st3, fake, ls2, fake, ks3, fake,
                                    vs3, fake, fake, fake, fake, fake, 1 << 40,
                                    None) == kvec.KVEC_ERR_INVALID
    st4 = (ctypes.c_int64 * 4)(32 * 64 * 128, 32 * 64 * 128, 64 * 128, 128)
    ks4 = (ctypes.c_int64 * 4)(8 * 32768 * 128, 8 * 32768 * 128, 32768 * 128, 128)
    ls3 = (ctypes.c_int64 * 3)(32 * 64, 32 * 64, 64)
    assert lib.kvec_evict_model_lse(ctypes.byref(c), fake, st4, None, ls3, fake, ks4, fake, ks4,
                                    fake, fake, fake, fake, fake, 1 << 40, None,
                                    None) == kvec.KVEC_ERR_INVALID
    assert lib.kvec_evict_model_lse(ctypes.byref(c), fake, st4, fake, ls3, fake, ks4, fake, ks4,
                                    fake, fake, fake, fake, fake, 16, None,
                                    None) == kvec.KVEC_ERR_WORKSPACE
    # several steps in one call: step count, outputs, strides, workspace
    st5 = (ctypes.c_int64 * 5)(0, 32 * 64 * 128, 32 * 64 * 128, 64 * 128, 128)
    ks5 = (ctypes.c_int64 * 5)(32 * 8 * 32768 * 128, 8 * 32768 * 128, 8 * 32768 * 128, 32768 * 128, 128)
    steps = lib.kvec_evict_model_steps
    for n in (0, -1, 1 << 16):
        assert steps(ctypes.byref(c), n, fake, st5, fake, ks5, fake, ks5, fake, fake, fake, fake,
                     fake, 1 << 40, None) == kvec.KVEC_ERR_INVALID
    assert steps(ctypes.byref(c), 2, fake, st5, fake, ks5, fake, ks5, None, fake, fake, fake, fake,
                 1 << 40, None) == kvec.KVEC_ERR_INVALID
    assert steps(ctypes.byref(c), 2, fake, None, fake, ks5, fake, ks5, fake, fake, fake, fake, fake,
                 1 << 40, None) == kvec.KVEC_ERR_INVALID
    bad5 = (ctypes.c_int64 * 5)(3, 8 * 32768 * 128, 8 * 32768 * 128, 32768 * 128, 128)
    assert steps(ctypes.byref(c), 2, fake, st5, fake, bad5, fake, ks5, fake, fake, fake, fake, fake,
                 1 << 40, None) == kvec.KVEC_ERR_INVALID
    assert steps(ctypes.byref(c), 2, fake, st5, fake, ks5, fake, ks5, fake, fake, fake, fake, fake,
                 16, None) == kvec.KVEC_ERR_WORKSPACE
    # ... with the normalisers given: the lse pointer and strides are checked first
    ls4 = (ctypes.c_int64 * 4)(0, 32 * 64, 32 * 64, 64)
    lsteps = lib.kvec_evict_model_lse_steps
    def lcall(n=2, lse=fake, lstr=ls4, ws_bytes=1 << 40):
        return lsteps(ctypes.byref(c), n, fake, st5, lse, lstr, fake, ks5, fake, ks5, fake, fake, fake,
                      fake, fake, ws_bytes, None)
    assert lcall(lse=None) == kvec.KVEC_ERR_INVALID
    assert lcall(lse=ctypes.c_void_p((1 << 20) + 2)) == kvec.KVEC_ERR_INVALID
    assert lcall(lstr=None) == kvec.KVEC_ERR_INVALID
    assert lcall(lstr=(ctypes.c_int64 * 4)(-1, 32 * 64, 32 * 64, 64)) == kvec.KVEC_ERR_INVALID
    assert lcall(n=0) == kvec.KVEC_ERR_INVALID
    assert lcall(ws_bytes=16) == kvec.KVEC_ERR_WORKSPACE


def test_decode_validation():
    lib = kvec.load()
    c = _cfg().c()
    fake = ctypes.c_void_p(1 << 20)
    qs = (ctypes.c_int64 * 2)(32 * 128, 128)
    cs = (ctypes.c_int64 * 2)(8 * 1024 * 128, 1024 * 128)
    ok = dict(n=1024, ws=1 << 40)
    assert kvec.kvec_decode_workspace_size(_cfg(), 1024) > 0
    def call(q=fake, kc=fake, n=1024, idx=None, out=fake, ws_bytes=1 << 40, cstr=cs):
        return lib.kvec_decode_attention(ctypes.byref(c), q, qs, kc, fake, cstr, n, idx, out, fake,
                                         ws_bytes, None)
    assert call(n=0) == kvec.KVEC_ERR_INVALID
    assert call(n=(1 << 20) + 1) == kvec.KVEC_ERR_INVALID
    assert call(n=1000, idx=fake) == kvec.KVEC_ERR_INVALID        # idx needs n_ctx >= B
    assert call(q=ctypes.c_void_p((1 << 20) + 4)) == kvec.KVEC_ERR_INVALID
    assert call(out=None) == kvec.KVEC_ERR_INVALID
    assert call(cstr=(ctypes.c_int64 * 2)(8 * 1024 * 128, 1024 * 128 + 1)) == kvec.KVEC_ERR_INVALID
    assert call(ws_bytes=16) == kvec.KVEC_ERR_WORKSPACE


def test_noalloc_decode_validation():
    """The allocation-free decode entry rejects, before any device call, what
    kvec_decode_attention rejects and plans beyond its fixed 4 MiB scratch."""
    lib = kvec.load()
    fake = ctypes.c_void_p(1 << 20)
    qs = (ctypes.c_int64 * 2)(32 * 128, 128)
    cs = (ctypes.c_int64 * 2)(8 * 1024 * 128, 1024 * 128)
    def call(cfg, q=fake, n=1024, idx=None, out=fake):
        c = cfg.c()
        return lib.kvec_decode_attention_noalloc(ctypes.byref(c), q, qs, fake, fake, cs, n, idx,
                                                 out, None)
    assert call(_cfg(), n=0) == kvec.KVEC_ERR_INVALID
    assert call(_cfg(), n=1000, idx=fake) == kvec.KVEC_ERR_INVALID
    assert call(_cfg(), out=None) == kvec.KVEC_ERR_INVALID
    assert call(_cfg(batch=0)) == kvec.KVEC_ERR_INVALID
    big = _cfg(batch=256)   # 256 x 8 heads: one chunk each, 4.26 MB of partial states
    assert kvec.kvec_decode_workspace_size(big, 1024) > 4 << 20
    assert call(big) == kvec.KVEC_ERR_WORKSPACE


def test_profile_points():
    assert kvec.kvec_profile_points(_cfg()) == 32 + 12
    assert kvec.kvec_profile_points_lse(_cfg()) == 32 + 8
    assert kvec.kvec_profile_points_lse(_cfg(seq_len=512, budget=1024)) == 0
    assert kvec.kvec_profile_points_lse(_cfg(batch=0)) == -1


def test_status_strings():
    for s in range(5):
        assert isinstance(kvec.status_string(s), str) and kvec.status_string(s)
    assert kvec.status_string(99) == "unknown status"


def test_plain_c_client(tmp_path):
    """include/kvec.h compiles as C99 and a C program linked against libkvec.so
    runs the host-only calls (no GPU needed)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    kvec.load()
    exe = tmp_path / "abi_check"
    libdir = os.path.dirname(kvec.LIB_PATH)
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           os.path.join(ROOT, "tests", "c", "abi_check.c"), "-L", libdir, "-lkvec",
           f"-Wl,-rpath,{libdir}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert "abi_check: ok" in r.stdout
