"""CPU checks of the C-ABI library: it loads, exports every declared symbol, and its host-side
validation and workspace plan behave as include/tilemix.h states (no kernel is launched)."""

import ctypes
import os
import re
import subprocess

import pytest

import paper_2608_17336_amd as tm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tilemix.h")

pytestmark = pytest.mark.skipif(not os.path.exists(tm.library_path()),
                                reason="libtilemix.so not built (run __graft_entry__.build())")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tilemix_[a-z0-9_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert _declared_functions() == sorted(tm.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = tm.load_library()
    for name in _declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", tm.library_path()], capture_output=True,
                         text=True).stdout
    for name in _declared_functions():
        assert re.search(rf"\bT {name}$", out, re.M), name


def _cp(**kw):
    base = dict(batch=1, heads_q=32, heads_kv=8, len_q=8192, len_k=8192, head_dim=128,
                block_m=128, block_n=64, group_size=1, causal=True, scale=0.0884)
    base.update(kw)
    return tm.Params(**base)


def test_words_per_row():
    assert tm.tilemix_route_words_per_row(_cp()) == 2                       # 128 groups
    assert tm.tilemix_route_words_per_row(_cp(len_q=4096, len_k=4096)) == 1
    assert tm.tilemix_route_words_per_row(_cp(len_q=131072, len_k=131072, group_size=16)) == 2
    assert tm.tilemix_route_words_per_row(_cp(len_q=131072, len_k=131072, group_size=1)) == 32
    assert tm.tilemix_route_words_per_row(_cp(head_dim=96)) == 0            # invalid -> 0


def test_workspace_matches_quantize_once_accounting():
    # H_q=32, H_k=8, L=8192, d=128.  The attention kernel quantizes each query block in the
    # prologue of the workgroup that owns it, so the workspace holds K8 (8 MiB), the key scales
    # (128 blocks x 8 heads, FP16) and the V tiles (|V| = 16 MiB); the fused mode only the V tiles.
    n = tm.tilemix_workspace_size(_cp())
    k8 = 8192 * 8 * 128
    scales = 128 * 8 * 2
    vt = 8192 * 8 * 128 * 2
    assert k8 + scales + vt <= n <= k8 + scales + vt + 4 * 256
    nf = tm.tilemix_fused_workspace_size(_cp())
    assert vt <= nf <= vt + 2 * 256


@pytest.mark.parametrize("kw,status", [
    (dict(heads_q=30), 2),          # H_q % H_k
    (dict(head_dim=96), 3),
    (dict(block_m=256), 3),
    (dict(block_n=128), 3),
    (dict(group_size=0), 2),
    (dict(len_q=0), 2),
    (dict(scale=-1.0), 2),
    (dict(route_hint=1), 2),
])
def test_validation_errors(kw, status):
    with pytest.raises(tm.TilemixError) as e:
        tm.tilemix_workspace_size(_cp(**kw))
    assert e.value.status == status
    assert tm.load_library().tilemix_last_error().decode()


def test_prefill_rejects_before_launch():
    lib = tm.load_library()
    cp = _cp().c()
    # NULL tensors
    st = lib.tilemix_prefill(ctypes.byref(cp), None, None, None, None, None, None, 0, None)
    assert st == 1
    # misaligned pointers (never dereferenced: validation fails first)
    fake = ctypes.c_void_p(0x1001)
    st = lib.tilemix_prefill(ctypes.byref(cp), fake, fake, fake, fake, fake, fake, 1 << 30, None)
    assert st == 4
    # workspace too small
    ok = ctypes.c_void_p(0x100000)
    st = lib.tilemix_prefill(ctypes.byref(cp), ok, ok, ok, ok, ok, ok, 1024, None)
    assert st == 5
    assert b"needed" in lib.tilemix_last_error()
    # params NULL
    assert lib.tilemix_prefill(None, ok, ok, ok, ok, ok, ok, 1 << 40, None) == 1
    assert lib.tilemix_status_string(5) == b"workspace missing or too small"


def test_debug_and_quantize_reject_before_launch():
    lib = tm.load_library()
    cp = _cp().c()
    ok = ctypes.c_void_p(0x100000)
    assert lib.tilemix_debug_qk_int32(ctypes.byref(cp), ok, ok, ok, -1, ok, None) == 2
    assert lib.tilemix_debug_qk_int32(ctypes.byref(cp), ok, ok, ok, 0, ok, None) == 0   # nothing to do
    assert lib.tilemix_quantize(ctypes.byref(cp), None, ok, ok, ok, ok, ok, None) == 1


def test_decode_rejects_before_launch():
    # Every call below fails a host-side check, so no kernel is launched (the pointers are fake).
    lib = tm.load_library()
    ok = ctypes.c_void_p(0x100000)
    dp = dict(len_q=1, len_k=5000, heads_q=64, heads_kv=8, group_size=8)

    def call(cp, ptr=ok, ws=None, ws_bytes=1 << 40):
        return lib.tilemix_decode(ctypes.byref(cp.c()), ptr, ptr, ptr, ptr, ptr, ptr, ptr, ptr, ws,
                                  ws_bytes, None)

    assert call(_cp(**dp)) == 5                                  # shapes pass; no workspace
    assert call(_cp(**dict(dp, len_q=2))) == 3                   # one query token only
    assert call(_cp(**dict(dp, heads_q=136, heads_kv=8))) == 3   # G = 17 > 16
    assert call(_cp(**dict(dp, len_k=262145))) == 3              # past the longest cache
    assert call(_cp(**dict(dp, len_k=262144))) == 5
    assert call(_cp(**dp), ptr=None) == 1
    assert call(_cp(**dp), ptr=ctypes.c_void_p(0x1001)) == 4
    assert call(_cp(**dp), ws=ctypes.c_void_p(0x100080)) == 4
    # partial results: B * H_q * ceil(L_k / 512) chunks of (max, normalizer, d floats) while the
    # batch holds at most 2048 key tiles (one tile per wave of each 8-wave workgroup)
    need = tm.tilemix_decode_workspace_size(_cp(**dp))
    assert need >= 64 * 10 * (2 + 128) * 4
    assert call(_cp(**dp), ws=ok, ws_bytes=need - 1) == 5
    assert b"needed" in lib.tilemix_last_error()


def test_noalloc_rejects_before_launch():
    # Host-side checks only: every call below returns before any device call.
    lib = tm.load_library()
    ok = ctypes.c_void_p(0x100000)
    big = _cp(batch=4, heads_q=64, len_q=65536, len_k=65536, group_size=8)   # 1.6 GB workspace
    assert tm.tilemix_workspace_size(big) > tm.NOALLOC_SCRATCH_BYTES
    st = lib.tilemix_prefill_noalloc(ctypes.byref(big.c()), ok, ok, ok, ok, ok, None)
    assert st == 5
    assert b"at most 134217728" in lib.tilemix_last_error()
    small = _cp()
    assert tm.tilemix_workspace_size(small) <= tm.NOALLOC_SCRATCH_BYTES
    assert lib.tilemix_prefill_noalloc(ctypes.byref(small.c()), None, ok, ok, ok, ok, None) == 1
    assert lib.tilemix_prefill_noalloc(ctypes.byref(small.c()), ok, ok, ok, ok, None, None) == 1
    fake = ctypes.c_void_p(0x100001)
    assert lib.tilemix_prefill_noalloc(ctypes.byref(small.c()), fake, ok, ok, ok, ok, None) == 4
    assert lib.tilemix_prefill_noalloc(None, ok, ok, ok, ok, ok, None) == 1


def test_one_hip_runtime_after_load():
    # Loading the library before torch would map a second HIP runtime (torch's wheel carries its
    # own under the same soname), whose device list the first one owns.
    import sys
    code = ("import os, sys; sys.path.insert(0, %r); import paper_2608_17336_amd as tm; "
            "tm.load_library(); maps = open('/proc/%%d/maps' %% os.getpid()).read(); "
            "print(len({l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}))" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_decode_varlen_rejects_before_launch():
    lib = tm.load_library()
    ok = ctypes.c_void_p(0x100000)
    cp = _cp(len_q=1, len_k=5000, heads_q=64, heads_kv=8, group_size=8).c()
    args = [ok] * 8 + [ok, 1 << 40, None]
    assert lib.tilemix_decode_varlen(ctypes.byref(cp), None, *args) == 1
    assert lib.tilemix_decode_varlen(ctypes.byref(cp), ctypes.c_void_p(0x100002), *args) == 4
    bad = _cp(len_q=2, len_k=5000, heads_q=64, heads_kv=8).c()
    assert lib.tilemix_decode_varlen(ctypes.byref(bad), ok, *args) == 3
