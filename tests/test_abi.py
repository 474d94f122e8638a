"""The C ABI loads, exports every declared symbol, and validates on the host.

No compute call is made here: every call below fails host-side validation
before anything would be launched, so these run without a GPU.
"""
import ctypes
import os
import re

import pytest

import paper_2511_03092_amd as snap

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "snapstream.h")
FAKE = 0x100000  # aligned, never dereferenced (validation fails first)


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(snap_[a-z_]+)\s*\(", src)))


def _params(**kw):
    base = dict(n_q_heads=32, n_kv_heads=8, d_qk=128, d_v=128, sink=4, recent=1024, topk=3068,
                obs_window=32, pool_kernel=7)
    base.update(kw)
    return snap.Params(**base)


def test_library_exports_every_declared_symbol():
    L = snap.lib()
    names = _declared()
    assert set(names) == set(snap.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def test_debug_build_exports_the_same_symbols_and_release_refuses_checks():
    """The debug build (device-side invariant checks) has the same entry
    points; the release build answers snap_debug_checks with
    SNAP_ERR_UNSUPPORTED and zero flags, without touching the device."""
    D = snap.load(snap.DEBUG_LIB_PATH)
    for n in _declared():
        assert hasattr(D, n), n
    flags = ctypes.c_uint32(7)
    assert snap.lib().snap_debug_checks(ctypes.byref(flags), 1) == snap.SNAP_ERR_UNSUPPORTED
    assert flags.value == 0
    assert snap.lib().snap_debug_checks(None, 1) == snap.SNAP_ERR_INVALID_ARG


def test_status_strings():
    for s in range(5):
        assert snap.snap_status_str(s)
    assert snap.snap_status_str(0) == "ok"


def test_workspace_queries_are_host_only():
    p = _params()
    ws = snap.snap_compress_workspace(p, 1, 32768)
    # at least A and P over the padded length
    assert ws >= 2 * 8 * 32768 * 4
    assert snap.snap_compress_workspace(p, 8, 131072) > ws
    assert snap.snap_decode_workspace(p, 8) > 0
    assert snap.snap_compress_workspace(_params(pool_kernel=4), 1, 100) == 0
    assert snap.snap_decode_workspace(_params(n_q_heads=30), 1) == 0


def _compress_status(p, ws_bytes=1 << 30, **kw):
    L = snap.lib()
    cache = snap.SnapCache(FAKE, FAKE if not p.v_in_k else None, None, None, 4)
    args = dict(pos=FAKE, n_topk=FAKE, n_seq=1, slot_ids=FAKE, lengths=FAKE, max_len=4096,
                q=FAKE, k=FAKE, v=None if p.v_in_k else FAKE, ws=FAKE)
    args.update(kw)
    st = L.snap_compress(ctypes.byref(p.c()), ctypes.byref(cache), args["pos"], args["n_topk"], args["n_seq"],
                         args["slot_ids"], args["lengths"], args["max_len"], args["q"], args["k"], args["v"],
                         None, None, args["ws"], ws_bytes, None)
    return st, L.snap_last_error().decode()


@pytest.mark.parametrize("bad,code", [
    (dict(n_q_heads=30), snap.SNAP_ERR_INVALID_ARG),
    (dict(recent=0), snap.SNAP_ERR_INVALID_ARG),
    (dict(pool_kernel=6), snap.SNAP_ERR_INVALID_ARG),
    (dict(pool_kernel=65), snap.SNAP_ERR_INVALID_ARG),
    (dict(d_qk=96, d_v=96), snap.SNAP_ERR_UNSUPPORTED),
    (dict(n_q_heads=64, n_kv_heads=2), snap.SNAP_ERR_UNSUPPORTED),
    (dict(in_dtype=snap.SNAP_F32, kv_dtype=snap.SNAP_BF16), snap.SNAP_ERR_UNSUPPORTED),
    (dict(obs_window=128), snap.SNAP_ERR_UNSUPPORTED),
    (dict(norm=5), snap.SNAP_ERR_INVALID_ARG),
    (dict(sm_scale=1e-31), snap.SNAP_ERR_INVALID_ARG),
    (dict(sm_scale=float("inf")), snap.SNAP_ERR_INVALID_ARG),
])
def test_invalid_params_rejected(bad, code):
    st, msg = _compress_status(_params(**bad))
    assert st == code and msg


def test_workspace_too_small():
    p = _params()
    need = snap.snap_compress_workspace(p, 1, 4096)
    st, msg = _compress_status(p, ws_bytes=need - 1)
    assert st == snap.SNAP_ERR_WORKSPACE and str(need) in msg
    st, _ = _compress_status(p, ws=FAKE + 16)  # not 256-byte aligned
    assert st == snap.SNAP_ERR_WORKSPACE


def test_null_and_misaligned_pointers():
    p = _params()
    assert _compress_status(p, k=None)[0] == snap.SNAP_ERR_INVALID_ARG
    assert _compress_status(p, q=FAKE + 2)[0] == snap.SNAP_ERR_INVALID_ARG
    assert _compress_status(p, lengths=None)[0] == snap.SNAP_ERR_INVALID_ARG
    assert _compress_status(p, max_len=0)[0] == snap.SNAP_ERR_INVALID_ARG
    lat = _params(n_q_heads=8, n_kv_heads=1, d_qk=576, d_v=512, v_in_k=True)
    assert _compress_status(lat, v=FAKE)[0] == snap.SNAP_ERR_INVALID_ARG
    assert _compress_status(_params(v_in_k=False, d_qk=576, d_v=512, n_q_heads=8, n_kv_heads=1))[0] == \
        snap.SNAP_ERR_UNSUPPORTED


def test_fp8_cache_needs_scales():
    p = _params(kv_dtype=snap.SNAP_FP8_E4M3)
    st, msg = _compress_status(p)
    assert st == snap.SNAP_ERR_INVALID_ARG and "scale" in msg


def test_empty_batch_is_a_no_op():
    # n_seq == 0 returns before any launch
    st, _ = _compress_status(_params(), n_seq=0)
    assert st == snap.SNAP_OK


def test_decode_and_append_validation():
    L = snap.lib()
    p = _params()
    cache = snap.SnapCache(FAKE, FAKE, None, None, 4)
    st = L.snap_decode_attn(ctypes.byref(p.c()), ctypes.byref(cache), FAKE, FAKE, 2, FAKE, FAKE, FAKE,
                            snap.SNAP_BF16, FAKE, 16, None)
    assert st == snap.SNAP_ERR_WORKSPACE
    st = L.snap_decode_attn(ctypes.byref(p.c()), ctypes.byref(cache), FAKE, FAKE, 2, FAKE, FAKE, FAKE,
                            7, FAKE, 1 << 30, None)
    assert st == snap.SNAP_ERR_INVALID_ARG
    st = L.snap_cache_append(ctypes.byref(p.c()), ctypes.byref(cache), FAKE, 2, FAKE, FAKE, None, None)
    assert st == snap.SNAP_ERR_INVALID_ARG  # v_new missing
    assert L.snap_advance(FAKE, 0, 1, FAKE, None) == snap.SNAP_ERR_INVALID_ARG
    assert L.snap_advance(FAKE, 4, 0, FAKE, None) == snap.SNAP_OK


def test_decode_step_validation():
    """snap_decode_step checks everything snap_cache_append and
    snap_decode_attn check, before any launch."""
    L = snap.lib()
    p = _params()
    cache = snap.SnapCache(FAKE, FAKE, None, None, 4)
    big = 1 << 30

    def step(q=FAKE, k_new=FAKE, v_new=FAKE, out=FAKE, out_dtype=snap.SNAP_BF16, ws=FAKE, ws_bytes=big, n=2,
             params=p, c=cache):
        return L.snap_decode_step(ctypes.byref(params.c()), ctypes.byref(c), FAKE, FAKE, n, FAKE, q, k_new, v_new,
                                  out, out_dtype, ws, ws_bytes, None)

    assert step(k_new=None) == snap.SNAP_ERR_INVALID_ARG
    assert step(k_new=FAKE + 4) == snap.SNAP_ERR_INVALID_ARG           # misaligned
    assert step(v_new=None) == snap.SNAP_ERR_INVALID_ARG               # GQA cache needs v_new
    assert step(q=None) == snap.SNAP_ERR_INVALID_ARG
    assert step(out=FAKE + 8) == snap.SNAP_ERR_INVALID_ARG
    assert step(out_dtype=snap.SNAP_FP8_E4M3) == snap.SNAP_ERR_INVALID_ARG
    assert step(ws_bytes=16) == snap.SNAP_ERR_WORKSPACE
    assert step(ws=FAKE + 64) == snap.SNAP_ERR_WORKSPACE               # not 256-byte aligned
    assert step(n=-1) == snap.SNAP_ERR_INVALID_ARG
    assert step(n=0) == snap.SNAP_OK                                   # no-op
    assert step(params=_params(pool_kernel=4)) == snap.SNAP_ERR_INVALID_ARG
    # latent cache: values live in K, so v_new must be absent
    lat = _params(n_q_heads=8, n_kv_heads=1, d_qk=576, d_v=512, v_in_k=1, recent=4096, topk=28668)
    lcache = snap.SnapCache(FAKE, None, None, None, 4)
    assert step(params=lat, c=lcache, ws_bytes=16) == snap.SNAP_ERR_WORKSPACE   # v_new ignored, then ws
    assert b"workspace" in snap.lib().snap_last_error()


def test_noalloc_step_validation():
    """snap_decode_step_noalloc makes snap_decode_step's checks and refuses a
    call whose partials would not fit the library's scratch array, before any
    device query (so on a host without a GPU)."""
    L = snap.lib()
    p = _params()
    cache = snap.SnapCache(FAKE, FAKE, None, None, 4)

    def step(n=2, params=p, c=cache, v_new=FAKE, out_dtype=snap.SNAP_BF16):
        return L.snap_decode_step_noalloc(ctypes.byref(params.c()), ctypes.byref(c), FAKE, FAKE, n, FAKE, FAKE,
                                          FAKE, v_new, FAKE, out_dtype, None)

    assert step(v_new=None) == snap.SNAP_ERR_INVALID_ARG
    assert step(out_dtype=snap.SNAP_FP8_E4M3) == snap.SNAP_ERR_INVALID_ARG
    assert step(n=0) == snap.SNAP_OK
    assert step(params=_params(pool_kernel=4)) == snap.SNAP_ERR_INVALID_ARG
    # latent rows (512 value dims) for 8191 sequences of 8 heads: one chunk
    # each, 8191 * 8 * 512 * 4 bytes of partials > the 32 MiB array
    lat = _params(n_q_heads=8, n_kv_heads=1, d_qk=576, d_v=512, v_in_k=1, recent=4096, topk=28668)
    lcache = snap.SnapCache(FAKE, None, None, None, 4)
    n = 8191
    assert snap.snap_decode_workspace(lat, n) > (32 << 20)
    assert step(n=n, params=lat, c=lcache, v_new=None) == snap.SNAP_ERR_WORKSPACE
    assert b"scratch" in L.snap_last_error()


def test_prefill_validation():
    """snap_prefill: the shapes it supports, its workspace and pointer checks,
    all before any launch."""
    L = snap.lib()
    p = _params()
    cache = snap.SnapCache(FAKE, FAKE, None, None, 4)
    need = snap.snap_prefill_workspace(p, 1, 4096)
    # the compress workspace plus the window queries and the transposed V
    assert need >= snap.snap_compress_workspace(p, 1, 4096) + 32 * 32 * 128 * 2 + 8 * 128 * 4096 * 2
    assert snap.snap_prefill_workspace(_params(pool_kernel=4), 1, 100) == 0

    def pre(params=p, q=FAKE, k=FAKE, v=FAKE, out=FAKE, ws=FAKE, ws_bytes=1 << 34, n_seq=1, max_len=4096):
        return L.snap_prefill(ctypes.byref(params.c()), ctypes.byref(cache), FAKE, FAKE, n_seq, FAKE, FAKE, max_len,
                              q, k, v, out, None, None, ws, ws_bytes, None)

    assert pre(out=None) == snap.SNAP_ERR_INVALID_ARG
    assert pre(out=FAKE + 2) == snap.SNAP_ERR_INVALID_ARG
    assert pre(v=None) == snap.SNAP_ERR_INVALID_ARG
    assert pre(q=FAKE + 8) == snap.SNAP_ERR_INVALID_ARG
    assert pre(ws_bytes=need - 1) == snap.SNAP_ERR_WORKSPACE
    assert pre(ws=FAKE + 64) == snap.SNAP_ERR_WORKSPACE
    assert pre(n_seq=0) == snap.SNAP_OK
    assert pre(max_len=0) == snap.SNAP_ERR_INVALID_ARG
    # unsupported shapes and dtypes
    assert pre(params=_params(in_dtype=snap.SNAP_F32, kv_dtype=snap.SNAP_F32)) == snap.SNAP_ERR_UNSUPPORTED
    assert pre(params=_params(n_q_heads=48, n_kv_heads=4)) == snap.SNAP_ERR_UNSUPPORTED  # G = 12
    assert pre(params=_params(n_q_heads=24, n_kv_heads=4, obs_window=16)) == snap.SNAP_ERR_UNSUPPORTED  # G = 6
    lat = _params(n_q_heads=8, n_kv_heads=1, d_qk=576, d_v=512, v_in_k=1, recent=4096, topk=28668)
    lcache = snap.SnapCache(FAKE, None, None, None, 4)
    assert L.snap_prefill(ctypes.byref(lat.c()), ctypes.byref(lcache), FAKE, FAKE, 1, FAKE, FAKE, 4096, FAKE, FAKE,
                          None, FAKE, None, None, FAKE, 1 << 34, None) == snap.SNAP_ERR_UNSUPPORTED
    # a supported fp8 cache still needs its scales
    assert pre(params=_params(kv_dtype=snap.SNAP_FP8_E4M3)) == snap.SNAP_ERR_INVALID_ARG


def test_prefill_attn_validation():
    L = snap.lib()
    p = _params()

    def att(params=p, q=FAKE, k=FAKE, v=FAKE, out=FAKE, ws=FAKE, ws_bytes=1 << 34, n_seq=1, max_len=4096, lengths=FAKE):
        return L.snap_prefill_attn(ctypes.byref(params.c()), n_seq, lengths, max_len, q, k, v, out, ws, ws_bytes, None)

    need = snap.snap_prefill_workspace(p, 1, 4096)
    assert att(out=None) == snap.SNAP_ERR_INVALID_ARG
    assert att(lengths=None) == snap.SNAP_ERR_INVALID_ARG
    assert att(k=FAKE + 4) == snap.SNAP_ERR_INVALID_ARG
    assert att(ws_bytes=need - 1) == snap.SNAP_ERR_WORKSPACE
    assert att(n_seq=0) == snap.SNAP_OK
    assert att(params=_params(d_qk=576, d_v=512, v_in_k=1, n_q_heads=8, n_kv_heads=1)) == snap.SNAP_ERR_UNSUPPORTED
    assert att(params=_params(pool_kernel=2)) == snap.SNAP_ERR_INVALID_ARG


def test_fp8_qk_validation():
    assert _compress_status(_params(fp8_qk=2))[0] == snap.SNAP_ERR_INVALID_ARG
    assert _compress_status(_params(fp8_qk=1))[0] == snap.SNAP_ERR_UNSUPPORTED  # bf16 cache
    assert _compress_status(_params(fp8_qk=1, kv_dtype=snap.SNAP_FP8_E4M3, d_qk=64, d_v=64))[0] == \
        snap.SNAP_ERR_UNSUPPORTED
    # a supported fp8 setting fails later (the fake cache has no scales), not on fp8_qk
    st, msg = _compress_status(_params(fp8_qk=1, kv_dtype=snap.SNAP_FP8_E4M3))
    assert st == snap.SNAP_ERR_INVALID_ARG and "scale" in msg


def test_kv_reuse_validation():
    """The decode load hint: the three snap_kv_reuse values pass the parameter
    checks (a workspace size comes back), anything else is refused."""
    for bad in (-1, 3, 7):
        assert _compress_status(_params(kv_reuse=bad))[0] == snap.SNAP_ERR_INVALID_ARG
    for ok in (snap.SNAP_KV_AUTO, snap.SNAP_KV_STREAM, snap.SNAP_KV_KEEP):
        assert snap.snap_decode_workspace(_params(kv_reuse=ok), 4) > 0


def test_launch_grid_limits():
    """Sizes whose per-(sequence, head) launch grids would not fit are refused
    before any launch."""
    L = snap.lib()
    p = _params()
    assert _compress_status(p, n_seq=8192)[0] == snap.SNAP_ERR_UNSUPPORTED  # 8192 x 8 KV heads
    cache = snap.SnapCache(FAKE, FAKE, None, None, 4)
    st = L.snap_decode_attn(ctypes.byref(p.c()), ctypes.byref(cache), FAKE, FAKE, 4096, FAKE, FAKE, FAKE,
                            snap.SNAP_BF16, FAKE, 1 << 34, None)
    assert st == snap.SNAP_ERR_UNSUPPORTED  # 4096 x 32 query heads
    st = L.snap_prefill_attn(ctypes.byref(p.c()), 64, FAKE, 1 << 28, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 62, None)
    assert st == snap.SNAP_ERR_UNSUPPORTED  # 512 groups x 2^23 position blocks


def test_library_binds_to_torchs_hip_runtime():
    """Loaded before anything imported torch, the library still ends up on
    torch's HIP runtime (the one that owns the device memory the binding
    passes in): one libamdhip64 in the process, not two."""
    import subprocess
    import sys
    code = ("import sys; sys.path.insert(0, %r)\n"
            "import paper_2511_03092_amd as snap\n"
            "snap.lib()\n"
            "print(sorted(set(l.split()[-1] for l in open('/proc/self/maps') if 'amdhip64' in l)))\n") % ROOT
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    maps = eval(out.stdout.strip().splitlines()[-1])
    assert len(maps) == 1 and "torch" in maps[0], maps


def test_header_compiles_and_links_as_c(tmp_path):
    """tests/c_abi_host.c, a plain C11 caller, compiles against the header
    with -Wall -Werror, links the built library and gets workspace sizes and
    a refused parameter back without a GPU."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    exe = tmp_path / "c_abi_host"
    libdir = os.path.dirname(snap.LIB_PATH)
    r = subprocess.run([cc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
                        os.path.join(ROOT, "tests", "c_abi_host.c"), "-L", libdir, "-lsnapstream",
                        "-Wl,-rpath," + libdir, "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "status 1 invalid argument" in out.stdout and "pool_kernel" in out.stdout, out.stdout
