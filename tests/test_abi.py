"""C-ABI checks that need no GPU: the library loads, exports what include/bd.h
declares, sizes workspaces, and rejects bad arguments on the host before any
launch (every call here is refused by validation, so no kernel runs)."""
import ctypes
import os
import re

import pytest

import paper_2606_00144_amd as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bd.h")

FAKE = 0x10000000          # a 256-byte aligned non-NULL address that is never dereferenced


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\**\s+\**(bd_[a-z_0-9]+)\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(bd.library_path):
        from paper_2606_00144_amd import build
        build.build_library()
    return bd.lib()


def test_exports_every_declared_symbol(L):
    names = header_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(bd._SIGNATURES)


def test_version_and_status_strings(L):
    assert L.bd_abi_version() == 3
    for s in range(5):
        assert L.bd_status_string(s)
    assert L.bd_status_string(99) == b"unknown status"


def _kv(**over):
    d = bd.KvDesc()
    d.k = d.v = FAKE
    d.num_seqs, d.num_kv_heads, d.head_dim, d.max_seq_len = 2, 8, 128, 4096
    d.seq_lens = FAKE
    d.stride_head, d.stride_tok, d.stride_seq = 4096 * 128, 128, 8 * 4096 * 128
    for k, v in over.items():
        setattr(d, k, v)
    return d


def _verify(L, kv, hq=32, gamma=5, ws=FAKE, wsb=1 << 40, q=FAKE, out=FAKE, scale=0.088):
    return L.bd_verify_attn(ctypes.byref(kv) if kv is not None else None, q, hq, gamma, scale, out, None, ws, wsb, None)


def test_verify_rejections(L):
    assert _verify(L, None) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(head_dim=64)) == bd.BD_ERR_UNSUPPORTED
    assert _verify(L, _kv(k=0)) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(k=FAKE + 8)) == bd.BD_ERR_INVALID_ARG             # misaligned K
    assert _verify(L, _kv(seq_lens=0)) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(), hq=30) == bd.BD_ERR_INVALID_ARG                # Hq % Hkv != 0
    assert _verify(L, _kv(), gamma=-1) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(), q=0) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(), out=FAKE + 2) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(), scale=float("nan")) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(), scale=0.0) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(), scale=-0.088) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(stride_tok=100)) == bd.BD_ERR_INVALID_ARG
    assert _verify(L, _kv(page_table=FAKE, page_size=16, max_pages_per_seq=10, num_pages=100,
                          stride_page=8 * 16 * 128)) == bd.BD_ERR_INVALID_ARG   # 4096 > 10 * 16
    assert _verify(L, _kv(), ws=None) == bd.BD_ERR_WORKSPACE
    assert _verify(L, _kv(), ws=FAKE + 64) == bd.BD_ERR_WORKSPACE
    assert _verify(L, _kv(), wsb=16) == bd.BD_ERR_WORKSPACE
    assert b"workspace" in L.bd_last_error()


def test_verify_noalloc_rejections(L):
    # refused by host validation: nothing is launched and no device is touched
    na = lambda kv, **a: L.bd_verify_attn_noalloc(ctypes.byref(kv), a.get("q", FAKE), 32, a.get("g", 5), 0.088,
                                                  a.get("out", FAKE), None, None)
    assert na(_kv(), g=-1) == bd.BD_ERR_INVALID_ARG
    assert na(_kv(), out=FAKE + 2) == bd.BD_ERR_INVALID_ARG
    assert na(_kv(head_dim=64)) == bd.BD_ERR_UNSUPPORTED
    # 64 sequences x 32 KV heads paged up to 16384 rows in pages of 8 (the per-key table bounds the
    # splits to 2,048 keys): the plan's records exceed the fixed scratch
    big = _kv(num_seqs=64, num_kv_heads=32, max_seq_len=16384, page_table=FAKE, page_size=8,
              max_pages_per_seq=2048, num_pages=131072, stride_page=32 * 8 * 128, stride_head=8 * 128)
    assert na(big) == bd.BD_ERR_UNSUPPORTED
    assert b"scratch" in L.bd_last_error()


def test_decode_select_multiview_accept_rejections(L):
    kv = _kv()
    assert L.bd_sparse_decode_attn(ctypes.byref(kv), FAKE, 32, FAKE, -1, FAKE, 0.1, FAKE, None, FAKE, 1 << 40, None) == 1
    assert L.bd_sparse_decode_attn(ctypes.byref(kv), FAKE, 32, FAKE, 64, None, 0.1, FAKE, None, FAKE, 1 << 40, None) == 1
    assert L.bd_sparse_decode_attn(ctypes.byref(kv), FAKE, 32, FAKE, 64, FAKE, 0.1, FAKE, None, None, 0, None) == 3
    sel = lambda **a: L.bd_select_kv(ctypes.byref(a.get("kv", kv)), FAKE, 32, a.get("W", 32), a.get("B", 256),
                                     a.get("P", 7), 0.1, None, FAKE, FAKE, None, FAKE, 1 << 40, None)
    assert sel(W=0) == 1
    assert sel(W=64, B=32) == 1
    assert sel(P=4) == 1
    assert sel(P=301) == 2
    assert sel(kv=_kv(max_seq_len=40000)) == 2                              # prefix above BD_SELECT_MAX_PREFIX
    ch = lambda **a: L.bd_select_kv_chunks(ctypes.byref(kv), FAKE, 32, 32, a.get("B", 256), a.get("s", 8),
                                           a.get("cw", 0), 0.1, None, FAKE, FAKE, None, FAKE, 1 << 40, None)
    assert ch(s=0) == 1
    assert ch(cw=2) == 1                                                     # the switch is 0 or 1
    assert ch(B=16) == 1                                                     # budget below the window
    assert ch(B=2 ** 31 - 8) == 1                                            # B + W slots overflow int32
    mv = lambda **a: L.bd_multiview_attn(ctypes.byref(kv), FAKE, 32, a.get("C", 64), a.get("V", 4), FAKE, 1024, FAKE,
                                         0.1, a.get("ov", FAKE), None, None, a.get("of", FAKE), None, a.get("o32f"),
                                         FAKE, 1 << 40, None)
    assert mv(C=0) == 1
    assert mv(V=0, of=None) == 1
    assert mv(ov=None) == 1
    assert mv(o32f=FAKE + 8) == 1                                            # misaligned fp32 output
    assert mv(V=64) == 2                                     # block mode: 64 views + the full cache > 64 branches
    acc = lambda **a: L.bd_accept_len(a.get("lg", FAKE), a.get("rs", 32000), a.get("dr", FAKE), 2, a.get("g", 5),
                                      32000, FAKE, None, None, FAKE, 1 << 40, None)
    assert acc(lg=None) == 1
    assert acc(rs=100) == 1
    assert acc(g=64) == 2
    assert acc(dr=None) == 1


def test_multiview_bwd_rejections(L):
    kv = _kv()

    def bwd(**a):
        g = lambda n, d=FAKE: a.get(n, d)
        return L.bd_multiview_attn_bwd(ctypes.byref(g("kv", kv)), g("q"), 32, g("C", 64), g("V", 4), g("idx"), 1024,
                                       g("nsel"), g("scale", 0.1), g("ov"), g("lv"), g("dov"), g("of"), g("lf"),
                                       g("dof"), g("dq"), g("dk"), g("dv"), g("ws"), g("wsb", 1 << 40), None)
    assert bwd(C=0) == bd.BD_ERR_INVALID_ARG
    assert bwd(C=2048) == bd.BD_ERR_UNSUPPORTED                             # block above 1024 rows
    assert bwd(V=0, dof=None, of=None, lf=None) == bd.BD_ERR_INVALID_ARG   # no branch at all
    assert bwd(lv=None) == bd.BD_ERR_INVALID_ARG                          # views need their lse
    assert bwd(dov=FAKE + 4) == bd.BD_ERR_INVALID_ARG
    assert bwd(lf=None) == bd.BD_ERR_INVALID_ARG                          # full branch half given
    assert bwd(of=None) == bd.BD_ERR_INVALID_ARG
    assert bwd(dq=None) == bd.BD_ERR_INVALID_ARG
    assert bwd(dk=None) == bd.BD_ERR_INVALID_ARG                          # dk without dv
    assert bwd(scale=float("inf")) == bd.BD_ERR_INVALID_ARG
    assert bwd(q=FAKE + 2) == bd.BD_ERR_INVALID_ARG
    assert bwd(kv=_kv(v=0)) == bd.BD_ERR_INVALID_ARG
    assert bwd(ws=None) == bd.BD_ERR_WORKSPACE
    assert bwd(wsb=1024) == bd.BD_ERR_WORKSPACE
    big = _kv(num_seqs=4096, num_kv_heads=8, max_seq_len=64, stride_seq=8 * 64 * 128, stride_head=64 * 128)
    assert bwd(kv=big) == bd.BD_ERR_UNSUPPORTED                           # counter lines exhausted
    assert bwd(V=64) == bd.BD_ERR_UNSUPPORTED                             # 65 branches


def test_workspace_sizes(L):
    v = L.bd_verify_attn_workspace_bytes(8, 8, 32, 5, 16384)
    assert v > 0 and v % 256 == 0
    assert L.bd_sparse_decode_attn_workspace_bytes(8, 8, 32, 1024) > 0
    assert L.bd_select_kv_workspace_bytes(8, 8, 32, 32, 16384) >= 8 * 8 * 16384 * 4
    assert L.bd_multiview_attn_workspace_bytes(4, 8, 32, 64, 4, 2048, 8192, 1) > 0
    w = L.bd_multiview_attn_bwd_workspace_bytes(4, 8, 32, 64, 4, 2048, 8192, 1)
    assert w > (1 << 20) and w % 256 == 0
    assert L.bd_multiview_attn_bwd_workspace_bytes(4, 8, 32, 0, 4, 2048, 8192, 1) == 0
    assert L.bd_accept_len_workspace_bytes(8, 5, 128256) > 0
    assert L.bd_verify_attn_workspace_bytes(0, 8, 32, 5, 16384) == 0        # invalid shape -> 0


def test_update_rejections(L):
    A = lambda kv, n=1, kn=FAKE, idx=None, nsel=None, ld=0: L.bd_cache_append(
        ctypes.byref(kv) if kv is not None else None, kn, FAKE, n, idx, ld, nsel, None)
    assert A(None) == bd.BD_ERR_INVALID_ARG
    assert A(_kv(), n=-1) == bd.BD_ERR_INVALID_ARG
    assert A(_kv(), n=0) == bd.BD_OK                                        # nothing to do, nothing launched
    assert A(_kv(), kn=0) == bd.BD_ERR_INVALID_ARG
    assert A(_kv(), kn=FAKE + 4) == bd.BD_ERR_INVALID_ARG                   # misaligned rows
    assert A(_kv(), idx=FAKE) == bd.BD_ERR_INVALID_ARG                      # idx without nsel
    assert A(_kv(), idx=FAKE, nsel=FAKE, ld=-1) == bd.BD_ERR_INVALID_ARG
    assert A(_kv(head_dim=64)) == bd.BD_ERR_UNSUPPORTED
    R = L.bd_cache_rollback
    assert R(None, None, FAKE, 2, 5, None, None, None) == bd.BD_ERR_INVALID_ARG
    assert R(FAKE, None, None, 2, 5, None, None, None) == bd.BD_ERR_INVALID_ARG
    assert R(FAKE, None, FAKE, 0, 5, None, None, None) == bd.BD_ERR_INVALID_ARG
    assert R(FAKE, None, FAKE, 2, -1, None, None, None) == bd.BD_ERR_INVALID_ARG
    assert R(FAKE, None, FAKE, 2, 5, FAKE, FAKE, None) == bd.BD_ERR_INVALID_ARG     # base_nsel without nsel


_EXTREME = [-2 ** 31, -1, 0, 1, 2, 7, 8, 32, 33, 64, 4096, 16384, 32768, 65536, 2 ** 24, 2 ** 30, 2 ** 31 - 1]


def test_workspace_sizes_of_extreme_shapes(L):
    """Every size function answers for any arguments (0 for shapes its operation rejects) and never
    fails: seeded random and extreme arguments.  Built with the host sanitizers (build.py
    --host-sanitize) this run also shows that the planning arithmetic stays in range."""
    import random
    sizes = {n: len(sig[1]) for n, sig in bd._SIGNATURES.items() if n.endswith("_workspace_bytes")}
    rng = random.Random(11)
    for name, nargs in sizes.items():
        f = getattr(L, name)
        for _ in range(3000):
            args = [rng.choice(_EXTREME) if rng.random() < 0.6 else rng.randint(-10, 70000) for _ in range(nargs)]
            assert f(*args) >= 0, (name, args)
    # shapes the operations reject give 0
    assert L.bd_verify_attn_workspace_bytes(2 ** 16, 2 ** 9, 2 ** 9, 5, 4096) == 0       # more than 2^24 pairs
    assert L.bd_verify_attn_workspace_bytes(8, 8, 32, 4096, 16384) == 0                   # gamma above 4095
    assert L.bd_sparse_decode_attn_workspace_bytes(8, 1, 2 ** 17, 1024) == 0              # group above 2^16
    assert L.bd_select_kv_workspace_bytes(8, 8, 32, 2 ** 31 - 1, 16384) == 0              # window * group
    assert L.bd_select_kv_workspace_bytes(8, 8, 32, 32, 40000) == 0                       # prefix above the cap
    assert L.bd_multiview_attn_workspace_bytes(4, 8, 32, 2 ** 19, 4, 2048, 8192, 1) == 0  # block * group
    assert L.bd_multiview_attn_bwd_workspace_bytes(4, 8, 32, 64, 64, 2048, 8192, 1) == 0  # 65 branches
    assert L.bd_accept_len_workspace_bytes(8, 64, 128256) == 0                            # gamma above 63


def test_extreme_shapes_are_refused_before_launch(L):
    """Sizes whose plans would leave 32- or 64-bit range are refused by the host checks."""
    assert _verify(L, _kv(num_seqs=2 ** 20, num_kv_heads=32), hq=32) == bd.BD_ERR_UNSUPPORTED   # 2^25 pairs
    assert _verify(L, _kv(num_kv_heads=1), hq=2 ** 17) == bd.BD_ERR_UNSUPPORTED                 # group 2^17
    assert _verify(L, _kv(), gamma=2 ** 31 - 1) == bd.BD_ERR_INVALID_ARG
    kv = _kv()
    sel = lambda W, hq: L.bd_select_kv(ctypes.byref(kv), FAKE, hq, W, 2 ** 31 - 1, 7, 0.1, None, FAKE, FAKE, None,
                                       FAKE, 1 << 40, None)
    assert sel(2 ** 31 - 1, 64) == bd.BD_ERR_UNSUPPORTED       # window * group overflows 32 bits
    assert sel(4096, 64) == bd.BD_ERR_UNSUPPORTED
    mv = lambda C, V: L.bd_multiview_attn(ctypes.byref(kv), FAKE, 32, C, V, FAKE, 2 ** 31 - 1, FAKE, 0.1, FAKE, None,
                                          None, FAKE, None, None, FAKE, 1 << 40, None)
    assert mv(1, 2 ** 31 - 1) == bd.BD_ERR_UNSUPPORTED           # views x pairs: too many work units
    assert mv(64, 2 ** 31 - 1) == bd.BD_ERR_UNSUPPORTED          # block mode: too many branches
    assert mv(2 ** 31 - 1, 4) == bd.BD_ERR_UNSUPPORTED           # block * group


def test_header_serves_a_c_program(L, tmp_path):
    """include/bd.h compiles as C11 (warnings as errors for the program's own code) and a C program
    links against the library and calls it: a refused call gives its status and reason."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    src = tmp_path / "abi.c"
    src.write_text(
        '#include "bd.h"\n#include <stdio.h>\n'
        "int main(void) {\n"
        "  bd_kv_desc kv = {0};\n"
        "  kv.head_dim = 64;\n"
        "  bd_status st = bd_verify_attn(&kv, NULL, 32, 5, 0.1f, NULL, NULL, NULL, 0, NULL);\n"
        '  printf("%d %d %s\\n", bd_abi_version(), (int)st, bd_last_error());\n'
        "  return st == BD_ERR_UNSUPPORTED ? 0 : 1;\n"
        "}\n")
    exe = tmp_path / "abi"
    libdir = os.path.dirname(bd.library_path)
    libname = os.path.basename(bd.library_path)
    r = subprocess.run([gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-isystem", "/opt/rocm/include",
                        "-D__HIP_PLATFORM_AMD__", f"-I{os.path.dirname(HEADER)}", str(src), f"-L{libdir}",
                        f"-l:{libname}", f"-Wl,-rpath,{libdir}", "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, (out.stdout, out.stderr)
    version, status, reason = out.stdout.split(" ", 2)
    assert int(version) == L.bd_abi_version() and int(status) == bd.BD_ERR_UNSUPPORTED
    assert "head_dim 64" in reason
