"""The C-ABI library loads on a CPU-only host and exports every entry point
that include/*.h declares (no compute call is made here)."""
import ctypes
import glob
import os
import re

import paper_2607_23250_amd as pl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b(libra_\w+)\s*\(", src, re.M):
            names.add(m.group(1))
    return names


def test_header_declares_the_entry_points():
    assert _declared() == set(pl.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = pl.lib()
    for name in _declared():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_strerror_names_every_code():
    L = pl.lib()
    for code in (0, -1, -2, -3, -4, -5):
        assert L.libra_strerror(code).decode() != "unknown error"
    assert L.libra_strerror(-99).decode() == "unknown error"


def test_workspace_size_rejects_bad_shapes():
    assert pl.libra_attn_workspace_size(4, 2, 100, 100, 4, 2, 128, False) > 0
    assert pl.libra_attn_workspace_size(4, 2, 100, 100, 4, 2, 128, True) > 0
    assert pl.libra_attn_workspace_size(4, 2, 100, 100, 4, 3, 128, False) == 0   # 3 does not divide 4
    assert pl.libra_attn_workspace_size(4, 2, 100, 100, 4, 2, 96, False) == 0    # head_dim 96
    assert pl.libra_attn_workspace_size(-1, 2, 100, 100, 4, 2, 64, True) == 0


def test_attention_entry_points_validate_before_touching_the_device():
    L = pl.lib()
    ws = ctypes.create_string_buffer(1024)
    # unsupported head_dim: rejected before any pointer is used
    rc = L.libra_attn_fwd(None, None, None, None, 1, None, 1, 10, 10, 2, 1, 96, 0.0, None, None,
                          ws, 1024, None)
    assert rc == pl.LIBRA_EUNSUPPORTED
    # NULL tensors with tiles present
    rc = L.libra_attn_fwd(None, None, None, None, 1, None, 1, 10, 10, 2, 1, 64, 0.0, None, None,
                          ws, 1024, None)
    assert rc == pl.LIBRA_EINVAL
    assert b"NULL" in L.libra_last_error()
    # no tiles: nothing to do
    rc = L.libra_attn_fwd(None, None, None, None, 1, None, 0, 10, 10, 2, 1, 64, 0.0, None, None,
                          None, 0, None)
    assert rc == pl.LIBRA_OK
    # unknown flag
    rc = L.libra_attn_bwd(None, None, None, None, None, None, None, 1, None, 0, 10, 10, 2, 1, 64,
                          0.0, None, ws, ws, 8, None, 0, None)
    assert rc == pl.LIBRA_EINVAL
    # workspace too small (fake non-NULL pointers; rejected on the host)
    fake = ctypes.c_void_p(4096)
    rc = L.libra_attn_fwd(fake, fake, fake, fake, 1, fake, 1, 10, 10, 2, 1, 64, 0.0, fake, fake,
                          ctypes.c_void_p(4096), 16, None)
    assert rc == pl.LIBRA_ENOSPC
    # misaligned workspace
    rc = L.libra_attn_fwd(fake, fake, fake, fake, 1, fake, 1, 10, 10, 2, 1, 64, 0.0, fake, fake,
                          ctypes.c_void_p(4096 + 8), 1 << 30, None)
    assert rc == pl.LIBRA_EINVAL


def test_skipped_tiles_query_rejects_null_arguments():
    """The documented route to the skipped-tile count validates its arguments
    on the host (no device access for NULL pointers)."""
    import ctypes as C
    L = pl.lib()
    n = C.c_int32(-7)
    assert L.libra_attn_skipped_tiles(None, C.byref(n), None) == pl.LIBRA_EINVAL
    assert L.libra_attn_skipped_tiles(C.c_void_p(256), None, None) == pl.LIBRA_EINVAL
    assert n.value == -7
    assert pl.LIBRA_WS_SKIPPED_OFFSET == 16


def test_noalloc_forward_rejects_oversize_on_the_host():
    """libra_attn_fwd_noalloc checks its sizes against the built-in scratch
    before touching the device: a tile count whose work items exceed it is
    LIBRA_ENOSPC (pointers are never dereferenced on the host)."""
    import ctypes as C
    L = pl.lib()
    dummy = C.c_void_p(256)
    T = pl.LIBRA_FWD_NOALLOC_MAX_WORKSPACE // 32
    assert pl.libra_attn_workspace_size(T, 4, 4096, 4096, 8, 2, 128, False) > \
        pl.LIBRA_FWD_NOALLOC_MAX_WORKSPACE
    rc = L.libra_attn_fwd_noalloc(dummy, dummy, dummy, dummy, 4, dummy, T, 4096, 4096, 8, 2, 128,
                                  C.c_float(0.0), dummy, dummy, None)
    assert rc == pl.LIBRA_ENOSPC
    assert b"built-in scratch" in L.libra_last_error()
    rc = L.libra_attn_fwd_noalloc(dummy, dummy, dummy, dummy, 4, dummy, 16, 4096, 4096, 8, 2, 96,
                                  C.c_float(0.0), dummy, dummy, None)
    assert rc == pl.LIBRA_EUNSUPPORTED
