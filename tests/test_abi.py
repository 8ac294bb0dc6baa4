"""The C-ABI library loads and exports every entry point include/arckv.h declares (CPU only)."""

import ctypes
import os
import re

import pytest

import paper_2606_21238_amd as ak
from paper_2606_21238_amd import _lib

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "arckv.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(arckv_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_symbols():
    decl = declared_functions()
    assert decl == sorted(_lib.SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_version_and_pool_bytes():
    assert ak.lib().arckv_version() == 1
    assert ak.pool_bytes(10, 8, 128) == 10 * 8 * 16 * 128 * 2
    assert ak.pool_bytes(-1, 8, 128) == -1


def test_device_calls_validate_arguments_without_touching_a_device():
    L = ak.lib()
    # unsupported head_dim / group size are refused before any launch
    assert L.arckv_kv_scatter(None, None, None, None, None, 4, 4, 2, 96, None) == _lib.EUNSUPPORTED
    assert L.arckv_prefill_attention(None, None, None, None, None, 1, None, None, 1, 1, 1, None, 1, 0,
                                     256, 12, 4, 128, 0.1, None, 0, None) == _lib.EUNSUPPORTED
    assert L.arckv_prefill_attention(None, None, None, None, None, 1, None, None, 1, 1, 1, None, 1, 0,
                                     256, 8, 4, 128, 0.1, None, 0, None) == _lib.EINVAL
    assert b"NULL" in L.arckv_last_error()
    assert L.arckv_prefill_attention(None, None, None, None, None, 1, None, None, 1, 1, 1, None, 1, 0,
                                     200, 8, 4, 128, 0.1, None, 0, None) == _lib.EINVAL
    assert b"tile_cols" in L.arckv_last_error()
    # nothing to do is a no-op
    assert L.arckv_kv_scatter(None, None, None, None, None, 0, 4, 2, 64, None) == _lib.OK
    # misaligned pools or rows are refused before any launch (the addresses are never read)
    a, m = 0x20000, 0x20008
    assert L.arckv_kv_scatter(a, m, a, a, a, 4, 4, 2, 64, None) == _lib.EINVAL
    assert b"aligned" in L.arckv_last_error()


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="not built"):
        _lib.load(str(tmp_path / "nope.so"))


def test_qkv_rope_validates_arguments_without_touching_a_device():
    L = ak.lib()
    args = lambda d, theta, t=4: (None, None, t, 64, 4, 2, d, None, None, 1, theta, None, 0, None, None, None, None)
    assert L.arckv_qkv_rope(*args(96, 1.0e6)) == _lib.EUNSUPPORTED
    assert L.arckv_qkv_rope(*args(128, 1.0)) == _lib.EINVAL
    assert L.arckv_qkv_rope(*args(128, 1.0e6)) == _lib.EINVAL          # NULL pointers
    assert b"NULL" in L.arckv_last_error()
    assert L.arckv_qkv_rope(*args(128, 1.0e6, t=0)) == _lib.OK         # nothing to do
    # the fused kernel's tiling: hidden in steps of 32, outputs in steps of 128
    assert L.arckv_qkv_rope(None, None, 4, 48, 4, 2, 128, None, None, 1, 1.0e6, None, 0, None, None, None,
                            None) == _lib.EUNSUPPORTED
    assert L.arckv_qkv_rope(None, None, 4, 64, 5, 1, 64, None, None, 1, 1.0e6, None, 0, None, None, None,
                            None) == _lib.EUNSUPPORTED
    # misaligned outputs are refused before any device work (the addresses are never read)
    a, m = 0x10000, 0x10002
    assert L.arckv_qkv_rope(a, a, 4, 64, 4, 2, 128, a, a, 1, 1.0e6, a, 1 << 20, a, m, a, None) == _lib.EINVAL
    assert b"aligned" in L.arckv_last_error()
    # the workspace holds 4 tokens x 64 (cos, sin) pairs of fp32: one byte short is refused
    assert L.arckv_qkv_rope(a, a, 4, 64, 4, 2, 128, a, a, 1, 1.0e6, a, 4 * 4 * 128 - 1, a, a, a,
                            None) == _lib.ENOSPC


def test_qkv_rope_to_pool_validates_arguments_without_touching_a_device():
    """The producer that writes K/V into the pool shares the producer's checks and adds its own
    (pool size, slot mapping); every refusal happens before any device work, so the fake
    addresses below are never read."""
    L = ak.lib()
    a, m = 0x10000, 0x10002

    def call(t=4, d=128, nb=8, slots=a, kp=a, ws=1 << 20, theta=1.0e6):
        return L.arckv_qkv_rope_to_pool(a, a, t, 64, 4, 2, d, a, a, 1, theta, a, ws, a, kp, a, nb, slots, None)

    assert call(d=96) == _lib.EUNSUPPORTED
    assert call(theta=1.0) == _lib.EINVAL
    assert call(nb=0) == _lib.EINVAL and b"num_blocks" in L.arckv_last_error()
    assert call(nb=(1 << 27) + 1) == _lib.EINVAL
    assert call(slots=None) == _lib.EINVAL and b"NULL" in L.arckv_last_error()
    assert call(kp=m) == _lib.EINVAL and b"aligned" in L.arckv_last_error()
    assert call(ws=4 * 4 * 128 - 1) == _lib.ENOSPC
    assert call(t=0) == _lib.OK                                        # nothing to do


def test_device_checks_only_in_the_checked_build():
    """The product build has no device checks (EUNSUPPORTED, no GPU touched); the checked
    debug build exists beside it and exports the same calls."""
    bits, count = _lib.i32(), _lib.i64()
    assert ak.lib().arckv_device_checks(bits, count, 0, None) == _lib.EUNSUPPORTED
    assert b"without" in ak.lib().arckv_last_error()
    from paper_2606_21238_amd.build import CHECKED_LIB
    chk = _lib.load(CHECKED_LIB)
    for name in _lib._SIGS:
        assert hasattr(chk, name), name
