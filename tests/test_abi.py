"""The C ABI without a GPU: the header compiles as C, libdla.so loads and
exports every entry point the header declares, and host-side argument checks
return their status codes without touching a device."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dla.h")


def _declared():
    """Entry points declared by every header under include/."""
    names = set()
    for f in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(dla_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_header_compiles_as_c(tmp_path):
    c = tmp_path / "t.c"
    c.write_text('#include "dla.h"\n#include "dla_peak.h"\n'
                 'int main(void){dla_cache_desc d={1,1,1,64,64,DLA_BF16};(void)d;return 0;}\n')
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    "-fsyntax-only", str(c)], check=True)


def test_library_exports_every_declared_symbol():
    from paper_2606_10650_amd import dla
    lib = dla.lib()
    names = _declared()
    assert "dla_prefill" in names and "dla_decode_step" in names
    for n in names:
        assert hasattr(lib, n), f"{n} declared in dla.h but not exported"
    assert set(dla.EXPORTED) == set(names)


def test_host_side_errors():
    from paper_2606_10650_amd import dla
    L = dla.lib()
    lay = dla.Layout()
    bad = [dla.CacheDesc(1, 1, 8, 96, 64), dla.CacheDesc(1, 1, 2000, 64, 64)]
    for d in bad:
        assert L.dla_cache_layout_of(ctypes.byref(d), ctypes.byref(lay)) == dla.DLA_ERR_UNSUPPORTED
    d = dla.CacheDesc(0, 1, 8, 64, 64)
    assert L.dla_cache_layout_of(ctypes.byref(d), ctypes.byref(lay)) == dla.DLA_ERR_INVALID_ARG
    d = dla.CacheDesc(2, 3, 8, 64, 128)
    assert L.dla_cache_layout_of(ctypes.byref(d), ctypes.byref(lay)) == dla.DLA_OK
    assert lay.total_bytes == lay.states_offset + 6 * 8 * 64 * 128 * 4
    n = ctypes.c_size_t(0)
    assert L.dla_state_cache_alloc(ctypes.byref(d), None, ctypes.byref(n), None) == dla.DLA_OK
    assert n.value == lay.total_bytes
    p = dla.Params(0.5, 1e-6, 1e-6, 0)
    fake = ctypes.c_void_p(0x1000)
    # missing k
    st = L.dla_prefill(ctypes.byref(d), fake, fake, None, fake, fake, None, 10, 1, ctypes.byref(p),
                       fake, 1, None, None, None, None, None, fake, 1 << 30, None)
    assert st == dla.DLA_ERR_INVALID_ARG
    assert L.dla_get_last_error() == dla.DLA_ERR_INVALID_ARG
    # workspace too small
    st = L.dla_prefill(ctypes.byref(d), fake, fake, fake, fake, fake, None, 10, 1, ctypes.byref(p),
                       fake, 1, None, None, None, None, None, fake, 16, None)
    assert st == dla.DLA_ERR_WORKSPACE
    # readout events: a negative count, or a count without the array
    for n_ev, arr in ((-1, None), (4, None)):
        pe = dla.Params(0.5, 1e-6, 1e-6, 0, None, arr, n_ev)
        st = L.dla_prefill(ctypes.byref(d), fake, fake, fake, fake, fake, None, 10, 1,
                           ctypes.byref(pe), fake, 1, None, None, None, None, None, fake, 1 << 30,
                           None)
        assert st == dla.DLA_ERR_INVALID_ARG, n_ev
    # a pipelined call needs no more workspace than a serial one (the same pool
    # when every state copy fits the budget, plus the scan carry)
    wp, wsr = ctypes.c_size_t(0), ctypes.c_size_t(0)
    d16 = dla.CacheDesc(4, 16, 128, 128, 128)
    assert L.dla_prefill_workspace_size(ctypes.byref(d16), 16384, 1, 0, ctypes.byref(wp)) == 0
    assert L.dla_prefill_workspace_size(ctypes.byref(d16), 16384, 1, dla.DLA_SERIAL_STAGES,
                                        ctypes.byref(wsr)) == 0
    assert wp.value >= wsr.value and wp.value - wsr.value < (1 << 24)
    # bad dtype
    st = L.dla_prefill(ctypes.byref(d), fake, fake, fake, fake, fake, None, 10, 7, ctypes.byref(p),
                       fake, 1, None, None, None, None, None, fake, 1 << 30, None)
    assert st == dla.DLA_ERR_INVALID_ARG
    # T = 0 is a no-op
    st = L.dla_prefill(ctypes.byref(d), fake, fake, fake, fake, fake, None, 0, 1, ctypes.byref(p),
                       fake, 1, None, None, None, None, None, None, 0, None)
    assert st == dla.DLA_OK
    # decode without q but with readout
    st = L.dla_decode_step(ctypes.byref(d), fake, None, fake, fake, fake, None, 1,
                           ctypes.byref(p), fake, 1, None, None, None, None, None, None)
    assert st == dla.DLA_ERR_INVALID_ARG
    assert dla.status_string(dla.DLA_ERR_WORKSPACE) == "workspace missing or too small"
    ws = ctypes.c_size_t(0)
    assert L.dla_prefill_workspace_size(ctypes.byref(d), 1000, 1, 0, ctypes.byref(ws)) == dla.DLA_OK
    assert ws.value >= 6 * 1000 * 12


def _header(B, H, C, dk, dv, flags=0, state_dtype=0, magic=0x31414C44, version=2):
    import struct
    return struct.pack("<II5iIi", magic, version, B, H, C, dk, dv, flags, state_dtype) + bytes(220)


def test_header_check_on_a_host_copy():
    """dla_cache_header_check (host only) accepts the header a cache of the
    descriptor is made with and refuses any difference: magic, version, shape
    or state type."""
    from paper_2606_10650_amd import dla
    d = dla.CacheDesc(2, 3, 8, 64, 128)
    assert dla.header_check(d, _header(2, 3, 8, 64, 128, flags=1)) == 1
    for bad in (_header(2, 3, 8, 64, 128, magic=0x31414C45), _header(2, 3, 8, 64, 128, version=1),
                _header(2, 3, 16, 64, 128), _header(2, 4, 8, 64, 128), _header(1, 3, 8, 64, 128),
                _header(2, 3, 8, 128, 128), _header(2, 3, 8, 64, 64),
                _header(2, 3, 8, 64, 128, state_dtype=1)):
        with pytest.raises(dla.DLAError) as e:
            dla.header_check(d, bad)
        assert e.value.status == dla.DLA_ERR_CACHE_MISMATCH
    L = dla.lib()
    assert L.dla_cache_header_check(ctypes.byref(d), None, None) == dla.DLA_ERR_INVALID_ARG


def test_state_type_of_the_descriptor():
    """The descriptor's state type must be float32 or bfloat16; float32 caches
    have no open region."""
    from paper_2606_10650_amd import dla
    L = dla.lib()
    lay = dla.Layout()
    d = dla.CacheDesc(2, 3, 8, 64, 128, 7)
    assert L.dla_cache_layout_of(ctypes.byref(d), ctypes.byref(lay)) == dla.DLA_ERR_INVALID_ARG
    d = dla.CacheDesc(2, 3, 8, 64, 128, dla.DLA_F32)
    assert L.dla_cache_layout_of(ctypes.byref(d), ctypes.byref(lay)) == dla.DLA_OK
    assert lay.open_offset == 0


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    from paper_2606_10650_amd import dla
    monkeypatch.setattr(dla, "_lib", None)
    monkeypatch.setattr(dla, "_LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(RuntimeError, match="missing"):
        dla.lib()


@pytest.mark.parametrize("dtype", [0, 1])  # DLA_F32, DLA_BF16
def test_every_supported_shape_passes_the_prefill_shape_check(dtype):
    """Every head dimension pair and capacity the header declares supported
    gets past dla_prefill's shape checks (the stages' LDS working sets fit):
    with no workspace the call stops at DLA_ERR_WORKSPACE, before any device
    access."""
    from paper_2606_10650_amd import dla
    L = dla.lib()
    p = dla.Params(0.5, 1e-6, 1e-6, 0)
    fake = ctypes.c_void_p(0x1000)
    for dk in (64, 128):
        for dv in (64, 128):
            for C in (1, 8, 128, 256, 512, 1000, 1024):
                d = dla.CacheDesc(1, 2, C, dk, dv)
                st = L.dla_prefill(ctypes.byref(d), fake, fake, fake, fake, fake, fake, 4096, dtype,
                                   ctypes.byref(p), fake, dtype, None, None, None, None, None,
                                   None, 0, None)
                assert st == dla.DLA_ERR_WORKSPACE, (dk, dv, C, dtype, st)


def test_prefill_segment_counts():
    """Segment plan (host only): a pipelined prefill of the 16k-token workload
    runs as a ramp of five segments; serial stages keep one segment while the
    state copies fit the pool budget; a call of one chunk is never split."""
    from paper_2606_10650_amd import dla
    L = dla.lib()

    def count(B, H, C, d, T, dtype, flags):
        desc = dla.CacheDesc(B, H, C, d, d)
        n = ctypes.c_int32(0)
        assert L.dla_prefill_segment_count(ctypes.byref(desc), T, dtype, flags,
                                           ctypes.byref(n)) == dla.DLA_OK
        return n.value

    assert count(4, 16, 128, 128, 16384, dla.DLA_BF16, 0) == 5   # 2, 3, 5, 8, 14 chunks
    assert count(4, 16, 128, 128, 16384, dla.DLA_BF16, dla.DLA_SERIAL_STAGES) == 1
    # 64k tokens at C = 256: the pool budget splits even the serial call
    assert count(1, 32, 256, 128, 65536, dla.DLA_BF16, dla.DLA_SERIAL_STAGES) == 4
    assert count(1, 32, 256, 128, 65536, dla.DLA_BF16, 0) >= 4
    assert count(1, 2, 16, 128, 512, dla.DLA_BF16, 0) == 1
    assert count(1, 2, 16, 128, 1100, dla.DLA_BF16, 0) == 2
    assert count(1, 2, 16, 128, 0, dla.DLA_BF16, 0) == 1
    assert count(1, 2, 16, 128, 1100, dla.DLA_BF16, dla.DLA_SKIP_READOUT) == 1
    # a state-copy budget in the flags: 1 GiB splits the 16k-token workload
    # (256 MiB of copies per chunk) into segments of at most 4 chunks, 256 MiB
    # into single chunks; the workspace shrinks with it; bad budgets are refused
    serial = dla.DLA_SERIAL_STAGES
    assert count(4, 16, 128, 128, 16384, dla.DLA_BF16, serial | dla._flags(False, False, 30)) == 8
    assert count(4, 16, 128, 128, 16384, dla.DLA_BF16, serial | dla._flags(False, False, 28)) == 32
    assert count(4, 16, 128, 128, 16384, dla.DLA_BF16, dla._flags(False, False, 30)) == 9
    ws = []
    for kb in (0, 31, 30, 29):
        d = dla.CacheDesc(4, 16, 128, 128, 128)
        n = ctypes.c_size_t(0)
        assert L.dla_prefill_workspace_size(ctypes.byref(d), 16384, dla.DLA_BF16,
                                            dla._flags(False, False, kb), ctypes.byref(n)) == 0
        ws.append(n.value)
    assert ws == sorted(ws, reverse=True) and ws[-1] < (1 << 30) < ws[0]
    for kb in (19, 41, 255):
        d = dla.CacheDesc(4, 16, 128, 128, 128)
        n = ctypes.c_size_t(0)
        assert L.dla_prefill_workspace_size(ctypes.byref(d), 16384, dla.DLA_BF16,
                                            dla._flags(False, False, kb),
                                            ctypes.byref(n)) == dla.DLA_ERR_INVALID_ARG
    # segment starts: the ramp of the 16k-token workload (2, 3, 5, 8, 14 chunks of 512)
    desc = dla.CacheDesc(4, 16, 128, 128, 128)
    arr = (ctypes.c_int32 * 8)(*([-7] * 8))
    assert L.dla_prefill_segment_starts(ctypes.byref(desc), 16384, dla.DLA_BF16, 0, arr, 8) == 0
    assert list(arr)[:6] == [0, 1024, 2560, 5120, 9216, -7]
