"""CPU tests of the binding's tensor checks (no GPU, no library call).

The C entry points take bare device addresses, so the binding is the only
place that can see where a tensor lives, how wide a cos/sin table is and
how long the tensors behind a prebuilt argument struct stay alive. These
tests call the checking helpers directly with CPU tensors; on the CPU a
tensor's device index is -1, which stands in for "the cache's device" where
a check must pass.
"""
import gc
import weakref

import pytest
import torch

import paper_2609_37241_amd as tri
from paper_2609_37241_amd import _check_cos_sin, _dims, _like, _on, _vector


def test_host_tensor_is_rejected_before_any_native_call():
    x = torch.zeros(4, 8)
    with pytest.raises(ValueError, match="on the CPU"):
        _on(x, "x", 0)
    with pytest.raises(ValueError, match="cuda:0"):
        _dims(x, "x", 2, 0)
    with pytest.raises(ValueError, match="cache's device"):
        _like(x, "out", (4, 8), torch.float32, 0)
    with pytest.raises(ValueError, match="cache's device"):
        _vector(torch.zeros(8), "w", 8, torch.float32, 0)


def test_shape_checks_still_come_first():
    x = torch.zeros(4, 8)
    with pytest.raises(ValueError, match="expected 2 dims"):
        _dims(torch.zeros(8), "x", 2, 0)
    with pytest.raises(ValueError, match=r"expected \(4, 8\)"):
        _like(torch.zeros(4, 9), "out", x.shape, x.dtype, 0)


def test_matching_device_passes():
    x = torch.zeros(4, 8)
    assert _dims(x, "x", 2, -1) == (4, 8)
    _like(x, "out", (4, 8), torch.float32, -1)
    _vector(torch.zeros(8), "w", 8, torch.float32, -1)


def test_cos_sin_table_width_must_equal_the_rotated_span():
    hd = 128
    ok = tri.rope_ext(cos_sin=torch.zeros(300, hd))
    _check_cos_sin(ok, hd, -1)
    narrow = tri.rope_ext(cos_sin=torch.zeros(300, 64))
    with pytest.raises(ValueError, match="rows of 128 floats"):
        _check_cos_sin(narrow, hd, -1)
    partial = tri.rope_ext(rotary_dim=64, cos_sin=torch.zeros(300, 64))
    _check_cos_sin(partial, hd, -1)
    wide = tri.rope_ext(rotary_dim=64, cos_sin=torch.zeros(300, 128))
    with pytest.raises(ValueError, match="rows of 64 floats"):
        _check_cos_sin(wide, hd, -1)


def test_cos_sin_table_must_be_on_the_cache_device():
    ext = tri.rope_ext(cos_sin=torch.zeros(10, 64))
    with pytest.raises(ValueError, match="cos_sin: tensor on the CPU"):
        _check_cos_sin(ext, 64, 0)


def test_cos_sin_set_by_hand_is_refused():
    ext = tri.RopeExt()
    ext.cos_sin = 4096
    ext.cos_sin_len = 10
    with pytest.raises(ValueError, match="rope_ext"):
        _check_cos_sin(ext, 64, -1)
    _check_cos_sin(tri.RopeExt(), 64, -1)       # no table: nothing to check
    _check_cos_sin(None, 64, -1)


def test_rope_ext_keeps_its_table_alive():
    t = torch.zeros(10, 64)
    ref = weakref.ref(t)
    ext = tri.rope_ext(cos_sin=t)
    del t
    gc.collect()
    assert ref() is not None and ext.cos_sin == ref().data_ptr()
    del ext
    gc.collect()
    assert ref() is None


class _NullStream:
    cuda_stream = 0        # the null stream, named without asking torch for a device


_NULL_STREAM = _NullStream()


class _Shell(tri.SpecCache):
    """A cache that was never created: nothing to release."""

    def close(self):
        self._h = None


def _recording_cache():
    """A SpecCache shell that only records: prepare() runs the op method,
    whose one entry call is noted, never issued (no library call here)."""
    import ctypes as C
    c = object.__new__(_Shell)
    c._h = C.c_void_p(0x1000)
    c._dev = -1            # a CPU tensor's device index: the checks pass
    c._rec = None
    c.misses_handled = 0
    return c


def test_prepare_converts_every_argument_once():
    """The prepared call holds the op's arguments (without the stream) as
    C objects of the entry point's parameter types, and the method's result."""
    import ctypes as C
    from paper_2609_37241_amd import _lib as L
    c = _recording_cache()
    x = torch.zeros(4, 8, dtype=torch.bfloat16)
    w = torch.ones(8, dtype=torch.bfloat16)
    y = torch.empty_like(x)
    p = c.prepare("rmsnorm", x, w, 1e-6, out=y, stream=_NULL_STREAM)
    assert p.result is y
    types = L.SIGNATURES["tri_rmsnorm"][1]
    assert len(p._cargs) == len(types) - 1                   # the stream comes per call
    assert isinstance(p._cargs[0], C.c_void_p) and p._cargs[0].value == 0x1000
    for t, a in zip(types[1:-1], p._cargs[1:]):
        assert type(a) is t, (t, a)
    assert p._cargs[1].value == L.BF16 and p._cargs[-1].value == pytest.approx(1e-6)
    assert (p._cargs[2].value, p._cargs[4].value) == (x.data_ptr() or None, w.data_ptr() or None)
    assert [a.value for a in p._cargs[6:9]] == [8, 4, 8]      # y row stride, T, H


def test_prepare_keeps_the_struct_of_a_prebuilt_chain_call():
    import ctypes as C
    c = _recording_cache()
    args = tri.ChainArgs()
    p = c.prepare("decode_chain_args", args, _NULL_STREAM)
    (ref,) = p._cargs[1:]
    assert type(ref).__name__ == "CArgObject" and ref._obj is args   # passed by reference
    assert isinstance(p._cargs[0], C.c_void_p)


def test_prepare_refuses_what_is_not_an_op_call():
    c = _recording_cache()
    for bad in ("close", "prepare", "_call", "no_such_op"):
        with pytest.raises(ValueError):
            c.prepare(bad)
    c.close()
    with pytest.raises(tri.TriError):
        c.prepare("rmsnorm", torch.zeros(1, 8), torch.ones(8), 1e-6, stream=_NULL_STREAM)
