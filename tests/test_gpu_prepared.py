"""GPU: prepared calls (SpecCache.prepare) -- one op call marshalled once and
issued again -- against the binding's ordinary method calls and the oracle,
on caches with kernel arguments and with resident argument blocks.

Each case prints its name (pytest -v) before touching the GPU. Inputs from
`workloads`, expected values from `oracle`.
"""
import pytest
import torch

from oracle import ops as O
from tests.parity import check
from tests.test_gpu_parity import DEV, host
from tests.test_gpu_resident import _op_case, _to_device
import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


PREPARED = {
    # op case -> (method, positional inputs, keyword outputs, result names)
    "rmsnorm_bf16": ("rmsnorm", ("x", "w", 1e-6), {"out": "y"}, ("y",)),
    "rmsnorm_f32_1024x128": ("rmsnorm", ("x", "w", 1e-6), {"out": "y"}, ("y",)),
    "residual_bf16": ("residual_rmsnorm", ("x", "r", "w", 1e-6),
                      {"out": "y", "residual_out": "ro"}, ("y", "res_out")),
    "rope_bf16": ("rope_qk", ("q", "k", "pos", 5e5), {}, ()),
    "swiglu_bf16": ("swiglu", ("g", "u"), {"out": "o"}, ("out",)),
    "silu_bf16": ("silu", ("a",), {"out": "o"}, ("out",)),
    "add_f32": ("add", ("a", "b"), {"out": "o"}, ("out",)),
    "masked_fill_bf16": ("masked_fill", ("a", "m", -1e4), {"out": "o"}, ("out",)),
}
ALLOC = {"y": "x", "ro": "x", "o": None}


def _inputs(name, d):
    """Positional arguments and output tensors of the prepared call."""
    method, pos, kw, _ = PREPARED[name]
    args = tuple(d[a] if isinstance(a, str) else a for a in pos)
    outs = {}
    for k, n in kw.items():
        like = d[ALLOC[n]] if ALLOC[n] else next(v for v in d.values()
                                                  if v.dtype != torch.int32 and v.dim() == 2
                                                  and v.dtype != torch.uint8)
        outs[k] = d.setdefault(n, torch.empty_like(like))
    return method, args, outs


@pytest.mark.parametrize("resident", [False, True], ids=["kernel_args", "resident"])
@pytest.mark.parametrize("name", list(PREPARED))
def test_prepared_call_equals_the_method_and_the_oracle(tri, name, resident):
    """The prepared call, issued three times with the inputs refreshed in
    place, gives the method call's outputs bit for bit and the oracle's."""
    dt, h, want, run = _op_case(name, seed=len(name) * 31)
    c = tri.SpecCache(resident_args=resident)          # no auto-install: a MISS first
    ref = tri.SpecCache(auto_install=True)
    try:
        a, b = _to_device(h, dt), _to_device(h, dt)
        method, args, outs = _inputs(name, b)
        p = c.prepare(method, *args, **outs)
        for call in range(3):
            for d in (a, b):
                for k, v in _to_device(h, dt).items():
                    d[k].copy_(v)
            got = run(ref, a)                           # the ordinary method
            p()
            torch.cuda.synchronize()
            for n in want:
                g = {"y": "y", "res_out": "ro", "out": "o"}.get(n, n)
                check(f"{name} call {call} {n}", host(b[g]), host(got[n]), dt, exact=True)
        assert c.misses_handled == 1 and c.stats()["hits"] == 3
        if resident:
            info = c.resident_info()
            assert info["held"] == 1 and info["launches"] == 3, info
        for n, w in want.items():
            g = {"y": "y", "res_out": "ro", "out": "o"}.get(n, n)
            check(f"{name} {n} vs oracle", host(b[g]), w, dt, exact=n in ("res_out",))
    finally:
        torch.cuda.synchronize()
        c.close()
        ref.close()


def test_prepared_chain_follows_new_data(tri):
    """A prepared decode chain on a resident cache: five steps with new
    inputs written into the same tensors, each the oracle's result."""
    cfg = wl.LLAMA7B_DECODE
    inp = wl.host_inputs(cfg)
    d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    c = tri.SpecCache(auto_install=True, resident_args=True)
    try:
        p = c.prepare("decode_chain", d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                      d["gate"], d["up"], cfg.eps, cfg.base)
        y, ro, out = p.result
        for step in range(5):
            new = wl.host_inputs(cfg, seed=800 + step)
            for k in ("x", "residual", "w", "q", "k", "pos", "gate", "up"):
                d[k].copy_(wl.to_torch(new[k], cfg.dtype, DEV))
            torch.cuda.synchronize()
            p()
            torch.cuda.synchronize()
            want = O.decode_chain(new, cfg.eps, cfg.base, cfg.dtype)
            for n, t in (("y", y), ("out", out), ("q", d["q"]), ("k", d["k"])):
                check(f"step {step} {n}", host(t), want[n], cfg.dtype)
            check(f"step {step} res_out", host(ro), want["res_out"], cfg.dtype, exact=True)
        assert c.resident_info() == {"enabled": 1, "held": 1, "launches": 5}
    finally:
        torch.cuda.synchronize()
        c.close()


def test_prepare_refuses_what_is_not_one_op_call(tri):
    c = tri.SpecCache()
    x = torch.zeros((1, 64), device=DEV)
    w = torch.ones(64, device=DEV)
    try:
        for bad in ("close", "prepare", "_call", "stats", "no_such_op"):
            with pytest.raises(ValueError):
                c.prepare(bad)
        p = c.prepare("rmsnorm", x, w, 1e-6)
        assert c.stats()["calls"] == 0                  # preparing launches nothing
        with pytest.raises(ValueError):                 # checks run once, at prepare
            c.prepare("rmsnorm", x, torch.ones(63, device=DEV), 1e-6)
    finally:
        torch.cuda.synchronize()
        c.close()
    with pytest.raises(tri.TriError):                   # the cache is gone
        p()
