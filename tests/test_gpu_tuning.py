"""GPU checks of install-time tuning: every candidate plan of a key computes
the oracle's result, and tuned caches (timed, stored, compiled) do too.

Each case prints its name and candidate before touching the GPU. Inputs come
from the seeded generators in `workloads`; expected values only from
`oracle`.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
from oracle import selection as S
from tests.parity import binding_rope_ext, check, oracle_rope_kw
from tests.test_gpu_parity import CHAIN_CFGS, MEDIUM, host, rng
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


def say(*a):
    print(*a, flush=True)


# ---- cases: host inputs, a run through a cache, the oracle's outputs -------------------
class ChainCase:
    def __init__(self, cfg):
        self.cfg = cfg
        self.name = cfg.name

    def host(self):
        return wl.host_inputs(self.cfg)

    def run(self, tri, cache, inp):
        cfg = self.cfg
        d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
        rope = binding_rope_ext(tri, cfg.rope_ext) if cfg.rope_ext else None
        y, ro, out = cache.decode_chain(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"],
                                        d["gate"], d["up"], cfg.eps, cfg.base,
                                        q_norm_w=d.get("q_norm_w"), k_norm_w=d.get("k_norm_w"),
                                        rope=rope)
        return dict(y=y, res_out=ro, out=out, q=d["q"], k=d["k"])

    def oracle(self, inp):
        cfg = self.cfg
        if cfg.rope_ext:
            inp = dict(inp, rope_ext=oracle_rope_kw(cfg.rope_ext))
        return O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)

    dtype = property(lambda self: self.cfg.dtype)
    exact = ("res_out",)


class NormCase:
    def __init__(self, dtype, T, H, res):
        self.dtype, self.T, self.H, self.res = dtype, T, H, res
        self.name = f"{'res_' if res else ''}rmsnorm-{dtype}-{T}x{H}"
        self.exact = ("res_out",)

    def host(self):
        r = rng(self.T * 131 + self.H)
        return dict(x=wl.host_array(r, (self.T, self.H), self.dtype),
                    r=wl.host_array(r, (self.T, self.H), self.dtype),
                    w=wl.host_weight(r, self.H, self.dtype))

    def run(self, tri, cache, inp):
        d = {k: wl.to_torch(v, self.dtype, DEV) for k, v in inp.items()}
        if self.res:
            y, ro = cache.residual_rmsnorm(d["x"], d["r"], d["w"], 1e-6)
            return dict(y=y, res_out=ro)
        return dict(y=cache.rmsnorm(d["x"], d["w"], 1e-6))

    def oracle(self, inp):
        if self.res:
            y, h = O.residual_rmsnorm(inp["x"], inp["r"], inp["w"], 1e-6, self.dtype)
            return dict(y=y, res_out=h)
        return dict(y=O.rmsnorm(inp["x"], inp["w"], 1e-6, self.dtype))


class RopeCase:
    def __init__(self, dtype, T, nq, nk, hd, base, ext=None, qkn=False):
        self.dtype, self.T, self.nq, self.nk, self.hd, self.base = dtype, T, nq, nk, hd, base
        self.ext, self.qkn = ext, qkn
        self.name = f"{'qkn_' if qkn else ''}rope-{dtype}-{T}-{nq}x{nk}x{hd}-{ext or 'plain'}"
        self.exact = ()

    def host(self):
        r = rng(self.T * 7 + self.nq * 13 + self.hd)
        return dict(q=wl.host_array(r, (self.T, self.nq, self.hd), self.dtype),
                    k=wl.host_array(r, (self.T, self.nk, self.hd), self.dtype),
                    pos=r.integers(0, 8192, size=self.T).astype(np.int32),
                    qw=wl.host_weight(r, self.hd, self.dtype),
                    kw=wl.host_weight(r, self.hd, self.dtype))

    def run(self, tri, cache, inp):
        d = {k: wl.to_torch(v, self.dtype, DEV) for k, v in inp.items()}
        kd = d["k"] if self.nk else None
        cache.rope(d["q"], kd, d["pos"], self.base,
                   ext=binding_rope_ext(tri, self.ext) if self.ext else None,
                   q_w=d["qw"] if self.qkn else None, k_w=d["kw"] if self.qkn else None)
        return dict(q=d["q"], k=d["k"]) if self.nk else dict(q=d["q"])

    def oracle(self, inp):
        kw = oracle_rope_kw(self.ext)
        if self.qkn:
            kw.update(q_w=inp["qw"], k_w=inp["kw"], eps=1e-6)
        wq, wk = O.rope_ext(inp["q"], inp["k"], inp["pos"], self.base, self.dtype, **kw)
        return dict(q=wq, k=wk) if self.nk else dict(q=wq)


class EltCase:
    def __init__(self, op, dtype, T, W):
        self.op, self.dtype, self.T, self.W = op, dtype, T, W
        self.name = f"{op}-{dtype}-{T}x{W}"
        self.exact = ("out",) if op != "silu" and op != "swiglu" else ()

    def host(self):
        r = rng(self.T * 17 + self.W + len(self.op))
        return dict(a=wl.host_array(r, (self.T, self.W), self.dtype, outliers=True),
                    b=wl.host_array(r, (self.T, self.W), self.dtype),
                    m=(r.random((self.T, self.W)) < 0.3).astype(np.uint8))

    def run(self, tri, cache, inp):
        a = wl.to_torch(inp["a"], self.dtype, DEV)
        b = wl.to_torch(inp["b"], self.dtype, DEV)
        if self.op == "silu":
            return dict(out=cache.silu(a))
        if self.op == "add":
            return dict(out=cache.add(a, b))
        if self.op == "swiglu":
            return dict(out=cache.swiglu(a, b))
        return dict(out=cache.masked_fill(a, torch.from_numpy(inp["m"]).to(DEV), -1e4))

    def oracle(self, inp):
        if self.op == "silu":
            return dict(out=O.silu(inp["a"], self.dtype))
        if self.op == "add":
            return dict(out=O.add(inp["a"], inp["b"], self.dtype))
        if self.op == "swiglu":
            return dict(out=O.swiglu(inp["a"], inp["b"], self.dtype))
        return dict(out=O.masked_fill(inp["a"], inp["m"], -1e4, self.dtype))


CASES = ([ChainCase(c) for c in CHAIN_CFGS + MEDIUM]
         + [NormCase(d, T, H, res) for (d, T, H) in
            ((nm.BF16, 9, 512), (nm.F32, 5, 256), (nm.BF16, 13, 1024), (nm.BF16, 6, 4096),
             (nm.BF16, 3, 32768), (nm.F32, 67, 16384)) for res in (False, True)]
         + [RopeCase(nm.BF16, 8, 32, 8, 128, 5e5), RopeCase(nm.F32, 19, 4, 4, 64, 1e4),
            RopeCase(nm.BF16, 37, 32, 8, 128, 5e5), RopeCase(nm.BF16, 17, 64, 8, 128, 5e5),
            RopeCase(nm.F32, 3, 3, 0, 128, 1e4),
            RopeCase(nm.BF16, 5, 16, 16, 256, 1e4, ext=dict(rotary_dim=64, interleaved=1)),
            RopeCase(nm.F32, 6, 8, 2, 128, 5e5, ext=dict(rotary_dim=64)),
            RopeCase(nm.BF16, 5, 32, 8, 128, 1e6, qkn=True),
            RopeCase(nm.F32, 3, 4, 2, 64, 1e6, qkn=True),
            RopeCase(nm.BF16, 4, 8, 2, 128, 5e5, ext=dict(interleaved=1), qkn=True)]
         + [EltCase("swiglu", d, T, W) for (d, T, W) in
            ((nm.BF16, 1, 11008), (nm.BF16, 300, 688), (nm.F32, 130, 1000),
             (nm.BF16, 8, 14336), (nm.F32, 4, 688))]
         + [EltCase(op, d, T, W) for (op, d, T, W) in
            (("add", nm.BF16, 100, 4096), ("silu", nm.F32, 130, 1000),
             ("masked_fill", nm.BF16, 130, 4096), ("add", nm.BF16, 1, 4096),
             ("silu", nm.BF16, 100, 11008), ("masked_fill", nm.F32, 3, 1024))])


def check_all(case, outs, want, what):
    for n, t in outs.items():
        check(f"{what} {n}", host(t), want[n], case.dtype, exact=n in case.exact)


def key_of(tri, case, inp):
    """The key a call of `case` makes (read back from a scratch cache)."""
    probe = tri.SpecCache()
    try:
        case.run(tri, probe, inp)
        torch.cuda.synchronize()
        (key,) = probe.export_keys()
        assert probe.version_info(0).n_candidates == len(S.candidates(key))
        return key
    finally:
        probe.close()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_every_candidate_matches_the_oracle(tri, case):
    inp = case.host()
    key = key_of(tri, case, inp)
    want = case.oracle(inp)
    cands = S.candidates(key)
    for i, cand in enumerate(cands):
        say(f"{case.name}: candidate {i} of {len(cands)} {cand}")
        c = tri.SpecCache()
        try:
            c.install_key(key, i)
            outs = case.run(tri, c, inp)
            torch.cuda.synchronize()
            assert c.stats()["misses"] == 0
            v = c.version_info(0)
            assert (v.candidate, v.variant, v.rope_slices) == (i, cand.variant, cand.slices)
            check_all(case, outs, want, f"candidate {i}")
        finally:
            c.close()


TUNED = [CASES[i] for i in (0, 1, 2, 3, 7)] + [c for c in CASES if not isinstance(c, ChainCase)]


@pytest.mark.parametrize("case", TUNED, ids=lambda c: c.name)
def test_tuned_cache_matches_the_oracle(tri, case):
    inp = case.host()
    say(f"{case.name}: autotune")
    c = tri.SpecCache(auto_install=True, autotune=True)
    try:
        outs = case.run(tri, c, inp)
        torch.cuda.synchronize()
        v = c.version_info(0)
        say(f"  kept candidate {v.candidate} of {v.n_candidates} (tuned {v.tuned}, "
            f"{v.tune_ms:.2f} ms)")
        assert v.tuned == (S.TUNE_MEASURED if v.n_candidates > 1 else S.TUNE_NONE)
        check_all(case, outs, case.oracle(inp), "tuned")
        # the tuned version serves the next call as a hit
        outs = case.run(tri, c, case.host())
        torch.cuda.synchronize()
        assert c.stats()["hits"] == 1 and c.stats()["misses"] == 1
    finally:
        c.close()


def test_stored_choice_is_reused(tri, tmp_path):
    case = ChainCase(wl.LLAMA7B_DECODE)
    inp = case.host()
    say("store: first cache times")
    a = tri.SpecCache(auto_install=True, autotune=True, code_dir=str(tmp_path))
    try:
        case.run(tri, a, inp)
        torch.cuda.synchronize()
        va = a.version_info(0)
        assert va.tuned == S.TUNE_MEASURED
    finally:
        a.close()
    files = [p.name for p in tmp_path.iterdir()]
    assert len(files) == 1 and files[0].startswith("tri-tune-")
    say("store: second cache reads")
    b = tri.SpecCache(auto_install=True, autotune=True, code_dir=str(tmp_path))
    try:
        outs = case.run(tri, b, inp)
        torch.cuda.synchronize()
        vb = b.version_info(0)
        assert (vb.tuned, vb.candidate) == (S.TUNE_STORED, va.candidate)
        check_all(case, outs, case.oracle(inp), "stored")
    finally:
        b.close()


@pytest.mark.parametrize("cfg", [wl.LLAMA7B_DECODE, wl.TINY_F32], ids=lambda c: c.name)
def test_compiled_tuned_plan_equals_the_pinned_precompiled_candidate(tri, cfg):
    case = ChainCase(cfg)
    inp = case.host()
    say(f"{cfg.name}: JIT + autotune")
    j = tri.SpecCache(auto_install=True, autotune=True, jit=True)
    p = tri.SpecCache()
    try:
        oj = case.run(tri, j, inp)
        torch.cuda.synchronize()
        v = j.version_info(0)
        assert v.jit == 1 and v.tuned == S.TUNE_MEASURED
        p.install_key(j.export_keys()[0], v.candidate)
        op = case.run(tri, p, inp)
        torch.cuda.synchronize()
        for n in oj:
            check(n, host(oj[n]), host(op[n]), cfg.dtype, exact=True)
    finally:
        torch.cuda.synchronize()
        j.close()
        p.close()


def test_tuned_plans_export_and_reinstall_without_timing(tri):
    """A tuned set of versions (keys + kept candidates) reinstalls in a cache
    without the tuning flag: same plans, nothing timed, same results."""
    say("export / import of tuned plans")
    cases = [CASES[0], CASES[1], CASES[7]] + [c for c in CASES if isinstance(c, EltCase)][:3]
    a = tri.SpecCache(auto_install=True, autotune=True)
    b = tri.SpecCache()
    try:
        inps = [c.host() for c in cases]
        outs_a = []
        for c, inp in zip(cases, inps):
            outs_a.append(c.run(tri, a, inp))
        torch.cuda.synchronize()
        plans = a.export_plans()
        assert len(plans) == len(cases)
        b.import_plans(plans)
        for i, (key, cand) in enumerate(plans):
            v = b.version_info(i)
            assert (tuple(v.key), v.candidate, v.tuned) == (tuple(key), cand, S.TUNE_NONE)
        for c, inp, oa in zip(cases, inps, outs_a):
            ob = c.run(tri, b, inp)
            torch.cuda.synchronize()
            for n in oa:
                check(n, host(ob[n]), host(oa[n]), c.dtype, exact=True)
        assert b.stats()["misses"] == 0
    finally:
        torch.cuda.synchronize()
        a.close()
        b.close()
