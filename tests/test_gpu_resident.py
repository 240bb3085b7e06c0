"""GPU: launches from resident argument blocks (TRI_CACHE_RESIDENT_ARGS) --
the fused chain, the three-launch chain and every standalone op -- against
the ordinary launches and the CPU oracle.

A resident launch takes no kernel arguments and finds its block in the
device's table of its kernel family through its LDS allocation; its outputs
must equal an ordinary launch's bit for bit and the oracle's, follow the
data behind the held pointers on every call, and stay right when a slot is
rewritten for another cache or a hit is replayed from a graph.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
from tests.parity import binding_rope_ext, check
from tests.test_gpu_parity import CHAIN_CFGS, DEV, MEDIUM, chain_oracle, host
import workloads as wl

pytestmark = pytest.mark.gpu
SLOTS = 40


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


def make_cache(tri, **kw):
    return tri.SpecCache(auto_install=True, **kw)


def device_inputs(cfg, seed=None):
    inp = wl.host_inputs(cfg) if seed is None else wl.host_inputs(cfg, seed=seed)
    d = {k: wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
    d["y"], d["res_out"] = torch.empty_like(d["x"]), torch.empty_like(d["x"])
    d["out"] = torch.empty_like(d["gate"])
    return inp, d


def args_of(tri, cache, cfg, d):
    rope = binding_rope_ext(tri, cfg.rope_ext) if cfg.rope_ext else None
    a, _ = cache.chain_args(d["x"], d["residual"], d["w"], d["q"], d["k"], d["pos"], d["gate"],
                            d["up"], cfg.eps, cfg.base, y=d["y"], residual_out=d["res_out"],
                            out=d["out"], q_norm_w=d.get("q_norm_w"),
                            k_norm_w=d.get("k_norm_w"), rope=rope)
    return a


def same_outputs(tag, a, b, dtype):
    for n in ("y", "res_out", "q", "k", "out"):
        check(f"{tag} {n}", host(a[n]), host(b[n]), dtype, exact=True)


def test_the_device_passes_the_lds_channel_check(tri):
    c = make_cache(tri, resident_args=True)
    try:
        assert c.resident_info() == {"enabled": 1, "held": 0, "launches": 0}
    finally:
        c.close()


@pytest.mark.parametrize("cfg", CHAIN_CFGS + MEDIUM, ids=lambda c: c.name)
def test_resident_chain_equals_ordinary_and_oracle(tri, cfg):
    """Decode sizes and 65-301 tokens (grids beyond 512 workgroups take one
    of the first ten slots)."""
    inp, a = device_inputs(cfg)
    b = {k: v.clone() for k, v in a.items()}
    q0, k0 = a["q"].clone(), a["k"].clone()
    plain, res = make_cache(tri), make_cache(tri, resident_args=True)
    try:
        aa, ab = args_of(tri, plain, cfg, a), args_of(tri, res, cfg, b)
        for call in range(3):
            if call:
                for d in (a, b):                      # undo the in-place rotation
                    d["q"].copy_(q0)
                    d["k"].copy_(k0)
            plain.decode_chain_args(aa)
            res.decode_chain_args(ab)
            torch.cuda.synchronize()
            same_outputs(f"call {call}", b, a, cfg.dtype)
            assert res.last_selection().as_tuple() == plain.last_selection().as_tuple()
        n = res.last_selection().n_launches          # fused, or three launches
        assert res.resident_info() == {"enabled": 1, "held": n, "launches": 3 * n}
        assert plain.resident_info()["launches"] == 0
        want = chain_oracle(inp, cfg)
        for n in ("y", "q", "k", "out"):
            check(n, host(b[n]), want[n], cfg.dtype)
        check("res_out", host(b["res_out"]), want["res_out"], cfg.dtype, exact=True)
    finally:
        torch.cuda.synchronize()
        plain.close()
        res.close()


def test_resident_blocks_read_new_data_on_every_call(tri):
    """Only pointers are held: new positions, activations and weights written
    into the same tensors give the oracle's result for the new data."""
    cfg = wl.LLAMA7B_DECODE
    _, d = device_inputs(cfg)
    c = make_cache(tri, resident_args=True)
    try:
        a = args_of(tri, c, cfg, d)
        for step in range(5):
            inp = wl.host_inputs(cfg, seed=500 + step)
            for k in ("x", "residual", "w", "q", "k", "pos", "gate", "up"):
                d[k].copy_(wl.to_torch(inp[k], cfg.dtype, DEV))
            torch.cuda.synchronize()
            c.decode_chain_args(a)
            torch.cuda.synchronize()
            want = O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)
            for n in ("y", "q", "k", "out"):
                check(f"step {step} {n}", host(d[n]), want[n], cfg.dtype)
            check(f"step {step} res_out", host(d["res_out"]), want["res_out"], cfg.dtype,
                  exact=True)
        assert c.resident_info() == {"enabled": 1, "held": 1, "launches": 5}
    finally:
        torch.cuda.synchronize()
        c.close()


def _layer_stack(tri, cache, cfg, n, seed):
    """n dependent layers (layer l + 1 reads layer l's residual output)."""
    layers, args = [], []
    prev = None
    for l in range(n):
        _, d = device_inputs(cfg, seed=seed + l)
        if prev is not None:
            d["residual"] = prev
        args.append(args_of(tri, cache, cfg, d))
        layers.append(d)
        prev = d["res_out"]
    return layers, args


def test_more_layers_than_slots_match_ordinary_layers(tri):
    """45 layers: the first 40 blocks are held, the last 5 launch with kernel
    arguments; two steps, every output equal to an ordinary cache's."""
    cfg = wl.GQA_DECODE
    n = SLOTS + 5
    plain, res = make_cache(tri), make_cache(tri, resident_args=True)
    try:
        la, aa = _layer_stack(tri, plain, cfg, n, 700)
        lb, ab = _layer_stack(tri, res, cfg, n, 700)
        for step in range(2):
            if step:
                for l in range(n):
                    fresh = wl.host_inputs(cfg, seed=900 + l)
                    for k in ("x", "q", "k", "gate", "up"):
                        src = wl.to_torch(fresh[k], cfg.dtype, DEV)
                        la[l][k].copy_(src)
                        lb[l][k].copy_(src)
                torch.cuda.synchronize()
            plain.decode_chain_layers(aa)
            res.decode_chain_layers(ab)
            torch.cuda.synchronize()
            for l in range(n):
                same_outputs(f"step {step} layer {l}", lb[l], la[l], cfg.dtype)
        info = res.resident_info()
        assert info["held"] == SLOTS and info["launches"] == 2 * SLOTS
    finally:
        torch.cuda.synchronize()
        plain.close()
        res.close()


def test_a_freed_slot_serves_another_cache(tri):
    """Cache A holds slot blocks for its buffers and is destroyed; cache B's
    block is then written into a freed slot: B's outputs are B's data's."""
    cfg = wl.LLAMA7B_DECODE
    inp_a, da = device_inputs(cfg, seed=41)
    inp_b, db = device_inputs(cfg, seed=42)
    a_cache = make_cache(tri, resident_args=True)
    a_cache.decode_chain_args(args_of(tri, a_cache, cfg, da))
    torch.cuda.synchronize()
    assert a_cache.resident_info()["launches"] == 1
    a_cache.close()
    b_cache = make_cache(tri, resident_args=True)
    try:
        b_cache.decode_chain_args(args_of(tri, b_cache, cfg, db))
        torch.cuda.synchronize()
        assert b_cache.resident_info() == {"enabled": 1, "held": 1, "launches": 1}
        want = O.decode_chain(inp_b, cfg.eps, cfg.base, cfg.dtype)
        for n in ("y", "q", "k", "out"):
            check(n, host(db[n]), want[n], cfg.dtype)
        want_a = O.decode_chain(inp_a, cfg.eps, cfg.base, cfg.dtype)
        for n in ("y", "out"):
            check(f"A {n}", host(da[n]), want_a[n], cfg.dtype)
    finally:
        torch.cuda.synchronize()
        b_cache.close()


def test_resident_hit_replays_from_a_hip_graph(tri):
    """A hit on a held block captured in a graph: replays, with eager work
    and synchronisations in between, equal direct ordinary calls on twin
    buffers bit for bit. A block first seen under capture is not written
    (the captured launch carries its arguments)."""
    cfg = wl.LLAMA7B_DECODE
    _, A = device_inputs(cfg)
    B = {k: v.clone() for k, v in A.items()}
    _, C2 = device_inputs(cfg, seed=77)
    res, plain = make_cache(tri, resident_args=True), make_cache(tri)
    try:
        args_a, args_b = args_of(tri, res, cfg, A), args_of(tri, plain, cfg, B)
        args_c = args_of(tri, res, cfg, C2)
        q0, k0 = A["q"].clone(), A["k"].clone()
        res.decode_chain_args(args_a)              # holds A's block
        plain.decode_chain_args(args_b)            # installs the ordinary version
        torch.cuda.synchronize()
        for d in (A, B):
            d["q"].copy_(q0)
            d["k"].copy_(k0)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            res.decode_chain_args(args_a, stream=torch.cuda.current_stream())
            res.decode_chain_args(args_c, stream=torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert res.resident_info()["held"] == 1    # C2's block was not written
        check("q before replay", host(A["q"]), host(B["q"]), cfg.dtype, exact=True)
        for step in range(4):
            for d in (A, B):
                d["x"].mul_(0.5).add_(0.25)
            torch.cuda.synchronize()
            g.replay()
            plain.decode_chain_args(args_b)
            torch.cuda.synchronize()
            same_outputs(f"replay {step}", A, B, cfg.dtype)
    finally:
        torch.cuda.synchronize()
        res.close()
        plain.close()


# ---- the standalone ops and the three-launch chain -----------------------------------
def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _out(d, name, like):
    """Output tensor `name` of d, allocated on first use: calls reuse it, so
    a cache sees the same argument block every time."""
    if name not in d:
        d[name] = torch.empty_like(like)
    return d[name]


def _op_case(name, seed):
    """(host inputs, oracle outputs, runner) of one standalone op call. The
    runner takes a cache and device copies of the inputs (outputs kept in the
    same dict) and returns the device outputs by name (in-place outputs
    included)."""
    r = rng(seed)
    bf, f32 = nm.BF16, nm.F32
    if name in ("rmsnorm_bf16", "rmsnorm_f32_1024x128", "rmsnorm_wide_bf16"):
        dt, T, H = {"rmsnorm_bf16": (bf, 1, 4096), "rmsnorm_f32_1024x128": (f32, 1024, 128),
                    "rmsnorm_wide_bf16": (bf, 2, 57344)}[name]
        h = {"x": wl.host_array(r, (T, H), dt), "w": wl.host_weight(r, H, dt)}
        want = {"y": O.rmsnorm(h["x"], h["w"], 1e-6, dt)}
        return dt, h, want, lambda c, d: {
            "y": c.rmsnorm(d["x"], d["w"], 1e-6, out=_out(d, "y", d["x"]))}
    if name in ("residual_bf16", "residual_split_bf16"):
        T, H = (4, 8192) if name == "residual_bf16" else (2, 65536)
        h = {"x": wl.host_array(r, (T, H), bf), "r": wl.host_array(r, (T, H), bf),
             "w": wl.host_weight(r, H, bf)}
        y, ro = O.residual_rmsnorm(h["x"], h["r"], h["w"], 1e-6, bf)

        def run(c, d):
            y_, ro_ = c.residual_rmsnorm(d["x"], d["r"], d["w"], 1e-6, out=_out(d, "y", d["x"]),
                                         residual_out=_out(d, "ro", d["x"]))
            return {"y": y_, "res_out": ro_}
        return bf, h, {"y": y, "res_out": ro}, run
    if name in ("rope_bf16", "qk_norm_rope_bf16"):
        T, nq, nk, hd = 2, 32, 8, 128
        pos = r.integers(0, 8192, size=T).astype(np.int32)
        h = {"q": wl.host_array(r, (T, nq, hd), bf), "k": wl.host_array(r, (T, nk, hd), bf),
             "pos": pos}
        if name == "rope_bf16":
            q, k = O.rope_qk(h["q"], h["k"], pos, 5e5, bf)

            def run(c, d):
                c.rope_qk(d["q"], d["k"], d["pos"], 5e5)
                return {"q": d["q"], "k": d["k"]}
        else:
            h["qw"], h["kw"] = wl.host_weight(r, hd, bf), wl.host_weight(r, hd, bf)
            q, k = O.qk_norm_rope(h["q"], h["k"], pos, 1e6, h["qw"], h["kw"], 1e-6, bf)

            def run(c, d):
                c.qk_norm_rope(d["q"], d["k"], d["pos"], d["qw"], d["kw"], 1e6, 1e-6)
                return {"q": d["q"], "k": d["k"]}
        return bf, h, {"q": q, "k": k}, run
    if name == "swiglu_bf16":
        h = {"g": wl.host_array(r, (1, 11008), bf), "u": wl.host_array(r, (1, 11008), bf)}
        return bf, h, {"out": O.swiglu(h["g"], h["u"], bf)}, \
            lambda c, d: {"out": c.swiglu(d["g"], d["u"], out=_out(d, "o", d["g"]))}
    if name == "silu_bf16":
        h = {"a": wl.host_array(r, (1, 4096), bf, outliers=True)}
        return bf, h, {"out": O.silu(h["a"], bf)}, \
            lambda c, d: {"out": c.silu(d["a"], out=_out(d, "o", d["a"]))}
    if name == "add_f32":
        h = {"a": wl.host_array(r, (2, 4096), f32), "b": wl.host_array(r, (2, 4096), f32)}
        return f32, h, {"out": O.add(h["a"], h["b"], f32)}, \
            lambda c, d: {"out": c.add(d["a"], d["b"], out=_out(d, "o", d["a"]))}
    if name == "masked_fill_bf16":
        h = {"a": wl.host_array(r, (2, 4096), bf),
             "m": (r.random((2, 4096)) < 0.3).astype(np.uint8)}
        return bf, h, {"out": O.masked_fill(h["a"], h["m"], -1e4, bf)}, \
            lambda c, d: {"out": c.masked_fill(d["a"], d["m"], -1e4, out=_out(d, "o", d["a"]))}
    if name == "embedding_bf16":
        h = {"t": wl.host_array(r, (4000, 4096), bf),
             "ids": r.integers(-2, 4002, size=8).astype(np.int32)}
        return bf, h, {"out": O.embedding(h["t"], h["ids"], bf)}, \
            lambda c, d: {"out": c.embedding(
                d["t"], d["ids"], out=_out(d, "o", torch.empty((8, 4096), dtype=d["t"].dtype,
                                                                device=DEV)))}
    raise ValueError(name)


OPS = ["rmsnorm_bf16", "rmsnorm_f32_1024x128", "rmsnorm_wide_bf16", "residual_bf16",
       "residual_split_bf16", "rope_bf16", "qk_norm_rope_bf16", "swiglu_bf16", "silu_bf16",
       "add_f32", "masked_fill_bf16", "embedding_bf16"]
EXACT = {"res_out", "out"}   # outputs the oracle fixes bit for bit (silu's aside)


def _to_device(h, dt):
    out = {}
    for k, v in h.items():
        if k in ("pos", "ids", "m"):
            out[k] = torch.from_numpy(v).to(DEV)
        else:
            out[k] = wl.to_torch(v, dt, DEV)
    return out


@pytest.mark.parametrize("name", OPS)
def test_resident_standalone_op_equals_ordinary_and_oracle(tri, name):
    """Three calls on each cache with the same inputs: the resident cache's
    outputs equal the ordinary cache's bit for bit and the oracle's."""
    dt, h, want, run = _op_case(name, seed=len(name) * 31)
    plain, res = make_cache(tri), make_cache(tri, resident_args=True)
    try:
        a, b = _to_device(h, dt), _to_device(h, dt)
        for call in range(3):
            for d in (a, b):                  # inputs afresh (RoPE works in place)
                for k, v in _to_device(h, dt).items():
                    d[k].copy_(v)
            ga = run(plain, a)
            gb = run(res, b)
            torch.cuda.synchronize()
            for n in want:
                check(f"{name} call {call} {n}", host(gb[n]), host(ga[n]), dt, exact=True)
            assert res.last_selection().as_tuple()[3:] == plain.last_selection().as_tuple()[3:]
        info = res.resident_info()
        # the plain wide-row norm has no argument-free form: kernel arguments
        held = 0 if name == "rmsnorm_wide_bf16" else 1
        assert info["held"] == held and info["launches"] == 3 * held, info
        for n, w in want.items():
            exact = n in EXACT and name != "silu_bf16"
            check(f"{name} {n} vs oracle", host(gb[n]), w, dt, exact=exact)
    finally:
        torch.cuda.synchronize()
        plain.close()
        res.close()


def test_resident_three_launch_chain(tri):
    """An unaligned GQA chain runs three launches (norm, RoPE, SwiGLU): each
    from its family's resident table, outputs equal to the ordinary cache's
    and the oracle's."""
    cfg = wl.GQA_DECODE
    inp = wl.host_inputs(cfg)
    from tests.test_gpu_parity import empty_like_layout, place

    def dev_inputs():
        d = {k: place(v, cfg.dtype, "unaligned") if k not in ("w", "pos") else
             wl.to_torch(v, cfg.dtype, DEV) for k, v in inp.items()}
        d["y"], d["res_out"], d["out"] = (empty_like_layout(d["x"]), empty_like_layout(d["x"]),
                                          empty_like_layout(d["gate"]))
        return d
    a, b = dev_inputs(), dev_inputs()
    plain, res = make_cache(tri), make_cache(tri, resident_args=True)
    try:
        plain.decode_chain_args(args_of(tri, plain, cfg, a))
        res.decode_chain_args(args_of(tri, res, cfg, b))
        torch.cuda.synchronize()
        assert res.last_selection().n_launches == 3
        assert res.resident_info() == {"enabled": 1, "held": 3, "launches": 3}
        same_outputs("three launches", b, a, cfg.dtype)
        want = O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)
        for n in ("y", "q", "k", "out"):
            check(n, host(b[n]), want[n], cfg.dtype)
        check("res_out", host(b["res_out"]), want["res_out"], cfg.dtype, exact=True)
    finally:
        torch.cuda.synchronize()
        plain.close()
        res.close()


def test_captured_step_of_held_blocks_replays_like_direct_calls(tri):
    """A decode step whose layers' blocks are held, captured with
    tri_graph_build_layers: every replay (new data, same pointers) equals an
    ordinary cache's direct call on twin buffers bit for bit, and its first
    layer the oracle."""
    cfg = wl.GQA_DECODE
    n = 4
    plain, res = make_cache(tri), make_cache(tri, resident_args=True)
    graph = None
    try:
        la, aa = _layer_stack(tri, plain, cfg, n, 1300)
        lb, ab = _layer_stack(tri, res, cfg, n, 1300)
        res.decode_chain_layers(ab)                  # holds the four blocks
        torch.cuda.synchronize()
        graph = res.build_graph(ab)
        assert graph.launch_count == n
        for rep in range(3):
            fresh = [wl.host_inputs(cfg, seed=1400 + 10 * rep + l) for l in range(n)]
            for l in range(n):
                for k in ("x", "q", "k", "gate", "up") + (("residual",) if l == 0 else ()):
                    src = wl.to_torch(fresh[l][k], cfg.dtype, DEV)
                    la[l][k].copy_(src)
                    lb[l][k].copy_(src)
            torch.cuda.synchronize()
            graph.launch()
            plain.decode_chain_layers(aa)
            torch.cuda.synchronize()
            for l in range(n):
                same_outputs(f"replay {rep} layer {l}", lb[l], la[l], cfg.dtype)
            want = O.decode_chain({k: fresh[0][k] for k in ("x", "residual", "q", "k", "gate",
                                                             "up")}
                                  | {"w": host(lb[0]["w"]), "pos": host(lb[0]["pos"])},
                                  cfg.eps, cfg.base, cfg.dtype)
            for nme in ("out", "q", "y"):
                check(f"replay {rep} {nme}[0] vs oracle", host(lb[0][nme]), want[nme], cfg.dtype)
        assert res.resident_info()["held"] == n
    finally:
        torch.cuda.synchronize()
        if graph is not None:
            graph.close()
        plain.close()
        res.close()


def test_one_resident_cache_on_two_streams(tri):
    """Calls alternate between two streams (two buffer sets, one held block
    each, the second written while the first stream's launches may still
    run); every chain matches the oracle."""
    cfg = wl.LLAMA7B_DECODE
    streams = [torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV)]
    c = make_cache(tri, resident_args=True)
    try:
        sets = []
        for i, s in enumerate(streams):
            inp, d = device_inputs(cfg, seed=1500 + i)
            sets.append((inp, d, d["q"].clone(), d["k"].clone(), args_of(tri, c, cfg, d), s))
        torch.cuda.synchronize()
        for it in range(100):
            for inp, d, q0, k0, a, s in sets:
                with torch.cuda.stream(s):
                    d["q"].copy_(q0)
                    d["k"].copy_(k0)
                c.decode_chain_args(a, stream=s)
        torch.cuda.synchronize()
        for inp, d, q0, k0, a, s in sets:
            want = O.decode_chain(inp, cfg.eps, cfg.base, cfg.dtype)
            for n in ("y", "q", "k", "out"):
                check(n, host(d[n]), want[n], cfg.dtype)
            check("res_out", host(d["res_out"]), want["res_out"], cfg.dtype, exact=True)
        assert c.resident_info() == {"enabled": 1, "held": 2, "launches": 200}
    finally:
        torch.cuda.synchronize()
        c.close()


def test_captured_step_of_new_blocks_carries_arguments(tri):
    """A step captured before any of its blocks is held: the capture writes
    no block (its launches carry their arguments), the replays equal direct
    ordinary calls, and later direct calls then hold the blocks."""
    cfg = wl.GQA_DECODE
    n = 3
    plain, res = make_cache(tri), make_cache(tri, resident_args=True)
    graph = None
    try:
        la, aa = _layer_stack(tri, plain, cfg, n, 1600)
        lb, ab = _layer_stack(tri, res, cfg, n, 1600)
        graph = res.build_graph(ab)                  # installs, then captures
        assert res.resident_info()["held"] == 0
        for rep in range(2):
            fresh = [wl.host_inputs(cfg, seed=1700 + 10 * rep + l) for l in range(n)]
            for l in range(n):
                for k in ("x", "q", "k", "gate", "up") + (("residual",) if l == 0 else ()):
                    src = wl.to_torch(fresh[l][k], cfg.dtype, DEV)
                    la[l][k].copy_(src)
                    lb[l][k].copy_(src)
            torch.cuda.synchronize()
            graph.launch()
            plain.decode_chain_layers(aa)
            torch.cuda.synchronize()
            for l in range(n):
                same_outputs(f"replay {rep} layer {l}", lb[l], la[l], cfg.dtype)
        want = O.decode_chain({k: fresh[0][k] for k in ("x", "residual", "q", "k", "gate", "up")}
                              | {"w": host(lb[0]["w"]), "pos": host(lb[0]["pos"])},
                              cfg.eps, cfg.base, cfg.dtype)
        check("out[0] vs oracle", host(lb[0]["out"]), want["out"], cfg.dtype)
        assert res.resident_info()["held"] == 0
        res.decode_chain_layers(ab)                  # outside a capture: held now
        torch.cuda.synchronize()
        assert res.resident_info()["held"] == n
    finally:
        torch.cuda.synchronize()
        if graph is not None:
            graph.close()
        plain.close()
        res.close()


def test_mixed_stream_from_resident_blocks(tri):
    """All 10,000 calls of the mixed stream (1-512 tokens, two dtypes, odd
    layouts) on a resident cache: every selection record against the
    oracle's model, outputs against the oracle every 50th call and on every
    miss; nearly every launch takes a held block."""
    from oracle import selection as S
    from tests.test_gpu_parity import _mixed_stream_on_gpu
    c = tri.SpecCache(resident_args=True)
    try:
        _mixed_stream_on_gpu(tri, c, S.SpecCacheModel())
        info = c.resident_info()
        assert info["enabled"] == 1 and info["launches"] > 9000, info
    finally:
        torch.cuda.synchronize()
        c.close()
