"""The allocation-free FFN entry point (promoe_expert_ffn_noalloc) through the
C ABI: its outputs must equal promoe_expert_ffn's on the same routing, on
consecutive calls whose second step is smaller than the first (the scratch
array keeps the previous call's contents), and it must refuse steps beyond its
limits before any device work."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import parity_util as pu  # noqa: E402
from synth import configs, model as sm  # noqa: E402

from paper_2410_22134_amd import PromoeError  # noqa: E402
from paper_2410_22134_amd.model import SyntheticModel  # noqa: E402
from paper_2410_22134_amd.stack import Stack  # noqa: E402

CASES = [
    # name, config, token counts of consecutive calls (largest first)
    ("small_bf16", pu.SMALL, (8, 2)),
    ("small_int4", pu.SMALL.with_(weight_format="int4"), (13, 3)),
    ("deepseek16b_2layers", configs.C2.with_(n_layers=2), (8, 1)),
]


def _log(*a):
    print(*a, flush=True)


def _layer_outputs(m, sts, plan, noalloc):
    """route -> FFN (either entry point) for each (layer, T) of the plan; returns the y's and ids."""
    out = []
    for l, T, x in plan:
        st = sts[T]
        st.x.copy_(x)
        m.ctx.route(l, st.x, T, st.ids, st.w, st.s)
        ffn = m.ctx.expert_ffn_noalloc if noalloc else m.ctx.expert_ffn
        ffn(l, st.x, T, st.ids, st.w, st.s, st.y)
        torch.cuda.synchronize()
        out.append(tuple(pu.to_np(t).copy() for t in (st.y, st.ids, st.w, st.s)))
    return out


@pytest.mark.parametrize("name,cfg,Ts", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_expert_ffn(name, cfg, Ts):
    m = SyntheticModel(cfg, max_tokens=max(Ts))
    try:
        sts = {T: Stack(m, T) for T in Ts}
        xs = {}
        plan = []
        for T in Ts:                   # every layer at the larger step, then every layer at the smaller
            for l in range(cfg.n_layers):
                x = sm.layer_input(cfg, l, T, tag=1200 + T)
                xs[(l, T)] = x
                plan.append((l, T, torch.from_numpy(x.view(np.int16)).cuda()))
        ref = _layer_outputs(m, sts, plan, noalloc=False)
        m.open()                       # same warm cache: the same plans in the same order
        got = _layer_outputs(m, sts, plan, noalloc=True)
        for (l, T, _), r, g in zip(plan, ref, got):
            _log("noalloc", name, "layer", l, "T", T)
            for u, v in zip(r[1:], g[1:]):
                assert np.array_equal(u, v)          # same routing on both runs
            yr, yg = pu.f64(r[0], cfg.dtype), pu.f64(g[0], cfg.dtype)
            pu.check_bf16_output(yg, yr, ("noalloc vs expert_ffn", name, l, T))
            assert np.array_equal(r[0], g[0]), (name, l, T)   # the same kernels: bit for bit
            # and the oracle's bar on the allocation-free output itself
            x64 = pu.f64(xs[(l, T)], cfg.dtype)
            rec = pu.LayerRecord()
            rec.ids, rec.w, rec.s, rec.y = g[1], g[2], g[3], g[0]
            g_ids, w_ref, s_ref, _ = pu.check_route(cfg, m, l, x64, rec)
            pu.check_ffn(cfg, m, l, x64, g_ids, w_ref, s_ref, g[0])
    finally:
        m.close()


def test_noalloc_refuses_steps_beyond_its_limits():
    # more than 64 routed pairs: refused, and the pending route is still
    # consumed by promoe_expert_ffn
    cfg, T = pu.SMALL, 40
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        st.x.copy_(torch.from_numpy(sm.layer_input(cfg, 0, T, tag=1300).view(np.int16)).cuda())
        m.ctx.route(0, st.x, T, st.ids, st.w, st.s)
        with pytest.raises(PromoeError) as e:
            m.ctx.expert_ffn_noalloc(0, st.x, T, st.ids, st.w, st.s, st.y)
        assert e.value.code == -1
        m.ctx.expert_ffn(0, st.x, T, st.ids, st.w, st.s, st.y)
        m.ctx.sync()
    finally:
        m.close()
    # 64 pairs whose shared-expert activations alone fill the 8 MiB: refused
    # (the context is then closed with its route pending)
    cfg, T = pu.SMALL.with_(name="wide_shared", n_layers=1, top_k=1, shared_inter=65536), 64
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        st.x.copy_(torch.from_numpy(sm.layer_input(cfg, 0, T, tag=1301).view(np.int16)).cuda())
        m.ctx.route(0, st.x, T, st.ids, st.w, st.s)
        with pytest.raises(PromoeError) as e:
            m.ctx.expert_ffn_noalloc(0, st.x, T, st.ids, st.w, st.s, st.y)
        assert e.value.code == -1 and "scratch" in str(e.value)
        m.ctx.sync()
    finally:
        m.close()
