"""GPU edge cases through the C ABI, checked against the oracle: ragged token
counts on the MFMA path, every expert routed through a one-slot cache, reactive
mode, external pushes, and the host-side error returns."""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import parity_util as pu  # noqa: E402
from oracle import cache as ocache  # noqa: E402
from synth import configs, model as sm  # noqa: E402
from synth.configs import Workload  # noqa: E402

from paper_2410_22134_amd import ABLATION, FLAG_FILL_BY_DEADLINE, FLAG_NO_PREFETCH, FLAG_NO_REORDER, FLAG_STATIC  # noqa: E402,E501
from paper_2410_22134_amd import PRIO_HIGH, PRIO_LOW, PromoeError  # noqa: E402
from paper_2410_22134_amd import _abi  # noqa: E402
from paper_2410_22134_amd.model import SyntheticModel  # noqa: E402
from paper_2410_22134_amd.stack import Stack  # noqa: E402

SMALL = pu.SMALL


def _log(*a):
    print(*a, flush=True)


def _step_diff(i, a, b):
    """What differs between two runs' residuals after step i: the count of
    unequal elements, the largest difference and the first unequal row."""
    ne = a != b
    rows = np.nonzero(ne.any(axis=1))[0] if a.ndim == 2 else np.nonzero(ne)[0]
    return ("step", i, "unequal", int(ne.sum()), "max_abs", float(np.abs(a - b).max()),
            "first_row", int(rows[0]) if rows.size else -1)


@pytest.mark.parametrize("T", [1, 5, 13, 77, 130])
def test_ragged_token_counts(T):
    cfg = SMALL
    _log("ragged T", T)
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for l in range(cfg.n_layers):
            pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=T))
        pu.check_counters(m, lcs)
    finally:
        m.close()


def test_shared_gateup_half_height_tail_tiles():
    # A one-job gate/up launch whose 256-row tiles overrun whole rounds of the
    # 256 CUs: 2000 tokens x 40 n-tiles of the shared expert = 8 x 40 = 320
    # tiles, so 256 full tiles run and the last 8 n-tiles go in 128-row tiles,
    # the last of which holds 80 tokens.  Every row is compared.
    cfg = SMALL.with_(name="tail_tiles", shared_inter=5120, n_layers=1,
                      workloads=(Workload("prefill", 2000, 1),))
    T = 2000
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        pu.moe_layer_check(cfg, m, st, 0, None, sm.layer_input(cfg, 0, T, tag=7), predict=False)
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 40])
def test_every_expert_through_one_slot(T):
    # k = E: every expert is routed; with one slot each fill must wait for the
    # previous expert's read (deferred fills), in decode (GEMV) and prefill (GEMM)
    cfg = SMALL.with_(top_k=8, slots=1, n_layers=2)
    _log("one slot T", T)
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for step in range(2):
            for l in range(cfg.n_layers):
                pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=100 + step))
        pu.check_counters(m, lcs)
        assert m.ctx.stats()["deferred"] > 0
    finally:
        m.close()


def test_reactive_mode_matches_demand_only_lru():
    cfg = SMALL
    m = SyntheticModel(cfg, max_tokens=4, flags=FLAG_NO_PREFETCH)
    try:
        st = Stack(m, 4)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for step in range(4):
            for l in range(cfg.n_layers):
                x = sm.layer_input(cfg, l, 4, tag=200 + step)
                # predictions are computed but not acted on: replay precise plans only
                pu.moe_layer_check(cfg, m, st, l, lcs, x, predict=False)
        pu.check_counters(m, lcs)
        s = m.ctx.stats()
        assert s["spec_issued"] == 0 and s["bytes_low"] == 0
    finally:
        m.close()


@pytest.mark.parametrize("limit,T", [(1, 1), (2, 6), (-1, 3)])
def test_spec_fill_limit(limit, T):
    # predicted plans fill at most `limit` slots (-1: none); host pushes are not limited
    cfg = SMALL
    _log("spec fill limit", limit, "T", T)
    m = SyntheticModel(cfg, max_tokens=T, spec_fill_limit=limit)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        b = pu.fill_budget(limit)
        for step in range(4):
            for l in range(cfg.n_layers):
                pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=400 + step), budget=b)
        m.ctx.prefetch(0, [0, 1, 2, 3], PRIO_LOW)
        pu.check_plan_spec(lcs[0], [0, 1, 2, 3], m.ctx.last_plan(0, 0), predicted=False)
        pu.moe_layer_check(cfg, m, st, 0, lcs, sm.layer_input(cfg, 0, T, tag=499), predict=False)
        pu.check_counters(m, lcs)
        if limit < 0:
            assert m.ctx.stats(1)["spec_issued"] == 0
    finally:
        m.close()


@pytest.mark.parametrize("limit,T", [(0, 1), (2, 4), (1, 77)])
def test_fill_by_deadline(limit, T):
    # Speculative fills budgeted by the copy time left before the target route:
    # each plan records the budget it was given (host timing), and the oracle
    # replays every plan with that budget; outputs, plans and counters exact.
    cfg = SMALL
    _log("fill by deadline, limit", limit, "T", T)
    m = SyntheticModel(cfg, max_tokens=T, flags=FLAG_FILL_BY_DEADLINE, spec_fill_limit=limit)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        budgets = []
        for step in range(6):
            for l in range(cfg.n_layers):
                pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=1400 + step), budget=None)
                tgt = sm.predictor_target(cfg, l)
                if tgt is not None:
                    budgets.append(m.ctx.last_plan(tgt, 0)["fill_budget"])
        pu.check_counters(m, lcs)
        assert budgets[0] == 0                      # no route interval measured yet: no fills
        cap = limit if limit > 0 else 64
        assert all(0 <= b <= cap for b in budgets), budgets
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 77])
@pytest.mark.parametrize("mode", list(ABLATION))
def test_ablation_modes(mode, T):
    # every ablation step and the static baseline: plans, counters and outputs
    flags = ABLATION[mode]
    cfg = SMALL.with_(slots=5)
    _log("ablation", mode, "T", T)
    m = SyntheticModel(cfg, max_tokens=T, flags=flags)
    try:
        st = Stack(m, T)
        pinned = cfg.slots - 2 if flags & FLAG_STATIC else 0
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots, pinned=pinned) for l in range(cfg.n_layers)}
        predict = not flags & FLAG_NO_PREFETCH
        for step in range(3):
            for l in range(cfg.n_layers):
                pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=500 + step), predict=predict,
                                   reorder=not flags & FLAG_NO_REORDER)
        pu.check_counters(m, lcs)
        if pinned:
            for l in range(cfg.n_layers):
                assert m.ctx.slot_table(l)[:pinned] == list(range(pinned))
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 5, 13, 77])
def test_int4_experts(T):
    # 4-bit routed experts through the dequantising GEMVs (token groups of 1, 2, 4, 8)
    cfg = SMALL.with_(weight_format="int4")
    _log("int4 T", T)
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for step in range(2):
            for l in range(cfg.n_layers):
                pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=600 + step))
        pu.check_counters(m, lcs)
        assert m.ctx.stats()["bytes_high"] % cfg.chunk_bytes == 0
    finally:
        m.close()


@pytest.mark.parametrize("T", [77, 300])
def test_down_over_single_column_ranges(T):
    # hidden 384 is not a multiple of 256, so the down GEMM runs 128-column tiles
    # (the column-pair tiles need H % 256 == 0); 300 tokens use 256-row tiles
    cfg = SMALL.with_(name="h384", hidden=384, n_layers=2)
    _log("h384 T", T)
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for l in range(cfg.n_layers):
            pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=900 + T))
        pu.check_counters(m, lcs)
    finally:
        m.close()


def test_int4_prefill_long_rows():
    # 4-bit experts whose rows exceed 256 chunks of 8 weights (hidden 2304, inter
    # 2176), so the dequantising expansion loops over each row
    cfg = SMALL.with_(name="int4_long", hidden=2304, inter=2176, shared_inter=512, n_layers=2,
                      weight_format="int4")
    T = 77
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for l in range(cfg.n_layers):
            pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=950))
        pu.check_counters(m, lcs)
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 77])
def test_predict_before_or_after_route(T):
    # The layer loop predicts after the route (look-ahead >= 1), and for large
    # steps after the FFN call; predicting first fuses the gate rows into the
    # predictor pass instead.  Every order must give the same ids, weights,
    # predictions, outputs and cache plans, bit for bit (the route-first order
    # is the one the oracle checks elsewhere).
    cfg = SMALL
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        runs = []
        for when in ("first", "after_route", "after_ffn"):
            m.open()
            got = []
            for step in range(2):
                for l in range(cfg.n_layers):
                    st.x.copy_(torch.from_numpy(sm.layer_input(cfg, l, T, tag=980 + step).view(np.int16)).cuda())
                    ctx = m.ctx
                    if when == "first":
                        ctx.predict(l, st.x, T, st.pred_ids)
                    order = ctx.route(l, st.x, T, st.ids, st.w, st.s)
                    if when == "after_route":
                        ctx.predict(l, st.x, T, st.pred_ids)
                    ctx.expert_ffn(l, st.x, T, st.ids, st.w, st.s, st.y)
                    if when == "after_ffn":
                        ctx.predict(l, st.x, T, st.pred_ids)
                    torch.cuda.synchronize()
                    got.append((order, *(t.cpu().numpy().copy() for t in (st.ids, st.w, st.s, st.pred_ids, st.y)),
                                m.ctx.last_plan(l, 1)["slot"]))
            runs.append(got)
        names = ("ids", "w", "s", "pred_ids", "y")
        for mode, other in zip(("after_route", "after_ffn"), runs[1:]):
            for i, (a, b) in enumerate(zip(runs[0], other)):
                where = (mode, "step", i // cfg.n_layers, "layer", i % cfg.n_layers)
                assert a[0] == b[0] and a[6] == b[6], where
                for name, u, v in zip(names, a[1:6], b[1:6]):
                    assert np.array_equal(u, v), (where, name, int((u != v).sum()))
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 4, 77])
def test_route_and_ffn_on_different_streams(T):
    # An FFN call on another stream than its route must order itself after the
    # route's top-k and plan (ids, weights, slots, permutation).  With 77 tokens
    # over 8 experts and 4 slots every expert is routed, so each fill overwrites
    # a slot that a resident expert of the same step reads, and the route also
    # launches the first of those readers on its own stream.  At 1 and 4 tokens
    # (the GEMV path) nothing but the plan links the two streams.  Outputs, ids,
    # weights and plans must equal the one-stream run bit for bit.
    cfg = SMALL
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        runs = []
        for split in (False, True):
            m.open()
            got = []
            for step in range(2):
                for l in range(cfg.n_layers):
                    st.x.copy_(torch.from_numpy(sm.layer_input(cfg, l, T, tag=990 + step).view(np.int16)).cuda())
                    ctx = m.ctx
                    cur = torch.cuda.current_stream()
                    rs, fs = (s1, s2) if split else (cur, cur)
                    rs.wait_stream(cur)
                    fs.wait_stream(cur)
                    order = ctx.route(l, st.x, T, st.ids, st.w, st.s, stream=rs)
                    ctx.predict(l, st.x, T, st.pred_ids, stream=rs)
                    ctx.expert_ffn(l, st.x, T, st.ids, st.w, st.s, st.y, stream=fs)
                    cur.wait_stream(rs)
                    cur.wait_stream(fs)
                    torch.cuda.synchronize()
                    got.append((order, *(t.cpu().numpy().copy() for t in (st.ids, st.w, st.s, st.y)),
                                m.ctx.last_plan(l, 1)["slot"]))
            runs.append(got)
        if T == 77:
            assert len(runs[0][0][0]) == cfg.n_experts  # every expert routed: fills wait for resident reads
        for a, b in zip(*runs):
            assert a[0] == b[0] and a[5] == b[5]
            for u, v in zip(a[1:5], b[1:5]):
                assert np.array_equal(u, v)
    finally:
        m.close()


def test_external_pushes_low_and_high():
    cfg = SMALL.with_(n_layers=1, lookahead=0)
    m = SyntheticModel(cfg, max_tokens=2)
    try:
        st = Stack(m, 2)
        lc = ocache.LayerCache(cfg.n_experts, cfg.slots)
        for i, (ids, prio) in enumerate((([5, 6], PRIO_LOW), ([7, 1, 4], PRIO_HIGH), ([0], PRIO_LOW))):
            m.ctx.prefetch(0, ids, prio)
            pu.check_plan_spec(lc, ids, m.ctx.last_plan(0, 0), predicted=False)
            pu.moe_layer_check(cfg, m, st, 0, {0: lc}, sm.layer_input(cfg, 0, 2, tag=300 + i), predict=False)
        pu.check_counters(m, {0: lc})
        assert m.ctx.stats()["bytes_high"] > 0
    finally:
        m.close()


def test_error_returns():
    cfg = SMALL.with_(n_layers=1, lookahead=0)
    m = SyntheticModel(cfg, max_tokens=4)
    try:
        st = Stack(m, 4)
        ctx = m.ctx
        with pytest.raises(PromoeError) as e:
            ctx.route(0, st.x, 5, st.ids, st.w, st.s)          # T > max_tokens
        assert e.value.code == -1
        for call in (lambda: ctx.route(0, st.x, 0, st.ids, st.w, st.s),      # empty step
                     lambda: ctx.predict(0, st.x, 0, st.pred_ids),
                     lambda: ctx.attn_surrogate(0, st.h, 0, st.x),
                     lambda: ctx.residual_add(st.h, st.y, 0)):
            with pytest.raises(PromoeError) as e:
                call()
            assert e.value.code == -1
        with pytest.raises(PromoeError) as e:
            ctx.route(1, st.x, 1, st.ids, st.w, st.s)          # layer out of range
        assert e.value.code == -1
        with pytest.raises(PromoeError) as e:
            ctx.route_predict(0, st.x, 1, st.ids, st.w, st.s, st.pred_ids)  # look-ahead 0
        assert e.value.code == -1
        with pytest.raises(PromoeError) as e:
            ctx.expert_ffn(0, st.x, 1, st.ids, st.w, st.s, st.y)  # no route before
        assert e.value.code == -4
        with pytest.raises(PromoeError) as e:
            ctx.prefetch(0, [3, 3])                              # duplicate ids
        assert e.value.code == -1
        with pytest.raises(PromoeError) as e:
            ctx.prefetch(0, list(range(cfg.slots + 1)))           # more than the slots
        assert e.value.code == -1
        ctx.route(0, st.x, 1, st.ids, st.w, st.s)
        with pytest.raises(PromoeError) as e:
            ctx.route(0, st.x, 1, st.ids, st.w, st.s)           # route while one is pending
        assert e.value.code == -4
        with pytest.raises(PromoeError) as e:
            ctx.expert_ffn(0, st.x, 2, st.ids, st.w, st.s, st.y)  # T differs from the route
        assert e.value.code == -4
        ctx.expert_ffn(0, st.x, 1, st.ids, st.w, st.s, st.y)
        ctx.sync()
    finally:
        m.close()
    # unsupported shapes are refused before any device work
    c = _abi.Config()
    c.n_layers, c.hidden, c.n_experts, c.top_k, c.inter = 1, 256, 65, 2, 512
    c.slots_per_layer, c.max_tokens, c.dtype = 4, 4, _abi.PROMOE_BF16
    h = ctypes.c_void_p()
    buf = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), buf.numel(), ctypes.byref(h)) == -5
    c.n_experts, c.hidden = 8, 250
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), buf.numel(), ctypes.byref(h)) == -5
    c.hidden = 256
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), 100, ctypes.byref(h)) == -1
    c.spec_fill_limit = -2
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), buf.numel(), ctypes.byref(h)) == -1
    c.spec_fill_limit, c.flags, c.slots_per_layer = 0, FLAG_STATIC, 2   # static needs C >= 3
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), buf.numel(), ctypes.byref(h)) == -1
    c.flags, c.slots_per_layer, c.weight_format = 0, 4, _abi.WEIGHTS_INT4
    c.inter = 520                                                      # int4 needs multiples of 128
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), buf.numel(), ctypes.byref(h)) == -5
    c.weight_format, c.inter, c.pred_hidden = _abi.WEIGHTS_DENSE, 512, 60   # predictor width % 8
    assert _abi.lib().promoe_create(ctypes.byref(c), buf.data_ptr(), buf.numel(), ctypes.byref(h)) == -5


@pytest.mark.parametrize("fmt", ["dense", "int4"])
@pytest.mark.parametrize("T", [1, 4, 77])
def test_route_predict_in_one_call(T, fmt):
    # promoe_route_predict is promoe_route then promoe_predict: per-token predicted
    # ids, both plans, the counters and every output as the oracle's
    cfg = SMALL.with_(weight_format=fmt)
    _log("route_predict T", T, fmt)
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        lcs = {l: ocache.LayerCache(cfg.n_experts, cfg.slots) for l in range(cfg.n_layers)}
        for step in range(3):
            for l in range(cfg.n_layers):
                pu.moe_layer_check(cfg, m, st, l, lcs, sm.layer_input(cfg, l, T, tag=800 + step), combined=True)
        pu.check_counters(m, lcs)
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 4, 77])
@pytest.mark.parametrize("lookahead", [0, 1])
def test_stack_step_in_one_call(T, lookahead):
    # promoe_stack_step runs the layer loop of the separate calls: the residual
    # stream after each step, the plans and every counter match them bit for bit
    cfg = SMALL.with_(lookahead=lookahead)
    _log("stack_step T", T, "lookahead", lookahead)
    m = SyntheticModel(cfg, max_tokens=T)
    try:
        st = Stack(m, T)
        runs = []
        for native in (False, True):
            m.open()
            hs, plans = [], []
            for step in range(3):
                h0 = torch.from_numpy(sm.stack_input(cfg, 990 + step, T)).cuda()
                hs.append(pu.to_np(st.step(h0, native=native)).copy())
                plans.append([(m.ctx.last_plan(l, 0)["slot"], m.ctx.last_plan(l, 1)["slot"])
                              for l in range(cfg.n_layers)])
            runs.append((hs, plans, [m.ctx.stats(l) for l in range(cfg.n_layers)]))
        (h_a, p_a, s_a), (h_b, p_b, s_b) = runs
        for i, (a, b) in enumerate(zip(h_a, h_b)):
            assert np.array_equal(a, b), _step_diff(i, a, b)
        assert p_a == p_b
        for l, (a, b) in enumerate(zip(s_a, s_b)):
            for c in ocache.COUNTERS:
                assert a[c] == b[c], (l, c)
    finally:
        m.close()


@pytest.mark.parametrize("T", [1, 4])
def test_stack_step_all_resident_lazy_routes(T):
    # With every expert of every layer resident, the layer loop's routes return
    # without waiting for their plans on the host and the plans are taken in
    # later.  The residual stream, the plans, the device counters, the in-time
    # predictions and the launches' profiled bytes must equal those of the
    # separate calls (whose routes wait, since they ask for the order) bit for
    # bit; a run of steps with no host read in between lets the plans queue up.
    cfg = SMALL.with_(lookahead=1, slots=SMALL.n_experts)
    _log("stack_step all resident T", T)
    m = SyntheticModel(cfg, max_tokens=T, flags=_abi.FLAG_PROFILE)
    try:
        st = Stack(m, T)
        runs = []
        for native in (False, True):
            m.open(flags=_abi.FLAG_PROFILE)
            hs, plans = [], []
            for step in range(14):
                h0 = torch.from_numpy(sm.stack_input(cfg, 995 + step, T)).cuda()
                hs.append(pu.to_np(st.step(h0, native=native)).copy())
                if step < 2 or step == 13:
                    plans.append([(m.ctx.last_plan(l, 0)["slot"], m.ctx.last_plan(l, 1)["slot"])
                                  for l in range(cfg.n_layers)])
            runs.append((hs, plans, [m.ctx.stats(l) for l in range(cfg.n_layers)], m.ctx.stats(-1)))
        (h_a, p_a, s_a, t_a), (h_b, p_b, s_b, t_b) = runs
        assert t_a["lazy_routes"] == 0 and t_b["lazy_routes"] == 14 * cfg.n_layers, (t_a["lazy_routes"],
                                                                                     t_b["lazy_routes"])
        for i, (a, b) in enumerate(zip(h_a, h_b)):
            assert np.array_equal(a, b), _step_diff(i, a, b)
        assert p_a == p_b
        for l, (a, b) in enumerate(zip(s_a, s_b)):
            for c in ocache.COUNTERS:
                assert a[c] == b[c], (l, c)
        assert t_a["miss"] == 0 and t_a["pred_in_time"] == t_a["pred_correct"] > 0
        assert t_b["pred_in_time"] == t_a["pred_in_time"]
        assert t_b["k_launches"][:2] == t_a["k_launches"][:2]
        assert t_b["k_bytes"][:2] == t_a["k_bytes"][:2]
    finally:
        m.close()


# The batch-1 layer loop at the model shapes' hidden and predictor widths: the
# RMSNorms folded into the attention and gate GEMVs (hidden 2048, 4096 and 3584
# take different register layouts there) and the prediction inside the plan
# kernel (predictor width 512) must give the separate calls' residual stream,
# plans and counters bit for bit -- with part of the experts cached, and for
# the DeepSeek shape also with every expert resident (lazy routes).
STACK_SHAPES = [
    ("c2_deepseek16b", configs.C2.with_(n_layers=3), None),
    ("c2_deepseek16b_all_resident", configs.C2.with_(n_layers=3), "all"),
    ("c4_mixtral_int4", configs.C4.with_(n_layers=3, weight_format="int4", lookahead=1), None),
    ("c5_qwen2_57b_int4", configs.C5.with_(n_layers=3, weight_format="int4"), None),
]


@pytest.mark.parametrize("name,cfg,slots", STACK_SHAPES, ids=[c[0] for c in STACK_SHAPES])
def test_stack_step_model_shapes(name, cfg, slots):
    _log("stack_step shape", name)
    if slots == "all":
        cfg = cfg.with_(slots=cfg.n_experts)
    m = SyntheticModel(cfg, max_tokens=1, gen_threads=8)
    try:
        st = Stack(m, 1)
        runs = []
        for native in (False, True):
            m.open(spec_fill_limit=1)
            hs, plans = [], []
            for step in range(3):
                h0 = torch.from_numpy(sm.stack_input(cfg, 960 + step, 1)).cuda()
                hs.append(pu.to_np(st.step(h0, native=native)).copy())
                plans.append([(m.ctx.last_plan(l, 0)["slot"], m.ctx.last_plan(l, 1)["slot"])
                              for l in range(cfg.n_layers)])
            runs.append((hs, plans, [m.ctx.stats(l) for l in range(cfg.n_layers)], m.ctx.stats(-1)))
        (h_a, p_a, s_a, t_a), (h_b, p_b, s_b, t_b) = runs
        if slots == "all":
            assert t_b["lazy_routes"] == 3 * cfg.n_layers and t_a["miss"] == 0
        for i, (a, b) in enumerate(zip(h_a, h_b)):
            assert np.array_equal(a, b), ("step", i, int((a != b).sum()))
        assert p_a == p_b
        for l, (a, b) in enumerate(zip(s_a, s_b)):
            for c in ocache.COUNTERS:
                assert a[c] == b[c], (l, c)
        if slots == "all":  # with copies in flight it depends on their timing
            assert t_a["pred_in_time"] == t_b["pred_in_time"]
    finally:
        m.close()
