"""The layer loop's call order (CPU, no library): with a look-ahead the route of
layer l comes before its prediction, so the speculative copies for layer l + d
queue behind layer l's precise ones; with look-ahead 0 the prediction plans the
layer the route then uses, so it comes first."""
import types

import pytest

torch = pytest.importorskip("torch")

from paper_2410_22134_amd.stack import Stack  # noqa: E402
from synth import configs  # noqa: E402


class _Ctx:
    def __init__(self):
        self.calls = []

    def predict(self, l, *a, **k):
        self.calls.append(("predict", l))

    def route(self, l, *a, **k):
        self.calls.append(("route", l))
        return []

    def route_predict(self, l, *a, **k):
        self.calls += [("route", l), ("predict", l)]
        return []

    def expert_ffn(self, l, *a, **k):
        self.calls.append(("ffn", l))

    def attn_surrogate(self, l, *a, **k):
        self.calls.append(("attn", l))

    def residual_add(self, *a, **k):
        self.calls.append(("res", None))


def _stack(cfg, T=1, flags=0):
    m = types.SimpleNamespace(cfg=cfg, ctx=_Ctx(), device="cpu", flags=flags)
    return Stack(m, T), m.ctx


@pytest.mark.parametrize("base", [configs.C2, configs.C3])
def test_route_before_predict_with_lookahead(base):
    cfg = base.with_(n_layers=3)
    st, ctx = _stack(cfg)
    st.step(torch.zeros(1, cfg.hidden))
    per_layer = [c for c in ctx.calls if c[0] in ("route", "predict", "ffn")]
    assert per_layer == [(n, l) for l in range(3) for n in ("route", "predict", "ffn")]


@pytest.mark.parametrize("T", [1, 512])
def test_route_predict_ffn_at_any_step_size(T):
    cfg = configs.C3.with_(n_layers=2)
    st, ctx = _stack(cfg, T)
    st.step(torch.zeros(T, cfg.hidden))
    per_layer = [c for c in ctx.calls if c[0] in ("route", "predict", "ffn")]
    assert per_layer == [(n, l) for l in range(2) for n in ("route", "predict", "ffn")]


def test_predict_first_at_lookahead_zero():
    cfg = configs.C1
    st, ctx = _stack(cfg)
    st.moe_layer(0)
    assert ctx.calls == [("predict", 0), ("route", 0), ("ffn", 0)]


def test_no_prediction_when_disabled():
    cfg = configs.C2.with_(n_layers=2)
    st, ctx = _stack(cfg)
    st.moe_layer(1, predict=False)
    assert ctx.calls == [("route", 1), ("ffn", 1)]


def test_no_prediction_without_prefetching():
    # a context opened without prefetching reads no prediction: the step skips it
    from paper_2410_22134_amd import FLAG_NO_PREFETCH
    cfg = configs.C2.with_(n_layers=2)
    st, ctx = _stack(cfg, flags=FLAG_NO_PREFETCH)
    st.step(torch.zeros(1, cfg.hidden))
    assert not [c for c in ctx.calls if c[0] == "predict"]
    st.step(torch.zeros(1, cfg.hidden), predict=True)
    assert [c for c in ctx.calls if c[0] == "predict"] == [("predict", 0), ("predict", 1)]
