"""ctypes binding of libpromoe.so (include/promoe.h).  Argument marshalling only:
every step of the path runs in the library's HIP kernels.  Importing this module
without the built library raises immediately -- there is no fallback."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("PROMOE_LIB", os.path.join(HERE, "libpromoe.so"))

PROMOE_F32, PROMOE_BF16 = 0, 1
WEIGHTS_DENSE, WEIGHTS_INT4 = 0, 1
PRIO_LOW, PRIO_HIGH = 0, 1
FLAG_PROFILE, FLAG_NO_PREFETCH, FLAG_NO_CHUNK, FLAG_NO_PREEMPT, FLAG_NO_REORDER, FLAG_STATIC = 1, 2, 4, 8, 16, 32
FLAG_FILL_BY_DEADLINE = 64

_i32, _i64, _vp, _sz, _dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_double


class Config(ctypes.Structure):
    _fields_ = [("n_layers", _i32), ("hidden", _i32), ("n_experts", _i32), ("top_k", _i32), ("inter", _i32),
                ("shared_inter", _i32), ("shared_gate", _i32), ("renorm", _i32), ("router_bias", _i32),
                ("slots_per_layer", _i32), ("lookahead", _i32), ("pred_hidden", _i32), ("max_tokens", _i32),
                ("dtype", _i32), ("copy_subchunk_bytes", _i64), ("copy_window", _i32), ("flags", _i32),
                ("spec_fill_limit", _i32), ("weight_format", _i32), ("link_gb_per_s", ctypes.c_float)]


STAT_COUNTERS = ("prec_access", "hit", "miss", "spec_issued", "spec_resident", "spec_used", "spec_wasted", "evict",
                 "pred_n", "pred_correct")


class Stats(ctypes.Structure):
    _fields_ = [(n, _i64) for n in STAT_COUNTERS] + [
        ("copies_high", _i64), ("copies_low", _i64), ("bytes_high", _i64), ("bytes_low", _i64),
        ("low_purged", _i64), ("deferred", _i64), ("pred_in_time", _i64),
        ("k_launches", _i64 * 6), ("k_ms", _dbl * 6), ("k_bytes", _dbl * 6), ("k_flops", _dbl * 6),
        ("stall_ms", _dbl), ("copy_ms", _dbl), ("lazy_routes", _i64)]

    def as_dict(self):
        d = {n: int(getattr(self, n)) for n in STAT_COUNTERS}
        for n in ("copies_high", "copies_low", "bytes_high", "bytes_low", "low_purged", "deferred", "pred_in_time"):
            d[n] = int(getattr(self, n))
        for n in ("k_launches", "k_ms", "k_bytes", "k_flops"):
            d[n] = list(getattr(self, n))
        d["stall_ms"] = float(self.stall_ms)
        d["lazy_routes"] = int(self.lazy_routes)
        return d


class Plan(ctypes.Structure):
    _fields_ = [("n", _i32)] + [(n, _i32 * 64) for n in ("expert", "slot", "flag", "victim", "after", "count")] + \
        [("fill_budget", _i32)]

    def as_dict(self):
        n = self.n
        return {"n": n, "fill_budget": int(self.fill_budget),
                **{f: list(getattr(self, f))[:n] for f in ("expert", "slot", "flag", "victim", "after", "count")}}


class PromoeError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {code} ({detail})")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2410_22134_amd.build.build() "
                          "(there is no non-HIP fallback)")
    l = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    sig = {
        "promoe_create": ([P(Config), _vp, _sz, P(_vp)], ctypes.c_int),
        "promoe_destroy": ([_vp], ctypes.c_int),
        "promoe_set_layer": ([_vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
        "promoe_set_attn": ([_vp, ctypes.c_int, _vp], ctypes.c_int),
        "promoe_set_expert_host": ([_vp, ctypes.c_int, ctypes.c_int, _vp], ctypes.c_int),
        "promoe_set_initial_cache": ([_vp, ctypes.c_int, _vp, ctypes.c_int], ctypes.c_int),
        "promoe_predict": ([_vp, ctypes.c_int, _vp, ctypes.c_int, _vp, _vp, _vp, _vp], ctypes.c_int),
        "promoe_route": ([_vp, ctypes.c_int, _vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
        "promoe_route_predict": ([_vp, ctypes.c_int, _vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp],
                                 ctypes.c_int),
        "promoe_stack_step": ([_vp, _vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_int, _vp],
                              ctypes.c_int),
        "promoe_prefetch": ([_vp, ctypes.c_int, _vp, ctypes.c_int, ctypes.c_int, _vp], ctypes.c_int),
        "promoe_expert_ffn": ([_vp, ctypes.c_int, _vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
        "promoe_expert_ffn_noalloc": ([_vp, ctypes.c_int, _vp, ctypes.c_int, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
        "promoe_cache_stats": ([_vp, ctypes.c_int, P(Stats)], ctypes.c_int),
        "promoe_reset_stats": ([_vp], ctypes.c_int),
        "promoe_slot_table": ([_vp, ctypes.c_int, _vp], ctypes.c_int),
        "promoe_last_plan": ([_vp, ctypes.c_int, ctypes.c_int, P(Plan)], ctypes.c_int),
        "promoe_sync": ([_vp], ctypes.c_int),
        "promoe_attn_surrogate": ([_vp, ctypes.c_int, _vp, ctypes.c_int, _vp, _vp], ctypes.c_int),
        "promoe_residual_add": ([_vp, _vp, _vp, ctypes.c_int, _vp], ctypes.c_int),
        "promoe_host_alloc": ([_sz, P(_vp)], ctypes.c_int),
        "promoe_host_free": ([_vp], ctypes.c_int),
        "promoe_expert_bytes": ([P(Config)], _sz),
        "promoe_strerror": ([ctypes.c_int], ctypes.c_char_p),
        "promoe_last_error_string": ([], ctypes.c_char_p),
        "promoe_peak_hbm_read": ([_vp, _sz, _vp, ctypes.c_int, _vp], ctypes.c_int),
        "promoe_peak_mfma_bf16": ([_vp, ctypes.c_int, ctypes.c_int, _vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(l, name)
        fn.argtypes = args
        fn.restype = res
    _lib = l
    return l


def exported_symbols():
    return [n for n in ("promoe_create", "promoe_destroy", "promoe_set_layer", "promoe_set_attn",
                        "promoe_set_expert_host", "promoe_set_initial_cache", "promoe_predict", "promoe_route",
                        "promoe_route_predict", "promoe_prefetch", "promoe_expert_ffn", "promoe_expert_ffn_noalloc", "promoe_cache_stats",
                        "promoe_reset_stats",
                        "promoe_slot_table", "promoe_last_plan", "promoe_sync", "promoe_attn_surrogate",
                        "promoe_residual_add", "promoe_stack_step", "promoe_host_alloc", "promoe_host_free",
                        "promoe_expert_bytes",
                        "promoe_strerror", "promoe_last_error_string", "promoe_peak_hbm_read",
                        "promoe_peak_mfma_bf16")]


def peak_hbm_read(buf, nbytes: int, sink, blocks: int, stream=None) -> None:
    """One streaming read of `nbytes` of `buf` (see promoe_peak_hbm_read)."""
    check(lib().promoe_peak_hbm_read(_p(buf), nbytes, _p(sink), blocks, _stream(stream)), "peak_hbm_read")


def peak_mfma_bf16(sink, blocks: int, iters: int, stream=None) -> None:
    """Register-only MFMA loop (see promoe_peak_mfma_bf16)."""
    check(lib().promoe_peak_mfma_bf16(_p(sink), blocks, iters, _stream(stream)), "peak_mfma_bf16")


def check(rc: int, where: str) -> None:
    if rc != 0:
        l = lib()
        raise PromoeError(rc, where, f"{l.promoe_strerror(rc).decode()}; {l.promoe_last_error_string().decode()}")


def _p(t):
    """Device/host address of a tensor, an int address, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Context:
    """One promoe_ctx.  Tensors passed in must stay alive as long as the context."""

    def __init__(self, cfg: Config, cache_ptr: int, cache_bytes: int):
        self.cfg = cfg
        self._h = _vp()
        check(lib().promoe_create(ctypes.byref(cfg), cache_ptr, cache_bytes, ctypes.byref(self._h)), "promoe_create")
        self._keep = []
        # out-arrays of the per-layer calls, allocated once
        self._order = (ctypes.c_int32 * 64)()
        self._q = (ctypes.c_int32 * 64)()
        self._n = ctypes.c_int32(0)
        self._n_ref = ctypes.byref(self._n)

    def close(self):
        if self._h:
            check(lib().promoe_destroy(self._h), "promoe_destroy")
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # weights
    def set_layer(self, layer, wgate, bias=None, pw1=None, pw2=None, shared=None, shared_gate=None):
        self._keep += [wgate, bias, pw1, pw2, shared, shared_gate]
        check(lib().promoe_set_layer(self._h, layer, _p(wgate), _p(bias), _p(pw1), _p(pw2), _p(shared),
                                     _p(shared_gate)), "promoe_set_layer")

    def set_attn(self, layer, wattn):
        self._keep.append(wattn)
        check(lib().promoe_set_attn(self._h, layer, _p(wattn)), "promoe_set_attn")

    def set_expert_host(self, layer, expert, addr: int):
        check(lib().promoe_set_expert_host(self._h, layer, expert, addr), "promoe_set_expert_host")

    def set_initial_cache(self, layer, experts):
        arr = (ctypes.c_int32 * max(1, len(experts)))(*experts)
        check(lib().promoe_set_initial_cache(self._h, layer, arr, len(experts)), "promoe_set_initial_cache")

    # hot path
    def predict(self, layer, x, T, pred_ids=None, want_q=False, stream=None):
        check(lib().promoe_predict(self._h, layer, _p(x), T, _p(pred_ids), self._q if want_q else None,
                                   self._n_ref if want_q else None, _stream(stream)), "promoe_predict")
        return self._q[:self._n.value] if want_q else None

    def route(self, layer, x, T, ids, w, shared_scale=None, stream=None):
        check(lib().promoe_route(self._h, layer, _p(x), T, _p(ids), _p(w), _p(shared_scale), self._order,
                                 self._n_ref, _stream(stream)), "promoe_route")
        return self._order[:self._n.value]

    def route_predict(self, layer, x, T, ids, w, shared_scale=None, pred_ids=None, stream=None):
        """route then predict of one layer on one input, in one call (look-ahead >= 1)."""
        check(lib().promoe_route_predict(self._h, layer, _p(x), T, _p(ids), _p(w), _p(shared_scale),
                                         _p(pred_ids), self._order, self._n_ref, _stream(stream)),
              "promoe_route_predict")
        return self._order[:self._n.value]

    def prefetch(self, layer, ids, prio=PRIO_LOW, stream=None):
        arr = (ctypes.c_int32 * max(1, len(ids)))(*ids)
        check(lib().promoe_prefetch(self._h, layer, arr, len(ids), prio, _stream(stream)), "promoe_prefetch")

    def expert_ffn(self, layer, x, T, ids, w, shared_scale, y, stream=None):
        check(lib().promoe_expert_ffn(self._h, layer, _p(x), T, _p(ids), _p(w), _p(shared_scale), _p(y),
                                      _stream(stream)), "promoe_expert_ffn")

    def expert_ffn_noalloc(self, layer, x, T, ids, w, shared_scale, y, stream=None):
        """promoe_expert_ffn with its scratch in the library's static device array."""
        check(lib().promoe_expert_ffn_noalloc(self._h, layer, _p(x), T, _p(ids), _p(w), _p(shared_scale), _p(y),
                                              _stream(stream)), "promoe_expert_ffn_noalloc")

    # harness
    def attn_surrogate(self, layer, h, T, x_out, stream=None):
        check(lib().promoe_attn_surrogate(self._h, layer, _p(h), T, _p(x_out), _stream(stream)),
              "promoe_attn_surrogate")

    def residual_add(self, h, y, T, stream=None):
        check(lib().promoe_residual_add(self._h, _p(h), _p(y), T, _stream(stream)), "promoe_residual_add")

    def stack_step(self, h, T, x, y, ids, w, shared_scale=None, pred_ids=None, predict=True, stream=None):
        """Every layer of one step in one call (attention surrogate, prediction and
        route, expert FFN, residual add); h [T, H] fp32 is updated in place."""
        check(lib().promoe_stack_step(self._h, _p(h), T, _p(x), _p(y), _p(ids), _p(w), _p(shared_scale),
                                      _p(pred_ids), 1 if predict else 0, _stream(stream)), "promoe_stack_step")

    # state
    def stats(self, layer=-1) -> dict:
        s = Stats()
        check(lib().promoe_cache_stats(self._h, layer, ctypes.byref(s)), "promoe_cache_stats")
        return s.as_dict()

    def reset_stats(self):
        check(lib().promoe_reset_stats(self._h), "promoe_reset_stats")

    def slot_table(self, layer):
        arr = (ctypes.c_int32 * self.cfg.n_experts)()
        check(lib().promoe_slot_table(self._h, layer, arr), "promoe_slot_table")
        return list(arr)

    def last_plan(self, layer, kind):
        p = Plan()
        check(lib().promoe_last_plan(self._h, layer, kind, ctypes.byref(p)), "promoe_last_plan")
        return p.as_dict()

    def sync(self):
        check(lib().promoe_sync(self._h), "promoe_sync")


class HostBuffer:
    """Pinned host memory from promoe_host_alloc."""

    def __init__(self, nbytes: int):
        self.nbytes = nbytes
        p = _vp()
        check(lib().promoe_host_alloc(nbytes, ctypes.byref(p)), "promoe_host_alloc")
        self.addr = p.value

    def numpy(self, dtype, count=None, offset=0):
        import numpy as np
        dt = np.dtype(dtype)
        count = (self.nbytes - offset) // dt.itemsize if count is None else count
        buf = (ctypes.c_char * (count * dt.itemsize)).from_address(self.addr + offset)
        return np.frombuffer(buf, dtype=dt, count=count)

    def free(self):
        if self.addr:
            check(lib().promoe_host_free(self.addr), "promoe_host_free")
            self.addr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass
