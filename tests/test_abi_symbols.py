"""The C-ABI library loads on the CPU and exports every call include/promoe.h declares."""
import ctypes
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "promoe.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(promoe_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_hot_path_calls():
    names = _declared()
    for n in ("promoe_route", "promoe_predict", "promoe_prefetch", "promoe_expert_ffn", "promoe_cache_stats"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2410_22134_amd import _abi
    lib = ctypes.CDLL(_abi.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(_abi.exported_symbols()) == _declared()


def test_strerror_without_gpu():
    from paper_2410_22134_amd import _abi
    l = _abi.lib()
    assert l.promoe_strerror(0) == b"ok"
    assert l.promoe_strerror(-4) == b"call order violated"
    cfg = _abi.Config()
    cfg.inter, cfg.hidden, cfg.dtype = 1408, 2048, _abi.PROMOE_BF16
    assert l.promoe_expert_bytes(ctypes.byref(cfg)) == 17301504
