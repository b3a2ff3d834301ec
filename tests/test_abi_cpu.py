"""Host-only checks of the C ABI: the library loads, exports every entry point that
include/dvi.h declares, and validates configurations without touching a GPU."""
import ctypes
import os
import re

import pytest

from paper_2510_05421_amd import _abi
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "dvi.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dvi_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("dvi_prefill", "dvi_draft", "dvi_verify", "dvi_commit", "dvi_update_drafter"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = _abi.load()
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert set(_abi.SIGNATURES) == set(_declared())


def _cfg(shape, **kw):
    from paper_2510_05421_amd.engine import EngineConfig
    c = EngineConfig.from_shape(shape, max_batch=kw.pop("max_batch", 1), max_seq=kw.pop("max_seq", 1100),
                                max_k_spec=kw.pop("max_k_spec", 8))
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_workspace_size_covers_weights_and_cache():
    from paper_2510_05421_amd.engine import workspace_bytes
    s = synth.SHAPE_7B
    cfg = _cfg(s, max_batch=8, max_seq=2320, max_k_spec=8)
    ws = workspace_bytes(cfg)
    params = s.n_layers * s.layer_params() + 2 * s.vocab * s.d_model
    kv = 2 * s.n_layers * 8 * s.kv_dim * 2320 * 2
    assert ws >= params * 2 + kv
    assert ws < (params * 2 + kv) * 1.1 + (1 << 30)


@pytest.mark.parametrize("bad", [
    dict(d_model=100), dict(head_dim=96), dict(n_kv_heads=3), dict(vocab=4001), dict(max_k_spec=17),
    dict(max_batch=9, max_k_spec=8), dict(lora_rank=0), dict(split_k=0), dict(split_k=99),
    dict(max_seq=10_000_000),   # attention partials of 64 rows past 2 GiB (32-bit offsets)
])
def test_invalid_configs_are_rejected_on_the_host(bad):
    from paper_2510_05421_amd.engine import workspace_bytes
    assert workspace_bytes(_cfg(synth.TINY, **bad)) == 0


def test_create_argument_errors_need_no_gpu():
    lib = _abi.load()
    cfg = _cfg(synth.TINY).to_c()
    out = ctypes.c_void_p()
    assert lib.dvi_create(ctypes.byref(cfg), None, None, 0, None, ctypes.byref(out)) == _abi.ERR_ARG
    assert out.value is None
    assert lib.dvi_create(None, None, None, 0, None, None) == _abi.ERR_ARG
    bad = _cfg(synth.TINY, vocab=4001).to_c()
    w = _abi.Weights()
    assert lib.dvi_create(ctypes.byref(bad), ctypes.byref(w), ctypes.c_void_p(256), 1 << 30, None,
                          ctypes.byref(out)) == _abi.ERR_ARG
    # too small a workspace is a capacity error, detected before any device call
    good = _cfg(synth.TINY).to_c()
    assert lib.dvi_create(ctypes.byref(good), ctypes.byref(w), ctypes.c_void_p(256), 1024, None,
                          ctypes.byref(out)) == _abi.ERR_CAPACITY
    # calls on a null context are argument errors
    assert lib.dvi_draft(None, 4, None, None) == _abi.ERR_ARG
    assert lib.dvi_abort_step(None) == _abi.ERR_ARG
    assert lib.dvi_set_graphs(None, 1) == _abi.ERR_ARG
    assert lib.dvi_set_sampling(None, 1.0, 3) == _abi.ERR_ARG
    assert lib.dvi_decode_steps(None, 4, 8, None, None, None, None) == _abi.ERR_ARG
    assert lib.dvi_last_error(None) == b"null context"


def test_schedule_matches_closed_form():
    from paper_2510_05421_amd.schedule import KLRLSchedule
    s = KLRLSchedule(lambda0=1.0, lambda_kl_min=0.5, lambda_pg_max=1.0, w_rl=0.5, t_warmup=4, t_ramp=4)
    assert s.coeffs(0)["c_kl"] == 1.0 and s.coeffs(0)["c_ce"] == 0.0 and s.coeffs(0)["c_pg"] == 0.0
    c = s.coeffs(6)
    assert abs(c["c_kl"] - 0.75) < 1e-12 and abs(c["c_ce"] - 0.5) < 1e-12 and abs(c["c_pg"] - 0.25) < 1e-12
    assert s.coeffs(50)["c_kl"] == 0.5 and s.coeffs(50)["c_ce"] == 1.0
    assert abs(s.ema(0.0, 1.0) - 0.1) < 1e-12


def test_product_package_does_not_import_the_oracle():
    import subprocess, sys
    code = ("import sys; sys.path.insert(0, %r); import paper_2510_05421_amd.engine, paper_2510_05421_amd; "
            "print(any(m == 'oracle' or m.startswith('oracle.') for m in sys.modules))" % ROOT)
    out = subprocess.check_output([sys.executable, "-c", code], text=True).strip()
    assert out == "False"
    for dirpath, _, files in os.walk(os.path.join(ROOT, "paper_2510_05421_amd")):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in txt and "from oracle" not in txt, f
