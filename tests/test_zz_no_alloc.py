"""dvi_verify_static (the verify entry point that allocates nothing) against dvi_verify.

Both run the same kernels on the same drafted state; dvi_verify_static only keeps the attention
partials, merge counters and argmax partials in the library's static device array instead of the
workspace, and at 33-64 rows it reduces each GEMM tile's K pieces inside one launch where
dvi_verify spreads them over workgroups and adds them in a second launch (same order, same bits).
Its targets, accept lengths and logits must equal dvi_verify's bit for bit, on two calls in a row
(the second with fewer rows), and a verify that would need more than the array's size is
refused."""
import numpy as np
import pytest

import synth
from paper_2510_05421_amd import _abi
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _verify_static(eng):
    tg = np.empty((eng.batch, eng.k_spec), np.int32)
    m = np.empty(eng.batch, np.int32)
    st = eng.lib.dvi_verify_static(eng.ctx, tg.ctypes.data, m.ctypes.data)
    eng._check(st)
    return tg, m


def _both(eng, k, forced):
    """dvi_verify, then (the step aborted and drafted again) dvi_verify_static, on one state."""
    eng.draft(k, forced=forced)
    tg1, m1 = eng.verify(want=True)
    lg1 = eng.read_logits().copy()
    eng.abort()
    eng.draft(k, forced=forced)
    tg2, m2 = _verify_static(eng)
    lg2 = eng.read_logits().copy()
    return (tg1, m1, lg1), (tg2, m2, lg2)


@pytest.mark.parametrize("name,B,k", [("tiny", 3, 6), ("7b_L4", 3, 6), ("tiny", 6, 8), ("7b_L4", 6, 8),
                                      ("tiny", 8, 8), ("7b_L4", 8, 8)])
def test_verify_static_equals_verify(name, B, k):
    """18 rows (one-launch GEMMs on both sides), 48 and 64 rows (dvi_verify splits its GEMMs)."""
    shape = gu.SHAPES[name]
    P = 70
    prompts = synth.make_prompts(shape.vocab, B, P, 41)
    _say("verify_static %s B=%d P=%d k=%d then k=2" % (name, B, P, k))
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + 40, max_k_spec=k)
    ar, _ = eng.generate(prompts, 20, 1)
    eng.prefill(prompts)
    # first call: drafts = greedy continuation with one wrong position per sequence (none for
    # the sequences whose wrong position is k)
    wrong = [(0, 2, k, 1, 3, 5, k, 4)[b] for b in range(B)]
    forced = ar[:, 1:1 + k].copy()
    for b, j in enumerate(wrong):
        if j < k:
            forced[b, j] = (forced[b, j] + 1) % shape.vocab
    (tg1, m1, lg1), (tg2, m2, lg2) = _both(eng, k, forced)
    assert np.array_equal(tg1, tg2) and np.array_equal(m1, m2) and np.array_equal(lg1, lg2)
    assert list(m2) == wrong
    tok, n, m = eng.commit()
    # second call, fewer rows (k = 2), from the committed state
    forced2 = np.stack([ar[b, 1 + n[b]:3 + n[b]] for b in range(B)]).astype(np.int32)
    (tg1, m1, lg1), (tg2, m2, lg2) = _both(eng, 2, forced2)
    assert np.array_equal(tg1, tg2) and np.array_equal(m1, m2) and np.array_equal(lg1, lg2)
    tok, n, m = eng.commit()
    assert np.all(m == 2)
    eng.close()


def test_verify_static_refuses_more_than_its_scratch():
    """64 rows over a 2000-position context need about 35 MB of attention partials: refused with
    DVI_ERR_CAPACITY before anything is launched; the step can then be verified normally."""
    shape = gu.SHAPES["7b_L4"]
    B, P, k = 8, 2000, 8
    prompts = synth.make_prompts(shape.vocab, B, P, 43)
    eng, _ = gu.engine(shape, max_batch=B, max_seq=P + 16)
    eng.prefill(prompts)
    eng.draft(k)
    tg = np.empty((B, k), np.int32)
    m = np.empty(B, np.int32)
    st = eng.lib.dvi_verify_static(eng.ctx, tg.ctypes.data, m.ctypes.data)
    assert st == _abi.ERR_CAPACITY
    assert b"static scratch" in eng.lib.dvi_last_error(eng.ctx)
    eng.verify()
    eng.commit()
    eng.close()
