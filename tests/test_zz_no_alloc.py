"""lmop_eval_rows_noalloc (scratch in the library's static device array, no
allocation) against lmop_eval_rows through the C ABI: two calls in a row,
the second with a smaller input, give the same bits as the allocating entry
point; the 1B-shape case needs smaller batches than the default budget to
fit the array, and with the logit dump smaller still."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

from synth import SHAPES, make_weights, make_workload
from tests.parity import assert_typed

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31808_amd import lmop
    return lmop


def _both(ctx, wl, **kw):
    a, da = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.type_spec, eos=wl.eos,
                          max_tokens=wl.max_tokens, **kw)
    held = ctx.memory()["device_bytes"]
    b, db = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.type_spec, eos=wl.eos,
                          max_tokens=wl.max_tokens, no_alloc=True, **kw)
    assert ctx.memory()["device_bytes"] == held  # the library allocated nothing
    assert a.tobytes() == b.tobytes()
    if da is not None:
        assert np.array_equal(da, db, equal_nan=True)
    return a


def test_noalloc_tiny_two_calls(L):
    shape = SHAPES["tiny"]
    w = make_weights(shape, seed=1234)
    ctx = L.Context(shape, device=0, stream=torch.cuda.current_stream().cuda_stream)
    ctx.load_weights(w)
    for name, rows in (("filter_tiny", 64), ("filter_tiny", 9), ("options_tiny", 40),
                       ("options_tiny", 3)):
        wl = make_workload(name, n_rows=rows)
        pre = ctx.set_prefix(wl.prefix)
        _log(f"no-alloc {name} {rows} rows")
        out = _both(ctx, wl, prefix=pre, debug_logits=True)
        if wl.kind != 3:
            assert_typed(out, wl.kind, len(wl.allowed), wl.allowed)
        ctx.release_prefix(pre)
    # integer outputs (decode groups in the static array), larger then smaller
    wl = make_workload("filter_tiny")
    digits = np.random.default_rng(3).choice(shape.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(shape.vocab) if t not in digits))
    pre = ctx.set_prefix(wl.prefix)
    for rows in (64, 5):
        sub = wl.subset(range(rows))
        a, _ = ctx.eval_rows(sub.tokens, sub.offsets, 2, digits, eos=eos, max_tokens=4,
                             prefix=pre)
        b, _ = ctx.eval_rows(sub.tokens, sub.offsets, 2, digits, eos=eos, max_tokens=4,
                             prefix=pre, no_alloc=True)
        assert a.tobytes() == b.tobytes(), rows
    ctx.release_prefix(pre)
    ctx.close()


def test_noalloc_1b_shape_shrinks_batches(L):
    # 2 layers of the 1B shape: ~40 KB of scratch per token, so the default
    # 16,384-token batch does not fit the 256 MiB array; the logit dump
    # (0.5 MB per row) shrinks batches further
    shape = dataclasses.replace(SHAPES["1b"], n_layers=2)
    w = make_weights(shape, seed=1234, device="cuda", n_layers=2)
    torch.cuda.synchronize()
    ctx = L.Context(shape, device=0, stream=torch.cuda.current_stream().cuda_stream,
                    max_seq=16384)
    ctx.load_weights(w)
    wl = make_workload("filter_1b")
    pre = ctx.set_prefix(wl.prefix)
    for rows, dump in ((600, False), (250, False), (40, True), (7, True)):
        sub = wl.subset(range(rows))
        _log(f"no-alloc 1B-shape: {rows} rows ({sub.n_suffix_tokens} tokens), dump {dump}")
        out = _both(ctx, sub, prefix=pre, debug_logits=dump)
        assert_typed(out, sub.kind, len(sub.allowed), sub.allowed)
    # a row whose batch cannot fit the array (~41 KB per token) is refused
    # with the sizes, before any device work
    with pytest.raises(L.LmopError) as ei:
        ctx.eval_rows(np.ones(9000, np.int32), [0, 9000], 0, wl.allowed, prefix=pre,
                      no_alloc=True)
    assert ei.value.status == L.LMOP_ERR_OOM and "no-allocation" in str(ei.value)
    ctx.release_prefix(pre)
    ctx.close()
    del w
    torch.cuda.empty_cache()
