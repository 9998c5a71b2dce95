"""GPU parity at the full model shapes (1B and 8B) through the C ABI.

Each test evaluates the whole synthetic table in the launch configuration the
benchmark times (default batch budget, whole-table call), then evaluates a
sample of its rows again with logit dumps and compares those with the fp32
oracle (the precision the target names for its CPU forward).  The library's
results do not depend on which other rows share a call, so the sampled call
must reproduce the full call's typed outputs and log-probabilities exactly.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import KIND_ENUM, OracleLM
from synth import SHAPES, make_weights, make_workload, parity_rows
from tests.parity import assert_automaton, assert_typed, compare

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


def _model(L, name):
    shape = SHAPES[name]
    w = make_weights(shape, seed=1234, device="cuda")
    torch.cuda.synchronize()
    ctx = L.Context(shape, device=0, stream=torch.cuda.current_stream().cuda_stream)
    ctx.load_weights(w)
    return w, ctx


@pytest.fixture(scope="module")
def m8b(L):
    _log("8B: weights on the GPU, library load, oracle setup")
    w, ctx = _model(L, "8b")
    orc = OracleLM(w, SHAPES["8b"], dtype=np.float32, cache_dequant=True)
    yield w, ctx, orc
    ctx.close()
    del w
    torch.cuda.empty_cache()


def _same_rows(full, sub, rows, label):
    # bit for bit (NaN fields, as in restricted mode, compare equal too)
    for j, r in enumerate(rows):
        assert full[r].tobytes() == sub[j].tobytes(), f"{label}: row {r} differs between calls"


def _check_filter(ctx, orc, wl, pre, sample, label):
    _log(f"{label}: full table ({wl.n_rows} rows, {wl.n_suffix_tokens} tokens)")
    full, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre)
    assert_typed(full, wl.kind, len(wl.allowed), wl.allowed)
    sub = wl.subset(sample)
    out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre,
                             debug_logits=True)
    _same_rows(full, out, sample, label)
    _log(f"{label}: oracle on {len(sample)} rows ({sub.n_suffix_tokens} suffix tokens)")
    ref = orc.eval_workload(sub, keep_logits=True)
    st = compare(ref, out, dbg, label)
    _log(label, st)
    return st


def _sample(wl, n, seed):
    return parity_rows(wl, n, seed)


def _forced(orc, sub, out, ref):
    """The oracle teacher-forced on the library's tokens, for the rows whose
    token path left the oracle's after a sub-margin step (None elsewhere)."""
    R = sub.n_rows
    div = [r for r in range(R)
           if list(out["tokens"][r][: out["n_tokens"][r]]) != list(ref["tokens"][r][: ref["n_tokens"][r]])]
    if not div:
        return None
    f = orc.eval_workload(sub, rows=div, keep_logits=True,
                          forced=[out["tokens"][r][: out["n_tokens"][r]] for r in div])
    logits = [None] * R
    for j, r in enumerate(div):
        logits[r] = f["logits"][j]
    return {"logits": logits}


def test_filter_1b_sampled_rows(L):
    w, ctx = _model(L, "1b")
    orc = OracleLM(w, SHAPES["1b"], dtype=np.float32, cache_dequant=True)
    wl = make_workload("filter_1b")
    pre = ctx.set_prefix(wl.prefix)
    _check_filter(ctx, orc, wl, pre, _sample(wl, 256, 1), "filter_1b")
    ctx.close()
    del w, orc
    torch.cuda.empty_cache()


def test_filter_8b_sampled_rows(m8b):
    w, ctx, orc = m8b
    wl = make_workload("filter_8b")
    pre = ctx.set_prefix(wl.prefix)
    _check_filter(ctx, orc, wl, pre, _sample(wl, 64, 2), "filter_8b")
    ctx.release_prefix(pre)


def test_filter_8b_restricted_head(m8b):
    """The whole table with the restricted head, then sampled rows against
    the oracle's allowed logits."""
    w, ctx, orc = m8b
    wl = make_workload("filter_8b")
    pre = ctx.set_prefix(wl.prefix)
    _log(f"filter_8b restricted: full table ({wl.n_rows} rows)")
    full, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre,
                            head_restricted=True)
    assert_typed(full, wl.kind, len(wl.allowed), wl.allowed)
    assert np.all(np.isnan(full["logprob_full"]))
    sample = _sample(wl, 16, 5)
    sub = wl.subset(sample)
    out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre,
                             debug_logits=True, head_restricted=True)
    _same_rows(full, out, sample, "filter_8b restricted")
    _log(f"filter_8b restricted: oracle on {len(sample)} rows")
    ref = orc.eval_workload(sub, keep_logits=True)
    st = compare(ref, out, dbg, "filter_8b restricted", cols=wl.allowed)
    _log("filter_8b restricted", st)
    ctx.release_prefix(pre)


def test_options_8b_sampled_rows(m8b, L):
    """24 multi-token options (a token trie, up to 3 tokens) over the whole
    8B-shape table, then sampled rows against the oracle."""
    w, ctx, orc = m8b
    wl = make_workload("options_8b")
    pre = ctx.set_prefix(wl.prefix)
    kw = dict(eos=wl.eos, max_tokens=wl.max_tokens, prefix=pre)
    _log(f"options_8b: full table ({wl.n_rows} rows)")
    full, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.automaton, **kw)
    assert_automaton(full, wl.automaton, wl.eos, wl.max_tokens)
    sample = _sample(wl, 16, 7)
    sub = wl.subset(sample)
    out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.automaton, debug_logits=True,
                             **kw)
    _same_rows(full, out, sample, "options_8b")
    _log(f"options_8b: oracle on {len(sample)} rows")
    ref = orc.eval_workload(sub, keep_logits=True)
    st = compare(ref, out, dbg, "options_8b", orc_forced=_forced(orc, sub, out, ref))
    _log("options_8b", st)
    ctx.release_prefix(pre)


def test_map_int_8b_dedup_and_sampled_rows(m8b, L):
    w, ctx, orc = m8b
    wl = make_workload("map_int_8b")
    pre = ctx.set_prefix(wl.prefix)
    _log(f"map_int_8b: full table ({wl.n_rows} rows)")
    full, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, eos=wl.eos,
                            max_tokens=wl.max_tokens, prefix=pre)
    assert_typed(full, wl.kind, 10, wl.allowed, wl.eos, wl.max_tokens)
    # early dedup: every duplicate gets its representative's result, bit for bit
    rep, n_unique = L.lmop_dedup_rows(wl.tokens, wl.offsets)
    assert 2300 < n_unique < 3000
    assert np.array_equal(full, full[rep])
    # 64 distinct suffixes (the longest and shortest among them), each with
    # up to two of its duplicate rows
    rng = np.random.default_rng(3)
    reps_all = np.unique(rep)
    lens = np.diff(wl.offsets)[reps_all]
    reps = {int(reps_all[np.argmax(lens)]), int(reps_all[np.argmin(lens)]), int(rep[0]),
            int(rep[-1])}
    while len(reps) < 64:
        reps.add(int(rng.choice(reps_all)))
    rows, uniq = [], []
    for r in sorted(reps):
        dup = np.nonzero(rep == r)[0]
        uniq.append(len(rows))
        rows.extend(dup[:2].tolist())
    assert len(rows) > len(uniq)  # some suffixes do repeat
    sub = wl.subset(rows)
    out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, eos=wl.eos,
                             max_tokens=wl.max_tokens, prefix=pre, debug_logits=True)
    _same_rows(full, out, rows, "map_int_8b")
    sub_u = wl.subset([rows[j] for j in uniq])
    _log(f"map_int_8b: oracle on {len(uniq)} distinct rows")
    ref = orc.eval_workload(sub_u, keep_logits=True)
    st = compare(ref, out[uniq], dbg[uniq], "map_int_8b",
                 orc_forced=_forced(orc, sub_u, out[uniq], ref))
    _log("map_int_8b", st)
    ctx.release_prefix(pre)


def test_join_8b_sampled_pairs(m8b):
    w, ctx, orc = m8b
    wl = make_workload("join_8b")
    root = ctx.set_prefix(wl.prefix)
    _log(f"join_8b: {len(wl.children)} child prefixes in one batched call")
    kids = ctx.set_prefixes(wl.children, parent=root)
    row_prefix = [kids[int(i)] for i in wl.row_child]
    _log(f"join_8b: full table ({wl.n_rows} pairs)")
    full, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, row_prefix=row_prefix)
    assert_typed(full, wl.kind, 2, wl.allowed)
    # 4 left values (first, last, two seeded) x 16 right values (first, last,
    # 14 seeded): 64 pairs over 4 child prefixes
    rng = np.random.default_rng(6)
    lefts = sorted({0, 199} | set(rng.choice(np.arange(1, 199), 2, replace=False).tolist()))
    rights = sorted({0, 199} | set(rng.choice(np.arange(1, 199), 14, replace=False).tolist()))
    rows = [200 * a + b for a in lefts for b in rights]
    sub = wl.subset(rows)
    out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed,
                             row_prefix=[row_prefix[r] for r in rows], debug_logits=True)
    _same_rows(full, out, rows, "join_8b")
    # the sampled pairs against children made one at a time: the same bits
    single = {int(wl.row_child[r]): None for r in rows}
    for i in single:
        single[i] = ctx.set_prefix(wl.children[i], parent=root)
    out1, dbg1 = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed,
                               row_prefix=[single[int(wl.row_child[r])] for r in rows],
                               debug_logits=True)
    assert out1.tobytes() == out.tobytes() and np.array_equal(dbg1, dbg)
    for p in single.values():
        ctx.release_prefix(p)
    _log(f"join_8b: oracle on {len(rows)} pairs")
    ref = orc.eval_workload(sub, keep_logits=True)
    st = compare(ref, out, dbg, "join_8b")
    _log("join_8b", st)
    for k in kids:
        ctx.release_prefix(k)
    ctx.release_prefix(root)


def test_filter_8b_fp8_sampled_rows(L):
    """FP8 (E4M3, per-channel scales) weights at the 8B shape: the whole
    filter table, then sampled rows against the oracle of the same weights."""
    shape = SHAPES["8b"]
    _log("8B fp8: weights on the GPU, library load")
    w = make_weights(shape, seed=1234, device="cuda", fmt="fp8_e4m3")
    torch.cuda.synchronize()
    ctx = L.Context(shape, device=0, stream=torch.cuda.current_stream().cuda_stream)
    ctx.load_weights(w)
    orc = OracleLM(w, shape, dtype=np.float32, cache_dequant=False)
    wl = make_workload("filter_8b")
    pre = ctx.set_prefix(wl.prefix)
    _check_filter(ctx, orc, wl, pre, _sample(wl, 8, 3), "filter_8b fp8")
    ctx.close()
    del w, orc
    torch.cuda.empty_cache()


def test_head_tiles_8b_shape(L):
    """The LM head at the 8B shape (V = 128,256, d = 4,096) on a model with no
    decoder layers: 300 one-token rows in one batch (one 320-row head tile)
    and in batches of at most 100 rows (the 256-row tile) give the same bits,
    and sampled rows match the fp32 oracle."""
    import dataclasses

    shape = dataclasses.replace(SHAPES["8b"], n_layers=0)
    w = make_weights(shape, seed=4321, device="cuda", n_layers=0)
    torch.cuda.synchronize()
    ctx = L.Context(shape, device=0, stream=torch.cuda.current_stream().cuda_stream)
    ctx.load_weights(w)
    rng = np.random.default_rng(5)
    toks = rng.integers(0, shape.vocab, size=300).astype(np.int32)
    offs = np.arange(301, dtype=np.int64)
    allowed = rng.choice(shape.vocab, 24, replace=False).astype(np.int32)
    _log("8B head: 300 rows in one batch, then in batches of 100")
    full, _ = ctx.eval_rows(toks, offs, KIND_ENUM, allowed, no_dedup=True)
    small, _ = ctx.eval_rows(toks, offs, KIND_ENUM, allowed, no_dedup=True, max_batch_tokens=100)
    assert full.tobytes() == small.tobytes()
    assert_typed(full, KIND_ENUM, len(allowed), allowed)
    sample = [0, 77, 150, 256, 299]
    st_toks = toks[sample]
    out, dbg = ctx.eval_rows(st_toks, np.arange(len(sample) + 1, dtype=np.int64), KIND_ENUM,
                             allowed, no_dedup=True, debug_logits=True)
    _same_rows(full, out, sample, "8B head")
    orc = OracleLM(w, shape, dtype=np.float32)
    ref = orc.eval_rows(np.zeros(0, dtype=np.int32), [toks[i:i + 1] for i in sample], KIND_ENUM,
                        allowed, keep_logits=True)
    st = compare(ref, out, dbg, "8B head")
    _log("8B head", st)
    ctx.close()
    del w, orc
    torch.cuda.empty_cache()


def test_llmqa_8b_width_past_4096_positions(L):
    """LLMQA (Sec. 2.3.1: one prompt over a whole data subset) at the 8B
    width with 2 layers: one 256 + 8,192-token prompt, so RoPE angles,
    own-KV slots and attention walks run past position 4,096, against the
    fp32 oracle (the multi-token option decoded under its trie)."""
    import dataclasses
    shape = dataclasses.replace(SHAPES["8b"], n_layers=2)
    w = make_weights(shape, seed=1234, device="cuda", n_layers=2)
    torch.cuda.synchronize()
    ctx = L.Context(shape, device=0, stream=torch.cuda.current_stream().cuda_stream,
                    max_seq=9216)
    ctx.load_weights(w)
    wl = make_workload("qa_8b")
    assert len(wl.prefix) + wl.n_suffix_tokens > 8192
    pre = ctx.set_prefix(wl.prefix)
    kw = dict(eos=wl.eos, max_tokens=wl.max_tokens, prefix=pre, debug_logits=True)
    _log("llmqa 8B-width: eval")
    out, dbg = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.automaton, **kw)
    assert_automaton(out, wl.automaton, wl.eos, wl.max_tokens)
    # a batch budget below the prompt's length gives the same bits
    o1, d1 = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.automaton, max_batch_tokens=1000,
                           **kw)
    assert o1.tobytes() == out.tobytes() and np.array_equal(d1, dbg, equal_nan=True)
    _log("llmqa 8B-width: oracle")
    orc = OracleLM(w, shape, dtype=np.float32)
    ref = orc.eval_workload(wl, keep_logits=True)
    st = compare(ref, out, dbg, "llmqa 8B width", orc_forced=_forced(orc, wl, out, ref))
    _log("llmqa 8B width", st)
    ctx.release_prefix(pre)
    ctx.close()
    del w, orc
    torch.cuda.empty_cache()
