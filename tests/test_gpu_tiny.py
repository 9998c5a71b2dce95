"""GPU parity of the whole row-evaluation path on the tiny decoder (2 layers,
d 256, 4 heads, vocab 2048) against the fp64 oracle, through the C ABI.
Sizes span several GEMM and attention tiles with ragged tails."""
import dataclasses
import sys

import numpy as np
import pytest
import torch

from oracle import KIND_BOOL, KIND_ENUM, KIND_INT, OracleLM
from oracle.lmop_oracle import KIND_AUTOMATON
from synth import SHAPES, make_weights, make_workload
from tests.parity import assert_automaton, assert_typed, compare

pytestmark = pytest.mark.gpu
TINY = SHAPES["tiny"]


def _log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_31808_amd import lmop
    return lmop


@pytest.fixture(scope="module")
def tiny(L):
    w = make_weights(TINY, seed=1234)
    orc = OracleLM(w, TINY)
    ctx = L.Context(TINY, device=0)
    ctx.load_weights(w)  # host weights
    return w, orc, ctx


def _run(ctx, wl, prefix, **kw):
    return ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, eos=wl.eos,
                         max_tokens=wl.max_tokens, prefix=prefix, debug_logits=True, **kw)


def test_zero_layer_model_head_only(L):
    """L = 0: embedding -> final RMSNorm -> LM head -> constrained pick."""
    w = make_weights(TINY, seed=77, n_layers=0)
    shape0 = dataclasses.replace(TINY, n_layers=0)
    orc = OracleLM(w, shape0)
    ctx = L.Context(shape0, device=0)
    ctx.load_weights(w)
    wl = make_workload("filter_tiny", n_rows=20)
    _log("zero-layer: eval")
    out, dbg = _run(ctx, wl, None)
    ref = orc.eval_workload(dataclasses.replace(wl, prefix=np.zeros(0, np.int32)),
                            keep_logits=True)
    st = compare(ref, out, dbg, "zero-layer")
    _log("zero-layer", st)
    assert_typed(out, wl.kind, len(wl.allowed), wl.allowed)


def test_tiny_filter_with_prefix(tiny, L):
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    _log("tiny filter: set_prefix")
    pre = ctx.set_prefix(wl.prefix)
    _log("tiny filter: eval 64 rows")
    out, dbg = _run(ctx, wl, pre)
    ref = orc.eval_workload(wl, keep_logits=True)
    st = compare(ref, out, dbg, "filter_tiny")
    _log("filter_tiny", st)
    assert st["exact_checked"] >= 32
    assert_typed(out, wl.kind, 2, wl.allowed)
    ctx.release_prefix(pre)


def test_tiny_device_weights_match_host_weights(tiny, L):
    w, orc, ctx = tiny
    ctx2 = L.Context(TINY, device=0)
    ctx2.load_weights(w.to("cuda"))
    wl = make_workload("filter_tiny", n_rows=24)
    p1, p2 = ctx.set_prefix(wl.prefix), ctx2.set_prefix(wl.prefix)
    o1, d1 = _run(ctx, wl, p1)
    o2, d2 = _run(ctx2, wl, p2)
    assert np.array_equal(d1, d2) and np.array_equal(o1, o2)


def test_tiny_no_prefix_and_empty_suffix(tiny, L):
    w, orc, ctx = tiny
    rng = np.random.default_rng(3)
    rows = [rng.integers(0, TINY.vocab, size=int(n)).astype(np.int32)
            for n in (1, 2, 63, 64, 65, 130, 7)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    allowed = rng.choice(TINY.vocab, 5, replace=False)
    out, dbg = ctx.eval_rows(np.concatenate(rows), offs, KIND_ENUM, allowed, debug_logits=True)
    ref = orc.eval_rows(None, rows, KIND_ENUM, allowed, keep_logits=True)
    _log("no prefix", compare(ref, out, dbg, "no-prefix"))
    # empty suffix rows take the prefix's last position
    prefix = rng.integers(0, TINY.vocab, size=50).astype(np.int32)
    pre = ctx.set_prefix(prefix)
    rows2 = [np.zeros(0, np.int32), rows[0], np.zeros(0, np.int32), rows[3]]
    offs2 = np.concatenate([[0], np.cumsum([len(r) for r in rows2])])
    out2, dbg2 = ctx.eval_rows(np.concatenate(rows2), offs2, KIND_ENUM, allowed, prefix=pre,
                               debug_logits=True)
    ref2 = orc.eval_rows(prefix, rows2, KIND_ENUM, allowed, keep_logits=True)
    _log("empty suffix", compare(ref2, out2, dbg2, "empty-suffix"))
    assert np.array_equal(dbg2[0], dbg2[2])
    ctx.release_prefix(pre)


def test_tiny_join_two_level_prefix(tiny, L):
    w, orc, ctx = tiny
    rng = np.random.default_rng(4)
    root_t = rng.integers(0, TINY.vocab, size=70).astype(np.int32)
    kids_t = [rng.integers(0, TINY.vocab, size=int(n)).astype(np.int32) for n in (8, 17, 32, 9)]
    rights = [rng.integers(0, TINY.vocab, size=int(n)).astype(np.int32) for n in (8, 20, 31, 12, 5)]
    root = ctx.set_prefix(root_t)
    kids = [ctx.set_prefix(k, parent=root) for k in kids_t]
    rc = [i for i in range(4) for _ in range(5)]
    rows = [rights[j] for i in range(4) for j in range(5)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    allowed = rng.choice(TINY.vocab, 2, replace=False)
    out, dbg = ctx.eval_rows(np.concatenate(rows), offs, KIND_BOOL, allowed,
                             row_prefix=[kids[i] for i in rc], debug_logits=True)
    ref = orc.eval_rows(root_t, rows, KIND_BOOL, allowed, children=kids_t, row_child=rc,
                        keep_logits=True)
    _log("join", compare(ref, out, dbg, "join"))
    ctx.release_prefix(root)  # children keep it alive
    out2, _ = ctx.eval_rows(np.concatenate(rows), offs, KIND_BOOL, allowed,
                            row_prefix=[kids[i] for i in rc])
    assert np.array_equal(out2, out)
    for k in kids:
        ctx.release_prefix(k)


def test_tiny_batched_children_equal_single(tiny, L):
    """Children made in one lmop_set_prefixes call share a KV store at 8-aligned
    offsets; rows evaluated against them equal, bit for bit, rows evaluated
    against children made one at a time (also rows with no suffix, which read
    the child's stored hidden state), and releasing some keeps the rest valid."""
    w, orc, ctx = tiny
    rng = np.random.default_rng(41)
    root_t = rng.integers(0, TINY.vocab, size=45).astype(np.int32)
    lens = (1, 8, 17, 64, 65, 9, 30)
    kids_t = [rng.integers(0, TINY.vocab, size=n).astype(np.int32) for n in lens]
    root = ctx.set_prefix(root_t)
    single = [ctx.set_prefix(k, parent=root) for k in kids_t]
    _log("batched children: set_prefixes")
    batched = ctx.set_prefixes(kids_t, parent=root)
    rights = [rng.integers(0, TINY.vocab, size=int(n)).astype(np.int32) for n in (0, 7, 23)]
    rc = [i for i in range(len(lens)) for _ in rights]
    rows = [r for _ in lens for r in rights]
    toks = np.concatenate(rows)
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    allowed = rng.choice(TINY.vocab, 3, replace=False)
    o1, d1 = ctx.eval_rows(toks, offs, KIND_ENUM, allowed,
                           row_prefix=[single[i] for i in rc], debug_logits=True)
    o2, d2 = ctx.eval_rows(toks, offs, KIND_ENUM, allowed,
                           row_prefix=[batched[i] for i in rc], debug_logits=True)
    assert o1.tobytes() == o2.tobytes() and np.array_equal(d1, d2)
    ref = orc.eval_rows(root_t, rows, KIND_ENUM, allowed, children=kids_t, row_child=rc,
                        keep_logits=True)
    _log("batched children", compare(ref, o2, d2, "batched children"))
    for i in (0, 3, 5):
        ctx.release_prefix(batched[i])
    keep = [i for i in range(len(lens)) if i not in (0, 3, 5)]
    sel = [j for j, i in enumerate(rc) if i in keep]
    rows_k = [rows[j] for j in sel]
    offs_k = np.concatenate([[0], np.cumsum([len(r) for r in rows_k])])
    o3, d3 = ctx.eval_rows(np.concatenate(rows_k), offs_k, KIND_ENUM, allowed,
                           row_prefix=[batched[rc[j]] for j in sel], debug_logits=True)
    assert o3.tobytes() == o1[sel].tobytes() and np.array_equal(d3, d1[sel])
    for i in keep:
        ctx.release_prefix(batched[i])
    for p in single:
        ctx.release_prefix(p)
    ctx.release_prefix(root)


def test_tiny_int_decode(L):
    w = make_weights(TINY, seed=1234)
    rng = np.random.default_rng(5)
    digits = rng.choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    w.lm_head[eos] *= 3  # make EOS competitive so that numbers of every length appear
    orc = OracleLM(w, TINY)
    ctx = L.Context(TINY, device=0)
    ctx.load_weights(w)
    prefix = rng.integers(0, TINY.vocab, size=40).astype(np.int32)
    rows = [rng.integers(0, TINY.vocab, size=int(rng.integers(1, 40))).astype(np.int32)
            for _ in range(48)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    pre = ctx.set_prefix(prefix)
    out, dbg = ctx.eval_rows(np.concatenate(rows), offs, KIND_INT, digits, eos=eos, max_tokens=4,
                             prefix=pre, debug_logits=True)
    ref = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4, keep_logits=True)
    forced = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4,
                           forced=[out["tokens"][r][: out["n_tokens"][r]] for r in range(48)],
                           keep_logits=True)
    st = compare(ref, out, dbg, "int", orc_forced=forced)
    _log("int decode", st)
    assert_typed(out, KIND_INT, 10, digits, eos, 4)
    lens = set(out["n_tokens"].tolist())
    assert len(lens) >= 2, lens
    # decode steps run per group of batches: the same bits for any batching
    # (40-token batches: several batches per group and several groups), with
    # and without the logit dump (the look-ahead path)
    toks = np.concatenate(rows)
    out_b, dbg_b = ctx.eval_rows(toks, offs, KIND_INT, digits, eos=eos, max_tokens=4,
                                 prefix=pre, debug_logits=True, max_batch_tokens=40)
    assert out_b.tobytes() == out.tobytes()
    assert np.array_equal(dbg_b, dbg, equal_nan=True)
    for mbt in (0, 40, 97):
        out_n, _ = ctx.eval_rows(toks, offs, KIND_INT, digits, eos=eos, max_tokens=4,
                                 prefix=pre, max_batch_tokens=mbt)
        assert out_n.tobytes() == out.tobytes(), mbt
    # the same with the restricted head (digits and EOS only)
    out_r, dbg_r = ctx.eval_rows(np.concatenate(rows), offs, KIND_INT, digits, eos=eos,
                                 max_tokens=4, prefix=pre, debug_logits=True, head_restricted=True)
    forced_r = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4,
                             forced=[out_r["tokens"][r][: out_r["n_tokens"][r]] for r in range(48)],
                             keep_logits=True)
    st_r = compare(ref, out_r, dbg_r, "int restricted", orc_forced=forced_r,
                   cols=list(digits) + [eos])
    _log("int decode, restricted head", st_r)
    assert_typed(out_r, KIND_INT, 10, digits, eos, 4)


def test_tiny_options_automaton(tiny, L):
    """Multi-token options as a token trie: every row's output is one whole
    option, parity with the oracle (teacher-forced where a sub-margin step
    diverged), the restricted head, and any batching giving the same bits."""
    w, orc, ctx = tiny
    wl = make_workload("options_tiny")
    aut = wl.automaton
    pre = ctx.set_prefix(wl.prefix)
    kw = dict(eos=wl.eos, max_tokens=wl.max_tokens, prefix=pre)
    _log("options: eval")
    out, dbg = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, aut, debug_logits=True,
                             **kw)
    assert_automaton(out, aut, wl.eos, wl.max_tokens)
    final = {f: o for o, f in enumerate(_final_states(wl.options, aut))}
    for r in range(wl.n_rows):
        o = final[int(out["value"][r])]
        assert out["tokens"][r][:out["n_tokens"][r]].tolist() == wl.options[o].tolist()
    ref = orc.eval_workload(wl, keep_logits=True)
    forced = orc.eval_rows(wl.prefix, [wl.suffix(r) for r in range(wl.n_rows)], KIND_AUTOMATON,
                           aut, max_tokens=wl.max_tokens, keep_logits=True,
                           forced=[out["tokens"][r][: out["n_tokens"][r]]
                                   for r in range(wl.n_rows)])
    st = compare(ref, out, dbg, "options", orc_forced=forced)
    _log("options", st)
    assert len(set(out["value"].tolist())) >= 3
    # the restricted head computes only the trie's tokens
    out_r, dbg_r = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, aut, debug_logits=True,
                                 head_restricted=True, **kw)
    cols = sorted(set(np.asarray(aut.edge_token).tolist()))
    forced_r = orc.eval_rows(wl.prefix, [wl.suffix(r) for r in range(wl.n_rows)], KIND_AUTOMATON,
                             aut, max_tokens=wl.max_tokens, keep_logits=True,
                             forced=[out_r["tokens"][r][: out_r["n_tokens"][r]]
                                     for r in range(wl.n_rows)])
    _log("options, restricted head",
         compare(ref, out_r, dbg_r, "options restricted", orc_forced=forced_r, cols=cols))
    assert_automaton(out_r, aut, wl.eos, wl.max_tokens)
    # batching does not change a bit
    for mbt in (40, 97):
        o2, d2 = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, aut, debug_logits=True,
                               max_batch_tokens=mbt, **kw)
        assert o2.tobytes() == out.tobytes() and np.array_equal(d2, dbg, equal_nan=True), mbt
    ctx.release_prefix(pre)


@pytest.mark.parametrize("grammar", ["list", "record"])
def test_tiny_list_and_record_grammars(tiny, L, grammar):
    """Collection and JSON-shaped outputs as token automata: a list of 1..3
    items with a separator (quantifier {1,3}) and a two-field record; every
    output is a string of the grammar, parity with the oracle (teacher-forced
    where a sub-margin step diverged), and batching gives the same bits."""
    from synth import automaton_of_list, automaton_of_record
    w, orc, ctx = tiny
    V = TINY.vocab
    rng = np.random.default_rng(57)
    ids = rng.choice(V, size=40, replace=False).astype(np.int32)
    eos = int(ids[0])
    if grammar == "list":
        heads = ids[1:4]
        items = [np.array([heads[0]]), np.array([heads[0], ids[4]]), np.array([heads[1], ids[5]]),
                 np.array([heads[2]]), np.array([ids[6], ids[7]])]
        aut = automaton_of_list(items, sep=int(ids[8]), lo=1, hi=3)
    else:
        aut = automaton_of_record(int(ids[9]), int(ids[10]), int(ids[11]),
                                  [("enum", int(ids[12]), ids[13:18].tolist()),
                                   ("int", int(ids[18]), ids[19:29].tolist(), 2)])
    max_tokens = 8
    wl = make_workload("filter_tiny", n_rows=48)
    pre = ctx.set_prefix(wl.prefix)
    kw = dict(eos=eos, max_tokens=max_tokens, prefix=pre)
    _log(f"{grammar} grammar: eval")
    out, dbg = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, aut, debug_logits=True, **kw)
    assert_automaton(out, aut, eos, max_tokens)
    ref = orc.eval_rows(wl.prefix, [wl.suffix(r) for r in range(wl.n_rows)], KIND_AUTOMATON, aut,
                        eos=eos, max_tokens=max_tokens, keep_logits=True)
    forced = orc.eval_rows(wl.prefix, [wl.suffix(r) for r in range(wl.n_rows)], KIND_AUTOMATON,
                           aut, eos=eos, max_tokens=max_tokens, keep_logits=True,
                           forced=[out["tokens"][r][: out["n_tokens"][r]]
                                   for r in range(wl.n_rows)])
    st = compare(ref, out, dbg, grammar, orc_forced=forced)
    _log(grammar, st)
    assert len(set(map(tuple, out["tokens"].tolist()))) >= 2
    for mbt in (40, 97):
        o2, d2 = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, aut, debug_logits=True,
                               max_batch_tokens=mbt, **kw)
        assert o2.tobytes() == out.tobytes() and np.array_equal(d2, dbg, equal_nan=True), mbt
    ctx.release_prefix(pre)


def _final_states(options, aut):
    off, tok, nxt = (np.asarray(aut.edge_offset), np.asarray(aut.edge_token),
                     np.asarray(aut.edge_next))
    out = []
    for o in options:
        st = 0
        for t in o.tolist():
            edges = tok[off[st]:off[st + 1]].tolist()
            st = int(nxt[off[st] + edges.index(t)])
        out.append(st)
    return out


def test_tiny_automaton_equals_enum_and_int(tiny, L):
    """ENUM and INT written as token automata give the same bits as the
    built-in kinds (value aside: the automaton reports the final state)."""
    from synth import Automaton
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    V = TINY.vocab
    rng = np.random.default_rng(31)
    opts = rng.choice(V, 5, replace=False).astype(np.int32)
    star = Automaton(6, np.array([0, 5, 5, 5, 5, 5, 5], np.int32), opts,
                     np.arange(1, 6, dtype=np.int32), np.array([0, 1, 1, 1, 1, 1], np.uint8))
    e, de = ctx.eval_rows(wl.tokens, wl.offsets, KIND_ENUM, opts, prefix=pre, debug_logits=True)
    a, da = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, star, max_tokens=2,
                          prefix=pre, debug_logits=True)
    for k in ("logprob", "logprob_full", "n_tokens", "tokens"):
        assert np.array_equal(a[k], e[k]), k
    assert np.array_equal(a["value"], e["value"] + 1)
    assert np.array_equal(da[:, :1], de)
    digits = rng.choice(V, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(V) if t not in digits))
    ints = Automaton(5, np.array([0, 10, 20, 30, 40, 40], np.int32), np.tile(digits, 4),
                     np.repeat(np.arange(1, 5, dtype=np.int32), 10),
                     np.array([0, 1, 1, 1, 1], np.uint8))
    i, di = ctx.eval_rows(wl.tokens, wl.offsets, KIND_INT, digits, eos=eos, max_tokens=4,
                          prefix=pre, debug_logits=True)
    a, da = ctx.eval_rows(wl.tokens, wl.offsets, L.LMOP_AUTOMATON, ints, eos=eos, max_tokens=4,
                          prefix=pre, debug_logits=True)
    for k in ("logprob", "logprob_full", "n_tokens", "tokens"):
        assert np.array_equal(a[k], i[k]), k
    assert np.array_equal(da, di, equal_nan=True)
    ctx.release_prefix(pre)


def _take(ref, rows):
    """The oracle's results for the listed rows only."""
    out = {k: np.asarray(v)[rows] for k, v in ref.items() if k != "logits"}
    if "logits" in ref:
        out["logits"] = [ref["logits"][r] for r in rows]
    return out


def _check_limit_vs_oracle(ref, out, dbg, k, v, label):
    """Against the oracle: the k-th row (table order) whose oracle value is v
    is where the scan must stop, and every row up to it is evaluated when the
    oracle's margins there exceed 0.1 (their values are then certain); every
    evaluated row's logits are within the tolerance of the oracle's."""
    ev = np.nonzero(out["n_tokens"] > 0)[0]
    st = compare(_take(ref, ev), out[ev], dbg[ev], label)
    hits = np.nonzero(ref["value"] == v)[0]
    stop = int(hits[k - 1]) if len(hits) >= k else len(out) - 1
    if np.all(ref["margin"][: stop + 1] > 0.1):
        assert np.all(out["n_tokens"][: stop + 1] > 0), f"{label}: a row before the stop skipped"
        assert np.sum(out["value"][ev] == v) >= min(k, len(hits)), label
    return st, stop


def _check_limit(full, out, k, v, label):
    """Rows up to the k-th with value v equal the full evaluation bit for bit;
    later rows are either evaluated (and equal) or marked skipped."""
    hits = np.nonzero(full["value"] == v)[0]
    last = int(hits[k - 1]) if len(hits) >= k else len(full) - 1
    assert out[: last + 1].tobytes() == full[: last + 1].tobytes(), label
    for r in range(last + 1, len(full)):
        if out["n_tokens"][r] == 0:
            assert out["value"][r] == -1 and np.isnan(out["logprob"][r]), label
            assert np.all(out["tokens"][r] == -1), label
        else:
            assert out[r].tobytes() == full[r].tobytes(), label
    return int(np.sum(out["n_tokens"] > 0))


def test_tiny_limit_early_exit(tiny, L):
    """LIMIT k: evaluation stops once k rows (in table order) have the wanted
    value; every row up to the k-th such row is exactly as without a limit."""
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    # duplicates (dedup) and small batches, so the stop comes early
    idx = np.array(list(range(64)) + [3, 3, 10, 5, 63, 0])
    sub = wl.subset(idx)
    full, dfull = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre,
                                max_batch_tokens=64, debug_logits=True)
    ref = orc.eval_workload(sub, keep_logits=True)
    compare(ref, full, dfull, "limit: whole table")
    # the wanted value is the oracle's most frequent one
    v = int(np.bincount(ref["value"]).argmax())
    for k in (1, 4, 9):
        out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre,
                                 max_batch_tokens=64, limit=k, limit_value=v, debug_logits=True)
        n_eval = _check_limit(full, out, k, v, f"limit {k}")
        st, stop = _check_limit_vs_oracle(ref, out, dbg, k, v, f"limit {k} vs oracle")
        _log(f"limit {k}: {n_eval} of {len(idx)} rows evaluated, oracle stop row {stop}, {st}")
        assert n_eval < len(idx)
    # more than the table holds: every row is evaluated
    out, _ = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre,
                           max_batch_tokens=64, limit=len(idx) + 1, limit_value=v)
    assert out.tobytes() == full.tobytes()
    # with the logit dump, skipped rows' logits are NaN
    out, dbg = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre,
                             max_batch_tokens=64, limit=2, limit_value=v, debug_logits=True)
    skipped = out["n_tokens"] == 0
    assert skipped.any() and np.all(np.isnan(dbg[skipped]))
    # integer outputs: the stop waits for each decode group's last step
    digits = np.random.default_rng(3).choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    fi, _ = ctx.eval_rows(sub.tokens, sub.offsets, KIND_INT, digits, eos=eos, max_tokens=3,
                          prefix=pre, max_batch_tokens=64)
    refi = orc.eval_rows(wl.prefix, [sub.suffix(r) for r in range(sub.n_rows)], KIND_INT, digits,
                         eos=eos, max_tokens=3, keep_logits=True)
    vi = int(np.bincount(refi["value"]).argmax())
    oi, di = ctx.eval_rows(sub.tokens, sub.offsets, KIND_INT, digits, eos=eos, max_tokens=3,
                           prefix=pre, max_batch_tokens=64, limit=2, limit_value=vi,
                           debug_logits=True)
    _check_limit(fi, oi, 2, vi, "int limit")
    ev = np.nonzero(oi["n_tokens"] > 0)[0]
    if all(list(oi["tokens"][r][: oi["n_tokens"][r]]) == list(refi["tokens"][r][: refi["n_tokens"][r]])
           for r in ev):
        _check_limit_vs_oracle(refi, oi, di, 2, vi, "int limit vs oracle")
    ctx.release_prefix(pre)


def test_tiny_llmqa_long_prompt(tiny, L):
    """LLMQA (one prompt holding a whole data subset): two 1,596-token
    prompts, each one row, against the oracle; one row per batch (a budget
    below the row's length) gives the same bits."""
    w, orc, ctx = tiny
    wl = make_workload("qa_tiny")
    pre = ctx.set_prefix(wl.prefix)
    kw = dict(eos=wl.eos, max_tokens=wl.max_tokens, prefix=pre, debug_logits=True)
    _log("llmqa: eval")
    out, dbg = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.automaton, **kw)
    assert_automaton(out, wl.automaton, wl.eos, wl.max_tokens)
    ref = orc.eval_workload(wl, keep_logits=True)
    forced = orc.eval_workload(wl, keep_logits=True,
                               forced=[out["tokens"][r][: out["n_tokens"][r]]
                                       for r in range(wl.n_rows)])
    _log("llmqa", compare(ref, out, dbg, "llmqa", orc_forced=forced))
    o1, d1 = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.automaton, max_batch_tokens=700,
                           **kw)
    assert o1.tobytes() == out.tobytes() and np.array_equal(d1, dbg, equal_nan=True)
    ctx.release_prefix(pre)


def test_tiny_cascade_row_mask(tiny, L):
    """Cascade filtering: a second predicate evaluated only on the rows the
    first one kept equals that predicate on those rows alone, bit for bit;
    the other rows are skipped (also with duplicates and a LIMIT)."""
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    idx = np.array(list(range(64)) + [3, 3, 10, 5, 63, 0])
    sub = wl.subset(idx)
    first, _ = ctx.eval_rows(sub.tokens, sub.offsets, sub.kind, sub.allowed, prefix=pre)
    keep = first["value"] == 1
    assert 0 < keep.sum() < len(idx)
    # the first predicate's mask agrees with the oracle's wherever the
    # oracle's margin decides it
    ref1 = orc.eval_workload(sub)
    sure = ref1["margin"] > 0.1
    assert np.array_equal(keep[sure], ref1["value"][sure] == 1)
    opts2 = np.random.default_rng(41).choice(TINY.vocab, 6, replace=False).astype(np.int32)
    second, d2 = ctx.eval_rows(sub.tokens, sub.offsets, KIND_ENUM, opts2, prefix=pre,
                               row_mask=keep, debug_logits=True)
    # the rows the mask keeps against the oracle's second predicate on them
    kept_rows = np.nonzero(keep)[0]
    ref2 = orc.eval_rows(wl.prefix, [sub.suffix(int(r)) for r in kept_rows], KIND_ENUM, opts2,
                         keep_logits=True)
    _log("cascade second predicate vs oracle",
         compare(ref2, second[kept_rows], d2[kept_rows], "cascade second"))
    alone = sub.subset(np.nonzero(keep)[0])
    ref, dref = ctx.eval_rows(alone.tokens, alone.offsets, KIND_ENUM, opts2, prefix=pre,
                              debug_logits=True)
    assert second[keep].tobytes() == ref.tobytes()
    assert np.array_equal(d2[keep], dref)
    sk = second[~keep]
    assert np.all(sk["value"] == -1) and np.all(sk["n_tokens"] == 0)
    assert np.all(np.isnan(sk["logprob"])) and np.all(np.isnan(d2[~keep]))
    # with a limit: the mask's rows in table order, stopping at the k-th hit
    v = int(np.bincount(ref["value"]).argmax())
    lim, _ = ctx.eval_rows(sub.tokens, sub.offsets, KIND_ENUM, opts2, prefix=pre, row_mask=keep,
                           limit=2, limit_value=v, max_batch_tokens=64)
    kept = np.nonzero(keep)[0]
    hits = kept[second["value"][kept] == v]
    stop = int(hits[1]) if len(hits) >= 2 else len(idx) - 1
    head = [r for r in kept if r <= stop]
    assert lim[head].tobytes() == second[head].tobytes()
    assert np.all(lim["n_tokens"][~keep] == 0)
    ctx.release_prefix(pre)


@pytest.fixture(scope="module")
def tiny_fp8(L):
    w = make_weights(TINY, seed=1234, fmt="fp8_e4m3")
    orc = OracleLM(w, TINY)
    ctx = L.Context(TINY, device=0)
    ctx.load_weights(w)
    return w, orc, ctx


def test_tiny_fp8_weights(tiny_fp8, L):
    """FP8 (E4M3, per-channel scale) weights: the filter, an integer decode
    and a two-level join against the oracle of the same FP8 weights; batching
    does not change a bit; device-resident weights load the same."""
    w, orc, ctx = tiny_fp8
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    _log("fp8: filter")
    out, dbg = _run(ctx, wl, pre)
    ref = orc.eval_workload(wl, keep_logits=True)
    _log("fp8 filter", compare(ref, out, dbg, "fp8 filter"))
    assert_typed(out, wl.kind, len(wl.allowed), wl.allowed)
    o2, d2 = _run(ctx, wl, pre, max_batch_tokens=50)
    assert o2.tobytes() == out.tobytes() and np.array_equal(d2, dbg)
    rng = np.random.default_rng(8)
    digits = rng.choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    rows = [wl.suffix(r) for r in range(24)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    oi, di = ctx.eval_rows(np.concatenate(rows), offs, KIND_INT, digits, eos=eos, max_tokens=3,
                           prefix=pre, debug_logits=True)
    ri = orc.eval_rows(wl.prefix, rows, KIND_INT, digits, eos=eos, max_tokens=3, keep_logits=True)
    fi = orc.eval_rows(wl.prefix, rows, KIND_INT, digits, eos=eos, max_tokens=3, keep_logits=True,
                       forced=[oi["tokens"][r][: oi["n_tokens"][r]] for r in range(24)])
    _log("fp8 int", compare(ri, oi, di, "fp8 int", orc_forced=fi))
    kids = ctx.set_prefixes([wl.suffix(40)[:9], wl.suffix(41)[:20]], parent=pre)
    jrows = [wl.suffix(r) for r in range(6)]
    rc = [0, 1, 0, 1, 1, 0]
    jo, jd = ctx.eval_rows(np.concatenate(jrows), np.concatenate([[0], np.cumsum([len(r) for r in jrows])]),
                           KIND_BOOL, wl.allowed, row_prefix=[kids[i] for i in rc],
                           debug_logits=True)
    jr = orc.eval_rows(wl.prefix, jrows, KIND_BOOL, wl.allowed,
                       children=[wl.suffix(40)[:9], wl.suffix(41)[:20]], row_child=rc,
                       keep_logits=True)
    _log("fp8 join", compare(jr, jo, jd, "fp8 join"))
    for k in kids:
        ctx.release_prefix(k)
    ctx.release_prefix(pre)
    # the same weights from device memory
    ctx2 = L.Context(TINY, device=0)
    ctx2.load_weights(w.to("cuda:0"))
    p2 = ctx2.set_prefix(wl.prefix)
    o3, d3 = _run(ctx2, wl, p2)
    assert o3.tobytes() == out.tobytes() and np.array_equal(d3, dbg)
    ctx2.close()


@pytest.mark.parametrize("seed", [101, 202, 303])
def test_tiny_mixed_features_random(tiny, L, seed):
    """Seeded mixes of the features in one call: rows under a root prefix, a
    child prefix or none, empty suffixes, duplicates, one of the four output
    types, the full or restricted head and a random batch budget, against the
    oracle (typed outputs exact where the margin allows)."""
    from synth import automaton_of_options
    w, orc, ctx = tiny
    V = TINY.vocab
    rng = np.random.default_rng(seed)
    root_t = rng.integers(0, V, size=int(rng.integers(1, 150))).astype(np.int32)
    kid_t = rng.integers(0, V, size=int(rng.integers(1, 70))).astype(np.int32)
    root = ctx.set_prefix(root_t)
    kid = ctx.set_prefixes([kid_t], parent=root)[0]
    n = int(rng.integers(8, 40))
    where = rng.integers(0, 3, size=n)  # 0: none, 1: root, 2: child
    rows = []
    for r in range(n):
        lo = 1 if where[r] == 0 else 0
        rows.append(rng.integers(0, V, size=int(rng.integers(lo, 90))).astype(np.int32))
    for r in rng.choice(n, size=min(4, n - 1), replace=False):  # duplicates
        rows[r], where[r] = rows[0].copy(), where[0]
    offs = np.concatenate([[0], np.cumsum([len(x) for x in rows])])
    toks = np.concatenate(rows) if offs[-1] else np.zeros(0, np.int32)
    rp = [None if where[r] == 0 else (root if where[r] == 1 else kid) for r in range(n)]
    kind = int(rng.integers(0, 4))
    eos, max_tokens, spec = -1, 1, None
    if kind == KIND_BOOL:
        spec = rng.choice(V, 2, replace=False).astype(np.int32)
    elif kind == KIND_ENUM:
        spec = rng.choice(V, int(rng.integers(1, 30)), replace=False).astype(np.int32)
    elif kind == KIND_INT:
        spec = rng.choice(V, 10, replace=False).astype(np.int32)
        eos = int(next(t for t in range(V) if t not in spec))
        max_tokens = int(rng.integers(1, 5))
    else:
        _, spec, _ = automaton_of_options(int(rng.integers(2, 20)), V, rng, max_len=3)
        max_tokens = 3
    restricted = bool(rng.integers(0, 2))
    mbt = int(rng.choice([0, 40, 120]))
    _log(f"seed {seed}: {n} rows, kind {kind}, restricted {restricted}, budget {mbt}")
    out, dbg = ctx.eval_rows(toks, offs, kind, spec, eos=eos, max_tokens=max_tokens,
                             row_prefix=rp, debug_logits=True, head_restricted=restricted,
                             max_batch_tokens=mbt)
    # the oracle, per prefix level
    for lvl in range(3):
        idx = [r for r in range(n) if where[r] == lvl]
        if not idx:
            continue
        kw = dict(eos=eos, max_tokens=max_tokens, keep_logits=True)
        pre = None if lvl == 0 else root_t
        ch = dict(children=[kid_t], row_child=[0] * len(idx)) if lvl == 2 else {}
        sub = [rows[r] for r in idx]
        ref = orc.eval_rows(pre, sub, kind, spec, **kw, **ch)
        forced = orc.eval_rows(pre, sub, kind, spec, **kw, **ch,
                               forced=[out["tokens"][r][: out["n_tokens"][r]] for r in idx])
        cols = None
        if restricted:
            cols = (sorted(set(np.asarray(spec.edge_token).tolist())) if kind == 3
                    else list(spec) + ([eos] if kind == KIND_INT else []))
        _log(f"  level {lvl}", compare(ref, out[idx], dbg[idx], f"seed {seed} level {lvl}",
                                       orc_forced=forced, cols=cols))
    ctx.release_prefix(kid)
    ctx.release_prefix(root)


def test_tiny_sampled_profiling(tiny, L):
    """Kernel timing on a sample: every launch is counted, the first and then
    every period-th launch of each kernel is timed; the results do not
    change."""
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny", n_rows=40)
    pre = ctx.set_prefix(wl.prefix)
    ref, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre,
                           max_batch_tokens=97)
    counts = {}
    for period in (1, 3):
        ctx.set_profiling(period)
        out, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre,
                               max_batch_tokens=97)
        st = ctx.kernel_stats()
        ctx.set_profiling(0)
        assert out.tobytes() == ref.tobytes()
        for name, s in st.items():
            assert s["timed"] == (s["launches"] + period - 1) // period, (name, s)
            assert s["ms"] > 0 and s["flops"] >= 0
        counts[period] = {k: v["launches"] for k, v in st.items()}
    assert counts[1] == counts[3] and counts[1]["gemm_w4a16_qkv"] >= 2 * TINY.n_layers
    ctx.release_prefix(pre)


@pytest.mark.parametrize("n_rows", [300, 600])
def test_ragged_vocab_and_wide_batch(L, n_rows):
    """A vocabulary that is not a multiple of the head's 128-entry chunk
    (1,999 = 15 x 128 + 79) and a batch of 300 or 600 rows, which the head
    covers with one or two 320-token tiles (the second partly filled):
    logits and typed outputs against the oracle, every row; the same bits
    when the rows are batched in small pieces, which take the 256-token tile."""
    shape = dataclasses.replace(TINY, name="tiny_v1999", vocab=1999, n_layers=1, shape_id=7)
    w = make_weights(shape, seed=99)
    orc = OracleLM(w, shape)
    ctx = L.Context(shape, device=0)
    ctx.load_weights(w)
    rng = np.random.default_rng(12)
    prefix = rng.integers(0, shape.vocab, size=40).astype(np.int32)
    rows = [rng.integers(0, shape.vocab, size=int(rng.integers(1, 6))).astype(np.int32)
            for _ in range(n_rows)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    toks = np.concatenate(rows)
    # allowed tokens include the last vocabulary entries (the ragged chunk)
    allowed = np.array([1998, 1990, 1920, 5, 700], dtype=np.int32)
    pre = ctx.set_prefix(prefix)
    _log(f"ragged vocab: eval {n_rows} rows in one batch")
    out, dbg = ctx.eval_rows(toks, offs, KIND_ENUM, allowed, prefix=pre, debug_logits=True,
                             no_dedup=True)
    ref = orc.eval_rows(prefix, rows, KIND_ENUM, allowed, keep_logits=True)
    st = compare(ref, out, dbg, "ragged vocab")
    _log("ragged vocab", st)
    assert st["exact_checked"] >= n_rows // 2
    assert_typed(out, KIND_ENUM, len(allowed), allowed)
    o2, d2 = ctx.eval_rows(toks, offs, KIND_ENUM, allowed, prefix=pre, debug_logits=True,
                           no_dedup=True, max_batch_tokens=37)
    assert o2.tobytes() == out.tobytes() and np.array_equal(d2, dbg)
    ctx.release_prefix(pre)
    ctx.close()


def test_head_dim_128_attention(L):
    """Attention with 128-dimensional heads (the 8B head width) at a small
    size: grouped queries (G = 2), a root and a child prefix, rows long
    enough for several 128-vector query tiles, against the oracle; the same
    bits for any batching."""
    shape = dataclasses.replace(TINY, name="tiny_hd128", n_heads=2, n_kv_heads=1, head_dim=128,
                                shape_id=8)
    w = make_weights(shape, seed=5)
    orc = OracleLM(w, shape)
    ctx = L.Context(shape, device=0)
    ctx.load_weights(w)
    rng = np.random.default_rng(21)
    root_t = rng.integers(0, shape.vocab, size=100).astype(np.int32)
    kid_t = rng.integers(0, shape.vocab, size=37).astype(np.int32)
    root = ctx.set_prefix(root_t)
    kid = ctx.set_prefixes([kid_t], parent=root)[0]
    lens = [1, 2, 63, 64, 65, 130, 7, 90, 150, 33, 0, 5]
    rows = [rng.integers(0, shape.vocab, size=n).astype(np.int32) for n in lens]
    offs = np.concatenate([[0], np.cumsum(lens)])
    toks = np.concatenate(rows)
    allowed = rng.choice(shape.vocab, 6, replace=False).astype(np.int32)
    for pre, label, kw in ((root, "root", {}), (kid, "child",
                                                 dict(children=[kid_t], row_child=[0] * len(rows)))):
        _log(f"hd 128, {label} prefix: eval")
        out, dbg = ctx.eval_rows(toks, offs, KIND_ENUM, allowed, prefix=pre, debug_logits=True,
                                 no_dedup=True)
        ref = orc.eval_rows(root_t, rows, KIND_ENUM, allowed, keep_logits=True, **kw)
        _log(f"hd 128 {label}", compare(ref, out, dbg, f"hd 128 {label}"))
        o2, d2 = ctx.eval_rows(toks, offs, KIND_ENUM, allowed, prefix=pre, debug_logits=True,
                               no_dedup=True, max_batch_tokens=70)
        assert o2.tobytes() == out.tobytes() and np.array_equal(d2, dbg)
    ctx.release_prefix(kid)
    ctx.release_prefix(root)
    ctx.close()


def test_tiny_max_sizes(tiny, L):
    """Maximum sizes: an integer type with max_tokens = 8 (numbers of up to 8
    digits fill the result's token array), and 2,100 one-to-three-token rows
    (more than one batch's 2,048-row cap; the LM head runs eight 256-row
    column tiles); against the oracle."""
    w, orc, ctx = tiny
    rng = np.random.default_rng(77)
    prefix = rng.integers(0, TINY.vocab, size=20).astype(np.int32)
    pre = ctx.set_prefix(prefix)
    digits = rng.choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    rows = [rng.integers(0, TINY.vocab, size=int(rng.integers(1, 12))).astype(np.int32)
            for _ in range(24)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    _log("max sizes: 8-digit integers")
    out, dbg = ctx.eval_rows(np.concatenate(rows), offs, KIND_INT, digits, eos=eos, max_tokens=8,
                             prefix=pre, debug_logits=True)
    ref = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=8, keep_logits=True)
    forced = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=8, keep_logits=True,
                           forced=[out["tokens"][r][: out["n_tokens"][r]] for r in range(24)])
    _log("max_tokens 8", compare(ref, out, dbg, "max_tokens 8", orc_forced=forced))
    assert_typed(out, KIND_INT, 10, digits, eos=eos, max_tokens=8)
    assert int(np.max(out["n_tokens"])) == 8
    _log("max sizes: 2,100 rows")
    rows = [rng.integers(0, TINY.vocab, size=int(rng.integers(1, 4))).astype(np.int32)
            for _ in range(2100)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    allowed = rng.choice(TINY.vocab, 5, replace=False).astype(np.int32)
    out, dbg = ctx.eval_rows(np.concatenate(rows), offs, KIND_ENUM, allowed, prefix=pre,
                             debug_logits=True, no_dedup=True)
    ref = orc.eval_rows(prefix, rows, KIND_ENUM, allowed, keep_logits=True)
    st = compare(ref, out, dbg, "2100 rows")
    _log("2100 rows", st)
    assert st["exact_checked"] >= 1000
    ctx.release_prefix(pre)


def test_tiny_restricted_head(tiny, L):
    """Restricted head: only the allowed tokens' logits are computed; typed
    outputs and allowed-set log-probabilities match the oracle and the full
    head, logprob_full is NaN."""
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    out, dbg = _run(ctx, wl, pre, head_restricted=True)
    ref = orc.eval_workload(wl, keep_logits=True)
    st = compare(ref, out, dbg, "restricted", cols=wl.allowed)
    _log("restricted head", st)
    assert st["exact_checked"] >= 32
    assert_typed(out, wl.kind, 2, wl.allowed)
    full, _ = _run(ctx, wl, pre)
    clear = ref["margin"] > 0.1
    assert np.array_equal(out["value"][clear], full["value"][clear])
    assert np.allclose(out["logprob"], full["logprob"], atol=1e-3)
    ctx.release_prefix(pre)


def test_tiny_prefix_cached_equals_inlined(tiny, L):
    """Prefix reuse changes nothing but cost: the rows evaluated against a
    cached prefix agree with the same rows carrying the prefix tokens
    inline (and with the oracle's full forward)."""
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny", n_rows=24)
    pre = ctx.set_prefix(wl.prefix)
    cached, dc = _run(ctx, wl, pre)
    rows = [np.concatenate([wl.prefix, wl.suffix(r)]) for r in range(wl.n_rows)]
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    inl, di = ctx.eval_rows(np.concatenate(rows), offs, wl.kind, wl.allowed, debug_logits=True)
    ref = orc.eval_workload(wl, keep_logits=True)
    _log("cached", compare(ref, cached, dc, "cached"))
    _log("inlined", compare(ref, inl, di, "inlined"))
    sigma = float(np.std(dc))
    assert np.abs(dc - di).max() <= 0.05 * sigma
    clear = ref["margin"] > 0.1
    assert np.array_equal(cached["value"][clear], inl["value"][clear])
    ctx.release_prefix(pre)


def test_tiny_edge_cases(tiny, L):
    """A single allowed option (log-probability exactly 0), a one-token
    integer, a 300-token row beside one-token rows under a batch budget
    smaller than the long row, and rows with and without a prefix in one call."""
    w, orc, ctx = tiny
    V = TINY.vocab
    rng = np.random.default_rng(11)
    prefix = rng.integers(0, V, size=130).astype(np.int32)
    pre = ctx.set_prefix(prefix)
    rows = [rng.integers(0, V, size=n).astype(np.int32) for n in (300, 1, 1, 17, 64)]
    toks = np.concatenate(rows)
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])

    one = [int(rng.integers(0, V))]
    out, dbg = ctx.eval_rows(toks, offs, KIND_ENUM, one, prefix=pre, debug_logits=True,
                             max_batch_tokens=100)
    assert np.all(out["value"] == 0) and np.all(out["logprob"] == 0.0)
    ref = orc.eval_rows(prefix, rows, KIND_ENUM, one, keep_logits=True)
    _log("one option", compare(ref, out, dbg, "one option"))

    digits = rng.choice(V, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(V) if t not in digits))
    out1, dbg1 = ctx.eval_rows(toks, offs, KIND_INT, digits, eos=eos, max_tokens=1, prefix=pre,
                               debug_logits=True)
    ref1 = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=1, keep_logits=True)
    _log("int, one token", compare(ref1, out1, dbg1, "int, one token"))
    assert np.all(out1["n_tokens"] == 1)
    assert_typed(out1, KIND_INT, 10, digits, eos, 1)

    allowed = rng.choice(V, 2, replace=False).astype(np.int32)
    with_p, without_p = [0, 2, 4], [1, 3]
    rp = [pre if i in with_p else None for i in range(len(rows))]
    outm, dbgm = ctx.eval_rows(toks, offs, KIND_BOOL, allowed, row_prefix=rp, debug_logits=True)
    refa = orc.eval_rows(prefix, [rows[i] for i in with_p], KIND_BOOL, allowed, keep_logits=True)
    refb = orc.eval_rows(None, [rows[i] for i in without_p], KIND_BOOL, allowed, keep_logits=True)
    _log("mixed, with prefix", compare(refa, outm[with_p], dbgm[with_p], "mixed, with prefix"))
    _log("mixed, no prefix", compare(refb, outm[without_p], dbgm[without_p], "mixed, no prefix"))
    ctx.release_prefix(pre)


def test_tiny_row_at_max_seq(tiny, L):
    """A row whose last decode step sits at position max_seq - 1 (the last
    RoPE table entry and KV slot), under a batch budget smaller than the row."""
    w, orc, _ = tiny
    V, max_seq = TINY.vocab, 600
    ctx = L.Context(TINY, device=0, max_seq=max_seq)
    ctx.load_weights(w)
    rng = np.random.default_rng(12)
    prefix = rng.integers(0, V, size=130).astype(np.int32)
    pre = ctx.set_prefix(prefix)
    digits = rng.choice(V, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(V) if t not in digits))
    rows = [rng.integers(0, V, size=n).astype(np.int32) for n in (max_seq - 130 - 3, 5)]
    toks = np.concatenate(rows)
    offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
    _log("max_seq row: eval")
    out, dbg = ctx.eval_rows(toks, offs, KIND_INT, digits, eos=eos, max_tokens=4, prefix=pre,
                             debug_logits=True, max_batch_tokens=64)
    ref = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4, keep_logits=True)
    forced = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4,
                           forced=[out["tokens"][r][: out["n_tokens"][r]] for r in range(2)],
                           keep_logits=True)
    _log("max_seq row", compare(ref, out, dbg, "max_seq row", orc_forced=forced))
    assert_typed(out, KIND_INT, 10, digits, eos, 4)
    # one token more does not fit
    long_row = np.concatenate([rows[0], [1]]).astype(np.int32)
    with pytest.raises(L.LmopError):
        ctx.eval_rows(long_row, [0, len(long_row)], KIND_INT, digits, eos=eos, max_tokens=4,
                      prefix=pre)
    ctx.release_prefix(pre)


def test_tiny_dedup_and_batch_invariance(tiny, L):
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    # a table with duplicated rows
    idx = np.array([0, 5, 0, 7, 5, 5, 9, 0, 63, 9])
    sub = wl.subset(idx)
    o1, d1 = _run(ctx, sub, pre)
    o2, d2 = _run(ctx, sub, pre, no_dedup=True)
    o3, d3 = _run(ctx, sub, pre, max_batch_tokens=17)  # one row per batch
    _log("dedup vs no-dedup per-row max|dz|:", np.abs(d1 - d2).max(axis=(1, 2)))
    _log("dedup vs one-row batches per-row max|dz|:", np.abs(d1 - d3).max(axis=(1, 2)))
    assert np.array_equal(o1, o2) and np.array_equal(d1, d2)
    assert np.array_equal(o1, o3) and np.array_equal(d1, d3)
    for a, b in [(0, 2), (0, 7), (1, 4), (1, 5), (6, 9)]:
        assert np.array_equal(o1[a], o1[b])
    # results do not depend on the other rows of the call
    full, dfull = _run(ctx, wl, pre)
    for j, r in enumerate(idx):
        assert np.array_equal(full[r], o1[j]) and np.array_equal(dfull[r], d1[j])
    # nor on the row order
    perm = np.random.default_rng(6).permutation(wl.n_rows)
    pw = wl.subset(perm)
    op, dp = _run(ctx, pw, pre)
    assert np.array_equal(op, full[perm]) and np.array_equal(dp, dfull[perm])
    ctx.release_prefix(pre)


def test_tiny_workspace(tiny, L):
    """Scratch carved from a caller's torch allocation: the same bits as
    library-allocated scratch, also when the workspace is small enough to
    force smaller batches and decode groups; the library allocates no scratch
    of its own meanwhile; a workspace too small for one row is LMOP_ERR_OOM
    with a readable message."""
    w, orc, ref_ctx = tiny
    wl = make_workload("filter_tiny")
    digits = np.random.default_rng(3).choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    pre_ref = ref_ctx.set_prefix(wl.prefix)
    want_b, dwant_b = ref_ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre_ref,
                                        debug_logits=True)
    want_i, dwant_i = ref_ctx.eval_rows(wl.tokens, wl.offsets, KIND_INT, digits, eos=eos,
                                        max_tokens=4, prefix=pre_ref, debug_logits=True)
    ref_ctx.release_prefix(pre_ref)
    ctx = L.Context(TINY, device=0, stream=torch.cuda.current_stream().cuda_stream)
    ctx.load_weights(w)
    held = ctx.memory()["device_bytes"]  # weights and the rotary table
    for mib in (64, 2):
        # NaN bit patterns everywhere: whatever must start at zero is cleared
        buf = torch.full((mib << 18,), float("nan"), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        ctx.set_workspace(buf.data_ptr(), buf.numel() * 4)
        pre = ctx.set_prefix(wl.prefix)
        with_prefix = ctx.memory()["device_bytes"]
        got_b, dgot_b = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre,
                                      debug_logits=True)
        got_i, dgot_i = ctx.eval_rows(wl.tokens, wl.offsets, KIND_INT, digits, eos=eos,
                                      max_tokens=4, prefix=pre, debug_logits=True)
        assert got_b.tobytes() == want_b.tobytes() and np.array_equal(dgot_b, dwant_b), mib
        assert got_i.tobytes() == want_i.tobytes(), mib
        assert np.array_equal(dgot_i, dwant_i, equal_nan=True), mib
        mem = ctx.memory()
        assert mem["device_bytes"] == with_prefix  # no scratch of the library's own
        assert 0 < mem["workspace_peak"] <= mem["workspace_bytes"] == mib << 20
        _log(f"workspace {mib} MiB: peak {mem['workspace_peak']} bytes, library holds "
             f"{mem['device_bytes']} (weights {held})")
        ctx.release_prefix(pre)
        ctx.set_workspace(0, 0)
        del buf
    small = torch.empty(1 << 14, dtype=torch.float32, device="cuda")
    ctx.set_workspace(small.data_ptr(), small.numel() * 4)
    pre = None
    with pytest.raises(L.LmopError) as ei:
        pre = ctx.set_prefix(wl.prefix)
    assert ei.value.status == L.LMOP_ERR_OOM and "workspace" in str(ei.value)
    ctx.set_workspace(0, 0)
    pre = ctx.set_prefix(wl.prefix)
    ctx.set_workspace(small.data_ptr(), small.numel() * 4)
    with pytest.raises(L.LmopError) as ei:
        ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre)
    assert ei.value.status == L.LMOP_ERR_OOM and "bytes" in str(ei.value)
    # the ctx stays usable after the failed call
    ctx.set_workspace(0, 0)
    again, _ = ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre)
    assert again.tobytes() == want_b.tobytes()
    ctx.release_prefix(pre)
    ctx.close()


@pytest.mark.gpu
def test_tiny_device_error_is_sticky(tiny, L, monkeypatch):
    """A HIP launch failure in the middle of a forward pass (forced from the
    host: the library's launch-failure hook fails the 3rd attention launch
    without launching it) returns LMOP_ERR_DEVICE naming the kernel; every
    later call on that ctx is refused with the same status and the first
    cause; a fresh ctx on the same device still gives the reference bits."""
    w, orc, ref_ctx = tiny
    wl = make_workload("filter_tiny")
    pre_ref = ref_ctx.set_prefix(wl.prefix)
    want = ref_ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre_ref)
    ref_ctx.release_prefix(pre_ref)
    monkeypatch.setenv("LMOP_INJECT_LAUNCH_FAILURE", "attention:3")
    ctx = L.Context(TINY, device=0, stream=torch.cuda.current_stream().cuda_stream)
    monkeypatch.delenv("LMOP_INJECT_LAUNCH_FAILURE")
    ctx.load_weights(w)
    pre = ctx.set_prefix(wl.prefix)  # two attention launches (two layers)
    with pytest.raises(L.LmopError) as ei:
        ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre)
    assert ei.value.status == L.LMOP_ERR_DEVICE
    assert "attention" in str(ei.value) and "injected" in str(ei.value)
    for call in (lambda: ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre),
                 lambda: ctx.set_prefix(wl.prefix)):
        with pytest.raises(L.LmopError) as ei2:
            call()
        assert ei2.value.status == L.LMOP_ERR_DEVICE
        assert "earlier error" in str(ei2.value) and "injected" in str(ei2.value)
    ctx.close()
    fresh = L.Context(TINY, device=0, stream=torch.cuda.current_stream().cuda_stream)
    fresh.load_weights(w)
    pre = fresh.set_prefix(wl.prefix)
    got = fresh.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre)
    assert got[0].tobytes() == want[0].tobytes()
    fresh.close()


@pytest.mark.gpu
def test_tiny_min_workspace_runs(tiny, L):
    """A workspace of exactly the size lmop_plan_rows names as the minimum
    runs the call on the GPU (one row per pass at this size), with results
    equal bit for bit to library-allocated scratch, for a yes/no and an
    integer type; the plan of a single-step call on a device ctx equals the
    host-only ctx's."""
    w, orc, ref_ctx = tiny
    wl = make_workload("filter_tiny")
    digits = np.random.default_rng(3).choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    cases = [((wl.tokens, wl.offsets, wl.kind, wl.allowed), {}),
             ((wl.tokens, wl.offsets, KIND_INT, digits), dict(eos=eos, max_tokens=4))]
    pre_ref = ref_ctx.set_prefix(wl.prefix)
    wants = [ref_ctx.eval_rows(*a, prefix=pre_ref, debug_logits=True, **k) for a, k in cases]
    ref_ctx.release_prefix(pre_ref)
    host = L.Context(TINY, device=-1)
    host.load_weights(w)
    ctx = L.Context(TINY, device=0, stream=torch.cuda.current_stream().cuda_stream)
    ctx.load_weights(w)
    a0, k0 = cases[0]
    assert ctx.plan_rows(*a0, **k0) == host.plan_rows(*a0, **k0)
    pre = ctx.set_prefix(wl.prefix)
    for (a, k), (want, dwant) in zip(cases, wants):
        plan = ctx.plan_rows(*a, prefix=pre, debug_logits=True, **k)
        need = plan["min_workspace_bytes"]
        buf = torch.full((need // 4 + 64,), float("nan"), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        ctx.set_workspace(buf.data_ptr(), need)
        small = ctx.plan_rows(*a, prefix=pre, debug_logits=True, **k)
        got, dgot = ctx.eval_rows(*a, prefix=pre, debug_logits=True, **k)
        ctx.set_workspace(0, 0)
        del buf
        _log(f"minimum workspace {need} bytes: {small['batches']} passes "
             f"(library scratch: {plan['batches']} passes, {plan['scratch_bytes']} bytes)")
        assert small["batches"] > plan["batches"]
        assert got.tobytes() == want.tobytes()
        assert np.array_equal(dgot, dwant, equal_nan=True)
    ctx.close()
    host.close()


@pytest.mark.gpu
def test_tiny_plan_matches_run(tiny, L):
    """lmop_plan_rows describes what the call then does: every forward pass
    launches the embedding once, so a single-step call launches it once per
    planned pass; an integer call adds, per decode group, between one and
    max_tokens - 1 decode passes."""
    w, orc, ctx = tiny
    wl = make_workload("filter_tiny")
    pre = ctx.set_prefix(wl.prefix)
    digits = np.random.default_rng(3).choice(TINY.vocab, 10, replace=False).astype(np.int32)
    eos = int(next(t for t in range(TINY.vocab) if t not in digits))
    for budget in (97, 300, 0):
        plan = ctx.plan_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre,
                             max_batch_tokens=budget)
        ctx.set_profiling(1)
        ctx.eval_rows(wl.tokens, wl.offsets, wl.kind, wl.allowed, prefix=pre,
                      max_batch_tokens=budget)
        st = ctx.kernel_stats()
        ctx.set_profiling(0)
        assert st["embed"]["launches"] == plan["batches"], (budget, plan)
        plan_i = ctx.plan_rows(wl.tokens, wl.offsets, KIND_INT, digits, eos=eos, max_tokens=4,
                               prefix=pre, max_batch_tokens=budget)
        ctx.set_profiling(1)
        ctx.eval_rows(wl.tokens, wl.offsets, KIND_INT, digits, eos=eos, max_tokens=4, prefix=pre,
                      max_batch_tokens=budget)
        st = ctx.kernel_stats()
        ctx.set_profiling(0)
        n = st["embed"]["launches"]
        g = plan_i["decode_groups"]
        assert plan_i["batches"] + g <= n <= plan_i["batches"] + 3 * g, (budget, plan_i, n)
        _log(f"budget {budget}: {plan['batches']} passes; integer: {plan_i['batches']} passes, "
             f"{g} decode groups, {n} forward passes run")
    ctx.release_prefix(pre)
