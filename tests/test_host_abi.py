"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every call its header declares, validates arguments and deduplicates rows."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2606_31808_amd import lmop as L
from synth import SHAPES, make_weights

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TINY = SHAPES["tiny"]


def test_header_declarations_are_exported():
    with open(os.path.join(ROOT, "include", "lmop.h")) as f:
        hdr = f.read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    declared = set(re.findall(r"\b(lmop_[a-z_]+)\s*\(", hdr))
    assert declared == set(L.EXPORTED)
    lib = C.CDLL(L.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name


def test_status_strings():
    for st in (0, -1, -2, -3, -4, -5):
        assert L._lib.lmop_status_string(st)


def _host_ctx(shape=TINY):
    return L.Context(shape, device=-1)


def _expect(status, fn, *a, **k):
    with pytest.raises(L.LmopError) as ei:
        fn(*a, **k)
    assert ei.value.status == status, str(ei.value)
    return str(ei.value)


def test_config_validation():
    base = L.config_from_shape(TINY)
    for field, val, st in [("head_dim", 96, L.LMOP_ERR_UNSUPPORTED),
                           ("n_kv_heads", 3, L.LMOP_ERR_UNSUPPORTED),
                           ("d_model", 200, L.LMOP_ERR_UNSUPPORTED),
                           ("group_size", 64, L.LMOP_ERR_UNSUPPORTED),
                           ("max_seq", (1 << 20) + 1, L.LMOP_ERR_UNSUPPORTED),
                           ("max_seq", -1, L.LMOP_ERR_INVALID_ARG),
                           ("vocab", 0, L.LMOP_ERR_INVALID_ARG),
                           ("d_ff", -1, L.LMOP_ERR_INVALID_ARG)]:
        cfg = L.lmop_config.from_buffer_copy(base)
        setattr(cfg, field, val)
        msg = _expect(st, L.lmop_create, cfg, -1)
        assert msg  # lmop_last_error(NULL) explains the failed create


@pytest.fixture(scope="module")
def tiny_w():
    return make_weights(TINY, seed=5)


def test_state_and_weight_validation(tiny_w):
    ctx = _host_ctx()
    _expect(L.LMOP_ERR_STATE, ctx.eval_rows, [1], [0, 1], L.LMOP_BOOL, [1, 2])
    _expect(L.LMOP_ERR_STATE, ctx.set_prefix, [1, 2])
    bad = make_weights(TINY, seed=5, n_layers=1)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.load_weights, bad)
    import dataclasses
    l0 = tiny_w.layers[0]
    tiny_w.layers[0] = dataclasses.replace(l0, w_down=l0.w_gate)
    try:
        _expect(L.LMOP_ERR_INVALID_ARG, ctx.load_weights, tiny_w)
    finally:
        tiny_w.layers[0] = l0
    ctx.load_weights(tiny_w)


def test_eval_argument_validation(tiny_w):
    ctx = _host_ctx()
    ctx.load_weights(tiny_w)
    V = TINY.vocab
    ok = dict(kind=L.LMOP_BOOL, allowed=[3, 4])
    # valid arguments on a host-only ctx stop at UNSUPPORTED after validation
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [1, 2, 3], [0, 2, 3], **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, V, 3], [0, 2, 3], **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, -1, 3], [0, 2, 3], **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, 2, 3], [0, 3, 2], **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, 2, 3], [1, 2, 3], **ok)
    # a row with neither prefix nor suffix tokens
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, 2], [0, 2, 2], **ok)
    # type checks
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], L.LMOP_BOOL, [3])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], L.LMOP_ENUM, [3, 3])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], L.LMOP_ENUM, [V + 5])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], 7, [1, 2])
    digits = list(range(10, 20))
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], L.LMOP_INT, digits[:9], eos=5,
            max_tokens=4)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], L.LMOP_INT, digits, eos=12,
            max_tokens=4)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1], [0, 1], L.LMOP_INT, digits, eos=5,
            max_tokens=9)
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [1], [0, 1], L.LMOP_INT, digits, eos=5,
            max_tokens=8)
    # options: the restricted head is a valid mode; unknown flags and a
    # negative batch budget are not
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [1, 2, 3], [0, 2, 3], head_restricted=True, **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, L.lmop_eval_rows, ctx.ctx, [1, 2, 3], [0, 2, 3], L.LMOP_BOOL,
            [3, 4], flags=4)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, 2, 3], [0, 2, 3], max_batch_tokens=-1, **ok)
    # too long for max_seq (4096 by default)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, np.ones(4097, np.int32), [0, 4097], **ok)
    # zero rows is a no-op
    out, _ = ctx.eval_rows([], [0], **ok)
    assert len(out) == 0


def test_prefix_lifetimes(tiny_w):
    ctx = _host_ctx()
    ctx.load_weights(tiny_w)
    root = ctx.set_prefix([1, 2, 3])
    assert L.lmop_prefix_length(root) == 3
    child = ctx.set_prefix([4, 5], parent=root)
    assert L.lmop_prefix_length(child) == 5
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.set_prefix, [6], parent=child)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_prefix, [])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_prefix, [TINY.vocab])
    ok = dict(kind=L.LMOP_BOOL, allowed=[3, 4])
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [7], [0, 1], prefix=child, **ok)
    # an empty suffix is fine with a prefix
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [], [0, 0], prefix=root, **ok)
    ctx.release_prefix(root)  # parent released first: lives on while the child exists
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [7], [0, 1], prefix=root, **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.release_prefix, root)
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [7], [0, 1], prefix=child, **ok)
    ctx.release_prefix(child)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [7], [0, 1], prefix=child, **ok)
    # prefixes of another ctx are rejected
    other = _host_ctx()
    other.load_weights(tiny_w)
    p2 = other.set_prefix([1])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [7], [0, 1], prefix=p2, **ok)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [7], [0, 1], row_prefix=[p2], **ok)
    # reloading weights invalidates prefixes
    p3 = ctx.set_prefix([9])
    ctx.load_weights(tiny_w)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [7], [0, 1], prefix=p3, **ok)


def test_set_prefixes_validation(tiny_w):
    ctx = _host_ctx()
    _expect(L.LMOP_ERR_STATE, ctx.set_prefixes, [[1, 2]])
    ctx.load_weights(tiny_w)
    assert ctx.set_prefixes([]) == []
    root = ctx.set_prefix([1, 2, 3])
    kids = ctx.set_prefixes([[4, 5], [6], [7, 8, 9]], parent=root)
    assert [L.lmop_prefix_length(k) for k in kids] == [5, 4, 6]
    assert len({k.value for k in kids}) == 3
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.set_prefixes, [[6]], parent=kids[0])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_prefixes, [[1], []], parent=root)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_prefixes, [[1], [TINY.vocab]], parent=root)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_prefixes, [[1] * 4096], parent=root)
    # the root outlives its release while batched children exist; children free one by one
    ctx.release_prefix(root)
    ctx.release_prefix(kids[1])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.release_prefix, kids[1])
    ctx.release_prefix(kids[0])
    ctx.release_prefix(kids[2])


def _py_dedup(rows, keys):
    first = {}
    rep = []
    for i, (r, k) in enumerate(zip(rows, keys)):
        rep.append(first.setdefault((k, tuple(r)), i))
    return rep, len(first)


def test_dedup_matches_brute_force():
    rng = np.random.default_rng(0)
    for trial in range(20):
        pool = [rng.integers(0, 5, size=rng.integers(0, 4)) for _ in range(12)]
        rows = [pool[rng.integers(0, len(pool))] for _ in range(200)]
        keys = rng.integers(0, 3, size=200) if trial % 2 else np.zeros(200, np.int64)
        offs = np.concatenate([[0], np.cumsum([len(r) for r in rows])])
        toks = np.concatenate(rows).astype(np.int32) if offs[-1] else np.zeros(0, np.int32)
        rep, nu = L.lmop_dedup_rows(toks, offs, keys if trial % 2 else None)
        want, wn = _py_dedup([r.tolist() for r in rows], keys.tolist())
        assert nu == wn and rep.tolist() == want


def test_dedup_rejects_bad_csr():
    with pytest.raises(L.LmopError):
        L.lmop_dedup_rows([1, 2], [0, 2, 1])
    with pytest.raises(L.LmopError):
        L.lmop_dedup_rows([1, 2], [1, 2])
    rep, nu = L.lmop_dedup_rows([], [0])
    assert nu == 0 and len(rep) == 0


def test_fp8_weights_load_on_host_ctx():
    w8 = make_weights(TINY, seed=5, fmt="fp8_e4m3")
    ctx = _host_ctx()
    ctx.load_weights(w8)  # validation passes; a host-only ctx keeps nothing
    w8.layers[0].wq.fmt = "int4_g32"
    with pytest.raises(ValueError):
        ctx.load_weights(w8)


def test_limit_validation(tiny_w):
    ctx = _host_ctx()
    ctx.load_weights(tiny_w)
    ok = dict(kind=L.LMOP_BOOL, allowed=[3, 4])
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, 2, 3], [0, 2, 3], limit=-1, **ok)
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, [1, 2, 3], [0, 2, 3], limit=1, **ok)


def test_automaton_validation(tiny_w):
    from synth import Automaton
    ctx = _host_ctx()
    ctx.load_weights(tiny_w)
    V = TINY.vocab

    def aut(off, tok, nxt, acc):
        return Automaton(len(acc), np.array(off, np.int32), np.array(tok, np.int32),
                         np.array(nxt, np.int32), np.array(acc, np.uint8))

    good = aut([0, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1])
    run = lambda a, eos=-1, mt=3: ctx.eval_rows([1, 2], [0, 2], L.LMOP_AUTOMATON, a, eos=eos,
                                                max_tokens=mt)
    # valid: stops at UNSUPPORTED (host-only ctx) after validation
    _expect(L.LMOP_ERR_UNSUPPORTED, run, good)
    _expect(L.LMOP_ERR_UNSUPPORTED, run, good, eos=9)
    bad = [
        (aut([0, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1]), dict(mt=0)),
        (aut([0, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1]), dict(mt=9)),
        (aut([1, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1]), {}),      # offset[0] != 0
        (aut([0, 3, 2, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1]), {}),      # decreasing
        (aut([0, 2, 3, 3], [5, V, 7], [1, 2, 2], [0, 1, 1]), {}),      # token outside V
        (aut([0, 2, 3, 3], [5, 5, 7], [1, 2, 2], [0, 1, 1]), {}),      # repeated in a state
        (aut([0, 2, 3, 3], [5, 6, 7], [1, 3, 2], [0, 1, 1]), {}),      # next out of range
        (aut([0, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 0]), {}),      # dead non-accepting
        (aut([0, 0, 1, 1], [7], [2], [1, 1, 1]), {}),                  # start without edges
        (aut([0, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1]), dict(eos=6)),   # EOS is an edge
        (aut([0, 2, 3, 3], [5, 6, 7], [1, 2, 2], [0, 1, 1]), dict(eos=V)),
    ]
    for a, kw in bad:
        _expect(L.LMOP_ERR_INVALID_ARG, run, a, **kw)
    # more than 4096 distinct tokens
    n = 4097
    big = aut([0, n] + [n] * n, list(range(n)), list(range(1, n + 1)), [0] + [1] * n)
    _expect(L.LMOP_ERR_INVALID_ARG, run, big)


def test_profiling_period_validation():
    ctx = _host_ctx()
    _expect(-1, ctx.set_profiling, -1)
    for period in (0, 1, 5, True, False):
        ctx.set_profiling(period)
    assert ctx.kernel_stats() == {}
    ctx.close()


def test_binding_constants_match_header():
    """The flag values the binding passes are the header's."""
    hdr = open(os.path.join(ROOT, "include", "lmop.h")).read()
    defs = dict(re.findall(r"#define\s+(LMOP_\w+)\s+(\d+)u", hdr))
    assert defs == {"LMOP_NO_DEDUP": "1", "LMOP_HEAD_RESTRICTED": "2", "LMOP_W_INT4_G32": "0",
                    "LMOP_W_FP8_E4M3": "1"}
    assert (L.LMOP_W_INT4_G32, L.LMOP_W_FP8_E4M3) == (0, 1)
    assert L.LMOP_NO_DEDUP == 1 and L.LMOP_HEAD_RESTRICTED == 2
    kinds = dict(re.findall(r"(LMOP_(?:BOOL|ENUM|INT|AUTOMATON))\s*=\s*(\d+)", hdr))
    assert kinds == {"LMOP_BOOL": "0", "LMOP_ENUM": "1", "LMOP_INT": "2", "LMOP_AUTOMATON": "3"}
    assert (L.LMOP_BOOL, L.LMOP_ENUM, L.LMOP_INT, L.LMOP_AUTOMATON) == (0, 1, 2, 3)


def test_binding_shares_torchs_hip_runtime():
    """Imported on its own, the binding still loads torch's HIP runtime before
    the library, so the process maps exactly one libamdhip64: torch's."""
    import json
    import subprocess
    import sys

    import torch

    code = ("import json, paper_2606_31808_amd.lmop\n"
            "maps = open('/proc/self/maps').read().splitlines()\n"
            "print(json.dumps(sorted({l.split()[-1] for l in maps if 'libamdhip64' in l})))")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True,
                         check=True, timeout=300).stdout
    paths = json.loads(out.strip().splitlines()[-1])
    torch_lib = os.path.realpath(os.path.join(os.path.dirname(torch.__file__), "lib"))
    assert len(paths) == 1, paths
    assert os.path.realpath(paths[0]).startswith(torch_lib), paths


def test_workspace_validation_and_plan(tiny_w):
    """lmop_set_workspace checks its arguments; on a host-only ctx the call
    still plans its batches against the workspace, so a workspace too small
    for one row is LMOP_ERR_OOM, and one that holds a row but not the
    default token budget is a valid (smaller-batch) plan."""
    from synth import make_workload
    ctx = _host_ctx()
    ctx.load_weights(tiny_w)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_workspace, 0x1000, 0)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_workspace, 0, 4096)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.set_workspace, 0x1010, 4096)
    wl = make_workload("filter_tiny")
    args = (wl.tokens, wl.offsets, wl.kind, wl.allowed)
    # no device is touched: the pointer is only a number to a host-only ctx
    ctx.set_workspace(1 << 20, 64 << 10)
    msg = _expect(L.LMOP_ERR_OOM, ctx.eval_rows, *args)
    assert "workspace" in msg and "bytes" in msg
    ctx.set_workspace(1 << 20, 2 << 20)
    msg = _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, *args)
    n_small = int(msg.split(" batches")[0].split("(")[-1])
    ctx.set_workspace(1 << 20, 1 << 30)
    msg = _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, *args)
    n_big = int(msg.split(" batches")[0].split("(")[-1])
    assert n_big == 1 and n_small > 1  # the whole table fits one default batch
    # integer outputs: decode groups are sized from the workspace too
    digits = np.arange(10, 20, dtype=np.int32)
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, wl.tokens, wl.offsets, L.LMOP_INT, digits,
            eos=5, max_tokens=4)
    ctx.set_workspace(0, 0)
    mem = ctx.memory()
    assert mem["workspace_bytes"] == 0 and mem["device_bytes"] == 0
    # the no-allocation entry point validates exactly like lmop_eval_rows
    _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, *args, no_alloc=True)
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.eval_rows, [1, TINY.vocab], [0, 2], L.LMOP_BOOL, [1, 2],
            no_alloc=True)
    # a row too long for the static array: 256 MiB / ~6 KB per tiny-model token
    big = L.Context(TINY, device=-1, max_seq=1 << 17)
    big.load_weights(tiny_w)
    msg = _expect(L.LMOP_ERR_OOM, big.eval_rows, np.ones(100000, np.int32), [0, 100000],
                  L.LMOP_BOOL, [1, 2], no_alloc=True)
    assert "no-allocation" in msg


def test_plan_rows_host(tiny_w):
    """lmop_plan_rows on a host-only ctx: the batch plan of the call without
    running it.  Checked against what the plan must satisfy: rows counted
    after deduplication and the row mask; every pass within the token budget
    unless one row alone exceeds it; passes at least total / budget; one
    decode group per pass for single-step types; min_workspace_bytes is the
    exact threshold of lmop_eval_rows in a workspace (one byte less is
    LMOP_ERR_OOM, that size plans)."""
    from synth import make_workload
    ctx = _host_ctx()
    ctx.load_weights(tiny_w)
    wl = make_workload("filter_tiny")
    lens = np.diff(wl.offsets)
    args = (wl.tokens, wl.offsets, wl.kind, wl.allowed)
    pl = ctx.plan_rows(*args)
    assert pl["unique_rows"] == wl.n_rows and pl["batches"] == 1
    assert pl["max_batch_tokens"] == lens.sum() <= pl["batch_tokens"]
    assert pl["decode_groups"] == 1
    assert 0 < pl["own_kv_bytes"] < pl["scratch_bytes"]
    assert 0 < pl["min_workspace_bytes"] <= pl["scratch_bytes"] + 256
    for budget in (50, 200, 777):
        p = ctx.plan_rows(*args, max_batch_tokens=budget)
        assert p["batch_tokens"] == budget
        assert p["max_batch_tokens"] <= max(budget, lens.max())
        assert p["batches"] >= -(-lens.sum() // budget)
        assert p["decode_groups"] == p["batches"]
        assert p["min_workspace_bytes"] == pl["min_workspace_bytes"]
    # duplicates and the row mask shrink the evaluated rows
    toks = np.concatenate([wl.tokens, wl.tokens])
    offs = np.concatenate([wl.offsets, wl.offsets[1:] + wl.offsets[-1]])
    assert ctx.plan_rows(toks, offs, wl.kind, wl.allowed)["unique_rows"] == wl.n_rows
    assert ctx.plan_rows(toks, offs, wl.kind, wl.allowed, no_dedup=True)["unique_rows"] == 2 * wl.n_rows
    mask = np.arange(wl.n_rows) % 3 == 0
    assert ctx.plan_rows(*args, row_mask=mask)["unique_rows"] == mask.sum()
    # integer outputs keep KV for the decode steps: a larger own-KV store
    digits = np.arange(10, 20, dtype=np.int32)
    pi = ctx.plan_rows(wl.tokens, wl.offsets, L.LMOP_INT, digits, eos=5, max_tokens=4)
    assert pi["own_kv_bytes"] > pl["own_kv_bytes"] and pi["decode_groups"] >= 1
    # the workspace threshold, for both types
    for a, k in ((args, {}), ((wl.tokens, wl.offsets, L.LMOP_INT, digits), dict(eos=5, max_tokens=4))):
        need = ctx.plan_rows(*a, **k)["min_workspace_bytes"]
        ctx.set_workspace(1 << 20, need - 1)
        _expect(L.LMOP_ERR_OOM, ctx.eval_rows, *a, **k)
        _expect(L.LMOP_ERR_OOM, ctx.plan_rows, *a, **k)
        ctx.set_workspace(1 << 20, need)
        _expect(L.LMOP_ERR_UNSUPPORTED, ctx.eval_rows, *a, **k)
        small = ctx.plan_rows(*a, **k)
        assert small["scratch_bytes"] <= need and small["batches"] >= ctx.plan_rows(*a, **k)["batches"]
        ctx.set_workspace(0, 0)
    # argument errors are the call's own
    _expect(L.LMOP_ERR_INVALID_ARG, ctx.plan_rows, [1, TINY.vocab], [0, 2], L.LMOP_BOOL, [1, 2])
    assert ctx.plan_rows([], [0], L.LMOP_BOOL, [1, 2])["batches"] == 0
    # the logit dump's scratch is planned when asked for
    dump = ctx.plan_rows(*args, debug_logits=True)
    assert dump["scratch_bytes"] >= pl["scratch_bytes"] + wl.n_rows * TINY.vocab * 4
    assert dump["min_workspace_bytes"] > pl["min_workspace_bytes"]
