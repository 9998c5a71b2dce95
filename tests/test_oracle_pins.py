"""Pins the oracle to facts outside itself: hand-worked fixtures, closed forms,
invariants, special cases that reduce to a few matrix products, and brute
force on tiny inputs.  CPU only."""
import dataclasses
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import (KIND_BOOL, KIND_ENUM, KIND_INT, OracleLM, attention, constrained_pick,
                    decode_nibbles, dequant, rms_norm, rope, silu)
from oracle.lmop_oracle import KIND_AUTOMATON, automaton_steps, decode_e4m3, dequant_fp8
from synth import (SHAPES, Automaton, ModelShape, automaton_of_list, automaton_of_record,
                   make_weights, make_workload, option_trie, quantize_fp8_e4m3, quantize_int4_g32)

GOLD = os.path.join(os.path.dirname(__file__), "golden")

# every matrix of this model is non-square, so a transposed operand cannot
# pass silently; d_ff = 80 is not a multiple of 32 (partial last group)
MICRO = ModelShape("micro", 2, 48, 4, 2, 16, 80, 97, 1e4, shape_id=90)


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- int4 layout
def test_nibble_layout_matches_hand_table():
    g = _gold("int4_nibbles.json")
    b = np.array(g["bytes"], dtype=np.uint8)[None, :]
    codes = decode_nibbles(b).reshape(-1, 2)
    assert codes.tolist() == g["codes"]


def test_dequant_is_code_times_scale_for_all_codes():
    rng = np.random.default_rng(0)
    # 16 codes x 8 rows; each row one random fp16 scale per group
    codes = np.tile(np.arange(-8, 8), 4)[None, :].repeat(8, 0)  # [8][64]
    nib = (codes & 0xF).astype(np.uint8)
    packed = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    scales = rng.uniform(1e-4, 2.0, size=(8, 2)).astype(np.float16)
    for dt in (np.float32, np.float64):
        w = dequant(packed, scales, 64, dt)
        for n in range(8):
            for k in range(64):
                # python float product of an int and an fp16 value is exact
                assert float(w[n, k]) == float(codes[n, k]) * float(scales[n, k // 32])


def test_quant_roundtrip_error_bound_and_requant_identity():
    g = torch.Generator().manual_seed(3)
    w = torch.randn(64, 80, generator=g) * 0.02  # 80 = 2.5 groups
    qw, sc = quantize_int4_g32(w)
    assert qw.shape == (64, 48) and sc.shape == (64, 3)
    wd = dequant(qw.numpy(), sc.numpy(), 80, np.float64)
    s = np.repeat(sc.numpy().astype(np.float64), 32, axis=1)[:, :80]
    wn = w.double().numpy()
    inside = np.abs(wn / s) <= 7.0
    assert np.all(np.abs(wn - wd)[inside] <= s[inside] / 2 + 1e-12)
    # dequantised weights requantise to the same codes with the same scales
    q2 = np.clip(np.rint(wd / s), -8, 7)
    assert np.array_equal(q2, decode_nibbles(qw.numpy())[:, :80])
    # pad features of the partial group carry code 0
    assert np.all(decode_nibbles(qw.numpy())[:, 80:] == 0)


# ---------------------------------------------------------------- rmsnorm / silu
def test_e4m3_hand_values():
    # sign | exponent (bias 7) | mantissa, OCP E4M3 "fn"
    hand = {0x38: 1.0, 0x3C: 1.5, 0x40: 2.0, 0x7E: 448.0, 0x08: 2.0 ** -6, 0x01: 2.0 ** -9,
            0x07: 7 * 2.0 ** -9, 0x00: 0.0, 0xB8: -1.0, 0xFE: -448.0, 0x30: 0.5, 0x77: 240.0}
    got = decode_e4m3(np.array(list(hand)))
    assert got.tolist() == list(hand.values())
    assert np.isnan(decode_e4m3(np.array([0x7F, 0xFF]))).all()
    assert math.copysign(1.0, float(decode_e4m3(np.array([0x80]))[0])) == -1.0


def test_e4m3_decode_matches_torch_for_every_code():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = decode_e4m3(np.arange(256))
    assert np.array_equal(np.isnan(ours), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(ours[ok], ref[ok])


def test_fp8_quantiser_error_bound_and_requant_identity():
    g = torch.Generator().manual_seed(5)
    w = torch.randn(64, 200, generator=g) * 0.02
    w[3, 7] = 0.0
    w[5] = 0.0  # an all-zero row takes scale 1
    q, sc = quantize_fp8_e4m3(w)
    assert q.dtype == torch.uint8 and sc.shape == (64,) and sc[5] == 1.0
    deq = dequant_fp8(q.numpy(), sc.numpy())
    x = w.double().numpy() / sc.double().numpy()[:, None]
    err = np.abs(deq / sc.double().numpy()[:, None] - x)
    normal = np.abs(x) >= 2.0 ** -6
    # round to nearest: half a unit in the last place (3 mantissa bits)
    assert np.all(err[normal] <= np.abs(x[normal]) * 2.0 ** -4 + 1e-12)
    assert np.all(err[~normal] <= 2.0 ** -10 + 1e-12)
    # the largest magnitude of every nonzero row is exactly 448
    assert np.allclose(np.abs(deq / sc.double().numpy()[:, None]).max(axis=1)[np.arange(64) != 5],
                       448.0)
    q2, _ = quantize_fp8_e4m3(torch.from_numpy(deq).float())
    assert torch.equal(q2, q)


def test_fp8_model_prefix_cached_equals_full_forward():
    w = make_weights(MICRO, seed=13, fmt="fp8_e4m3")
    assert w.layers[0].wq.fmt == "fp8_e4m3" and w.layers[0].wq.scales.dtype == torch.float32
    orc = OracleLM(w, MICRO)
    rng = np.random.default_rng(17)
    prefix = rng.integers(0, MICRO.vocab, size=9)
    rows = _rand_rows(rng, 5, 1, 7, MICRO.vocab)
    res = orc.eval_rows(prefix, rows, KIND_ENUM, np.array([3, 50, 7]), keep_logits=True)
    for r in range(5):
        z = orc.logits(orc.forward_sequence(np.concatenate([prefix, rows[r]]))[-1])[0]
        assert np.allclose(res["logits"][r][0], z, atol=1e-11)


def test_rmsnorm_hand_value_and_unit_rms():
    y = rms_norm(np.array([3.0, 4.0]), np.ones(2), 0.0)
    assert np.allclose(y, [3 / math.sqrt(12.5), 4 / math.sqrt(12.5)], rtol=0, atol=1e-15)
    x = np.random.default_rng(1).normal(size=(5, 33))
    y = rms_norm(x, np.ones(33), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, atol=1e-14)
    assert np.allclose(rms_norm(7.5 * x, np.ones(33), 0.0), y, atol=1e-14)  # scale invariant
    gam = np.arange(33.0)
    assert np.allclose(rms_norm(x, gam, 0.0), y * gam, atol=1e-13)


def test_silu_closed_form():
    assert silu(np.array(0.0)) == 0.0
    assert math.isclose(float(silu(np.array(1.0))), 1 / (1 + math.exp(-1)), rel_tol=1e-15)
    assert math.isclose(float(silu(np.array(-1.0))), -1 / (1 + math.e), rel_tol=1e-14)
    x = np.linspace(-6, 6, 25)
    assert np.allclose(silu(x) - silu(-x), x, atol=1e-14)  # a*sig(a) + a*sig(-a) = a
    assert math.isclose(float(silu(np.array(40.0))), 40.0, rel_tol=1e-15)
    assert abs(float(silu(np.array(-800.0)))) < 1e-300


# ---------------------------------------------------------------- rope
def test_rope_hand_values():
    g = _gold("rope_rotate_half.json")
    for c in g["cases"]:
        x = np.array(c["x"], dtype=np.float64)[None, None, :]
        y = rope(x, np.array([c["pos"]]), g["theta"])[0, 0]
        assert np.allclose(y, c["y"], rtol=0, atol=1e-15), c


def test_rope_norm_and_relative_position():
    rng = np.random.default_rng(2)
    q = rng.normal(size=(6, 3, 32))
    k = rng.normal(size=(6, 3, 32))
    pos = np.array([0, 1, 5, 17, 100, 4095])
    rq = rope(q, pos, 5e5)
    assert np.allclose(np.linalg.norm(rq, axis=-1), np.linalg.norm(q, axis=-1), atol=1e-12)
    # q.k after rotation depends only on the position difference
    for shift in (1, 37, 1000):
        a = np.einsum("thd,shd->tsh", rope(q, pos, 5e5), rope(k, pos[::-1].copy(), 5e5))
        b = np.einsum("thd,shd->tsh", rope(q, pos + shift, 5e5), rope(k, pos[::-1] + shift, 5e5))
        assert np.allclose(a, b, atol=1e-9)


# ---------------------------------------------------------------- attention
def _naive_attention(q, k, v, n_visible):
    tq, hq, hd = q.shape
    _, hkv, _ = k.shape
    out = np.zeros_like(q)
    for i in range(tq):
        for j in range(hq):
            g = (j * hkv) // hq
            sc = [sum(q[i, j, d] * k[t, g, d] for d in range(hd)) / math.sqrt(hd)
                  for t in range(n_visible[i])]
            m = max(sc)
            e = [math.exp(s - m) for s in sc]
            tot = sum(e)
            for d in range(hd):
                out[i, j, d] = sum(e[t] * v[t, g, d] for t in range(n_visible[i])) / tot
    return out


def test_attention_matches_naive_loops():
    rng = np.random.default_rng(4)
    q = rng.normal(size=(5, 4, 8))
    k = rng.normal(size=(9, 2, 8))
    v = rng.normal(size=(9, 2, 8))
    nv = np.array([5, 6, 7, 8, 9])
    assert np.allclose(attention(q, k, v, nv), _naive_attention(q, k, v, nv), atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(5)
    k = rng.normal(size=(6, 2, 8))
    v = rng.normal(size=(6, 2, 8))
    q = rng.normal(size=(6, 4, 8))
    # one visible key => output is that key's value
    o = attention(q, k, v, np.ones(6, dtype=int))
    for j in range(4):
        assert np.allclose(o[:, j], v[0, j // 2][None, :], atol=1e-15)
    # zero queries => equal scores => running mean of the visible values
    o = attention(np.zeros_like(q), k, v, np.arange(1, 7))
    for i in range(6):
        for j in range(4):
            assert np.allclose(o[i, j], v[: i + 1, j // 2].mean(0), atol=1e-14)
    # GQA with hkv == hq is plain multi-head attention per head
    o1 = attention(q[:, :2], k, v, np.arange(1, 7))
    for j in range(2):
        oj = attention(q[:, j:j + 1], k[:, j:j + 1], v[:, j:j + 1], np.arange(1, 7))
        assert np.allclose(o1[:, j], oj[:, 0], atol=1e-14)


# ---------------------------------------------------------------- constrained step
def test_constrained_pick_hand_values():
    g = _gold("constrained_pick.json")
    z = np.array(g["z"])
    for c in g["cases"]:
        i, lp, lpf, m = constrained_pick(z, c["allowed"])
        assert i == c["index"]
        assert math.isclose(lp, c["logprob"], abs_tol=1e-14)
        assert math.isclose(lpf, c["logprob_full"], abs_tol=1e-14)
        want_m = math.inf if c["margin"] == "inf" else c["margin"]
        assert m == want_m or math.isclose(m, want_m, abs_tol=1e-14)


def test_constrained_pick_invariants():
    rng = np.random.default_rng(6)
    for _ in range(50):
        z = rng.normal(size=300) * 3
        a = rng.choice(300, size=rng.integers(1, 30), replace=False)
        i, lp, lpf, m = constrained_pick(z, a)
        assert z[a[i]] == z[a].max()
        assert lp <= 0 and lpf <= lp + 1e-15
        za = z[a]
        assert math.isclose(np.exp(za - (za[i] - lp)).sum(), 1.0, rel_tol=1e-12)
        if len(a) == 1:
            assert lp == 0.0


# ---------------------------------------------------------------- whole model
@pytest.fixture(scope="module")
def micro():
    w = make_weights(MICRO, seed=11)
    return w, OracleLM(w, MICRO)


def _rand_rows(rng, n, lo, hi, V):
    return [rng.integers(0, V, size=int(rng.integers(lo, hi + 1))) for _ in range(n)]


def test_prefix_cached_equals_full_forward(micro):
    w, orc = micro
    rng = np.random.default_rng(7)
    prefix = rng.integers(0, MICRO.vocab, size=11)
    rows = _rand_rows(rng, 6, 1, 9, MICRO.vocab) + [np.zeros(0, dtype=np.int64)]
    allowed = np.array([3, 50, 7])
    res = orc.eval_rows(prefix, rows, KIND_ENUM, allowed, keep_logits=True)
    for r, s in enumerate(rows):
        seq = np.concatenate([prefix, s])
        x = orc.forward_sequence(seq)
        z = orc.logits(x[-1])[0]
        assert np.allclose(res["logits"][r][0], z, rtol=0, atol=1e-11)
        i, lp, lpf, _ = constrained_pick(z, allowed)
        assert res["value"][r] == i and math.isclose(res["logprob"][r], lp, abs_tol=1e-12)
        assert math.isclose(res["logprob_full"][r], lpf, abs_tol=1e-12)


def test_two_level_prefix_equals_full_forward(micro):
    w, orc = micro
    rng = np.random.default_rng(8)
    prefix = rng.integers(0, MICRO.vocab, size=7)
    kids = _rand_rows(rng, 3, 2, 5, MICRO.vocab)
    rows = _rand_rows(rng, 6, 1, 4, MICRO.vocab)
    rc = [0, 2, 1, 1, 0, 2]
    res = orc.eval_rows(prefix, rows, KIND_BOOL, [4, 9], children=kids, row_child=rc,
                        keep_logits=True)
    for r in range(6):
        seq = np.concatenate([prefix, kids[rc[r]], rows[r]])
        z = orc.logits(orc.forward_sequence(seq)[-1])[0]
        assert np.allclose(res["logits"][r][0], z, atol=1e-11)


def test_zero_layers_is_one_matvec():
    w = make_weights(MICRO, seed=12, n_layers=0)
    orc = OracleLM(w, MICRO)
    e = w.tok_embedding.double().numpy()
    head = w.lm_head.double().numpy()
    t = np.array([5, 17, 42])
    x = e[42]
    want = (x / np.sqrt(np.mean(x * x) + MICRO.rms_eps)) @ head.T
    got = orc.logits(orc.forward_sequence(t)[-1])[0]
    assert np.allclose(got, want, atol=1e-13)


def _zero(m):
    m.qweight.zero_()


def test_zero_output_projections_make_layers_identity():
    w = make_weights(MICRO, seed=13)
    for l in w.layers:
        _zero(l.wo)
        _zero(l.w_down)
    orc = OracleLM(w, MICRO)
    w0 = make_weights(MICRO, seed=13, n_layers=0)
    orc0 = OracleLM(w0, MICRO)
    t = np.array([1, 2, 3, 60, 96])
    assert np.allclose(orc.forward_sequence(t), orc0.forward_sequence(t), atol=1e-14)


def test_one_token_attention_block_is_two_linear_maps():
    # with one token, attention returns that token's value: the block is
    # x + (RMSNorm(x) Wv^T, repeated per query head group) Wo^T
    w = make_weights(MICRO, seed=14, n_layers=1)
    _zero(w.layers[0].w_down)
    orc = OracleLM(w, MICRO)
    L = w.layers[0]
    wv = dequant(L.wv.qweight.numpy(), L.wv.scales.numpy(), L.wv.k)
    wo = dequant(L.wo.qweight.numpy(), L.wo.scales.numpy(), L.wo.k)
    x = w.tok_embedding.double().numpy()[33]
    h = x / np.sqrt(np.mean(x * x) + MICRO.rms_eps)
    v = (h @ wv.T).reshape(MICRO.n_kv_heads, MICRO.head_dim)
    rep = MICRO.n_heads // MICRO.n_kv_heads
    o = np.repeat(v, rep, axis=0).reshape(-1)  # query head j reads kv head j // rep
    want = x + o @ wo.T
    assert np.allclose(orc.forward_sequence([33])[-1], want, atol=1e-13)


def _attention_layer_by_scalar_loops(w, tokens):
    """One decoder layer whose down projection is zero, written out with
    scalar loops and the math module from the layer's definition: RMSNorm,
    the q/k/v maps, rotate-half RoPE on q and k at positions 0, 1, 2, ...
    (pair (m, m + hd/2) turned by pos * theta^(-2m/hd)), query head j reading
    kv head floor(j * n_kv / n_q), a softmax over the keys at or before the
    query, and the output map added to the residual."""
    sh = MICRO
    hd, half, nq, nkv = sh.head_dim, sh.head_dim // 2, sh.n_heads, sh.n_kv_heads
    L = w.layers[0]
    dq = lambda m: dequant(m.qweight.numpy(), m.scales.numpy(), m.k).tolist()
    wq, wk, wv, wo = dq(L.wq), dq(L.wk), dq(L.wv), dq(L.wo)
    emb = w.tok_embedding.double().numpy()
    d = sh.d_model
    xs, qs, ks, vs = [], [], [], []
    for pos, t in enumerate(tokens):
        x = [float(v) for v in emb[t]]
        r = 1.0 / math.sqrt(sum(v * v for v in x) / d + sh.rms_eps)
        h = [v * r for v in x]
        lin = lambda W: [sum(W[n][c] * h[c] for c in range(d)) for n in range(len(W))]
        q, k, v = lin(wq), lin(wk), lin(wv)

        def rot(vec, heads):
            out = list(vec)
            for j in range(heads):
                for m in range(half):
                    a = pos * sh.rope_theta ** (-2.0 * m / hd)
                    x1, x2 = vec[j * hd + m], vec[j * hd + m + half]
                    out[j * hd + m] = x1 * math.cos(a) - x2 * math.sin(a)
                    out[j * hd + m + half] = x1 * math.sin(a) + x2 * math.cos(a)
            return out
        xs.append(x)
        qs.append(rot(q, nq))
        ks.append(rot(k, nkv))
        vs.append(v)
    out = []
    for i in range(len(tokens)):
        o = [0.0] * (nq * hd)
        for j in range(nq):
            g = j * nkv // nq
            sc = [sum(qs[i][j * hd + m] * ks[s][g * hd + m] for m in range(hd)) / math.sqrt(hd)
                  for s in range(i + 1)]
            top = max(sc)
            e = [math.exp(v - top) for v in sc]
            tot = sum(e)
            for m in range(hd):
                o[j * hd + m] = sum(e[s] / tot * vs[s][g * hd + m] for s in range(i + 1))
        out.append([xs[i][n] + sum(wo[n][c] * o[c] for c in range(nq * hd)) for n in range(d)])
    return np.array(out)


def test_multi_token_attention_block_scalar_loops():
    # three tokens: RoPE turns q and k (not v) at positions 1 and 2, the
    # softmax weighs several keys, and the two kv heads serve four query heads
    w = make_weights(MICRO, seed=16, n_layers=1)
    _zero(w.layers[0].w_down)
    orc = OracleLM(w, MICRO)
    toks = [33, 7, 81]
    want = _attention_layer_by_scalar_loops(w, toks)
    assert np.allclose(orc.forward_sequence(toks), want, rtol=0, atol=1e-12)
    # the same through row evaluation: a 1-token prefix and a 2-token suffix
    res = orc.eval_rows(np.array(toks[:1]), [np.array(toks[1:])], KIND_ENUM, [1, 2, 3],
                        keep_logits=True)
    x = want[-1]
    hn = x / math.sqrt(float(np.mean(x * x)) + MICRO.rms_eps)
    z = hn @ w.lm_head.double().numpy().T
    assert np.allclose(res["logits"][0][0], z, rtol=0, atol=1e-12)


def test_mlp_block_closed_form():
    # attention output projection zeroed: the layer is x + swiglu(RMSNorm(x)) Wd^T
    w = make_weights(MICRO, seed=15, n_layers=1)
    _zero(w.layers[0].wo)
    orc = OracleLM(w, MICRO)
    L = w.layers[0]
    dq = lambda m: dequant(m.qweight.numpy(), m.scales.numpy(), m.k)
    wg, wu, wd = dq(L.w_gate), dq(L.w_up), dq(L.w_down)
    x = w.tok_embedding.double().numpy()[[4, 8, 15]]
    h = x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + MICRO.rms_eps)
    g = h @ wg.T
    want = x + ((g / (1 + np.exp(-g))) * (h @ wu.T)) @ wd.T
    assert np.allclose(orc.forward_sequence([4, 8, 15]), want, atol=1e-13)


def test_causality(micro):
    _, orc = micro
    a = orc.forward_sequence([1, 2, 3, 4, 5, 6])
    b = orc.forward_sequence([1, 2, 3, 90, 91])
    assert np.allclose(a[:3], b[:3], atol=1e-14)
    assert not np.allclose(a[3], b[3])


def test_int_decode_matches_full_recompute():
    w = make_weights(MICRO, seed=11)
    eos = 3
    w.lm_head[eos] *= 4  # widen the EOS logit so that some rows stop early
    orc = OracleLM(w, MICRO)
    rng = np.random.default_rng(9)
    prefix = rng.integers(0, MICRO.vocab, size=6)
    digits = np.array([10, 11, 12, 13, 14, 15, 16, 17, 18, 19])
    rows = _rand_rows(rng, 12, 1, 5, MICRO.vocab)
    res = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4, keep_logits=True)
    n_eos = n_full = 0
    for r in range(12):
        n = res["n_tokens"][r]
        toks = res["tokens"][r][:n].tolist()
        assert 1 <= n <= 4 and toks[0] in digits.tolist()
        assert all(t in digits.tolist() for t in toks[:-1])
        if toks[-1] == eos:
            n_eos += 1
        else:
            assert n == 4
            n_full += 1
        val = int("".join(str(digits.tolist().index(t)) for t in toks if t != eos))
        assert res["value"][r] == val
        # each step's logits equal a full forward over the extended sequence
        lp = lpf = 0.0
        for s in range(n):
            seq = np.concatenate([prefix, rows[r], toks[:s]])
            z = orc.logits(orc.forward_sequence(seq)[-1])[0]
            assert np.allclose(res["logits"][r][s], z, atol=1e-11)
            allowed = digits if s == 0 else np.concatenate([digits, [eos]])
            i, a, b, _ = constrained_pick(z, allowed)
            assert allowed[i] == toks[s]
            lp += a
            lpf += b
        assert math.isclose(res["logprob"][r], lp, abs_tol=1e-12)
        assert math.isclose(res["logprob_full"][r], lpf, abs_tol=1e-12)
    assert n_eos >= 1 and n_full >= 1


def _star(tokens):
    """ENUM as a token automaton: state 0 -> one leaf per option."""
    n = len(tokens)
    off = np.array([0] + [n] * (n + 1), dtype=np.int32)
    return Automaton(n + 1, off, np.asarray(tokens, dtype=np.int32),
                     np.arange(1, n + 1, dtype=np.int32),
                     np.array([0] + [1] * n, dtype=np.uint8))


def _int_automaton(digits, max_digits=4):
    """INT as a token automaton: state k = k digits so far."""
    n = max_digits + 1
    off = np.array([10 * min(s, max_digits) for s in range(n + 1)], dtype=np.int32)
    tok = np.tile(np.asarray(digits, dtype=np.int32), max_digits)
    nxt = np.repeat(np.arange(1, max_digits + 1, dtype=np.int32), 10)
    acc = np.array([0] + [1] * max_digits, dtype=np.uint8)
    return Automaton(n, off, tok, nxt, acc)


def test_automaton_steps_hand_example():
    # state 0: 7 -> 1, 5 -> 2; state 1 (accepting): 5 -> 2, 9 -> 3; 2, 3 accepting leaves
    aut = Automaton(4, np.array([0, 2, 4, 4, 4], np.int32), np.array([7, 5, 9, 5], np.int32),
                    np.array([1, 2, 3, 2], np.int32), np.array([0, 1, 1, 1], np.uint8))
    g = automaton_steps(aut, eos=42)
    assert g[0][0].tolist() == [7, 5] and g[0][1] == [1, 2]
    # token order is first appearance in the edge list (7, 5, 9), then EOS
    assert g[1][0].tolist() == [5, 9, 42] and g[1][1] == [2, 3, None]
    assert g[2][0].tolist() == [42] and g[3][1] == [None]
    assert [a.tolist() for a, _ in automaton_steps(aut, eos=-1)][1] == [5, 9]


def test_option_trie_hand_example():
    aut, final = option_trie([np.array([4, 8]), np.array([4, 9, 1]), np.array([6])])
    # states: 0, [4]=1, [4,8]=2, [4,9]=3, [4,9,1]=4, [6]=5
    assert aut.n_states == 6
    assert aut.edge_offset.tolist() == [0, 2, 4, 4, 5, 5, 5]
    assert aut.edge_token.tolist() == [4, 6, 8, 9, 1]
    assert aut.edge_next.tolist() == [1, 5, 2, 3, 4]
    assert aut.accepting.tolist() == [0, 0, 1, 0, 1, 1]
    assert final.tolist() == [2, 4, 5]


def test_automaton_star_equals_enum(micro):
    _, orc = micro
    rng = np.random.default_rng(21)
    prefix = rng.integers(0, MICRO.vocab, size=7)
    rows = _rand_rows(rng, 9, 1, 6, MICRO.vocab)
    opts = np.array([30, 5, 61, 12])
    e = orc.eval_rows(prefix, rows, KIND_ENUM, opts)
    a = orc.eval_rows(prefix, rows, KIND_AUTOMATON, _star(opts), max_tokens=3)
    assert np.array_equal(a["value"], e["value"] + 1)
    for k in ("logprob", "logprob_full", "n_tokens", "tokens", "margin"):
        assert np.array_equal(a[k], e[k]), k


def test_automaton_int_grammar_equals_int():
    w = make_weights(MICRO, seed=11)
    eos = 3
    w.lm_head[eos] *= 4
    orc = OracleLM(w, MICRO)
    rng = np.random.default_rng(9)
    prefix = rng.integers(0, MICRO.vocab, size=6)
    digits = np.array([10, 11, 12, 13, 14, 15, 16, 17, 18, 19])
    rows = _rand_rows(rng, 12, 1, 5, MICRO.vocab)
    i = orc.eval_rows(prefix, rows, KIND_INT, digits, eos=eos, max_tokens=4)
    a = orc.eval_rows(prefix, rows, KIND_AUTOMATON, _int_automaton(digits), eos=eos, max_tokens=4)
    for k in ("logprob", "logprob_full", "n_tokens", "tokens", "margin"):
        assert np.array_equal(a[k], i[k]), k
    n_digits = np.array([n - (t[n - 1] == eos) for n, t in zip(i["n_tokens"], i["tokens"])])
    assert np.array_equal(a["value"], n_digits)


def test_automaton_trie_decode_matches_full_recompute(micro):
    _, orc = micro
    rng = np.random.default_rng(23)
    prefix = rng.integers(0, MICRO.vocab, size=5)
    options = [np.array(o) for o in ([40, 2], [40, 7, 9], [40, 7, 1], [66], [21, 2, 2])]
    aut, final = option_trie(options)
    g = automaton_steps(aut, eos=-1)
    rows = _rand_rows(rng, 16, 1, 6, MICRO.vocab)
    res = orc.eval_rows(prefix, rows, KIND_AUTOMATON, aut, max_tokens=3, keep_logits=True)
    seen = set()
    for r in range(16):
        n = res["n_tokens"][r]
        toks = res["tokens"][r][:n].tolist()
        # the output is exactly the option whose final state is the value
        o = final.tolist().index(res["value"][r])
        assert toks == options[o].tolist()
        seen.add(o)
        st, lp, lpf = 0, 0.0, 0.0
        for s in range(n):
            seq = np.concatenate([prefix, rows[r], toks[:s]])
            z = orc.logits(orc.forward_sequence(seq)[-1])[0]
            assert np.allclose(res["logits"][r][s], z, atol=1e-11)
            allowed, to = g[st]
            ci, a, b, _ = constrained_pick(z, allowed)
            assert allowed[ci] == toks[s]
            lp, lpf, st = lp + a, lpf + b, to[ci]
        assert math.isclose(res["logprob"][r], lp, abs_tol=1e-12)
        assert math.isclose(res["logprob_full"][r], lpf, abs_tol=1e-12)
    assert len(seen) >= 2


def test_automaton_endings(micro):
    _, orc = micro
    rng = np.random.default_rng(25)
    rows = _rand_rows(rng, 6, 1, 4, MICRO.vocab)
    # a chain 0 -> 1 -> 2 -> 3 with only state 3 accepting: cut after 2 tokens
    chain = Automaton(4, np.array([0, 1, 2, 3, 3], np.int32), np.array([5, 6, 7], np.int32),
                      np.array([1, 2, 3], np.int32), np.array([0, 0, 0, 1], np.uint8))
    res = orc.eval_rows(None, rows, KIND_AUTOMATON, chain, max_tokens=2)
    assert np.all(res["value"] == -1) and np.all(res["n_tokens"] == 2)
    assert np.all(res["tokens"][:, :2] == [5, 6]) and np.all(res["logprob"] == 0.0)
    res = orc.eval_rows(None, rows, KIND_AUTOMATON, chain, max_tokens=3)
    assert np.all(res["value"] == 3) and np.all(res["n_tokens"] == 3)
    # an accepting state with edges ends on EOS or runs on
    fork = Automaton(3, np.array([0, 1, 2, 2], np.int32), np.array([5, 6], np.int32),
                     np.array([1, 2], np.int32), np.array([0, 1, 1], np.uint8))
    w2 = make_weights(MICRO, seed=11)
    w2.lm_head[9] *= 6
    o2 = OracleLM(w2, MICRO)
    res = o2.eval_rows(None, rows, KIND_AUTOMATON, fork, eos=9, max_tokens=3)
    for r in range(6):
        toks = res["tokens"][r][:res["n_tokens"][r]].tolist()
        assert toks in ([5, 9], [5, 6])
        assert res["value"][r] == (1 if toks == [5, 9] else 2)
    lp = res["logprob"]
    assert np.all(lp <= 0.0)


def _language(aut, max_len):
    """Every token string an output can be: the paths from state 0 that stop
    in an accepting state (found by brute-force search)."""
    out = set()

    def walk(st, path):
        if aut.accepting[st]:
            out.add(tuple(path))
        if len(path) < max_len:
            for e in range(aut.edge_offset[st], aut.edge_offset[st + 1]):
                walk(int(aut.edge_next[e]), path + [int(aut.edge_token[e])])

    walk(0, [])
    return out


def _assert_deterministic(aut):
    for st in range(aut.n_states):
        t = aut.edge_token[aut.edge_offset[st]:aut.edge_offset[st + 1]].tolist()
        assert len(set(t)) == len(t), st


def test_list_automaton_language():
    # items with a shared first token, one a prefix of another
    items = [np.array(x) for x in ([4], [4, 9], [6], [7, 7])]
    sep = 2
    for lo, hi in ((1, 1), (1, 3), (2, 3), (3, 3)):
        aut = automaton_of_list(items, sep=sep, lo=lo, hi=hi)
        _assert_deterministic(aut)
        want = set()
        for n in range(lo, hi + 1):
            for combo in itertools.product(items, repeat=n):
                want.add(tuple(sum(([sep] * (j > 0) + it.tolist()
                                    for j, it in enumerate(combo)), [])))
        assert _language(aut, 3 * hi) == want, (lo, hi)
    with pytest.raises(ValueError):
        automaton_of_list(items, sep=9, lo=1, hi=2)   # the separator is an item token
    with pytest.raises(ValueError):
        automaton_of_list(items, sep=sep, lo=0, hi=2)
    with pytest.raises(ValueError):
        automaton_of_list(items, sep=sep, lo=3, hi=2)


def test_record_automaton_language():
    digits = list(range(10, 20))
    fields = [("enum", 50, [60, 61, 62]), ("int", 51, digits, 2)]
    aut = automaton_of_record(1, 3, 2, fields)
    _assert_deterministic(aut)
    want = {tuple([1, 50, v, 2, 51] + list(d) + [3])
            for v in (60, 61, 62) for n in (1, 2) for d in itertools.product(digits, repeat=n)}
    assert _language(aut, 12) == want
    # one accepting state, without edges: a complete record ends the output
    (end,) = np.flatnonzero(aut.accepting)
    assert aut.edge_offset[end] == aut.edge_offset[end + 1]
    with pytest.raises(ValueError):
        automaton_of_record(1, 12, 2, fields)         # the closing token is a digit
    with pytest.raises(ValueError):
        automaton_of_record(1, 3, 2, [("int", 51, digits[:9], 2)])


@pytest.mark.parametrize("grammar", ["list", "record"])
def test_grammar_decode_matches_full_recompute(micro, grammar):
    """Greedy constrained decoding over a list or record grammar: every output
    is a string of the grammar, and each step's logits, pick and
    log-probabilities equal a full recompute of the sequence so far."""
    _, orc = micro
    rng = np.random.default_rng(31)
    eos = 91  # with these rows, some lists end early on EOS
    if grammar == "list":
        items = [np.array(x) for x in ([40, 2], [40, 7], [66], [21, 5])]
        aut, max_tokens = automaton_of_list(items, sep=9, lo=1, hi=3), 8
    else:
        aut = automaton_of_record(30, 31, 32, [("enum", 33, [60, 61, 62]),
                                               ("int", 34, list(range(70, 80)), 2)])
        max_tokens = 8
    lang = _language(aut, max_tokens)
    g = automaton_steps(aut, eos=eos)
    prefix = rng.integers(0, MICRO.vocab, size=5)
    rows = _rand_rows(rng, 12, 1, 6, MICRO.vocab)
    res = orc.eval_rows(prefix, rows, KIND_AUTOMATON, aut, eos=eos, max_tokens=max_tokens,
                        keep_logits=True)
    ends, eos_ends = 0, 0
    for r in range(12):
        n = res["n_tokens"][r]
        toks = res["tokens"][r][:n].tolist()
        body = toks[:-1] if toks[-1] == eos else toks
        if res["value"][r] >= 0:
            assert tuple(body) in lang
            ends += 1
            eos_ends += toks[-1] == eos
        st, lp, lpf = 0, 0.0, 0.0
        for s in range(n):
            seq = np.concatenate([prefix, rows[r], toks[:s]])
            z = orc.logits(orc.forward_sequence(seq)[-1])[0]
            assert np.allclose(res["logits"][r][s], z, atol=1e-11)
            allowed, to = g[st]
            ci, a, b, _ = constrained_pick(z, allowed)
            assert allowed[ci] == toks[s]
            lp, lpf = lp + a, lpf + b
            st = to[ci] if to[ci] is not None else st
        assert math.isclose(res["logprob"][r], lp, abs_tol=1e-12)
        assert math.isclose(res["logprob_full"][r], lpf, abs_tol=1e-12)
    assert ends == 12
    if grammar == "list":
        assert 0 < eos_ends < 12  # both endings: EOS after fewer items, and {3} reached
    else:
        assert eos_ends == 0      # a complete record ends by itself


def test_batch_and_order_invariance(micro):
    _, orc = micro
    rng = np.random.default_rng(10)
    prefix = rng.integers(0, MICRO.vocab, size=5)
    rows = _rand_rows(rng, 8, 1, 6, MICRO.vocab)
    allowed = [1, 2, 3, 4, 5]
    full = orc.eval_rows(prefix, rows, KIND_ENUM, allowed, keep_logits=True)
    perm = rng.permutation(8)
    pr = orc.eval_rows(prefix, [rows[i] for i in perm], KIND_ENUM, allowed, keep_logits=True)
    for j, i in enumerate(perm):
        assert np.allclose(pr["logits"][j][0], full["logits"][i][0], atol=1e-12)
        assert pr["value"][j] == full["value"][i]
    one = orc.eval_rows(prefix, rows[3:4], KIND_ENUM, allowed, keep_logits=True)
    assert np.allclose(one["logits"][0][0], full["logits"][3][0], atol=1e-12)


def test_logit_std_matches_closed_form():
    # final hidden has unit RMS and W_lm ~ N(0, 0.02^2): std(z) ~ 0.02 sqrt(d)
    wl = make_workload("filter_tiny", n_rows=16)
    w = make_weights(SHAPES["tiny"], seed=1234)
    orc = OracleLM(w, SHAPES["tiny"])
    res = orc.eval_workload(wl, keep_logits=True)
    z = np.stack([res["logits"][r][0] for r in range(16)])
    assert abs(z.std() / (0.02 * math.sqrt(256)) - 1) < 0.1
    assert set(res["value"].tolist()) <= {0, 1}
    assert np.all(res["logprob"] <= 0)


def test_fp32_and_fp64_oracles_agree(micro):
    w, orc = micro
    o32 = OracleLM(w, MICRO, dtype=np.float32)
    t = [5, 6, 7, 8, 9, 10]
    a = orc.logits(orc.forward_sequence(t)[-1])
    b = o32.logits(o32.forward_sequence(t)[-1])
    assert np.max(np.abs(a - b)) < 1e-4 * np.std(a)


def test_workload_recipes():
    wl = make_workload("filter_8b")
    lens = np.diff(wl.offsets)
    assert wl.n_rows == 10000 and len(wl.prefix) == 512 and len(wl.allowed) == 24
    assert lens.min() >= 8 and lens.max() <= 512 and abs(lens.mean() - 60) < 2
    wl = make_workload("filter_1b")
    lens = np.diff(wl.offsets)
    assert wl.n_rows == 4096 and abs(lens.mean() - 40) < 2 and lens.max() <= 256
    wl = make_workload("map_int_8b")
    assert wl.n_rows == 20000 and wl.eos not in wl.allowed.tolist()
    uniq = {tuple(wl.suffix(r).tolist()) for r in range(wl.n_rows)}
    assert 2300 < len(uniq) < 3000
    wl = make_workload("join_8b")
    assert wl.n_rows == 40000 and len(wl.children) == 200 and wl.row_child[-1] == 199
    assert len(wl.prefix) == 320
