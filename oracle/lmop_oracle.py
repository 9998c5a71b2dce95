"""Oracle: a plain, slow CPU evaluation of LM-operator rows.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import, call or execute this module.
It shares no code with the library and imports nothing from it.

What it computes (the paper's row-wise LM function, Sec. 2.3.2 "llmmap"):
for every row r the sequence t = prefix ++ suffix_r (prefix = the shared
instruction part of the prompt template, Appendix "Prompts"; the row's
values are the suffix) is run through a decoder LM and the next token is
chosen under the operator's return-type constraint (Sec. 2.3 "Constrained
Decoding": bool, an `options` set, or an integer).  The paper does not
describe the model; its shape is a Llama-style decoder:

  x0 = E[t]                                   (token embedding)
  per layer:  h = RMSNorm(x) * g_attn
              q, k, v = h Wq^T, h Wk^T, h Wv^T ; RoPE (rotate-half) on q, k
              o_i = sum_{j<=i} softmax_j(q_i . k_j / sqrt(hd)) v_j   (GQA)
              x += o Wo^T
              h2 = RMSNorm(x) * g_mlp
              x += (silu(h2 Wg^T) * (h2 Wu^T)) Wd^T
  z = RMSNorm(x_last) * g_final  W_lm^T

Weights are W4A16 (Sec. 3.2, Table "tab:models"): each linear matrix is
int4 with one fp16 scale per 32 input features; the oracle multiplies the
stored code by the stored scale, which is exact in fp32 and fp64.

Precision: float64 by default; float32 on request (the large shapes, where
fp64 would double the CPU time).  The constrained step and the integer
decode follow the readings listed in the design notes: ties go to the first
allowed token; `logprob` is the log-softmax over the step's allowed set and
`logprob_full` over the whole vocabulary; an integer is a digit string with
no EOS at the first step and at most `max_tokens` tokens including EOS.
Multi-token outputs (option strings, other regular types) follow a token
automaton: each step allows the current state's edge tokens (and EOS in an
accepting state), as listed in automaton_steps.

Evaluation with a shared prefix computes the prefix's keys and values once
and lets each row attend to them.  Causal attention makes that identical to
the full per-row forward (`forward_sequence`), which the tests check by
brute force on small models.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Sequence

import numpy as np

KIND_BOOL, KIND_ENUM, KIND_INT, KIND_AUTOMATON = 0, 1, 2, 3
GROUP = 32

# two's-complement value of every nibble 0..15
_NIBBLE_VALUE = np.array([v if v < 8 else v - 16 for v in range(16)], dtype=np.int8)
# byte -> (value of low nibble, value of high nibble)
_BYTE_PAIR = np.stack([_NIBBLE_VALUE[np.arange(256) & 15], _NIBBLE_VALUE[np.arange(256) >> 4]],
                      axis=1)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def decode_nibbles(qweight: np.ndarray) -> np.ndarray:
    """int4 codes [N][2*B] from packed bytes [N][B]: feature 2j is the low
    nibble of byte j, feature 2j+1 the high nibble; two's complement."""
    n, nb = qweight.shape
    return _BYTE_PAIR[qweight].reshape(n, 2 * nb)


def dequant(qweight: np.ndarray, scales: np.ndarray, k: int, dtype=np.float64) -> np.ndarray:
    """W'[n, j] = q[n, j] * s[n, j // 32] for j < k (W4A16 weights, Sec. 3.2).

    The product of a 4-bit integer and an fp16 scale is exact in fp32/fp64.
    Rows are split across threads; each element is still that one product.
    """
    qweight = np.asarray(qweight)
    scales = np.asarray(scales)
    n, nb = qweight.shape
    kp = 2 * nb
    assert kp % GROUP == 0 and scales.shape == (n, kp // GROUP) and k <= kp
    lut = _BYTE_PAIR.astype(dtype)
    out = np.empty((n, kp), dtype=dtype)
    step = 256

    def work(r0):
        r1 = min(n, r0 + step)
        q = lut[qweight[r0:r1]].reshape(r1 - r0, kp // GROUP, GROUP)
        s = scales[r0:r1].astype(dtype)[:, :, None]
        np.multiply(q, s, out=out[r0:r1].reshape(r1 - r0, kp // GROUP, GROUP))

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(work, range(0, n, step)))
    return out[:, :k] if k != kp else out


def decode_e4m3(codes: np.ndarray) -> np.ndarray:
    """Value of each FP8 code in the OCP 8-bit floating-point format E4M3
    (the "fn" variant: no infinities, S.1111.111 is NaN, largest finite
    448): sign bit, 4 exponent bits with bias 7, 3 mantissa bits; exponent
    field 0 holds the subnormals m/8 * 2^-6."""
    c = np.arange(256)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 7
    mag = np.where(e == 0, (m / 8.0) * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    table = sign * mag
    table[(c & 0x7F) == 0x7F] = np.nan
    return table[np.asarray(codes, dtype=np.int64)]


def dequant_fp8(codes: np.ndarray, scales: np.ndarray, dtype=np.float64) -> np.ndarray:
    """W'[n, j] = e4m3(q[n, j]) * s[n] (FP8 weights with one scale per output
    channel, the layout of FP8 checkpoints).  An E4M3 value has 4 significant
    bits, so with an fp32 scale the product is exact in fp64."""
    codes = np.asarray(codes)
    scales = np.asarray(scales, dtype=np.float64)
    assert codes.ndim == 2 and scales.shape == (codes.shape[0],)
    out = decode_e4m3(codes) * scales[:, None]
    return out.astype(dtype)


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gamma over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gamma.astype(x.dtype)


def silu(a: np.ndarray) -> np.ndarray:
    """a * sigmoid(a) = a / (1 + e^-a)."""
    with np.errstate(over="ignore"):
        return a / (1.0 + np.exp(-a))


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [T][H][hd] at integer positions pos [T].

    Pair (i, i + hd/2) is rotated by angle pos * theta^(-2i/hd); the angle,
    its cosine and sine are computed in float64.
    """
    t, h, hd = x.shape
    half = hd // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c = np.cos(ang).astype(x.dtype)[:, None, :]
    s = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x1 * s + x2 * c], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_visible: np.ndarray) -> np.ndarray:
    """Scaled dot-product attention with a visibility limit per query.

    q [Tq][Hq][hd], k, v [Tk][Hkv][hd]; query i sees keys 0 .. n_visible[i]-1.
    Query head j reads key/value head floor(j * Hkv / Hq) (grouped-query).
    """
    tq, hq, hd = q.shape
    tk, hkv, _ = k.shape
    n_visible = np.asarray(n_visible)
    assert n_visible.shape == (tq,) and np.all(n_visible >= 1) and np.all(n_visible <= tk)
    mask = np.arange(tk)[None, :] < n_visible[:, None]
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for j in range(hq):
        g = j * hkv // hq
        s = (q[:, j, :] @ k[:, g, :].T) * scale
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, j, :] = p @ v[:, g, :]
    return out


def _lse(z: np.ndarray) -> float:
    m = np.max(z)
    return float(m + np.log(np.sum(np.exp(z - m))))


def constrained_pick(z: np.ndarray, allowed: Sequence[int]):
    """Type-constrained choice of the next token (Sec. 2.3 "Constrained Decoding").

    Returns (i*, logprob, logprob_full, margin): i* = first index of the
    largest z[allowed[i]]; logprob = z[a*] - LSE_i z[allowed[i]] (the
    distribution renormalised over the allowed set); logprob_full =
    z[a*] - LSE over the whole vocabulary; margin = gap between the two
    largest allowed logits (inf with one allowed token).
    """
    za = np.asarray(z)[np.asarray(allowed)]
    i = int(np.argmax(za))  # numpy returns the first maximum
    lp = float(za[i] - _lse(za))
    lpf = float(za[i] - _lse(np.asarray(z)))
    if len(za) > 1:
        srt = np.sort(za)
        margin = float(srt[-1] - srt[-2])
    else:
        margin = float("inf")
    return i, lp, lpf, margin


def automaton_steps(aut, eos: int):
    """The constrained-decoding grammar of a token automaton (multi-token
    options and other regular output types, Sec. 2.3 "Constrained Decoding").

    `aut` has n_states, edge_offset [n_states + 1], edge_token, edge_next and
    accepting [n_states]; state 0 is the start.  Returns, per state, the
    allowed tokens of a step in that state and the state each one leads to
    (None for EOS).  The allowed tokens are the state's edge tokens ordered by
    where each token first appears in edge_token (this order breaks ties),
    followed by EOS when the state is accepting and an EOS token is given.
    """
    off = np.asarray(aut.edge_offset)
    tok = np.asarray(aut.edge_token)
    nxt = np.asarray(aut.edge_next)
    acc = np.asarray(aut.accepting)
    first = {}
    for t in tok.tolist():
        first.setdefault(t, len(first))
    out = []
    for st in range(int(aut.n_states)):
        edges = sorted(zip(tok[off[st]:off[st + 1]].tolist(), nxt[off[st]:off[st + 1]].tolist()),
                       key=lambda e: first[e[0]])
        allowed = [t for t, _ in edges]
        to = [int(n) for _, n in edges]
        if acc[st] and eos >= 0:
            allowed.append(int(eos))
            to.append(None)
        out.append((np.array(allowed, dtype=np.int64), to))
    return out


def _np(t):
    """Host numpy view/copy of a torch tensor or array-like."""
    if hasattr(t, "detach"):
        t = t.detach()
        if t.device.type != "cpu":
            t = t.cpu()
        return t.numpy()
    return np.asarray(t)


class _Node:
    """A run of tokens that attends to its ancestors' tokens and causally to itself."""

    def __init__(self, tokens: np.ndarray, parent: Optional["_Node"]):
        self.tokens = np.asarray(tokens, dtype=np.int64)
        self.parent = parent
        self.start = 0 if parent is None else parent.start + parent.n
        self.k: List[np.ndarray] = []
        self.v: List[np.ndarray] = []
        self.x_last: Optional[np.ndarray] = None

    @property
    def n(self) -> int:
        return len(self.tokens)

    def chain(self) -> List["_Node"]:
        """This node and its ancestors, root first, skipping empty runs."""
        out = []
        nd = self
        while nd is not None:
            if nd.n > 0:
                out.append(nd)
            nd = nd.parent
        return out[::-1]


class OracleLM:
    """The decoder LM of the module docstring over one set of quantised weights.

    `weights` is duck-typed: .tok_embedding, .lm_head ([V][d] fp16),
    .final_norm, and .layers with .attn_norm, .mlp_norm and the quantised
    matrices .wq .wk .wv .wo .w_gate .w_up .w_down (each .qweight, .scales,
    .n, .k), as torch tensors or numpy arrays.  `shape` supplies n_heads,
    n_kv_heads, head_dim, rms_eps and rope_theta.
    """

    def __init__(self, weights, shape, dtype=np.float64, cache_dequant: Optional[bool] = None):
        self.shape = shape
        self.dtype = np.dtype(dtype)
        self.emb = _np(weights.tok_embedding)
        self.lm_head = _np(weights.lm_head)
        self.final_norm = _np(weights.final_norm)
        self.layers = []
        for l in weights.layers:
            mats = {}
            for name in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
                m = getattr(l, name)
                mats[name] = (_np(m.qweight), _np(m.scales), int(m.n), int(m.k),
                              getattr(m, "fmt", "int4_g32"))
            self.layers.append((_np(l.attn_norm), _np(l.mlp_norm), mats))
        n_params = sum(m[2] * m[3] for _, _, mats in self.layers for m in mats.values())
        if cache_dequant is None:
            cache_dequant = n_params * self.dtype.itemsize < (4 << 30)
        self._cache = {} if cache_dequant else None
        self._head = None

    # -- weights -------------------------------------------------------
    def layer_weights(self, l: int):
        if self._cache is not None and l in self._cache:
            return self._cache[l]
        g1, g2, mats = self.layers[l]
        w = {name: (dequant_fp8(q, s, self.dtype) if fmt == "fp8_e4m3"
                    else dequant(q, s, k, self.dtype))
             for name, (q, s, n, k, fmt) in mats.items()}
        out = (g1, g2, w)
        if self._cache is not None:
            self._cache[l] = out
        return out

    def head_weights(self) -> np.ndarray:
        if self._head is None:
            self._head = self.lm_head.astype(self.dtype)
        return self._head

    # -- plain full forward over one sequence (the definition) ----------
    def forward_sequence(self, tokens: Sequence[int]) -> np.ndarray:
        """Final-layer hidden states [T][d] of one sequence at positions 0..T-1."""
        sh = self.shape
        t = np.asarray(tokens, dtype=np.int64)
        T = len(t)
        x = self.emb[t].astype(self.dtype)
        pos = np.arange(T)
        for l in range(len(self.layers)):
            g1, g2, w = self.layer_weights(l)
            h = rms_norm(x, g1, sh.rms_eps)
            q = (h @ w["wq"].T).reshape(T, sh.n_heads, sh.head_dim)
            k = (h @ w["wk"].T).reshape(T, sh.n_kv_heads, sh.head_dim)
            v = (h @ w["wv"].T).reshape(T, sh.n_kv_heads, sh.head_dim)
            q = rope(q, pos, sh.rope_theta)
            k = rope(k, pos, sh.rope_theta)
            o = attention(q, k, v, pos + 1)
            x = x + o.reshape(T, -1) @ w["wo"].T
            h2 = rms_norm(x, g2, sh.rms_eps)
            x = x + (silu(h2 @ w["w_gate"].T) * (h2 @ w["w_up"].T)) @ w["w_down"].T
        return x

    def logits(self, x_last: np.ndarray) -> np.ndarray:
        """z = RMSNorm(x) * g_final  W_lm^T for hidden rows x_last [R][d]."""
        h = rms_norm(np.atleast_2d(x_last).astype(self.dtype), self.final_norm, self.shape.rms_eps)
        return h @ self.head_weights().T

    # -- forward over a forest of token runs, layer by layer ------------
    def _run(self, nodes: List[_Node]) -> None:
        """Runs the new `nodes` through every layer.  Their ancestors must have
        been run before or appear earlier in `nodes`.  Stores per-layer
        post-RoPE keys and values on each node and its last hidden state."""
        nodes = [nd for nd in nodes if nd.n > 0]
        if not nodes:
            return
        sh = self.shape
        sizes = [nd.n for nd in nodes]
        cuts = np.concatenate([[0], np.cumsum(sizes)])
        T = int(cuts[-1])
        toks = np.concatenate([nd.tokens for nd in nodes])
        pos = np.concatenate([nd.start + np.arange(nd.n) for nd in nodes])
        x = self.emb[toks].astype(self.dtype)
        for nd in nodes:
            nd.k, nd.v = [], []
        for l in range(len(self.layers)):
            g1, g2, w = self.layer_weights(l)
            h = rms_norm(x, g1, sh.rms_eps)
            q = rope((h @ w["wq"].T).reshape(T, sh.n_heads, sh.head_dim), pos, sh.rope_theta)
            k = rope((h @ w["wk"].T).reshape(T, sh.n_kv_heads, sh.head_dim), pos, sh.rope_theta)
            v = (h @ w["wv"].T).reshape(T, sh.n_kv_heads, sh.head_dim)
            for i, nd in enumerate(nodes):
                nd.k.append(k[cuts[i]:cuts[i + 1]])
                nd.v.append(v[cuts[i]:cuts[i + 1]])
            o = np.empty_like(q)
            for i, nd in enumerate(nodes):
                chain = nd.chain()
                kk = np.concatenate([c.k[l] for c in chain])
                vv = np.concatenate([c.v[l] for c in chain])
                past = nd.start
                o[cuts[i]:cuts[i + 1]] = attention(q[cuts[i]:cuts[i + 1]], kk, vv,
                                                   past + np.arange(nd.n) + 1)
            x = x + o.reshape(T, -1) @ w["wo"].T
            h2 = rms_norm(x, g2, sh.rms_eps)
            x = x + (silu(h2 @ w["w_gate"].T) * (h2 @ w["w_up"].T)) @ w["w_down"].T
        for i, nd in enumerate(nodes):
            nd.x_last = x[cuts[i + 1] - 1].copy()

    # -- the operator -----------------------------------------------------
    def eval_rows(self, prefix, suffixes: Sequence[np.ndarray], kind: int, allowed,
                  eos: int = -1, max_tokens: int = 1, children=None, row_child=None,
                  forced: Optional[Sequence[Sequence[int]]] = None, keep_logits: bool = False):
        """Evaluates every row once (LLMMap, Sec. 2.3.2) and returns a dict of
        per-row arrays: value, logprob, logprob_full, n_tokens, tokens [R][8],
        margin (smallest top-two allowed gap over the row's steps) and, with
        keep_logits, logits[r] = list of per-step logit vectors.

        `kind` KIND_AUTOMATON takes a token automaton as `allowed` (see
        automaton_steps); the value is then the final state.

        Sequences are prefix ++ children[row_child[r]] ++ suffixes[r].  The
        prefix (and each child) is run once and its keys/values are reused by
        every row below it.  `forced[r]`, if given, replaces the chosen token
        of each step (teacher forcing) while logits/picks are still reported.
        """
        grammar = None
        if kind == KIND_AUTOMATON:
            grammar = automaton_steps(allowed, eos)
            edge_off = np.asarray(allowed.edge_offset)
            accepting = np.asarray(allowed.accepting)
        else:
            allowed = np.asarray(allowed, dtype=np.int64)
        R = len(suffixes)
        root = _Node(np.asarray(prefix), None) if prefix is not None and len(prefix) else None
        kids = []
        if children is not None:
            kids = [_Node(np.asarray(c), root) for c in children]
        rows = []
        for r in range(R):
            parent = root
            if row_child is not None:
                parent = kids[int(row_child[r])]
            rows.append(_Node(np.asarray(suffixes[r]), parent))
        self._run(([root] if root is not None else []) + kids + rows)

        def last_hidden(nd: _Node):
            while nd is not None and nd.n == 0:
                nd = nd.parent
            if nd is None:
                raise ValueError("row with empty prefix and empty suffix")
            return nd.x_last

        value = np.zeros(R, dtype=np.int64)
        lp = np.zeros(R, dtype=np.float64)
        lpf = np.zeros(R, dtype=np.float64)
        ntok = np.zeros(R, dtype=np.int32)
        toks = np.full((R, 8), -1, dtype=np.int32)
        margin = np.full(R, np.inf)
        logits_out = [[] for _ in range(R)]
        tails = list(rows)
        live = list(range(R))
        digits: List[List[int]] = [[] for _ in range(R)]
        state = np.zeros(R, dtype=np.int64)  # automaton state of each row
        steps = 1 if kind not in (KIND_INT, KIND_AUTOMATON) else max_tokens
        for step in range(steps):
            if not live:
                break
            xs = np.stack([last_hidden(tails[r]) for r in live])
            z = self.logits(xs)
            if kind == KIND_INT and step > 0:
                step_allowed = np.concatenate([allowed, [eos]])
            elif kind != KIND_AUTOMATON:
                step_allowed = allowed
            next_live = []
            for i, r in enumerate(live):
                zi = z[i]
                if kind == KIND_AUTOMATON:
                    step_allowed, step_to = grammar[int(state[r])]
                if keep_logits:
                    logits_out[r].append(zi.copy())
                ci, a, b, m = constrained_pick(zi, step_allowed)
                tok = int(step_allowed[ci])
                if forced is not None and step < len(forced[r]):
                    tok = int(forced[r][step])
                    ci = int(np.nonzero(step_allowed == tok)[0][0])
                    zsel = zi[step_allowed]
                    a = float(zsel[ci] - _lse(zsel))
                    b = float(zi[tok] - _lse(zi))
                lp[r] += a
                lpf[r] += b
                margin[r] = min(margin[r], m)
                toks[r, ntok[r]] = tok
                ntok[r] += 1
                if kind == KIND_INT:
                    if tok == eos:
                        continue
                    digits[r].append(ci)
                    if ntok[r] < max_tokens:
                        next_live.append(r)
                elif kind == KIND_AUTOMATON:
                    # the output ends with EOS, in an accepting state without
                    # edges, or after max_tokens; the value is the final state,
                    # -1 if that state is not accepting
                    if step_to[ci] is None:
                        value[r] = state[r]
                        continue
                    state[r] = step_to[ci]
                    s_new = int(state[r])
                    ends = edge_off[s_new + 1] == edge_off[s_new] or ntok[r] >= max_tokens
                    if ends:
                        value[r] = s_new if accepting[s_new] else -1
                    else:
                        next_live.append(r)
                else:
                    value[r] = ci
            if kind in (KIND_INT, KIND_AUTOMATON) and next_live:
                new = [_Node(np.array([toks[r, ntok[r] - 1]]), tails[r]) for r in next_live]
                for r, nd in zip(next_live, new):
                    tails[r] = nd
                self._run(new)
            live = next_live
        if kind == KIND_INT:
            for r in range(R):
                v = 0
                for dgt in digits[r]:
                    v = 10 * v + dgt
                value[r] = v
        out = dict(value=value, logprob=lp, logprob_full=lpf, n_tokens=ntok, tokens=toks,
                   margin=margin)
        if keep_logits:
            out["logits"] = logits_out
        return out

    def eval_workload(self, wl, rows=None, **kw):
        """eval_rows over a synthetic table (or the listed rows of it)."""
        idx = range(wl.n_rows) if rows is None else rows
        sufs = [wl.suffix(int(r)) for r in idx]
        rc = None if wl.row_child is None else [int(wl.row_child[int(r)]) for r in idx]
        allowed = wl.automaton if getattr(wl, "automaton", None) is not None else wl.allowed
        return self.eval_rows(wl.prefix, sufs, wl.kind, allowed, eos=wl.eos,
                              max_tokens=wl.max_tokens, children=wl.children, row_child=rc, **kw)
