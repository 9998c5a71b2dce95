"""Seeded model weights and row tables shaped like the paper's LLMMap workloads.

The paper runs its LM functions over database rows: one prompt per row
(LLMMap, Sec. 2.3.2 "Refined LLMMap Prompting Pattern"), the rows sharing
the instruction text of the prompt template (Appendix "Prompts"), with
duplicate inputs removed first (Sec. 2.4 "Early Deduplication") and joins
evaluated as LLMMap over DB-built pairs (Sec. 4.1, the ecomm self-join CTE).
It publishes neither its datasets nor its checkpoints, so every input here is
synthetic: uniform random token ids, a Llama-shaped decoder with N(0, 0.02)
weights quantised to symmetric int4 with one fp16 scale per 32 consecutive
input features (W4A16, Sec. 3.2 Table "tab:models"), and suffix lengths drawn
to match the workload recipes below.

Weight tensors are drawn with torch on a chosen device (the 8B shape has
7e9 parameters; drawing them on the host would take minutes), so a given
seed yields the same weights on the same device type.  Row tables are drawn
with numpy PCG64 and are identical everywhere.

Layout of a quantised matrix W [N][K] (y = x W^T):
  qweight uint8 [N][Kp/2], Kp = K rounded up to 32; feature k sits in the
  low nibble of byte k//2 when k is even, the high nibble when odd; each
  nibble is a two's-complement int4 in [-8, 7]; pad features have q = 0.
  scales float16 [N][Kp/32]: one scale per (row, group of 32 features).
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np
import torch

GROUP = 32


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rope_theta: float
    rms_eps: float = 1e-5
    group_size: int = GROUP
    shape_id: int = 0


SHAPES = {
    "tiny": ModelShape("tiny", 2, 256, 4, 4, 64, 688, 2048, 1e4, shape_id=1),
    "1b": ModelShape("1b", 16, 2048, 32, 8, 64, 8192, 128256, 5e5, shape_id=2),
    "8b": ModelShape("8b", 32, 4096, 32, 8, 128, 14336, 128256, 5e5, shape_id=3),
}


@dataclasses.dataclass
class QMat:
    qweight: torch.Tensor  # int4_g32: uint8 [N][Kp/2]; fp8_e4m3: uint8 codes [N][K]
    scales: torch.Tensor   # int4_g32: float16 [N][Kp/32]; fp8_e4m3: float32 [N]
    n: int
    k: int
    fmt: str = "int4_g32"


@dataclasses.dataclass
class Layer:
    attn_norm: torch.Tensor  # float32 [d]
    mlp_norm: torch.Tensor   # float32 [d]
    wq: QMat
    wk: QMat
    wv: QMat
    wo: QMat
    w_gate: QMat
    w_up: QMat
    w_down: QMat


@dataclasses.dataclass
class Weights:
    shape: ModelShape
    tok_embedding: torch.Tensor  # float16 [V][d]
    lm_head: torch.Tensor        # float16 [V][d]
    final_norm: torch.Tensor     # float32 [d]
    layers: List[Layer]

    def to(self, device) -> "Weights":
        def qm(m: QMat) -> QMat:
            return QMat(m.qweight.to(device), m.scales.to(device), m.n, m.k, m.fmt)
        layers = [Layer(l.attn_norm.to(device), l.mlp_norm.to(device), qm(l.wq), qm(l.wk),
                        qm(l.wv), qm(l.wo), qm(l.w_gate), qm(l.w_up), qm(l.w_down))
                  for l in self.layers]
        return Weights(self.shape, self.tok_embedding.to(device), self.lm_head.to(device),
                       self.final_norm.to(device), layers)


def _seed(*parts: int) -> int:
    state = np.random.SeedSequence([int(p) for p in parts]).generate_state(2, np.uint32)
    return int((int(state[0]) << 31) ^ int(state[1])) & ((1 << 62) - 1)


def _normal(shape, std: float, seed: int, device) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32) * std


def quantize_int4_g32(w: torch.Tensor):
    """Symmetric int4 with one fp16 scale per 32 consecutive input features.

    Input generation, not part of the operator: s = fp16(max|w| / 7) per
    group (1 if that is 0), q = clip(round_half_even(w / s), -8, 7).  Returns
    (qweight uint8 [N][Kp/2], scales float16 [N][Kp/32]).
    """
    n, k = w.shape
    kp = (k + GROUP - 1) // GROUP * GROUP
    if kp != k:
        w = torch.nn.functional.pad(w, (0, kp - k))
    g = w.reshape(n, kp // GROUP, GROUP)
    s = (g.abs().amax(-1) / 7.0).to(torch.float16)
    s = torch.where(s == 0, torch.ones_like(s), s)
    q = torch.round(g / s.float().unsqueeze(-1)).clamp_(-8, 7).to(torch.int16).reshape(n, kp)
    lo = q[:, 0::2] & 0xF
    hi = q[:, 1::2] & 0xF
    packed = (lo | (hi << 4)).to(torch.uint8)
    return packed.contiguous(), s.contiguous()


def quantize_fp8_e4m3(w: torch.Tensor):
    """FP8 (OCP e4m3, "fn" variant: max 448, no infinities) with one fp32
    scale per output channel, the layout of FP8 checkpoints.

    Input generation, not part of the operator: s = max|w| / 448 per row (1
    if that is 0), q = e4m3(round to nearest even of w / s, clamped to
    +-448).  Returns (codes uint8 [N][K], scales float32 [N])."""
    s = w.abs().amax(-1) / 448.0
    s = torch.where(s == 0, torch.ones_like(s), s)
    q = (w / s.unsqueeze(-1)).clamp_(-448.0, 448.0).to(torch.float8_e4m3fn)
    return q.view(torch.uint8).contiguous(), s.float().contiguous()


def make_weights(shape: ModelShape, seed: int = 1234, device="cpu", std: float = 0.02,
                 n_layers: Optional[int] = None, fmt: str = "int4_g32") -> Weights:
    """Random-init weights of `shape`, linear layers quantised to int4 g32
    (fmt "int4_g32") or to FP8 e4m3 with per-channel scales ("fp8_e4m3").

    Each tensor has its own stream keyed by (seed, shape, layer, tensor), so a
    model with fewer layers is a prefix of the full one.
    """
    dev = torch.device(device)
    sid = shape.shape_id
    d, hd = shape.d_model, shape.head_dim
    nq, nkv, f = shape.n_heads * hd, shape.n_kv_heads * hd, shape.d_ff
    L = shape.n_layers if n_layers is None else n_layers

    def qmat(layer: int, tid: int, n: int, k: int) -> QMat:
        w = _normal((n, k), std, _seed(seed, sid, layer, tid), dev)
        if fmt == "fp8_e4m3":
            qw, sc = quantize_fp8_e4m3(w)
        else:
            qw, sc = quantize_int4_g32(w)
        del w
        return QMat(qw, sc, n, k, fmt)

    emb = _normal((shape.vocab, d), std, _seed(seed, sid, 10_000, 0), dev).to(torch.float16)
    head = _normal((shape.vocab, d), std, _seed(seed, sid, 10_000, 1), dev).to(torch.float16)
    ones = torch.ones(d, dtype=torch.float32, device=dev)
    layers = []
    for l in range(L):
        layers.append(Layer(
            attn_norm=ones.clone(), mlp_norm=ones.clone(),
            wq=qmat(l, 0, nq, d), wk=qmat(l, 1, nkv, d), wv=qmat(l, 2, nkv, d),
            wo=qmat(l, 3, d, nq), w_gate=qmat(l, 4, f, d), w_up=qmat(l, 5, f, d),
            w_down=qmat(l, 6, d, f)))
    return Weights(shape, emb, head, ones.clone(), layers)


# --------------------------------------------------------------------------
# Row tables
# --------------------------------------------------------------------------

KIND_BOOL, KIND_ENUM, KIND_INT, KIND_AUTOMATON = 0, 1, 2, 3


@dataclasses.dataclass
class Automaton:
    """A token automaton (data only): state 0 starts; state s has the edges
    edge_token[edge_offset[s]:edge_offset[s+1]] -> edge_next[...];
    accepting[s] != 0 lets an output end in s."""
    n_states: int
    edge_offset: np.ndarray   # int32 [n_states + 1]
    edge_token: np.ndarray    # int32 [n_edges]
    edge_next: np.ndarray     # int32 [n_edges]
    accepting: np.ndarray     # uint8 [n_states]


def option_trie(options) -> "tuple[Automaton, np.ndarray]":
    """The prefix tree of token-string options: one state per distinct option
    prefix (state 0 = empty), edges in order of first use, the state of each
    whole option accepting.  Returns the automaton and, per option, its
    final state."""
    children = [dict()]
    final = []
    for opt in options:
        st = 0
        for t in (int(x) for x in opt):
            nxt = children[st].get(t)
            if nxt is None:
                nxt = len(children)
                children[st][t] = nxt
                children.append(dict())
            st = nxt
        final.append(st)
    n = len(children)
    off = np.zeros(n + 1, dtype=np.int32)
    tok, nx = [], []
    for s in range(n):
        for t, c in children[s].items():
            tok.append(t)
            nx.append(c)
        off[s + 1] = len(tok)
    acc = np.zeros(n, dtype=np.uint8)
    acc[final] = 1
    aut = Automaton(n, off, np.array(tok, dtype=np.int32), np.array(nx, dtype=np.int32), acc)
    return aut, np.array(final, dtype=np.int64)


def automaton_of_options(n_options: int, V: int, rng, max_len: int = 3, n_heads: int = 8):
    """Options of 1..max_len tokens whose first tokens come from a pool of
    n_heads ids (so the options share prefixes), no option a prefix of
    another: a synthetic multi-token option set and its trie."""
    heads = rng.choice(V, size=n_heads, replace=False)
    opts, seen = [], set()
    while len(opts) < n_options:
        n = int(rng.integers(1, max_len + 1))
        o = tuple([int(heads[rng.integers(0, n_heads)])] +
                  [int(x) for x in rng.integers(0, V, size=n - 1)])
        clash = any(o == q[:len(o)] or q == o[:len(q)] for q in seen)
        if not clash:
            seen.add(o)
            opts.append(np.array(o, dtype=np.int32))
    aut, final = option_trie(opts)
    return opts, aut, final


def _automaton_of_dicts(edges, accepting) -> Automaton:
    """Packs per-state {token: next state} dicts (edge order = insertion
    order) and accepting flags into the CSR automaton."""
    off, tok, nxt = [0], [], []
    for e in edges:
        for t, c in e.items():
            tok.append(int(t))
            nxt.append(int(c))
        off.append(len(tok))
    return Automaton(len(edges), np.array(off, dtype=np.int32), np.array(tok, dtype=np.int32),
                     np.array(nxt, dtype=np.int32), np.array(accepting, dtype=np.uint8))


def automaton_of_list(items, sep: int, lo: int, hi: int) -> Automaton:
    """A collection output (Sec. 2.3: a list return type with a regex-style
    quantifier {lo,hi}): lo..hi items, each one of the token strings
    `items`, with the token `sep` between two items.  The automaton is hi
    copies of the items' trie; copy c holds item c + 1.  Where an item ends
    in copy c, `sep` leads to copy c + 1 (if c + 1 < hi) and the output may
    end (if c + 1 >= lo).  {3} is lo = hi = 3."""
    if not 1 <= lo <= hi:
        raise ValueError(f"quantifier {{{lo},{hi}}}: need 1 <= lo <= hi")
    if any(int(sep) in {int(t) for t in it} for it in items):
        raise ValueError("the separator is a token of an item")
    trie, final = option_trie(items)
    n = trie.n_states
    ends = set(int(f) for f in final)
    edges, acc = [], []
    for c in range(hi):
        for st in range(n):
            e = {int(trie.edge_token[i]): c * n + int(trie.edge_next[i])
                 for i in range(trie.edge_offset[st], trie.edge_offset[st + 1])}
            if st in ends and c + 1 < hi:
                e[int(sep)] = (c + 1) * n
            edges.append(e)
            acc.append(1 if st in ends and c + 1 >= lo else 0)
    return _automaton_of_dicts(edges, acc)


def automaton_of_record(open_tok: int, close_tok: int, sep: int, fields) -> Automaton:
    """A JSON-shaped record over token ids (Sec. 5: a JSON object with a given
    schema): open_tok, the fields in order separated by sep, close_tok.  A
    field is ("enum", key, values): its key token (standing for the
    `"name":` text) and one of the single-token values; or ("int", key,
    digits, max_digits): its key token and 1..max_digits of the 10 digit
    tokens.  The state after close_tok is the only accepting state and has
    no edges, so a complete record ends the output."""
    edges, acc = [], []

    def new():
        edges.append({})
        acc.append(0)
        return len(edges) - 1

    def add(st, t, nx):
        if int(t) in edges[st]:
            raise ValueError(f"token {t} has two meanings in one state")
        edges[st][int(t)] = nx

    exits = [new()]
    for i, f in enumerate(fields):
        lit = open_tok if i == 0 else sep
        st = new()
        for e in exits:
            add(e, lit, st)
        key = new()
        add(st, f[1], key)
        if f[0] == "enum":
            after = new()
            for v in f[2]:
                add(key, v, after)
            exits = [after]
        elif f[0] == "int":
            digits, max_digits = f[2], int(f[3])
            if len(digits) != 10 or max_digits < 1:
                raise ValueError("an int field needs 10 digit tokens and max_digits >= 1")
            exits, prev = [], key
            for _ in range(max_digits):
                d = new()
                for t in digits:
                    add(prev, t, d)
                exits.append(d)
                prev = d
        else:
            raise ValueError(f"unknown field kind {f[0]!r}")
    end = new()
    for e in exits:
        add(e, close_tok, end)
    acc[end] = 1
    return _automaton_of_dicts(edges, acc)


@dataclasses.dataclass
class Workload:
    """A table of rows for one LM-operator call.

    Every row's sequence is prefix ++ child[row_child[r]] (if any) ++ suffix_r.
    `tokens`/`offsets` is the CSR of the row suffixes.
    """
    name: str
    shape: ModelShape
    prefix: np.ndarray                  # int32 [P]
    tokens: np.ndarray                  # int32 [sum S_r]
    offsets: np.ndarray                 # int64 [n_rows + 1]
    kind: int
    allowed: np.ndarray                 # int32 [n_allowed]; INT: the 10 digit tokens
    eos: int = -1
    max_tokens: int = 1
    children: Optional[List[np.ndarray]] = None   # second-level prefixes (joins)
    row_child: Optional[np.ndarray] = None         # int32 [n_rows]
    automaton: Optional[Automaton] = None          # KIND_AUTOMATON: the output grammar
    options: Optional[List[np.ndarray]] = None     # its option strings, if it is a trie

    @property
    def n_rows(self) -> int:
        return len(self.offsets) - 1

    @property
    def type_spec(self):
        """What the output type is given by: the automaton for
        KIND_AUTOMATON, otherwise the allowed token list."""
        return self.automaton if self.kind == KIND_AUTOMATON else self.allowed

    def suffix(self, r: int) -> np.ndarray:
        return self.tokens[self.offsets[r]:self.offsets[r + 1]]

    def row_prefix(self, r: int) -> np.ndarray:
        if self.row_child is None:
            return self.prefix
        return np.concatenate([self.prefix, self.children[int(self.row_child[r])]])

    def subset(self, rows) -> "Workload":
        rows = np.asarray(rows, dtype=np.int64)
        parts = [self.suffix(int(r)) for r in rows]
        lens = np.array([len(p) for p in parts], dtype=np.int64)
        offs = np.zeros(len(rows) + 1, dtype=np.int64)
        np.cumsum(lens, out=offs[1:])
        toks = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
        rc = None if self.row_child is None else self.row_child[rows].astype(np.int32)
        return dataclasses.replace(self, name=f"{self.name}[subset {len(rows)}]", tokens=toks,
                                   offsets=offs, row_child=rc)

    @property
    def n_suffix_tokens(self) -> int:
        return int(self.offsets[-1])


def parity_rows(wl: "Workload", n: int, seed: int) -> List[int]:
    """n row indices of a table for a parity sample: its longest row, its
    shortest, the first and the last, the rest drawn uniformly (seeded)."""
    lens = np.diff(wl.offsets)
    rng = np.random.default_rng(seed)
    pick = {int(np.argmax(lens)), int(np.argmin(lens)), 0, wl.n_rows - 1}
    n = min(n, wl.n_rows)
    while len(pick) < n:
        pick.add(int(rng.integers(0, wl.n_rows)))
    return sorted(pick)


def _csr(parts):
    lens = np.array([len(p) for p in parts], dtype=np.int64)
    offs = np.zeros(len(parts) + 1, dtype=np.int64)
    np.cumsum(lens, out=offs[1:])
    toks = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
    return toks, offs


def _lognormal_lengths(rng, n, mean, lo, hi, sigma=0.75):
    mu = math.log(mean) - sigma * sigma / 2.0
    return np.clip(np.rint(rng.lognormal(mu, sigma, size=n)), lo, hi).astype(np.int64)


def make_workload(name: str, seed: int = 7, n_rows: Optional[int] = None) -> Workload:
    """Synthetic LM-operator table.  `name` is one of WORKLOADS.

    filter_tiny   tiny decoder, 64 rows, prefix 96, suffix U{16..48}, bool
    filter_1b     1B shape, 4,096 rows, prefix 384, suffix lognormal mean 40 in [8,256], bool
    filter_8b     8B shape, 10,000 rows, prefix 512, suffix lognormal mean 60 in [8,512],
                  enum over 24 tokens
    map_int_8b    8B shape, prefix 256, 20,000 rows drawn Zipf(1.1) from 5,000 distinct
                  suffixes of U{24..64} tokens; integer output over 10 digits + EOS, <= 4 tokens
    join_8b       8B shape, instruction 320, 200 left x 200 right values of U{8..32} tokens,
                  all 40,000 pairs left-major; bool; one child prefix per left value
    options_tiny  as filter_tiny, output one of 24 options of 1..3 tokens (a token trie)
    options_8b    as filter_8b, output one of 24 options of 1..3 tokens (a token trie)
    qa_tiny       LLMQA: tiny decoder, 2 prompts of 96 + 1,500 tokens, one of 24 options
    qa_8b         LLMQA: 8B shape, one prompt of 256 + 8,192 tokens, one of 24 options
    `n_rows` truncates the table to its first rows (same draws otherwise).
    """
    cfg = WORKLOADS[name]
    rng = np.random.default_rng([seed, cfg["id"]])
    shape = SHAPES[cfg["shape"]]
    V = shape.vocab
    prefix = rng.integers(0, V, size=cfg["prefix"], dtype=np.int64).astype(np.int32)
    n_allowed = cfg["n_allowed"]
    allowed = rng.choice(V, size=n_allowed, replace=False).astype(np.int32)
    eos = -1
    if cfg["kind"] == KIND_INT:
        while True:
            e = int(rng.integers(0, V))
            if e not in set(allowed.tolist()):
                eos = e
                break
    children = row_child = None
    automaton = options = None
    if cfg["kind"] == KIND_AUTOMATON:
        options, automaton, _ = automaton_of_options(cfg["n_allowed"], V, rng,
                                                     max_len=cfg["max_tokens"])
        allowed = np.zeros(0, dtype=np.int32)
    if name == "map_int_8b":
        n_distinct, n_total = 5000, 20000
        lens = rng.integers(24, 65, size=n_distinct)
        distinct = [rng.integers(0, V, size=int(s)).astype(np.int32) for s in lens]
        ranks = np.arange(1, n_distinct + 1, dtype=np.float64)
        p = ranks ** -1.1
        p /= p.sum()
        perm = rng.permutation(n_distinct)
        draws = rng.choice(n_distinct, size=n_total, p=p)
        parts = [distinct[perm[k]] for k in draws]
    elif name == "join_8b":
        n_left = n_right = 200
        llen = rng.integers(8, 33, size=n_left)
        rlen = rng.integers(8, 33, size=n_right)
        children = [rng.integers(0, V, size=int(s)).astype(np.int32) for s in llen]
        rights = [rng.integers(0, V, size=int(s)).astype(np.int32) for s in rlen]
        parts = [rights[j] for i in range(n_left) for j in range(n_right)]
        row_child = np.repeat(np.arange(n_left, dtype=np.int32), n_right)
    else:
        n = cfg["rows"]
        if cfg["len"][0] == "uniform":
            lens = rng.integers(cfg["len"][1], cfg["len"][2] + 1, size=n)
        elif cfg["len"][0] == "fixed":
            lens = np.full(n, cfg["len"][1], dtype=np.int64)
        else:
            lens = _lognormal_lengths(rng, n, cfg["len"][1], cfg["len"][2], cfg["len"][3])
        parts = [rng.integers(0, V, size=int(s)).astype(np.int32) for s in lens]
    if n_rows is not None:
        parts = parts[:n_rows]
        if row_child is not None:
            row_child = row_child[:n_rows]
    toks, offs = _csr(parts)
    return Workload(name=name, shape=shape, prefix=prefix, tokens=toks, offsets=offs,
                    kind=cfg["kind"], allowed=allowed, eos=eos, max_tokens=cfg["max_tokens"],
                    children=children, row_child=row_child, automaton=automaton,
                    options=options)


WORKLOADS = {
    "filter_tiny": dict(id=1, shape="tiny", rows=64, prefix=96, len=("uniform", 16, 48),
                        kind=KIND_BOOL, n_allowed=2, max_tokens=1),
    "filter_1b": dict(id=2, shape="1b", rows=4096, prefix=384, len=("lognormal", 40, 8, 256),
                      kind=KIND_BOOL, n_allowed=2, max_tokens=1),
    "filter_8b": dict(id=3, shape="8b", rows=10000, prefix=512, len=("lognormal", 60, 8, 512),
                      kind=KIND_ENUM, n_allowed=24, max_tokens=1),
    "map_int_8b": dict(id=4, shape="8b", rows=20000, prefix=256, len=None,
                       kind=KIND_INT, n_allowed=10, max_tokens=4),
    "join_8b": dict(id=5, shape="8b", rows=40000, prefix=320, len=None,
                    kind=KIND_BOOL, n_allowed=2, max_tokens=1),
    "options_tiny": dict(id=6, shape="tiny", rows=64, prefix=96, len=("uniform", 16, 48),
                         kind=KIND_AUTOMATON, n_allowed=24, max_tokens=3),
    "options_8b": dict(id=7, shape="8b", rows=10000, prefix=512, len=("lognormal", 60, 8, 512),
                       kind=KIND_AUTOMATON, n_allowed=24, max_tokens=3),
    # LLMQA (Sec. 2.3.1): one long prompt holding a whole subset of the data
    "qa_tiny": dict(id=8, shape="tiny", rows=2, prefix=96, len=("fixed", 1500),
                    kind=KIND_AUTOMATON, n_allowed=24, max_tokens=3),
    "qa_8b": dict(id=9, shape="8b", rows=1, prefix=256, len=("fixed", 8192),
                  kind=KIND_AUTOMATON, n_allowed=24, max_tokens=3),
}
