"""Comparison of the library's results with the oracle's.

Tolerance (stated for this operator): every compared logit satisfies
|z_gpu - z_oracle| <= 0.05 * std(oracle logits), the std pooled over all
compared logits of the call; typed outputs (value, tokens) agree exactly on
every row whose smallest top-two allowed-logit margin in the oracle exceeds
0.1.  Multi-step (integer) rows compare step s only while the library's
tokens of steps < s equal the oracle's; a row whose path diverged after a
sub-margin step is checked by teacher forcing the oracle on the library's
tokens (so every step's logits are still compared).
"""
import numpy as np

TOL_REL = 0.05
MARGIN = 0.1


def compare(orc, out, dbg, label="", orc_forced=None, cols=None):
    """orc: oracle eval_rows dict (keep_logits=True); out: library results;
    dbg: library logits [R][steps][V]; orc_forced: oracle re-run with
    forced = library tokens (needed only if some row's path diverged).
    cols: the allowed token ids (INT: EOS included) when the library ran the
    restricted head; then only those logits exist (the rest must be NaN),
    the scale is still the std of the oracle's full logits, and
    logprob_full must be NaN."""
    if cols is not None:
        cols = np.asarray(cols)
        others = np.ones(dbg.shape[-1], bool)
        others[cols] = False

    def pick(zg, zo):
        if cols is None:
            return zg, zo
        assert np.all(np.isnan(zg[others])), f"{label}: restricted logits outside the allowed set"
        return zg[cols], zo[cols]
    R = len(out)
    diffs, refs = [], []
    n_exact = n_checked = 0
    diverged = []
    worst = 0.0
    for r in range(R):
        ot = orc["tokens"][r][: orc["n_tokens"][r]].tolist()
        gt = out["tokens"][r][: out["n_tokens"][r]].tolist()
        for s, zo in enumerate(orc["logits"][r]):
            if s > 0 and ot[:s] != gt[:s]:
                break
            zg, zc = pick(dbg[r, s], zo)
            assert np.all(np.isfinite(zg)), f"{label} row {r} step {s}: non-finite logits"
            d = np.abs(zg.astype(np.float64) - zc)
            diffs.append(d.max())
            refs.append(zo)
        if ot != gt:
            diverged.append(r)
        if orc["margin"][r] > MARGIN:
            n_checked += 1
            assert ot == gt and int(out["value"][r]) == int(orc["value"][r]), (
                f"{label} row {r}: typed output differs with margin {orc['margin'][r]:.3f}: "
                f"gpu {gt} / {out['value'][r]} vs oracle {ot} / {orc['value'][r]}")
            n_exact += 1
    if diverged and orc_forced is not None:
        for r in diverged:
            for s, zo in enumerate(orc_forced["logits"][r]):
                zg, zc = pick(dbg[r, s], zo)
                diffs.append(np.abs(zg.astype(np.float64) - zc).max())
                refs.append(zo)
    sigma = float(np.concatenate(refs).std())
    worst = float(max(diffs)) if diffs else 0.0
    ratio = worst / sigma
    assert ratio <= TOL_REL, f"{label}: max|dlogit| = {worst:.4g} = {ratio:.4f} sigma > {TOL_REL}"
    # the log-probabilities follow from the logits: at most twice the logit error each step
    same = [r for r in range(R) if r not in diverged]
    if same:
        steps = np.array([out["n_tokens"][r] for r in same])
        dlp = np.abs(out["logprob"][same] - orc["logprob"][same])
        dlpf = np.abs(out["logprob_full"][same] - orc["logprob_full"][same])
        bound = 2 * worst * steps + 1e-3 * steps
        assert np.all(dlp <= bound), f"{label}: logprob off by {dlp.max():.4g}"
        if cols is None:
            assert np.all(dlpf <= bound + 1e-3 * steps), f"{label}: logprob_full off by {dlpf.max():.4g}"
    if cols is not None:
        assert np.all(np.isnan(out["logprob_full"])), f"{label}: restricted head gave logprob_full"
    return dict(max_abs=worst, sigma=sigma, ratio=ratio, rows=R, exact_checked=n_checked,
                diverged=len(diverged))


def assert_typed(out, kind, n_allowed, allowed, eos=-1, max_tokens=1):
    """Every result is a well-formed value of its type (Sec. 2.3 "Constrained Decoding")."""
    allowed = list(map(int, allowed))
    for r in range(len(out)):
        n = int(out["n_tokens"][r])
        toks = out["tokens"][r][:n].tolist()
        assert np.all(out["tokens"][r][n:] == -1)
        assert out["logprob"][r] <= 1e-6
        assert np.isnan(out["logprob_full"][r]) or out["logprob_full"][r] <= out["logprob"][r] + 1e-5
        if kind == 2:
            assert 1 <= n <= max_tokens and toks[0] in allowed
            assert all(t in allowed for t in toks[:-1])
            assert toks[-1] in allowed or (toks[-1] == eos and n >= 2)
            if toks[-1] != eos:
                assert n == max_tokens
            digits = [allowed.index(t) for t in toks if t != eos]
            assert int(out["value"][r]) == int("".join(map(str, digits)))
        else:
            assert n == 1 and toks[0] in allowed
            assert allowed[int(out["value"][r])] == toks[0]
            assert 0 <= out["value"][r] < n_allowed


def assert_automaton(out, aut, eos=-1, max_tokens=1):
    """Every result is a path of the token automaton from state 0 that ends
    on EOS, at an accepting state without edges or after max_tokens; the
    value is the final state, -1 if that state is not accepting."""
    off, tok, nxt, acc = (np.asarray(aut.edge_offset), np.asarray(aut.edge_token),
                          np.asarray(aut.edge_next), np.asarray(aut.accepting))
    for r in range(len(out)):
        n = int(out["n_tokens"][r])
        toks = out["tokens"][r][:n].tolist()
        assert np.all(out["tokens"][r][n:] == -1)
        assert 1 <= n <= max_tokens and out["logprob"][r] <= 1e-6
        st, ended = 0, None
        for i, t in enumerate(toks):
            assert ended is None, f"row {r}: token after the end"
            if eos >= 0 and t == eos:
                assert acc[st], f"row {r}: EOS in a non-accepting state"
                ended = st
                continue
            edges = tok[off[st]:off[st + 1]].tolist()
            assert t in edges, f"row {r}: token {t} is not an edge of state {st}"
            st = int(nxt[off[st] + edges.index(t)])
            if off[st + 1] == off[st]:
                ended = st
        if ended is None:
            assert n == max_tokens, f"row {r}: stopped early in state {st}"
            ended = st
        want = ended if acc[ended] else -1
        assert int(out["value"][r]) == want, f"row {r}: value {out['value'][r]} != {want}"
