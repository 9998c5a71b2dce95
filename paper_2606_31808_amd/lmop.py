"""Python binding of liblmop (include/lmop.h): argument marshalling only.

Every computation runs in the library's HIP kernels; this module converts
numpy / torch arguments to the C structs and back.  The functions keep the C
names (lmop_create, lmop_load_weights, lmop_set_prefix, lmop_eval_rows, ...);
`Context` bundles them for convenience.  If the built library is missing,
importing the binding raises: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "liblmop.so")

LMOP_OK, LMOP_ERR_INVALID_ARG, LMOP_ERR_STATE, LMOP_ERR_OOM, LMOP_ERR_DEVICE, \
    LMOP_ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
LMOP_BOOL, LMOP_ENUM, LMOP_INT, LMOP_AUTOMATON = 0, 1, 2, 3
LMOP_W_INT4_G32, LMOP_W_FP8_E4M3 = 0, 1
_WEIGHT_FORMATS = {"int4_g32": LMOP_W_INT4_G32, "fp8_e4m3": LMOP_W_FP8_E4M3}
LMOP_NO_DEDUP = 1
LMOP_HEAD_RESTRICTED = 2

EXPORTED = (
    "lmop_create", "lmop_destroy", "lmop_last_error", "lmop_status_string", "lmop_load_weights",
    "lmop_set_prefix", "lmop_set_prefixes", "lmop_release_prefix", "lmop_prefix_length", "lmop_eval_rows",
    "lmop_dedup_rows", "lmop_set_profiling", "lmop_get_kernel_stats", "lmop_set_workspace",
    "lmop_get_memory", "lmop_eval_rows_noalloc", "lmop_plan_rows",
)
# size of the static device array lmop_eval_rows_noalloc carves its scratch from
LMOP_NOALLOC_SCRATCH_BYTES = 256 << 20


class lmop_config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ff", C.c_int32),
                ("vocab", C.c_int32), ("group_size", C.c_int32), ("rms_eps", C.c_float),
                ("rope_theta", C.c_float), ("max_seq", C.c_int32)]


class lmop_qmat(C.Structure):
    _fields_ = [("qweight", C.c_void_p), ("scales", C.c_void_p), ("n", C.c_int32),
                ("k", C.c_int32)]


class lmop_layer(C.Structure):
    _fields_ = [("attn_norm", C.c_void_p), ("mlp_norm", C.c_void_p), ("wq", lmop_qmat),
                ("wk", lmop_qmat), ("wv", lmop_qmat), ("wo", lmop_qmat), ("w_gate", lmop_qmat),
                ("w_up", lmop_qmat), ("w_down", lmop_qmat)]


class lmop_weights(C.Structure):
    _fields_ = [("tok_embedding", C.c_void_p), ("lm_head", C.c_void_p),
                ("final_norm", C.c_void_p), ("layers", C.POINTER(lmop_layer)),
                ("n_layers", C.c_int32), ("on_device", C.c_int32), ("format", C.c_int32)]


class lmop_automaton(C.Structure):
    _fields_ = [("n_states", C.c_int32), ("edge_offset", C.POINTER(C.c_int32)),
                ("edge_token", C.POINTER(C.c_int32)), ("edge_next", C.POINTER(C.c_int32)),
                ("accepting", C.POINTER(C.c_uint8))]


class lmop_type(C.Structure):
    _fields_ = [("kind", C.c_int32), ("tokens", C.POINTER(C.c_int32)), ("n_tokens", C.c_int32),
                ("eos_token", C.c_int32), ("max_tokens", C.c_int32),
                ("automaton", C.POINTER(lmop_automaton))]


class lmop_result(C.Structure):
    _fields_ = [("value", C.c_int64), ("logprob", C.c_float), ("logprob_full", C.c_float),
                ("n_tokens", C.c_int32), ("tokens", C.c_int32 * 8)]


class lmop_eval_opts(C.Structure):
    _fields_ = [("flags", C.c_uint32), ("max_batch_tokens", C.c_int32),
                ("debug_logits", C.POINTER(C.c_float)), ("limit", C.c_int32),
                ("limit_value", C.c_int64), ("row_mask", C.POINTER(C.c_uint8))]


class lmop_memory_stats(C.Structure):
    _fields_ = [("device_bytes", C.c_uint64), ("device_peak", C.c_uint64),
                ("workspace_bytes", C.c_uint64), ("workspace_peak", C.c_uint64)]


class lmop_eval_plan(C.Structure):
    _fields_ = [("unique_rows", C.c_int32), ("batches", C.c_int32), ("batch_tokens", C.c_int32),
                ("max_batch_tokens", C.c_int32), ("decode_groups", C.c_int32),
                ("pad_", C.c_int32), ("scratch_bytes", C.c_uint64), ("own_kv_bytes", C.c_uint64),
                ("min_workspace_bytes", C.c_uint64)]


class lmop_kernel_stat(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("launches", C.c_int64), ("timed_launches", C.c_int64),
                ("total_ms", C.c_double), ("flops", C.c_double), ("bytes", C.c_double)]


RESULT_DTYPE = np.dtype([("value", "<i8"), ("logprob", "<f4"), ("logprob_full", "<f4"),
                         ("n_tokens", "<i4"), ("tokens", "<i4", (8,)), ("_pad", "<i4")])
assert C.sizeof(lmop_result) == RESULT_DTYPE.itemsize


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_31808_amd.build`")
    # torch ships its own HIP runtime under the same soname.  Loading it first
    # makes the library bind to that one runtime: the streams and device
    # pointers torch hands over are only valid there, and a second runtime
    # loaded beside it finds no devices.
    import torch  # noqa: F401
    lib = C.CDLL(LIB_PATH)
    vp, i32, st = C.c_void_p, C.c_int32, C.c_int
    sig = {
        "lmop_create": (st, [C.POINTER(lmop_config), i32, vp, C.POINTER(vp)]),
        "lmop_destroy": (None, [vp]),
        "lmop_last_error": (C.c_char_p, [vp]),
        "lmop_status_string": (C.c_char_p, [st]),
        "lmop_load_weights": (st, [vp, C.POINTER(lmop_weights)]),
        "lmop_set_prefix": (st, [vp, vp, C.POINTER(C.c_int32), i32, C.POINTER(vp)]),
        "lmop_set_prefixes": (st, [vp, vp, C.POINTER(C.c_int32), C.POINTER(C.c_int64), i32,
                                   C.POINTER(vp)]),
        "lmop_release_prefix": (st, [vp, vp]),
        "lmop_prefix_length": (i32, [vp]),
        "lmop_eval_rows": (st, [vp, vp, C.POINTER(vp), C.POINTER(C.c_int32),
                                C.POINTER(C.c_int64), i32, C.POINTER(lmop_type), vp,
                                C.POINTER(lmop_eval_opts)]),
        "lmop_eval_rows_noalloc": (st, [vp, vp, C.POINTER(vp), C.POINTER(C.c_int32),
                                        C.POINTER(C.c_int64), i32, C.POINTER(lmop_type), vp,
                                        C.POINTER(lmop_eval_opts)]),
        "lmop_plan_rows": (st, [vp, vp, C.POINTER(vp), C.POINTER(C.c_int32),
                                C.POINTER(C.c_int64), i32, C.POINTER(lmop_type),
                                C.POINTER(lmop_eval_opts), C.POINTER(lmop_eval_plan)]),
        "lmop_set_workspace": (st, [vp, vp, C.c_size_t]),
        "lmop_get_memory": (st, [vp, C.POINTER(lmop_memory_stats)]),
        "lmop_dedup_rows": (st, [C.POINTER(C.c_int32), C.POINTER(C.c_int64), i32,
                                 C.POINTER(C.c_int64), C.POINTER(C.c_int32),
                                 C.POINTER(C.c_int32)]),
        "lmop_set_profiling": (st, [vp, i32]),
        "lmop_get_kernel_stats": (st, [vp, C.POINTER(lmop_kernel_stat), i32,
                                       C.POINTER(C.c_int32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


class LmopError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_lib.lmop_status_string(status).decode()} ({status}): {message}")
        self.status = status


def _check(status: int, ctx) -> None:
    if status != LMOP_OK:
        msg = _lib.lmop_last_error(ctx)
        raise LmopError(status, msg.decode() if msg else "")


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _ptr(a: np.ndarray, ct):
    return a.ctypes.data_as(C.POINTER(ct))


# ---------------------------------------------------------------- C-named calls
def lmop_create(cfg: lmop_config, device: int = 0, stream: Optional[int] = None):
    out = C.c_void_p()
    st = _lib.lmop_create(C.byref(cfg), device, C.c_void_p(stream or 0), C.byref(out))
    _check(st, None)
    return out


def lmop_destroy(ctx) -> None:
    _lib.lmop_destroy(ctx)


def _tensor_ptr(t, keep):
    """Device or host address of a contiguous torch tensor / numpy array."""
    if hasattr(t, "data_ptr"):
        t = t.contiguous()
        keep.append(t)
        return t.data_ptr(), t.device.type != "cpu"
    a = np.ascontiguousarray(t)
    keep.append(a)
    return a.ctypes.data, False


def lmop_load_weights(ctx, weights) -> None:
    """weights: object with tok_embedding, lm_head (fp16 [V][d]), final_norm, layers[...]
    (attn_norm, mlp_norm, wq .. w_down each with qweight/scales/n/k and a format name
    `fmt`, "int4_g32" (default) or "fp8_e4m3"), all on one device."""
    keep = []
    where = set()

    def p(t):
        a, dev = _tensor_ptr(t, keep)
        where.add(dev)
        return a

    def qm(m):
        return lmop_qmat(p(m.qweight), p(m.scales), int(m.n), int(m.k))

    L = len(weights.layers)
    arr = (lmop_layer * max(L, 1))()
    for i, l in enumerate(weights.layers):
        arr[i] = lmop_layer(p(l.attn_norm), p(l.mlp_norm), qm(l.wq), qm(l.wk), qm(l.wv), qm(l.wo),
                            qm(l.w_gate), qm(l.w_up), qm(l.w_down))
    fmts = {getattr(getattr(l, nm), "fmt", "int4_g32") for l in weights.layers
            for nm in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")}
    if len(fmts) > 1:
        raise ValueError("all linear maps must have one weight format")
    fmt = _WEIGHT_FORMATS[fmts.pop() if fmts else "int4_g32"]
    w = lmop_weights(p(weights.tok_embedding), p(weights.lm_head), p(weights.final_norm),
                     C.cast(arr, C.POINTER(lmop_layer)), L, 0, fmt)
    if len(where) != 1:
        raise ValueError("weights must all be on the host or all on the device")
    w.on_device = 1 if where.pop() else 0
    _check(_lib.lmop_load_weights(ctx, C.byref(w)), ctx)


def lmop_set_prefix(ctx, tokens, parent=None):
    t = _i32(tokens)
    out = C.c_void_p()
    _check(_lib.lmop_set_prefix(ctx, parent, _ptr(t, C.c_int32), len(t), C.byref(out)), ctx)
    return out


def lmop_set_prefixes(ctx, token_lists, parent=None):
    lists = [_i32(t) for t in token_lists]
    n = len(lists)
    offs = np.zeros(n + 1, dtype=np.int64)
    offs[1:] = np.cumsum([len(t) for t in lists])
    t = np.concatenate(lists) if n else np.zeros(0, dtype=np.int32)
    t = np.ascontiguousarray(t, dtype=np.int32)
    out = (C.c_void_p * max(n, 1))()
    _check(_lib.lmop_set_prefixes(ctx, parent, _ptr(t, C.c_int32), _ptr(offs, C.c_int64), n,
                                  out), ctx)
    return [C.c_void_p(out[i]) for i in range(n)]


def lmop_release_prefix(ctx, prefix) -> None:
    _check(_lib.lmop_release_prefix(ctx, prefix), ctx)


def lmop_prefix_length(prefix) -> int:
    return int(_lib.lmop_prefix_length(prefix))


def lmop_eval_rows(ctx, tokens, offsets, kind: int, allowed: Sequence[int], eos: int = -1,
                   max_tokens: int = 1, prefix=None, row_prefix=None, flags: int = 0,
                   max_batch_tokens: int = 0, debug_logits: bool = False, vocab: int = 0,
                   limit: int = 0, limit_value: int = 1, row_mask=None, no_alloc: bool = False):
    """Returns a structured numpy array of lmop_result (value, logprob, logprob_full,
    n_tokens, tokens) and, with debug_logits, fp32 logits [n_rows][steps][vocab].
    For LMOP_AUTOMATON, `allowed` is an object with n_states, edge_offset,
    edge_token, edge_next and accepting arrays.  no_alloc calls
    lmop_eval_rows_noalloc (scratch in the library's static array) instead."""
    toks, offs, n, ty, opts, rp, keep = _call_args(tokens, offsets, kind, allowed, eos, max_tokens,
                                                   row_prefix, flags, max_batch_tokens, limit,
                                                   limit_value, row_mask)
    out = np.zeros(max(n, 0), dtype=RESULT_DTYPE)
    steps = max_tokens if kind in (LMOP_INT, LMOP_AUTOMATON) else 1
    dbg = None
    if debug_logits:
        if vocab <= 0:
            raise ValueError("debug_logits needs vocab")
        dbg = np.empty((n, steps, vocab), dtype=np.float32)
        opts.debug_logits = _ptr(dbg, C.c_float)
    fn = _lib.lmop_eval_rows_noalloc if no_alloc else _lib.lmop_eval_rows
    _check(fn(ctx, prefix, rp, _ptr(toks, C.c_int32), _ptr(offs, C.c_int64), n, C.byref(ty),
              out.ctypes.data, C.byref(opts)), ctx)
    del keep
    return out, dbg


def lmop_plan_rows(ctx, tokens, offsets, kind: int, allowed: Sequence[int], eos: int = -1,
                   max_tokens: int = 1, prefix=None, row_prefix=None, flags: int = 0,
                   max_batch_tokens: int = 0, limit: int = 0, limit_value: int = 1,
                   row_mask=None, debug_logits: bool = False) -> dict:
    """lmop_plan_rows: the plan lmop_eval_rows would use for these arguments
    (a dict of lmop_eval_plan's fields); runs nothing on the device.
    debug_logits plans the logit dump's scratch (the library writes nothing)."""
    toks, offs, n, ty, opts, rp, keep = _call_args(tokens, offsets, kind, allowed, eos, max_tokens,
                                                   row_prefix, flags, max_batch_tokens, limit,
                                                   limit_value, row_mask)
    if debug_logits:
        dummy = np.zeros(1, dtype=np.float32)
        keep.append(dummy)
        opts.debug_logits = _ptr(dummy, C.c_float)
    pl = lmop_eval_plan()
    _check(_lib.lmop_plan_rows(ctx, prefix, rp, _ptr(toks, C.c_int32), _ptr(offs, C.c_int64), n,
                               C.byref(ty), C.byref(opts), C.byref(pl)), ctx)
    del keep
    return {k: int(getattr(pl, k)) for k, _ in lmop_eval_plan._fields_ if k != "pad_"}


def _call_args(tokens, offsets, kind, allowed, eos, max_tokens, row_prefix, flags,
               max_batch_tokens, limit, limit_value, row_mask):
    """The marshalled arguments shared by lmop_eval_rows and lmop_plan_rows:
    token and offset arrays, row count, lmop_type, lmop_eval_opts, the row
    prefix array, and the arrays those structs point into (kept alive by the
    caller until the call returns)."""
    toks = _i32(tokens)
    offs = _i64(offsets)
    n = len(offs) - 1
    keep = []
    if kind == LMOP_AUTOMATON:
        eo, et, en = _i32(allowed.edge_offset), _i32(allowed.edge_token), _i32(allowed.edge_next)
        ac = np.ascontiguousarray(np.asarray(allowed.accepting, dtype=np.uint8))
        keep = [eo, et, en, ac]
        aut = lmop_automaton(int(allowed.n_states), _ptr(eo, C.c_int32), _ptr(et, C.c_int32),
                             _ptr(en, C.c_int32), _ptr(ac, C.c_uint8))
        ty = lmop_type(kind, None, 0, int(eos), int(max_tokens), C.pointer(aut))
    else:
        al = _i32(allowed)
        keep = [al]
        ty = lmop_type(kind, _ptr(al, C.c_int32), len(al), int(eos), int(max_tokens), None)
    keep.append(ty)
    opts = lmop_eval_opts(flags, max_batch_tokens, None, int(limit), int(limit_value), None)
    if row_mask is not None:
        mk = np.ascontiguousarray(np.asarray(row_mask, dtype=bool).astype(np.uint8))
        if len(mk) != n:
            raise ValueError("row_mask needs one entry per row")
        keep.append(mk)
        opts.row_mask = _ptr(mk, C.c_uint8)
    rp = None
    if row_prefix is not None:
        rp = (C.c_void_p * max(n, 1))(*[r.value if isinstance(r, C.c_void_p) else r
                                        for r in row_prefix])
    return toks, offs, n, ty, opts, rp, keep


def lmop_dedup_rows(tokens, offsets, keys=None):
    toks = _i32(tokens)
    offs = _i64(offsets)
    n = len(offs) - 1
    rep = np.zeros(max(n, 0), dtype=np.int32)
    nu = C.c_int32()
    kp = None
    if keys is not None:
        k = _i64(keys)
        kp = _ptr(k, C.c_int64)
    st = _lib.lmop_dedup_rows(_ptr(toks, C.c_int32), _ptr(offs, C.c_int64), n, kp,
                              _ptr(rep, C.c_int32), C.byref(nu))
    if st != LMOP_OK:
        raise LmopError(st, "invalid CSR arguments")
    return rep, int(nu.value)


def lmop_eval_rows_noalloc(ctx, tokens, offsets, kind: int, allowed, **kw):
    """lmop_eval_rows_noalloc: lmop_eval_rows with no device allocation."""
    return lmop_eval_rows(ctx, tokens, offsets, kind, allowed, no_alloc=True, **kw)


def lmop_set_workspace(ctx, ptr: int, nbytes: int) -> None:
    """Scratch carved from the caller's device memory [ptr, ptr + nbytes)
    (e.g. a torch tensor's data_ptr()); (0, 0) returns to library scratch."""
    _check(_lib.lmop_set_workspace(ctx, C.c_void_p(ptr or None), C.c_size_t(nbytes)), ctx)


def lmop_get_memory(ctx) -> dict:
    m = lmop_memory_stats()
    _check(_lib.lmop_get_memory(ctx, C.byref(m)), ctx)
    return {k: int(getattr(m, k)) for k, _ in lmop_memory_stats._fields_}


def lmop_set_profiling(ctx, period) -> None:
    """period: False/0 off, True/1 time every launch, N time every N-th launch
    of each kernel."""
    _check(_lib.lmop_set_profiling(ctx, int(period)), ctx)


def lmop_get_kernel_stats(ctx):
    n = C.c_int32()
    _check(_lib.lmop_get_kernel_stats(ctx, None, 0, C.byref(n)), ctx)
    arr = (lmop_kernel_stat * max(n.value, 1))()
    _check(_lib.lmop_get_kernel_stats(ctx, arr, n.value, C.byref(n)), ctx)
    return {arr[i].name.decode(): dict(launches=arr[i].launches, timed=arr[i].timed_launches,
                                       ms=arr[i].total_ms, flops=arr[i].flops, bytes=arr[i].bytes)
            for i in range(n.value)}


# ---------------------------------------------------------------- convenience
def config_from_shape(shape, max_seq: int = 0) -> lmop_config:
    return lmop_config(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                       shape.head_dim, shape.d_ff, shape.vocab, shape.group_size,
                       shape.rms_eps, shape.rope_theta, max_seq)


class Context:
    """One lmop ctx on a HIP device (device=-1: host-only, validation only)."""

    def __init__(self, shape, device: int = 0, stream: Optional[int] = None, max_seq: int = 0,
                 n_layers: Optional[int] = None):
        cfg = config_from_shape(shape, max_seq)
        if n_layers is not None:
            cfg.n_layers = n_layers
        self.vocab = shape.vocab
        self.ctx = lmop_create(cfg, device, stream)

    def close(self):
        if self.ctx:
            lmop_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load_weights(self, weights):
        lmop_load_weights(self.ctx, weights)

    def set_prefix(self, tokens, parent=None):
        return lmop_set_prefix(self.ctx, tokens, parent)

    def set_prefixes(self, token_lists, parent=None):
        return lmop_set_prefixes(self.ctx, token_lists, parent)

    def release_prefix(self, p):
        lmop_release_prefix(self.ctx, p)

    def eval_rows(self, tokens, offsets, kind, allowed, eos=-1, max_tokens=1, prefix=None,
                  row_prefix=None, no_dedup=False, max_batch_tokens=0, debug_logits=False,
                  head_restricted=False, limit=0, limit_value=1, row_mask=None, no_alloc=False):
        flags = (LMOP_NO_DEDUP if no_dedup else 0) | (LMOP_HEAD_RESTRICTED if head_restricted else 0)
        return lmop_eval_rows(self.ctx, tokens, offsets, kind, allowed, eos, max_tokens, prefix,
                              row_prefix, flags, max_batch_tokens, debug_logits, self.vocab,
                              limit, limit_value, row_mask, no_alloc)

    def plan_rows(self, tokens, offsets, kind, allowed, eos=-1, max_tokens=1, prefix=None,
                  row_prefix=None, no_dedup=False, max_batch_tokens=0, head_restricted=False,
                  limit=0, limit_value=1, row_mask=None, debug_logits=False) -> dict:
        flags = (LMOP_NO_DEDUP if no_dedup else 0) | (LMOP_HEAD_RESTRICTED if head_restricted else 0)
        return lmop_plan_rows(self.ctx, tokens, offsets, kind, allowed, eos, max_tokens, prefix,
                              row_prefix, flags, max_batch_tokens, limit, limit_value, row_mask,
                              debug_logits)

    def set_workspace(self, ptr: int, nbytes: int):
        lmop_set_workspace(self.ctx, ptr, nbytes)

    def memory(self) -> dict:
        return lmop_get_memory(self.ctx)

    def set_profiling(self, period):
        lmop_set_profiling(self.ctx, period)

    def kernel_stats(self):
        return lmop_get_kernel_stats(self.ctx)
