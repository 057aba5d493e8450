"""Thin Python binding of the SEED C ABI (include/seed.h).

Each ``seed_*`` function here marshals arguments for the C function of the same name; all work
runs in the HIP library. PyTorch supplies only device memory (the weight arena, KV pool and
workspace) and the HIP stream. If the built library is missing, loading fails loudly: there is
no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16 = 0, 1

PHASE_VERIFY, PHASE_DRAFT, PHASE_PREFILL = 0, 1, 2
OP_SETUP, OP_QKV, OP_ATTN, OP_COMBINE, OP_O, OP_GATEUP, OP_DOWN, OP_HEAD, OP_ACCEPT, OP_HEAD_ARGMAX, OP_TOPK = range(11)


def kernel_id(phase: int, op: int) -> int:
    return phase * 16 + op


class SeedError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        super().__init__(f"{func} failed ({status}): {msg}")
        self.status = status


class SeedConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "n_dec_layers", "hidden", "n_heads", "n_kv_heads", "head_dim", "ffn", "vocab")] + [
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float)] + [
        (n, ctypes.c_int32) for n in ("dtype", "max_batch", "max_ctx", "max_draft", "kv_block")]


class SeedTensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("data", ctypes.c_void_p), ("dtype", ctypes.c_int32),
                ("on_device", ctypes.c_int32), ("ndim", ctypes.c_int32), ("shape", ctypes.c_int64 * 2)]


class SeedGenOpts(ctypes.Structure):
    _fields_ = [("k", ctypes.c_int32), ("max_new", ctypes.c_int32), ("eos_id", ctypes.c_int32),
                ("sim_accept", ctypes.c_int32), ("forced_trace", ctypes.POINTER(ctypes.c_int32)),
                ("use_graph", ctypes.c_int32)]


class SeedTreeOpts(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("max_depth", ctypes.c_int32), ("n_levels", ctypes.c_int32),
                ("thr", ctypes.c_float * 4), ("k", ctypes.c_int32 * 4), ("k_rest", ctypes.c_int32),
                ("max_nodes", ctypes.c_int32)]


def tree_opts(max_depth: int, tau: float | None = None, table=None, rest: int | None = None,
              max_nodes: int | None = None) -> SeedTreeOpts:
    """The paper's dynamic-drafting options (seed_tree_defaults), with optional overrides; table is
    a sequence of (threshold, fan-out) pairs."""
    o = SeedTreeOpts()
    load_library().seed_tree_defaults(ctypes.byref(o), max_depth)
    if tau is not None:
        o.tau = tau
    if table is not None:
        o.n_levels = len(table)
        for j, (thr, k) in enumerate(table):
            o.thr[j], o.k[j] = thr, k
    if rest is not None:
        o.k_rest = rest
    if max_nodes is not None:
        o.max_nodes = max_nodes
    return o


class SeedStats(ctypes.Structure):
    _fields_ = [("rounds", ctypes.c_int64), ("drafted", ctypes.c_int64), ("accepted", ctypes.c_int64),
                ("prefill_ms", ctypes.c_double), ("decode_ms", ctypes.c_double),
                ("n_accept_log", ctypes.POINTER(ctypes.c_int32)), ("n_accept_log_cap", ctypes.c_int64),
                ("verify_ms", ctypes.c_double), ("draft_ms", ctypes.c_double)]


EXPORTS = ("seed_arena_bytes", "seed_create", "seed_load_weights", "seed_prefill", "seed_draft",
           "seed_verify", "seed_rounds", "seed_generate", "seed_get_tokens", "seed_read_kv", "seed_kernel_timing",
           "seed_kernel_timing_read", "seed_last_error", "seed_destroy", "seed_spec_kv_bytes",
           "seed_spec_forward", "seed_spec_forward_noalloc", "seed_verify_tree", "seed_tree_defaults",
           "seed_draft_tree", "seed_generate_tree")

_LIB = None
_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)


def lib_path() -> str:
    return _build.LIB


def load_library(path: str | None = None):
    """Load the built HIP library (``build()`` first). Raises if it is missing."""
    global _LIB
    if _LIB is not None and path is None:
        return _LIB
    path = path or lib_path()
    if not os.path.exists(path):
        raise FileNotFoundError(f"SEED HIP library not built: {path} (run __graft_entry__.build())")
    # torch ships its own HIP runtime; load it first so the library binds to that same runtime
    # (two HIP runtimes in one process do not share devices, streams or allocations)
    import torch  # noqa: F401

    lib = ctypes.CDLL(path)
    sig = {
        "seed_arena_bytes": [ctypes.POINTER(SeedConfig), ctypes.POINTER(ctypes.c_size_t),
                             ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)],
        "seed_create": [ctypes.POINTER(SeedConfig), _P, _P, _P, _P, ctypes.POINTER(_P)],
        "seed_load_weights": [_P, ctypes.POINTER(SeedTensor), ctypes.c_int32],
        "seed_prefill": [_P, ctypes.c_int32, _I32P, _I32P],
        "seed_draft": [_P, ctypes.c_int32, _I32P, _P],
        "seed_verify": [_P, ctypes.c_int32, _I32P, _I32P, _I32P, _P],
        "seed_rounds": [_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32],
        "seed_generate": [_P, ctypes.c_int32, _I32P, _I32P, ctypes.POINTER(SeedGenOpts), _I32P, _I32P,
                          ctypes.POINTER(SeedStats)],
        "seed_get_tokens": [_P, ctypes.c_int32, _I32P, ctypes.c_int32, _I32P],
        "seed_read_kv": [_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, _P],
        "seed_kernel_timing": [_P, ctypes.c_int32, ctypes.c_int32],
        "seed_kernel_timing_read": [_P, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double)],
        "seed_spec_kv_bytes": [ctypes.POINTER(SeedConfig), ctypes.POINTER(ctypes.c_size_t)],
        "seed_verify_tree": [_P, ctypes.c_int32, _I32P, _I32P, _I32P, _I32P, _I32P, _P],
        "seed_tree_defaults": [ctypes.POINTER(SeedTreeOpts), ctypes.c_int32],
        "seed_draft_tree": [_P, ctypes.POINTER(SeedTreeOpts), _I32P, _I32P, _I32P, ctypes.POINTER(ctypes.c_float), _P],
        "seed_generate_tree": [_P, _I32P, ctypes.c_int32, ctypes.POINTER(SeedTreeOpts), ctypes.POINTER(SeedGenOpts),
                               _I32P, _I32P, ctypes.POINTER(SeedStats)],
        "seed_spec_forward": [_P, ctypes.c_int32, _I32P, ctypes.c_int32, _P, _P, _P, ctypes.POINTER(ctypes.c_double)],
        "seed_spec_forward_noalloc": [_P, ctypes.c_int32, _I32P, ctypes.c_int32, _P, _P, ctypes.POINTER(ctypes.c_double)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.seed_last_error.argtypes = []
    lib.seed_last_error.restype = ctypes.c_char_p
    lib.seed_destroy.argtypes = [_P]
    lib.seed_destroy.restype = None
    lib.seed_tree_defaults.restype = None
    if path == lib_path():
        _LIB = lib
    return lib


def _check(status: int, func: str):
    if status != 0:
        raise SeedError(status, func, load_library().seed_last_error().decode())


def _i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(_I32P)


def make_config(model, max_batch: int, max_ctx: int, max_draft: int) -> SeedConfig:
    """seed_config from a model description with the attributes of ``synth.Config``."""
    return SeedConfig(model.n_layers, model.n_dec_layers, model.hidden, model.n_heads, model.n_kv_heads,
                      model.head_dim, model.ffn, model.vocab, float(model.rope_base), float(model.rms_eps),
                      BF16 if model.dtype == "bf16" else F32, max_batch, max_ctx, max_draft, 16)


# ----------------------------------------------------------------------------------------------
# one function per C entry point
# ----------------------------------------------------------------------------------------------
def seed_arena_bytes(cfg: SeedConfig):
    w, kv, ws = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(load_library().seed_arena_bytes(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(kv), ctypes.byref(ws)),
           "seed_arena_bytes")
    return w.value, kv.value, ws.value


def seed_create(cfg: SeedConfig, stream: int, weight_arena: int, kv_pool: int, workspace: int) -> int:
    out = _P()
    _check(load_library().seed_create(ctypes.byref(cfg), stream, weight_arena, kv_pool, workspace, ctypes.byref(out)),
           "seed_create")
    return out.value


def seed_load_weights(ctx: int, tensors):
    """tensors: list of (name, data_ptr, dtype, on_device, shape)."""
    arr = (SeedTensor * len(tensors))()
    names = []
    for i, (name, ptr, dt, dev, shape) in enumerate(tensors):
        names.append(name.encode())
        arr[i].name = names[-1]
        arr[i].data = ptr
        arr[i].dtype = dt
        arr[i].on_device = int(dev)
        arr[i].ndim = len(shape)
        for j, s in enumerate(shape):
            arr[i].shape[j] = s
    _check(load_library().seed_load_weights(ctx, arr, len(tensors)), "seed_load_weights")


def seed_prefill(ctx: int, prompts):
    lens, lp = _i32([len(p) for p in prompts])
    toks, tp = _i32(np.concatenate([np.asarray(p) for p in prompts]))
    _check(load_library().seed_prefill(ctx, len(prompts), tp, lp), "seed_prefill")


def seed_draft(ctx: int, k: int, B: int, logits_ptr: int | None = None):
    out = np.zeros(B * k, dtype=np.int32)
    _check(load_library().seed_draft(ctx, k, out.ctypes.data_as(_I32P), logits_ptr), "seed_draft")
    return out.reshape(B, k)


def seed_verify(ctx: int, k: int, B: int, drafts=None, logits_ptr: int | None = None):
    na = np.zeros(B, dtype=np.int32)
    bo = np.zeros(B, dtype=np.int32)
    dp = None
    if drafts is not None:
        d, dp = _i32(np.asarray(drafts).reshape(-1))
    _check(load_library().seed_verify(ctx, k, dp, na.ctypes.data_as(_I32P), bo.ctypes.data_as(_I32P), logits_ptr),
           "seed_verify")
    return na, bo


def seed_rounds(ctx: int, k: int, n_rounds: int, use_graph: bool = False):
    _check(load_library().seed_rounds(ctx, k, n_rounds, int(use_graph)), "seed_rounds")


def seed_generate(ctx: int, prompts, k: int, max_new: int, eos_id: int = -1, sim_accept: int = -1,
                  forced_trace=None, use_graph: bool = False, log_cap: int = 0):
    B = len(prompts)
    lens, lp = _i32([len(p) for p in prompts])
    toks, tp = _i32(np.concatenate([np.asarray(p) for p in prompts]))
    opts = SeedGenOpts()
    opts.k, opts.max_new, opts.eos_id, opts.sim_accept, opts.use_graph = k, max_new, eos_id, sim_accept, int(use_graph)
    if forced_trace is not None:
        tr, trp = _i32(np.asarray(forced_trace).reshape(-1))
        opts.forced_trace = trp
    out = np.zeros(B * max_new, dtype=np.int32)
    counts = np.zeros(B, dtype=np.int32)
    stats = SeedStats()
    log = np.full(max(log_cap, 1) * B, -2, dtype=np.int32)
    if log_cap > 0:
        stats.n_accept_log = log.ctypes.data_as(_I32P)
        stats.n_accept_log_cap = log_cap
    _check(load_library().seed_generate(ctx, B, tp, lp, ctypes.byref(opts), out.ctypes.data_as(_I32P),
                                        counts.ctypes.data_as(_I32P), ctypes.byref(stats)), "seed_generate")
    st = {"rounds": stats.rounds, "drafted": stats.drafted, "accepted": stats.accepted,
          "prefill_ms": stats.prefill_ms, "decode_ms": stats.decode_ms, "verify_ms": stats.verify_ms,
          "draft_ms": stats.draft_ms}
    if log_cap > 0:
        st["n_accept_log"] = log.reshape(-1, B)[:min(stats.rounds, log_cap)]
    return out.reshape(B, max_new), counts, st


def seed_get_tokens(ctx: int, b: int, cap: int):
    out = np.zeros(cap, dtype=np.int32)
    n = ctypes.c_int32()
    _check(load_library().seed_get_tokens(ctx, b, out.ctypes.data_as(_I32P), cap, ctypes.byref(n)), "seed_get_tokens")
    return out[:min(cap, n.value)]


def seed_read_kv(cfg: SeedConfig, ctx: int, b: int, layer: int, pos0: int, n: int):
    """Cached keys and values of sequence b, layer ``layer``, positions pos0..pos0+n-1, as float32
    arrays [n, n_kv_heads, head_dim] (bf16 caches are widened exactly)."""
    shape = (n, cfg.n_kv_heads, cfg.head_dim)
    dt = np.uint16 if cfg.dtype == BF16 else np.float32
    k = np.zeros(shape, dtype=dt)
    v = np.zeros(shape, dtype=dt)
    _check(load_library().seed_read_kv(ctx, b, layer, pos0, n, k.ctypes.data_as(_P), v.ctypes.data_as(_P)),
           "seed_read_kv")
    if dt is np.uint16:
        return ((k.astype(np.uint32) << 16).view(np.float32), (v.astype(np.uint32) << 16).view(np.float32))
    return k, v


def seed_kernel_timing(ctx: int, kid: int, enable: bool):
    _check(load_library().seed_kernel_timing(ctx, kid, int(enable)), "seed_kernel_timing")


def seed_kernel_timing_read(ctx: int):
    n, ms = ctypes.c_int64(), ctypes.c_double()
    _check(load_library().seed_kernel_timing_read(ctx, ctypes.byref(n), ctypes.byref(ms)), "seed_kernel_timing_read")
    return n.value, ms.value


def seed_spec_kv_bytes(cfg: SeedConfig) -> int:
    n = ctypes.c_size_t()
    _check(load_library().seed_spec_kv_bytes(ctypes.byref(cfg), ctypes.byref(n)), "seed_spec_kv_bytes")
    return n.value


def seed_spec_forward(ctx: int, tokens, block: int, shallow_kv: int, logits: int, row_nll: int | None = None,
                      want_loss: bool = True):
    t, tp = _i32(tokens)
    loss = ctypes.c_double()
    _check(load_library().seed_spec_forward(ctx, len(t), tp, block, shallow_kv, logits, row_nll,
                                            ctypes.byref(loss) if want_loss else None), "seed_spec_forward")
    return loss.value if want_loss else None


def seed_spec_forward_noalloc(ctx: int, tokens, block: int, logits: int, row_nll: int | None = None,
                              want_loss: bool = True):
    """seed_spec_forward with the pass's own keys/values in the library's fixed scratch array."""
    t, tp = _i32(tokens)
    loss = ctypes.c_double()
    _check(load_library().seed_spec_forward_noalloc(ctx, len(t), tp, block, logits, row_nll,
                                                    ctypes.byref(loss) if want_loss else None),
           "seed_spec_forward_noalloc")
    return loss.value if want_loss else None


def seed_verify_tree(ctx: int, tokens, parents, logits_ptr: int | None = None):
    t, tp = _i32(tokens)
    pa, pp = _i32(parents)
    path = np.zeros(len(t), dtype=np.int32)
    n_path, bonus = ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().seed_verify_tree(ctx, len(t), tp, pp, path.ctypes.data_as(_I32P), ctypes.byref(n_path),
                                           ctypes.byref(bonus), logits_ptr), "seed_verify_tree")
    return [int(x) for x in path[:n_path.value]], bonus.value


def seed_draft_tree(ctx: int, opts: SeedTreeOpts, logits_ptr: int | None = None):
    toks = np.zeros(64, dtype=np.int32)
    par = np.zeros(64, dtype=np.int32)
    p0 = np.zeros(opts.max_depth, dtype=np.float32)
    n = ctypes.c_int32()
    _check(load_library().seed_draft_tree(ctx, ctypes.byref(opts), toks.ctypes.data_as(_I32P), par.ctypes.data_as(_I32P),
                                          ctypes.byref(n), p0.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                          logits_ptr), "seed_draft_tree")
    k = n.value
    depth = 0
    while depth + 1 < k and par[depth + 1] == depth:
        depth += 1
    return [int(x) for x in toks[:k]], [int(x) for x in par[:k]], p0[:depth]


def seed_generate_tree(ctx: int, prompt, opts: SeedTreeOpts, max_new: int, eos_id: int = -1,
                       use_graph: bool = False, log_cap: int = 0, sim_accept: int = -1, forced_trace=None):
    toks, tp = _i32(np.asarray(prompt))
    g = SeedGenOpts()
    g.k, g.max_new, g.eos_id, g.sim_accept, g.use_graph = 0, max_new, eos_id, sim_accept, int(use_graph)
    if forced_trace is not None:
        tr, trp = _i32(np.asarray(forced_trace).reshape(-1))
        g.forced_trace = trp
    out = np.zeros(max_new, dtype=np.int32)
    count = ctypes.c_int32()
    stats = SeedStats()
    log = np.full(max(log_cap, 1), -2, dtype=np.int32)
    if log_cap > 0:
        stats.n_accept_log = log.ctypes.data_as(_I32P)
        stats.n_accept_log_cap = log_cap
    _check(load_library().seed_generate_tree(ctx, tp, len(toks), ctypes.byref(opts), ctypes.byref(g),
                                             out.ctypes.data_as(_I32P), ctypes.byref(count), ctypes.byref(stats)),
           "seed_generate_tree")
    st = {"rounds": stats.rounds, "drafted": stats.drafted, "accepted": stats.accepted,
          "prefill_ms": stats.prefill_ms, "decode_ms": stats.decode_ms, "verify_ms": stats.verify_ms,
          "draft_ms": stats.draft_ms}
    if log_cap > 0:
        st["n_accept_log"] = log[:min(stats.rounds, log_cap)]
    return out[:count.value], st


def seed_destroy(ctx: int):
    load_library().seed_destroy(ctx)


# ----------------------------------------------------------------------------------------------
# convenience owner of the torch buffers
# ----------------------------------------------------------------------------------------------
class Decoder:
    """Owns the device buffers of one context and forwards to the seed_* calls."""

    def __init__(self, model, max_batch: int, max_ctx: int, max_draft: int, device: str = "cuda", stream=None):
        import torch

        self.torch = torch
        self.model = model
        self.cfg = make_config(model, max_batch, max_ctx, max_draft)
        wb, kvb, wsb = seed_arena_bytes(self.cfg)
        dev = torch.device(device)
        # a stream of our own (default priority): HIP graph capture cannot use the null stream
        self.stream = stream if stream is not None else torch.cuda.Stream(device=dev)
        self.weights = torch.empty(wb, dtype=torch.uint8, device=dev)
        self.kv = torch.empty(kvb, dtype=torch.uint8, device=dev)
        self.workspace = torch.empty(wsb, dtype=torch.uint8, device=dev)
        self.bytes = {"weights": wb, "kv": kvb, "workspace": wsb}
        self.ctx = seed_create(self.cfg, self.stream.cuda_stream, self.weights.data_ptr(), self.kv.data_ptr(),
                               self.workspace.data_ptr())
        self.B = 0

    def load_weights(self, weights: dict, on_device: bool = True):
        """weights: name -> ndarray (uint16 bf16 bit patterns or float32), uploaded one at a time."""
        torch = self.torch
        dt = self.cfg.dtype
        for name, arr in weights.items():
            a = np.ascontiguousarray(arr)
            if on_device:
                t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(self.weights.device)
                seed_load_weights(self.ctx, [(name, t.data_ptr(), dt, True, a.shape)])
                del t
            else:
                seed_load_weights(self.ctx, [(name, a.ctypes.data, dt, False, a.shape)])
        torch.cuda.synchronize(self.weights.device)

    def prefill(self, prompts):
        self.B = len(prompts)
        seed_prefill(self.ctx, prompts)

    def draft(self, k: int, logits: bool = False):
        lg = self._logits(self.B * k) if logits else None
        d = seed_draft(self.ctx, k, self.B, lg.data_ptr() if lg is not None else None)
        return d, (self._host(lg, (self.B, k)) if logits else None)

    def verify(self, k: int, drafts=None, logits: bool = False):
        lg = self._logits(self.B * (k + 1)) if logits else None
        na, bo = seed_verify(self.ctx, k, self.B, drafts, lg.data_ptr() if lg is not None else None)
        return na, bo, (self._host(lg, (self.B, k + 1)) if logits else None)

    def rounds(self, k: int, n: int, use_graph: bool = False):
        seed_rounds(self.ctx, k, n, use_graph)

    def generate(self, prompts, k: int, max_new: int, **kw):
        self.B = len(prompts)
        return seed_generate(self.ctx, prompts, k, max_new, **kw)

    def tokens(self, b: int):
        return seed_get_tokens(self.ctx, b, self.cfg.max_ctx)

    def read_kv(self, b: int, layer: int, pos0: int, n: int):
        """Keys, values [n, n_kv_heads, head_dim] (float32) cached for sequence b, layer ``layer``."""
        return seed_read_kv(self.cfg, self.ctx, b, layer, pos0, n)

    def draft_tree(self, opts: SeedTreeOpts, logits: bool = False):
        """One round's dynamic drafting: (tokens, parents, p0 per step, logits [steps, vocab] or None)."""
        lg = self._logits(opts.max_depth) if logits else None
        toks, par, p0 = seed_draft_tree(self.ctx, opts, lg.data_ptr() if lg is not None else None)
        return toks, par, p0, (self._host(lg, (opts.max_depth,))[:len(p0)] if logits else None)

    def generate_tree(self, prompt, opts: SeedTreeOpts, max_new: int, **kw):
        """Dynamic drafting with tree verification for one prompt: (tokens, stats)."""
        self.B = 1
        return seed_generate_tree(self.ctx, prompt, opts, max_new, **kw)

    def verify_tree(self, tokens, parents, logits: bool = False):
        """Tree-based verification of one packed draft tree: (accepted path nodes, bonus token,
        logits [n, vocab] or None)."""
        lg = self._logits(len(tokens)) if logits else None
        path, bonus = seed_verify_tree(self.ctx, tokens, parents, lg.data_ptr() if lg is not None else None)
        return path, bonus, (self._host(lg, (len(tokens),)) if logits else None)

    def spec_forward(self, tokens, block: int, logits: bool = True):
        """Forward pass of the speculative drafting objective on one sequence: (drafter logits
        [n-1, vocab] or None, per-row negative log-likelihoods [n-1], L_spec)."""
        torch = self.torch
        n = len(tokens)
        if getattr(self, "_skv", None) is None:
            self._skv = torch.empty(seed_spec_kv_bytes(self.cfg), dtype=torch.uint8, device=self.weights.device)
        lg = self._logits(max(n - 1, 1))
        nll = torch.empty(max(n - 1, 1), dtype=torch.float32, device=self.weights.device)
        loss = seed_spec_forward(self.ctx, tokens, block, self._skv.data_ptr(), lg.data_ptr(), nll.data_ptr())
        self.B = 1
        self.stream.synchronize()
        return (self._host(lg, (n - 1,)) if logits else None), nll.cpu().numpy()[:n - 1], loss

    def _logits(self, rows):
        return self.torch.empty(rows * self.cfg.vocab, dtype=self.torch.float32, device=self.weights.device)

    def _host(self, t, shape):
        self.stream.synchronize()
        return t.cpu().numpy().reshape(*shape, self.cfg.vocab)

    def close(self):
        if getattr(self, "ctx", None):
            seed_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
