"""Seeded synthetic inputs for the SEED decode path: model configs, random-init weights, prompts.

This module holds no arithmetic of the method. It only draws inputs (weights, prompt tokens,
prompt lengths) from fixed seeds so that the HIP path, the CPU oracle and the benchmark all see
identical values. It imports nothing from the rest of the package.

Shapes follow the decoder-only transformer of the paper's Preliminaries (per-layer attention +
SwiGLU MLP, tied input/output embedding) with the model sizes of Appendix E (the 28-layer
1.7B-scale shape and the 36-layer 4B-scale shape).

Weights: every linear/embedding tensor is N(0, 0.02), norm gains are 1.0. Tensor ``i`` (in the
order of :func:`tensor_specs`) is drawn in chunks of 2**24 elements, chunk ``c`` from
``numpy.random.default_rng([seed, i, c])``, so tensors can be drawn in parallel threads and any
tensor can be regenerated alone. For bf16 models the float32 draw is rounded to bf16 with
round-to-nearest-even; the oracle receives those same values widened back to float32.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F32 = "f32"
BF16 = "bf16"

_CHUNK = 1 << 24


@dataclasses.dataclass(frozen=True)
class Config:
    """Model shape plus the decode workload it is measured on."""

    name: str
    n_layers: int          # l
    n_dec_layers: int      # l - l'  (the decoder = last layers)
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_base: float
    rms_eps: float = 1e-6
    dtype: str = BF16
    # workload
    prompt_len: int = 32
    gen_len: int = 64
    k: int = 4
    batch: int = 1
    prompt_len_range: tuple | None = None   # (lo, hi) inclusive, per-sequence lengths

    @property
    def n_enc_layers(self) -> int:
        return self.n_layers - self.n_dec_layers

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# Tiny parity model: 4 layers = 2 encoder + 2 decoder, fp32.
C1_TINY = Config("tiny-4L-h256", 4, 2, 256, 4, 4, 64, 1024, 1024, 1e4, dtype=F32,
                 prompt_len=32, gen_len=64, k=4, batch=1)
# 28-layer 1.7B-scale shape (Appendix E), 26 encoder + 2 decoder, bf16.
C2_28L = Config("28L-h2048", 28, 2, 2048, 16, 8, 128, 6144, 151936, 1e6, dtype=BF16,
                prompt_len=512, gen_len=256, k=4, batch=1)
# 36-layer 4B-scale shape (Appendix E), 34 encoder + 2 decoder, bf16.
C3_4B = Config("4B-36L-h2560", 36, 2, 2560, 32, 8, 128, 9728, 151936, 1e6, dtype=BF16,
               prompt_len=1024, gen_len=512, k=4, batch=1)
# Same 4B shape, batch 8 with ragged prompt lengths in [256, 2048].
C4_4B_B8 = C3_4B.replace(name="4B-36L-h2560-b8", batch=8, prompt_len_range=(256, 2048))
# Same 4B shape, long context.
C5_4B_LONG = C3_4B.replace(name="4B-36L-h2560-16k", prompt_len=16384, gen_len=1024)

CONFIGS = {c.name: c for c in (C1_TINY, C2_28L, C3_4B, C4_4B_B8, C5_4B_LONG)}


def tensor_specs(cfg: Config):
    """Ordered list of (name, shape, kind) with kind in {"normal", "ones"}.

    Linear weights use the [out_features, in_features] layout. ``embed`` is the tied
    embedding / LM-head matrix [vocab, hidden].
    """
    H, F = cfg.hidden, cfg.ffn
    specs = [("embed", (cfg.vocab, H), "normal")]
    for i in range(cfg.n_layers):
        p = f"layers.{i}."
        specs += [
            (p + "attn_norm", (H,), "ones"),
            (p + "wq", (cfg.q_dim, H), "normal"),
            (p + "wk", (cfg.kv_dim, H), "normal"),
            (p + "wv", (cfg.kv_dim, H), "normal"),
            (p + "wo", (H, cfg.q_dim), "normal"),
            (p + "mlp_norm", (H,), "ones"),
            (p + "w_gate", (F, H), "normal"),
            (p + "w_up", (F, H), "normal"),
            (p + "w_down", (H, F), "normal"),
        ]
    specs.append(("final_norm", (H,), "ones"))
    return specs


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even), returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to float32 exactly."""
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _round_chunk_to_bf16(v: np.ndarray, out16: np.ndarray) -> None:
    """RNE-round float32 ``v`` to bf16 bits into ``out16`` (same length), in place on ``v``."""
    u = v.view(np.uint32)
    b = u >> np.uint32(16)
    b &= np.uint32(1)
    b += np.uint32(0x7FFF)
    b += u
    b >>= np.uint32(16)
    out16[:] = b


def make_weights(cfg: Config, seed: int = 0, std: float = 0.02, enc_out_scale: float = 1.0):
    """Random-init weights for ``cfg``.

    Returns ``dict name -> ndarray``. For bf16 configs the arrays are uint16 bf16 bit patterns;
    for fp32 configs they are float32. Use :func:`weights_as_f32` to get float32 views for the
    oracle.

    ``enc_out_scale`` multiplies the standard deviation of the encoder layers' output
    projections (``wo``, ``w_down`` of layers < l'). Values below 1 shrink what the encoder adds
    to the residual stream, which makes the drafter agree with the verifier more often; tests use
    it to exercise partial and full acceptance with random weights.
    """
    as_bf16 = cfg.dtype == BF16
    n_enc = cfg.n_layers - cfg.n_dec_layers
    out = {}
    jobs = []
    for idx, (name, shape, kind) in enumerate(tensor_specs(cfg)):
        n = int(np.prod(shape))
        if kind == "ones":
            a = np.ones(n, dtype=np.float32)
            out[name] = (f32_to_bf16_bits(a) if as_bf16 else a).reshape(shape)
            continue
        s = std
        if name.startswith("layers.") and name.endswith((".wo", ".w_down")):
            if int(name.split(".")[1]) < n_enc:
                s = std * enc_out_scale
        flat = np.empty(n, dtype=np.uint16 if as_bf16 else np.float32)
        out[name] = flat.reshape(shape)
        jobs += [(idx, c, flat, s) for c in range((n + _CHUNK - 1) // _CHUNK)]

    def fill(job):
        idx, c, flat, s = job
        lo = c * _CHUNK
        hi = min(len(flat), lo + _CHUNK)
        v = np.random.default_rng([seed, idx, c]).standard_normal(hi - lo, dtype=np.float32)
        v *= np.float32(s)
        if as_bf16:
            _round_chunk_to_bf16(v, flat[lo:hi])
        else:
            flat[lo:hi] = v

    with ThreadPoolExecutor(_threads()) as pool:
        list(pool.map(fill, jobs))
    return out


def weights_as_f32(cfg: Config, weights: dict) -> dict:
    """float32 copies of ``weights`` (bf16 bit patterns widened exactly)."""
    if cfg.dtype != BF16:
        return {k: np.asarray(v, dtype=np.float32) for k, v in weights.items()}
    out = {}
    jobs = []
    for k, v in weights.items():
        src = v.reshape(-1)
        dst = np.empty(src.shape, dtype=np.uint32)
        out[k] = dst.view(np.float32).reshape(v.shape)
        jobs += [(src, dst, c) for c in range((len(src) + _CHUNK - 1) // _CHUNK)]

    def widen(job):
        src, dst, c = job
        lo = c * _CHUNK
        hi = min(len(src), lo + _CHUNK)
        d = dst[lo:hi]
        d[:] = src[lo:hi]
        d <<= np.uint32(16)

    with ThreadPoolExecutor(_threads()) as pool:
        list(pool.map(widen, jobs))
    return out


def make_prompt_lengths(cfg: Config, seed: int = 2) -> list:
    """Per-sequence prompt lengths: fixed ``prompt_len`` or uniform in ``prompt_len_range``."""
    if cfg.prompt_len_range is None:
        return [cfg.prompt_len] * cfg.batch
    lo, hi = cfg.prompt_len_range
    g = np.random.default_rng(seed)
    return [int(x) for x in g.integers(lo, hi + 1, size=cfg.batch)]


def make_prompts(cfg: Config, seed: int = 1, lengths=None) -> list:
    """Uniform-random token prompts (one int32 array per sequence), i.i.d. over [0, vocab)."""
    if lengths is None:
        lengths = make_prompt_lengths(cfg)
    g = np.random.default_rng(seed)
    return [g.integers(0, cfg.vocab, size=n, dtype=np.int64).astype(np.int32) for n in lengths]
