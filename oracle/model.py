"""The decoder-only transformer f of the paper's Preliminaries, in plain NumPy.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``): never imported by the HIP path.

f maps tokens to next-token logits (Preliminaries, Eq. 1): H^0 = W_in X, each layer maps
H^{i-1} -> H^i while caching keys/values, and the last hidden state is projected with W_out.
The paper fixes the model family (Qwen3-Base shapes, Appendix E) but not the layer internals; the
readings used here are:

* pre-norm blocks: h += Attn(RMSNorm(h)); h += MLP(RMSNorm(h)); a final RMSNorm before the head.
* RMSNorm(x) = x / sqrt(mean(x^2) + eps) * g.
* rotary position embedding, "rotate-half" pairing (i, i + d/2), theta_i = base^(-2i/d),
  absolute positions; angles are formed in float64.
* grouped-query attention: query head j uses KV head j // (n_heads / n_kv_heads); scores are
  q.k / sqrt(d); row r attends to every position <= its own.
* SwiGLU MLP: down(silu(gate(x)) * up(x)); no biases anywhere.
* tied embedding: W_out = W_in (Appendix E).
* storage precision: the paper does not state the inference precision. A bf16 model stores its
  weights and its KV cache in bfloat16, so each key/value is rounded to bf16 (round to nearest
  even) as it is produced, before any attention reads it. All arithmetic (norms, products,
  softmax, residual stream, logits) runs in ``dtype``: float32 by default, float64 for the pins
  that need it.
"""
from __future__ import annotations

import numpy as np


def round_to_bf16(x):
    """Round to the nearest bfloat16 (ties to even) and return the value in x's dtype."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.asarray(x).dtype)


def rmsnorm(x, g, eps):
    """RMSNorm over the last axis followed by the per-feature gain g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def silu(x):
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def rope_cos_sin(positions, head_dim, base):
    """cos/sin tables [n, head_dim/2] for the given absolute positions (float64)."""
    half = head_dim // 2
    inv_freq = float(base) ** (-(np.arange(half, dtype=np.float64) * 2.0) / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x, cos, sin):
    """Rotate x [n, heads, head_dim]: pair (i, i + d/2) is rotated by angle pos * theta_i."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c = cos[:, None, :].astype(x.dtype)
    s = sin[:, None, :].astype(x.dtype)
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q, K, V, q_pos):
    """Causal grouped-query attention.

    q [R, n_heads, d] are the queries of rows at absolute positions q_pos [R];
    K, V [L, n_kv, d] hold the keys/values of absolute positions 0..L-1.
    Row r attends to positions 0..q_pos[r]. Returns [R, n_heads, d].
    """
    R, nh, d = q.shape
    L, nkv, _ = K.shape
    rep = nh // nkv
    # query head j = kv * rep + g uses KV head kv: group the query heads by KV head and let the
    # matrix products broadcast over the group (no copy of K/V per query head)
    qg = q.reshape(R, nkv, rep, d).transpose(1, 2, 0, 3)               # [nkv, rep, R, d]
    Kt = K.transpose(1, 2, 0)[:, None]                                   # [nkv, 1, d, L]
    Vt = V.transpose(1, 0, 2)[:, None]                                   # [nkv, 1, L, d]
    s = np.matmul(qg, Kt) / np.sqrt(d).astype(q.dtype)                   # [nkv, rep, R, L]
    allowed = np.arange(L)[None, :] <= np.asarray(q_pos)[:, None]      # [R, L]
    s = np.where(allowed, s, -np.inf)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    o = np.matmul(p, Vt)                                                 # [nkv, rep, R, d]
    return o.transpose(2, 0, 1, 3).reshape(R, nh, d)                     # [R, nh, d]


class Model:
    """Weights of f plus the per-layer block, embedding and head."""

    def __init__(self, cfg, weights, dtype=np.float32, kv_bf16=None):
        self.cfg = cfg
        self.dtype = np.dtype(dtype)
        self.kv_bf16 = (getattr(cfg, "dtype", "f32") == "bf16") if kv_bf16 is None else kv_bf16
        self.w = {k: np.asarray(v, dtype=self.dtype) for k, v in weights.items()}

    @property
    def n_layers(self):
        return self.cfg.n_layers

    @property
    def first_decoder_layer(self):
        """l' : layers [0, l') are the encoder, [l', l) the decoder (Sec. 3.1, Eq. 3-4)."""
        return self.cfg.n_layers - self.cfg.n_dec_layers

    def embed(self, tokens):
        """H^0 = W_in X (Preliminaries)."""
        return self.w["embed"][np.asarray(tokens, dtype=np.int64)].copy()

    def head(self, h):
        """Logits H^l W_out^T with the final RMSNorm; W_out is tied to W_in (Appendix E)."""
        c = self.cfg
        return rmsnorm(h, self.w["final_norm"], c.rms_eps) @ self.w["embed"].T

    def kv(self, i, h, pos):
        """Keys and values [n, n_kv, d] that layer f_i produces for rows h [n, H] at absolute
        positions ``pos``: RMSNorm, the key/value projections, rotary embedding of the keys, and
        the cache's storage rounding. They depend on the row alone, not on the context."""
        c = self.cfg
        W = self.w
        p = f"layers.{i}."
        n = h.shape[0]
        a = rmsnorm(h, W[p + "attn_norm"], c.rms_eps)
        k = (a @ W[p + "wk"].T).reshape(n, c.n_kv_heads, c.head_dim)
        v = (a @ W[p + "wv"].T).reshape(n, c.n_kv_heads, c.head_dim)
        cos, sin = rope_cos_sin(np.asarray(pos, dtype=np.int64), c.head_dim, c.rope_base)
        k = apply_rope(k, cos, sin)
        if self.kv_bf16:
            k, v = round_to_bf16(k), round_to_bf16(v)
        return k, v

    def block(self, i, h, pos, K_prefix, V_prefix):
        """Layer f_i on rows h [n, H] at consecutive absolute positions ``pos``.

        K_prefix/V_prefix [pos[0], n_kv, d] are the keys/values this layer holds for the
        positions before pos[0]. Returns (new h, keys [n, n_kv, d], values [n, n_kv, d]) where
        the keys/values are those of the n new rows.
        """
        c = self.cfg
        W = self.w
        p = f"layers.{i}."
        n = h.shape[0]
        pos = np.asarray(pos, dtype=np.int64)
        assert K_prefix.shape[0] == pos[0] and np.all(np.diff(pos) == 1)
        a = rmsnorm(h, W[p + "attn_norm"], c.rms_eps)
        q = (a @ W[p + "wq"].T).reshape(n, c.n_heads, c.head_dim)
        k = (a @ W[p + "wk"].T).reshape(n, c.n_kv_heads, c.head_dim)
        v = (a @ W[p + "wv"].T).reshape(n, c.n_kv_heads, c.head_dim)
        cos, sin = rope_cos_sin(pos, c.head_dim, c.rope_base)
        q = apply_rope(q, cos, sin)
        k = apply_rope(k, cos, sin)
        if self.kv_bf16:
            k, v = round_to_bf16(k), round_to_bf16(v)
        K = np.concatenate([K_prefix, k], axis=0)
        V = np.concatenate([V_prefix, v], axis=0)
        o = attention(q, K, V, pos)
        h = h + o.reshape(n, c.n_heads * c.head_dim) @ W[p + "wo"].T
        m = rmsnorm(h, W[p + "mlp_norm"], c.rms_eps)
        h = h + (silu(m @ W[p + "w_gate"].T) * (m @ W[p + "w_up"].T)) @ W[p + "w_down"].T
        return h, k, v


class KVCache:
    """Per-layer key/value cache KV^i with an explicit valid length per layer.

    Positions [0, valid[i]) of layer i hold keys/values; writes must append at valid[i]
    (so every truncation of Algorithm 2 is explicit and checked).
    """

    def __init__(self, cfg, capacity, dtype=np.float32):
        shape = (cfg.n_layers, capacity, cfg.n_kv_heads, cfg.head_dim)
        self.K = np.zeros(shape, dtype=dtype)
        self.V = np.zeros(shape, dtype=dtype)
        self.valid = np.zeros(cfg.n_layers, dtype=np.int64)

    def prefix(self, i, n):
        """Keys/values of layer i for positions [0, n); they must all be valid."""
        assert n <= self.valid[i], (i, n, self.valid[i])
        return self.K[i, :n], self.V[i, :n]

    def append(self, i, pos0, k, v):
        """Store keys/values for positions pos0 .. pos0+len(k)-1 of layer i."""
        assert pos0 == self.valid[i], (i, pos0, self.valid[i])
        self.K[i, pos0:pos0 + len(k)] = k
        self.V[i, pos0:pos0 + len(v)] = v
        self.valid[i] = pos0 + len(k)

    def truncate(self, n):
        """Truncate(KV, n) of Algorithm 2: keep positions [0, n) in every layer."""
        self.valid = np.minimum(self.valid, n)


def run_layers(model, cache, layers, h, pos0):
    """Run layers ``layers`` on rows h at positions pos0.., reading/extending ``cache``."""
    n = h.shape[0]
    pos = np.arange(pos0, pos0 + n)
    for i in layers:
        Kp, Vp = cache.prefix(i, pos0)
        h, k, v = model.block(i, h, pos, Kp, Vp)
        cache.append(i, pos0, k, v)
    return h


def full_forward(model, tokens, return_kv=False, row_block=256):
    """f over a whole sequence with no cache: logits for every position [n, V].

    Rows are processed in blocks of ``row_block`` only to bound memory; each row still attends
    to exactly positions 0..its own. With ``return_kv`` also returns per-layer K, V [l, n, n_kv, d].
    """
    c = model.cfg
    tokens = np.asarray(tokens, dtype=np.int64)
    n = len(tokens)
    Ks = np.zeros((c.n_layers, n, c.n_kv_heads, c.head_dim), dtype=model.dtype)
    Vs = np.zeros_like(Ks)
    logits = np.zeros((n, c.vocab), dtype=model.dtype)
    for s in range(0, n, row_block):
        e = min(n, s + row_block)
        h = model.embed(tokens[s:e])
        for i in range(c.n_layers):
            h, k, v = model.block(i, h, np.arange(s, e), Ks[i, :s], Vs[i, :s])
            Ks[i, s:e] = k
            Vs[i, s:e] = v
        logits[s:e] = model.head(h)
    if return_kv:
        return logits, Ks, Vs
    return logits


def sampled_kv_first_layers(model, tokens, positions):
    """Keys/values of layers 0 and 1 at a few positions of one sequence, one position at a time.

    Layer 0's keys/values depend on each token alone, so they are formed for every position of
    the prefix; layer 1's at position j need layer 0's output at j, i.e. one row of layer 0
    attending to positions 0..j. This reaches long prefixes (16k tokens) that a full forward
    pass could not. Returns four arrays [len(positions), n_kv, d]: K0, V0, K1, V1.
    """
    positions = [int(j) for j in positions]
    tokens = np.asarray(tokens, dtype=np.int64)
    n = max(positions) + 1
    h0 = model.embed(tokens[:n])
    K0, V0 = model.kv(0, h0, np.arange(n))
    out = [[], [], [], []]
    for j in positions:
        h1, _, _ = model.block(0, h0[j:j + 1], [j], K0[:j], V0[:j])
        k1, v1 = model.kv(1, h1, [j])
        for lst, x in zip(out, (K0[j], V0[j], k1[0], v1[0])):
            lst.append(x)
    return tuple(np.stack(x) for x in out)
