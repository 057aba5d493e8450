"""Shared helpers of the GPU tests: decoder construction and oracle comparisons.

Inputs reach the oracle only from ``synth`` (seeded weights and prompts); the GPU path receives
the same inputs plus, where a test drives it step by step, tokens the oracle produced. Nothing
the GPU computes is fed back into the oracle.
"""
import sys

import numpy as np

from oracle import model as om
from oracle import seed as os_
from paper_2609_36590_amd import binding, synth


# rows one GPU pass verifies at most (seed_config: max_batch * (max_draft + 1) <= 64); a draft
# tree compared with the GPU's is built by the oracle under the same node budget
GPU_ROWS = 64


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def decoder(cfg, weights, max_batch=1, max_ctx=256, max_draft=6):
    say(f"[gpu] decoder {cfg.name} dtype={cfg.dtype} B<={max_batch} ctx={max_ctx} d<={max_draft}")
    dec = binding.Decoder(cfg, max_batch=max_batch, max_ctx=max_ctx, max_draft=max_draft)
    dec.load_weights(weights)
    return dec


def oracle_model(cfg, weights, dtype=np.float32):
    return om.Model(cfg, synth.weights_as_f32(cfg, weights), dtype)


def top2_gap(logits):
    s = np.sort(logits, axis=-1)
    return s[..., -1] - s[..., -2]


def first_ambiguous(rounds, tol):
    """Index of the first round whose verification has a row with a top-2 gap <= 2*tol."""
    for i, rd in enumerate(rounds):
        if np.any(top2_gap(rd.verify_logits) <= 2 * tol):
            return i
    return len(rounds)


def committed_before(prompt, toks, p):
    """X[0..p] of the oracle's decode (prompt followed by generated tokens)."""
    full = np.concatenate([np.asarray(prompt), np.asarray(toks)])
    return full[:p + 1]


def check_round(dec, prompt, toks, rd, tol, k):
    """Drive the GPU through one oracle round from the same committed prefix and compare every
    draft and verify logit row. Returns the max abs errors (draft, verify)."""
    ctx = committed_before(prompt, toks, rd.p)
    dec.prefill([ctx.astype(np.int32)])
    d, qlog = dec.draft(k, logits=True)
    derr = float(np.abs(qlog[0, 0] - rd.draft_logits[0]).max())
    for i in range(1, k):
        # later draft steps are comparable while the drafted tokens agree
        if not np.array_equal(d[0, :i], rd.drafts[1:i + 1]):
            break
        derr = max(derr, float(np.abs(qlog[0, i] - rd.draft_logits[i]).max()))
    for i in range(k):
        if top2_gap(rd.draft_logits[i]) > 2 * tol and np.array_equal(d[0, :i], rd.drafts[1:i + 1]):
            assert d[0, i] == rd.drafts[i + 1], (rd.p, i)
    na, bo, vlog = dec.verify(k, drafts=np.asarray(rd.drafts[1:], dtype=np.int32)[None], logits=True)
    verr = float(np.abs(vlog[0] - rd.verify_logits).max())
    if np.all(top2_gap(rd.verify_logits) > 2 * tol):
        assert na[0] == rd.n_accept and bo[0] == rd.bonus, (rd.p, na, rd.n_accept, bo, rd.bonus)
    return derr, verr


def bf16_ulp(x):
    """Spacing of bfloat16 values at |x| (8 significand bits): 2^(e - 8) for |x| = m 2^e."""
    _, e = np.frexp(np.abs(np.asarray(x, dtype=np.float64)))
    return np.ldexp(1.0, e - 8)


def compare_kv(got, ref, bf16, tol32=1e-4, what=""):
    """Cached keys/values of the GPU against the oracle's. A bf16 cache rounds both sides' fp32
    values to bfloat16, so an element may differ by one bf16 step where the unrounded values
    straddle a rounding boundary (plus 1e-3 for the rounding-order noise of values near zero);
    an fp32 cache is compared within tol32. Returns (max abs error, fraction exactly equal)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    d = np.abs(got - ref)
    if bf16:
        bound = bf16_ulp(np.maximum(np.abs(got), np.abs(ref))) + 1e-3
        worst = float((d - bound).max())
        assert worst <= 0, (what, worst, float(d.max()))
    else:
        assert float(d.max()) <= tol32, (what, float(d.max()))
    same = float(np.mean(d == 0))
    say(f"[gpu] {what}: max |kv - oracle| = {d.max():.3g}, {100 * same:.2f}% identical")
    return float(d.max()), same
