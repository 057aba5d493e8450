"""GPU parity of the forward pass of the speculative drafting objective (Algorithm 1, L_spec)
against the oracle's block-by-block loop.

Tiny models (fp32: logits within 1e-4; bf16 weights and caches: 2e-2), block sizes from 1 to
larger than the sequence; a 100-token sequence runs as one wide pass of 99 rows with a ragged last
token tile, and an 1100-token one makes blocks straddle the 1024-row passes of the GPU path (rows
of one block computed in two passes read each other's keys/values from the pass's own cache). Per-row negative log-likelihoods within the logit tolerance (+ rounding of the
log-sum-exp), L_spec within n times that. The decoder-only split (n_dec = l) must reproduce the
full model's causal logits for every block size.
"""
import numpy as np
import pytest

from gpu_common import decoder, oracle_model, say
from oracle import model as om
from oracle import seed as os_
from paper_2609_36590_amd import synth

pytestmark = pytest.mark.gpu

TINY_BF16 = synth.C1_TINY.replace(name="tiny-4L-h256-bf16", dtype=synth.BF16)


def _run(cfg, n, blocks, tol, seed=0):
    w = synth.make_weights(cfg, seed=seed)
    x = synth.make_prompts(cfg.replace(prompt_len=n), seed=seed + 7)[0]
    m = oracle_model(cfg, w)
    dec = decoder(cfg, w, max_batch=1, max_ctx=n + 8, max_draft=4)
    try:
        for b in blocks:
            say(f"[gpu] spec forward {cfg.name} n={n} block={b}")
            ref, ref_loss = os_.spec_forward(m, x, b)
            lg, nll, loss = dec.spec_forward(x, b)
            err = float(np.abs(lg - ref).max())
            z = ref.astype(np.float64)
            zm = z.max(axis=1, keepdims=True)
            ref_nll = zm[:, 0] + np.log(np.exp(z - zm).sum(axis=1)) - z[np.arange(n - 1), np.asarray(x[1:])]
            nerr = float(np.abs(nll - ref_nll).max())
            say(f"[gpu]   max |logits - oracle| = {err:.3g}, max |nll - oracle| = {nerr:.3g}, "
                f"L_spec {loss:.6g} vs {ref_loss:.6g}")
            assert err <= tol
            assert nerr <= 2 * tol
            assert abs(loss - ref_loss) <= 2 * tol * (n - 1)
    finally:
        dec.close()


@pytest.mark.parametrize("cfg,tol", [(synth.C1_TINY, 1e-4), (TINY_BF16, 2e-2)], ids=["f32", "bf16"])
def test_spec_forward_matches_oracle(cfg, tol):
    _run(cfg, 33, [1, 4, 16, 64], tol)


def test_one_ragged_wide_pass():
    _run(synth.C1_TINY, 100, [5, 16, 30], 1e-4, seed=3)


def test_blocks_straddle_passes():
    # 1099 rows: passes of 1024 and 75; blocks of 5 and 30 cross row 1024, blocks of 16 end on it
    _run(synth.C1_TINY, 1100, [5, 16, 30], 1e-4, seed=4)


def test_two_tokens():
    _run(synth.C1_TINY, 2, [1, 4], 1e-4, seed=5)


def test_decoder_only_split_is_the_full_model():
    cfg = synth.C1_TINY.replace(name="tiny-4L-h256-dec4", n_dec_layers=4)
    w = synth.make_weights(cfg, seed=1)
    x = synth.make_prompts(cfg, seed=9)[0]
    m = oracle_model(cfg, w)
    full = om.full_forward(m, x)[:-1]
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(x) + 8, max_draft=4)
    try:
        for b in (1, 3, 8):
            lg, _, _ = dec.spec_forward(x, b)
            assert float(np.abs(lg - full).max()) <= 1e-4
    finally:
        dec.close()


@pytest.mark.parametrize("cfg,tol", [(synth.C1_TINY, 1e-4), (TINY_BF16, 2e-2)], ids=["f32", "bf16"])
def test_shallow_buffer_contents_do_not_matter(cfg, tol):
    """The caller's buffer for the pass's own keys/values may hold anything (here every byte
    0xFF: NaN in fp32 and bf16); the call clears it, so the logits still match the oracle."""
    w = synth.make_weights(cfg, seed=0)
    x = synth.make_prompts(cfg.replace(prompt_len=37), seed=17)[0]
    m = oracle_model(cfg, w)
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(x) + 8, max_draft=4)
    try:
        dec.spec_forward(x, 4)          # allocates the shallow buffer
        dec._skv.fill_(255)
        lg, _, _ = dec.spec_forward(x, 4)
        ref, _ = os_.spec_forward(m, x, 4)
        err = float(np.abs(lg - ref).max())
        say(f"[gpu] {cfg.name}: shallow buffer of 0xFF bytes, max |logits - oracle| = {err:.3g}")
        assert np.all(np.isfinite(lg)) and err <= tol
    finally:
        dec.close()
