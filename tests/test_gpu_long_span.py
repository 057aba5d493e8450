"""GPU parity of the wider attention groups against the oracle.

A decoder's context and batch capacities fix how many positions one attention workgroup covers:
for one sequence 64 up to 4096, 128 up to 8192 and 256 beyond (several sequences take 128 from 2049
on), so that a query's merge tree depends only on absolute positions.
The other GPU tests run small capacities (64-position groups); these cases build the tiny models
with capacities 6000 and 9000 and a 600-token prompt, so the 128- and 256-position groups run
several groups per query and merge them in the combine kernel, for each attention variant:

* Algorithm 2 rounds (causal verification rows, drafting steps over deep and shallow entries),
  teacher-forced from the oracle's own decode, every draft and verify logit row;
* tree verification (ancestor mask) over consecutive rounds, some ending on a sibling leaf;
* the block-causal drafter pass of the speculative drafting objective (Algorithm 1).

A fifth case gives the bf16 model a capacity of 250000 positions: its block table (62.5 KB) no
longer fits the LDS of the one-launch pass attention beside the tile slots, so the prompt's prefill
and the drafting objective's pass run on the split-KV kernel and its merge instead (the path every
capacity beyond ~131k positions takes).

fp32 models within 1e-4, bf16 within 2e-2 (max abs over all logits).
"""
import numpy as np
import pytest

from gpu_common import check_round, decoder, oracle_model, say, top2_gap
from oracle import seed as os_
from paper_2609_36590_amd import synth
from test_gpu_tree import _oracle_rounds

pytestmark = pytest.mark.gpu

K = 4
PROMPT = 600
TINY_BF16 = synth.C1_TINY.replace(name="tiny-4L-h256-bf16", dtype=synth.BF16)
CASES = [(synth.C1_TINY, 1e-4, 6000), (synth.C1_TINY, 1e-4, 9000), (TINY_BF16, 2e-2, 6000), (TINY_BF16, 2e-2, 9000),
         (TINY_BF16, 2e-2, 250000)]
IDS = ["f32-span128", "f32-span256", "bf16-span128", "bf16-span256", "bf16-no-pass-kernel"]


@pytest.mark.parametrize("cfg,tol,cap", CASES, ids=IDS)
def test_rounds_match_oracle(cfg, tol, cap):
    w = synth.make_weights(cfg, seed=0, enc_out_scale=0.1)
    prompt = synth.make_prompts(cfg.replace(prompt_len=PROMPT), seed=11)[0]
    m = oracle_model(cfg, w)
    toks, rounds = os_.generate(m, prompt, K, 24, record=True)
    dec = decoder(cfg, w, max_batch=1, max_ctx=cap, max_draft=K)
    try:
        worst_d = worst_v = 0.0
        for rd in rounds:
            dmax, vmax = check_round(dec, prompt, toks, rd, tol, K)
            worst_d, worst_v = max(worst_d, dmax), max(worst_v, vmax)
        say(f"[gpu] {cfg.name} capacity {cap}: {len(rounds)} rounds, max |draft - oracle| = {worst_d:.3g}, "
            f"max |verify - oracle| = {worst_v:.3g}")
        assert worst_d <= tol and worst_v <= tol
    finally:
        dec.close()


@pytest.mark.parametrize("cfg,tol,cap", CASES, ids=IDS)
def test_tree_rounds_match_oracle(cfg, tol, cap):
    w = synth.make_weights(cfg, seed=0, enc_out_scale=0.1)
    prompt = synth.make_prompts(cfg.replace(prompt_len=PROMPT), seed=12)[0]
    m = oracle_model(cfg, w)
    rounds = _oracle_rounds(m, prompt, 3, 6, (0, 2, 1, 3))
    dec = decoder(cfg, w, max_batch=1, max_ctx=cap, max_draft=K)
    try:
        dec.prefill([prompt])
        worst, checked = 0.0, 0
        for rd in rounds:
            path, bonus, lg = dec.verify_tree(rd.tree.tokens, rd.tree.parents, logits=True)
            worst = max(worst, float(np.abs(lg - rd.verify_logits).max()))
            if np.any(top2_gap(rd.verify_logits) <= 2 * tol):
                say(f"[gpu] p={rd.p}: near tie, stopping the comparison")
                break
            assert path == rd.path and bonus == rd.bonus, (rd.p, path, rd.path, bonus, rd.bonus)
            checked += 1
        say(f"[gpu] {cfg.name} capacity {cap}: {checked} tree rounds, max |logits - oracle| = {worst:.3g}")
        assert worst <= tol and checked >= 3
    finally:
        dec.close()


@pytest.mark.parametrize("cfg,tol,cap", CASES, ids=IDS)
def test_spec_forward_matches_oracle(cfg, tol, cap):
    w = synth.make_weights(cfg, seed=0)
    x = synth.make_prompts(cfg.replace(prompt_len=PROMPT), seed=13)[0]
    m = oracle_model(cfg, w)
    dec = decoder(cfg, w, max_batch=1, max_ctx=cap, max_draft=K)
    try:
        for b in (4, 100):
            ref, ref_loss = os_.spec_forward(m, x, b)
            lg, _, loss = dec.spec_forward(x, b)
            err = float(np.abs(lg - ref).max())
            say(f"[gpu] {cfg.name} capacity {cap} block {b}: max |logits - oracle| = {err:.3g}, "
                f"L_spec {loss:.6g} vs {ref_loss:.6g}")
            assert err <= tol
            assert abs(loss - ref_loss) <= 2 * tol * (len(x) - 1)
    finally:
        dec.close()
