"""GPU tree-based verification (Tree-Based Verification; Fig. 3 right) against the oracle.

The oracle drafts trees on the tiny models (encoder output projections damped so that the
verifier agrees with the drafter's top-1 chain) and, in scheduled rounds, swaps the token of the
chain node at depth d with its first sibling's: the verifier then accepts that sibling, a leaf,
and the round ends there, so its keys/values must move from the leaf's packed slot to position
p + d. The GPU verifies the oracle's trees round after round from one prefill, so every round also
checks the previous rounds' commits. Every node's logits must be within the tolerance (fp32 1e-4,
bf16 2e-2), and the accepted path and bonus must match wherever the oracle's top-2 gaps leave no
doubt.
"""
import numpy as np
import pytest

from gpu_common import decoder, oracle_model, say, top2_gap
from oracle import seed as os_
from oracle import tree as ot
from paper_2609_36590_amd import binding, synth

pytestmark = pytest.mark.gpu

TINY_BF16 = synth.C1_TINY.replace(name="tiny-4L-h256-bf16", dtype=synth.BF16)


def _swap_chain_with_sibling(tree, d):
    """Exchange the tokens of the chain node at depth d and of its first sibling (same parent)."""
    j = next((i for i in range(len(tree.tokens)) if tree.depths[i] == d and i != d), None)
    if d < len(tree.tokens) and tree.depths[d] == d and j is not None:
        tree.tokens[d], tree.tokens[j] = tree.tokens[j], tree.tokens[d]


def _oracle_rounds(m, prompt, depth, n_rounds, schedule):
    st = os_.prefill(m, [int(x) for x in prompt], len(prompt) + n_rounds * (depth + 1) + 70)
    rounds = []
    for r in range(n_rounds):
        tree = ot.draft_tree(st, 0.0, depth)
        if schedule[r % len(schedule)]:
            _swap_chain_with_sibling(tree, schedule[r % len(schedule)])
        logits, kv = ot.verify_tree(st, tree)
        path, bonus = ot.accept_tree(tree, logits)
        rounds.append(ot.TreeRound(st.p, tree, logits, path, bonus))
        ot.commit_tree(st, tree, kv, path, bonus)
    return rounds


@pytest.mark.parametrize("cfg,tol,depth,schedule", [
    (synth.C1_TINY, 1e-4, 3, (0, 1, 3, 2)),
    (synth.C1_TINY, 1e-4, 6, (2, 0, 6, 4, 1)),
    (TINY_BF16, 2e-2, 4, (3, 1, 0, 4)),
], ids=["f32-d3", "f32-d6", "bf16-d4"])
def test_tree_rounds_match_oracle(cfg, tol, depth, schedule):
    w = synth.make_weights(cfg, seed=0, enc_out_scale=0.1)
    prompt = synth.make_prompts(cfg)[0]
    m = oracle_model(cfg, w)
    n_rounds = 8
    rounds = _oracle_rounds(m, prompt, depth, n_rounds, schedule)
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + n_rounds * (depth + 1) + 70, max_draft=6)
    try:
        dec.prefill([prompt])
        worst, leaf_ends, checked = 0.0, 0, 0
        for rd in rounds:
            say(f"[gpu] p={rd.p}: {len(rd.tree.tokens)} nodes")
            path, bonus, lg = dec.verify_tree(rd.tree.tokens, rd.tree.parents, logits=True)
            worst = max(worst, float(np.abs(lg - rd.verify_logits).max()))
            if np.any(top2_gap(rd.verify_logits) <= 2 * tol):
                say(f"[gpu] p={rd.p}: near tie, stopping the comparison")
                break
            assert path == rd.path and bonus == rd.bonus, (rd.p, path, rd.path, bonus, rd.bonus)
            checked += 1
            leaf_ends += bool(rd.path) and rd.path[-1] != len(rd.path)
        say(f"[gpu] {cfg.name} depth {depth}: {checked} rounds, {leaf_ends} ended on a leaf, "
            f"max |logits - oracle| = {worst:.3g}")
        assert worst <= tol
        assert checked == n_rounds and leaf_ends >= 3
        full = list(prompt) + [t for rd in rounds for t in [rd.tree.tokens[j] for j in rd.path] + [rd.bonus]]
        np.testing.assert_array_equal(dec.tokens(0), full)
    finally:
        dec.close()


def test_root_only_tree_is_a_plain_step():
    """A one-node tree verifies the pending token alone: the bonus is the greedy next token."""
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=2)
    prompt = synth.make_prompts(cfg, seed=4)[0]
    m = oracle_model(cfg, w)
    ref = os_.greedy_brute_force(m, prompt, 3)
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + 8, max_draft=4)
    try:
        dec.prefill([prompt])
        for i in range(3):
            path, bonus, _ = dec.verify_tree([int(dec.tokens(0)[-1])], [-1])
            assert path == [] and bonus == int(ref[i])
    finally:
        dec.close()


def test_tree_argument_errors():
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=0)
    dec = decoder(cfg, w, max_batch=1, max_ctx=128, max_draft=4)
    try:
        with pytest.raises(binding.SeedError):
            dec.verify_tree([1, 2], [-1, 0])   # before prefill
        dec.prefill([synth.make_prompts(cfg)[0]])
        t0 = len(dec.tokens(0))
        for toks, par in (([1, 2], [0, 0]), ([1, 2, 3], [-1, 0, 2]), ([1, cfg.vocab], [-1, 0]), ([], []),
                          ([1] * 65, [-1] + list(range(64)))):
            with pytest.raises(binding.SeedError):
                dec.verify_tree(toks, par)
        assert len(dec.tokens(0)) == t0
    finally:
        dec.close()
