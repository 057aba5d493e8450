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

from gpu_common import GPU_ROWS, decoder, oracle_model, say, top2_gap
from oracle import model as om
from oracle import seed as os_
from oracle import tree as ot
from paper_2609_36590_amd import binding, synth

pytestmark = pytest.mark.gpu

TINY_BF16 = synth.C1_TINY.replace(name="tiny-4L-h256-bf16", dtype=synth.BF16)
# a wide FFN and 32 query heads: a depth-1 tree of 11 nodes runs the O and down projections split-K
WIDE = synth.C1_TINY.replace(name="wide-4L-h256-f8192", ffn=8192, n_heads=32, n_kv_heads=8, head_dim=128)


def _swap_chain_with_sibling(tree, d):
    """Exchange the tokens of the chain node at depth d and of its first sibling (same parent)."""
    j = next((i for i in range(len(tree.tokens)) if tree.depths[i] == d and i != d), None)
    if d < len(tree.tokens) and tree.depths[d] == d and j is not None:
        tree.tokens[d], tree.tokens[j] = tree.tokens[j], tree.tokens[d]


def _oracle_rounds(m, prompt, depth, n_rounds, schedule):
    st = os_.prefill(m, [int(x) for x in prompt], len(prompt) + n_rounds * (depth + 1) + 70)
    rounds = []
    for r in range(n_rounds):
        tree = ot.draft_tree(st, 0.0, depth, max_nodes=GPU_ROWS)
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
    (WIDE, 1e-4, 1, (1, 0, 1, 1)),
], ids=["f32-d3", "f32-d6", "bf16-d4", "wide-f32-d1"])
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


# ---------------------------------------------------------------------------------------------
# dynamic drafting (Confidence-Aware Dynamic Drafting) and the end-to-end tree decoding loop
# ---------------------------------------------------------------------------------------------
THRESHOLDS = tuple(t for t, _ in ot.FANOUT)
GAIN = 20.0   # sharpened logits are GAIN times larger, and so are their absolute errors


def _sharp_weights(cfg, gain=GAIN, enc=0.3, std=0.05, seed=0):
    """Random weights whose final-norm gain sharpens the softmax, so that the top-1 probabilities
    spread over every level of the top-p table."""
    w = synth.make_weights(cfg, seed=seed, std=std, enc_out_scale=enc)
    g = np.full(w["final_norm"].shape, gain, dtype=np.float32)
    w["final_norm"] = synth.f32_to_bf16_bits(g) if cfg.dtype == synth.BF16 else g
    return w


def _step_ambiguous(logits, p0, k, tau, tol, order=True):
    """Could logits within tol of these change the step's decisions: fan-out, stop, the top-1
    token, which tokens are candidates and (order=True) their ranking?"""
    if min(abs(p0 - x) for x in THRESHOLDS + (tau,)) <= 4 * tol:
        return True
    top = np.sort(np.asarray(logits, dtype=np.float64))[::-1][:k + 1]
    gaps = -np.diff(top)
    if order:
        return bool(np.any(gaps <= 2 * tol))
    return bool(gaps[0] <= 2 * tol or gaps[k - 1] <= 2 * tol)


def _tree_ambiguous(tree, tau, tol, order=True):
    return any(_step_ambiguous(tree.draft_logits[i], tree.p0[i], ot.fanout(tree.p0[i]), tau, tol, order)
               for i in range(len(tree.p0)))


@pytest.mark.parametrize("cfg,tol,tau,depth", [
    (synth.C1_TINY, 1e-4, 0.0, 6), (synth.C1_TINY, 1e-4, 0.7, 8), (TINY_BF16, 2e-2, 0.5, 6),
], ids=["f32-tau0-d6", "f32-tau0.7-d8", "bf16-tau0.5-d6"])
def test_drafting_matches_oracle(cfg, tol, tau, depth):
    """Teacher-forced rounds: the GPU drafts from the same committed state as the oracle (both
    then verify the oracle's tree); drafter logits, p0 and, where no decision is within the
    tolerance of a boundary, the packed tree must match."""
    tol = tol * GAIN
    w = _sharp_weights(cfg)
    prompt = synth.make_prompts(cfg)[0]
    m = oracle_model(cfg, w)
    n_rounds = 10
    cap = len(prompt) + n_rounds * (depth + 1) + 70
    st = os_.prefill(m, [int(x) for x in prompt], cap)
    dec = decoder(cfg, w, max_batch=1, max_ctx=cap, max_draft=depth)
    opts = binding.tree_opts(depth, tau=tau)
    try:
        dec.prefill([prompt])
        same_trees, levels, worst = 0, set(), 0.0
        for r in range(n_rounds):
            tree = ot.draft_tree(st, tau, depth, max_nodes=GPU_ROWS)
            toks, par, p0, lg = dec.draft_tree(opts, logits=True)
            say(f"[gpu] round {r}: oracle {len(tree.tokens)} nodes / {len(tree.p0)} steps, "
                f"GPU {len(toks)} nodes / {len(p0)} steps")
            # drafter logits of the steps fed the same chain tokens
            same = 1
            while (same < min(len(p0), len(tree.p0)) and toks[same] == tree.tokens[same]):
                same += 1
            worst = max(worst, float(np.abs(lg[:same] - tree.draft_logits[:same]).max()))
            np.testing.assert_allclose(p0[:same], tree.p0[:same], rtol=4 * tol, atol=1e-7)
            if not _tree_ambiguous(tree, tau, tol):
                assert toks == tree.tokens and par == tree.parents, r
                same_trees += 1
                levels |= {ot.fanout(x) for x in tree.p0}
            # both sides verify the oracle's tree
            logits, kv = ot.verify_tree(st, tree)
            path, bonus = ot.accept_tree(tree, logits)
            ot.commit_tree(st, tree, kv, path, bonus)
            dec.verify_tree(tree.tokens, tree.parents)
        say(f"[gpu] {same_trees}/{n_rounds} trees compared, fan-outs {sorted(levels)}, max |logits - oracle| = {worst:.3g}")
        assert worst <= tol
        if cfg.dtype == synth.F32:   # bf16's tolerance leaves few decisions unambiguous
            assert same_trees >= n_rounds // 2 and len(levels) >= 3
    finally:
        dec.close()


def _oracle_ok_prefix(m, prompt, toks, tol):
    """Length of the greedy continuation whose every choice has a top-2 gap above 2 tol."""
    lg = om.full_forward(m, list(prompt) + [int(x) for x in toks])[len(prompt) - 1:-1]
    amb = np.nonzero(top2_gap(lg) <= 2 * tol)[0]
    return int(amb[0]) if len(amb) else len(toks)


@pytest.mark.parametrize("cfg,tol,tau,depth,graph", [
    (synth.C1_TINY, 1e-4, 0.7, 8, False), (synth.C1_TINY, 1e-4, 0.7, 8, True),
    (synth.C1_TINY, 1e-4, 0.0, 5, True), (TINY_BF16, 2e-2, 0.5, 6, True),
], ids=["f32-tau0.7-eager", "f32-tau0.7-graph", "f32-tau0-graph", "bf16-tau0.5-graph"])
def test_generate_tree_is_lossless(cfg, tol, tau, depth, graph):
    """End to end: the committed tokens are the GPU's plain greedy decode (up to the first near
    tie of the oracle's greedy logits), and each round's accepted path length equals the oracle's
    tree decoding while no decision is ambiguous."""
    tol = tol * GAIN
    w = _sharp_weights(cfg, enc=0.05)
    prompt = synth.make_prompts(cfg)[0]
    m = oracle_model(cfg, w)
    max_new = 64
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + max_new + 2 * 65 + 8, max_draft=depth)
    try:
        ref, _, _ = dec.generate([prompt], 0, max_new)
        opts = binding.tree_opts(depth, tau=tau)
        toks, st = dec.generate_tree(prompt, opts, max_new, use_graph=graph, log_cap=256)
        n_ok = _oracle_ok_prefix(m, prompt, ref[0], tol)
        say(f"[gpu] {st['rounds']} rounds, {st['accepted']} accepted of {st['drafted']} drafted nodes, "
            f"{n_ok} unambiguous tokens")
        assert len(toks) == max_new
        np.testing.assert_array_equal(toks[:n_ok], ref[0][:n_ok])
        assert st["accepted"] > 0
        # the oracle's rounds, compared while every draft and verification decision is clear
        _, rounds = ot.generate_tree(m, prompt, tau, depth, max_new, record=True, max_nodes=GPU_ROWS)
        log = st["n_accept_log"]
        compared, t_gpu, t_or = 0, 0, 0
        for i, rd in enumerate(rounds):
            if i >= len(log) or t_gpu != t_or:   # both sides must start the round at the same position
                break
            visited = [0] + list(rd.path)   # the nodes whose argmax the acceptance reads
            if not (_tree_ambiguous(rd.tree, tau, tol, order=False)
                    or np.any(top2_gap(rd.verify_logits[visited]) <= 2 * tol)):
                assert log[i] == len(rd.path), (i, list(log[:i + 1]), [len(x.path) for x in rounds[:i + 1]])
                compared += 1
            t_gpu += int(log[i]) + 1
            t_or += len(rd.path) + 1
        say(f"[gpu] {compared} rounds match the oracle's accepted lengths")
        if cfg.dtype == synth.F32:   # bf16's tolerance leaves few decisions unambiguous
            assert compared >= 3
    finally:
        dec.close()


def test_generate_tree_eos_and_short_runs():
    cfg = synth.C1_TINY
    w = _sharp_weights(cfg, enc=0.05)
    prompt = synth.make_prompts(cfg)[0]
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + 40 + 2 * 65 + 8, max_draft=6)
    try:
        ref, _, _ = dec.generate([prompt], 0, 40)
        opts = binding.tree_opts(6, tau=0.5)
        one, st = dec.generate_tree(prompt, opts, 1, use_graph=True)
        np.testing.assert_array_equal(one, ref[0][:1])
        eos = int(ref[0][17])
        first = int(np.nonzero(ref[0] == eos)[0][0])
        toks, st = dec.generate_tree(prompt, opts, 40, eos_id=eos, use_graph=True)
        np.testing.assert_array_equal(toks, ref[0][:first + 1])
        with pytest.raises(binding.SeedError):
            dec.generate_tree(prompt, binding.tree_opts(7), 8)        # max_depth > max_draft
        with pytest.raises(binding.SeedError):
            dec.generate_tree(prompt, binding.tree_opts(4, table=((0.5, 1), (0.6, 3))), 8)   # increasing
    finally:
        dec.close()


@pytest.mark.parametrize("table,depth", [(((-1.0, 1),), 4), (((-1.0, 3),), 5)], ids=["chain-d4", "fan3-d5"])
def test_generate_tree_forced_acceptance(table, depth):
    """Benchmark mode: with the greedy continuation as the forced trace, every round accepts
    exactly sim_accept chain nodes (random weights accept almost nothing by themselves), and the
    output is still the greedy decode."""
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=3)
    prompt = synth.make_prompts(cfg, seed=2)[0]
    max_new = 48
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + max_new + 2 * 65 + 8, max_draft=depth)
    try:
        ref, _, _ = dec.generate([prompt], 0, max_new)
        opts = binding.tree_opts(depth, tau=0.0, table=table, rest=1)
        for a in (0, 2, depth):
            for graph in (False, True):
                toks, st = dec.generate_tree(prompt, opts, max_new, use_graph=graph, log_cap=256,
                                             sim_accept=a, forced_trace=ref[0])
                np.testing.assert_array_equal(toks, ref[0])
                log = st["n_accept_log"]
                say(f"[gpu] {table} a={a} graph={graph}: {st['rounds']} rounds, log {list(log)}")
                assert np.all(log[:-2] >= a)   # a leaf may extend a path by the trace's next token
                assert st["rounds"] <= -(-max_new // (a + 1))
    finally:
        dec.close()
