"""Pins of the dynamic-drafting / tree-verification oracle (oracle/tree.py).

* the top-p fan-out table at its boundaries;
* every tree node's verification logits equal a brute-force full recomputation of the committed
  prefix followed by the node's path (the tree mask hides other branches, nothing else);
* losslessness: the token stream equals brute-force greedy decoding for several thresholds,
  depths and splits;
* with fan-out 1 and no confidence stop, the tree is a chain and every round equals Algorithm 2
  with d = max_depth (drafts, acceptance, bonus);
* with no encoder (n_dec = l) and fan-out 1, the whole chain is accepted every round.
"""
import numpy as np
import pytest

from oracle import model as om
from oracle import seed as os_
from oracle import tree as ot
from paper_2609_36590_amd import synth

SMALL = synth.Config("s4", 4, 2, 64, 4, 2, 16, 96, 61, 1e4, dtype=synth.F32)
CHAIN = ((-1.0, 1),)   # every p0 > -1: fan-out 1


def _model(n_dec=2, enc_out_scale=0.3, seed=0, std=0.2):
    cfg = SMALL.replace(n_dec_layers=n_dec)
    w = synth.make_weights(cfg, seed=seed, std=std, enc_out_scale=enc_out_scale)
    return om.Model(cfg, w, np.float64)


def _prompt(n, seed=1):
    return [int(x) for x in np.random.default_rng(seed).integers(0, SMALL.vocab, size=n)]


def test_fanout_table_boundaries():
    assert ot.fanout(0.96) == 1 and ot.fanout(0.95) == 3
    assert ot.fanout(0.81) == 3 and ot.fanout(0.8) == 5
    assert ot.fanout(0.51) == 5 and ot.fanout(0.5) == 10 and ot.fanout(0.0) == 10


def test_tree_logits_are_each_path_recomputed():
    m = _model()
    prompt = _prompt(11)
    st = os_.prefill(m, prompt, 64)
    tree = ot.draft_tree(st, tau=0.0, max_depth=3)
    assert len(tree.tokens) > 4     # siblings exist (random weights: p0 is small, fan-out 10)
    logits, _ = ot.verify_tree(st, tree)
    for i in range(len(tree.tokens)):
        seq = list(prompt) + [tree.tokens[j] for j in tree.path(i)[1:]]
        ref = om.full_forward(m, seq)[-1]
        np.testing.assert_allclose(logits[i], ref, rtol=1e-9, atol=1e-11)


@pytest.mark.parametrize("tau,depth,n_dec", [(0.0, 3, 2), (0.3, 4, 2), (1.0, 2, 1), (0.0, 5, 3)])
def test_lossless_against_brute_force(tau, depth, n_dec):
    m = _model(n_dec=n_dec)
    prompt = _prompt(9, seed=3)
    toks, rounds = ot.generate_tree(m, prompt, tau, depth, 24, record=True)
    np.testing.assert_array_equal(toks, os_.greedy_brute_force(m, prompt, 24))
    assert sum(len(r.path) for r in rounds) > 0     # some drafts were accepted


def test_chain_tree_is_algorithm_2():
    m = _model()
    prompt = _prompt(10, seed=4)
    toks_t, rt = ot.generate_tree(m, prompt, 0.0, 4, 20, table=CHAIN, rest=1, record=True)
    toks_a, ra = os_.generate(m, prompt, 4, 20, record=True)
    np.testing.assert_array_equal(toks_t, toks_a)
    assert len(rt) == len(ra)
    for a, b in zip(rt, ra):
        assert a.tree.tokens == list(b.drafts)
        np.testing.assert_allclose(a.tree.draft_logits, b.draft_logits, rtol=1e-9, atol=1e-11)
        np.testing.assert_allclose(a.verify_logits, b.verify_logits, rtol=1e-9, atol=1e-11)
        assert len(a.path) == b.n_accept and a.bonus == b.bonus


def test_no_encoder_accepts_the_whole_chain():
    m = _model(n_dec=SMALL.n_layers)
    _, rounds = ot.generate_tree(m, _prompt(8, seed=5), 0.0, 3, 16, table=CHAIN, rest=1, record=True)
    assert all(len(r.path) == 3 for r in rounds)


def test_siblings_are_leaves_and_packed_after_the_chain():
    m = _model()
    st = os_.prefill(m, _prompt(7, seed=6), 32)
    tree = ot.draft_tree(st, tau=0.0, max_depth=3)
    chain = [0] + [i for i in range(1, len(tree.tokens)) if tree.parents[i] == i - 1 and tree.depths[i] == i]
    assert len(chain) == 4
    for i in range(len(chain), len(tree.tokens)):
        assert tree.parents[i] in chain and all(tree.parents[j] != i for j in range(len(tree.tokens)))
        assert tree.depths[i] == tree.depths[tree.parents[i]] + 1


def test_ranking_breaks_ties_to_the_lower_id():
    z = np.array([1.0, 3.0, 3.0, 2.0, 3.0, -1.0])
    p0, order = ot._confidence(z)
    assert list(order) == [1, 2, 4, 3, 0, 5]
    e = np.exp(z - 3.0)
    assert abs(p0 - 1.0 / e.sum()) < 1e-15


@pytest.mark.parametrize("gain,tau,depth", [(1.0, 0.0, 3), (8.0, 0.0, 4), (20.0, 0.7, 6), (40.0, 0.5, 6),
                                            (60.0, 0.0, 5)])
def test_drafting_steps_match_an_independent_softmax_and_sort(gain, tau, depth):
    """p0, fan-out, candidates and the tau stop of every drafting step against a torch float64
    softmax and a stable torch sort of the recorded drafter logits; the final-norm gain scales the
    logits so that p0 moves across the top-p table's levels."""
    from tree_pins import check_drafting_steps
    cfg = SMALL.replace(n_dec_layers=2)
    w = synth.make_weights(cfg, seed=0, std=0.2, enc_out_scale=0.3)
    w["final_norm"] = w["final_norm"] * gain
    m = om.Model(cfg, w, np.float64)
    seen = set()
    for seed in range(4):
        st = os_.prefill(m, _prompt(9, seed=20 + seed), 96)
        tree = ot.draft_tree(st, tau, depth)
        seen.update(check_drafting_steps(tree, tau, depth, ot.FANOUT, ot.FANOUT_REST))
    assert seen


def test_every_fanout_level_is_exercised():
    """Across the scaled models of the test above, every level of the table (1, 3, 5, 10) occurs."""
    from tree_pins import check_drafting_steps
    cfg = SMALL.replace(n_dec_layers=2)
    seen = set()
    for gain in (1.0, 8.0, 20.0, 40.0, 60.0):
        w = synth.make_weights(cfg, seed=0, std=0.2, enc_out_scale=0.3)
        w["final_norm"] = w["final_norm"] * gain
        m = om.Model(cfg, w, np.float64)
        for seed in range(4):
            st = os_.prefill(m, _prompt(9, seed=20 + seed), 96)
            seen.update(check_drafting_steps(ot.draft_tree(st, 0.0, 6), 0.0, 6, ot.FANOUT, ot.FANOUT_REST))
    assert seen >= {1, 3, 5, 10}, seen


def test_unbounded_by_default_and_budget_when_asked():
    """The paper sets no node budget: a depth-6 tree at fan-out 10 holds 61 nodes by default, and a
    budget of 20 cuts the fan-out to the nodes left and stops drafting once none are left."""
    m = _model()
    st = os_.prefill(m, _prompt(7, seed=6), 96)
    full = ot.draft_tree(st, 0.0, 6)
    assert len(full.tokens) == 1 + 6 * 10
    st.cache.truncate(st.t - 1)     # drop the shallow entries of the first drafting (Alg. 2's truncate)
    cut = ot.draft_tree(st, 0.0, 6, max_nodes=20)
    assert len(cut.tokens) == 20 and len(cut.p0) == 2
