"""The tree oracle's pins catch plausible mistakes: each test plants one mistake in oracle/tree.py
(on the CPU, via monkeypatch) and checks that the pin guarding that step would fail: per-node
logits against a brute-force recomputation of the node's path, losslessness against brute-force
greedy decoding, and the fan-out table's boundaries."""
import numpy as np

from oracle import model as om
from oracle import seed as os_
from oracle import tree as ot
from paper_2609_36590_amd import synth

SMALL = synth.Config("s4", 4, 2, 64, 4, 2, 16, 96, 61, 1e4, dtype=synth.F32)


def _model(n_dec=2, enc_out_scale=0.3):
    cfg = SMALL.replace(n_dec_layers=n_dec)
    return om.Model(cfg, synth.make_weights(cfg, seed=0, std=0.2, enc_out_scale=enc_out_scale), np.float64)


def _prompt(n, seed):
    return [int(x) for x in np.random.default_rng(seed).integers(0, SMALL.vocab, size=n)]


def _path_logit_error(m, prompt, depth=3):
    """Largest deviation of any node's verification logits from a full recomputation of the
    committed prefix followed by the node's path (the per-node pin)."""
    st = os_.prefill(m, prompt, 64)
    tree = ot.draft_tree(st, tau=0.0, max_depth=depth)
    logits, _ = ot.verify_tree(st, tree)
    err = 0.0
    for i in range(len(tree.tokens)):
        seq = list(prompt) + [tree.tokens[j] for j in tree.path(i)[1:]]
        err = max(err, float(np.abs(logits[i] - om.full_forward(m, seq)[-1]).max()))
    return err


def test_unplanted_tree_passes_the_pins():
    m = _model()
    assert _path_logit_error(m, _prompt(11, 1)) < 1e-9
    toks, _ = ot.generate_tree(m, _prompt(9, 3), 0.0, 3, 20)
    np.testing.assert_array_equal(toks, os_.greedy_brute_force(m, _prompt(9, 3), 20))


def test_causal_mask_over_packed_order_breaks_path_pin(monkeypatch):
    # every node seeing all earlier packed nodes (a chain mask) lets siblings leak into each other
    def causal(tree):
        n = len(tree.tokens)
        return np.tril(np.ones((n, n), dtype=bool))

    monkeypatch.setattr(ot, "_ancestor_mask", causal)
    assert _path_logit_error(_model(), _prompt(11, 1)) > 1e-3


def test_rotary_position_by_slot_breaks_path_pin(monkeypatch):
    # nodes rotated by their packed slot p + i instead of their depth p + depth(i) (the ancestor
    # mask comes from the parents and stays right)
    orig = ot.verify_tree

    def by_slot(st, tree):
        return orig(st, ot.Tree(tree.tokens, tree.parents, list(range(len(tree.tokens))), tree.p0,
                                tree.draft_logits))

    monkeypatch.setattr(ot, "verify_tree", by_slot)
    assert _path_logit_error(_model(), _prompt(11, 1)) > 1e-3


def test_inclusive_fanout_thresholds_break_boundary_pin():
    # p0 >= threshold instead of p0 > threshold: the boundary values take the smaller fan-out
    def fanout_ge(p0, table=ot.FANOUT, rest=ot.FANOUT_REST):
        for thr, k in table:
            if p0 >= thr:
                return k
        return rest

    assert fanout_ge(0.95) != ot.fanout(0.95) and fanout_ge(0.8) != ot.fanout(0.8)
    assert fanout_ge(0.5) != ot.fanout(0.5)


def test_bonus_from_the_root_breaks_lossless_pin(monkeypatch):
    # the bonus token taken at the root instead of the last accepted node
    good = ot.accept_tree

    def bad(tree, logits):
        path, _ = good(tree, logits)
        return path, int(np.argmax(logits[0]))

    monkeypatch.setattr(ot, "accept_tree", bad)
    m = _model(enc_out_scale=0.05)
    prompt = _prompt(9, 3)
    toks, rounds = ot.generate_tree(m, prompt, 0.0, 3, 20, record=True)
    assert any(r.path for r in rounds)
    assert not np.array_equal(toks, os_.greedy_brute_force(m, prompt, 20))


def test_accepting_any_node_with_the_token_breaks_lossless_pin(monkeypatch):
    # a match anywhere in the tree (not only among the current node's children) is accepted
    def bad(tree, logits):
        node, path = 0, []
        while True:
            g = int(np.argmax(logits[node]))
            nxt = next((c for c in range(1, len(tree.tokens)) if tree.tokens[c] == g and c not in path
                        and c != node), None)
            if nxt is None:
                break
            path.append(nxt)
            node = nxt
        return path, int(np.argmax(logits[node]))

    monkeypatch.setattr(ot, "accept_tree", bad)
    m = _model(enc_out_scale=0.3)
    caught = False
    for seed in range(3, 9):
        prompt = _prompt(9, seed)
        try:
            toks, _ = ot.generate_tree(m, prompt, 0.0, 3, 20)
        except (AssertionError, IndexError, ValueError):
            caught = True   # the cache refuses keys/values of a path that is not a chain of ancestors
            break
        if not np.array_equal(toks, os_.greedy_brute_force(m, prompt, 20)):
            caught = True
            break
    assert caught


def test_committing_packed_rows_breaks_lossless_pin(monkeypatch):
    # keys/values committed from the first packed rows (the top-1 chain) instead of the accepted
    # path: wrong whenever the path ends on a sibling leaf
    def bad_commit(st, tree, kv, path, bonus):
        rows = list(range(len(path) + 1))
        for i, (k, v) in enumerate(kv):
            st.cache.append(i, st.p, k[rows], v[rows])
        st.tokens.extend(int(tree.tokens[j]) for j in path)
        st.tokens.append(int(bonus))
        st.cache.truncate(st.t - 1)

    monkeypatch.setattr(ot, "commit_tree", bad_commit)
    m = _model(enc_out_scale=0.3)
    caught, leaf_rounds = False, 0
    for seed in range(3, 13):
        prompt = _prompt(9, seed)
        toks, rounds = ot.generate_tree(m, prompt, 0.0, 3, 20, record=True)
        leaf_rounds += sum(bool(r.path) and r.path[-1] != len(r.path) for r in rounds)
        if not np.array_equal(toks, os_.greedy_brute_force(m, prompt, 20)):
            caught = True
            break
    assert leaf_rounds > 0 and caught


def _confidence_pin_fails(monkeypatch, bad_confidence):
    """Plant bad_confidence as the drafting step's (p0, ranking) and report whether the
    independent softmax/sort pin (tests/tree_pins.py) rejects the drafted trees."""
    from tree_pins import check_drafting_steps
    monkeypatch.setattr(ot, "_confidence", bad_confidence)
    cfg = SMALL.replace(n_dec_layers=2)
    for gain in (1.0, 20.0, 40.0):
        w = synth.make_weights(cfg, seed=0, std=0.2, enc_out_scale=0.3)
        w["final_norm"] = w["final_norm"] * gain
        m = om.Model(cfg, w, np.float64)
        for seed in range(4):
            st = os_.prefill(m, _prompt(9, 20 + seed), 96)
            tree = ot.draft_tree(st, 0.5, 5)
            try:
                check_drafting_steps(tree, 0.5, 5, ot.FANOUT, ot.FANOUT_REST)
            except AssertionError:
                return True
    return False


def test_p0_from_the_second_ranked_token_breaks_confidence_pin(monkeypatch):
    # p0 read at rank 2 (the ranking itself right): every existing losslessness pin still passes,
    # the independent recomputation of p0 does not
    good = ot._confidence

    def second(logits):
        _, order = good(logits)
        z = np.asarray(logits, dtype=np.float64)
        pr = np.exp(z - z.max())
        pr /= pr.sum()
        return float(pr[order[1]]), order

    assert _confidence_pin_fails(monkeypatch, second)


def test_coarse_ranking_with_ties_to_the_higher_id_breaks_confidence_pin(monkeypatch):
    # the ranking taken over logits coarsened to quarters (so candidates tie) with ties broken
    # towards the higher token id; the tie rule itself is pinned directly in
    # test_oracle_tree.py::test_ranking_breaks_ties_to_the_lower_id
    def higher_first(logits):
        z = np.asarray(logits, dtype=np.float64)
        z = np.round(z * 4.0) / 4.0          # coarse logits: many exact ties among candidates
        pr = np.exp(z - z.max())
        pr /= pr.sum()
        order = np.lexsort((-np.arange(len(z)), -z))
        return float(pr[order[0]]), order

    assert _confidence_pin_fails(monkeypatch, higher_first)


def test_candidates_from_the_lowest_logits_break_confidence_pin(monkeypatch):
    # ranking reversed: the fan-out's candidates taken from the bottom of the distribution
    good = ot._confidence

    def reversed_rank(logits):
        p0, order = good(logits)
        return p0, order[::-1]

    assert _confidence_pin_fails(monkeypatch, reversed_rank)
