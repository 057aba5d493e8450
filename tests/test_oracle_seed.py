"""Pins for the oracle's Algorithm 2: lossless decoding against brute-force greedy, per-round
acceptance against brute-force prefix matching, verify rows against full recomputation, the
incremental drafter against the parallel block-mask drafter pass, and the method's special
cases (d = 0 is plain greedy; l' = 0 accepts everything; no decoder layers = closed form)."""
import numpy as np
import pytest

from oracle import model as om
from oracle import seed as os_
from paper_2609_36590_amd import synth

# 4 layers so that every split n_dec in 0..4 exists; GQA 4q/2kv.
SMALL = synth.Config("s4", 4, 2, 64, 4, 2, 16, 96, 61, 1e4, dtype=synth.F32)


def _model(cfg, n_dec=None, enc_out_scale=1.0, seed=0, dtype=np.float64, std=0.2):
    if n_dec is not None:
        cfg = cfg.replace(n_dec_layers=n_dec)
    w = synth.make_weights(cfg, seed=seed, std=std, enc_out_scale=enc_out_scale)
    return om.Model(cfg, w, dtype)


def _prompt(cfg, n, seed=1):
    return np.random.default_rng(seed).integers(0, cfg.vocab, size=n)


def test_verify_rows_equal_full_recompute():
    m = _model(SMALL)
    prompt = _prompt(SMALL, 12)
    st = os_.prefill(m, prompt, 64)
    drafts = np.array([prompt[-1], 5, 17, 3, 40])
    logits = os_.verify(st, drafts)
    for r in range(len(drafts)):
        seq = list(prompt) + list(drafts[1:r + 1])
        np.testing.assert_allclose(logits[r], om.full_forward(m, seq)[-1], rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("n_dec", [1, 2, 3])
def test_incremental_draft_equals_block_mask_pass(n_dec):
    m = _model(SMALL, n_dec=n_dec)
    prompt = _prompt(SMALL, 15, seed=2)
    st = os_.prefill(m, prompt, 64)
    # advance one round so the deep cache comes from a verification, not only the prefill
    d, ql = os_.draft(st, 3)
    n, b = os_.accept(d, os_.verify(st, d))
    os_.commit(st, d, n, b)
    ctx = list(st.tokens)
    drafts, qlog = os_.draft(st, 5)
    ref = os_.block_draft_logits(m, ctx, drafts[1:5])
    np.testing.assert_allclose(qlog, ref, rtol=1e-9, atol=1e-11)


def test_draft_without_decoder_layers_is_head_of_raw_embedding():
    m = _model(SMALL, n_dec=0)
    st = os_.prefill(m, _prompt(SMALL, 9), 32)
    drafts, qlog = os_.draft(st, 3)
    E = m.w["embed"]
    for i in range(3):
        e = E[drafts[i]]
        closed = (e / np.sqrt(np.mean(e * e) + SMALL.rms_eps)) @ E.T
        np.testing.assert_allclose(qlog[i], closed, rtol=1e-12, atol=1e-13)


@pytest.fixture(scope="module")
def damped():
    """One weight set (encoder output projections damped so drafts are often right) and its
    brute-force greedy continuation, shared by every split."""
    cfg = SMALL
    w = synth.make_weights(cfg, seed=3, std=0.2, enc_out_scale=0.15)
    prompt = _prompt(cfg, 10, seed=4)
    # 24 tokens are generated; 7 more let the last round's drafts be checked too
    ref = os_.greedy_brute_force(om.Model(cfg, w, np.float64), prompt, 24 + 7)
    return w, prompt, ref


@pytest.mark.parametrize("n_dec", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("d", [0, 1, 2, 3, 4, 5, 6])
def test_lossless_against_brute_force(damped, n_dec, d):
    w, prompt, ref = damped
    m = om.Model(SMALL.replace(n_dec_layers=n_dec), w, np.float64)
    toks, rounds = os_.generate(m, prompt, d, 24, record=True)
    np.testing.assert_array_equal(toks, ref[:24])
    # every round's n_accept is the longest prefix of drafts that matches greedy decoding
    full = list(prompt) + list(ref)
    for rd in rounds:
        cont = full[rd.p + 1:rd.p + 1 + d]
        n = 0
        assert len(cont) == d
        while n < d and rd.drafts[n + 1] == cont[n]:
            n += 1
        assert rd.n_accept == n
        assert rd.bonus == full[rd.p + 1 + rd.n_accept]


def test_damped_model_exercises_partial_acceptance(damped):
    w, prompt, ref = damped
    m = om.Model(SMALL, w, np.float64)
    _, rounds = os_.generate(m, prompt, 4, 24, record=True)
    seen = {r.n_accept for r in rounds}
    assert len(seen) >= 2 and max(seen) >= 1, seen


def test_decoder_is_whole_model_accepts_every_draft():
    m = _model(SMALL, n_dec=SMALL.n_layers, seed=5)
    prompt = _prompt(SMALL, 8, seed=6)
    toks, rounds = os_.generate(m, prompt, 4, 20, record=True)
    assert all(r.n_accept == 4 for r in rounds)
    np.testing.assert_array_equal(toks, os_.greedy_brute_force(m, prompt, 20))


def test_draft_length_zero_is_plain_greedy():
    m = _model(SMALL, seed=7)
    prompt = _prompt(SMALL, 6, seed=8)
    toks, rounds = os_.generate(m, prompt, 0, 12, record=True)
    assert len(rounds) == 12 and all(r.n_accept == 0 for r in rounds)
    np.testing.assert_array_equal(toks, os_.greedy_brute_force(m, prompt, 12))


@pytest.mark.parametrize("j", [0, 1, 2, 3, 4])
def test_forced_drafts_accept_exactly_the_greedy_prefix(j):
    m = _model(SMALL, seed=9)
    prompt = _prompt(SMALL, 7, seed=10)
    g = os_.greedy_brute_force(m, prompt, 6)
    st = os_.prefill(m, prompt, 32)
    drafts = [prompt[-1]] + list(g[:j])
    if j < 4:
        drafts += [(g[j] + 1) % SMALL.vocab] + [0] * (3 - j)
    n, bonus = os_.accept(np.array(drafts), os_.verify(st, np.array(drafts)))
    assert n == j and bonus == g[j]


def test_commit_keeps_deep_cache_for_accepted_tokens_only():
    m = _model(SMALL, seed=11)
    prompt = _prompt(SMALL, 9, seed=12)
    st = os_.prefill(m, prompt, 32)
    assert st.cache.valid.tolist() == [8] * SMALL.n_layers
    d, _ = os_.draft(st, 3)
    dec = m.first_decoder_layer
    assert st.cache.valid[dec:].tolist() == [11] * (SMALL.n_layers - dec)
    assert st.cache.valid[:dec].tolist() == [8] * dec
    n, b = os_.accept(d, os_.verify(st, d))
    os_.commit(st, d, n, b)
    assert st.cache.valid.tolist() == [st.t - 1] * SMALL.n_layers


def test_eos_stops_generation():
    m = _model(SMALL, seed=13)
    prompt = _prompt(SMALL, 5, seed=14)
    ref = os_.greedy_brute_force(m, prompt, 10)
    eos = int(ref[4])
    first = list(ref).index(eos)
    toks, _ = os_.generate(m, prompt, 3, 10, eos=eos)
    np.testing.assert_array_equal(toks, ref[:first + 1])


def test_fp32_oracle_tracks_fp64_on_tiny_config():
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=0)
    prompt = synth.make_prompts(cfg)[0][:16]
    l32 = om.full_forward(om.Model(cfg, w, np.float32), prompt)
    l64 = om.full_forward(om.Model(cfg, w, np.float64), prompt)
    assert np.abs(l32 - l64).max() < 1e-5


# ---- forward pass of the speculative drafting objective (Algorithm 1) ----

def _spec_case(n_dec, n=13, seed=4):
    m = _model(SMALL, n_dec=n_dec, seed=seed)
    return m, _prompt(SMALL, n, seed=seed + 1)


def test_spec_forward_block_one_is_first_draft_step_everywhere():
    """b = 1: row q sees the deep cache of X[0..q-1] and only its own raw embedding, i.e. the
    first drafting step after a prefill of X[0..q] (cached path of Algorithm 2)."""
    m, x = _spec_case(2)
    logits, _ = os_.spec_forward(m, x, 1)
    for q in range(len(x) - 1):
        st = os_.prefill(m, x[:q + 1], 32)
        _, ql = os_.draft(st, 1)
        np.testing.assert_allclose(logits[q], ql[0], rtol=1e-9, atol=1e-11)


def test_spec_forward_single_block_is_the_decoder_alone():
    """b >= n: no deep context at all; the decoder layers act as a causal LM over H^0."""
    m, x = _spec_case(2)
    logits, _ = os_.spec_forward(m, x, 64)
    sub_cfg = SMALL.replace(n_layers=2, n_dec_layers=2)
    L0 = SMALL.n_layers - 2
    w = {}
    for k, v in m.w.items():
        if k.startswith("layers."):
            i = int(k.split(".")[1])
            if i >= L0:
                w[f"layers.{i - L0}." + k.split(".", 2)[2]] = v
        else:
            w[k] = v
    sub = om.Model(sub_cfg, w, np.float64)
    ref = om.full_forward(sub, x[:-1])
    np.testing.assert_allclose(logits, ref, rtol=1e-9, atol=1e-11)


@pytest.mark.parametrize("b", [1, 3, 5])
def test_spec_forward_without_encoder_is_the_full_model(b):
    """n_dec = l: the drafter is the whole model, so every block reproduces causal f."""
    m, x = _spec_case(SMALL.n_layers)
    logits, _ = os_.spec_forward(m, x, b)
    np.testing.assert_allclose(logits, om.full_forward(m, x)[:-1], rtol=1e-9, atol=1e-11)


@pytest.mark.parametrize("b", [2, 4])
def test_spec_forward_blocks_are_independent_drafts(b):
    """Each block equals the block-mask drafter pass from the committed prefix X[0..s] with the
    block's tokens as teacher-forced draft inputs."""
    m, x = _spec_case(2, n=12)
    logits, _ = os_.spec_forward(m, x, b)
    for s in range(0, len(x) - 1, b):
        e = min(s + b, len(x) - 1)
        ref = os_.block_draft_logits(m, x[:s + 1], x[s + 1:e])
        np.testing.assert_allclose(logits[s:e], ref, rtol=1e-9, atol=1e-11)


def test_spec_loss_is_the_summed_negative_log_likelihood():
    m, x = _spec_case(2)
    logits, loss = os_.spec_forward(m, x, 3)
    z = logits.astype(np.float64)
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    ref = -sum(np.log(p[q, x[q + 1]]) for q in range(len(x) - 1))
    assert abs(loss - ref) <= 1e-9 * abs(ref)


def test_row_blocked_prefill_is_the_same_cache():
    """Prefill in row blocks (bounded memory for long prompts) fills the same cache as one pass."""
    cfg = synth.C1_TINY
    mm = om.Model(cfg, synth.weights_as_f32(cfg, synth.make_weights(cfg, seed=2)), np.float64)
    prompt = synth.make_prompts(cfg.replace(prompt_len=45), seed=4)[0]
    a = os_.prefill(mm, prompt, 64)
    b = os_.prefill(mm, prompt, 64, row_block=16)
    np.testing.assert_array_equal(a.cache.valid, b.cache.valid)
    np.testing.assert_allclose(b.cache.K, a.cache.K, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(b.cache.V, a.cache.V, rtol=1e-12, atol=1e-14)
