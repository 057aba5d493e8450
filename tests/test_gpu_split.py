"""GPU parity across encoder/decoder splits (the decoder-size sweep of Fig. 6 and Table 4).

The tiny fp32 model (4 layers) is run with every split n_dec = l - l' in {0, 1, 3, 4} (n_dec = 2
is the default case of test_gpu_parity.py); weights are damped (encoder output projections x0.1)
so that drafts are accepted in part. For each split:

* every round, teacher-forced from the oracle's decode, has draft and verify logits within 1e-4
  of the oracle, and matching drafts / n_accept / bonus where the oracle's top-2 gap allows;
* the speculative decode (k=4) equals plain greedy decoding (k=0) bit for bit;
* n_dec = l (no encoder): the drafter is the verifier, so every round accepts all k drafts;
* n_dec = 0: the drafter is the LM head on the normalised raw embedding, and the draft logits
  equal that closed form computed by the oracle.
"""
import numpy as np
import pytest

from gpu_common import check_round, decoder, first_ambiguous, oracle_model, say
from oracle import model as om
from oracle import seed as os_
from paper_2609_36590_amd import synth

pytestmark = pytest.mark.gpu

K = 4
TOL = 1e-4


@pytest.fixture(scope="module", params=[0, 1, 3, 4], ids=lambda n: f"n_dec={n}")
def split(request):
    n_dec = request.param
    cfg = synth.C1_TINY.replace(name=f"tiny-4L-h256-dec{n_dec}", n_dec_layers=n_dec)
    w = synth.make_weights(cfg, seed=0, enc_out_scale=0.1)
    prompt = synth.make_prompts(cfg)[0]
    m = oracle_model(cfg, w)
    toks, rounds = os_.generate(m, prompt, K, cfg.gen_len, record=True)
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + cfg.gen_len + 2 * K + 2, max_draft=K)
    yield dict(n_dec=n_dec, cfg=cfg, w=w, m=m, prompt=prompt, toks=toks, rounds=rounds, dec=dec)
    dec.close()


def test_rounds_match_oracle(split):
    worst_d = worst_v = 0.0
    for rd in split["rounds"][:8]:
        dmax, vmax = check_round(split["dec"], split["prompt"], split["toks"], rd, TOL, K)
        worst_d, worst_v = max(worst_d, dmax), max(worst_v, vmax)
    say(f"[gpu] n_dec={split['n_dec']}: max |draft - oracle| = {worst_d:.3g}, max |verify - oracle| = {worst_v:.3g}")
    assert worst_d <= TOL and worst_v <= TOL


def test_speculative_equals_greedy_and_oracle(split):
    cfg, rounds = split["cfg"], split["rounds"]
    dec = split["dec"]
    g0, _, _ = dec.generate([split["prompt"]], 0, cfg.gen_len)
    g4, cnt, st = dec.generate([split["prompt"]], K, cfg.gen_len, log_cap=4 * cfg.gen_len)
    assert cnt[0] == cfg.gen_len
    np.testing.assert_array_equal(g4, g0)
    n_ok = first_ambiguous(rounds, TOL)
    upto = (rounds[n_ok].p + 1 - len(split["prompt"])) if n_ok < len(rounds) else cfg.gen_len
    np.testing.assert_array_equal(g4[0, :upto], split["toks"][:upto])
    log = st["n_accept_log"][:, 0]
    for i in range(n_ok):
        assert log[i] == rounds[i].n_accept, (i, log[i], rounds[i].n_accept)
    say(f"[gpu] n_dec={split['n_dec']}: mean accepted {st['accepted'] / st['rounds']:.2f} of {K}")
    if split["n_dec"] == cfg.n_layers:
        # the drafter runs the whole model: every draft is the verifier's own greedy token
        assert st["accepted"] == K * st["rounds"]


def test_no_decoder_layers_drafts_from_the_embedding(split):
    if split["n_dec"] != 0:
        pytest.skip("closed form only for n_dec = 0")
    cfg, m = split["cfg"], split["m"]
    dec = split["dec"]
    dec.prefill([split["prompt"]])
    d, qlog = dec.draft(K, logits=True)
    # draft[0] is the pending last prompt token; step i feeds draft[i-1] and no layer runs
    prev = [split["prompt"][-1]] + list(d[0, :-1])
    E = m.w["embed"].astype(np.float64)
    g = m.w["final_norm"].astype(np.float64)
    for i, x in enumerate(prev):
        h = E[x]
        a = h / np.sqrt(np.mean(h * h) + cfg.rms_eps) * g
        want = E @ a
        assert np.abs(qlog[0, i] - want).max() <= TOL
        assert d[0, i] == int(np.argmax(want))


@pytest.mark.slow
@pytest.mark.timeout(900)
@pytest.mark.parametrize("n_dec", [1, 4, 8], ids=lambda n: f"28L-n_dec={n}")
def test_split_first_round_at_full_size(n_dec):
    """The 28-layer bf16 model (512-token prompt) at other splits of the sweep: the first round's
    draft and verify logits within 2e-2 of the oracle (teacher-forced drafts), and the speculative
    decode equal to plain greedy decoding bit for bit."""
    tol = 2e-2
    cfg = synth.C2_28L.replace(name=f"28L-h2048-dec{n_dec}", n_dec_layers=n_dec)
    w = synth.make_weights(cfg, seed=0)
    prompt = synth.make_prompts(cfg)[0]
    dec = decoder(cfg, w, max_batch=1, max_ctx=len(prompt) + 24 + 2 * K + 2, max_draft=K)
    try:
        dec.prefill([prompt])
        d, qlog = dec.draft(K, logits=True)
        say(f"[gpu] oracle prefill {cfg.name}")
        st = os_.prefill(oracle_model(cfg, w), prompt, len(prompt) + K + 2)
        drafts, ref_q = os_.draft(st, K)
        ref_v = os_.verify(st, drafts)
        same = 1
        while same < K and np.array_equal(d[0, :same], drafts[1:same + 1]):
            same += 1
        derr = float(np.abs(qlog[0, :same] - ref_q[:same]).max())
        dec.prefill([prompt])
        _, _, vlog = dec.verify(K, drafts=np.asarray(drafts[1:], dtype=np.int32)[None], logits=True)
        verr = float(np.abs(vlog[0] - ref_v).max())
        say(f"[gpu] {cfg.name}: max |draft - oracle| = {derr:.3g}, max |verify - oracle| = {verr:.3g}")
        assert derr <= tol and verr <= tol
        out4, _, _ = dec.generate([prompt], K, 24, use_graph=True)
        out0, _, _ = dec.generate([prompt], 0, 24, use_graph=True)
        np.testing.assert_array_equal(out4, out0)
    finally:
        dec.close()
