"""GPU tests of the runtime around the kernels: batches with ragged prompts and acceptance,
graph replay, forced acceptance, EOS, long contexts that span several attention groups, the
step-wise calls, and the error paths of the C ABI (state is left unchanged after an error)."""
import numpy as np
import pytest

from gpu_common import compare_kv, decoder, first_ambiguous, oracle_model, say, top2_gap
from oracle import model as om
from oracle import seed as os_
from paper_2609_36590_amd import binding, synth

pytestmark = pytest.mark.gpu

BF16_TINY = synth.C1_TINY.replace(name="tiny-bf16", dtype=synth.BF16)


@pytest.fixture(scope="module")
def batch_dec():
    cfg = BF16_TINY
    w = synth.make_weights(cfg, seed=3, enc_out_scale=0.1)
    dec = decoder(cfg, w, max_batch=4, max_ctx=600, max_draft=6)
    yield cfg, w, dec
    dec.close()


def _prompts(cfg, lens, seed=7):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, cfg.vocab, size=n).astype(np.int32) for n in lens]


def test_batch_equals_each_sequence_alone(batch_dec):
    cfg, w, dec = batch_dec
    prompts = _prompts(cfg, [5, 70, 33, 300])
    say("[gpu] batch of 4 ragged prompts vs alone")
    out_b, cnt_b, st = dec.generate(prompts, 4, 48, log_cap=64)
    assert (cnt_b == 48).all()
    log = st["n_accept_log"]
    assert len({int(x) for x in log[log >= 0]}) >= 2, "acceptance should vary across rounds"
    for i, p in enumerate(prompts):
        out_1, _, _ = dec.generate([p], 4, 48)
        np.testing.assert_array_equal(out_b[i], out_1[0])
        out_g, _, _ = dec.generate([p], 0, 48)
        np.testing.assert_array_equal(out_b[i], out_g[0])


def test_graph_replay_equals_eager(batch_dec):
    cfg, w, dec = batch_dec
    prompts = _prompts(cfg, [40, 9], seed=8)
    say("[gpu] graph vs eager")
    a, _, sa = dec.generate(prompts, 3, 40, use_graph=False, log_cap=64)
    b, _, sb = dec.generate(prompts, 3, 40, use_graph=True, log_cap=64)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(sa["n_accept_log"], sb["n_accept_log"])


@pytest.mark.parametrize("a", [0, 1, 2, 3, 4])
def test_forced_acceptance(batch_dec, a):
    cfg, w, dec = batch_dec
    prompts = _prompts(cfg, [30, 12], seed=9)
    trace, _, _ = dec.generate(prompts, 0, 40)
    say(f"[gpu] forced acceptance a={a}")
    out, cnt, st = dec.generate(prompts, 4, 40, sim_accept=a, forced_trace=trace, log_cap=64)
    np.testing.assert_array_equal(out, trace)
    log = st["n_accept_log"]
    for b in range(2):
        live = log[:, b][log[:, b] >= 0]
        # every round that ends inside the trace accepts exactly a drafts
        assert (live[:-1] == a).all(), (a, live)
    assert st["rounds"] == -(-40 // (a + 1))


def test_eos_stops_each_sequence(batch_dec):
    cfg, w, dec = batch_dec
    prompts = _prompts(cfg, [20, 25], seed=10)
    ref, _, _ = dec.generate(prompts, 0, 30)
    eos = int(ref[0, 6])
    out, cnt, _ = dec.generate(prompts, 4, 30, eos_id=eos)
    for b in range(2):
        hits = np.nonzero(ref[b] == eos)[0]
        n = hits[0] + 1 if len(hits) else 30
        assert cnt[b] == n
        np.testing.assert_array_equal(out[b, :n], ref[b, :n])
        assert (out[b, n:] == -1).all()


def test_rounds_and_stepwise_calls_agree_with_generate(batch_dec):
    cfg, w, dec = batch_dec
    prompts = _prompts(cfg, [17, 64], seed=11)
    ref, _, _ = dec.generate(prompts, 0, 60)
    dec.prefill(prompts)
    binding.seed_rounds(dec.ctx, 4, 6, True)
    for b in range(2):
        toks = dec.tokens(b)
        n = len(toks) - len(prompts[b])
        assert n >= 6
        np.testing.assert_array_equal(toks[len(prompts[b]):], ref[b, :n])
    # the step-wise calls: draft, then verify the device drafts
    dec.prefill(prompts)
    total = [0, 0]
    for _ in range(5):
        d, _ = dec.draft(3)
        na, bo, _ = dec.verify(3)
        for b in range(2):
            total[b] += na[b] + 1
    for b in range(2):
        toks = dec.tokens(b)
        np.testing.assert_array_equal(toks[len(prompts[b]):], ref[b, :total[b]])


@pytest.mark.parametrize("B,k", [(4, 15), (64, 0)], ids=["4x16-rows", "64x1-rows"])
def test_maximum_rows_per_pass(B, k):
    """Passes of the maximum 64 rows (max_batch * (max_draft + 1)): 4 sequences drafting 15 tokens,
    and 64 sequences of plain greedy decoding, each against its own decode alone."""
    cfg = BF16_TINY
    w = synth.make_weights(cfg, seed=3, enc_out_scale=0.1)
    dec = decoder(cfg, w, max_batch=B, max_ctx=160, max_draft=k)
    try:
        rng = np.random.default_rng(12)
        prompts = _prompts(cfg, [int(x) for x in rng.integers(1, 100, size=B)], seed=13)
        say(f"[gpu] {B} sequences, k={k}: {B * (k + 1)} rows per verification")
        out, cnt, st = dec.generate(prompts, k, 24, log_cap=64)
        assert (cnt == 24).all()
        if k:
            log = st["n_accept_log"]
            assert log[log >= 0].max() >= 2, "some rounds should accept several drafts"
        for b in ([0, 1, 2, 3] if B == 4 else [0, 17, 40, 63]):
            alone, _, _ = dec.generate([prompts[b]], 0, 24)
            np.testing.assert_array_equal(out[b], alone[0])
    finally:
        dec.close()


def test_long_context_spans_several_attention_groups():
    """A 700-token context crosses two 256-position group boundaries (cross-group merge)."""
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=4)
    prompt = _prompts(cfg, [700], seed=12)[0]
    m = oracle_model(cfg, w)
    st = os_.prefill(m, prompt, 760)
    drafts, qlog = os_.draft(st, 4)
    vlog = os_.verify(st, drafts)
    dec = decoder(cfg, w, max_batch=1, max_ctx=760, max_draft=4)
    try:
        dec.prefill([prompt])
        d, q = dec.draft(4, logits=True)
        _, _, v = dec.verify(4, drafts=drafts[1:][None].astype(np.int32), logits=True)
        err_q = np.abs(q[0, 0] - qlog[0]).max()
        err_v = np.abs(v[0] - vlog).max()
        say(f"[gpu] long context: draft err {err_q:.2e}, verify err {err_v:.2e}")
        assert err_q <= 1e-4 and err_v <= 1e-4
        g0, _, _ = dec.generate([prompt], 0, 24)
        g4, _, _ = dec.generate([prompt], 4, 24)
        np.testing.assert_array_equal(g0, g4)
        ref, _ = os_.generate(m, prompt, 4, 24)
        gap_ok = all(top2_gap(vlog) > 2e-4)
        if gap_ok:
            assert g4[0, 0] == ref[0]
    finally:
        dec.close()


@pytest.mark.parametrize("cfg", [synth.C1_TINY, BF16_TINY], ids=["fp32", "bf16"])
def test_cache_contents_match_oracle(cfg):
    """After prefill, a draft and a verification of the oracle's drafts, every layer's cached keys
    and values of every position 0..p+k (the deep entries verification wrote over the drafts'
    shallow ones included) equal those of the oracle's full forward over the same tokens; the
    sequences are ragged and batched, so their blocks interleave in the paged pool."""
    k = 4
    w = synth.make_weights(cfg, seed=6)
    m = oracle_model(cfg, w)
    prompts = _prompts(cfg, [37, 70, 21], seed=14)
    dec = decoder(cfg, w, max_batch=3, max_ctx=100, max_draft=k)
    try:
        dec.prefill(prompts)
        d, _ = dec.draft(k)
        dec.verify(k)
        for b, pr in enumerate(prompts):
            toks = np.concatenate([pr, d[b]])
            _, Ks, Vs = om.full_forward(m, toks, return_kv=True)
            for layer in range(cfg.n_layers):
                kg, vg = dec.read_kv(b, layer, 0, len(toks))
                compare_kv(kg, Ks[layer], cfg.dtype == synth.BF16, what=f"seq {b} layer {layer} keys")
                compare_kv(vg, Vs[layer], cfg.dtype == synth.BF16, what=f"seq {b} layer {layer} values")
        with pytest.raises(binding.SeedError) as e:
            dec.read_kv(0, 0, 0, 1000)
        assert e.value.status == -1
        with pytest.raises(binding.SeedError) as e:
            dec.read_kv(0, cfg.n_layers, 0, 1)
        assert e.value.status == -1
    finally:
        dec.close()


def test_one_token_prompts_and_one_new_token():
    """Degenerate lengths: prompts of 1 and 2 tokens (no cache entry exists before the first
    verification; the first drafts attend only to their own entries) batched with a 17-token one,
    and a single generated token. Speculative decoding equals plain greedy decoding bit for bit,
    and each sequence follows the oracle's Algorithm 2 (logits of the first verification within
    1e-4; tokens up to the first round whose top-2 gap is within twice that)."""
    cfg, k, n = synth.C1_TINY, 4, 12
    w = synth.make_weights(cfg, seed=9)
    m = oracle_model(cfg, w)
    prompts = _prompts(cfg, [1, 2, 17], seed=16)
    dec = decoder(cfg, w, max_batch=3, max_ctx=40, max_draft=k)
    try:
        out, cnt, _ = dec.generate(prompts, k, n)
        greedy, _, _ = dec.generate(prompts, 0, n)
        assert np.all(cnt == n)
        np.testing.assert_array_equal(out, greedy)
        for i, p in enumerate(prompts):
            ref, rounds = os_.generate(m, p, k, n, record=True)
            n_ok = first_ambiguous(rounds, 1e-4)
            upto = (rounds[n_ok].p + 1 - len(p)) if n_ok < len(rounds) else n
            say(f"[gpu] prompt of {len(p)} tokens: {upto} of {n} tokens compared with the oracle")
            np.testing.assert_array_equal(out[i, :upto], ref[:upto])
            rd = rounds[0]
            dec.prefill([p])
            _, _, vlog = dec.verify(k, drafts=np.asarray(rd.drafts[1:], np.int32)[None], logits=True)
            assert float(np.abs(vlog[0] - rd.verify_logits).max()) <= 1e-4
            one, c1, _ = dec.generate([p], k, 1)
            assert c1[0] == 1 and one[0, 0] == greedy[i, 0]
    finally:
        dec.close()


WIDE = synth.C1_TINY.replace(name="wide-4L-h256-f8192", ffn=8192, n_heads=32, n_kv_heads=8, head_dim=128)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16], ids=["fp32", "bf16"])
def test_wide_batch_equals_each_sequence_alone(dtype):
    """A wide FFN (8192): the batch's verification passes (4 x 5 = 20 rows) run gate/up in the
    chunked kernel and the other projections split-K, each sequence alone (5 rows) and plain
    greedy decoding (1 row) the narrow kernels; every sequence's tokens must be identical."""
    cfg = WIDE.replace(dtype=dtype)
    w = synth.make_weights(cfg, seed=8)
    prompts = _prompts(cfg, [30, 19, 41, 26], seed=15)
    dec = decoder(cfg, w, max_batch=4, max_ctx=120, max_draft=4)
    try:
        out, cnt, _ = dec.generate(prompts, 4, 40, use_graph=True)
        assert np.all(cnt == 40)
        for i, p in enumerate(prompts):
            alone, _, _ = dec.generate([p], 4, 40)
            greedy, _, _ = dec.generate([p], 0, 40)
            np.testing.assert_array_equal(out[i], alone[0])
            np.testing.assert_array_equal(out[i], greedy[0])
    finally:
        dec.close()


def test_error_paths_leave_state_unchanged(batch_dec):
    cfg, w, dec = batch_dec
    lib = binding.load_library()
    fresh = decoder(cfg, w, max_batch=2, max_ctx=80, max_draft=4)
    try:
        with pytest.raises(binding.SeedError) as e:
            fresh.draft(2)
        assert e.value.status == -2
        prompts = _prompts(cfg, [10, 20], seed=13)
        with pytest.raises(binding.SeedError) as e:
            fresh.prefill(_prompts(cfg, [5, 5, 5]))
        assert e.value.status == -3
        with pytest.raises(binding.SeedError) as e:
            fresh.prefill([np.array([1, 2, cfg.vocab], np.int32)])
        assert e.value.status == -1
        with pytest.raises(binding.SeedError) as e:
            fresh.prefill([np.zeros(80, np.int32)])
        assert e.value.status == -3
        fresh.prefill(prompts)
        before = [fresh.tokens(b) for b in range(2)]
        with pytest.raises(binding.SeedError) as e:
            fresh.draft(5)
        assert e.value.status == -1
        with pytest.raises(binding.SeedError) as e:
            fresh.verify(3)
        assert e.value.status == -2          # no drafts of length 3 since the last commit
        with pytest.raises(binding.SeedError) as e:
            fresh.verify(2, drafts=np.array([[1, -1], [0, 0]], np.int32))
        assert e.value.status == -1
        with pytest.raises(binding.SeedError) as e:
            binding.seed_rounds(fresh.ctx, 4, 40, False)
        assert e.value.status == -3
        assert lib.seed_last_error()
        for b in range(2):
            np.testing.assert_array_equal(fresh.tokens(b), before[b])
        # still usable, and the result equals a run that never saw the errors
        out, _, _ = fresh.generate(prompts, 2, 20)
        ref, _, _ = dec.generate(prompts, 2, 20)
        np.testing.assert_array_equal(out, ref)
        with pytest.raises(binding.SeedError) as e:
            fresh.generate(prompts, 2, 70)
        assert e.value.status == -3
    finally:
        fresh.close()


def test_rejected_generate_calls_leave_the_state_readable(batch_dec):
    """seed_generate with a forced trace out of range and seed_generate_tree with bad options are
    rejected before the previous decoding state is touched: its tokens stay readable."""
    cfg, w, _ = batch_dec
    dec = decoder(cfg, w, max_batch=2, max_ctx=200, max_draft=4)
    try:
        prompts = _prompts(cfg, [9, 14], seed=21)
        out, _, _ = dec.generate(prompts, 2, 12)
        before = [dec.tokens(b) for b in range(2)]
        bad = np.zeros((2, 12), np.int32)
        bad[1, 5] = cfg.vocab
        with pytest.raises(binding.SeedError) as e:
            dec.generate(prompts, 2, 12, sim_accept=1, forced_trace=bad)
        assert e.value.status == -1
        with pytest.raises(binding.SeedError) as e:
            dec.generate_tree(prompts[0], binding.tree_opts(7), 8)            # max_depth > max_draft
        assert e.value.status == -1
        with pytest.raises(binding.SeedError) as e:
            dec.generate_tree(prompts[0], binding.tree_opts(3, table=((0.5, 1), (0.6, 3))), 8)
        assert e.value.status == -1
        for b in range(2):
            np.testing.assert_array_equal(dec.tokens(b), before[b])
    finally:
        dec.close()


@pytest.mark.parametrize("graph", [False, True], ids=["eager", "graph"])
def test_stats_report_step_latencies(batch_dec, graph):
    """seed_stats carries the medians of the verification and drafting-step latencies stamped by
    the kernels inside the rounds; one round's stamped phases fit inside the call's decode time."""
    cfg, w, dec = batch_dec
    prompts = _prompts(cfg, [40, 33], seed=5)
    _, _, st = dec.generate(prompts, 4, 40, use_graph=graph)
    say(f"[gpu] k=4: rounds {st['rounds']}, verify {st['verify_ms']:.4f} ms, draft step {st['draft_ms']:.4f} ms, "
        f"decode {st['decode_ms']:.3f} ms")
    assert st["verify_ms"] > 0 and st["draft_ms"] > 0
    assert st["verify_ms"] + 4 * st["draft_ms"] <= st["decode_ms"] / st["rounds"] * 1.05
    _, _, st0 = dec.generate(prompts, 0, 20, use_graph=graph)
    assert st0["verify_ms"] > 0 and st0["draft_ms"] == 0
    _, st_t = dec.generate_tree(prompts[0], binding.tree_opts(3), 16, use_graph=graph)
    assert st_t["verify_ms"] > 0 and st_t["draft_ms"] > 0


def test_missing_weights_are_reported():
    cfg = synth.C1_TINY
    w = synth.make_weights(cfg, seed=0)
    dec = binding.Decoder(cfg, max_batch=1, max_ctx=64, max_draft=2)
    try:
        part = {k: v for k, v in w.items() if k != "layers.1.w_up"}
        dec.load_weights(part)
        with pytest.raises(binding.SeedError) as e:
            dec.prefill([np.arange(5, dtype=np.int32)])
        assert e.value.status == -2 and "layers.1.w_up" in str(e.value)
        with pytest.raises(binding.SeedError) as e:
            dec.load_weights({"layers.1.w_up": w["layers.1.w_up"][:, :64]})
        assert e.value.status == -1
        dec.load_weights({"layers.1.w_up": w["layers.1.w_up"]})
        dec.prefill([np.arange(5, dtype=np.int32)])
        # host-side sources take the same path as device sources
        host = binding.Decoder(cfg, max_batch=1, max_ctx=64, max_draft=2)
        host.load_weights(w, on_device=False)
        a, _, _ = dec.generate([np.arange(5, dtype=np.int32)], 2, 10)
        b, _, _ = host.generate([np.arange(5, dtype=np.int32)], 2, 10)
        np.testing.assert_array_equal(a, b)
        host.close()
    finally:
        dec.close()
