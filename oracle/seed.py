"""Algorithm 2 (SEED inference with fixed draft length), brute-force greedy decoding, the
parallel block-mask drafter pass, and the forward pass of the speculative drafting objective
(Algorithm 1, L_spec), in plain NumPy.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``): never imported by the HIP path.

Positions are 0-based. After any commit the sequence X[0..t-1] is committed, the cache holds
deep keys/values for positions 0..t-2 in every layer, and X[t-1] (position p = t-1) is the
pending token whose keys/values are not cached yet.

Readings (where the paper is silent or ambiguous):
* Initialisation (Alg. 2): f runs over the whole prompt, then the cache is truncated to t-1
  positions before the first draft, because the first draft step conditions on KV_{1:t-1}
  only. The first new token is therefore emitted by the first verification.
* The drafter (Sec. 3.1, Eq. 5) reads the decoder layers' own cache (layers l'..l-1): deep
  entries written by the previous verification for positions < p, plus the shallow entries it
  wrote itself at positions p.. during this drafting phase (the index range of Alg. 2's draft
  step covers them).
* Greedy argmax ties go to the lowest token id (``numpy.argmax``).
* The last round still drafts d tokens; the output is cut to T tokens.
* EOS (optional): generation of a sequence stops right after it emits ``eos``.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .model import KVCache, full_forward, run_layers


@dataclasses.dataclass
class Round:
    """Everything one draft-verify round of Algorithm 2 produced."""

    p: int                   # position of the pending token X[t-1]
    drafts: np.ndarray       # X_draft[0..d]   (X_draft[0] = pending token)
    draft_logits: np.ndarray  # q_1..q_d        [d, V]
    verify_logits: np.ndarray  # p_1..p_{d+1}   [d+1, V]
    n_accept: int
    bonus: int


class State:
    """Decode state of one sequence: committed tokens X[0..t-1] and the cache."""

    def __init__(self, model, prompt, capacity):
        self.model = model
        self.tokens = [int(x) for x in prompt]
        self.cache = KVCache(model.cfg, capacity, model.dtype)

    @property
    def t(self):
        return len(self.tokens)

    @property
    def p(self):
        return self.t - 1


def prefill(model, prompt, capacity, row_block=None):
    """Initialise KV_{1:t} with (f_dec o f_enc)(X_{1:t}), then keep positions [0, t-1) (Alg. 2).

    With ``row_block`` the prompt's rows go through the layers ``row_block`` rows at a time (each
    block after the earlier blocks filled the cache): every row still attends to exactly the
    positions up to its own, so the cache is the same; only the memory of the score matrices is
    bounded (a 16384-token prompt)."""
    st = State(model, prompt, capacity)
    n = len(st.tokens)
    step = n if row_block is None else row_block
    for s in range(0, n, step):
        h = model.embed(st.tokens[s:s + step])
        run_layers(model, st.cache, range(model.n_layers), h, s)
    st.cache.truncate(st.t - 1)
    return st


def draft(st, d):
    """Drafting phase of Alg. 2: d autoregressive steps of the decoder only.

    Step i feeds the raw embedding W_in X_draft[i-1] (Eq. 5) through layers l'..l-1 at position
    p+i-1, attending to that layer's cache, and takes the argmax. Returns (drafts[0..d],
    draft logits [d, V]).
    """
    m = st.model
    dec = range(m.first_decoder_layer, m.n_layers)
    drafts = [st.tokens[-1]]
    logits = []
    for i in range(1, d + 1):
        h = m.embed([drafts[i - 1]])
        h = run_layers(m, st.cache, dec, h, st.p + i - 1)
        q = m.head(h)[0]
        logits.append(q)
        drafts.append(int(np.argmax(q)))
    V = m.cfg.vocab
    return np.array(drafts, dtype=np.int64), (np.stack(logits) if logits else np.zeros((0, V), m.dtype))


def verify(st, drafts):
    """Verification phase of Alg. 2: truncate to t-1, then one full pass over X_draft[0..d].

    Row r sits at position p+r and attends to positions 0..p+r. Returns logits p_1..p_{d+1}.
    """
    m = st.model
    st.cache.truncate(st.t - 1)
    h = m.embed(drafts)
    h = run_layers(m, st.cache, range(m.n_layers), h, st.p)
    return m.head(h)


def accept(drafts, verify_logits):
    """Greedy acceptance of Alg. 2: the longest prefix with argmax p_i = X_draft[i], then the
    bonus token argmax p_{n_accept+1}."""
    d = len(drafts) - 1
    n = 0
    for i in range(1, d + 1):
        if int(np.argmax(verify_logits[i - 1])) == int(drafts[i]):
            n += 1
        else:
            break
    return n, int(np.argmax(verify_logits[n]))


def commit(st, drafts, n_accept, bonus):
    """Append X_draft[1..n_accept] and the bonus token; truncate the cache to t+n_accept
    positions (1-based), i.e. keep the deep KV of every committed token but the new pending one."""
    st.tokens.extend(int(x) for x in drafts[1:n_accept + 1])
    st.tokens.append(int(bonus))
    st.cache.truncate(st.t - 1)


def generate(model, prompt, d, max_new, eos=None, record=False, capacity=None):
    """Algorithm 2 end to end: returns (new tokens [max_new or fewer], list of Round)."""
    t0 = len(prompt)
    T = t0 + max_new
    if capacity is None:
        capacity = T + d + 1
    st = prefill(model, prompt, capacity)
    rounds = []
    while st.t < T:
        drafts, qlog = draft(st, d)
        plog = verify(st, drafts)
        n_acc, bonus = accept(drafts, plog)
        if record:
            rounds.append(Round(st.p, drafts, qlog, plog, n_acc, bonus))
        before = st.t
        commit(st, drafts, n_acc, bonus)
        if eos is not None:
            new = st.tokens[before:]
            if eos in new:
                del st.tokens[before + new.index(eos) + 1:]
                break
    return np.array(st.tokens[t0:T], dtype=np.int64), rounds


def greedy_brute_force(model, prompt, max_new, eos=None):
    """Non-speculative greedy decoding by full recomputation (no cache): X[s+1] = argmax f(X[0..s])."""
    toks = [int(x) for x in prompt]
    for _ in range(max_new):
        nxt = int(np.argmax(full_forward(model, toks)[-1]))
        toks.append(nxt)
        if eos is not None and nxt == eos:
            break
    return np.array(toks[len(prompt):], dtype=np.int64)


def greedy_cached(model, prompt, max_new, capacity=None):
    """Plain greedy decoding with the cache: prefill, then one single-row pass per token.

    Equivalent to Algorithm 2 with d = 0 (verify only the pending token, accept nothing, emit
    the bonus token)."""
    toks, _ = generate(model, prompt, 0, max_new, capacity=capacity)
    return toks


def block_draft_logits(model, context, draft_inputs):
    """Draft logits from the parallel block-mask formulation of the drafter (Sec. 3.2).

    ``context`` = X[0..p] (the last one is the pending token at the block start n' = p) and
    ``draft_inputs`` = X_draft[1..d-1]. The decoder layers run once, in parallel, over the raw
    embeddings H^0 of [X[p], X_draft[1..d-1]] at positions p..p+d-1, with causal attention inside
    the block and attention to the deep decoder keys/values KV^dec_{<p} of a full pass over
    X[0..p-1] (the conditioning of L_spec, Eq. 7). Returns q_1..q_d [d, V].
    """
    c = model.cfg
    context = [int(x) for x in context]
    p = len(context) - 1
    _, Ks, Vs = full_forward(model, context[:p], return_kv=True) if p > 0 else (
        None,
        np.zeros((c.n_layers, 0, c.n_kv_heads, c.head_dim), model.dtype),
        np.zeros((c.n_layers, 0, c.n_kv_heads, c.head_dim), model.dtype),
    )
    block = [context[p]] + [int(x) for x in draft_inputs]
    h = model.embed(block)
    pos = np.arange(p, p + len(block))
    for i in range(model.first_decoder_layer, c.n_layers):
        h, _, _ = model.block(i, h, pos, Ks[i], Vs[i])
    return model.head(h)


def spec_forward(model, tokens, b):
    """Forward pass of the speculative drafting objective L_spec of Algorithm 1.

    For every input position q = 0..n-2 (the drafter predicts X[q+1]) the block start is
    s = floor(q / b) * b (0-based form of Algorithm 1's n'). The decoder layers run over the raw
    embeddings H^0 of X[s..q] (causal inside the block) and attend to the deep decoder keys /
    values KV^dec of positions < s, which come from one full pass of f over the whole sequence.
    Written as Algorithm 1's loop over blocks, one block at a time; the GPU computes all blocks
    in one pass with the block-causal mask of Fig. 2 (right).

    Returns (logits [n-1, V], L_spec = sum over q of -log softmax(logits[q])[X[q+1]]).
    """
    c = model.cfg
    tokens = [int(x) for x in tokens]
    n = len(tokens)
    assert n >= 2 and b >= 1
    _, Ks, Vs = full_forward(model, tokens, return_kv=True)
    logits = np.zeros((n - 1, c.vocab), dtype=model.dtype)
    for s in range(0, n - 1, b):
        e = min(s + b, n - 1)                      # inputs X[s..e-1] predict X[s+1..e]
        h = model.embed(tokens[s:e])
        pos = np.arange(s, e)
        for i in range(model.first_decoder_layer, c.n_layers):
            h, _, _ = model.block(i, h, pos, Ks[i][:s], Vs[i][:s])
        logits[s:e] = model.head(h)
    z = logits.astype(np.float64)
    zmax = z.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(z - zmax).sum(axis=1))
    nll = lse - z[np.arange(n - 1), np.asarray(tokens[1:], dtype=np.int64)]
    return logits, float(nll.sum())
