"""Confidence-aware dynamic drafting with tree-based verification, the decoding mode of the
paper's main experiments (Method, "Adaptive Drafting with Tree-Based Verification"; appendix
paragraphs "Confidence-Aware Dynamic Drafting" and "Tree-Based Verification"; Fig. 3), in plain
NumPy.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``): never imported by the HIP path.

Readings (where the paper leaves the procedure open):
* Tree shape: each drafting step expands the current node into k candidates, the k tokens of
  highest drafter probability (ties to the lower token id), with k from the appendix's top-p
  table of the top-1 probability p0 (k = 1 if p0 > 0.95, 3 if 0.8 < p0 <= 0.95, 5 if
  0.5 < p0 <= 0.8, else 10). Only the top-1 candidate becomes the next current node and is drafted
  further; the other candidates are leaves.
* Stop rule: drafting stops after a step whose top-1 probability is below tau (that step's
  candidates are still verified), and after max_depth steps.
* Node budget: the paper sets none, so by default a tree is unbounded. A caller comparing with an
  implementation that verifies at most N rows in one pass passes max_nodes = N: a tree then holds
  at most N nodes, root included, a step's fan-out is cut to the nodes left and drafting stops
  once none are left.
* Packing: node 0 is the pending token X[p] (the root), then the top-1 chain in depth order, then
  the other candidates by depth and rank. Node i sits at rotary position p + depth(i).
* Verification: one full-model pass over the packed nodes; node i attends to the committed prefix
  (positions < p) and to the nodes on its own path from the root (itself included).
* Acceptance: starting at the root, move to the child whose token equals the verifier's argmax at
  the current node while one exists; the bonus token is the verifier's argmax at the last node
  reached. Commit: the accepted nodes' keys/values become the cache entries of positions
  p+1.., the root's that of p (the cache is truncated to the accepted path).
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .model import apply_rope, rmsnorm, rope_cos_sin, round_to_bf16, run_layers, silu
from .seed import prefill

# (threshold, k): k for the first threshold that p0 exceeds; FANOUT_REST below all of them
FANOUT = ((0.95, 1), (0.8, 3), (0.5, 5))
FANOUT_REST = 10


def fanout(p0, table=FANOUT, rest=FANOUT_REST):
    """Number of sibling candidates for top-1 probability p0 (the appendix's top-p rule)."""
    for thr, k in table:
        if p0 > thr:
            return k
    return rest


@dataclasses.dataclass
class Tree:
    tokens: list          # node tokens, node 0 = the root (pending token)
    parents: list         # parent node index, -1 for the root
    depths: list          # depth (root 0); rotary position p + depth
    p0: list              # top-1 drafter probability of each drafting step
    draft_logits: np.ndarray   # [steps, V]

    def path(self, i):
        """Node indices from the root to node i (both included)."""
        out = []
        while i >= 0:
            out.append(i)
            i = self.parents[i]
        return out[::-1]


def _ranked(logits):
    """Token ids by decreasing logit, ties to the lower id."""
    z = np.asarray(logits, dtype=np.float64)
    return np.lexsort((np.arange(len(z)), -z))


def _confidence(logits):
    """Top-1 probability p0 of one drafting step's logits (softmax in float64) and the token ids
    ranked by decreasing logit (ties to the lower id)."""
    z = np.asarray(logits, dtype=np.float64)
    pr = np.exp(z - z.max())
    pr /= pr.sum()
    order = _ranked(z)
    return float(pr[order[0]]), order


def draft_tree(st, tau, max_depth, table=FANOUT, rest=FANOUT_REST, max_nodes=None):
    """Dynamic drafting: decoder-only steps from the pending token (Eq. 5, as in Algorithm 2),
    each expanded into top-p candidates; stops by the confidence threshold tau or at max_depth
    (or, when max_nodes is given, once the tree holds max_nodes nodes)."""
    m = st.model
    dec = range(m.first_decoder_layer, m.n_layers)
    chain = [st.tokens[-1]]
    steps, p0s, logits = [], [], []
    nodes = 1
    for i in range(1, max_depth + 1):
        h = m.embed([chain[i - 1]])
        h = run_layers(m, st.cache, dec, h, st.p + i - 1)
        q = m.head(h)[0]
        p0, order = _confidence(q)
        k = fanout(p0, table, rest)
        if max_nodes is not None:
            k = min(k, max_nodes - nodes)
        cands = [int(x) for x in order[:k]]
        nodes += len(cands)
        steps.append(cands)
        p0s.append(p0)
        logits.append(q)
        chain.append(cands[0])
        if p0 < tau or (max_nodes is not None and nodes >= max_nodes):
            break
    tokens, parents, depths, chain_nodes = [chain[0]], [-1], [0], [0]
    for d, cands in enumerate(steps, 1):
        tokens.append(cands[0])
        parents.append(chain_nodes[-1])
        depths.append(d)
        chain_nodes.append(len(tokens) - 1)
    for d, cands in enumerate(steps, 1):
        for c in cands[1:]:
            tokens.append(c)
            parents.append(chain_nodes[d - 1])
            depths.append(d)
    V = m.cfg.vocab
    return Tree(tokens, parents, depths, p0s, np.stack(logits) if logits else np.zeros((0, V), m.dtype))


def _ancestor_mask(tree):
    n = len(tree.tokens)
    anc = np.zeros((n, n), dtype=bool)
    for i in range(n):
        anc[i, tree.path(i)] = True
    return anc


def _tree_block(model, i, h, pos, K_prefix, V_prefix, anc):
    """Layer f_i on the packed tree rows: like Model.block, but each row attends to the whole
    prefix and to its ancestor-or-self rows only (Tree-Based Verification)."""
    c = model.cfg
    W = model.w
    p = f"layers.{i}."
    n = h.shape[0]
    a = rmsnorm(h, W[p + "attn_norm"], c.rms_eps)
    q = (a @ W[p + "wq"].T).reshape(n, c.n_heads, c.head_dim)
    k = (a @ W[p + "wk"].T).reshape(n, c.n_kv_heads, c.head_dim)
    v = (a @ W[p + "wv"].T).reshape(n, c.n_kv_heads, c.head_dim)
    cos, sin = rope_cos_sin(pos, c.head_dim, c.rope_base)
    q = apply_rope(q, cos, sin)
    k = apply_rope(k, cos, sin)
    if model.kv_bf16:
        k, v = round_to_bf16(k), round_to_bf16(v)
    K = np.concatenate([K_prefix, k], axis=0)
    V = np.concatenate([V_prefix, v], axis=0)
    L = K.shape[0]
    allowed = np.concatenate([np.ones((n, L - n), dtype=bool), anc], axis=1)      # [n, L]
    rep = c.n_heads // c.n_kv_heads
    Kh = np.repeat(K, rep, axis=1).transpose(1, 2, 0)
    Vh = np.repeat(V, rep, axis=1).transpose(1, 0, 2)
    s = np.matmul(q.transpose(1, 0, 2), Kh) / np.sqrt(c.head_dim).astype(q.dtype)
    s = np.where(allowed[None], s, -np.inf)
    s = s - s.max(axis=-1, keepdims=True)
    pr = np.exp(s)
    pr = pr / pr.sum(axis=-1, keepdims=True)
    o = np.matmul(pr, Vh).transpose(1, 0, 2)
    h = h + o.reshape(n, c.n_heads * c.head_dim) @ W[p + "wo"].T
    mm = rmsnorm(h, W[p + "mlp_norm"], c.rms_eps)
    h = h + (silu(mm @ W[p + "w_gate"].T) * (mm @ W[p + "w_up"].T)) @ W[p + "w_down"].T
    return h, k, v


def verify_tree(st, tree):
    """Tree-based verification: truncate to the committed prefix, one full-model pass over the
    packed nodes with the tree attention mask. Returns (logits [n, V], per-layer (k, v) of the
    nodes)."""
    m = st.model
    st.cache.truncate(st.t - 1)
    h = m.embed(tree.tokens)
    pos = st.p + np.asarray(tree.depths, dtype=np.int64)
    anc = _ancestor_mask(tree)
    kv = []
    for i in range(m.n_layers):
        Kp, Vp = st.cache.prefix(i, st.p)
        h, k, v = _tree_block(m, i, h, pos, Kp, Vp, anc)
        kv.append((k, v))
    return m.head(h), kv


def accept_tree(tree, logits):
    """Longest accepted path from the root and the bonus token. Returns (path nodes without the
    root, bonus)."""
    n = len(tree.tokens)
    node, path = 0, []
    while True:
        g = int(np.argmax(logits[node]))
        nxt = next((c for c in range(n) if tree.parents[c] == node and tree.tokens[c] == g), None)
        if nxt is None:
            break
        path.append(nxt)
        node = nxt
    return path, int(np.argmax(logits[node]))


def commit_tree(st, tree, kv, path, bonus):
    """Append the accepted tokens and the bonus token; the cache keeps the root's and the
    accepted nodes' keys/values at positions p, p+1, .., p+len(path)."""
    rows = [0] + list(path)
    for i, (k, v) in enumerate(kv):
        st.cache.append(i, st.p, k[rows], v[rows])
    st.tokens.extend(int(tree.tokens[j]) for j in path)
    st.tokens.append(int(bonus))
    st.cache.truncate(st.t - 1)


@dataclasses.dataclass
class TreeRound:
    p: int
    tree: Tree
    verify_logits: np.ndarray
    path: list
    bonus: int


def generate_tree(model, prompt, tau, max_depth, max_new, table=FANOUT, rest=FANOUT_REST, record=False,
                  capacity=None, max_nodes=None):
    """Dynamic drafting with tree verification end to end: returns (new tokens, rounds)."""
    t0 = len(prompt)
    most = 1 + max_depth * max([k for _, k in table] + [rest])   # nodes of one unbounded tree
    cap = capacity or (t0 + max_new + (most if max_nodes is None else min(most, max_nodes)) + 2)
    st = prefill(model, [int(x) for x in prompt], cap)
    rounds = []
    while st.t - t0 < max_new:
        tree = draft_tree(st, tau, max_depth, table, rest, max_nodes)
        logits, kv = verify_tree(st, tree)
        path, bonus = accept_tree(tree, logits)
        if record:
            rounds.append(TreeRound(st.p, tree, logits, path, bonus))
        commit_tree(st, tree, kv, path, bonus)
    return np.array(st.tokens[t0:t0 + max_new], dtype=np.int64), rounds
