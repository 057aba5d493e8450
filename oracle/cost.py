"""The parameter-count cost model of Appendix E (Computational Cost Analysis).

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

Cost of a pass = number of weights it touches, in units of one full forward pass. Per layer:
attention W_Q, W_K, W_V, W_O plus a 3-matrix MLP (norm gains are not counted); the tied
embedding / LM head counts once. A round of fixed-length drafting costs
T_unit = d * c_draft + c_verify and commits n = d * r + 1 tokens, so the predicted throughput is
1000 / (T_unit * unit_ms) * n tokens/s.
"""
from __future__ import annotations


def attention_params(cfg):
    H = cfg.hidden
    return H * cfg.q_dim + 2 * H * cfg.kv_dim + cfg.q_dim * H


def mlp_params(cfg):
    return 3 * cfg.hidden * cfg.ffn


def layer_params(cfg):
    return attention_params(cfg) + mlp_params(cfg)


def embedding_params(cfg):
    return cfg.vocab * cfg.hidden


def full_params(cfg):
    return cfg.n_layers * layer_params(cfg) + embedding_params(cfg)


def draft_weights(cfg, n_dec=None):
    """Weights touched per SEED draft token: the decoder layers plus the head (Table 9)."""
    n_dec = cfg.n_dec_layers if n_dec is None else n_dec
    return n_dec * layer_params(cfg) + embedding_params(cfg)


def draft_cost(cfg, n_dec=None):
    """c_draft in units of one full pass."""
    return draft_weights(cfg, n_dec) / full_params(cfg)


def round_cost(d, c_draft, c_verify=1.0):
    """T_unit = d * c_draft + c_verify."""
    return d * c_draft + c_verify


def tokens_per_round(d, r):
    """n = d * r + 1 (accepted drafts plus the bonus token)."""
    return d * r + 1


def predicted_throughput(t_ms, n):
    """Predicted tokens/s = 1000 / T_ms * n."""
    return 1000.0 / t_ms * n
