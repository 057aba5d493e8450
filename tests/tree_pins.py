"""Independent recomputation of the confidence-aware drafting decisions (appendix,
"Confidence-Aware Dynamic Drafting"): from a tree's recorded per-step drafter logits, the top-1
probability p0 (a float64 torch softmax), the fan-out from the top-p table, the ranked candidates
(a stable descending torch sort, so the lower token id wins a tie) and the stop rule (the first
step whose p0 is below tau, else max_depth). Shares no code with oracle/tree.py."""
import torch


def expected_steps(draft_logits, tau, max_depth, table, rest):
    """(p0 per step, candidate ids per step) the rule yields from the recorded logits."""
    p0s, steps = [], []
    for z in draft_logits[:max_depth]:
        zt = torch.as_tensor(z, dtype=torch.float64)
        prob = torch.softmax(zt, dim=0)
        ids = torch.sort(-zt, stable=True).indices
        p0 = float(prob[ids[0]])
        k = rest
        for thr, kk in table:
            if p0 > thr:
                k = kk
                break
        p0s.append(p0)
        steps.append([int(x) for x in ids[:k]])
        if p0 < tau:
            break
    return p0s, steps


def check_drafting_steps(tree, tau, max_depth, table, rest):
    """The oracle's tree against the independent recomputation: step count (stop rule), p0,
    fan-out and the ranked candidates of every step (the chain node first, then its siblings)."""
    p0s, steps = expected_steps(tree.draft_logits, tau, max_depth, table, rest)
    assert len(tree.p0) == len(steps), (len(tree.p0), len(steps))
    for d, (p0, cands) in enumerate(zip(p0s, steps), 1):
        assert abs(tree.p0[d - 1] - p0) <= 1e-12 * max(1.0, p0), (d, tree.p0[d - 1], p0)
        at_depth = [tree.tokens[i] for i in range(len(tree.tokens)) if tree.depths[i] == d]
        assert at_depth == cands, (d, at_depth, cands)
    return [len(c) for c in steps]
