"""Writes c5_first_round.npz next to this script: the oracle's first draft-verify round of
Algorithm 2 (k = 4) on the 4B-36L-h2560 model (weights seed 0, bf16 weights and KV cache, float32
arithmetic) after its 16384-token prompt (prompt seed 1), i.e. the long-context workload's first
round: drafted tokens, draft logits [4, V], verify logits of the drafted rows [5, V], n_accept and
the bonus token, plus a digest of the prompt so a reader can check it is the same input.

Calls only oracle/ and the seeded input generators (synth); nothing here comes from the GPU path.
The prefill runs 256 rows at a time (the oracle's row-blocked prefill: the same cache, bounded
memory). About 20-40 minutes and ~28 GB of host memory on 8 cores.

    python tests/golden/make_c5_first_round.py
"""
import hashlib
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import model as om  # noqa: E402
from oracle import seed as os_  # noqa: E402
from paper_2609_36590_amd import synth  # noqa: E402

K = 4
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c5_first_round.npz")


def prompt_digest(prompt):
    return hashlib.sha256(np.asarray(prompt, dtype=np.int32).tobytes()).hexdigest()


def main():
    cfg = synth.C5_4B_LONG
    t0 = time.time()
    w = synth.make_weights(cfg, seed=0)
    m = om.Model(cfg, synth.weights_as_f32(cfg, w), np.float32)
    del w
    prompt = synth.make_prompts(cfg, seed=1)[0]
    assert len(prompt) == 16384
    print(f"weights ready {time.time() - t0:.0f} s; prefill of {len(prompt)} tokens", flush=True)
    st = os_.prefill(m, prompt, len(prompt) + K + 2, row_block=256)
    print(f"prefill done {time.time() - t0:.0f} s", flush=True)
    drafts, qlog = os_.draft(st, K)
    plog = os_.verify(st, drafts)
    n, bonus = os_.accept(drafts, plog)
    print(f"round done {time.time() - t0:.0f} s: drafts {drafts.tolist()} n_accept {n} bonus {bonus}", flush=True)
    np.savez_compressed(OUT, drafts=np.asarray(drafts, dtype=np.int64), draft_logits=qlog.astype(np.float32),
                        verify_logits=plog.astype(np.float32), n_accept=np.int64(n), bonus=np.int64(bonus),
                        p=np.int64(st.p), prompt_sha256=np.array(prompt_digest(prompt)), config=np.array(cfg.name))
    print(f"wrote {OUT}", flush=True)


if __name__ == "__main__":
    main()
