"""CPU oracle for the SEED draft-verify decode loop.

TEST INFRASTRUCTURE. This package is a plain, slow, independent NumPy statement of what the
decode path computes. Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import it. The HIP library never calls, links or imports anything here, and
nothing here imports the HIP library: the two share only the seeded inputs (weights, prompts),
which the callers pass in as arrays.

Modules:
  model  -- the decoder-only transformer f (Preliminaries, Eq. 1) with an explicit KV cache.
  seed   -- Algorithm 2 (fixed-length drafting + verification), brute-force greedy decoding
            and the parallel block-mask drafter pass (Sec. 3.2).
  tree   -- confidence-aware dynamic drafting with tree-based verification (the main-experiment
            decoding mode; appendix "Confidence-Aware Dynamic Drafting", "Tree-Based
            Verification", Fig. 3).
  cost   -- the parameter-count cost model of Appendix E (Tables 9 and 10).

Every function cites the passage it follows. Readings taken where the paper is silent are listed
in the module docstrings; the absolute values of logits are pinned by brute force and by an
independent library implementation of the same architecture, not by any number in the paper.
"""
