"""CPU oracle for the view-masked attention and the fused token log-prob.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
restatement of what the hot path computes.  Only the test-suite, the smoke
check and the benchmark's CPU-baseline leg may import it; the library and its
Python binding never do, and nothing here shares code with them.

* ``views``     replays the eviction record into the live view of every row
                (Eq. "live-view" of Section 3.2; Definition "trajectory tree",
                Appendix B.1).
* ``attention`` ordinary causal attention run once per branch layer, i.e. the
                LogitTree form (Section 4.1, Eq. "logittree-def"), which the
                materialisation-equivalence theorem (Section 4.3, Appendix C.3)
                says the packed 4D mask reproduces; plus the dense masked form
                of Eq. "4d-mask-def" for tiny inputs.
* ``logprob``   textbook log-softmax at the target id, importance ratio and
                clip (the GRPO ratio of Appendix C, "Pitfall A, RL view", and
                Appendix F hyper-parameters), and the closed-form gradient into
                the hidden states.

Every function is pinned by ``tests/test_oracle_*.py`` against values the paper
prints (``tests/golden/``), closed forms, brute force and invariants.  No
function here is "parity unpinned".
"""
