"""Plain CPU oracle of SpecBlock's block-expansion hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it, to check the HIP path and to time
a CPU baseline.  It shares no code with the HIP library or its binding; both
sides take their inputs from the ``synth`` generators only.

The oracle is written from the paper (SpecBlock: Block-Iterative Speculative
Decoding with Dynamic Tree Drafting):

* ``numerics``  RMSNorm, RoPE, SiLU, softmax attention and the bf16 rounding
                used to model the bf16 configurations, in float64;
* ``model``     the Llama-style target and the SpecBlock drafter block forward
                (Sec. 3.1, Eq. 1-3) over explicit rows with explicit visibility;
* ``rank``      the 15-dim distribution summary psi (App. B), the rank head
                (Eq. 4), the rank-to-bucket rule (Sec. 3.3) and the
                bucket-to-branching maps (App. A.5);
* ``tree``      the draft tree, rank-guided sibling attachment and next-block
                start selection (Sec. 3.2, Alg. 2);
* ``specdec``   prefill, one verifier iteration (Alg. 2: M block expansions,
                tree verification, greedy acceptance, commit) and plain greedy
                decoding of the target for the lossless check.
* ``sampling``  stochastic tree verification at temperature T > 0 (the
                paper's T = 1.0 setting): recursive rejection sampling of a
                node's children as point-mass drafts, then the residual draw.

Readings of points the paper leaves open are listed with the code that takes
them.  Floating point is float64 throughout; ``Numerics("bf16")`` additionally
rounds to bfloat16 at the points where the bf16 configurations store bf16
(GEMM inputs, Q/K/V, attention output), so the discrete decisions of a bf16
run can be compared with margins that reflect only accumulation order.

Parity status: every function here is pinned by ``tests/test_oracle_*.py``
except the next-block start-selection rule and the budget insertion order,
which the paper does not fix (parity unpinned: our reading).
"""
