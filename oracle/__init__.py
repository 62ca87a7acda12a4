"""CPU oracle for Batch-Max prefill-and-decode (P&D) KV-cache-compressed attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with
the HIP path (no kernels, headers, helpers, tables or constants); the two meet
only through the seeded input generator, which holds none of the method's
arithmetic.

Modules
-------
``pd``     numpy float64 oracle, one (sample, KV head) unit at a time, with
           full probability rows materialised (no online softmax, no fusion).
``micro``  pure-Python loop oracle for tiny inputs; exact rational arithmetic
           (``fractions.Fraction``) when every visible logit of a row is equal,
           e.g. all-zero keys, where softmax is exactly uniform.

Every function cites the passage of the paper (arXiv 2412.05693, "Batch-Max")
it follows: Sec. 3 (left-padded batch, cache bound), Sec. 3.1 with Algorithm 1
(block-wise prefill, eviction schedule), Sec. 3.2 (``sum_weights`` update and
the ``ave_weights`` eviction rule).

Pins (tests/test_oracle_pins.py) tie each function to something outside
itself: dense causal attention from ``torch.nn.functional.
scaled_dot_product_attention`` when nothing is evicted, the paper's stated
values of Sec. 3.2, a hand-derived exact worked example
(``tests/golden/uniform_worked_example.json``), brute-force subset selection,
score conservation, permutation and unit independence, and agreement of the two
independent implementations here.  The ranking inside the near-tie band (two
averages closer than 1e-6) is parity unpinned by construction.
"""
