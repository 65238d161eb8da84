"""fp64 CPU oracle for thin-key attention.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline use it; the GPU library never imports, links or calls it, and the two
share no code. ``oracle.prefill`` / ``oracle.decode`` are the C implementation
of the definition (Sec. 2.1, Eq. 4); ``brute`` is a pure-Python evaluator for
tiny inputs; ``factored`` is the SVD factorisation and query absorption of
Sec. 2.3 (Eq. 6-7)."""
