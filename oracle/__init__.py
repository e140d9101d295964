"""fp64 CPU oracle of the Monte Carlo mutation-selection method (MCA).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package: only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP library: not a
kernel, header, helper, table or constant generator.  The seeded input
generators (package ``workloads``) are the only code both sides consume, and
they hold none of the method's arithmetic.

Contents (each function cites the passage of the paper it follows):

* ``philox``     Philox4x64-10 counter-based generator, written from its
                 published definition (Salmon et al., SC'11), and the decoding
                 of one draw into a single-parameter mutation (Eq. 1, Eq. 12)
                 or a channel mutation (Sec. 2.3).
* ``mlp``        fp64 forward pass and average cross-entropy (Eq. 2) of a
                 bias-free MLP, by full recomputation (the definition), and an
                 fp64 incremental evaluator (Sec. 2.4: only the changed local
                 fields move) that carries the field changes layer to layer
                 and forms each sample's loss change from its logit change
                 by exact identities (so a change of 1e-11 on a loss of 2.3
                 keeps its digits), pinned against the definition in fp64
                 where changes are large and in long double where small.
* ``normmlp``    fp64 deep MLPs of Sec. 2.1: biases, normalized hidden fields
                 and the layer-sticky proposal schedule.
* ``transformer`` fp64 forward pass and loss of the pre-LN causal decoder.
* ``mca``        the selection loop (Eq. 1, Eq. 5, Eq. 6, and the Metropolis
                 rule of Eq. 7 as a per-candidate threshold) over K candidates
                 per step in stream order, with pruning moves first and
                 minibatch windows (Sec. 2.2).

Every function computes in float64 from fp32 state; the mutated parameter
itself is formed in fp32 exactly as a single-precision implementation would
(Sec. 2: computations in single precision).

Pin status: every function here is pinned by a test under ``tests/`` against
something other than itself (library routines, closed forms, brute force);
none is "parity unpinned".
"""
