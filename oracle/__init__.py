"""CPU oracle of the memory-based TGNN batch step -- TEST INFRASTRUCTURE ONLY.

This package is the independent checker of the GPU library.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it; the
product path never does, and it shares no code with the HIP kernels or their
binding (its only shared dependency is the seeded input generator ``synth``,
which holds none of the method's arithmetic).

It is written for clarity, not speed: NumPy, float64 arithmetic unless a
precision mode asks for the storage roundings the method defines, and the
steps in the paper's order.  Module map:

* ``tgn``        -- the batch step: most-recent message selection, message
                    construction (Eq. 1), GRU memory update (Eq. 2), temporal
                    adjacency, most-recent-k sampling, multi-head temporal
                    attention, and the hand-written backward pass.
* ``sequential`` -- the literal per-event reading of Eq. 1-2 (one event at a
                    time), used to pin the batched memory phase.
* ``bf16``       -- round-to-nearest-even conversion to bfloat16.
* ``depscan``    -- the offline backward dependency scan and mixed-batch
                    construction of Algorithm 1.
"""
