"""Plain fp64 CPU oracle for the replay-buffer policy-gradient hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and its
Python binding) imports, links or runs anything in this package; only the test
suite, the smoke check and the benchmark's CPU-baseline leg do.  The oracle and
the HIP path share no code: no kernels, headers, constants or helpers.  The only
thing both sides consume is the seeded synthetic-input generator, which holds
none of the method's arithmetic.

Each module follows one part of the paper (arXiv 2604.08706, "Efficient RL
Training for LLMs with Experience Replay"):

* ``philox``    -- the counter-based generator (Philox4x64-10, Salmon et al.,
                   SC'11) that drives every random draw of the sampler; the
                   paper is silent on the generator.
* ``buffer``    -- the FIFO replay buffer and its sampling rules
                   (Sec. 3.1; App. B "BufferStructure"; Sec. 5 "Further
                   optimization" and App. D.4 "Positive-bias sampling").
* ``advantage`` -- group-normalised advantages at insert time (App. D.2).
* ``logprob``   -- per-token policy log-probabilities from hidden states and the
                   LM-head weight (App. D.2, temperature 1).
* ``loss``      -- the clipped importance-weighted GRPO objective and its
                   gradient w.r.t. the token log-probabilities (App. D.2).
* ``grad``      -- backward of the log-probabilities to the hidden states and
                   the LM-head weight.

Parity status per function is stated in each module header.
"""
