"""CPU oracle for the speculative-decoding hot path (TEST INFRASTRUCTURE ONLY).

A plain, slow, float64 implementation of what the GPU path computes, written
from the paper and the works it cites for the draft-and-verify iteration:

  * ``model``    -- Llama-style decoder forward (embedding, RMSNorm, RoPE,
                    GQA attention over a KV cache, SwiGLU FFN, LM head), the
                    target verify pass over gamma+1 tokens and the draft's
                    single-token step;
  * ``philox``   -- Philox4x32-10 counter-based generator (Salmon et al.,
                    SC'11), used for every random draw;
  * ``sampling`` -- temperature softmax, the fixed-point inverse-CDF sampler,
                    the speculative-sampling accept/resample rule and its
                    greedy special case;
  * ``kvstate``  -- KV commit / rollback bookkeeping after an iteration;
  * ``specdec``  -- one draft-and-verify iteration end to end (the inner loop
                    of the paper's runtime, Sec. 3.4, Alg. 3).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path
and never imports it; inputs (weights, tokens, random words) come from
``paper_2608_10362_amd.synth`` as plain arrays.

Functions whose result is not pinned by a test against something other than
the oracle itself say "parity unpinned" in their docstring; every function
here is pinned (see tests/test_oracle_*.py).
"""
