"""CPU oracle for the merged actor update -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct numpy implementation of what the GPU path
computes, used to check it.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the product path never does, and
it shares no code with the HIP kernels or their binding.

  merge.py  Timeline merging (Section 4.4.2, Algorithm 1, token-level Match)
            and the flattening of surviving timelines into packed segments.
  model.py  One pre-norm decoder block, the LM head, token log-probs and the
            clipped policy-gradient loss (Section 3: GRPO-style updates,
            clip ratio 0.2 from the AIME case study in Section 6), forward and
            hand-written backward, all in float64.

Every function is pinned by tests that check it against closed forms, special
cases that reduce to library routines, brute force and finite differences.
"""
