"""CPU oracle for one Jacobi iteration of a causal decoder (Jacobi Forcing,
arXiv 2512.14681).

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
reference that the GPU path is checked against.  Only the tests, the smoke
check in ``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may
import it; the product path never does and shares no code with it.

Contents, each citing the passage it follows:

* ``numerics``   -- bf16 round-to-nearest-even emulation (the bf16 KV cache
                    of the bf16 model variant; not a paper passage).
* ``model``      -- the decoder forward pass over draft rows against an exact
                    prefix KV cache (Sec. 2.1 "Jacobi Decoding": one forward
                    pass under a causal mask yields every row's prediction).
* ``tree``       -- segments -> parent / position / visibility of the rows of
                    one step (Sec. 3.2: candidates verified side by side,
                    blocks concatenated; input assembly of App. A Alg. 1).
* ``jacobi``     -- greedy AR decoding (Eq. 1), the Jacobi update (Eq. 3),
                    longest-prefix acceptance, block mode (Eq. 4), running
                    window (Sec. 4.2, running-window variant) and the
                    pure fixed-point iteration of Eq. 3 without commits.
* ``multiblock`` -- multi-block decoding with rejection recycling (Sec. 3.2,
                    App. A Alg. 1).
* ``mock``       -- deterministic next-token backends used to drive the
                    decoding state machines without a transformer.
* ``trajectory`` -- Jacobi trajectories of blocks (Sec. 2.1), the noise
                    schedule (Eq. 7) and the unconverged-fraction point
                    selection (App. C).
* ``packed``     -- logits of a packed noisy/clean training sequence under
                    the noise-aware and the clean-context masks (Sec. 3.1,
                    App. C), by plain causal forwards over each chain.

Precision: fp64 by default (the plain definition); a float32 mode with the
same rounding points exists for the 7B-shaped model, whose fp64 weights would
not fit a test host comfortably.
"""
