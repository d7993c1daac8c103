"""CPU oracle for the relaxed online long convolution (test infrastructure).

This package is the correctness reference for the GPU library.  It is plain,
slow numpy code in fp64 over fp32 inputs.  Only the tests, the smoke check and
the CPU-baseline leg of the benchmark may import it; the product path never
does.  It shares no code with the GPU path: the only module both sides use is
the seeded input generator ``datagen`` (no convolution arithmetic in it).

Contents (all indices 0-based: positions 0..L-1, z_t = sum_{s<=t} y_s h_{t-s}):

* ``schedule``  -- the tile order of the relaxed algorithm (Alg. 1; Prop. 1).
* ``conv``      -- the plain definitions: the lazy O(L^2) sum (Eq. onlineConv,
  the "lazy approach" of Sec. 3.1.1), the static FFT convolution used at
  training time (Sec. 2.3.1) and the one-pole recurrence of a geometric
  filter (the LTI-SSM view, App. "State Space Models").
* ``relaxed``   -- the relaxed tiling itself: red cells and gray tiles in the
  order of Alg. 1 / Alg. 3, with the contribution block tau (Eq. taus)
  computed either directly or by the 2U-point cyclic FFT of App. B.
* ``feedback``  -- the elementwise chained block used by the synthetic
  workloads (y^{l+1}_t = 0.5 tanh(z^l_t) + x^l_t, layer 0 fed from the last
  layer at t-1).
* ``dd``        -- the relaxed online product with data-dependent filters
  (Alg. 5): rho_t revealed with y_t, parallelogram tiles of untruncated
  convolutions of two length-U blocks, every power of two U dividing t+1.
* ``block``     -- the blocks and sampler of the paper's synthetic model
  (Sec. 5): an MLP of hidden width 2D with GELU per layer, and the next
  token's input = the last layer's output plus noise.

Every function is pinned by tests in ``tests/test_oracle*.py`` and
``tests/test_schedule.py`` against closed forms, brute force and invariants
the paper fixes; none is marked "parity unpinned".
"""
