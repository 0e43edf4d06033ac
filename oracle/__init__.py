"""Float64 CPU oracle for sequence-bucketed RNN training (arXiv 1708.05604).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the package's
smoke check and the benchmark's CPU-baseline leg may import or run anything in
this directory.  The GPU path (``paper_1708_05604_amd``) never imports it, and
it never imports the GPU path: the two share only the seeded input generators
of ``paper_1708_05604_amd.synth``, which hold none of the method's arithmetic.

Modules
  bucketing  the dynamic-programming bucketing of Sec. III.A (eqs. 1-2 and the
             DYNAMICBUCKETING procedure), bucket assignment, padded-step counts
  schedule   the per-epoch batch schedule: buckets shortest first (Sec. IV.A),
             shuffled inside each bucket (Sec. III), cut into mini-batches
  rnn        LSTM / GRU forward and backpropagation-through-time in float64,
             per-frame softmax cross-entropy, SGD
  optim      ADADELTA, the update rule of the paper's training processes
             (Sec. III.B, step 4)
  ctc        the CTC loss of the paper's experiments (Sec. IV.A) and its
             gradient, log-space forward-backward over the blank-extended target
  aggregate  the epoch-end mean of parallel replicas with decay (Sec. III.B,
             eq. 3)

Every function is written to be checked by eye against the paper or against
textbook definitions, not to be fast.  Pins (brute force, closed forms, finite
differences, an independent library routine) live in tests/test_oracle_*.py.
"""
