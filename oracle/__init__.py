"""CPU oracle for checkpointed backpropagation through time.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute anything in this package: only the tests, the smoke check and the
CPU-baseline leg of the benchmark use it.  It shares no code with the GPU
path; the only thing both sides use is the seeded input generator in
``synth``.

Contents
  cells     float64 forward step and adjoint step of the three recurrent
            cells (tanh RNN, LSTM, residual MLP), written from the chain rule.
  bptt      conventional backpropagation through time that stores every
            state (the plain definition, Section 1.1 and Fig. 1 of the paper:
            memory linear in n, peak at the end of the forward pass).
  schedule  Revolve (binomial) counting and schedule generation, the
            asynchronous two-level policy of Section 2, its canonical text,
            a replayer and a symbolic checker.

Checkpointing only decides which states are recomputed, never what is
computed, so with a deterministic step function every valid schedule
reproduces the store-all result exactly; the replayer relies on that.
"""
