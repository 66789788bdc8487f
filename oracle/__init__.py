"""mLSTM cell oracle: TEST INFRASTRUCTURE ONLY.

Plain, slow CPU forms of the cell in fp64 that the HIP library is checked
against.  Only the tests, the smoke check and the benchmark's CPU-baseline
leg may use this package; the product path never imports it, and nothing
here imports the product package's kernels or binding.

* ``mlstm_oracle.c`` / ``coracle``: the recurrent form (Eqs. 2-5, 7-8) in C
  with OpenMP over independent sequences; the timed CPU baseline.
* ``mlstm_ref``: NumPy fp64 forms (recurrent, unstabilized, fully parallel,
  chunkwise) used to pin the C oracle and each other, the output gate and
  headwise norm, the gate pre-activations and the multi-head layer.
* ``mlstm_grad``: the gradients for the backward pass, by autograd over the
  step-by-step cell and in closed form over the parallel form.
"""
