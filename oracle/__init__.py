"""fp64 CPU oracle for the ResNet-18 training step and the dual-batch merge.

TEST INFRASTRUCTURE ONLY. This package is the slow, obviously-correct
reference that the HIP path is checked against. Only the test suite, the
smoke check in ``__graft_entry__`` and the CPU-baseline leg of ``bench.py``
may import it; the product path never does and must not fall back to it.

Everything here is written from the definitions (direct sums over kernel
taps, explicit batch-norm and softmax cross-entropy formulas, the merge rule
of the paper's model-update factor) in float64 NumPy, NCHW layout. It shares
no code, tables or helpers with the HIP library under
``paper_2509_26092_amd/``; neither side imports the other.

Modules
  ops      single operators (conv fwd / data-grad / weight-grad, BN, ReLU,
           pools, FC, softmax-CE, SGD-momentum, bf16 rounding)
  net      ResNet-18 variants, flat parameter-state layout, train step,
           eval forward
  merge    parameter-server merge with the model-update factor (Sec. 3.4)
           and the dual-batch planner arithmetic (Eqs. 2-8)
  philox   Philox4x32-10 and the dropout masks drawn from it

Parity status: every function is pinned by a ``-m "not gpu"`` test against
something other than itself (dense-matrix brute force, finite differences,
closed forms, invariants, the paper's Table 2 values), except the choices the
paper leaves open (BN epsilon/momentum, weight-decay scope, He fan mode, the
bf16 rounding points), which are conventions: "parity unpinned" for those
choices themselves, the arithmetic that uses them is pinned.
"""
