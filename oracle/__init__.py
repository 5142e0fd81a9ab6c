"""CPU oracle for packed multi-ragged pair-state computation.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link anything in this package: only the tests, the smoke check and the CPU
baseline leg of the benchmark use it, to check and to time the GPU path.

The oracle is a plain, slow, obviously correct float64 implementation written
from the paper ("DanLing NestedTensor: Composable Multi-Ragged Tensors for Deep
Learning").  Every operation unpacks each sample's dense element, runs textbook
dense math on it, and repacks the result: the reference-semantics contract of
Appendix A ("Reference semantics": the logical view of a packed result equals
the reference operation applied to the logical view of the inputs, which for
sample-local operations is the dense per-element computation).

Modules
  layout    offsets, row splits, coordinate map, gather lists (Sec. 3.1, 3.2)
  numerics  bf16 rounding, LayerNorm, activations, softmax
  ops       broadcast, LayerNorm+Linear, attention, triangle, segment reduce
  blocks    block compositions with the storage rounding points of the GPU path

Parity status per function is stated in each docstring; see also the pins in
tests/test_oracle_*.py.
"""
from . import layout, numerics, ops, blocks  # noqa: F401
