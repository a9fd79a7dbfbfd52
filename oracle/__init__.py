"""CPU oracle of FlashLoop's per-loop attention step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, deliberately unoptimised NumPy implementation of what the step computes, written from
the paper ("FlashLoop: Fast and Memory-Efficient Looped Transformers via Lazy Updates"), Sections 3-4
and Appendix D.  Floating-point work is fp64 except where an exact bf16/fp16/fp32 rounding sequence is
part of the definition (the residual codec and the selection keys, whose results are integers or bit
patterns).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may import this package.
The product (the HIP library and its Python binding) never imports, calls or links anything here, and
this package imports nothing from the product: the two share only the seeded input generator
(`workloads`), which holds none of the method's arithmetic.

Modules
  numerics   bf16 / fp16 rounding helpers (the oracle's own)
  select     token scores and nested top-k                      (Section 4.1, Appendix D.1, Eq. 5)
  codec      residual quantization, packing, reconstruction     (Section 4.3, Appendix D.3, Eqs. 4, 8)
  attention  dense loop, column statistics / selection, mass-corrected sparse update
                                                                 (Sections 3.2, 4.2, Appendix D.2, Eqs. 2, 3, 6, 7)
  chain      one layer end to end: loop-1 setup, then sparse loops 2..R

Parity status of each function is stated in its docstring; all are pinned by tests in
tests/test_oracle_*.py (see the pins listed there) except the accuracy of the approximation against
exact loop-r attention, which needs real model activations ("parity unpinned", diagnostic only).
"""
