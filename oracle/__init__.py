"""CPU oracle for the KDA step with a mixed-precision recurrent state.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or runs
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code with the
HIP library (``paper_2609_30950_amd``) and the library shares none with it.

Two arithmetic flavours are provided, each written straight from the paper
("Low-Bit Recurrent States in Hybrid Language Models"):

* TRUTH: float64 NumPy, used for output accuracy, closed forms and invariants.
* MIRROR: the float32 numerics contract (operation order, fused multiply-adds,
  reduction trees, rounding of scales) under which every discrete output
  (bit widths, clip-factor choice, codes, FP16 scales, decay codes) is
  reproducible bit for bit.  Where float32 decides an integer, the oracle takes
  that decision in float32 exactly as the kernels do.

Modules
-------
fp          exact float32 fma emulation, FP16 rounding, reduction trees
recurrence  gated delta rule (Sec. 2, eq. rule), TRUTH and MIRROR forms
stats       EMA decay/erase estimates, Gramian weights (Prop. 1, eq. gram,
            eq. weight), exact Gramian for pins, log-uniform rate codes
alloc       range normalisation and high-rate bit allocation (eq. alloc)
quant       symmetric row quantiser with fitted clip factor (Sec. 3)
record      byte layout of the packed per-head state record
step        decode step and chunked prefill drivers (write-back protocol)

Parity status per function is stated in each module docstring.
"""
