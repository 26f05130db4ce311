"""CPU oracle for the DASC state-checkpoint path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct restatement of what the paper defines, used to
check the HIP library.  Only the test-suite, the smoke entry point and the CPU
baseline leg of the benchmark may import it; the library never does, and the two
share no code (the only common module is the seeded input generator in
``workloads``, which holds none of the method's arithmetic).

Modules
  plan        static horizons, selection, ragged offsets, replay window, rank
              slices, compression ratios and matched-HBM slot count
              (Sec. 3.3 Eq. 2-3, Sec. 4.1 Eq. 6, Sec. 4.2 Eq. 7, Sec. 4.3,
              App. B, App. C.1 Eq. 8)
  pack        ragged pack and zero-fill restore on raw 32-bit words
              (Sec. 4.1-4.2, App. B "Scheme 2")
  recurrence  the gated delta rule of Eq. 1: per-token form, chunked WY form,
              the paper-orientation matrix form, and the refresh that writes
              back only omitted units (Sec. 3.1, Sec. 4.2)
  quant       symmetric INT8 checkpoint codec (App. E.1, Eq. 10)

Floating point is binary64 throughout unless the paper fixes the precision
(the INT8 codec computes in FP32 as App. E.1 states).
"""
