"""CPU oracle for the HiFA4 forward (test infrastructure only).

This package is a plain, slow, obviously-correct numpy implementation of what
the HiFA4 hot path computes, written from the paper (HiFA4: Training-Free 4-bit
FlashAttention on Ascend HIF4 NPUs, arXiv 2607.04302).  Only the test-suite,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with the HIP library and imports nothing from it.

Modules
  hif4        HIF4 group quantizer (Background, HIF4 paragraph; Section 4.1)
  softmax16   the FP16 softmax exponential E(x) (Appendix C, FP16 operations)
  smooth      Smooth-QK calibration, gate and application (Eq. 1, Sections 4.2-4.4)
  attention   the C4V16 tiled forward with P-Reordering (Algorithm 1, Thm. 1)
  qmean       the Q-Mean auxiliary (Algorithm 1, mu step; Section 4.6; App. C)

Parity status: every function here is pinned by a ``-m "not gpu"`` test against
something other than itself (exhaustive exact enumeration, closed forms from
Theorem 1, brute-force softmax attention, values printed in the paper).  What
remains unpinned is parity with Huawei's official HIF4 QDQ library, which is
not public: the bit-level reading of the format below is our own.
"""
