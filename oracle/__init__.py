"""CPU oracle for the CAT-Q calibration step.  TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy implementation of what the calibration hot path
computes, written from the paper (Sec. 2.2 learnable modulation, Eq. 3-4;
Sec. 2.3 softened ternarization, Eq. 5-6; Sec. 2.4 output reconstruction,
Eq. 7; App. B.2 group-wise quantisation).  It shares no code with the HIP
path, and the product never calls it: only the test-suite, the smoke check
and the benchmark's CPU-baseline leg may import it.

Modules
  lmst   group statistics, modulation, transition function f and its
         derivatives, hard ternarisation, fake weights, factor gradients,
         2-bit packing
  block  dense decoder-block forward/backward and the reconstruction loss
  moe    routed-expert block forward/backward
  calib  time-state schedule and AdamW on the factors (the trajectory's
         parity is unpinned: the paper prints none; AdamW and the learning
         rate are pinned against torch and closed forms)
"""
