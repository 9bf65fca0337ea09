"""Plain CPU oracle for the per-use backward-state check.

This package is TEST INFRASTRUCTURE. It is a slow, obviously correct fp64
restatement of what the GPU path computes, written from the paper's text:

* the FP8 store (per-tensor amax scaling, round-to-nearest-even and
  stochastic rounding; Sec. 2.1, App. D.2),
* the normalization store and its two uses (Sec. 3.1, Eq. norm-uses; App. D.4,
  Table "Store policies"),
* the attention correction term D and its backward (Sec. 2.1, Eq. dterm;
  App. D.2),
* a Linear backward whose incoming gradient is rounded to E5M2 (App. D.1,
  HYBRID recipe; the two-stage example of App. C.2),
* one decoder layer composing those stores (App. D.1, Table "Training recipes"),
* the trial statistics (App. C.4: mean error, se over trials, z; App. D.4: R).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call or execute anything in this package. The
product path (``paper_2609_39813_amd``) never imports it, and this package never
imports the product path: the two share no code.

Parity status of each function is stated in its module header.
"""
