"""Float64 CPU oracle for the per-head spectral-norm estimator and the
per-layer FP8 E4M3 scale factor.

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import anything here; the product path
(the HIP library and its Python binding) never does, and this package shares
no code with it.

Modules
-------
power_iteration  The method itself, in the paper's order and notation
                 (App. E, "Power Iteration for Spectral Norm Estimation" and
                 "Implicit GQA Power Iteration"), one head at a time (per-head
                 reading) and the paper-literal layer-concatenated form.
explicit         Textbook cross-checks that form M = W^Q W^{K T} explicitly:
                 dense power iteration, SVD and a QR-reduced exact sigma_1.
calibration      Eq. "scale", the gamma / alpha_min selection rule (Sec. 3.2)
                 and the overflow-probability terms T1, T2.
e4m3             Exact OCP E4M3FN encoder / decoder and the overflow predicate.
fp8_consumer     Stage 3 of the geometry-aware forward pass up to the E4M3
                 logits: S = Q K^T / sqrt(d_h), S / scale, codes, max |S~| and
                 the overflow count per head.

Every function here is pinned by the ``-m "not gpu"`` tests against values
the paper prints, closed forms or textbook routines; none is "parity
unpinned".
"""
