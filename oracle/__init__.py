"""Reference oracle for the IsoLoCo outer aggregation step.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 CPU
implementation of the IsoLoCo outer step (Algorithm 2 of "Can Model Merging
Improve Aggregation in DiLoCo?"), written from the paper so that the HIP path
can be checked against it.  Only the test suite, the smoke check of
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import it.
The product path (``paper_2607_03011_amd``) never imports, links or calls it,
and this package imports nothing from the product path.

Contents
--------
``jacobi``       one-sided (Hestenes) Jacobi SVD with round-robin pair ordering
``isoloco_step`` the outer step: pseudo-gradient mean (Algorithm 1's
                 pseudo-gradient, averaged as in Algorithm 2), the isotropic
                 correction of every exactly-2-D tensor (Algorithm 2's SVD
                 branch, i.e. Iso-C of Section 2.2), and Nesterov momentum
                 (Algorithm 2's last three assignments); and the variants
                 the paper studies: the fast five-step Newton-Schulz with the
                 RMS scale (Section 4.3), Muon's spectral scale (Appendix B),
                 standard momentum, correcting the momentum update instead
                 of the pseudo-gradient, and clipping only the singular
                 values above or below their mean (Section 4.5).

Every function is pinned by ``tests/test_oracle_pins.py`` against values fixed
by the mathematics (closed forms, invariants, library routines, brute force)
rather than against itself.  One function is not pinned beyond itself: the
behaviour on inputs whose smallest singular value is below float64 resolution
(parity unpinned; the pseudo-gradients of the benchmark are full rank).
"""
from .jacobi import jacobi_svd, polar_factor  # noqa: F401
from .isoloco_step import (  # noqa: F401
    NS5_COEFFS,
    NS5_STEPS,
    VARIANT_DEFAULT,
    clip_correct,
    correct_matrix,
    decode_bf16,
    heavy_ball_update,
    iso_correct,
    nesterov_update,
    newton_schulz5,
    outer_step,
    pseudo_gradient_mean,
    rms_singular_value,
    spectral_scale,
)
