"""One ALS half-sweep (the hot path of cuMF's alternating least squares) as hand-written
HIP kernels for the MI355X (gfx950), behind the C ABI of include/als.h.

``paper_1603_03820_amd.als`` is the ctypes binding (same names as the C entry points);
``paper_1603_03820_amd.driver`` runs whole iterations (update-X, update-Theta, RMSE) on top of it.
"""
from .als import (ALS_F_MAX, ALSError, Context, als_csr_to_csc, als_destroy,  # noqa: F401
                  als_half_sweep, als_init, als_plan, als_rmse, als_rmse_waves, als_status,
                  als_workspace_bytes)
