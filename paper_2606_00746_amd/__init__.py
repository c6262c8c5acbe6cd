"""MI355X-native GSPN line-scan propagation (libgspn).

The 2D line-scan recurrence of Generalized Spatial Propagation Networks,
h_i = w_i h_{i-1} + lambda_i * x_i with output y = sum_d u_d * h_d over four
scan directions, forward and backward, as hand-written HIP kernels for gfx950
behind a C ABI (``include/gspn.h``).  This package is the ctypes binding.
"""
from ._native import (ALL, B2T, BF16, BLOCKED, F32, L2R, LIB_PATH, OP_BWD, OP_BWD_BLOCKED,
                      OP_BWD_NORM, OP_BWD_NORM_RESERVE, OP_BWD_RESERVE, OP_FWD, OP_FWD_BLOCKED,
                      OP_FWD_NORM, OP_FWD_NORM_TRAIN, OP_FWD_TRAIN, PIXEL, R2L, T2B, GspnError, gspn_last_hip_error,
                      gspn_latent_fwd, gspn_latent_params, gspn_latent_workspace_size,
                      gspn_project, gspn_reserve_size, gspn_reserve_size_norm, gspn_scan_bwd,
                      gspn_scan_bwd_blocked, gspn_scan_bwd_norm, gspn_scan_bwd_norm_reserve,
                      gspn_scan_bwd_reserve, gspn_scan_bwd_slots, gspn_scan_bwd_static,
                      gspn_scan_fwd, gspn_scan_fwd_blocked, gspn_scan_fwd_norm,
                      gspn_scan_fwd_norm_train, gspn_scan_fwd_train, gspn_strerror, gspn_version,
                      gspn_workspace_size, gspn_workspace_size_slots, latent_fwd, latent_params,
                      load, project, reserve_size, scan_bwd, scan_bwd_norm,
                      scan_bwd_norm_reserve, scan_bwd_reserve, scan_fwd, scan_fwd_norm,
                      scan_fwd_norm_train, scan_fwd_train, workspace_size)

__all__ = ["ALL", "B2T", "BF16", "BLOCKED", "F32", "L2R", "LIB_PATH", "OP_BWD", "OP_BWD_BLOCKED",
           "OP_BWD_NORM", "OP_BWD_NORM_RESERVE", "OP_BWD_RESERVE", "OP_FWD", "OP_FWD_BLOCKED",
           "OP_FWD_NORM", "OP_FWD_NORM_TRAIN", "OP_FWD_TRAIN", "PIXEL", "R2L", "T2B", "GspnError", "gspn_last_hip_error",
           "gspn_latent_fwd", "gspn_latent_params", "gspn_latent_workspace_size", "gspn_project",
           "gspn_reserve_size", "gspn_reserve_size_norm", "gspn_scan_bwd", "gspn_scan_bwd_blocked",
           "gspn_scan_bwd_norm", "gspn_scan_bwd_norm_reserve", "gspn_scan_bwd_reserve", "gspn_scan_bwd_slots", "gspn_scan_bwd_static",
           "gspn_scan_fwd", "gspn_scan_fwd_blocked", "gspn_scan_fwd_norm", "gspn_scan_fwd_norm_train",
           "gspn_scan_fwd_train",
           "gspn_strerror", "gspn_version", "gspn_workspace_size", "gspn_workspace_size_slots",
           "latent_fwd", "latent_params", "load", "project", "reserve_size", "scan_bwd",
           "scan_bwd_norm", "scan_bwd_norm_reserve", "scan_bwd_reserve", "scan_fwd",
           "scan_fwd_norm", "scan_fwd_norm_train", "scan_fwd_train",
           "workspace_size"]
