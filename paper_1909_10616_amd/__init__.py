"""Tuned GEMM for MI355X (gfx950) with the G-BFS configuration search of
arxiv 1909.10616 (and its N-A2C and random-search tuners). The compute path is libgemmtune.so (HIP); this package only
binds it."""
from .gemmtune import (A_KMAJOR, ADJACENT, ANY_PAIR, BF16, F32, GemmTuneError, Space,  # noqa: F401
                       gemm_run, gt_compare, gt_measure, gt_reference_gemm, lower, tflops,
                       tune_gbfs, tune_na2c, tune_random)
