"""Tuned GEMM for MI355X (gfx950) with the G-BFS configuration search of
arxiv 1909.10616. The compute path is libgemmtune.so (HIP); this package only
binds it."""
from .gemmtune import (ADJACENT, ANY_PAIR, BF16, F32, GemmTuneError, Space, gemm_run,  # noqa: F401
                       gt_compare, gt_measure, gt_reference_gemm, lower, tflops, tune_gbfs,
                       tune_random)
