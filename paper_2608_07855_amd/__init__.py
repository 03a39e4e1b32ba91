"""CommitKV hot path on MI355X (gfx950): HIP kernels behind a C ABI.

The compute runs in ``libcommitkv.so`` (``python -m paper_2608_07855_amd.build``);
this package only marshals torch tensors into its calls.
"""
from .binding import (Agent, CKVError, Context, Pages, cache_view, ckv_classify_pages,  # noqa: F401
                      ckv_joint_test, ckv_measure_page_effects, ckv_measure_page_effects_batch,
                      ckv_measure_recorded, ckv_pool_scores,
                      ckv_select_and_compact,
                      kv_view, lib, version, window_view, PAPER_THRESHOLDS)
