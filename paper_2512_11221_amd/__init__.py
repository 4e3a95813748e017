"""MI355X (gfx950) decode-step library for ASR-KF-EGR (arXiv 2512.11221).

The HIP kernels and the C ABI live in libasrkf.so (csrc/, include/asrkf.h);
``_lib`` is the thin ctypes binding with the same function names.
"""
from ._lib import (AUTO, SR, WR, FR, NONE, BF16, F32, AsrkfError, load,  # noqa: F401
                   REL_ABS, REL_SOFTMAX, SCOPE_LAYER, SCOPE_TOKEN, CAND_OUTSIDE, CAND_INSIDE,
                   make_config, asrkf_init, asrkf_prefill, asrkf_decode_step,
                   asrkf_decode_step_static, asrkf_restore, asrkf_stats, asrkf_stats_reset, asrkf_set_timing, asrkf_timing_series, asrkf_reset,
                   asrkf_debug_delay_side, asrkf_get_state,
                   asrkf_get_seq, asrkf_get_residency, asrkf_schedule_table, asrkf_destroy,
                   asrkf_last_error)
