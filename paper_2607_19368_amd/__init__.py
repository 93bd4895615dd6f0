"""Spectral-LSH hot path on AMD MI355X (gfx950): HIP kernels behind the C ABI
of include/slh.h (libslh.so), with a thin ctypes binding (slh.py)."""
from .slh import (  # noqa: F401
    SLHError, load, slh_gen_params, slh_gen_start, slh_create, slh_set_option, slh_set_stream,
    slh_route, slh_feature_map, slh_lanczos, slh_simhash, slh_merge, slh_merge_async, slh_merge_wait, slh_merge_capacity,
    slh_copy_out, slh_load, slh_stage_times, slh_time_passes, slh_spectral_energy, slh_bucket_purity, slh_eigh_ritz, slh_peak_read, slh_peak_mfma, slh_merge_noalloc, compress,
)
