"""MI355X library for the batched multi-adapter linear layer of "Compress then
Serve" (arXiv 2407.00066): y_t = W x_t + U_k Sigma_{i(t)} V_k^T x_t.

The kernels and the C ABI live in libcts.so (include/cts.h); this package
binds it with ctypes.  torch is used only for device memory and streams.
"""
from ._binding import (CtsError, Problem, apply, apply_diag, apply_multi, apply_multi_packed, apply_multi_sorted,  # noqa: F401
                       apply_noalloc, apply_ranked, apply_uncompressed, apply_uncompressed_ranked,
                       bucketing_size, lib, make_problem, set_stage_events, sort_by_cluster, status_string,
                       validate_ids, workspace_bucketing, workspace_size, workspace_size_multi,
                       CTS_F32, CTS_BF16, NOALLOC_SCRATCH_BYTES)
