"""MI355X (gfx950) batched speculative-Jacobi rollout (HB-SJD).

Python binding of the C ABI in include/hbsjd.h: argument marshalling only;
every step of the rollout runs in the HIP library libhbsjd.so. PyTorch supplies
device memory and the stream. Importing this package does not load the
library; the first call does, and raises if it has not been built.
"""
from .binding import (  # noqa: F401
    DTYPE_BF16, DTYPE_F32, KERNELS, EXEC_AUTO, EXEC_COMPACT, EXEC_FULL, VERIFY_AR, VERIFY_AR_GREEDY,
    VERIFY_GREEDY, VERIFY_PROB, PROGRESS_INDEPENDENT, PROGRESS_SYNC,
    HbsjdError, Context, ModelDesc, hbsjd_bikl_rows, hbsjd_mfma_probe, hbsjd_philox, hbsjd_transform_rows,
    hbsjd_verify_probs,
    hbsjd_version,
    library_path, load_library,
)
