"""Batched, lossless speculative verification on one MI355X (gfx950).

Thin ctypes binding of ``libsdverify.so`` (the C-ABI declared in
``include/sdverify.h``).  Each function has the C name, marshals torch device
tensors, host integer arrays and the current HIP stream into the C call, and
raises :class:`SdError` on a non-zero status.  No step of the computation runs
in Python: every result comes from the HIP kernels, and the binding fails
loudly when the library has not been built.
"""

from ._binding import (  # noqa: F401
    SD_DTYPE_BF16,
    SD_DTYPE_F32,
    SD_ERR_CAPACITY,
    SD_ERR_HIP,
    SD_ERR_INVALID_ARGUMENT,
    SD_ERR_UNSUPPORTED,
    SD_ERR_WORKSPACE,
    SD_FLAG_PACKED_VOCAB,
    SD_OK,
    Dims,
    Expand,
    KVPages,
    KVPool,
    PreparedCall,
    Sampling,
    SdError,
    exported_symbols,
    library,
    library_path,
    prepare_acceptance_rate,
    prepare_verify_attention,
    prepare_verify_step,
    prepare_verify_step_paged,
    prepare_verify_step_sampled,
    prepare_verify_step_tree,
    sd_acceptance_rate,
    sd_expand_layer,
    sd_accept_resample,
    sd_accept_resample_sampled,
    sd_accept_tree,
    sd_pack_vocab,
    sd_status_string,
    sd_tree_commit_kv,
    sd_verify_attention,
    sd_verify_attention_paged,
    sd_verify_attention_tree,
    sd_verify_logits,
    sd_verify_step,
    sd_verify_step_static,
    sd_verify_step_paged,
    sd_verify_step_sampled,
    sd_verify_step_tree,
    sd_version,
    sd_vocab_kernel_name,
    sd_vocab_packed_bytes,
    sd_workspace_bytes,
)
