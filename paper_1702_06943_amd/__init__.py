"""MI355X-native tuple-oriented compression (TOC): encode on the host, run A.W,
G^T.A, decode, sparse-safe element-wise ops and dense A .+ c on the compressed
mini-batches with hand-written gfx950 kernels; pack batches into the paper's
physical encoding and build the decoding tree C' and the whole upload image from
it on the GPU; run
mini-batch gradient descent steps of linear models and of a feed-forward neural
network on the compressed batches;
encode many mini-batches at once on the GPU.

The functions are those of include/toc.h, called through ctypes; see binding.py.
"""

from .binding import (  # noqa: F401
    TocError, Enc, Dev, lib, LIB_PATH, BATCH_DTYPE, KEY_DTYPE, LINK_DTYPE,
    TOC_UPLOAD_KEEP_DEAD, TOC_UPLOAD_HOST, TOC_OP_RIGHT, TOC_OP_LEFT, TOC_OP_DECODE,
    TOC_MAP_SCALE, TOC_MAP_SQUARE,
    TOC_EINVAL, TOC_ENOMEM, TOC_ESIZE, TOC_EDEVICE, TOC_EUNSUPPORTED,
    toc_encode, toc_encode_batches, toc_enc_info_get, toc_enc_export,
    toc_upload_size, toc_upload, toc_dev_info_get, toc_dev_layout_get,
    toc_workspace_size, toc_right_mul, toc_left_mul, toc_left_mul_noalloc, toc_decode_csr,
    TOC_NOALLOC_SCRATCH_BYTES,
    toc_map_values, toc_decode_dense,
    TOC_CPRIME_LAYOUT, TOC_CPRIME_VALUE_INDEX, TOC_CPRIME_STARTS, TOC_CPRIME_CODE,
    TOC_CPRIME_NODES, TOC_CPRIME_ROWS, TOC_CPRIME_COLUMN, TOC_LEVEL_D, TOC_LEVEL_DEPTH,
    TOC_LEVEL_LIVE,
    toc_level_workspace_size, toc_level_build, toc_level_right_mul,
    toc_enc_pack, toc_phys_info_get, toc_cprime_workspace_size, toc_cprime_build,
    TOC_MGD_LINEAR, TOC_MGD_LOGISTIC, TOC_MGD_HINGE, toc_mgd_epoch, toc_mgd_workspace_size,
    toc_mgd_epoch_split,
    TOC_ENCDEV_ROWPTR, TOC_ENCDEV_SIZE, TOC_ENCDEV_COLUMN, TOC_ENCDEV_VALUE,
    toc_encode_device_workspace_size, toc_encode_device,
    toc_mlp_workspace_size, toc_mlp_epoch,
    TOC_INGEST_CHANGED, toc_ingest_workspace_size, toc_ingest_plan, toc_ingest_build,
)
