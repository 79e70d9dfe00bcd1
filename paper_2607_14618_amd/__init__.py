"""MI355X (gfx950) mixed-bit linear layer: PolyQ's decode GEMV and prefill GEMM.

Python binding of libpolyq.so (include/polyq.h).  The functions take torch
tensors for device memory and run on torch's current HIP stream.
"""
from ._lib import (Block, Layout, PolyQError, EXPORTS, LIB_PATH, lib, plan, pack, pack_rows, unpack,  # noqa
                   permute, gemv, gemv_batch, gemm, gemm_batch, gemv_workspace_bytes, gemm_workspace_bytes,
                   PreparedBatch, read_probe, channel_error, waterfill, quanta_match, cluster, allocate, bit_scaling,
                   SCALE_GRID)
from .layer import PackedLinear, decode_batch, prefill_batch, group_index, device_perm  # noqa: F401
