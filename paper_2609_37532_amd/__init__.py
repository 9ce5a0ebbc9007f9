"""MI355X-native verify path of block-diffusion speculative decoding (DScale).

Two operations behind the C ABI of ``libdsv.so`` (declared in
``include/dsv.h``), with hand-written HIP kernels for gfx950:

* ``verify_attn(q_packed, cu_qlens, kv_pages, page_table, ctx_lens, out)`` --
  ragged, packed verify attention over a paged bf16 GQA KV cache;
* ``accept(logits_packed, cu_qlens, draft_tokens, accept_len, next_token)`` --
  greedy acceptance (per-row vocabulary argmax + longest-prefix compare);

and the decision step that produces their packed layout:

* ``dvl_allocate_pack(...)`` -- DVL budget allocation and flat-buffer packing
  (verify lengths under the shared budget, the offsets, the packed rows).

``BucketSet`` holds fixed-address buffers and the captured decision and
verify graphs for a set of request-bucket sizes (``select_bucket``).

This module only marshals arguments; PyTorch provides device memory and
streams.  ``Graph`` captures and replays the calls with fixed buffer
addresses; ``KernelTimer`` times the kernels with HIP events, and
``read_probe`` measures the read rate of scattered 4 KiB tiles.
"""
from ._lib import (  # noqa: F401
    DSV_BF16,
    DVL_MAX_REQS,
    PRED_HIDDEN,
    DSV_F32,
    LIB_PATH,
    MAX_QLEN,
    PAGE_SIZE,
    TIMING_KINDS,
    AttnDims,
    DSVError,
    Graph,
    KernelTimer,
    accept,
    accept_noalloc,
    accept_stochastic,
    accept_stochastic_workspace_bytes,
    accept_workspace_bytes,
    alloc_workspace,
    attn_dims,
    dvl_allocate_pack,
    predictor_forward,
    predictor_workspace_bytes,
    load,
    read_probe,
    status_string,
    validate_metadata,
    verify_attn,
    verify_attn_workspace_bytes,
)
from .buckets import Bucket, BucketSet, select_bucket  # noqa: F401,E402
