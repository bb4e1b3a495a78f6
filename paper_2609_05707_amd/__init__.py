"""MI355X (gfx950) decode-step attention for Intra-Prompt Parallel Decoding.

The compute lives in libippd.so (hand-written HIP, C ABI in include/ippd.h);
``_lib`` is its ctypes binding and ``session.DecodeBatch`` a torch-side
holder of device buffers.  Importing this package does not load the library;
``load_library()`` does, and raises if it has not been built.
"""
from ._lib import (  # noqa: F401
    EXPORTED,
    IppdBatch,
    IppdKvCache,
    IppdError,
    load_library,
    ippd_load_context,
    ippd_load_segments,
    ippd_append_kv,
    ippd_decode_workspace_bytes,
    standard_decode_workspace_bytes,
    ippd_decode_attention,
    standard_decode_attention,
    ippd_decode_step,
    standard_decode_step,
)
