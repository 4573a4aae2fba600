"""KV-cache streaming (pack, unpack, swap) for one MI355X.

The product is the C-ABI library ``libdv.so`` declared in ``include/dv.h``;
``paper_2403_01876_amd.dv`` is its Python binding.
"""
from . import dv  # noqa: F401
from .dv import (Cache, DvError, dv_api_version, dv_cache_bytes, dv_packed_bytes,  # noqa: F401
                 dv_stream_in, dv_stream_out_prompt, dv_stream_out_token, dv_swap_in,
                 dv_swap_out)
