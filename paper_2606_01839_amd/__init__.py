"""MI355X-native paged-KV attention hot path under conversation-level disaggregated serving.

The C ABI (include/conserve_attn.h) lives in ``libconserve_attn.so`` (gfx950 HIP kernels);
``paper_2606_01839_amd.conserve`` is its Python binding.
"""
from .conserve import (KVPool, ConserveError, load_library, PAGE_TOKENS, EXPORTS,  # noqa: F401
                       CS_OK, CS_EINVAL, CS_ENOMEM, CS_ENOENT, CS_ESTATE, CS_ERANGE, CS_EHIP, CS_EBUSY,
                       CS_MIXED_LAYER_ORDERED,
                       Scheduler, prefill_curve_fit, prefill_curve_eval, provision_decoders,
                       place_least_occupied, device_info, probe_stream_read)
