"""FedOptima server hot path on MI355X (gfx950).

The compute lives in ``libfedoptima.so`` (HIP kernels behind a C ABI, see
``include/fedoptima.h``); ``api`` is its argument-marshalling binding.
"""
from . import api  # noqa: F401
from .api import (  # noqa: F401
    fo_async_aggregate, fo_pick_device, fo_server_step, fo_model_create, fo_model_destroy,
    fo_model_read, fo_model_write, fo_queues_create, fo_queues_destroy, fo_queues_push,
    fo_queues_push_model, fo_queues_in_service, fo_queues_release, fo_aggregate_pending,
    fo_aggregate_pending_all, fo_queues_stats, fo_queues_counters, fo_set_max_delay, fo_set_stream,
)
