"""MI355X (gfx950) implementation of the mixed step of heterogeneous batching: one forward over
a type-sorted batch of embedding chunks, generation prefill chunks and decode tokens, with the
incremental pooler on the embedding slice, the LM head on the rows that need next-token logits,
and a greedy sampler.

The compute lives in liborthrus.so (hand-written HIP kernels behind the C ABI declared in
include/orthrus.h).  ``_abi`` mirrors that ABI with the same names; ``runtime`` holds device
memory in torch tensors and marshals arguments.  Build with
``python -m paper_2609_25405_amd.build``.
"""
from ._abi import (LIB_PATH, OrthrusError, load, orthrus_device_error, orthrus_model_create,
                   orthrus_model_destroy, orthrus_plan, orthrus_profile_begin,
                   orthrus_profile_end, orthrus_sample_greedy, orthrus_step, orthrus_strerror,
                   orthrus_workspace_bytes, orthrus_workspace_init)

__all__ = ["LIB_PATH", "OrthrusError", "load", "orthrus_device_error", "orthrus_model_create",
           "orthrus_model_destroy", "orthrus_plan",
           "orthrus_profile_begin", "orthrus_profile_end", "orthrus_sample_greedy",
           "orthrus_step", "orthrus_strerror",
           "orthrus_workspace_bytes", "orthrus_workspace_init"]
