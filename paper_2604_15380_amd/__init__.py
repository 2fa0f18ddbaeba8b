"""MI355X-native batched PaiNN screening forward pass (HIP, gfx950).

Python binding of the C ABI in include/painn.h.  The functions below carry
the C names and only marshal arguments (device pointers come from torch
tensors, the stream from torch); every step of the computation runs in the
HIP kernels of libpainn.so.  Importing works without a GPU; calling anything
needs the built library and a device, and fails loudly otherwise.
"""
from .binding import (PAINN_BF16, PAINN_FP32, PAINN_FP64, PainnError,  # noqa: F401
                      lib_path, load_library, painn_build_graph, painn_build_graph_capped, painn_create,
                      painn_destroy, painn_forward, painn_forward_blend, painn_forward_features,
                      painn_graph_csr, painn_graph_free, painn_last_error,
                      painn_model_free, painn_model_options, painn_model_info, painn_model_load,
                      painn_model_load_buffer, painn_profile_enable, painn_profile_read,
                      painn_set_stream, painn_status_string, painn_synchronize)
from .runtime import Graph, Model, Runtime  # noqa: F401
