"""MI355X-native additively-quantized (AQ) layer: forward and codebook gradient.

The product is ``libaq.so`` (HIP kernels for gfx950 behind the C ABI in
``include/aq.h``); this package holds its sources (``csrc/``), the build
script and a ctypes binding with the same entry-point names.
"""
from .aq import (  # noqa: F401
    AQError,
    AQLayer,
    LIB_PATH,
    EXPORTED,
    load_library,
    make_desc,
    aq_layer_create,
    aq_layer_forward,
    aq_layer_forward_static,
    aq_layer_prepare,
    aq_layers_prepare,
    aq_layer_decode,
    aq_layer_codebook_grad,
    aq_layer_set_path,
    aq_layer_set_option,
    aq_layer_get_option,
    aq_layer_set_launch_events,
    aq_layer_last_launches,
    aq_layer_describe,
    OPTION_CODES,
    aq_layer_choose_path,
    aq_layer_destroy,
    aq_version,
)
