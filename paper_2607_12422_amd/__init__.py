"""MI355X-native PEFT-BD speculative step: HIP kernels behind a C ABI (libpbd).

``binding`` marshals arguments to the library (the product path); ``costmodel``
holds the paper's host-side cost arithmetic used for reporting; ``build``
compiles the library in-tree for gfx950.
"""
from . import binding, costmodel  # noqa: F401
from .binding import Engine, load_library, make_config, upload_weights  # noqa: F401
