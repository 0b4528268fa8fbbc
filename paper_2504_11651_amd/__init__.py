"""DFloat11 lossless BF16 weight decompression for MI355X (gfx950).

``codec`` binds libdf11.so (include/df11.h): host encoder and the HIP
decoder.  ``synth`` generates seeded synthetic LLM-shaped BF16 weights.
"""
from . import codec, synth  # noqa: F401
from .codec import (DeviceStream, HostStream, build_codebook, decode_block, encode,  # noqa: F401
                    make_layout, to_device, validate)
