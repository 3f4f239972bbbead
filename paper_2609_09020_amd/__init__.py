"""PIC synthesis decoder for AMD Instinct MI355X (gfx950).

The decoder's per-pixel synthesis (PIC, Sec. 3.1 and App. A): upsample every
level of a latent pyramid to full resolution and evaluate a small ReLU MLP per
pixel to RGB.  The work runs in hand-written HIP kernels behind a C ABI
(``include/pic_decode.h``); this package is the thin Python binding over it.
"""

from .decoder import (Decoder, PicError, fuse_modulation, load_library, make_desc,  # noqa: F401
                      pic_decode_create, pic_decode_destroy, pic_decode_query, pic_decode_run,
                      pic_decode_run_layers, pic_fuse_modulation, pic_status_string)
