"""PIC decoder for AMD Instinct MI355X (gfx950).

Three steps of PIC's decoder run in hand-written HIP kernels behind a C ABI:
  * the per-pixel synthesis (Sec. 3.1 and App. A): upsample every level of
    the latent pyramid to full resolution and evaluate a small ReLU MLP per
    pixel to RGB (``include/pic_decode.h``);
  * the latent decoding before it (Sec. 3.3, App. B Alg. 1): expand the ZpR
    symbol stream into 8x8 DCT blocks, inverse-transform them and place them
    in the pyramid (``include/pic_zpr.h``);
  * the entropy decoding before that (Sec. 3.3, Sec. 4.1): the Huffman
    bitstream back to the ZpR symbols (``include/pic_huff.h``).
This package is the thin Python binding over them.
"""

from .decoder import (Decoder, HuffDecoder, PicError, ZprDecoder, fuse_modulation,  # noqa: F401
                      load_library, make_desc, make_huff_desc, make_zpr_desc, pic_huff_create,
                      pic_huff_decode, pic_huff_destroy, pic_huff_query, pic_decode_create, pic_decode_destroy,
                      pic_decode_query, pic_decode_run, pic_decode_run_layers, pic_decode_run_noalloc,
                      pic_fuse_modulation,
                      pic_status_string, pic_zpr_create, pic_zpr_decode, pic_zpr_destroy,
                      pic_zpr_expand, pic_zpr_query)
