"""PIC synthesis decoder for AMD Instinct MI355X (gfx950).

The decoder's per-pixel synthesis (PIC, Sec. 3.1 and App. A): upsample every
level of a latent pyramid to full resolution and evaluate a small ReLU MLP per
pixel to RGB.  The work runs in hand-written HIP kernels behind a C ABI
(``include/pic_decode.h``); this package is the thin Python binding over it.
"""
