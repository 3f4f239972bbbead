"""Pins of the CPU oracle: checks against things other than the oracle itself.

Each ``check_*`` takes an oracle object (anything with ``decode``,
``upsample`` and ``level_dim`` like the ``oracle`` package) and raises
AssertionError on a mismatch.  ``test_oracle_pins.py`` runs them on the real
oracle; ``test_oracle_mutants.py`` runs them on deliberately broken copies of
the oracle's C source to show that each plausible slip is caught.

What pins what (PIC, Sec. 3.1 Eq. (2) for the pyramid, Sec. 4.1 and App. A
for the MLP):
  * level sizes        -- Eq. (2)'s H / 2^k for divisible sizes, the smallest
                          covering grid otherwise (brute force);
  * upsample           -- torch's bilinear ``interpolate`` (half-pixel,
                          scale 2^k) in fp64, a tent-kernel formulation in exact
                          rationals, constant and affine-ramp closed forms;
  * MLP                -- torch fp64 ``linear``/``relu`` on non-square layers
                          with nonzero biases, the relu(x) - relu(-x) identity
                          net, zero weights leaving the output bias;
  * epilogue           -- clamp and floor(255 c + 1/2) closed forms;
  * whole decode       -- exact rational brute force on tiny images.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np
import torch
import torch.nn.functional as F

from paper_2609_09020_amd import synth


# --------------------------------------------------------------- helpers

def _rand_latents(rng, H, W, L, batch=1, kind="int", scale=8):
    out = []
    for k in range(L):
        h, w = -(-H // (1 << k)), -(-W // (1 << k))
        if kind == "int":
            a = rng.integers(-scale, scale + 1, size=(batch, h, w)).astype(np.float32)
        else:
            a = rng.normal(0, scale, size=(batch, h, w)).astype(np.float32)
        out.append(a)
    return out


def _identity_net(L, channels):
    """relu(x) - relu(-x) = x: L -> 2L -> 2L -> 3 passing through the three
    given input channels exactly (weights [out][in], biases zero)."""
    W1 = np.concatenate([np.eye(L), -np.eye(L)], axis=0)          # [2L][L]
    W2 = np.eye(2 * L)                                              # [2L][2L]
    W3 = np.zeros((3, 2 * L))
    for c, ch in enumerate(channels):
        W3[c, ch] = 1.0
        W3[c, L + ch] = -1.0
    w = np.concatenate([W1.ravel(), W2.ravel(), W3.ravel()]).astype(np.float32)
    b = np.zeros(2 * L + 2 * L + 3, dtype=np.float32)
    return [L, 2 * L, 2 * L, 3], w, b


def _torch_upsample(latents, H, W):
    """torch fp64 bilinear upsample by 2^k with half-pixel centres, cropped."""
    chans = []
    for k, a in enumerate(latents):
        t = torch.from_numpy(a.astype(np.float64))[:, None]
        if k == 0:
            u = t
        else:
            u = F.interpolate(t, scale_factor=float(1 << k), mode="bilinear",
                              align_corners=False)
        assert u.shape[-2] >= H and u.shape[-1] >= W
        chans.append(u[:, 0, :H, :W])
    return torch.stack(chans, dim=1).numpy()


def _frac_decode(latents, weights, biases, widths, H, W):
    """Exact rational decode of one image.  The upsample is written as a
    separable tent (hat) kernel sum over every texel, with the source
    coordinate clamped to the grid: a different formulation from the
    oracle's two-tap interpolation that must agree with it exactly."""
    L = len(latents)
    half = Fraction(1, 2)

    def tent(t):
        t = abs(t)
        return 1 - t if t < 1 else Fraction(0)

    def src(o, k, n):
        s = (o + half) / (1 << k) - half
        return min(max(s, Fraction(0)), Fraction(n - 1))

    out = np.empty((3, H, W), dtype=object)
    nl = len(widths) - 1
    for y in range(H):
        for x in range(W):
            h = []
            for k in range(L):
                g = latents[k]
                hk, wk = g.shape
                sy, sx = src(y, k, hk), src(x, k, wk)
                v = Fraction(0)
                for i in range(hk):
                    ty = tent(sy - i)
                    if ty == 0:
                        continue
                    for j in range(wk):
                        tx = tent(sx - j)
                        if tx:
                            v += Fraction(float(g[i, j])) * ty * tx
                h.append(v)
            wo = bo = 0
            for l in range(nl):
                fin, fout = widths[l], widths[l + 1]
                g2 = []
                for j in range(fout):
                    acc = Fraction(float(biases[bo + j]))
                    for i in range(fin):
                        acc += Fraction(float(weights[wo + j * fin + i])) * h[i]
                    g2.append(max(acc, Fraction(0)) if l < nl - 1 else acc)
                h = g2
                wo += fin * fout
                bo += fout
            for c in range(3):
                out[c, y, x] = h[c]
    return out


# ------------------------------------------------------------------ pins

def check_level_dims(orc):
    # Eq. (2): H / 2^k exactly when divisible.
    for H in (256, 512, 768, 1536, 2048):
        for k in range(8):
            if H % (1 << k) == 0:
                assert orc.level_dim(H, k) == H // (1 << k)
    # Otherwise the smallest grid whose 2^k-times upsample covers H.
    for n in (1, 2, 3, 5, 17, 135, 2160):
        for k in range(10):
            m = 1
            while m * (1 << k) < n:
                m += 1
            assert orc.level_dim(n, k) == m, (n, k)


def check_upsample_constant(orc):
    for (H, W, L) in ((7, 5, 3), (16, 16, 4), (9, 13, 4), (1, 1, 3)):
        lat = []
        for k in range(L):
            h, w = orc.level_dim(H, k), orc.level_dim(W, k)
            lat.append(np.full((1, h, w), float(3 * k - 4.25), dtype=np.float32))
        u = orc.upsample(lat, H, W)
        for k in range(L):
            assert np.all(u[0, k] == 3 * k - 4.25), (H, W, k)


def check_upsample_affine(orc):
    a, b, c = 1.5, -0.75, 2.0
    H, W, L = 24, 40, 4
    lat = []
    for k in range(L):
        h, w = orc.level_dim(H, k), orc.level_dim(W, k)
        i, j = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
        lat.append((a * i + b * j + c).astype(np.float32)[None])
    u = orc.upsample(lat, H, W)
    for k in range(1, L):
        f = 1 << k
        h, w = orc.level_dim(H, k), orc.level_dim(W, k)
        sy = (np.arange(H) + 0.5) / f - 0.5
        sx = (np.arange(W) + 0.5) / f - 0.5
        iy = (sy >= 0) & (sy <= h - 1)
        ix = (sx >= 0) & (sx <= w - 1)
        want = a * sy[:, None] + b * sx[None, :] + c
        got = u[0, k]
        m = iy[:, None] & ix[None, :]
        assert np.array_equal(got[m], want[m]), k


def check_upsample_vs_torch(orc):
    rng = np.random.default_rng(11)
    for (H, W, L, kind) in ((64, 64, 4, "int"), (37, 53, 5, "int"), (48, 80, 6, "normal"),
                            (135, 240, 8, "int"), (3, 5, 3, "normal"), (1, 1, 2, "normal")):
        lat = _rand_latents(rng, H, W, L, batch=2, kind=kind, scale=8)
        got = orc.upsample(lat, H, W)
        want = _torch_upsample(lat, H, W)
        if kind == "int":
            assert np.array_equal(got, want), (H, W, L)
        else:
            np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-13)


def check_identity_net(orc):
    rng = np.random.default_rng(5)
    H, W, L = 21, 34, 5
    lat = _rand_latents(rng, H, W, L, batch=2, kind="normal", scale=4)
    u = orc.upsample(lat, H, W)
    for start in range(L):
        chans = [(start + i) % L for i in range(3)]
        widths, w, b = _identity_net(L, chans)
        wb = np.tile(w, (2, 1))
        bb = np.tile(b, (2, 1))
        raw = orc.decode(lat, wb, bb, widths, H, W, out="raw")
        for c, ch in enumerate(chans):
            assert np.array_equal(raw[:, c], u[:, ch]), (start, c)


def check_mlp_vs_torch(orc):
    rng = np.random.default_rng(7)
    for widths in ((5, 7, 3), (3, 11, 6, 3), (4, 3), (6, 9, 9, 9, 3)):
        H, W, L, batch = 13, 19, widths[0], 2
        lat = _rand_latents(rng, H, W, L, batch=batch, kind="normal", scale=2)
        nw, nb = synth.param_counts(widths)
        wts = rng.normal(0, 0.7, size=(batch, nw)).astype(np.float32)
        bs = rng.normal(0, 0.5, size=(batch, nb)).astype(np.float32)
        raw = orc.decode(lat, wts, bs, widths, H, W, out="raw")
        u = torch.from_numpy(orc.upsample(lat, H, W))           # [B][L][H][W]
        for bi in range(batch):
            h = u[bi].permute(1, 2, 0).reshape(-1, L)           # pixels x L
            wo = bo = 0
            for l in range(len(widths) - 1):
                fin, fout = widths[l], widths[l + 1]
                Wl = torch.from_numpy(wts[bi, wo:wo + fin * fout].astype(np.float64)).view(fout, fin)
                bl = torch.from_numpy(bs[bi, bo:bo + fout].astype(np.float64))
                h = F.linear(h, Wl, bl)
                if l < len(widths) - 2:
                    h = F.relu(h)
                wo += fin * fout
                bo += fout
            want = h.view(H, W, 3).permute(2, 0, 1).numpy()
            np.testing.assert_allclose(raw[bi], want, rtol=1e-12, atol=1e-12)


def check_epilogue_closed_forms(orc):
    # Zero weights: every pixel outputs the last layer's bias; clamp to [0, 1]
    # and quantise as floor(255 c + 1/2).
    H, W, L = 5, 6, 2
    widths = (2, 4, 3)
    lat = [np.ones((1, orc.level_dim(H, k), orc.level_dim(W, k)), np.float32) for k in range(L)]
    nw, nb = synth.param_counts(widths)
    cases = [((0.25, 0.75, 0.5), (64, 191, 128)),
             ((-3.0, 7.0, 1.0), (0, 255, 255)),
             ((0.0, 100 / 255, 0.998), (0, 100, 254))]
    for bias3, codes in cases:
        w = np.zeros((1, nw), np.float32)
        b = np.zeros((1, nb), np.float32)
        b[0, -3:] = bias3
        raw = orc.decode(lat, w, b, widths, H, W, out="raw")
        cl = orc.decode(lat, w, b, widths, H, W, out="clamped")
        q = orc.decode(lat, w, b, widths, H, W, out="u8")
        for c in range(3):
            bv = float(np.float32(bias3[c]))
            assert np.all(raw[0, c] == bv)
            assert np.all(cl[0, c] == min(max(bv, 0.0), 1.0))
            assert np.all(q[0, c] == codes[c]), (bias3, c, q[0, c, 0, 0])
    # Hidden-layer biases pass through ReLU before reaching the output.
    w = np.zeros((1, nw), np.float32)
    b = np.zeros((1, nb), np.float32)
    b[0, :4] = (0.5, -2.0, 0.25, 1.0)                 # hidden biases, ReLU -> (0.5, 0, 0.25, 1)
    w[0, 2 * 4:] = np.array([[1, 1, 0, 0], [0, 1, 1, 0], [0, 0, 0, 1]], np.float32).ravel()
    raw = orc.decode(lat, w, b, widths, H, W, out="raw")
    assert np.all(raw[0, 0] == 0.5) and np.all(raw[0, 1] == 0.25) and np.all(raw[0, 2] == 1.0)


def check_exact_rational(orc):
    rng = np.random.default_rng(3)
    for (H, W, L, widths) in ((4, 4, 2, (2, 4, 3)), (5, 3, 3, (3, 5, 4, 3)), (7, 6, 3, (3, 6, 3))):
        lat = _rand_latents(rng, H, W, L, batch=1, kind="int", scale=6)
        nw, nb = synth.param_counts(widths)
        wts = (rng.integers(-16, 17, size=(1, nw)) / 8).astype(np.float32)   # dyadic
        bs = (rng.integers(-8, 9, size=(1, nb)) / 16).astype(np.float32)
        want = _frac_decode([a[0] for a in lat], wts[0], bs[0], widths, H, W)
        raw = orc.decode(lat, wts, bs, widths, H, W, out="raw")
        q = orc.decode(lat, wts, bs, widths, H, W, out="u8")
        for c in range(3):
            for y in range(H):
                for x in range(W):
                    v = want[c, y, x]
                    assert Fraction(float(raw[0, c, y, x])) == v, (H, W, c, y, x)
                    cl = min(max(v, Fraction(0)), Fraction(1))
                    code = (255 * cl + Fraction(1, 2)).__floor__()
                    assert int(q[0, c, y, x]) == code


def check_f32_model(orc, workloads=("pic64", "kodak768", "uhd4k")):
    """The binary32 model against the fp64 definition: within 1e-5 on
    clamped output, identical upsample for integer latents (dyadic weights),
    and 8-bit codes identical wherever the fp64 value is not within 255e-5 of
    a rounding boundary."""
    for name in workloads:
        wl = synth.WORKLOADS[name]
        inp = synth.workload_inputs(wl)
        # crop to a strip of rows so the check stays fast on the big workloads
        rows = min(wl.height, 64)
        H = rows
        lat = []
        for k in range(wl.levels):
            h = orc.level_dim(H, k)
            lat.append(np.ascontiguousarray(inp.latents[k][:, :h]))
        args = (lat, inp.weights, inp.biases, wl.widths, H, wl.width)
        c64 = orc.decode(*args, out="clamped")
        c32 = orc.decode(*args, out="clamped", precision="f32")
        assert np.max(np.abs(c64 - c32)) <= 1e-5, name
        q64 = orc.decode(*args, out="u8")
        q32 = orc.decode(*args, out="u8", precision="f32")
        t = 255.0 * c64 + 0.5
        safe = np.abs(t - np.round(t)) > 255 * 1e-5
        assert np.array_equal(q64[safe], q32[safe]), name
        assert np.all(np.abs(q64.astype(int) - q32.astype(int)) <= 1)
        # identity net in binary32 exposes the binary32 upsample: exact here
        L = wl.levels
        widths, w, b = _identity_net(L, [0, L // 2, L - 1])
        r32 = orc.decode(lat, w[None], b[None], widths, H, wl.width, out="raw", precision="f32")
        u = orc.upsample(lat, H, wl.width)
        for c, ch in enumerate([0, L // 2, L - 1]):
            assert np.array_equal(r32[0, c].astype(np.float64), u[0, ch]), (name, ch)
    # nonzero biases, non-integer latents, several layers and images
    inp = synth.make_inputs(23, 37, 5, (5, 12, 9, 3), batch=3, seed=4, latent="normal",
                            latent_scale=1.5, bias="normal")
    r64 = orc.decode_inputs(inp, out="raw")
    r32 = orc.decode_inputs(inp, out="raw", precision="f32")
    assert np.max(np.abs(r64 - r32) / np.maximum(1.0, np.abs(r64))) <= 1e-5


def check_bf16_weights(orc):
    rng = np.random.default_rng(9)
    H, W, widths = 11, 9, (3, 8, 3)
    lat = _rand_latents(rng, H, W, 3, batch=2, kind="normal", scale=2)
    nw, nb = synth.param_counts(widths)
    w = rng.normal(0, 0.6, size=(2, nw)).astype(np.float32)
    b = rng.normal(0, 0.2, size=(2, nb)).astype(np.float32)
    bits = synth.f32_to_bf16_bits(w)
    widened = synth.bf16_bits_to_f32(bits)
    for prec in ("f64", "f32"):
        a = orc.decode(lat, w, b, widths, H, W, out="raw", precision=prec, weights_bf16=bits)
        c = orc.decode(lat, widened, b, widths, H, W, out="raw", precision=prec)
        assert np.array_equal(a, c), prec


def check_shared_weights(orc):
    rng = np.random.default_rng(2)
    H, W, widths = 10, 12, (3, 6, 3)
    lat = _rand_latents(rng, H, W, 3, batch=3, kind="normal", scale=2)
    nw, nb = synth.param_counts(widths)
    w = rng.normal(0, 0.6, size=nw).astype(np.float32)
    b = rng.normal(0, 0.2, size=nb).astype(np.float32)
    a = orc.decode(lat, w, b, widths, H, W, out="raw", shared=True)
    c = orc.decode(lat, np.tile(w, (3, 1)), np.tile(b, (3, 1)), widths, H, W, out="raw")
    assert np.array_equal(a, c)


def check_fuse_modulation(orc):
    """App. A: the fused layer applied to raw features equals the layer applied
    to the normalised and modulated features (checked on random features in
    fp64 with numpy, an independent evaluation of the unfused definition);
    gamma = sigma, beta = mu leaves the layer unchanged."""
    rng = np.random.default_rng(17)
    for fin, fout in ((7, 5), (16, 3), (40, 40), (1, 1)):
        W = rng.normal(0, 0.5, size=(fout, fin)).astype(np.float32)
        b = rng.normal(0, 0.5, size=fout).astype(np.float32)
        gamma = rng.normal(1, 0.5, size=fin).astype(np.float32)
        beta = rng.normal(0, 0.5, size=fin).astype(np.float32)
        mu = rng.normal(0, 2, size=fin).astype(np.float32)
        sigma = (np.abs(rng.normal(1, 0.5, size=fin)) + 0.1).astype(np.float32)
        wf, bf = orc.fuse_modulation(W, b, gamma, beta, mu, sigma)
        f = rng.normal(0, 3, size=(200, fin))
        g64, b64, m64, s64 = (a.astype(np.float64) for a in (gamma, beta, mu, sigma))
        unfused = (g64 * (f - m64) / s64 + b64) @ W.astype(np.float64).T + b.astype(np.float64)
        fused = f @ wf.T + bf
        np.testing.assert_allclose(fused, unfused, rtol=1e-12, atol=1e-11)
        wf2, bf2 = orc.fuse_modulation(W, b, sigma, mu, mu, sigma)   # modulation undoes the norm
        np.testing.assert_allclose(wf2, W.astype(np.float64), rtol=1e-15)
        np.testing.assert_allclose(bf2, b.astype(np.float64), rtol=1e-12, atol=1e-12)


ALL_CHECKS = [check_level_dims, check_upsample_constant, check_upsample_affine,
              check_upsample_vs_torch, check_identity_net, check_mlp_vs_torch,
              check_epilogue_closed_forms, check_exact_rational, check_f32_model,
              check_bf16_weights, check_shared_weights, check_fuse_modulation]

# the latent-decoding step (ZpR stream -> pyramid) has its pins in pins_zpr.py
from tests.pins_zpr import ZPR_CHECKS  # noqa: E402

ALL_CHECKS += ZPR_CHECKS

# the entropy-decoding step (Huffman bitstream -> symbols): pins_huff.py
from tests.pins_huff import HUFF_CHECKS  # noqa: E402

ALL_CHECKS += HUFF_CHECKS
