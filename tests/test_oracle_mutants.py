"""Planted mistakes in the oracle, on the CPU: each plausible slip in
pic_oracle.c (a dropped term, a wrong sign or index, a transposed operand, a
misplaced clamp) is compiled into a throw-away copy, and at least one pin in
tests/pins.py must reject that copy.  This shows the pins constrain every part
of the oracle, not just that the oracle agrees with itself."""
import os
import re
import tempfile

import pytest

import oracle
from oracle import build as obuild
from tests import pins

# (name, exact source fragment, replacement): pic_oracle.c (synthesis step)
MUTANTS = [
    ("drop_bias", "acc += (double)bias[bo + j];", ""),
    ("transpose_weights", "long idx = wo + (long)j * fin + i;\n                        double wv",
     "long idx = wo + (long)i * fout + j;\n                        double wv"),
    ("relu_on_last_layer", "g[j] = (l < nl - 1 && acc < 0.0) ? 0.0 : acc;",
     "g[j] = (acc < 0.0) ? 0.0 : acc;"),
    ("no_relu", "g[j] = (l < nl - 1 && acc < 0.0) ? 0.0 : acc;", "g[j] = acc;"),
    ("no_half_pixel", "double sy = ((double)y + 0.5) / f - 0.5;", "double sy = (double)y / f;"),
    ("swap_axes", "double ly = sy - y0, lx = sx - x0;", "double ly = sx - x0, lx = sy - y0;"),
    ("wrap_edge", "floor(sx);\n    int y1 = y0 + 1 < hk ? y0 + 1 : hk - 1;",
     "floor(sx);\n    int y1 = y0 + 1 < hk ? y0 + 1 : 0;"),
    ("no_low_clamp", "    if (sx < 0.0) sx = 0.0;\n    int y0", "    int y0"),
    ("flipped_lerp", "double top = (1.0 - lx) * a + lx * b;", "double top = lx * a + (1.0 - lx) * b;"),
    ("levels_reversed", "h[k] = upsample_f64(grid, hk[k], wk[k], k, y, x);",
     "h[L - 1 - k] = upsample_f64(grid, hk[k], wk[k], k, y, x);"),
    ("floor_level_dims", "return (int)((n + f - 1) / f);", "return (int)(n / f);"),
    ("u8_truncates", "((uint8_t *)out)[o] = (uint8_t)floor(255.0 * cl + 0.5);",
     "((uint8_t *)out)[o] = (uint8_t)floor(255.0 * cl);"),
    ("no_upper_clamp", "double cl = v < 0.0 ? 0.0 : (v > 1.0 ? 1.0 : v);",
     "double cl = v < 0.0 ? 0.0 : v;"),
    ("wrong_output_plane",
     "size_t o = (((size_t)b * 3 + c) * R + (y - y_begin)) * (size_t)W + x;\n                double v",
     "size_t o = (((size_t)b * 3 + (2 - c)) * R + (y - y_begin)) * (size_t)W + x;\n                double v"),
    ("f32_model_no_bias", "float acc = bias[bo + j];", "float acc = 0.0f;"),
    ("f32_model_transposed", "long idx = wo + (long)j * fin + i;\n                        float wv",
     "long idx = wo + (long)i * fout + j;\n                        float wv"),
    ("fuse_drops_beta", "mod += w * (double)beta[c];", ""),
    ("fuse_sigma_multiplies", "w_fused[(size_t)o * in + c] = w * (double)gamma[c] / (double)sigma[c];",
     "w_fused[(size_t)o * in + c] = w * (double)gamma[c] * (double)sigma[c];"),
    ("f32_model_u8_truncates", "(uint8_t)floorf(fmaf(cl, 255.0f, 0.5f))", "(uint8_t)floorf(cl * 255.0f)"),
]

# the same for zpr_oracle.c (latents from the ZpR symbol stream)
ZPR_MUTANTS = [
    ("zigzag_direction", "if (d % 2 == 1) {", "if (d % 2 == 0) {"),
    ("run_off_by_one", "int run = s - eob + 17;", "int run = s - eob + 16;"),
    ("run_threshold", "if (s >= eob - 16) {", "if (s >= eob - 17) {"),
    ("block_starts_at_marker", "long begin = g == 0 ? 0 : offsets[g - 1] + 1;",
     "long begin = g == 0 ? 0 : offsets[g - 1];"),
    ("literal_not_zigzagged", "blk[zz[produced]] = s;", "blk[produced] = s;"),
    ("idct_no_dc_norm", "double a = u == 0 ? sqrt(1.0 / 8.0) : 0.5;", "double a = 0.5;"),
    ("idct_transposed", "acc += C[x][u] * C[y][v] * S[u * 8 + v];", "acc += C[x][u] * C[y][v] * S[v * 8 + u];"),
    ("idct_cos_phase", "cos((2 * x + 1) * u * pi / 16.0)", "cos((2 * x) * u * pi / 16.0)"),
    ("idct_basis_transposed", "acc += C[x][u] * C[y][v] * S[u * 8 + v];", "acc += C[u][x] * C[v][y] * S[u * 8 + v];"),
    ("levels_finest_first", "for (int k = L - 1; k >= 0; --k) {", "for (int k = 0; k < L; ++k) {"),
    ("patch_grid_transposed", "int y = py * 8 + r, x = px * 8 + c;", "int y = px * 8 + r, x = py * 8 + c;"),
    ("patch_inner_transposed", "grid[(size_t)y * wk + x] = blk[r * 8 + c];",
     "grid[(size_t)y * wk + x] = blk[c * 8 + r];"),
    ("no_count_check", "if (m != nb || (n > 0 && symbols[n - 1] != eob))", "if (m > nb)"),
    ("symbol_above_eob_is_a_run", "if (s > eob) {\n                err |= ZO_ERR_SYMBOL;\n                continue;\n            }",
     ""),
    ("no_symbol_count_limit", "if (produced > 64 || end - begin > 64)", "if (produced > 64)"),
]

# the same for huff_oracle.c (symbols from the Huffman bitstream)
HUFF_MUTANTS = [
    ("lsb_first", "(bits[pos >> 3] >> (7 - (pos & 7))) & 1u", "(bits[pos >> 3] >> (pos & 7)) & 1u"),
    ("canonical_no_shift", "code = (code + (uint32_t)count[l - 1]) << 1;", "code = code + (uint32_t)count[l - 1];"),
    ("canonical_count_off_by_one", "code = (code + (uint32_t)count[l - 1]) << 1;",
     "code = (code + (uint32_t)count[l]) << 1;"),
    ("kraft_unchecked", "if (kraft > (1LL << HO_MAX_LEN))\n        return HO_ERR_TABLE;", ""),
    ("match_ignores_length", "if (lengths[i] == len && codes[i] == acc) {", "if (codes[i] == acc) {"),
    ("no_prefix_check", "if (found < 0 && !longer) {", "if (0) {"),
    ("value_is_index", "out[s] = values[found];", "out[s] = found;"),
]


def _caught(orc):
    for check in pins.ALL_CHECKS:
        try:
            check(orc)
        except (AssertionError, ValueError):
            return check.__name__
    return None


CASES = ([(obuild.SRC,) + m for m in MUTANTS] + [(obuild.ZPR_SRC,) + m for m in ZPR_MUTANTS] +
         [(obuild.HUFF_SRC,) + m for m in HUFF_MUTANTS])


@pytest.mark.parametrize("path,name,old,new", CASES, ids=[c[1] for c in CASES])
def test_mutant_is_caught(path, name, old, new, tmp_path):
    src = open(path).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique in {os.path.basename(path)}"
    mutated = src.replace(old, new)
    csrc = tmp_path / os.path.basename(path)
    csrc.write_text(mutated)
    srcs = [str(csrc) if s == path else s for s in obuild.SRCS]
    lib = str(tmp_path / f"libmutant_{name}.so")
    obuild.build(srcs=srcs, out=lib)
    orc = oracle.Oracle(lib)
    assert _caught(orc) is not None, f"no pin rejects the {name} mutant"
