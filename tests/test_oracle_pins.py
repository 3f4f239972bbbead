"""The CPU oracle against its pins (see tests/pins.py for what pins what)."""
import pytest

import oracle
from tests import pins


@pytest.fixture(scope="module")
def orc():
    return oracle.default()


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(orc, check):
    check(orc)


def test_rejects_bad_arguments(orc):
    import numpy as np
    lat = [np.zeros((1, 4, 4), np.float32), np.zeros((1, 2, 2), np.float32)]
    w = np.zeros((1, 2 * 4 + 4 * 3), np.float32)
    b = np.zeros((1, 7), np.float32)
    with pytest.raises(ValueError):       # widths[0] != number of levels
        orc.decode(lat, w, b, (3, 4, 3), 4, 4)
    with pytest.raises(ValueError):       # last width != 3
        orc.decode(lat, w, b, (2, 4, 4), 4, 4)
    with pytest.raises(ValueError):       # level 1 has the wrong shape
        orc.decode([lat[0], np.zeros((1, 3, 2), np.float32)], w, b, (2, 4, 3), 4, 4)


def test_row_range_matches_full_decode(orc):
    import numpy as np
    from paper_2609_09020_amd import synth
    inp = synth.make_inputs(37, 29, 4, (4, 9, 3), batch=2, seed=1, latent="normal", bias="normal")
    full = orc.decode_inputs(inp, out="raw")
    for rows in ((0, 37), (0, 1), (36, 37), (5, 20)):
        part = orc.decode_inputs(inp, out="raw", rows=rows)
        assert np.array_equal(full[:, :, rows[0]:rows[1]], part)
