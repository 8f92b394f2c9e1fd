"""Host-side V ring block layout (the map the binding uses to read a ring)."""
import numpy as np
import pytest

from paper_2607_18171_amd.binding import V_BLOCK, v_offsets


@pytest.mark.parametrize("C,d", [(64, 64), (136, 64), (240, 128), (264, 128), (28080, 128)])
def test_v_offsets_layout(C, d):
    off = v_offsets(C, d).numpy()
    assert off.shape == (C, d)
    # a bijection onto the head's C*d elements
    assert np.array_equal(np.sort(off.ravel()), np.arange(C * d))
    # storage built block by block: each block's [slots][d] tile stored d-major
    store = np.concatenate([np.arange(s0, min(s0 + V_BLOCK, C))[None, :].repeat(d, 0).ravel()
                            for s0 in range(0, C, V_BLOCK)])
    dims = np.concatenate([np.arange(d)[:, None].repeat(min(V_BLOCK, C - s0), 1).ravel()
                           for s0 in range(0, C, V_BLOCK)])
    assert np.array_equal(off[store, dims], np.arange(C * d))
    # 8-slot groups (C is a multiple of 8) are contiguous along each row
    g = off[0::8]
    for j in range(1, 8):
        assert np.array_equal(off[j::8], g + j)
