"""Host-side checks of the device data layouts (CPU only)."""

import pytest


@pytest.mark.parametrize("d", [64, 128])
def test_kv_plane_layouts_are_permutations(d):
    """Every (token, d) of a KV block plane has its own slot in the fragment
    layouts the attention kernels read (K and V planes)."""
    from tests.gpu_pair import kv_plane_index
    k, v = kv_plane_index(16, d)
    for idx in (k, v):
        assert sorted(idx.ravel().tolist()) == list(range(16 * d))
