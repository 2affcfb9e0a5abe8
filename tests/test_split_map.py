"""The workgroup-to-(row, chunk) map of the split-row softmax kernel
(csrc/softmax.hip, sm_split_kernel), restated and checked on the CPU: a
bijection onto (row, chunk) for every row count and chunk count, and with
the rows a multiple of 8 every chunk of a row on the XCD (blockIdx mod 8) of
its first chunk."""
import pytest


def split_map(b, rows, G):
    if rows % 8 == 0:
        sl = b >> 3
        return (b & 7) + 8 * (sl // G), sl % G
    return b // G, b % G


@pytest.mark.parametrize("rows", [1, 3, 8, 16, 64, 65, 120, 512])
@pytest.mark.parametrize("G", [1, 2, 8, 31, 256])
def test_split_map_is_a_bijection(rows, G):
    seen = {}
    for b in range(rows * G):
        rr, g = split_map(b, rows, G)
        assert 0 <= rr < rows and 0 <= g < G
        assert (rr, g) not in seen
        seen[(rr, g)] = b
    assert len(seen) == rows * G
    if rows % 8 == 0:
        for rr in range(rows):
            assert len({seen[(rr, g)] % 8 for g in range(G)}) == 1
