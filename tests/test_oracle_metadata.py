"""Pin the metadata closed form of Sec. VI-F against every printed cell of Table 3."""
import os

import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table3_metadata.txt")


def _rows():
    out = []
    with open(GOLDEN) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            p = line.split()
            out.append((p[0], int(p[1]), int(p[2]), [float(v) for v in p[3:]]))
    return out


@pytest.mark.parametrize("name,rows,cols,cells", _rows())
def test_table3(name, rows, cols, cells):
    for (tr, tc), (kb, pct, bits) in zip([(32, 128), (64, 256)], [cells[0:3], cells[3:6]]):
        m = oracle.metadata_bytes(rows, cols, tr, tc, 12)
        layer_bytes = rows * cols * 2
        assert round(m / 1024, 1) == kb, name
        assert round(100 * m / layer_bytes, 3) == pytest.approx(pct), name
        assert round(16 * m / layer_bytes, 4) == pytest.approx(bits), name
