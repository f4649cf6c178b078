"""Host check of the 32-bit lane offsets of the bf16 DMA kernels.

Every DMA lane reads through a buffer resource whose 64-bit base moves with
the tile or block (csrc/dma.h), plus a per-lane byte offset that must stay
below 2^32 (the offset register is 32 bits; the resource's record count
saturates at 4 GiB - 1).  The offsets below restate each kernel's formula;
the largest pair stride is the ending node's position stride n h 32 at the
largest accepted n = 8192 and h = 64.
"""
import pytest

MAX_N, MAX_H, D = 8192, 64, 32


def s_pos(node, n, h):
    return h * D if node == 0 else n * h * D


def s_row(node, n, h):
    return n * h * D if node == 0 else h * D


def max_offsets(node, n, h):
    """Largest lane byte offset of each DMA stream, per kernel."""
    sp = s_pos(node, n, h)
    sr = s_row(node, n, h)
    nkt = (n + 31) // 32
    hb = (h - 1) * D  # head offset folded into the lane offset (dkdv, db)
    chunk = 8 * 3  # channel chunk 8 c, c <= 3
    return {
        # fwd_dma: K/V tile positions p < 32; bias tiles 0..3 of the query block
        "fwd_dma kv": (31 * sp + chunk) * 2,
        "fwd_dma bias": (3 * nkt * 1024 + 256 * 3) * 4 + 16 * 63,
        # dq_dma: K/V tile positions p < 32; when one resource serves a wave's
        # units, the second row of the group rides in the lane offset (one row
        # stride, QD_ROWS = 2); bias quarters of one tile
        "dq_dma kv": (31 * sp + chunk) * 2 + sr * 2,
        "dq_dma bias": 1024 * 3 + 16 * 63,
        # dkdv_dma: query tile positions p < 32 plus the head; bias tiles 0..3
        "dkdv_dma qda": (31 * sp + hb + chunk) * 2,
        "dkdv_dma bias": (3 * nkt * 1024 + 256 * 3) * 4 + 16 * 63,
        # db_dma: block positions pp < 128 (the block's first key and query
        # are in the base) plus the head
        "db_dma kvq": (127 * sp + hb + chunk) * 2,
        "db_dma lse": ((n - 1) + 32 * 3 + 4 * 7) * 4,
    }


@pytest.mark.parametrize("node", [0, 1])
@pytest.mark.parametrize("n,h", [(MAX_N, MAX_H), (MAX_N, 1), (1056, 64), (4097, 4), (33, 64)])
def test_lane_offsets_fit_32_bits(node, n, h):
    for name, off in max_offsets(node, n, h).items():
        assert off < 2 ** 32, (name, node, n, h, off)


def test_largest_shape_is_the_binding_case():
    # the ending node's db_dma stream at the largest shape is the closest
    # to the limit (127 positions of 524288 elements each)
    worst = max(max_offsets(1, MAX_N, MAX_H).values())
    assert worst == max_offsets(1, MAX_N, MAX_H)["db_dma kvq"]
    assert worst > 0.99 * 2 ** 32 * (4261412864 / 2 ** 32)
