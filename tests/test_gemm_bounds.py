"""Host-side model of the bf16 GEMM's operand loads (csrc/gemm.hip): every
byte a load touches lies inside the operand, for ragged and exact tiles.

The kernel forms each 16-byte load from a buffer descriptor (base = first
row of the tile, range = bytes up to the end of the operand's last row), a
lane offset (the row inside the tile, 8 q + i / 8 for piece q and lane i,
and a swizzled 16-byte chunk) and a scalar offset (the K step).  The
hardware zero-fills a load whose lane offset is past the range and does not
range-check the scalar offset, so the rows past a ragged tile's end must be
caught by the lane offset and the K step must stay inside a row.  This model
recomputes those offsets the same way for every tile row, wave, piece, lane
and K step."""
import numpy as np
import pytest

BM, BK, WAVES, LOADS = 256, 64, 4, 8


def load_extents(M, K, ld, row_in_lane=True):
    """(lowest, highest) byte touched by the loads of every tile, relative to
    the operand's base, for all K steps the kernel issues (0 .. max(K/64, 4)).
    row_in_lane=False models the earlier layout (piece row in the scalar
    offset, outside the range check)."""
    tiles = (M + BM - 1) // BM
    kt = K // BK
    lane = np.arange(64)
    lo, hi = np.inf, -np.inf
    # the prologue issues steps 0..3, the loop steps up to K/64 - 1; a step
    # past the last one reloads the last one
    steps = np.minimum(np.arange(max(kt, 4)), kt - 1) * BK * 2
    for tm in range(tiles):
        m0 = tm * BM
        n_rec = ((M - m0 - 1) * ld + K) * 2
        for wave in range(WAVES):
            for u in range(LOADS):
                q = LOADS * wave + u
                c = (lane & 7) ^ (4 * (q & 1) + (lane >> 4))
                lane_part = (lane >> 3) * ld * 2 + c * 16
                piece = 8 * q * ld * 2
                vo = lane_part + piece if row_in_lane else lane_part
                live = vo < n_rec                       # otherwise zero-filled, nothing read
                if not live.any():
                    continue
                addr = m0 * ld * 2 + vo[live] + (0 if row_in_lane else piece)
                lo = min(lo, addr.min() + steps.min())
                hi = max(hi, addr.max() + steps.max() + 15)
    return lo, hi


@pytest.mark.parametrize("M,K,ld", [
    (75600, 5120, 5120),     # 720p activations: last tile of 80 rows
    (75600, 13824, 13824),   # MLP down operand (the workspace's last region)
    (64, 5120, 5120),        # the step's output projection weight (N = P = 64)
    (5, 128, 136),           # fewer than 8 rows, padded stride
    (256, 64, 64),           # exact tile, a single K step
    (300, 192, 200),         # ragged, odd K step count, padded stride
    (15360, 5120, 5120),     # QKV weight, exact tiles
])
def test_gemm_loads_stay_inside_operand(M, K, ld):
    lo, hi = load_extents(M, K, ld)
    last = ((M - 1) * ld + K) * 2 - 1      # the operand's last byte
    assert lo >= 0
    assert hi <= last, f"a load reaches byte {hi}, past the operand's last byte {last}"


def test_scalar_piece_offset_would_leave_the_operand():
    """With the piece row in the (unchecked) scalar offset, the 720p ragged
    tile reads past the operand's end: what the lane-offset layout prevents."""
    M, K, ld = 75600, 5120, 5120
    lo, hi = load_extents(M, K, ld, row_in_lane=False)
    assert hi > ((M - 1) * ld + K) * 2 - 1
