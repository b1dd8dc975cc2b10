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


def load_extents(M, K, ld, row_in_lane=True, tile=BM, loads=LOADS):
    """(lowest, highest) byte touched by the loads of every tile, relative to
    the operand's base, for all K steps the kernel issues (0 .. max(K/64, 4)).
    tile / loads: rows of the operand's tile and 1 KiB loads per wave (A: 256
    and 8; W: 256 and 8, or 192 and 6 for the narrow tiles).
    row_in_lane=False models the earlier layout (piece row in the scalar
    offset, outside the range check)."""
    assert tile == 8 * loads * WAVES
    tiles = (M + tile - 1) // tile
    kt = K // BK
    lane = np.arange(64)
    lo, hi = np.inf, -np.inf
    # the prologue issues steps 0..3, the loop steps up to K/64 - 1; a step
    # past the last one reloads the last one
    steps = np.minimum(np.arange(max(kt, 4)), kt - 1) * BK * 2
    for tm in range(tiles):
        m0 = tm * tile
        n_rec = ((M - m0 - 1) * ld + K) * 2
        for wave in range(WAVES):
            for u in range(loads):
                q = loads * wave + u
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


@pytest.mark.parametrize("N,K,ld", [
    (3072, 3072, 3072),      # image block: O, cross-Q, cross-O weights (16 narrow tiles)
    (9216, 3072, 3072),      # image block QKV weight
    (6144, 3072, 3072),      # image block text key/value weight
    (264, 64, 64),           # ragged: 2 narrow tiles, the second with 72 rows
    (2880, 768, 768),        # ragged, the tile-sequence test's weight
    (8, 128, 128),           # fewer rows than one load piece
])
def test_gemm_narrow_tile_weight_loads_stay_inside_operand(N, K, ld):
    lo, hi = load_extents(N, K, ld, tile=192, loads=6)
    last = ((N - 1) * ld + K) * 2 - 1
    assert lo >= 0
    assert hi <= last, f"a load reaches byte {hi}, past the operand's last byte {last}"


def lds_extent(bnt):
    """Highest LDS byte each kind of access of the bf16 GEMM touches, for
    output tiles of 256 x bnt, and the size of the kernel's LDS array."""
    row_bytes, stages, epi = BK * 2, 2, 32 * 256
    tile_a, tile_w = BM * row_bytes, bnt * row_bytes
    stage = tile_a + tile_w
    kla, klw = tile_a // 1024 // WAVES, tile_w // 1024 // WAVES
    wn, ni = bnt // 2, bnt // 64
    total = stages * stage + WAVES * epi
    hi = {}
    lane = np.arange(64)
    for step in range(stages):
        for wave in range(WAVES):
            a_home = step * stage + kla * wave * 1024 + lane * 16
            w_home = step * stage + tile_a + klw * wave * 1024 + lane * 16
            hi["store A"] = max(hi.get("store A", 0), (a_home + (kla - 1) * 1024).max() + 15)
            hi["store W"] = max(hi.get("store W", 0), (w_home + (klw - 1) * 1024).max() + 15)
            wm, wnn = wave >> 1, wave & 1
            fr, fh = lane & 31, lane >> 5
            sw = (fr >> 1) & 7
            for kk in range(4):
                fo_a = (wm * 128 + fr) * row_bytes + (((2 * kk + fh) ^ sw) << 4)
                fo_w = tile_a + (wnn * wn + fr) * row_bytes + (((2 * kk + fh) ^ sw) << 4)
                hi["read A"] = max(hi.get("read A", 0), (step * stage + fo_a + 3 * 32 * row_bytes).max() + 15)
                hi["read W"] = max(hi.get("read W", 0), (step * stage + fo_w + (ni - 1) * 32 * row_bytes).max() + 15)
            # A and W regions of a slot stay apart
            assert (a_home + (kla - 1) * 1024).max() + 15 < step * stage + tile_a
            assert (w_home + (klw - 1) * 1024).max() + 15 < (step + 1) * stage
    for wave in range(WAVES):
        hi["epilogue"] = max(hi.get("epilogue", 0), stages * stage + wave * epi + epi - 1)
    return hi, total


@pytest.mark.parametrize("bnt", [256, 192])
def test_gemm_lds_accesses_stay_inside_the_array(bnt):
    hi, total = lds_extent(bnt)
    for kind, h in hi.items():
        assert h < total, f"{kind} reaches LDS byte {h} of {total}"
    assert total <= 160 * 1024
