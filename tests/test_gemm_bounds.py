"""Host-side model of the bf16 GEMM's operand loads (csrc/gemm.hip): every
byte a load touches lies inside the operand, for ragged and exact tiles.

The kernel forms each 16-byte load from a buffer descriptor (base = first
row of the tile, range = bytes up to the end of the operand's last row), a
lane offset (row inside an 8-row piece and a swizzled 16-byte chunk) and a
scalar offset (the piece's first row, clamped to the last in-bounds piece,
plus the K step).  The hardware zero-fills a load whose lane offset is past
the range and does not range-check the scalar offset, so the scalar part
alone must keep every load inside the operand.  This model recomputes those
offsets the same way for every tile row, wave, piece, lane and K step."""
import numpy as np
import pytest

BM, BK, WAVES, LOADS = 256, 64, 4, 8


def load_extents(M, K, ld, ragged_rows=None):
    """(lowest, highest) byte touched by the loads of every tile, relative to
    the operand's base, for all K steps the kernel issues (0 .. max(K/64, 4))."""
    tiles = (M + BM - 1) // BM
    kt = K // BK
    lane = np.arange(64)
    lo, hi = np.inf, -np.inf
    for tm in range(tiles):
        m0 = tm * BM
        n_rec = ((M - m0 - 1) * ld + K) * 2
        rmax = max(min(M - m0, BM) - 8, 0)
        for wave in range(WAVES):
            for u in range(LOADS):
                q = LOADS * wave + u
                par = q & 1
                c = (lane & 7) ^ (4 * par + (lane >> 4))
                vo = (lane >> 3) * ld * 2 + c * 16
                live = vo < n_rec                       # otherwise zero-filled, nothing read
                if not live.any():
                    continue
                # the prologue issues steps 0..3, the loop steps up to K/64 - 1
                steps = np.minimum(np.arange(max(kt, 4)), kt - 1) * BK * 2
                base = m0 * ld * 2 + min(8 * q, rmax) * 2 * ld
                lo = min(lo, base + vo[live].min() + steps.min())
                hi = max(hi, base + vo[live].max() + steps.max() + 15)
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


def test_unclamped_offsets_would_leave_the_operand():
    """Without the clamp (scalar offset = 8 q rows) the 720p ragged tile reads
    past the end: what the clamp is there for."""
    M, K, ld = 75600, 5120, 5120
    m0 = (M // BM) * BM
    worst = m0 * ld * 2 + (8 * (LOADS * WAVES - 1) + 7) * ld * 2 + (K - 1) * 2
    assert worst > ((M - 1) * ld + K) * 2 - 1
