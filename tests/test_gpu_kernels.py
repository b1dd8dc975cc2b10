"""Per-kernel parity of the HIP path against the CPU oracle, through the C ABI.

Inputs are seeded (synth.draw); both sides read the same stored bits.  Sizes
span several tiles with ragged tails, packed batches of several requests,
single-row and empty requests."""
import numpy as np
import pytest
import torch

import synth
from oracle import dit_block as O
from gpu_util import require_gpu, dev, host, empty, check, log

pytestmark = pytest.mark.gpu


def _cu(lengths):
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)


def _req_of(cu):
    return np.concatenate([np.full(cu[r + 1] - cu[r], r) for r in range(len(cu) - 1)]).astype(np.int64)


# ------------------------------------------------------------------ LayerNorm


@pytest.mark.parametrize("dtype,D,lengths", [
    ("bf16", 3072, [5, 1000, 331]), ("bf16", 5120, [1, 257]), ("f32", 384, [64]), ("f32", 384, [3, 20, 41]),
    ("bf16", 8192, [3, 70]), ("bf16", 576, [33]), ("bf16", 1536, [2, 9]), ("f32", 4096, [9]), ("f32", 2816, [5])])
def test_adaln_modulate(dtype, D, lengths):
    B = require_gpu()
    log(f"case adaln_modulate {dtype} D={D} lengths={lengths}")
    cu = _cu(lengths)
    R, T = len(lengths), int(cu[-1])
    x = synth.draw((T, D), (1, D, T), dtype)
    mod = synth.draw((R, 6, D), (2, D, T), "f32", std=0.5)
    out = empty((T, D), dtype)
    mt = dev(mod)
    B.adaln_modulate(dev(x), mt[:, 3], mt[:, 4], 6 * D, cu, 1e-6, out)
    torch.cuda.synchronize()
    req = _req_of(cu)
    ref = O.modulate(O.layer_norm(O.decode(x), 1e-6), mod[req, 3].astype(np.float64), mod[req, 4].astype(np.float64))
    check(host(out), ref, dtype, "adaln_modulate")


@pytest.mark.parametrize("dtype,D,T", [("bf16", 5120, 777), ("f32", 384, 64), ("bf16", 8192, 37), ("bf16", 704, 50)])
def test_layer_norm_affine(dtype, D, T):
    B = require_gpu()
    log(f"case layer_norm_affine {dtype} D={D} T={T}")
    x = synth.draw((T, D), (3, D), dtype)
    g = synth.draw((D,), (4, D), dtype, mean=1.0, std=0.02)
    b = synth.draw((D,), (5, D), dtype, std=0.02)
    out = empty((T, D), dtype)
    B.layer_norm_affine(dev(x), dev(g), dev(b), 1e-6, out)
    torch.cuda.synchronize()
    ref = O.layer_norm(O.decode(x), 1e-6) * O.decode(g) + O.decode(b)
    check(host(out), ref, dtype, "layer_norm_affine")


# ------------------------------------------------------------------ GEMM

GEMM_CASES = [
    ("bf16", 1000, 768, 1024, [1000]),       # ragged M, several tiles
    ("bf16", 300, 264, 64, [100, 200]),       # N tail (not a multiple of 256), K = one tile
    ("bf16", 4096 + 77, 512, 3072, [4096, 77]),
    # 11 and 16 tile rows: rastered in groups of 8 tile rows (a full group and
    # a tail of 3; more tiles than compute units, so tile sequences)
    ("bf16", 2600, 1024, 384, [2600]),
    ("bf16", 3900, 5120 + 64, 384, [1900, 2000]),
    ("f32", 64, 1536, 384, [64]),
    ("f32", 77, 768, 384, [30, 47]),
]


class forced_tile_n:
    """Force the bf16 GEMM's output tile width (192 or 256) inside a with-block;
    0 (the per-shape choice) again afterwards."""

    def __init__(self, B, tile_n):
        self.B, self.tile_n = B, tile_n

    def __enter__(self):
        self.B.debug_gemm_tile_n(self.tile_n)

    def __exit__(self, *exc):
        self.B.debug_gemm_tile_n(0)


@pytest.mark.parametrize("dtype,M,N,K,lengths", GEMM_CASES)
@pytest.mark.parametrize("epi", [0, 1, 2, 3])
def test_linear(dtype, M, N, K, lengths, epi):
    """bf16: both output tile widths (256 and 192 columns), each against the oracle."""
    B = require_gpu()
    cu = _cu(lengths)
    a = synth.draw((M, K), (10, M, N, K), dtype)
    w = synth.draw((N, K), (11, M, N, K), dtype, std=0.02)
    b = synth.draw((N,), (12, M, N, K), dtype, std=0.02)
    res = synth.draw((M, N), (13, M, N, K), dtype)
    gate = synth.draw((len(lengths), 2 * N), (14, M, N, K), "f32", std=0.7)
    gt = dev(gate)
    z = O.linear(O.decode(a), O.decode(w), O.decode(b))
    if epi == 1:
        z = O.gelu_tanh(z)
    elif epi == 2:
        z = O.decode(res) + z
    elif epi == 3:
        z = O.decode(res) + gate[_req_of(cu), N:].astype(np.float64) * z
    for tile_n in ((256, 192) if dtype == "bf16" else (0,)):
        log(f"case linear {dtype} M={M} N={N} K={K} epi={epi} lengths={lengths} tile_n={tile_n}")
        out = empty((M, N), dtype)
        with forced_tile_n(B, tile_n):
            B.linear(dev(a), dev(w), dev(b), out, epi=epi, res=dev(res) if epi >= 2 else None,
                     gate=gt[:, N:] if epi == 3 else None, gate_stride=2 * N, cu_seqlens=cu if epi == 3 else None)
            torch.cuda.synchronize()
        check(host(out), z, dtype, f"linear epi={epi} tile_n={tile_n}")


@pytest.mark.parametrize("epi", [0, 1, 3])
def test_linear_tile_sequences(epi):
    """More output tiles (49 x 12 = 588, ragged in M and N) than compute units:
    each workgroup runs a sequence of 2 or 3 tiles and loads the next tile's
    first K steps while finishing the current one.  Checked on sampled rows
    covering the first, middle and last row of every tile row."""
    B = require_gpu()
    M, N, K, lengths = 12288 + 77, 2816 + 64, 768, [5000, 7365]
    cu = _cu(lengths)
    a = synth.draw((M, K), (15, M, N, K), "bf16")
    w = synth.draw((N, K), (16, M, N, K), "bf16", std=0.02)
    b = synth.draw((N,), (17, M, N, K), "bf16", std=0.02)
    res = synth.draw((M, N), (18, M, N, K), "bf16")
    gate = synth.draw((len(lengths), N), (19, M, N, K), "f32", std=0.7)
    rows = np.unique(np.concatenate([np.arange(0, M, 256), np.minimum(np.arange(0, M, 256) + 128, M - 1),
                                     np.minimum(np.arange(0, M, 256) + 255, M - 1), [M - 1],
                                     np.random.default_rng(7).integers(0, M, 200)]))
    z = O.linear(O.decode(a[rows]), O.decode(w), O.decode(b))
    if epi == 1:
        z = O.gelu_tanh(z)
    elif epi == 3:
        z = O.decode(res[rows]) + gate[_req_of(cu)[rows]].astype(np.float64) * z
    for tile_n in (256, 192):   # 49 x 12 or 49 x 15 tiles (the last column tile ragged in both)
        log(f"case linear tile sequences M={M} N={N} K={K} epi={epi} tile_n={tile_n}")
        out = empty((M, N), "bf16")
        with forced_tile_n(B, tile_n):
            B.linear(dev(a), dev(w), dev(b), out, epi=epi, res=dev(res) if epi >= 2 else None,
                     gate=dev(gate) if epi == 3 else None, gate_stride=N, cu_seqlens=cu if epi == 3 else None)
            torch.cuda.synchronize()
        check(host(out)[rows], z, "bf16", f"linear tile sequences epi={epi} tile_n={tile_n}")


def test_linear_inplace_residual():
    """res == out (the block updates x1 in place)."""
    B = require_gpu()
    log("case linear in-place residual bf16 M=515 N=512 K=256")
    M, N, K = 515, 512, 256
    a = synth.draw((M, K), (15,), "bf16")
    w = synth.draw((N, K), (16,), "bf16", std=0.05)
    r = synth.draw((M, N), (17,), "bf16")
    out = dev(r)
    B.linear(dev(a), dev(w), None, out, epi=2, res=out)
    torch.cuda.synchronize()
    check(host(out), O.decode(r) + O.linear(O.decode(a), O.decode(w), None), "bf16", "in-place residual")


# ------------------------------------------------------------ RMSNorm + rotary


@pytest.mark.parametrize("dtype,H,d,sections,lengths,grids,offsets", [
    ("bf16", 4, 128, (44, 42, 42), [700, 500], [(3, 10, 30), (2, 20, 20)], [0, 100]),
    ("bf16", 3, 128, (0, 64, 64), [1, 300], [(1, 4, 4), (1, 20, 16)], [5, 19]),
    ("f32", 6, 64, (0, 32, 32), [64], [(1, 8, 8)], [0]),
    ("bf16", 40, 128, (44, 42, 42), [90, 31], [(2, 9, 5), (1, 5, 7)], [0, 3]),
    ("bf16", 70, 128, (44, 42, 42), [20], [(1, 4, 5)], [0]),
    ("f32", 100, 64, (20, 22, 22), [17], [(1, 1, 17)], [0]),
])
def test_qk_norm_rope(dtype, H, d, sections, lengths, grids, offsets):
    B = require_gpu()
    log(f"case qk_norm_rope {dtype} H={H} d={d} sections={sections} lengths={lengths}")
    cu = _cu(lengths)
    T, D = int(cu[-1]), H * d
    qkv = synth.draw((T, 3 * D), (20, H, T), dtype)
    gq = synth.draw((d,), (21, H), dtype, mean=1.0, std=0.1)
    gk = synth.draw((d,), (22, H), dtype, mean=1.0, std=0.1)
    t = dev(qkv)
    vl = B.Varlen(cu, None, grids, offsets)
    B.qk_norm_rope(t[:, :D], t[:, D:2 * D], H, d, dev(gq), dev(gk), 1e-6, sections, 10000.0, vl)
    torch.cuda.synchronize()
    g = host(t)
    src = O.decode(qkv)
    cfg = O.BlockConfig(hidden=D, n_heads=H, head_dim=d, mlp_hidden=4, freq_dim=4, rope_sections=sections)
    ovl = O.Varlen(list(cu), [0] * len(cu), grids, offsets)
    rq = O.rope_for_rows(O.rms_norm_heads(src[:, :D], O.decode(gq), H, d, 1e-6), cfg, ovl)
    rk = O.rope_for_rows(O.rms_norm_heads(src[:, D:2 * D], O.decode(gk), H, d, 1e-6), cfg, ovl)
    check(g[:, :D], rq, dtype, "q")
    check(g[:, D:2 * D], rk, dtype, "k")
    assert np.array_equal(g[:, 2 * D:], src[:, 2 * D:]), "v must be untouched"


def test_rms_norm_only():
    """RMSNorm without rotary and without a second tensor (cross-attention query)."""
    B = require_gpu()
    log("case rms_norm only bf16 H=5 T=333")
    H, d, T = 5, 128, 333
    q = synth.draw((T, 2 * H * d), (23,), "bf16")
    g = synth.draw((d,), (24,), "bf16", mean=1.0, std=0.1)
    t = dev(q)
    B.qk_norm_rope(t[:, :H * d], None, H, d, dev(g), None, 1e-6)
    torch.cuda.synchronize()
    out = host(t)
    check(out[:, :H * d], O.rms_norm_heads(O.decode(q)[:, :H * d], O.decode(g), H, d, 1e-6), "bf16", "rms only")
    assert np.array_equal(out[:, H * d:], O.decode(q)[:, H * d:])


# ------------------------------------------------------------------ attention

ATTN_CASES = [
    # dtype, heads, d, query lengths, key lengths (None = self-attention)
    ("bf16", 3, 128, [1, 255, 256, 700, 64], None),
    ("bf16", 2, 128, [100, 0, 513], [77, 40, 512]),
    ("bf16", 1, 128, [2048], None),
    # the 8-wave shape (a key range over 1024) with requests of 1 to 5 key
    # tiles beside a long one: the loop's first, steady, tail and last steps
    ("bf16", 2, 128, [1100, 1, 64, 65, 190, 256, 257, 320], None),
    # the 4-wave shape with 2, 3, 4 and 16 key tiles
    ("bf16", 2, 128, [65, 129, 193, 5], [65, 129, 193, 1000]),
    ("f32", 6, 64, [64], None),
    ("f32", 6, 64, [64], [77]),
    ("f32", 2, 128, [5, 30], [7, 1]),
]


@pytest.mark.parametrize("dtype,H,d,lq,lk", ATTN_CASES)
def test_attention_varlen(dtype, H, d, lq, lk):
    B = require_gpu()
    log(f"case attention {dtype} H={H} d={d} lq={lq} lk={lk}")
    cu_q = _cu(lq)
    cu_k = cu_q if lk is None else _cu(lk)
    Tq, Tk, W = int(cu_q[-1]), int(cu_k[-1]), H * d
    # q, k, v as strided views of packed buffers, like the block's qkv
    qb = synth.draw((Tq, 3 * W), (30, H, Tq, Tk), dtype)
    kvb = synth.draw((Tk, 2 * W), (31, H, Tq, Tk), dtype)
    qt, kvt = dev(qb), dev(kvb)
    out = empty((Tq, W), dtype)
    B.attention_varlen(qt[:, :W], kvt[:, :W], kvt[:, W:], out, cu_q, cu_k, H, d)
    torch.cuda.synchronize()
    ref = O.attention_varlen(O.decode(qb)[:, :W], O.decode(kvb)[:, :W], O.decode(kvb)[:, W:], cu_q, cu_k, H, d)
    check(host(out), ref, dtype, "attention")


class forced_attention_split:
    """Force the bf16 attention's split into key pieces (2 or 4) inside a
    with-block; the choice per shape again afterwards."""

    def __init__(self, B, mode):
        self.B, self.mode = B, mode

    def __enter__(self):
        self.B.debug_attention_split(self.mode)

    def __exit__(self, *exc):
        self.B.debug_attention_split(0)


SPLIT_CASES = [
    # heads, query lengths, key lengths (None = self-attention)
    (2, [3000], None),                 # all 24 items split; keys ragged (47 tiles of 64, the last of 56)
    (2, [2600, 2100], None),           # the second request's 18 items split, the first's run whole
    (1, [300, 200], [4000, 2100]),     # cross-shaped ranges over 1024 keys, ragged in queries and keys
]


@pytest.mark.parametrize("pieces", [2, 4])
@pytest.mark.parametrize("H,lq,lk", SPLIT_CASES)
def test_attention_split_into_key_pieces(H, lq, lk, pieces):
    """Work items computed as 2 or 4 key pieces and merged equal the oracle;
    a second split call right after (another shape) reuses the pieces' array
    and is correct too."""
    B = require_gpu()
    d = 128
    cu_q = _cu(lq)
    cu_k = cu_q if lk is None else _cu(lk)
    Tq, Tk, W = int(cu_q[-1]), int(cu_k[-1]), H * d
    qb = synth.draw((Tq, W), (34, H, Tq, Tk), "bf16")
    kvb = synth.draw((Tk, 2 * W), (35, H, Tq, Tk), "bf16")
    ref = O.attention_varlen(O.decode(qb), O.decode(kvb)[:, :W], O.decode(kvb)[:, W:], cu_q, cu_k, H, d)
    # the second call: one request of 2500 rows, 1 head, self-attention
    qb2 = synth.draw((2500, 3 * d), (36, 1, 2500), "bf16")
    ref2 = O.attention_varlen(O.decode(qb2)[:, :d], O.decode(qb2)[:, d:2 * d], O.decode(qb2)[:, 2 * d:],
                              _cu([2500]), _cu([2500]), 1, d)
    log(f"case attention split H={H} lq={lq} lk={lk} pieces={pieces}")
    qt, kvt, q2 = dev(qb), dev(kvb), dev(qb2)
    out, out2 = empty((Tq, W), "bf16"), empty((2500, d), "bf16")
    with forced_attention_split(B, pieces):
        B.attention_varlen(qt, kvt[:, :W], kvt[:, W:], out, cu_q, cu_k, H, d)
        B.attention_varlen(q2[:, :d], q2[:, d:2 * d], q2[:, 2 * d:], out2, _cu([2500]), _cu([2500]), 1, d)
        torch.cuda.synchronize()
    check(host(out), ref, "bf16", f"attention split into {pieces}")
    check(host(out2), ref2, "bf16", f"attention split into {pieces}, second call")


class forced_attention_shape:
    """Force the bf16 attention's kernel shape (4 or 8 waves) and its split
    setting inside a with-block; the choices per call again afterwards."""

    def __init__(self, B, waves, split=0):
        self.B, self.waves, self.split = B, waves, split

    def __enter__(self):
        self.B.debug_attention_shape(self.waves)
        self.B.debug_attention_split(self.split)

    def __exit__(self, *exc):
        self.B.debug_attention_shape(0)
        self.B.debug_attention_split(0)


SHAPE_CASES = [
    # heads, query lengths, key lengths (None = self-attention), all over 1024 keys
    (2, [3000], None),                     # 47 key tiles, the last of 56 keys
    (2, [2600, 2100, 70], None),           # packed, ragged in queries and keys
    (1, [300, 200], [4000, 2100]),         # cross-shaped ranges
]


@pytest.mark.parametrize("H,lq,lk", SHAPE_CASES)
def test_attention_four_wave_shape_on_long_ranges(H, lq, lk):
    """The 4-wave shape (128 query rows per workgroup) forced on key ranges
    over 1024 equals the oracle, and the 8-wave shape without a split gives
    the same bits."""
    B = require_gpu()
    d = 128
    cu_q = _cu(lq)
    cu_k = cu_q if lk is None else _cu(lk)
    Tq, Tk, W = int(cu_q[-1]), int(cu_k[-1]), H * d
    qb = synth.draw((Tq, W), (37, H, Tq, Tk), "bf16")
    kvb = synth.draw((Tk, 2 * W), (38, H, Tq, Tk), "bf16")
    ref = O.attention_varlen(O.decode(qb), O.decode(kvb)[:, :W], O.decode(kvb)[:, W:], cu_q, cu_k, H, d)
    log(f"case attention 4-wave shape H={H} lq={lq} lk={lk}")
    qt, kvt = dev(qb), dev(kvb)
    out4, out8 = empty((Tq, W), "bf16"), empty((Tq, W), "bf16")
    with forced_attention_shape(B, 4):
        B.attention_varlen(qt, kvt[:, :W], kvt[:, W:], out4, cu_q, cu_k, H, d)
        torch.cuda.synchronize()
    with forced_attention_shape(B, 8, split=1):
        B.attention_varlen(qt, kvt[:, :W], kvt[:, W:], out8, cu_q, cu_k, H, d)
        torch.cuda.synchronize()
    check(host(out4), ref, "bf16", "attention, 4-wave shape")
    assert torch.equal(out4, out8), "the two shapes differ"


def test_attention_short_launch_takes_four_waves():
    """One request of 4,000 tokens x 24 heads (the image block's shape, ragged
    keys): its 8-wave items would end in a split last round, and the launch
    is short, so on 256 compute units it runs the 4-wave shape.  The first
    and last row of every 128-row query tile and the last rows equal the
    oracle, and the output equals the 8-wave shape's without a split."""
    B = require_gpu()
    H, d, T = 24, 128, 4000
    W = H * d
    cu = _cu([T])
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    waves = B.debug_attention_plan(cu, cu, H, cus)[0]
    log(f"case attention short launch H={H} T={T} on {cus} CUs: {waves} waves")
    if waves != 4:
        pytest.skip(f"{cus} compute units: the launch does not take the 4-wave shape")
    qkv = synth.draw((T, 3 * W), (39, H, T), "bf16")
    t = dev(qkv)
    out, out8 = empty((T, W), "bf16"), empty((T, W), "bf16")
    B.attention_varlen(t[:, :W], t[:, W:2 * W], t[:, 2 * W:], out, cu, cu, H, d)
    with forced_attention_shape(B, 8, split=1):
        B.attention_varlen(t[:, :W], t[:, W:2 * W], t[:, 2 * W:], out8, cu, cu, H, d)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.arange(0, T, 128), np.arange(127, T, 128), np.arange(T - 8, T)]))
    src = O.decode(qkv)
    ref = O.attention_varlen(src[:, :W], src[:, W:2 * W], src[:, 2 * W:], cu, cu, H, d, q_rows=rows)
    check(host(out)[rows], ref, "bf16", "attention, short launch")
    assert torch.equal(out, out8), "the two shapes differ"


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_attention_request_without_keys(dtype, d):
    """A request with queries but no keys gets rows of zeros; the packed
    request beside it still matches the oracle (its keys start at row 0)."""
    B = require_gpu()
    log(f"case attention without keys {dtype} d={d}")
    H, lq, lk = 2, [50, 30], [0, 70]
    cu_q, cu_k = _cu(lq), _cu(lk)
    W = H * d
    qb = synth.draw((80, 3 * W), (32, H, 80, 70), dtype)
    kvb = synth.draw((70, 2 * W), (33, H, 80, 70), dtype)
    qt, kvt = dev(qb), dev(kvb)
    out = dev(np.full((80, W), 7.0, dtype=np.float32)).to(qt.dtype)   # poison: every row is written
    B.attention_varlen(qt[:, :W], kvt[:, :W], kvt[:, W:], out, cu_q, cu_k, H, d)
    torch.cuda.synchronize()
    got = host(out)
    assert np.all(got[:50] == 0.0)
    ref = O.attention_varlen(O.decode(qb)[50:, :W], O.decode(kvb)[:, :W], O.decode(kvb)[:, W:], [0, 30], [0, 70], H, d)
    check(got[50:], ref, dtype, "attention")


@pytest.mark.parametrize("jump_key,big_val", [(100, 20.0), (1999, 20.0), (1500, 10.0)])
def test_attention_late_score_jump(jump_key, big_val):
    """A key far past the first tile whose score exceeds every earlier one by
    far more than the kernel's softmax headroom (2^64).  Key = 20 * ones
    scores 0.5 * 20 * 128 / sqrt(128) = 113 (163 in log2 units): its
    probability overflows fp32, the row sum is inf and the exact row max has
    to be found.  Key = 10 * ones scores 82 in log2 units: the row sum stays
    finite but above 2^64 and one recomputation with a shifted reference
    suffices."""
    B = require_gpu()
    log(f"case attention late score jump key={jump_key} value={big_val}")
    H, d, n = 2, 128, 2048
    W = H * d
    qkv = synth.draw((n, 3 * W), (33, jump_key), "bf16").copy()
    half = np.float32(0.5).view(np.uint32) >> 16          # bf16 bits of 0.5
    big = np.float32(big_val).view(np.uint32) >> 16
    qkv[:, :W] = half                                      # every query = 0.5 * ones
    qkv[jump_key, W:2 * W] = big                           # one key = big_val * ones
    t = dev(qkv)
    out = empty((n, W), "bf16")
    cu = [0, n]
    B.attention_varlen(t[:, :W], t[:, W:2 * W], t[:, 2 * W:], out, cu, cu, H, d)
    torch.cuda.synchronize()
    x = O.decode(qkv)
    ref = O.attention_varlen(x[:, :W], x[:, W:2 * W], x[:, 2 * W:], cu, cu, H, d)
    check(host(out), ref, "bf16", "attention late jump")


def test_attention_varlen_no_leakage():
    """A packed batch equals each request run alone (bitwise: same tiles)."""
    B = require_gpu()
    log("case attention packed vs alone bf16")
    H, d, lens = 2, 128, [300, 129, 600]
    cu = _cu(lens)
    W = H * d
    qkv = dev(synth.draw((int(cu[-1]), 3 * W), (32,), "bf16"))
    packed = empty((int(cu[-1]), W), "bf16")
    B.attention_varlen(qkv[:, :W], qkv[:, W:2 * W], qkv[:, 2 * W:], packed, cu, cu, H, d)
    for r in range(len(lens)):
        a, b = int(cu[r]), int(cu[r + 1])
        one = empty((b - a, W), "bf16")
        sub = qkv[a:b]
        B.attention_varlen(sub[:, :W], sub[:, W:2 * W], sub[:, 2 * W:], one, [0, b - a], [0, b - a], H, d)
        torch.cuda.synchronize()
        assert torch.equal(one, packed[a:b]), f"request {r} differs when packed"


# ------------------------------------------------------------ gated residual


@pytest.mark.parametrize("dtype,D,lengths", [("bf16", 3072, [10, 500, 3]), ("f32", 384, [64]), ("bf16", 8192, [7, 2]), ("f32", 4096, [5]), ("bf16", 5120, [33])])
def test_gated_residual(dtype, D, lengths):
    B = require_gpu()
    log(f"case gated_residual {dtype} D={D} lengths={lengths}")
    cu = _cu(lengths)
    T, R = int(cu[-1]), len(lengths)
    x = synth.draw((T, D), (40, D), dtype)
    z = synth.draw((T, D), (41, D), dtype)
    b = synth.draw((D,), (42, D), dtype, std=0.02)
    g = synth.draw((R, 6 * D), (43, D), "f32", std=0.7)
    out = empty((T, D), dtype)
    gt = dev(g)
    B.gated_residual(dev(x), dev(z), dev(b), gt[:, 2 * D:], 6 * D, cu, out)
    torch.cuda.synchronize()
    ref = O.decode(x) + g[_req_of(cu), 2 * D:3 * D].astype(np.float64) * (O.decode(z) + O.decode(b))
    check(host(out), ref, dtype, "gated_residual")


# ------------------------------------------------------------ conditioning


@pytest.mark.parametrize("name,n_req", [("tiny_image_fp32", 1), ("tiny_image_fp32", 3), ("image_1024", 3)])
def test_timestep_modulation(name, n_req):
    B = require_gpu()
    log(f"case timestep_modulation {name} n_req={n_req}")
    wl = synth.get_workload(name)
    names = ["w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada"]
    inp = synth.generate_block_inputs(wl, names)
    t = synth.draw((n_req,), (50, n_req), "f32", dist="uniform", lo=0.0, hi=1000.0)
    d = {k: dev(v) for k, v in inp.items()}
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    cfg = B.BlockConfig(wl.hidden, wl.n_heads, wl.head_dim, wl.mlp_hidden, wl.freq_dim, wl.rope_sections, tdt)
    mod = torch.empty((n_req, 6, wl.hidden), dtype=torch.float32, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    B.timestep_modulation(cfg, B.make_weights(d), dev(t), mod, ws)
    torch.cuda.synchronize()
    ow = {k: O.decode(v) for k, v in inp.items()}
    ref = O.conditioning(t.astype(np.float64), wl.freq_dim, ow)
    check(host(mod), ref, "f32" if wl.dtype == "f32" else "bf16", "modulation")
