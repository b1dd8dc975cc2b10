"""Thin ctypes binding of ``libditblock.so`` (argument marshalling only).

Every function here mirrors one ``extern "C"`` entry point of
``include/dit_block.h`` under the same name without the ``dit_`` prefix.
Tensors are torch tensors on the current ROCm device; their data pointers
and ``torch.cuda.current_stream()`` are passed straight through.  Nothing is
computed in Python: if the library is missing, every call raises.
"""
import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libditblock.so")

DIT_OK, DIT_ERR_INVALID_ARG, DIT_ERR_UNSUPPORTED, DIT_ERR_WORKSPACE, DIT_ERR_HIP = 0, -1, -2, -3, -4
DIT_F32, DIT_BF16 = 0, 1
EPI_NONE, EPI_GELU_TANH, EPI_RESIDUAL, EPI_GATED_RESIDUAL = 0, 1, 2, 3
MAX_REQ = 64

WEIGHT_FIELDS = (
    "w_t1", "b_t1", "w_t2", "b_t2", "w_ada", "b_ada",
    "w_qkv", "b_qkv", "g_q", "g_k", "w_o", "b_o",
    "g_ca", "b_ca", "w_cq", "b_cq", "w_ckv", "b_ckv", "g_cq", "g_ck", "w_co", "b_co",
    "w_up", "b_up", "w_dn", "b_dn",
)


class DitError(RuntimeError):
    def __init__(self, status: int, func: str, detail: str):
        self.status = status
        super().__init__(f"{func}: status {status}: {detail}")


class ExtensionMissing(RuntimeError):
    pass


class CConfig(ctypes.Structure):
    _fields_ = [
        ("hidden", ctypes.c_int), ("n_heads", ctypes.c_int), ("head_dim", ctypes.c_int),
        ("mlp_hidden", ctypes.c_int), ("freq_dim", ctypes.c_int),
        ("rope_sections", ctypes.c_int * 3), ("rope_theta", ctypes.c_float),
        ("qk_norm", ctypes.c_int), ("ln_eps", ctypes.c_float), ("rms_eps", ctypes.c_float),
        ("dtype", ctypes.c_int),
    ]


class CWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS]


class CVarlen(ctypes.Structure):
    _fields_ = [
        ("n_req", ctypes.c_int),
        ("cu_seqlens", ctypes.POINTER(ctypes.c_int32)),
        ("cu_seqlens_txt", ctypes.POINTER(ctypes.c_int32)),
        ("grid_fhw", ctypes.POINTER(ctypes.c_int32)),
        ("pos_offset", ctypes.POINTER(ctypes.c_int32)),
    ]


MODEL_FIELDS = ("w_t1", "b_t1", "w_t2", "b_t2", "w_pe", "b_pe", "w_hmod", "b_hmod", "w_out", "b_out")


class CModelConfig(ctypes.Structure):
    _fields_ = [("block", CConfig), ("n_blocks", ctypes.c_int), ("in_channels", ctypes.c_int),
                ("patch", ctypes.c_int * 3)]


class CModelWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in MODEL_FIELDS] + [("blocks", ctypes.POINTER(CWeights))]


class CSimConfig(ctypes.Structure):
    _fields_ = [("n_ranks", ctypes.c_int), ("n_degrees", ctypes.c_int), ("degrees", ctypes.POINTER(ctypes.c_int32)),
                ("n_classes", ctypes.c_int), ("cost_us", ctypes.POINTER(ctypes.c_int64)), ("policy", ctypes.c_int),
                ("group_size", ctypes.c_int)]


class CSimTrace(ctypes.Structure):
    _fields_ = [("n_req", ctypes.c_int64), ("arrival_us", ctypes.POINTER(ctypes.c_int64)),
                ("cls", ctypes.POINTER(ctypes.c_int32)), ("n_steps", ctypes.POINTER(ctypes.c_int32)),
                ("deadline_us", ctypes.POINTER(ctypes.c_int64))]


class CSimResult(ctypes.Structure):
    _fields_ = [("finish_us", ctypes.POINTER(ctypes.c_int64)), ("first_start_us", ctypes.POINTER(ctypes.c_int64)),
                ("dispatches", ctypes.POINTER(ctypes.c_int64)), ("events", ctypes.c_int64)]


SIM_FCFS_GROUPS, SIM_SRTF_GROUPS, SIM_EDF_BESTFIT = 0, 1, 2

MIG_SHARDED, MIG_REPLICATED, MIG_METADATA = 0, 1, 2
MIG_MAX_DIMS = 4


class CMigSlice(ctypes.Structure):
    _fields_ = [("rank", ctypes.c_int32), ("start", ctypes.c_int64 * MIG_MAX_DIMS),
                ("end", ctypes.c_int64 * MIG_MAX_DIMS)]


class CMigField(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("n_dims", ctypes.c_int), ("shape", ctypes.c_int64 * MIG_MAX_DIMS),
                ("elem_bytes", ctypes.c_int), ("n_src", ctypes.c_int), ("src", ctypes.POINTER(CMigSlice)),
                ("n_dst", ctypes.c_int), ("dst", ctypes.POINTER(CMigSlice))]


class CMigEntry(ctypes.Structure):
    _fields_ = [("src_index", ctypes.c_int32), ("dst_index", ctypes.c_int32), ("src_rank", ctypes.c_int32),
                ("dst_rank", ctypes.c_int32), ("src_off", ctypes.c_int64 * MIG_MAX_DIMS),
                ("dst_off", ctypes.c_int64 * MIG_MAX_DIMS), ("extent", ctypes.c_int64 * MIG_MAX_DIMS),
                ("bytes", ctypes.c_int64)]

_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ExtensionMissing(f"{LIB_PATH} not found: build it with paper_2606_13501_amd.build.build()")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    PC, PW, PV = ctypes.POINTER(CConfig), ctypes.POINTER(CWeights), ctypes.POINTER(CVarlen)
    PI = ctypes.POINTER(ctypes.c_int32)
    PM, PMW = ctypes.POINTER(CModelConfig), ctypes.POINTER(CModelWeights)
    sig = {
        "dit_block_workspace_size": (sz, [PC, PV]),
        "dit_block_forward": (i32, [PC, PW, PV, vp, vp, vp, vp, vp, vp, sz, vp]),
        "dit_block_pre_attention": (i32, [PC, PW, PV, vp, vp, vp, vp, vp, sz, vp]),
        "dit_block_post_attention": (i32, [PC, PW, PV, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "dit_timestep_modulation": (i32, [PC, PW, i32, vp, vp, vp, sz, vp]),
        "dit_timestep_modulation_noalloc": (i32, [PC, PW, i32, vp, vp, vp]),
        "dit_attention_varlen": (i32, [vp, vp, vp, vp, i64, i64, i64, i64, PI, PI, i32, i32, i32, f32, i32, vp]),
        "dit_adaln_modulate": (i32, [vp, vp, vp, i64, PI, i32, i32, f32, vp, i32, vp]),
        "dit_layer_norm_affine": (i32, [vp, vp, vp, i64, i32, f32, vp, i32, vp]),
        "dit_linear": (i32, [vp, i64, vp, i64, vp, vp, i64, i64, i32, i32, i32, vp, i64, vp, i64, PI, i32, i32, vp]),
        "dit_qk_norm_rope": (i32, [vp, vp, i64, i64, i32, i32, vp, vp, f32, PI, f32, PV, i32, vp]),
        "dit_gated_residual": (i32, [vp, vp, vp, vp, i64, PI, i32, i32, vp, i32, vp]),
        "dit_text_kv_elems": (sz, [PM, PV]),
        "dit_text_kv": (i32, [PM, PMW, PV, vp, vp, vp]),
        "dit_denoise_workspace_size": (sz, [PM, PV]),
        "dit_denoise_step": (i32, [PM, PMW, PV, vp, vp, vp, vp, vp, vp, sz, vp]),
        "dit_patchify": (i32, [PM, PV, vp, vp, vp]),
        "dit_unpatchify_euler": (i32, [PM, PV, vp, vp, vp, vp, vp]),
        "dit_simulate": (i32, [ctypes.POINTER(CSimConfig), ctypes.POINTER(CSimTrace), ctypes.POINTER(CSimResult)]),
        "dit_migration_plan": (i32, [ctypes.POINTER(CMigField), ctypes.POINTER(CMigEntry), i64,
                                     ctypes.POINTER(ctypes.c_int64)]),
        "dit_migration_execute": (i32, [ctypes.POINTER(CMigField), ctypes.POINTER(CMigEntry), i64,
                                        ctypes.POINTER(vp), ctypes.POINTER(vp), vp]),
        "dit_debug_gemm_tile_n": (i32, [i32]),
        "dit_debug_attention_split": (i32, [i32]),
        "dit_debug_attention_shape": (i32, [i32]),
        "dit_debug_attention_plan": (i32, [ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32), i32, i32, i32,
                                         ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int),
                                         ctypes.POINTER(ctypes.c_int)]),
        "dit_status_string": (ctypes.c_char_p, [i32]),
        "dit_last_error": (ctypes.c_char_p, []),
        "dit_abi_version": (i32, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def exported_symbols() -> Sequence[str]:
    return [n for n in ("dit_block_workspace_size", "dit_block_forward", "dit_block_pre_attention",
                        "dit_block_post_attention", "dit_timestep_modulation",
                        "dit_timestep_modulation_noalloc", "dit_attention_varlen",
                        "dit_adaln_modulate", "dit_layer_norm_affine", "dit_linear", "dit_qk_norm_rope",
                        "dit_gated_residual", "dit_text_kv_elems", "dit_text_kv", "dit_denoise_workspace_size",
                        "dit_denoise_step", "dit_patchify", "dit_unpatchify_euler", "dit_simulate",
                        "dit_migration_plan", "dit_migration_execute", "dit_debug_gemm_tile_n",
                        "dit_debug_attention_split", "dit_debug_attention_shape", "dit_debug_attention_plan",
                        "dit_status_string",
                        "dit_last_error", "dit_abi_version")]


def _check(status: int, func: str):
    if status != DIT_OK:
        detail = lib().dit_last_error().decode()
        raise DitError(status, func, detail)


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return DIT_BF16
    if dt == torch.float32:
        return DIT_F32
    raise ValueError(f"unsupported dtype {dt}")


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _pi(a: Optional[np.ndarray]):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


class BlockConfig:
    """Python view of dit_block_config."""

    def __init__(self, hidden, n_heads, head_dim, mlp_hidden, freq_dim, rope_sections, dtype,
                 rope_theta=10000.0, qk_norm=True, ln_eps=1e-6, rms_eps=1e-6):
        self.c = CConfig()
        self.c.hidden, self.c.n_heads, self.c.head_dim = hidden, n_heads, head_dim
        self.c.mlp_hidden, self.c.freq_dim = mlp_hidden, freq_dim
        for i in range(3):
            self.c.rope_sections[i] = int(rope_sections[i])
        self.c.rope_theta = rope_theta
        self.c.qk_norm = 1 if qk_norm else 0
        self.c.ln_eps, self.c.rms_eps = ln_eps, rms_eps
        self.c.dtype = dtype_code(dtype) if isinstance(dtype, torch.dtype) else int(dtype)


class Varlen:
    """Python view of dit_varlen; keeps its host arrays alive."""

    def __init__(self, cu_seqlens, cu_txt=None, grid_fhw=None, pos_offset=None):
        self.cu = _i32(cu_seqlens)
        self.cu_txt = _i32(cu_txt) if cu_txt is not None else None
        self.grid = _i32(np.asarray(grid_fhw).reshape(-1)) if grid_fhw is not None else None
        self.off = _i32(pos_offset) if pos_offset is not None else None
        self.c = CVarlen()
        self.c.n_req = len(self.cu) - 1
        self.c.cu_seqlens = _pi(self.cu)
        self.c.cu_seqlens_txt = _pi(self.cu_txt)
        self.c.grid_fhw = _pi(self.grid)
        self.c.pos_offset = _pi(self.off)


def make_weights(w: Dict[str, Optional[torch.Tensor]]) -> CWeights:
    cw = CWeights()
    for n in WEIGHT_FIELDS:
        t = w.get(n)
        setattr(cw, n, t.data_ptr() if t is not None else None)
    return cw


# ------------------------------------------------------------ entry points


def block_workspace_size(cfg: BlockConfig, vl: Varlen) -> int:
    return int(lib().dit_block_workspace_size(ctypes.byref(cfg.c), ctypes.byref(vl.c)))


def block_forward(cfg, weights: CWeights, vl, x, t, txt, y, ws, stream=None, mod=None):
    """mod: optional precomputed modulation [n_req, 6, D] fp32 (t may then be None)."""
    _check(lib().dit_block_forward(ctypes.byref(cfg.c), ctypes.byref(weights), ctypes.byref(vl.c), _ptr(x),
                                   _ptr(t), _ptr(mod), _ptr(txt), _ptr(y), _ptr(ws), ws.numel() * ws.element_size(),
                                   _stream(stream)), "dit_block_forward")


def block_pre_attention(cfg, weights, vl, x, t, mod, qkv, ws, stream=None):
    """t given: mod is written from t; t None: mod is read."""
    _check(lib().dit_block_pre_attention(ctypes.byref(cfg.c), ctypes.byref(weights), ctypes.byref(vl.c), _ptr(x),
                                         _ptr(t), _ptr(mod), _ptr(qkv), _ptr(ws), ws.numel() * ws.element_size(),
                                         _stream(stream)), "dit_block_pre_attention")


def block_post_attention(cfg, weights, vl, x, o, txt, mod, y, ws, stream=None, t=None):
    """mod None: the modulation is computed from t."""
    _check(lib().dit_block_post_attention(ctypes.byref(cfg.c), ctypes.byref(weights), ctypes.byref(vl.c), _ptr(x),
                                          _ptr(o), _ptr(txt), _ptr(t), _ptr(mod), _ptr(y), _ptr(ws),
                                          ws.numel() * ws.element_size(), _stream(stream)),
           "dit_block_post_attention")


def debug_gemm_tile_n(tile_n: int):
    """Force the bf16 GEMM's output tile width (192 or 256); 0 restores the choice per shape."""
    _check(lib().dit_debug_gemm_tile_n(int(tile_n)), "dit_debug_gemm_tile_n")


def debug_attention_split(mode: int):
    """bf16 self-attention's split of its last round: 2 or 4 forces that many key pieces, 1 never, 0 per shape."""
    _check(lib().dit_debug_attention_split(int(mode)), "dit_debug_attention_split")


def debug_attention_shape(waves: int):
    """bf16 attention's kernel shape: 4 or 8 waves forced, 0 chosen per call."""
    _check(lib().dit_debug_attention_shape(int(waves)), "dit_debug_attention_shape")


def debug_attention_plan(cu_q, cu_k, n_heads: int, compute_units: int):
    """(waves, split pieces, split items) of a bf16 attention call with these ranges (host only)."""
    n = len(cu_q) - 1
    cq = (ctypes.c_int32 * (n + 1))(*[int(x) for x in cu_q])
    ck = (ctypes.c_int32 * (n + 1))(*[int(x) for x in cu_k])
    w, sp, si = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(lib().dit_debug_attention_plan(cq, ck, n, int(n_heads), int(compute_units), ctypes.byref(w),
                                          ctypes.byref(sp), ctypes.byref(si)), "dit_debug_attention_plan")
    return w.value, sp.value, si.value


def timestep_modulation(cfg, weights, t, mod, ws, stream=None):
    _check(lib().dit_timestep_modulation(ctypes.byref(cfg.c), ctypes.byref(weights), int(t.numel()), _ptr(t),
                                         _ptr(mod), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "dit_timestep_modulation")


def timestep_modulation_noalloc(cfg, weights, t, mod, stream=None):
    """dit_timestep_modulation without a workspace (the library's static scratch)."""
    _check(lib().dit_timestep_modulation_noalloc(ctypes.byref(cfg.c), ctypes.byref(weights), int(t.numel()),
                                                 _ptr(t), _ptr(mod), _stream(stream)),
           "dit_timestep_modulation_noalloc")


def attention_varlen(q, k, v, o, cu_q, cu_k, n_heads, head_dim, softmax_scale=None, stream=None):
    """softmax_scale None: the library's default, 1/sqrt(head_dim)."""
    cq, ck = _i32(cu_q), _i32(cu_k)
    scale = 0.0 if softmax_scale is None else softmax_scale
    _check(lib().dit_attention_varlen(_ptr(q), _ptr(k), _ptr(v), _ptr(o), q.stride(0), k.stride(0), v.stride(0),
                                      o.stride(0), _pi(cq), _pi(ck), len(cq) - 1, n_heads, head_dim, scale,
                                      dtype_code(q.dtype), _stream(stream)), "dit_attention_varlen")


def adaln_modulate(x, shift, scale, mod_stride, cu_seqlens, eps, out, stream=None):
    cu = _i32(cu_seqlens)
    _check(lib().dit_adaln_modulate(_ptr(x), _ptr(shift), _ptr(scale), mod_stride, _pi(cu), len(cu) - 1,
                                    x.shape[-1], eps, _ptr(out), dtype_code(x.dtype), _stream(stream)),
           "dit_adaln_modulate")


def layer_norm_affine(x, gamma, beta, eps, out, stream=None):
    _check(lib().dit_layer_norm_affine(_ptr(x), _ptr(gamma), _ptr(beta), x.shape[0], x.shape[-1], eps, _ptr(out),
                                       dtype_code(x.dtype), _stream(stream)), "dit_layer_norm_affine")


def linear(a, w, bias, out, epi=EPI_NONE, res=None, gate=None, gate_stride=0, cu_seqlens=None, stream=None):
    cu = _i32(cu_seqlens) if cu_seqlens is not None else None
    _check(lib().dit_linear(_ptr(a), a.stride(0), _ptr(w), w.stride(0), _ptr(bias), _ptr(out), out.stride(0),
                            a.shape[0], w.shape[0], a.shape[1], epi, _ptr(res), res.stride(0) if res is not None else 0,
                            _ptr(gate), gate_stride, _pi(cu), (len(cu) - 1) if cu is not None else 0,
                            dtype_code(a.dtype), _stream(stream)), "dit_linear")


def qk_norm_rope(q, k, n_heads, head_dim, g_q, g_k, eps, rope_sections=(0, 0, 0), rope_theta=10000.0,
                 vl: Optional[Varlen] = None, stream=None):
    sec = (ctypes.c_int * 3)(*[int(s) for s in rope_sections])
    _check(lib().dit_qk_norm_rope(_ptr(q), _ptr(k), q.stride(0), q.shape[0], n_heads, head_dim, _ptr(g_q), _ptr(g_k),
                                  eps, ctypes.cast(sec, ctypes.POINTER(ctypes.c_int32)), rope_theta,
                                  ctypes.byref(vl.c) if vl is not None else None, dtype_code(q.dtype),
                                  _stream(stream)), "dit_qk_norm_rope")


def gated_residual(x, z, bias, gate, gate_stride, cu_seqlens, out, stream=None):
    cu = _i32(cu_seqlens)
    _check(lib().dit_gated_residual(_ptr(x), _ptr(z), _ptr(bias), _ptr(gate), gate_stride, _pi(cu), len(cu) - 1,
                                    x.shape[-1], _ptr(out), dtype_code(x.dtype), _stream(stream)),
           "dit_gated_residual")


# ------------------------------------------------------- the denoising step


class ModelConfig:
    """Python view of dit_model_config."""

    def __init__(self, block: BlockConfig, n_blocks: int, in_channels: int, patch):
        self.block = block
        self.c = CModelConfig()
        self.c.block = block.c
        self.c.n_blocks, self.c.in_channels = int(n_blocks), int(in_channels)
        for i in range(3):
            self.c.patch[i] = int(patch[i])


class ModelWeights:
    """Python view of dit_model_weights; keeps the host array of block weights alive."""

    def __init__(self, w: Dict[str, Optional[torch.Tensor]], blocks: Sequence[CWeights]):
        self.blocks = (CWeights * len(blocks))(*blocks)
        self.c = CModelWeights()
        for n in MODEL_FIELDS:
            t = w.get(n)
            setattr(self.c, n, t.data_ptr() if t is not None else None)
        self.c.blocks = ctypes.cast(self.blocks, ctypes.POINTER(CWeights))


def text_kv_elems(cfg: ModelConfig, vl: Varlen) -> int:
    return int(lib().dit_text_kv_elems(ctypes.byref(cfg.c), ctypes.byref(vl.c)))


def text_kv(cfg: ModelConfig, w: ModelWeights, vl: Varlen, txt, kv, stream=None):
    _check(lib().dit_text_kv(ctypes.byref(cfg.c), ctypes.byref(w.c), ctypes.byref(vl.c), _ptr(txt), _ptr(kv),
                             _stream(stream)), "dit_text_kv")


def denoise_workspace_size(cfg: ModelConfig, vl: Varlen) -> int:
    return int(lib().dit_denoise_workspace_size(ctypes.byref(cfg.c), ctypes.byref(vl.c)))


def denoise_step(cfg: ModelConfig, w: ModelWeights, vl: Varlen, latent, t, dt, kv, latent_out, ws, stream=None):
    _check(lib().dit_denoise_step(ctypes.byref(cfg.c), ctypes.byref(w.c), ctypes.byref(vl.c), _ptr(latent), _ptr(t),
                                  _ptr(dt), _ptr(kv), _ptr(latent_out), _ptr(ws), ws.numel() * ws.element_size(),
                                  _stream(stream)), "dit_denoise_step")


def patchify(cfg: ModelConfig, vl: Varlen, latent, tokens, stream=None):
    _check(lib().dit_patchify(ctypes.byref(cfg.c), ctypes.byref(vl.c), _ptr(latent), _ptr(tokens), _stream(stream)),
           "dit_patchify")


def unpatchify_euler(cfg: ModelConfig, vl: Varlen, latent, v, dt, latent_out, stream=None):
    _check(lib().dit_unpatchify_euler(ctypes.byref(cfg.c), ctypes.byref(vl.c), _ptr(latent), _ptr(v), _ptr(dt),
                                      _ptr(latent_out), _stream(stream)), "dit_unpatchify_euler")


# ------------------------------------------------------------ the simulator


def simulate(n_ranks: int, degrees, cost_us, policy: int, group_size: int, arrival_us, cls, n_steps,
             deadline_us=None) -> Dict[str, object]:
    """dit_simulate on host arrays.  cost_us: [n_classes][n_degrees] integer
    microseconds.  Returns finish_us, first_start_us (int64 arrays),
    dispatches (per degree) and events."""
    deg = _i32(degrees)
    cost = np.ascontiguousarray(np.asarray(cost_us, dtype=np.int64))
    arr = np.ascontiguousarray(np.asarray(arrival_us, dtype=np.int64))
    cl = _i32(cls)
    st = _i32(n_steps)
    dl = np.ascontiguousarray(np.asarray(deadline_us, dtype=np.int64)) if deadline_us is not None else None
    n = len(arr)
    fin = np.zeros(n, dtype=np.int64)
    first = np.zeros(n, dtype=np.int64)
    disp = np.zeros(len(deg), dtype=np.int64)
    p64 = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if a is not None else None
    cfg = CSimConfig(int(n_ranks), len(deg), _pi(deg), int(cost.shape[0]), p64(cost), int(policy), int(group_size))
    tr = CSimTrace(n, p64(arr), _pi(cl), _pi(st), p64(dl))
    res = CSimResult(p64(fin), p64(first), p64(disp), 0)
    _check(lib().dit_simulate(ctypes.byref(cfg), ctypes.byref(tr), ctypes.byref(res)), "dit_simulate")
    return {"finish": fin, "first_start": first, "dispatches": disp, "events": int(res.events)}


# ------------------------------------------------------------ migration


class MigField:
    """Python view of dit_mig_field; keeps its slice arrays alive.  src, dst:
    lists of (rank, start, end) boxes in global coordinates."""

    def __init__(self, kind: int, shape, elem_bytes: int, src, dst):
        self.src = (CMigSlice * max(1, len(src)))()
        self.dst = (CMigSlice * max(1, len(dst)))()
        for arr, sl in ((self.src, src), (self.dst, dst)):
            for k, (rank, a, b) in enumerate(sl):
                arr[k].rank = int(rank)
                for d in range(len(shape)):
                    arr[k].start[d], arr[k].end[d] = int(a[d]), int(b[d])
        self.c = CMigField()
        self.c.kind, self.c.n_dims, self.c.elem_bytes = int(kind), len(shape), int(elem_bytes)
        for d in range(len(shape)):
            self.c.shape[d] = int(shape[d])
        self.c.n_src, self.c.src = len(src), ctypes.cast(self.src, ctypes.POINTER(CMigSlice))
        self.c.n_dst, self.c.dst = len(dst), ctypes.cast(self.dst, ctypes.POINTER(CMigSlice))


def migration_plan(field: MigField):
    """The plan of a field as a ctypes array of CMigEntry (sized by a first call)."""
    n = ctypes.c_int64(0)
    st = lib().dit_migration_plan(ctypes.byref(field.c), None, 0, ctypes.byref(n))
    if st not in (DIT_OK, DIT_ERR_WORKSPACE):
        _check(st, "dit_migration_plan")
    entries = (CMigEntry * max(1, n.value))()
    _check(lib().dit_migration_plan(ctypes.byref(field.c), entries, n.value, ctypes.byref(n)), "dit_migration_plan")
    return entries, n.value


def migration_execute(field: MigField, entries, n: int, src_bufs, dst_bufs, stream=None):
    """Apply a plan on the current device: src_bufs / dst_bufs are tensors
    holding the slices densely, in the order of the field's slices."""
    sp = (ctypes.c_void_p * max(1, len(src_bufs)))(*[t.data_ptr() for t in src_bufs])
    dp = (ctypes.c_void_p * max(1, len(dst_bufs)))(*[t.data_ptr() for t in dst_bufs])
    _check(lib().dit_migration_execute(ctypes.byref(field.c), entries, n, sp, dp, _stream(stream)),
           "dit_migration_execute")
