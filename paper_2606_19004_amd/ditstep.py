"""Thin Python binding of libditstep.so (include/ditstep.h).

Argument marshalling only: every function takes torch tensors that already
live on the GPU, passes their device pointers, sizes and the current HIP
stream through ctypes, and raises DitError on a non-OK status. All
computation happens in the library's HIP kernels; there is no fallback. The
import fails loudly if the library has not been built
(``python -m paper_2606_19004_amd.build``).
"""
from __future__ import annotations

import ctypes as C
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# DITSTEP_LIB selects another build of the library (the DITSTEP_DEBUG build, libditstep_debug.so)
LIB_PATH = os.environ.get("DITSTEP_LIB") or os.path.join(_HERE, "libditstep.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_19004_amd.build`")
_lib = C.CDLL(LIB_PATH)

DIT_F32, DIT_BF16 = 0, 1
STATUS = {0: "DIT_OK", 1: "DIT_ERR_INVALID_ARG", 2: "DIT_ERR_SHAPE", 3: "DIT_ERR_DOMAIN", 4: "DIT_ERR_NAN",
          5: "DIT_ERR_UNSUPPORTED", 6: "DIT_ERR_HIP", 7: "DIT_ERR_WORKSPACE"}
EXPORTS = ("dit_abi_version", "dit_status_string", "dit_last_error_message", "dit_block_workspace_bytes",
           "dit_block_forward", "dit_block_mlp", "joint_attention", "flow_step", "flow_logprob", "group_reward_stats",
           "group_reward_stats_async", "dit_timestep_embed", "dit_timestep_embed_noalloc", "dit_patch_embed", "dit_final_layer", "dit_denoise_workspace_bytes",
           "dit_denoise_step", "dit_profile_begin", "dit_profile_end", "dit_teacache_init", "dit_teacache_gate",
           "dit_teacache_cache_bytes", "dit_denoise_step_teacache")


class DitError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


class BlockConfig(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("heads", C.c_int32), ("head_dim", C.c_int32), ("mlp_hidden", C.c_int32),
                ("n_img", C.c_int32), ("n_txt", C.c_int32), ("grid_h", C.c_int32), ("grid_w", C.c_int32),
                ("rope", C.c_int32), ("ln_eps", C.c_float), ("rope_theta", C.c_float), ("dtype", C.c_int32)]


_P2 = C.c_void_p * 2
_BLOCK_TENSORS = ("mod_w", "mod_b", "qkv_w", "qkv_b", "out_w", "out_b", "mlp1_w", "mlp1_b", "mlp2_w", "mlp2_b")
_STEP_TENSORS = ("t1_w", "t1_b", "t2_w", "t2_b", "in_w", "in_b", "fmod_w", "fmod_b", "fout_w", "fout_b")


class BlockWeights(C.Structure):
    _fields_ = [(n, _P2) for n in _BLOCK_TENSORS]


class StepWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _STEP_TENSORS]


class TeaCacheState(C.Structure):
    _fields_ = [("threshold", C.c_double), ("n_coef", C.c_int32), ("coef", C.c_double * 8),
                ("accumulated", C.c_double), ("has_prev", C.c_int32), ("has_residual", C.c_int32)]


class KernelStat(C.Structure):
    _fields_ = [("name", C.c_char * 40), ("launches", C.c_int32), ("total_ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_stream = C.c_void_p
_i32, _i64, _f32, _sz = C.c_int32, C.c_int64, C.c_float, C.c_size_t
_vp = C.c_void_p
_sigs = {
    "dit_abi_version": ([], _i32),
    "dit_status_string": ([_i32], C.c_char_p),
    "dit_last_error_message": ([], C.c_char_p),
    "dit_block_workspace_bytes": ([C.POINTER(BlockConfig), _i32], _sz),
    "dit_block_forward": ([C.POINTER(BlockConfig), C.POINTER(BlockWeights), _i32, _vp, _vp, _vp, _vp, _sz, _stream], _i32),
    "dit_block_mlp": ([C.POINTER(BlockConfig), C.POINTER(BlockWeights), _i32, _vp, _vp, _vp, _vp, _sz, _stream], _i32),
    "joint_attention": ([_vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i64, _i64, _i64, _i64, _i64, _i64, _f32, _i32,
                         _stream], _i32),
    "flow_step": ([_vp, _vp, _vp, _i64, _f32, _f32, _f32, _stream], _i32),
    "flow_logprob": ([_vp, _vp, _vp, _i32, _i64, _f32, _f32, _f32, _vp, _stream], _i32),
    "group_reward_stats": ([_vp, _i32, _i32, _f32, _i32, _vp, _vp, _vp, _vp, _vp, _stream], _i32),
    "group_reward_stats_async": ([_vp, _i32, _i32, _f32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _stream], _i32),
    "dit_timestep_embed": ([C.POINTER(BlockConfig), C.POINTER(StepWeights), _i32, _vp, _vp, _vp, _sz, _stream], _i32),
    "dit_timestep_embed_noalloc": ([C.POINTER(BlockConfig), C.POINTER(StepWeights), _i32, _vp, _vp, _stream], _i32),
    "dit_patch_embed": ([C.POINTER(BlockConfig), C.POINTER(StepWeights), _i32, _i32, _vp, _vp, _vp, _sz, _stream], _i32),
    "dit_final_layer": ([C.POINTER(BlockConfig), C.POINTER(StepWeights), _i32, _i32, _vp, _vp, _vp, _vp, _sz,
                         _stream], _i32),
    "dit_denoise_workspace_bytes": ([C.POINTER(BlockConfig), _i32, _i32], _sz),
    "dit_denoise_step": ([C.POINTER(BlockConfig), C.POINTER(StepWeights), C.POINTER(BlockWeights), _i32, _i32, _i32,
                          _f32, _f32, _f32, _vp, _vp, _vp, _vp, _vp, _sz, _stream], _i32),
    "dit_profile_begin": ([], _i32),
    "dit_teacache_init": ([C.POINTER(TeaCacheState), C.c_double, C.POINTER(C.c_double), _i32], _i32),
    "dit_teacache_gate": ([C.POINTER(TeaCacheState), C.c_double, _i32, C.POINTER(_i32)], _i32),
    "dit_teacache_cache_bytes": ([C.POINTER(BlockConfig), _i32], _sz),
    "dit_denoise_step_teacache": ([C.POINTER(BlockConfig), C.POINTER(StepWeights), C.POINTER(BlockWeights), _i32,
                                   _i32, _i32, _f32, _f32, _f32, _vp, _vp, _vp, _vp, C.POINTER(TeaCacheState), _i32,
                                   _vp, _sz, C.POINTER(_i32), C.POINTER(C.c_double), _vp, _sz, _stream], _i32),
    "dit_profile_end": ([C.POINTER(KernelStat), _i32, C.POINTER(_i32)], _i32),
}
for _name, (_args, _res) in _sigs.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res


def lib() -> C.CDLL:
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise DitError(status, _lib.dit_last_error_message().decode())


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _s(stream) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _dtype_code(dtype) -> int:
    if dtype in ("bf16", torch.bfloat16, DIT_BF16):
        return DIT_BF16
    if dtype in ("f32", torch.float32, DIT_F32):
        return DIT_F32
    raise ValueError(f"dtype {dtype!r}")


# ---------------------------------------------------------------------------
# structures
# ---------------------------------------------------------------------------
def block_config(hidden, heads, head_dim, mlp_hidden, n_img, n_txt, grid_h, grid_w, rope=True,
                 ln_eps=1e-6, rope_theta=1e4, dtype="bf16") -> BlockConfig:
    return BlockConfig(hidden, heads, head_dim, mlp_hidden, n_img, n_txt, grid_h, grid_w, int(bool(rope)),
                       ln_eps, rope_theta, _dtype_code(dtype))


def block_weights(img: dict, txt: dict) -> BlockWeights:
    """img/txt: {tensor name: device tensor} for the two streams (image = index 0)."""
    w = BlockWeights()
    for n in _BLOCK_TENSORS:
        setattr(w, n, _P2(_ptr(img.get(n)), _ptr(txt.get(n))))
    w._keep = (dict(img), dict(txt))   # the struct holds raw device pointers: keep the tensors alive with it
    return w


def step_weights(sw: dict) -> StepWeights:
    w = StepWeights()
    for n in _STEP_TENSORS:
        setattr(w, n, _ptr(sw.get(n)))
    w._keep = dict(sw)
    return w


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """A device byte buffer (torch's allocator returns >= 256-byte aligned blocks)."""
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------
def dit_abi_version() -> int:
    return _lib.dit_abi_version()


def dit_block_workspace_bytes(cfg: BlockConfig, batch: int) -> int:
    return _lib.dit_block_workspace_bytes(C.byref(cfg), batch)


def dit_block_forward(cfg, w, temb, x_img, x_txt, ws, stream=None):
    _check(_lib.dit_block_forward(C.byref(cfg), C.byref(w), temb.shape[0], _ptr(temb), _ptr(x_img), _ptr(x_txt),
                                  _ptr(ws), ws.numel() if ws is not None else 0, _s(stream)))


def dit_block_mlp(cfg, w, temb, x_img, x_txt, ws, stream=None):
    _check(_lib.dit_block_mlp(C.byref(cfg), C.byref(w), temb.shape[0], _ptr(temb), _ptr(x_img), _ptr(x_txt),
                              _ptr(ws), ws.numel() if ws is not None else 0, _s(stream)))


def joint_attention(q, k, v, o, batch, heads, seq, head_dim, qkv_strides, o_strides, scale=None, dtype="bf16",
                    stream=None):
    """q/k/v/o: device tensors (or views) whose element (b, s, h, e) sits at the given element strides."""
    if scale is None:
        scale = 1.0 / math.sqrt(head_dim)
    _check(_lib.joint_attention(_ptr(q), _ptr(k), _ptr(v), _ptr(o), batch, heads, seq, head_dim, *qkv_strides,
                                *o_strides, scale, _dtype_code(dtype), _s(stream)))


def flow_step(x, v, noise, t, t_next, noise_level, stream=None):
    _check(_lib.flow_step(_ptr(x), _ptr(v), _ptr(noise), x.numel(), t, t_next, noise_level, _s(stream)))


def flow_logprob(x, v, x_next, t, t_next, noise_level, logp, stream=None):
    """x, v, x_next: [batch][n] fp32 device tensors (any trailing shape, flattened per sample);
    logp: [batch] fp64 device tensor."""
    b = x.shape[0] if x.dim() > 0 else 0
    n = x.numel() // b if b else 0
    _check(_lib.flow_logprob(_ptr(x), _ptr(v), _ptr(x_next), b, n, t, t_next, noise_level, _ptr(logp), _s(stream)))


def group_reward_stats(rewards, adv_eps=1e-4, k_select=0, mean=None, std=None, adv=None, order=None, selected=None,
                       stream=None):
    g, n = rewards.shape
    _check(_lib.group_reward_stats(_ptr(rewards), g, n, adv_eps, k_select, _ptr(mean), _ptr(std), _ptr(adv),
                                   _ptr(order), _ptr(selected), _s(stream)))


def group_reward_stats_async(rewards, status, adv_eps=1e-4, k_select=0, mean=None, std=None, adv=None, order=None,
                             selected=None, stream=None):
    """status: one-element int32 device tensor; holds DIT_OK or DIT_ERR_NAN once the stream has run."""
    g, n = rewards.shape
    _check(_lib.group_reward_stats_async(_ptr(rewards), g, n, adv_eps, k_select, _ptr(mean), _ptr(std), _ptr(adv),
                                         _ptr(order), _ptr(selected), _ptr(status), _s(stream)))


def dit_timestep_embed(cfg, sw, t, temb, ws, stream=None):
    _check(_lib.dit_timestep_embed(C.byref(cfg), C.byref(sw), t.shape[0], _ptr(t), _ptr(temb), _ptr(ws),
                                   ws.numel(), _s(stream)))


def dit_timestep_embed_noalloc(cfg, sw, t, temb, stream=None):
    _check(_lib.dit_timestep_embed_noalloc(C.byref(cfg), C.byref(sw), t.shape[0], _ptr(t), _ptr(temb), _s(stream)))


def dit_patch_embed(cfg, sw, latent, x_img, ws, stream=None):
    _check(_lib.dit_patch_embed(C.byref(cfg), C.byref(sw), latent.shape[0], latent.shape[-1], _ptr(latent),
                                _ptr(x_img), _ptr(ws), ws.numel() if ws is not None else 0, _s(stream)))


def dit_final_layer(cfg, sw, temb, x_img, v, ws, stream=None):
    _check(_lib.dit_final_layer(C.byref(cfg), C.byref(sw), temb.shape[0], v.shape[-1], _ptr(temb), _ptr(x_img),
                                _ptr(v), _ptr(ws), ws.numel(), _s(stream)))


def dit_denoise_workspace_bytes(cfg, batch, latent_dim) -> int:
    return _lib.dit_denoise_workspace_bytes(C.byref(cfg), batch, latent_dim)


def dit_denoise_step(cfg, sw, blocks, t, t_next, noise_level, latent, x_txt, noise, v_out, ws, stream=None):
    arr = (BlockWeights * max(len(blocks), 1))(*blocks)
    _check(_lib.dit_denoise_step(C.byref(cfg), C.byref(sw), arr, len(blocks), latent.shape[0], latent.shape[-1],
                                 t, t_next, noise_level, _ptr(latent), _ptr(x_txt), _ptr(noise), _ptr(v_out),
                                 _ptr(ws), ws.numel(), _s(stream)))


def teacache_state(threshold, coef=()):
    st = TeaCacheState()
    c = (C.c_double * max(len(coef), 1))(*[float(x) for x in coef])
    _check(_lib.dit_teacache_init(C.byref(st), float(threshold), c, len(coef)))
    return st


def dit_teacache_gate(state, rel, force=False):
    run = _i32()
    _check(_lib.dit_teacache_gate(C.byref(state), float(rel), int(bool(force)), C.byref(run)))
    return bool(run.value)


def dit_teacache_cache_bytes(cfg, batch):
    return _lib.dit_teacache_cache_bytes(C.byref(cfg), batch)


def dit_denoise_step_teacache(cfg, sw, blocks, t, t_next, noise_level, latent, x_txt, noise, v_out, state, cache, ws,
                              force=False, stream=None):
    """Returns (ran_blocks, rel)."""
    arr = (BlockWeights * max(len(blocks), 1))(*blocks)
    ran, rel = _i32(), C.c_double()
    _check(_lib.dit_denoise_step_teacache(C.byref(cfg), C.byref(sw), arr, len(blocks), latent.shape[0],
                                          latent.shape[-1], t, t_next, noise_level, _ptr(latent), _ptr(x_txt),
                                          _ptr(noise), _ptr(v_out), C.byref(state), int(bool(force)), _ptr(cache),
                                          cache.numel(), C.byref(ran), C.byref(rel), _ptr(ws), ws.numel(),
                                          _s(stream)))
    return bool(ran.value), rel.value


def dit_profile_begin():
    _check(_lib.dit_profile_begin())


def dit_profile_end() -> list:
    """Per-kernel-class totals since dit_profile_begin: list of dicts (name, launches, total_ms, flops, bytes)."""
    cap = 64
    arr = (KernelStat * cap)()
    n = _i32(0)
    _check(_lib.dit_profile_end(arr, cap, C.byref(n)))
    return [{"name": arr[i].name.decode(), "launches": arr[i].launches, "total_ms": arr[i].total_ms,
             "flops": arr[i].flops, "bytes": arr[i].bytes} for i in range(min(n.value, cap))]
