"""ctypes binding of libfreqcache (include/freqcache.h).

Argument marshalling only: every computation runs in the HIP library.  Tensors
are torch tensors on the GPU; the binding checks their device, dtype,
contiguity and size against what the call will touch (the C ABI receives bare
pointers and cannot), then passes data pointers and torch's current stream.
The library must be built (paper_2604_24391_amd.build); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import torch  # imported before the library so both share torch's HIP runtime

from .build import LIB

c_int32, c_int64, c_double, c_float, c_void_p, c_char_p = (
    ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_float, ctypes.c_void_p,
    ctypes.c_char_p)

FC_OK = 0
STATUS = {0: "FC_OK", 1: "FC_ERR_INVALID_ARG", 2: "FC_ERR_SHAPE", 3: "FC_ERR_CAPACITY",
          4: "FC_ERR_HIP", 5: "FC_ERR_NO_DEVICE", 6: "FC_ERR_UNSUPPORTED"}
NSCALARS, NCOUNTS = 6, 4
SCALARS = ("sim_freq", "psi", "alpha", "mu", "sigma", "thr")
COUNTS = ("k_reuse", "k_cand", "k_final", "flushed")
FLAG_ALIGNED, FLAG_FRESH, FLAG_CAND = 1, 2, 4

EXPORTS = ("fc_version", "fc_last_error", "fc_create", "fc_destroy", "fc_select",
           "fc_select_noalloc", "fc_select_state_bytes", "fc_select_carry", "fc_cache_update",
           "fc_cache_update_layers", "fc_cache_step", "fc_layer_forward", "fc_layer_forward_trail", "fc_debug",
           "fc_phase_correlate", "fc_phase_correlate_rotation", "fc_vit_block_forward",
           "fc_vit_cache_update", "fc_vit_merger_forward", "fc_slot_state_bytes",
           "fc_slot_map_init",
           "fc_profile_enable", "fc_profile_only", "fc_profile_read")


class FcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class fc_caps(ctypes.Structure):
    _fields_ = [("max_batch", c_int32), ("max_height", c_int32), ("max_width", c_int32),
                ("max_tokens", c_int32), ("max_seq", c_int32), ("max_d_model", c_int32),
                ("max_ffn", c_int32), ("max_qkv", c_int32)]


class fc_select_params(ctypes.Structure):
    _fields_ = [("patch", c_int32), ("merge", c_int32), ("tau_mig", c_double),
                ("lambda_", c_double), ("alpha_min", c_double), ("alpha_max", c_double),
                ("adaptive", c_int32), ("alpha_fixed", c_double), ("entropy_norm", c_int32),
                ("tau_sim", c_double), ("no_align", c_int32), ("no_refresh", c_int32),
                ("align_pixel", c_int32), ("align_rotation", c_int32)]


class fc_select_out(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("sim", "energy", "reuse_mask", "recompute_idx",
                                        "n_recompute", "shift", "scalars", "counts", "flags")]


class fc_layer_desc(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("n_heads", c_int32), ("n_kv_heads", c_int32),
                ("head_dim", c_int32), ("d_ffn", c_int32), ("rms_eps", c_float),
                ("rope_theta", c_double)] + [
        (n, c_void_p) for n in ("w_qkv", "b_qkv", "w_o", "w_gate", "w_up", "w_down", "g_attn",
                                "g_mlp")]


class fc_kv_cache(ctypes.Structure):
    _fields_ = [("k", c_void_p), ("v", c_void_p), ("text_tokens", c_int32),
                ("frame_tokens", c_int32), ("window", c_int32), ("head", c_int32),
                ("grid_w", c_int32), ("mrope_section", c_int32 * 3), ("trail_tokens", c_int32),
                ("slot_map", c_void_p)]


_lib = None


class fc_vit_desc(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("n_heads", c_int32), ("head_dim", c_int32),
                ("d_ffn", c_int32), ("rms_eps", ctypes.c_float), ("rope_theta", c_double)] + \
        [(n, c_void_p) for n in ("w_qkv", "b_qkv", "w_o", "b_o", "w_gate_up", "b_gate_up",
                                 "w_down", "b_down", "g1", "g2")]


class fc_merger_desc(ctypes.Structure):
    _fields_ = [("d_model", c_int32), ("merge", c_int32), ("d_out", c_int32),
                ("rms_eps", ctypes.c_float)] + [(n, c_void_p) for n in ("g", "w1", "b1", "w2", "b2")]


class fc_vit_cache(ctypes.Structure):
    _fields_ = [("k", c_void_p), ("v", c_void_p), ("grid_h", c_int32), ("grid_w", c_int32),
                ("merge", c_int32), ("window", c_int32), ("k_prev", c_void_p),
                ("v_prev", c_void_p)]


def lib() -> ctypes.CDLL:
    """Load libfreqcache.so (fails loudly when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise FcError(6, f"{LIB} is missing: build it with "
                             "`python -m paper_2604_24391_amd.build` (there is no fallback)")
        L = ctypes.CDLL(LIB)
        L.fc_version.restype = c_char_p
        L.fc_last_error.restype = c_char_p
        L.fc_create.argtypes = [ctypes.POINTER(c_void_p), c_int32, ctypes.POINTER(fc_caps)]
        L.fc_destroy.argtypes = [c_void_p]
        L.fc_select.argtypes = [c_void_p, ctypes.POINTER(fc_select_params), c_void_p, c_void_p,
                                c_int32, c_int32, c_int32, ctypes.POINTER(fc_select_out),
                                c_void_p]
        L.fc_select_noalloc.argtypes = [ctypes.POINTER(fc_select_params), c_void_p, c_void_p,
                                        c_int32, c_int32, c_int32, ctypes.POINTER(fc_select_out),
                                        c_void_p]
        L.fc_select_state_bytes.argtypes = [c_int32, c_int32, c_int32]
        L.fc_select_state_bytes.restype = ctypes.c_size_t
        L.fc_select_carry.argtypes = [c_void_p, ctypes.POINTER(fc_select_params), c_void_p,
                                      c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                      ctypes.POINTER(fc_select_out), c_void_p]
        L.fc_cache_update.argtypes = [c_void_p, ctypes.POINTER(fc_layer_desc),
                                      ctypes.POINTER(fc_kv_cache), c_void_p, c_void_p, c_void_p,
                                      c_void_p, c_int32, c_int32, c_void_p]
        L.fc_cache_step.argtypes = [c_void_p, ctypes.POINTER(fc_layer_desc),
                                    ctypes.POINTER(fc_kv_cache), c_void_p, c_void_p, c_void_p,
                                    c_void_p, c_int32, c_int32, c_int32, c_void_p]
        L.fc_cache_update_layers.argtypes = [c_void_p, ctypes.POINTER(fc_layer_desc), c_int32,
                                             ctypes.POINTER(fc_kv_cache), ctypes.POINTER(c_void_p),
                                             ctypes.POINTER(c_void_p), c_void_p, c_void_p, c_int32,
                                             c_int32, c_void_p]
        L.fc_layer_forward.argtypes = [c_void_p, ctypes.POINTER(fc_layer_desc),
                                       ctypes.POINTER(fc_kv_cache), c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_int32, c_void_p]
        L.fc_layer_forward_trail.argtypes = [c_void_p, ctypes.POINTER(fc_layer_desc),
                                             ctypes.POINTER(fc_kv_cache), c_void_p, c_void_p,
                                             c_int32, c_void_p]
        L.fc_phase_correlate.argtypes = [c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                         c_void_p, c_void_p, c_void_p, c_void_p]
        L.fc_vit_block_forward.argtypes = [c_void_p, ctypes.POINTER(fc_vit_desc),
                                           ctypes.POINTER(fc_vit_cache), c_void_p, c_void_p,
                                           c_void_p, c_void_p, c_int32, c_void_p]
        L.fc_vit_cache_update.argtypes = [c_void_p, ctypes.POINTER(fc_vit_desc),
                                          ctypes.POINTER(fc_vit_cache), c_void_p, c_void_p,
                                          c_void_p, c_void_p, c_int32, c_void_p]
        L.fc_vit_merger_forward.argtypes = [c_void_p, ctypes.POINTER(fc_merger_desc), c_void_p,
                                            c_void_p, c_void_p, c_void_p, c_int32, c_int32,
                                            c_void_p]
        L.fc_phase_correlate_rotation.argtypes = [c_void_p, c_void_p, c_void_p, c_int32, c_int32,
                                                  c_int32, c_void_p, c_void_p, c_void_p]
        L.fc_slot_state_bytes.argtypes = [c_int32, c_int32]
        L.fc_slot_state_bytes.restype = ctypes.c_size_t
        L.fc_slot_map_init.argtypes = [c_void_p, ctypes.POINTER(fc_layer_desc),
                                       ctypes.POINTER(fc_kv_cache), c_int32, c_void_p]
        L.fc_debug.argtypes = [c_int32]
        L.fc_debug.restype = c_int32
        L.fc_profile_enable.argtypes = [c_void_p, c_int32]
        L.fc_profile_only.argtypes = [c_void_p, c_char_p]
        L.fc_profile_read.argtypes = [c_void_p, c_char_p, ctypes.POINTER(c_double),
                                      ctypes.POINTER(c_int64), c_int32]
        for n in ("fc_create", "fc_destroy", "fc_select", "fc_select_noalloc", "fc_select_carry",
                  "fc_cache_update", "fc_cache_update_layers", "fc_layer_forward",
                  "fc_layer_forward_trail", "fc_phase_correlate", "fc_phase_correlate_rotation",
                  "fc_vit_block_forward", "fc_vit_cache_update",
                  "fc_slot_map_init",
                  "fc_profile_enable",
                  "fc_profile_only", "fc_profile_read"):
            getattr(L, n).restype = c_int32
        _lib = L
    return _lib


def _check(status: int):
    if status != FC_OK:
        raise FcError(status, lib().fc_last_error().decode())


def fc_version() -> str:
    return lib().fc_version().decode()


def fc_last_error() -> str:
    return lib().fc_last_error().decode()


def _stream(stream):
    if stream is None:
        return c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return c_void_p(stream.cuda_stream)
    return c_void_p(int(stream))


def _ptr(t: torch.Tensor, dtype, numel: int, name: str):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, the call touches {numel}")
    if t.data_ptr() % 16:
        raise ValueError(f"{name} must be 16-byte aligned")
    return c_void_p(t.data_ptr())


# ------------------------------------------------------------------------------ context
@dataclass
class Caps:
    max_batch: int = 1
    max_height: int = 448
    max_width: int = 448
    max_tokens: int = 1024
    max_seq: int = 2176
    max_d_model: int = 3584
    max_ffn: int = 18944
    max_qkv: int = 4608

    def c(self) -> fc_caps:
        return fc_caps(*(int(getattr(self, f[0])) for f in fc_caps._fields_))


class Context:
    """An fc_ctx on one GPU (owns the library workspace)."""

    def __init__(self, caps: Caps, device: int = 0):
        self.caps = caps
        self.device = device
        h = c_void_p()
        cc = caps.c()
        _check(lib().fc_create(ctypes.byref(h), device, ctypes.byref(cc)))
        self.handle = h

    def close(self):
        if getattr(self, "handle", None) and self.handle.value:
            lib().fc_destroy(self.handle)
            self.handle = c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def fc_create(caps: Caps, device: int = 0) -> Context:
    return Context(caps, device)


def fc_destroy(ctx: Context):
    ctx.close()


# ------------------------------------------------------------------------------ selection
@dataclass
class SelectParams:
    """Selection hyper-parameters; defaults are the paper's (Sec. 6.4)."""
    patch: int = 14
    merge: int = 1
    tau_mig: float = 0.12
    lam: float = 0.25
    alpha_min: float = 0.08
    alpha_max: float = 0.5
    adaptive: bool = True
    alpha_fixed: float = 0.5
    entropy_norm: bool = True
    tau_sim: float = 0.0
    align: bool = True          # False: ablation "w/o Module I" (position-wise matching)
    refresh: bool = True        # False: ablation "w/o Module II" (no edge refresh)
    align_pixel: bool = False   # True: Module I's displacement from full-resolution luma
    align_rotation: bool = False  # with align_pixel: the rotation found and undone first

    @classmethod
    def naive(cls, tau: float, merge: int = 1) -> "SelectParams":
        """The paper's naive frequency baseline (Sec. 6.1): position-wise amplitude-spectrum
        similarity and static reuse of every token that reaches the fixed threshold tau.
        It is Algorithm 1 with alignment, refresh, the adaptive budget and the migration
        gate switched off (shift 0, no fresh token, a 100 % budget, tau_mig = 0) and the
        similarity floor at tau."""
        return cls(merge=merge, tau_mig=0.0, adaptive=False, alpha_fixed=1.0, tau_sim=tau,
                   align=False, refresh=False)

    def c(self) -> fc_select_params:
        return fc_select_params(self.patch, self.merge, self.tau_mig, self.lam, self.alpha_min,
                                self.alpha_max, int(self.adaptive), self.alpha_fixed,
                                int(self.entropy_norm), self.tau_sim, int(not self.align),
                                int(not self.refresh), int(self.align_pixel),
                                int(self.align_rotation))


@dataclass
class SelectOut:
    sim: torch.Tensor
    energy: torch.Tensor
    reuse_mask: torch.Tensor
    recompute_idx: torch.Tensor
    n_recompute: torch.Tensor
    shift: torch.Tensor
    scalars: torch.Tensor
    counts: torch.Tensor
    flags: torch.Tensor | None = None

    @staticmethod
    def alloc(B: int, N: int, device="cuda", flags: bool = True) -> "SelectOut":
        kw = dict(device=device)
        return SelectOut(
            sim=torch.empty(B, N, dtype=torch.float32, **kw),
            energy=torch.empty(B, N, dtype=torch.float64, **kw),
            reuse_mask=torch.empty(B, N, dtype=torch.uint8, **kw),
            recompute_idx=torch.empty(B, N, dtype=torch.int32, **kw),
            n_recompute=torch.empty(B, dtype=torch.int32, **kw),
            shift=torch.empty(B, 2, dtype=torch.int32, **kw),
            scalars=torch.empty(B, NSCALARS, dtype=torch.float64, **kw),
            counts=torch.empty(B, NCOUNTS, dtype=torch.int32, **kw),
            flags=torch.empty(B, N, dtype=torch.uint8, **kw) if flags else None)

    def c(self, B: int, N: int) -> fc_select_out:
        return fc_select_out(
            _ptr(self.sim, torch.float32, B * N, "sim"),
            _ptr(self.energy, torch.float64, B * N, "energy"),
            _ptr(self.reuse_mask, torch.uint8, B * N, "reuse_mask"),
            _ptr(self.recompute_idx, torch.int32, B * N, "recompute_idx"),
            _ptr(self.n_recompute, torch.int32, B, "n_recompute"),
            _ptr(self.shift, torch.int32, 2 * B, "shift"),
            _ptr(self.scalars, torch.float64, NSCALARS * B, "scalars"),
            _ptr(self.counts, torch.int32, NCOUNTS * B, "counts"),
            _ptr(self.flags, torch.uint8, B * N, "flags") if self.flags is not None
            else c_void_p(0))


def token_grid(H: int, W: int, prm: SelectParams):
    tp = prm.patch * prm.merge
    return H // tp, W // tp


def _select_args(prm: SelectParams, prev: torch.Tensor | None, cur: torch.Tensor,
                 out: SelectOut):
    if cur.dim() != 4 or cur.shape[1] != 3:
        raise ValueError("cur must be [B, 3, H, W]")
    B, _, H, W = cur.shape
    gh, gw = token_grid(H, W, prm)
    N = gh * gw
    pc = _ptr(cur, torch.float32, B * 3 * H * W, "cur")
    if prev is not None:
        if tuple(prev.shape) != tuple(cur.shape):
            raise ValueError("prev and cur shapes differ")
        pp = _ptr(prev, torch.float32, B * 3 * H * W, "prev")
    else:
        pp = c_void_p(0)
    return prm.c(), pp, pc, B, H, W, out.c(B, N)


def fc_select(ctx: Context, prm: SelectParams, prev: torch.Tensor | None, cur: torch.Tensor,
              out: SelectOut, stream=None):
    """Algorithm 1 for a [B, 3, H, W] float32 batch of frame pairs (prev may be None)."""
    cp, pp, pc, B, H, W, co = _select_args(prm, prev, cur, out)
    _check(lib().fc_select(ctx.handle, ctypes.byref(cp), pp, pc, B, H, W, ctypes.byref(co),
                           _stream(stream)))


def fc_select_noalloc(prm: SelectParams, prev: torch.Tensor | None, cur: torch.Tensor,
                      out: SelectOut, stream=None):
    """fc_select with the library's static scratch instead of a context (no device
    allocation; on the current device; at most 16 MiB of workspace)."""
    cp, pp, pc, B, H, W, co = _select_args(prm, prev, cur, out)
    _check(lib().fc_select_noalloc(ctypes.byref(cp), pp, pc, B, H, W, ctypes.byref(co),
                                   _stream(stream)))


def fc_phase_correlate(ctx: Context, prev: torch.Tensor | None, cur: torch.Tensor,
                       shift_px: torch.Tensor, peak: torch.Tensor | None = None,
                       response: torch.Tensor | None = None, stream=None):
    """Pixel-resolution phase correlation of a [B, 3, H, W] float32 batch of frame pairs
    (prev may be None): shift_px [B, 2] float64 sub-pixel displacement, optionally peak
    [B, 2] int32 integer peak and response [B, H, W] float64 surface."""
    if cur.dim() != 4 or cur.shape[1] != 3:
        raise ValueError("cur must be [B, 3, H, W]")
    B, _, H, W = cur.shape
    pc = _ptr(cur, torch.float32, B * 3 * H * W, "cur")
    if prev is not None:
        if tuple(prev.shape) != tuple(cur.shape):
            raise ValueError("prev and cur shapes differ")
        pp = _ptr(prev, torch.float32, B * 3 * H * W, "prev")
    else:
        pp = c_void_p(0)
    sp = _ptr(shift_px, torch.float64, 2 * B, "shift_px")
    pk = _ptr(peak, torch.int32, 2 * B, "peak") if peak is not None else c_void_p(0)
    rs = _ptr(response, torch.float64, B * H * W, "response") if response is not None else c_void_p(0)
    _check(lib().fc_phase_correlate(ctx.handle, pp, pc, B, H, W, sp, pk, rs, _stream(stream)))


def fc_phase_correlate_rotation(ctx: Context, prev: torch.Tensor | None, cur: torch.Tensor,
                                shift_px: torch.Tensor, angle: torch.Tensor | None = None,
                                stream=None):
    """Rotation of the current frames relative to the previous ones (angle [B] float64,
    radians) and the displacement of the frame centre after undoing it (shift_px [B, 2]
    float64)."""
    if cur.dim() != 4 or cur.shape[1] != 3:
        raise ValueError("cur must be [B, 3, H, W]")
    B, _, H, W = cur.shape
    pc = _ptr(cur, torch.float32, B * 3 * H * W, "cur")
    if prev is not None:
        if tuple(prev.shape) != tuple(cur.shape):
            raise ValueError("prev and cur shapes differ")
        pp = _ptr(prev, torch.float32, B * 3 * H * W, "prev")
    else:
        pp = c_void_p(0)
    ang = _ptr(angle, torch.float64, B, "angle") if angle is not None else c_void_p(0)
    _check(lib().fc_phase_correlate_rotation(ctx.handle, pp, pc, B, H, W, ang,
                                             _ptr(shift_px, torch.float64, 2 * B, "shift_px"),
                                             _stream(stream)))


def select_state_bytes(B: int, H: int, W: int) -> int:
    return int(lib().fc_select_state_bytes(B, H, W))


def select_state_alloc(B: int, H: int, W: int, device="cuda") -> torch.Tensor:
    """A device buffer for the carried selection state of B frames of H x W."""
    n = select_state_bytes(B, H, W)
    if n == 0:
        raise ValueError(f"no selection state for B={B} H={H} W={W}")
    return torch.empty(n, dtype=torch.uint8, device=device)


def fc_select_carry(ctx: Context, prm: SelectParams, state_prev: torch.Tensor | None,
                    cur: torch.Tensor, state_cur: torch.Tensor, out: SelectOut, stream=None):
    """fc_select with the previous frame's spectra carried in state_prev (None at the
    first step); this frame's spectra go to state_cur."""
    cp, _, pc, B, H, W, co = _select_args(prm, None, cur, out)
    n = select_state_bytes(B, H, W)
    ps = c_void_p(0) if state_prev is None else _ptr(state_prev, torch.uint8, n, "state_prev")
    pcur = _ptr(state_cur, torch.uint8, n, "state_cur")
    _check(lib().fc_select_carry(ctx.handle, ctypes.byref(cp), ps, pc, pcur, B, H, W,
                                 ctypes.byref(co), _stream(stream)))


# ------------------------------------------------------------------------------ layer
@dataclass
class LayerDesc:
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    weights: dict = field(repr=False)   # name -> bf16 GPU tensor
    rms_eps: float = 1e-6
    rope_theta: float = 1e6

    @property
    def qkv(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def c(self) -> fc_layer_desc:
        d, f, q, o = self.d_model, self.d_ffn, self.qkv, self.n_heads * self.head_dim
        w = self.weights
        sizes = dict(w_qkv=q * d, b_qkv=q, w_o=d * o, w_gate=f * d, w_up=f * d, w_down=d * f,
                     g_attn=d, g_mlp=d)
        ptrs = [_ptr(w[n], torch.bfloat16, sizes[n], n) for n in
                ("w_qkv", "b_qkv", "w_o", "w_gate", "w_up", "w_down", "g_attn", "g_mlp")]
        return fc_layer_desc(d, self.n_heads, self.n_kv_heads, self.head_dim, f, self.rms_eps,
                             self.rope_theta, *ptrs)


@dataclass
class KVCache:
    """One layer's token cache: k, v [B, S, n_kv, hd] bf16, S = T + W N; ring head."""
    k: torch.Tensor
    v: torch.Tensor
    text_tokens: int
    frame_tokens: int
    window: int
    head: int = 0
    # Multimodal RoPE (Qwen2.5-VL): frame token-grid width and rotary pairs per
    # (t, h, w) section; (0, 0, 0) = 1-D RoPE by prompt index
    grid_w: int = 0
    mrope: tuple = (0, 0, 0)
    trail_tokens: int = 0      # text tokens after the frames (recomputed every step)
    # slot state (slot_state_alloc) shared by every layer of the items, or None: rows
    # stored at their own index
    slot_map: torch.Tensor | None = None

    @property
    def S(self) -> int:
        return self.text_tokens + self.window * self.frame_tokens + self.trail_tokens

    def advance(self):
        """Move to the next step: the oldest frame's slot becomes the current one."""
        self.head = (self.head + 1) % self.window

    def c(self, B: int, kvw: int) -> fc_kv_cache:
        n = B * self.S * kvw
        return fc_kv_cache(_ptr(self.k, torch.bfloat16, n, "k"), _ptr(self.v, torch.bfloat16, n, "v"),
                           self.text_tokens, self.frame_tokens, self.window, self.head,
                           self.grid_w, (c_int32 * 3)(*self.mrope), self.trail_tokens,
                           _ptr(self.slot_map, torch.int32, B * self.S, "slot_map")
                           if self.slot_map is not None else c_void_p(0))

    def logical(self, t: torch.Tensor, B: int) -> torch.Tensor:
        """k or v in row order: rows gathered through the slot map (t itself without one)."""
        if self.slot_map is None:
            return t
        m = self.slot_map[:B * self.S].view(B, self.S).long()
        return torch.stack([t[b].index_select(0, m[b]) for b in range(B)])


def fc_layer_forward(ctx: Context, layer: LayerDesc, kv: KVCache, x_cur: torch.Tensor,
                     recompute_idx: torch.Tensor, n_recompute: torch.Tensor, y_cur: torch.Tensor,
                     stream=None):
    """Partial-recompute decoder layer over B items (x_cur, y_cur: [B, N, d] bf16)."""
    B = x_cur.shape[0]
    N, d = kv.frame_tokens, layer.d_model
    cl = layer.c()
    ck = kv.c(B, layer.n_kv_heads * layer.head_dim)
    _check(lib().fc_layer_forward(
        ctx.handle, ctypes.byref(cl), ctypes.byref(ck),
        _ptr(x_cur, torch.bfloat16, B * N * d, "x_cur"),
        _ptr(recompute_idx, torch.int32, B * N, "recompute_idx"),
        _ptr(n_recompute, torch.int32, B, "n_recompute"),
        _ptr(y_cur, torch.bfloat16, B * N * d, "y_cur"), B, _stream(stream)))


def fc_layer_forward_trail(ctx: Context, layer: LayerDesc, kv: KVCache, x_trail: torch.Tensor,
                           y_trail: torch.Tensor, stream=None):
    """The text rows after the frames (x_trail, y_trail: [B, U, d] bf16), all recomputed;
    call after fc_layer_forward of the same layer."""
    B = x_trail.shape[0]
    U, d = kv.trail_tokens, layer.d_model
    cl = layer.c()
    ck = kv.c(B, layer.n_kv_heads * layer.head_dim)
    _check(lib().fc_layer_forward_trail(ctx.handle, ctypes.byref(cl), ctypes.byref(ck),
                                        _ptr(x_trail, torch.bfloat16, B * U * d, "x_trail"),
                                        _ptr(y_trail, torch.bfloat16, B * U * d, "y_trail"), B,
                                        _stream(stream)))


def fc_cache_update(ctx: Context, layer: LayerDesc, kv: KVCache, y_prev: torch.Tensor,
                    y_cur: torch.Tensor, shift: torch.Tensor, reuse_mask: torch.Tensor,
                    grid_w: int, stream=None):
    """Copy each reused token's cached K/V and output rows from its aligned source."""
    B = y_cur.shape[0]
    N, d = kv.frame_tokens, layer.d_model
    cl = layer.c()
    ck = kv.c(B, layer.n_kv_heads * layer.head_dim)
    _check(lib().fc_cache_update(
        ctx.handle, ctypes.byref(cl), ctypes.byref(ck),
        _ptr(y_prev, torch.bfloat16, B * N * d, "y_prev"),
        _ptr(y_cur, torch.bfloat16, B * N * d, "y_cur"),
        _ptr(shift, torch.int32, 2 * B, "shift"),
        _ptr(reuse_mask, torch.uint8, B * N, "reuse_mask"), grid_w, B, _stream(stream)))


FC_ADVANCE_WINDOW, FC_REMAP = 1, 2


def fc_cache_step(ctx: Context, layer: LayerDesc, kv: KVCache, y_prev, y_cur, shift, reuse_mask,
                  grid_w: int, flags: int, B: int = 1, stream=None):
    """fc_cache_update with the window advance done by the library (FC_ADVANCE_WINDOW,
    FC_REMAP); the head the library writes is copied back into kv."""
    N, d = kv.frame_tokens, layer.d_model
    cl = layer.c()
    ck = kv.c(B, layer.n_kv_heads * layer.head_dim)
    remap = bool(flags & FC_REMAP)
    _check(lib().fc_cache_step(
        ctx.handle, ctypes.byref(cl), ctypes.byref(ck),
        _ptr(y_prev, torch.bfloat16, B * N * d, "y_prev") if remap else c_void_p(0),
        _ptr(y_cur, torch.bfloat16, B * N * d, "y_cur") if remap else c_void_p(0),
        _ptr(shift, torch.int32, 2 * B, "shift") if remap else c_void_p(0),
        _ptr(reuse_mask, torch.uint8, B * N, "reuse_mask") if remap else c_void_p(0),
        grid_w, flags, B, _stream(stream)))
    kv.head = int(ck.head)


def fc_cache_update_layers(ctx: Context, layer: LayerDesc, kvs, y_prevs, y_curs,
                           shift: torch.Tensor, reuse_mask: torch.Tensor, grid_w: int,
                           stream=None):
    """fc_cache_update over several layers' caches in one launch.

    kvs, y_prevs, y_curs: equal-length sequences (one entry per layer); the caches
    share their layout and have all been advanced to the same step."""
    n = len(kvs)
    if (y_prevs is None) != (y_curs is None):
        raise ValueError("fc_cache_update_layers: give both y_prevs and y_curs or neither")
    if n < 1 or (y_prevs is not None and (len(y_prevs) != n or len(y_curs) != n)):
        raise ValueError("fc_cache_update_layers: kvs, y_prevs and y_curs need one entry per layer")
    B = reuse_mask.shape[0]
    N, d = kvs[0].frame_tokens, layer.d_model
    kvw = layer.n_kv_heads * layer.head_dim
    cl = layer.c()
    cks = (fc_kv_cache * n)(*[kv.c(B, kvw) for kv in kvs])
    if y_prevs is None:
        yp = yc = None
    else:
        yp = (c_void_p * n)(*[_ptr(y, torch.bfloat16, B * N * d, "y_prev") for y in y_prevs])
        yc = (c_void_p * n)(*[_ptr(y, torch.bfloat16, B * N * d, "y_cur") for y in y_curs])
    _check(lib().fc_cache_update_layers(
        ctx.handle, ctypes.byref(cl), n, cks, yp, yc,
        _ptr(shift, torch.int32, 2 * B, "shift"),
        _ptr(reuse_mask, torch.uint8, B * N, "reuse_mask"), grid_w, B, _stream(stream)))


@dataclass
class VitDesc:
    """One vision-encoder block: bf16 device weights (w_gate_up stacks gate rows, then up
    rows; d_ffn a multiple of 64, padded with zeros if needed)."""
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    w: dict
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0

    def c(self) -> fc_vit_desc:
        d, f = self.d_model, self.d_ffn
        sizes = dict(w_qkv=3 * d * d, b_qkv=3 * d, w_o=d * d, b_o=d, w_gate_up=2 * f * d,
                     b_gate_up=2 * f, w_down=d * f, b_down=d, g1=d, g2=d)
        ptrs = [_ptr(self.w[k], torch.bfloat16, n, k) for k, n in sizes.items()]
        return fc_vit_desc(d, self.n_heads, self.head_dim, f, self.rms_eps, self.rope_theta, *ptrs)


@dataclass
class VitCache:
    """One block's encoder cache: k, v [B, grid_h grid_w merge^2, n_heads, head_dim] bf16
    (patch rows token-major); window: attention window side in merged tokens, 0 = full.
    k_prev, v_prev (fc_vit_cache_update only): the previous frame's cache in separate
    buffers, or None (k, v hold it and are remapped in place)."""
    k: torch.Tensor
    v: torch.Tensor
    grid_h: int
    grid_w: int
    merge: int = 2
    window: int = 4
    k_prev: torch.Tensor | None = None
    v_prev: torch.Tensor | None = None

    def c(self, B: int, d: int) -> fc_vit_cache:
        n = B * self.grid_h * self.grid_w * self.merge * self.merge * d
        kp = _ptr(self.k_prev, torch.bfloat16, n, "k_prev") if self.k_prev is not None else c_void_p(0)
        vp = _ptr(self.v_prev, torch.bfloat16, n, "v_prev") if self.v_prev is not None else c_void_p(0)
        return fc_vit_cache(_ptr(self.k, torch.bfloat16, n, "k"), _ptr(self.v, torch.bfloat16, n, "v"),
                            self.grid_h, self.grid_w, self.merge, self.window, kp, vp)


def fc_vit_block_forward(ctx: Context, layer: VitDesc, cache: VitCache, x: torch.Tensor,
                         recompute_idx: torch.Tensor, n_recompute: torch.Tensor, y: torch.Tensor,
                         stream=None):
    """One vision block over the patches of the recomputed merged tokens (x, y:
    [B, patches, d] bf16)."""
    B = y.shape[0]
    n = cache.grid_h * cache.grid_w
    rows = B * n * cache.merge * cache.merge * layer.d_model
    cl, cc = layer.c(), cache.c(B, layer.d_model)
    _check(lib().fc_vit_block_forward(
        ctx.handle, ctypes.byref(cl), ctypes.byref(cc), _ptr(x, torch.bfloat16, rows, "x"),
        _ptr(recompute_idx, torch.int32, B * n, "recompute_idx"),
        _ptr(n_recompute, torch.int32, B, "n_recompute"), _ptr(y, torch.bfloat16, rows, "y"), B,
        _stream(stream)))


def fc_vit_cache_update(ctx: Context, layer: VitDesc, cache: VitCache,
                        y_prev: torch.Tensor | None, y_cur: torch.Tensor | None,
                        shift: torch.Tensor, reuse_mask: torch.Tensor, stream=None):
    """The encoder cache's remap (y_prev = y_cur = None: no output rows moved)."""
    B = shift.shape[0]
    n = cache.grid_h * cache.grid_w
    rows = B * n * cache.merge * cache.merge * layer.d_model
    cl, cc = layer.c(), cache.c(B, layer.d_model)
    yp = _ptr(y_prev, torch.bfloat16, rows, "y_prev") if y_prev is not None else c_void_p(0)
    yc = _ptr(y_cur, torch.bfloat16, rows, "y_cur") if y_cur is not None else c_void_p(0)
    _check(lib().fc_vit_cache_update(
        ctx.handle, ctypes.byref(cl), ctypes.byref(cc), yp, yc,
        _ptr(shift, torch.int32, 2 * B, "shift"),
        _ptr(reuse_mask, torch.uint8, B * n, "reuse_mask"), B, _stream(stream)))


@dataclass
class MergerDesc:
    """The patch merger: bf16 device weights g [d_model], w1 [hidden, hidden], b1 [hidden],
    w2 [d_out, hidden], b2 [d_out] (hidden = merge^2 d_model)."""
    d_model: int
    merge: int
    d_out: int
    w: dict
    rms_eps: float = 1e-6

    def c(self) -> fc_merger_desc:
        h = self.merge * self.merge * self.d_model
        sizes = dict(g=self.d_model, w1=h * h, b1=h, w2=self.d_out * h, b2=self.d_out)
        ptrs = [_ptr(self.w[k], torch.bfloat16, n, k) for k, n in sizes.items()]
        return fc_merger_desc(self.d_model, self.merge, self.d_out, self.rms_eps, *ptrs)


def fc_vit_merger_forward(ctx: Context, merger: MergerDesc, y: torch.Tensor,
                          recompute_idx: torch.Tensor, n_recompute: torch.Tensor,
                          x_out: torch.Tensor, stream=None):
    """The merger for the recomputed tokens: y [B, tokens merge^2, d_model] bf16 ->
    x_out [B, tokens, d_out] bf16 (rows of recompute_idx only)."""
    B, n = recompute_idx.shape
    mm = merger.merge * merger.merge
    cm = merger.c()
    _check(lib().fc_vit_merger_forward(
        ctx.handle, ctypes.byref(cm), _ptr(y, torch.bfloat16, B * n * mm * merger.d_model, "y"),
        _ptr(recompute_idx, torch.int32, B * n, "recompute_idx"),
        _ptr(n_recompute, torch.int32, B, "n_recompute"),
        _ptr(x_out, torch.bfloat16, B * n * merger.d_out, "x_out"), n, B, _stream(stream)))


def slot_state_bytes(B: int, S: int) -> int:
    return int(lib().fc_slot_state_bytes(B, S))


def slot_state_alloc(B: int, S: int, device="cuda") -> torch.Tensor:
    """A slot state for B items of S cache rows (int32; set it up with fc_slot_map_init)."""
    n = slot_state_bytes(B, S)
    if n == 0:
        raise ValueError("slot_state_alloc: B and S must be positive")
    return torch.empty(n // 4, dtype=torch.int32, device=device)


def fc_slot_map_init(ctx: Context, layer: LayerDesc, kv: KVCache, B: int, stream=None):
    """Every row at its own pool row (the state that kv.slot_map points at)."""
    if kv.slot_map is None:
        raise ValueError("fc_slot_map_init: the cache has no slot map")
    cl = layer.c()
    ck = kv.c(B, layer.n_kv_heads * layer.head_dim)
    _check(lib().fc_slot_map_init(ctx.handle, ctypes.byref(cl), ctypes.byref(ck), B,
                                  _stream(stream)))


# ------------------------------------------------------------------------------ timing
def fc_debug(on: bool | None = None) -> bool:
    """Debug mode (process-wide): every kernel launch waits for its stream, so a fault
    inside a kernel is reported by the call that launched it.  None leaves the mode as it
    is; returns the previous mode."""
    return bool(lib().fc_debug(-1 if on is None else int(bool(on))))


def fc_profile_enable(ctx: Context, on: bool = True):
    _check(lib().fc_profile_enable(ctx.handle, int(on)))


def fc_profile_only(ctx: Context, name: str | None = None):
    """Time only kernel `name` (None: every kernel) while profiling is enabled."""
    _check(lib().fc_profile_only(ctx.handle, name.encode() if name else None))


def fc_profile_read(ctx: Context, name: str | None = None, reset: bool = False):
    """(total milliseconds, launches) of kernel `name` (all kernels when None)."""
    ms, n = c_double(), c_int64()
    _check(lib().fc_profile_read(ctx.handle, name.encode() if name else None, ctypes.byref(ms),
                                 ctypes.byref(n), int(reset)))
    return ms.value, n.value
