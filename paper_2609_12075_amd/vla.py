"""ctypes binding of libvla.so (argument marshalling only).

Names follow the C ABI in include/vla.h. Device buffers are torch tensors
(PyTorch provides device memory and streams); every step of the computation
runs in the library's HIP kernels. The library must have been built
(``python -m paper_2609_12075_amd.build``); loading raises otherwise — there
is no fallback path.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref
from typing import Optional

import numpy as np

from . import synth

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libvla.so")
_lib = None

VLA_OK, VLA_EINVAL, VLA_ENOMEM, VLA_EHIP, VLA_EUNSUPPORTED = range(5)

# every exported symbol declared by include/vla.h and include/vla_debug.h
EXPORTS = ["vla_weight_count", "vla_create_model", "vla_destroy_model", "vla_set_graphs", "vla_kv_bytes",
           "vla_prefill", "vla_prefill_ex", "vla_denoise", "vla_step", "vla_last_error", "vla_shutdown",
           "vla_debug_gemm", "vla_debug_gemm_bf16", "vla_debug_resid_norm", "vla_debug_gemm_rms", "vla_debug_resid_copy", "vla_debug_attention",
           "vla_debug_cu_probe", "vla_debug_replay_gemm", "vla_gemm_noalloc", "vla_debug_sync_probe",
           "vla_debug_gemm_plan"]


class VlaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"vla status {status}: {msg}")
        self.status = status


class VlaConfigC(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in (
        "dtype", "n_img", "img_hw", "patch", "vit_layers", "vit_d", "vit_heads", "vit_mlp", "n_text", "vocab",
        "llm_layers", "llm_d", "n_q", "n_kv", "head_dim", "llm_mlp", "head_kind", "act_layers", "act_d",
        "act_heads", "act_mlp", "horizon", "action_dim", "state_dim", "time_dim", "max_batch")] + [
        ("rope_base", ctypes.c_float), ("norm_eps", ctypes.c_float), ("pix_shuffle", ctypes.c_int)]


class StepArgsC(ctypes.Structure):
    _fields_ = [("vlm_model", ctypes.c_void_p), ("vlm_batch", ctypes.c_int),
                ("pixels", ctypes.c_void_p), ("text_ids", ctypes.c_void_p), ("state", ctypes.c_void_p),
                ("kv_out", ctypes.c_void_p),
                ("adit_model", ctypes.c_void_p), ("adit_batch", ctypes.c_int),
                ("kv_in", ctypes.c_void_p), ("noise", ctypes.c_void_p), ("steps", ctypes.c_int),
                ("actions_out", ctypes.c_void_p),
                ("vlm_cu_count", ctypes.c_int), ("adit_cu_count", ctypes.c_int), ("adit_done", ctypes.c_void_p)]


def lib():
    """Load libvla.so (once). Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} not built: run `python -m paper_2609_12075_amd.build`")
        # torch first: it loads the HIP runtime it ships, which the library's
        # own dependency then resolves to, so the process has one runtime
        import torch  # noqa: F401
        L = ctypes.CDLL(_LIB_PATH)
        vp, ci, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        L.vla_weight_count.argtypes = [ctypes.POINTER(VlaConfigC)]; L.vla_weight_count.restype = sz
        L.vla_create_model.argtypes = [ctypes.POINTER(VlaConfigC), vp, sz, ci, ctypes.POINTER(vp)]
        L.vla_create_model.restype = ci
        L.vla_destroy_model.argtypes = [vp]; L.vla_destroy_model.restype = None
        L.vla_set_graphs.argtypes = [vp, ci]; L.vla_set_graphs.restype = ci
        L.vla_kv_bytes.argtypes = [vp, ci]; L.vla_kv_bytes.restype = sz
        L.vla_prefill.argtypes = [vp, ci, vp, vp, vp, vp]; L.vla_prefill.restype = ci
        L.vla_prefill_ex.argtypes = [vp, ci, vp, vp, vp, vp, vp]; L.vla_prefill_ex.restype = ci
        L.vla_denoise.argtypes = [vp, ci, vp, vp, ci, vp, vp]; L.vla_denoise.restype = ci
        L.vla_step.argtypes = [ctypes.POINTER(StepArgsC), vp]; L.vla_step.restype = ci
        L.vla_last_error.argtypes = []; L.vla_last_error.restype = ctypes.c_char_p
        L.vla_debug_gemm.argtypes = [ci, ci, ci, vp, ci, ci, vp, ci, ci, vp, ci, vp, ci, vp]
        L.vla_debug_gemm.restype = ci
        L.vla_debug_gemm_bf16.argtypes = [ci, ci, ci, vp, ci, vp, ci, vp, ci, ci, ci, ctypes.c_float, vp, ci, vp]
        L.vla_debug_gemm_bf16.restype = ci
        L.vla_gemm_noalloc.argtypes = [ci, ci, ci, vp, ci, ci, vp, ci, ci, vp, ci, vp, ci, vp]
        L.vla_gemm_noalloc.restype = ci
        L.vla_debug_resid_norm.argtypes = [ci, ci, ci, vp, vp, vp, vp, vp, ci, vp, vp, ctypes.c_float, vp, vp]
        L.vla_debug_resid_norm.restype = ci
        L.vla_debug_gemm_rms.argtypes = [ci, ci, ci, vp, vp, vp, ctypes.c_float, vp, vp]
        L.vla_debug_gemm_rms.restype = ci
        L.vla_debug_resid_copy.argtypes = [ci, ci, ci, vp, vp, vp, vp, vp, ci, vp, ci, vp]
        L.vla_debug_resid_copy.restype = ci
        L.vla_debug_attention.argtypes = [ci, ci, ci, ci, ci, ci, vp, vp, vp, ci, vp, vp, ci, vp, vp]
        L.vla_debug_attention.restype = ci
        L.vla_debug_cu_probe.argtypes = [ci, ci, ci, ci, ci, ci, vp, vp]; L.vla_debug_cu_probe.restype = ci
        L.vla_debug_sync_probe.argtypes = [ci, ci, ci, ci, ci, vp, vp, vp, vp, vp]
        L.vla_debug_sync_probe.restype = ci
        L.vla_debug_gemm_plan.argtypes = [ci, ci, ci, ci, ci, ci, ci, ctypes.POINTER(ci)]
        L.vla_debug_gemm_plan.restype = ci
        L.vla_debug_replay_gemm.argtypes = [vp, ci, ci, ci, vp, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_int)]
        L.vla_debug_replay_gemm.restype = ci
        L.vla_shutdown.argtypes = []; L.vla_shutdown.restype = None
        _lib = L
        # atexit handlers run last-registered-first: torch, imported above,
        # registered its handlers already, so this teardown runs before them
        atexit.register(shutdown)
    return _lib


# objects holding library resources (models, schedulers), closed by shutdown()
_live = weakref.WeakSet()
# non-blocking streams created by nonblocking_stream(), destroyed by shutdown()
_streams = []


def register(obj):
    """Track an object with a close() method so shutdown() releases it."""
    _live.add(obj)


def shutdown():
    """Orderly teardown before the runtime unloads: wait for the GPU, close
    live schedulers and models, destroy the streams this module created, then
    vla_shutdown() (stream pool, events, hook workspaces)."""
    global _streams
    if _lib is None:
        return
    try:
        import torch
        if torch.cuda.is_available() and torch.cuda.is_initialized():
            torch.cuda.synchronize()
    except Exception:
        pass
    for obj in sorted(list(_live), key=lambda o: 0 if hasattr(o, "n_models") else 1):
        try:
            obj.close()
        except Exception:
            pass
    if _streams:
        for dev, s in _streams:
            try:
                _hip.hipSetDevice(ctypes.c_int(dev))
                _hip.hipStreamSynchronize(ctypes.c_void_p(s))
                _hip.hipStreamDestroy(ctypes.c_void_p(s))
            except Exception:
                pass
        _streams = []
    _lib.vla_shutdown()


def _check(status: int):
    if status != VLA_OK:
        raise VlaError(status, lib().vla_last_error().decode())


def config_struct(c: synth.VLAConfig) -> VlaConfigC:
    s = VlaConfigC()
    for name, _ in VlaConfigC._fields_:
        setattr(s, name, getattr(c, name))
    return s


def weight_count(c: synth.VLAConfig) -> int:
    s = config_struct(c)
    n = lib().vla_weight_count(ctypes.byref(s))
    if n == 0:
        raise VlaError(VLA_EINVAL, lib().vla_last_error().decode())
    return int(n)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    import torch
    assert isinstance(t, torch.Tensor) and t.is_cuda and t.is_contiguous(), "device tensors must be contiguous"
    return t.data_ptr()


def _ptr_rows(t) -> int:
    """Pointer of a 2-D device matrix whose rows are contiguous (a row
    stride of its own is passed separately)."""
    import torch
    assert isinstance(t, torch.Tensor) and t.is_cuda and t.dim() == 2 and t.stride(1) == 1, \
        "device matrices need contiguous rows"
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


class Model:
    """A model resident on one GPU (libvla's vla_model)."""

    def __init__(self, cfg: synth.VLAConfig, weights: np.ndarray, device: int = 0):
        self.cfg = cfg
        w = np.ascontiguousarray(weights, dtype=np.float32)
        s = config_struct(cfg)
        h = ctypes.c_void_p()
        _check(lib().vla_create_model(ctypes.byref(s), w.ctypes.data, w.size, device, ctypes.byref(h)))
        self.handle = h
        self.device = device
        register(self)

    def close(self):
        if getattr(self, "handle", None):
            lib().vla_destroy_model(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_graphs(self, enabled: bool):
        _check(lib().vla_set_graphs(self.handle, int(bool(enabled))))

    def kv_bytes(self, batch: int) -> int:
        n = lib().vla_kv_bytes(self.handle, batch)
        if n == 0:
            raise VlaError(VLA_EINVAL, lib().vla_last_error().decode())
        return int(n)

    def alloc_kv(self, batch: int):
        import torch
        return torch.empty(self.kv_bytes(batch), dtype=torch.uint8, device=f"cuda:{self.device}")

    def prefill(self, batch, pixels, text_ids, kv_out, state=None, stream=None):
        _check(lib().vla_prefill_ex(self.handle, batch, _ptr(pixels), _ptr(text_ids), _ptr(state), _ptr(kv_out),
                                    _stream(stream)))

    def replay_gemm(self, which: int, batch: int, iters: int, stream=None):
        """Enqueue `iters` launches of one stage projection. Returns (flops of
        one launch, plan dict: tile_n, tile_m, splits, mode, kind, stages, bk, kg, rms)."""
        f = ctypes.c_double(0.0)
        plan = (ctypes.c_int * 9)()
        _check(lib().vla_debug_replay_gemm(self.handle, which, batch, iters, _stream(stream), ctypes.byref(f), plan))
        return f.value, {"tile_n": plan[0], "tile_m": plan[1], "splits": plan[2], "mode": plan[3], "kind": plan[4],
                         "stages": plan[5], "bk": plan[6], "kg": plan[7], "rms": plan[8]}

    @staticmethod
    def kernel_symbol(plan):
        """Mangled-name fragment of the projection kernel a plan launches
        (the partial pass of a K-split plan is the STORE instantiation)."""
        mode = plan["mode"] if plan["splits"] == 1 else 0
        if plan["kind"] in (1, 4):
            return (f"gemm_stage_kernelILi{plan['tile_n']}ELi{plan['tile_m']}ELi{plan['stages']}ELi{mode}"
                    f"ELi{plan['bk']}ELi{plan['kg']}ELi{plan['rms']}E")
        if plan["kind"] == 2:
            return f"gemm_skinny_kernelILi{plan['tile_n'] // 16}ELi{mode}ELi{plan['rms']}E"
        if plan["kind"] == 3:
            return f"gemm_big_kernelILi{mode}E"
        return f"gemm_mfma_kernelILi{plan['tile_n']}ELi{plan['tile_m']}EDF16bLi{mode}E"

    def denoise(self, batch, kv, noise, steps, actions_out, stream=None):
        _check(lib().vla_denoise(self.handle, batch, _ptr(kv), _ptr(noise), steps, _ptr(actions_out),
                                 _stream(stream)))


_hip = None


def nonblocking_stream(device: int = 0):
    """A new non-blocking HIP stream on `device`, as a torch ExternalStream
    (torch creates blocking streams only). Passed as vla_step's join stream it
    lets the unrestricted action half run on it directly (see vla_step). The
    stream lives until shutdown() (registered to run at interpreter exit)."""
    global _hip
    import torch
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
    prev = torch.cuda.current_device()
    torch.cuda.set_device(device)
    try:
        s = ctypes.c_void_p()
        if _hip.hipStreamCreateWithFlags(ctypes.byref(s), ctypes.c_uint(1)) != 0:   # hipStreamNonBlocking
            raise VlaError(VLA_EHIP, "hipStreamCreateWithFlags failed")
        _streams.append((device, s.value))
    finally:
        torch.cuda.set_device(prev)
    return torch.cuda.ExternalStream(s.value, device=torch.device("cuda", device))


def step(vlm_model: Optional[Model], vlm_batch: int, pixels, text_ids, kv_out,
         adit_model: Optional[Model], adit_batch: int, kv_in, noise, steps: int, actions_out,
         vlm_cu_count: int = 256, adit_cu_count: int = 0, state=None, join_stream=None, adit_done=None):
    """One lockstep: prefill(vlm_batch) on the CU-restricted stream alongside
    denoise(adit_batch) on the action stream; join_stream waits for both.
    adit_done: a torch.cuda.Event (or raw hipEvent_t) recorded right after the
    action half."""
    a = StepArgsC()
    a.vlm_model = vlm_model.handle if vlm_model is not None else None
    a.vlm_batch = vlm_batch
    a.pixels, a.text_ids, a.state, a.kv_out = _ptr(pixels), _ptr(text_ids), _ptr(state), _ptr(kv_out)
    a.adit_model = adit_model.handle if adit_model is not None else None
    a.adit_batch = adit_batch
    a.kv_in, a.noise, a.steps, a.actions_out = _ptr(kv_in), _ptr(noise), steps, _ptr(actions_out)
    a.vlm_cu_count, a.adit_cu_count = vlm_cu_count, adit_cu_count
    if adit_done is not None:
        a.adit_done = adit_done.cuda_event if hasattr(adit_done, "cuda_event") else int(adit_done)
    _check(lib().vla_step(ctypes.byref(a), _stream(join_stream)))


# ---------------------------------------------------------------- test hooks
def _gemm_call(fn, A, Wt, bias, act, out, M, N, K, stream):
    import torch
    M = A.shape[0] if M is None else M
    N = Wt.shape[0] if N is None else N
    K = A.shape[1] if K is None else K
    if out is None:
        out = torch.empty(M, N, dtype=torch.float32, device=A.device)
    at = 1 if A.dtype == torch.bfloat16 else 0
    wt = 1 if Wt.dtype == torch.bfloat16 else 0
    _check(fn(M, N, K, _ptr(A), A.shape[1], at, _ptr(Wt), Wt.shape[1], wt, _ptr(bias), act, _ptr(out), out.shape[1],
              _stream(stream)))
    return out


def debug_gemm(A, Wt, bias=None, act=0, out=None, M=None, N=None, K=None, stream=None):
    return _gemm_call(lib().vla_debug_gemm, A, Wt, bias, act, out, M, N, K, stream)


def debug_gemm_bf16(A, Wt, bias=None, glu=False, act=0, rms=False, eps=1e-6, out=None, stream=None):
    """Projection with bf16 output: act(D + bias) [M][N], or with glu the
    gated-GELU form gelu(D[:, 2f] + b[2f]) * (D[:, 2f+1] + b[2f+1]) [M][N/2];
    D = A Wt^T, with rms the rows of A RMS-normalised inside the product;
    bf16 A [M][K], Wt [N][K]; out may be a 2-D bf16 view with contiguous rows."""
    import torch
    M, K = A.shape
    N = Wt.shape[0]
    if out is None:
        out = torch.empty(M, N // 2 if glu else N, dtype=torch.bfloat16, device=A.device)
    _check(lib().vla_debug_gemm_bf16(M, N, K, _ptr(A), A.stride(0), _ptr(Wt), Wt.stride(0), _ptr(bias), int(bool(glu)),
                                     act, int(bool(rms)), eps, _ptr_rows(out), out.stride(0), _stream(stream)))
    return out


def gemm_noalloc(A, Wt, bias=None, act=0, out=None, M=None, N=None, K=None, stream=None):
    """vla_gemm_noalloc: the projection of debug_gemm with its scratch in the
    library's static device array (no allocation)."""
    return _gemm_call(lib().vla_gemm_noalloc, A, Wt, bias, act, out, M, N, K, stream)


def debug_resid_norm(A, Wt, x, kind, g=None, b=None, bias=None, gate=None, eps=1e-6, stream=None):
    """x += gate * (A Wt^T + bias) in place; returns z = norm(x) (bf16)."""
    import torch
    M, K = A.shape
    N = Wt.shape[0]
    z = torch.empty(M, N, dtype=torch.bfloat16, device=A.device)
    _check(lib().vla_debug_resid_norm(M, N, K, _ptr(A), _ptr(Wt), _ptr(bias), _ptr(gate), _ptr(x), kind, _ptr(g),
                                      _ptr(b), ctypes.c_float(eps), _ptr(z), _stream(stream)))
    return z


def debug_gemm_rms(A, Wt, bias=None, eps=1e-6, stream=None):
    """rsqrt(mean_k A^2 + eps) * (A Wt^T) + bias per row, fp32 (A, Wt bf16)."""
    import torch
    M, K = A.shape
    N = Wt.shape[0]
    out = torch.empty(M, N, dtype=torch.float32, device=A.device)
    _check(lib().vla_debug_gemm_rms(M, N, K, _ptr(A), _ptr(Wt), _ptr(bias), ctypes.c_float(eps), _ptr(out),
                                    _stream(stream)))
    return out


def gemm_plan(M, N, K, mode=0, out_bf16=False, rms=False, norm_follows=False):
    """vla_debug_gemm_plan: the launch plan of a bf16 projection (host only)."""
    plan = (ctypes.c_int * 8)()
    _check(lib().vla_debug_gemm_plan(M, N, K, mode, int(bool(out_bf16)), int(bool(rms)), int(bool(norm_follows)), plan))
    keys = ("tile_n", "tile_m", "splits", "ksplit", "kind", "stages", "bk", "kg")
    return dict(zip(keys, list(plan)))


def debug_resid_copy(A, Wt, x, bias=None, gate=None, xb=None, stream=None):
    """x += gate * (A Wt^T + bias) in place; returns bf16(x) (in xb when
    given). x and xb may be 2-D views with contiguous rows."""
    import torch
    M, K = A.shape
    N = Wt.shape[0]
    if xb is None:
        xb = torch.empty(M, N, dtype=torch.bfloat16, device=A.device)
    _check(lib().vla_debug_resid_copy(M, N, K, _ptr(A), _ptr(Wt), _ptr(bias), _ptr(gate), _ptr_rows(x), x.stride(0),
                                      _ptr_rows(xb), xb.stride(0), _stream(stream)))
    return xb


def debug_attention(q, k0, v0, k1=None, v1=None, stream=None):
    import torch
    B, Hq, Lq, hd = q.shape
    Hkv, len0 = k0.shape[1], k0.shape[2]
    len1 = 0 if k1 is None else k1.shape[2]
    o = torch.empty(B, Lq, Hq * hd, dtype=q.dtype, device=q.device)
    et = 1 if q.dtype == torch.bfloat16 else 0
    _check(lib().vla_debug_attention(B, Hq, Hkv, Lq, hd, et, _ptr(q), _ptr(k0), _ptr(v0), len0, _ptr(k1), _ptr(v1),
                                     len1, _ptr(o), _stream(stream)))
    return o


def debug_sync_probe(kind: int, grid: int, iters: int, words: int = 0, spin_limit: int = 200000, buf=None, ctr=None,
                     err=None, sink=None, stream=None):
    """vla_debug_sync_probe: kind 0 `iters` empty kernels, 1 `iters` kernels
    writing `words` floats per block, 2 one kernel running `iters` grid
    barriers (ctr must be zero; err collects spin overruns)."""
    _check(lib().vla_debug_sync_probe(kind, grid, iters, words, spin_limit, _ptr(buf), _ptr(ctr), _ptr(err), _ptr(sink),
                                      _stream(stream)))


def debug_cu_probe(cu_count: int, blocks: int, spin: int = 200, from_top: bool = False, device: int = 0, stream=None,
                   via_graph: bool = False):
    import torch
    out = torch.zeros(2 * blocks, dtype=torch.int32, device=f"cuda:{device}")
    _check(lib().vla_debug_cu_probe(device, cu_count, int(from_top), blocks, spin, int(via_graph), _ptr(out),
                                    _stream(stream)))
    return out
