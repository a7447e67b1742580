"""Python binding of libfdllm.so, the gfx950 Fast-dLLM++ commit selector.

Thin ctypes marshalling of the C ABI declared in include/fdllm.h: every
function takes torch tensors that already live on the GPU, checks their
dtype/shape/contiguity, and passes raw device pointers plus the current HIP
stream.  All arithmetic happens in the HIP kernels; there is no CPU fallback,
and loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libfdllm.so")
BENCH_LIB_PATH = os.path.join(_PKG, "libfdllm_bench.so")

BF16, F32 = 0, 1
SEL_THRESHOLD, SEL_FACTOR, SEL_PROFILE, SEL_ROBUST = 0, 1, 2, 3
SELECTORS = {"threshold": SEL_THRESHOLD, "factor": SEL_FACTOR, "profile": SEL_PROFILE,
             "robust": SEL_ROBUST}
MAX_BLOCK = 1024

OK = 0
ERR_INVALID_ARG, ERR_UNSUPPORTED_DTYPE, ERR_SIZE, ERR_WORKSPACE, ERR_HIP = -1, -2, -3, -4, -5
ERR_BOUNDS, ERR_BLOCK_TOO_LARGE, ERR_NONFINITE, ERR_SCRATCH = -6, -7, -8, -9
MAX_ABS_LOGIT = 1.0e7
STATIC_SCRATCH_BYTES = 8 << 20

EXPORTS = ("fdllm_confidence", "fdllm_select_profile", "fdllm_select_factor",
           "fdllm_select_threshold", "fdllm_select_robust", "fdllm_reveal", "fdllm_decode_step",
           "fdllm_workspace_size", "fdllm_status_string", "fdllm_synth_logits",
           "fdllm_advance_blocks", "fdllm_generation_workspace_size", "fdllm_generation_create",
           "fdllm_generation_run", "fdllm_generation_destroy", "fdllm_lmhead_workspace_size",
           "fdllm_lmhead_confidence", "fdllm_lmhead_decode_step", "fdllm_check_inputs",
           "fdllm_decode_step_static")


class GenerationDesc(ctypes.Structure):
    """fdllm_generation_desc (include/fdllm.h), field for field."""
    _fields_ = [("B", ctypes.c_int), ("G", ctypes.c_int), ("blk", ctypes.c_int), ("V", ctypes.c_int),
                ("seed", ctypes.c_uint64), ("sel", ctypes.c_int), ("param", ctypes.c_float),
                ("eta", ctypes.c_void_p), ("eta_uniform", ctypes.c_float),
                ("max_steps", ctypes.c_int), ("chunk", ctypes.c_int), ("use_graph", ctypes.c_int),
                ("logits", ctypes.c_void_p), ("mask", ctypes.c_void_p), ("x", ctypes.c_void_p),
                ("block_start", ctypes.c_void_p), ("block_end", ctypes.c_void_p),
                ("n_commit_hist", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t)]

BENCH_EXPORTS = ("fdllm_stream_read",)

_lib = None
_bench_lib = None


class FdllmError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libfdllm.so (built by paper_2606_02955_amd.build); raises if absent."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise FileNotFoundError(
            f"{p} is missing: build it first (python -m paper_2606_02955_amd.build)")
    lib = ctypes.CDLL(p)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.fdllm_confidence.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    for name in ("fdllm_select_profile", "fdllm_select_factor", "fdllm_select_threshold"):
        getattr(lib, name).argtypes = [vp, vp, vp, vp, vp, i32, i32, f32, vp, vp, vp]
        getattr(lib, name).restype = i32
    lib.fdllm_select_robust.argtypes = [vp, vp, vp, f32, vp, vp, vp, i32, i32, f32, vp, vp, vp]
    lib.fdllm_select_robust.restype = i32
    lib.fdllm_reveal.argtypes = [vp, vp, vp, vp, i32, i32, vp]
    lib.fdllm_decode_step.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp, i32, f32, vp, f32,
                                      vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.fdllm_decode_step_static.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp, i32, f32, vp,
                                             f32, vp, vp, vp, vp, vp, vp, vp]
    lib.fdllm_check_inputs.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp, vp]
    lib.fdllm_workspace_size.argtypes = [i32, i32, i32, i32, ctypes.POINTER(sz)]
    lib.fdllm_status_string.argtypes = [i32]
    lib.fdllm_status_string.restype = ctypes.c_char_p
    lib.fdllm_lmhead_workspace_size.argtypes = [i32, i32, i32, i32, ctypes.POINTER(sz)]
    lib.fdllm_lmhead_confidence.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                            vp, sz, vp]
    lib.fdllm_lmhead_decode_step.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, i32, f32,
                                             vp, f32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.fdllm_synth_logits.argtypes = [vp, i32, i32, i32, i32, vp, vp, ctypes.c_uint64, i32, vp]
    lib.fdllm_advance_blocks.argtypes = [vp, vp, vp, i32, i32, i32, vp, vp]
    dp = ctypes.POINTER(GenerationDesc)
    lib.fdllm_generation_workspace_size.argtypes = [dp, ctypes.POINTER(sz)]
    lib.fdllm_generation_create.argtypes = [dp, ctypes.POINTER(vp)]
    lib.fdllm_generation_run.argtypes = [vp, vp, ctypes.POINTER(i32)]
    lib.fdllm_generation_destroy.argtypes = [vp]
    for name in ("fdllm_confidence", "fdllm_reveal", "fdllm_decode_step", "fdllm_workspace_size",
                 "fdllm_decode_step_static", "fdllm_check_inputs",
                 "fdllm_synth_logits", "fdllm_advance_blocks", "fdllm_generation_workspace_size",
                 "fdllm_lmhead_workspace_size", "fdllm_lmhead_confidence", "fdllm_lmhead_decode_step",
                 "fdllm_generation_create", "fdllm_generation_run", "fdllm_generation_destroy"):
        getattr(lib, name).restype = i32
    if path is None:
        _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().fdllm_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != OK:
        raise FdllmError(status, where)


def _ptr(t: Optional[torch.Tensor], dtype=None, shape=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise ValueError(f"logits must be bfloat16 or float32, got {t.dtype}")


def fdllm_confidence(logits, mask, block_start, block_end, tokens, conf, eps=None, lse=None):
    """Greedy token / confidence / eps / lse of every candidate (see fdllm.h)."""
    B, L, V = logits.shape
    lib = load()
    st = lib.fdllm_confidence(
        _ptr(logits, name="logits"), _dtype_code(logits), B, L, V,
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), _ptr(tokens, torch.int32, (B, L), "tokens"),
        _ptr(conf, torch.float32, (B, L), "conf"), _ptr(eps, torch.float32, (B, L), "eps"),
        _ptr(lse, torch.float32, (B, L), "lse"), _stream(logits.device))
    _check(st, "fdllm_confidence")


def _select(name, conf, eps, mask, block_start, block_end, param, commit, n_commit=None):
    B, L = conf.shape
    lib = load()
    st = getattr(lib, name)(
        _ptr(conf, torch.float32, (B, L), "conf"), _ptr(eps, torch.float32, (B, L), "eps"),
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), B, L, float(param),
        _ptr(commit, torch.uint8, (B, L), "commit"), _ptr(n_commit, torch.int32, (B,), "n_commit"),
        _stream(conf.device))
    _check(st, name)


def fdllm_select_profile(conf, eps, mask, block_start, block_end, f, commit, n_commit=None):
    _select("fdllm_select_profile", conf, eps, mask, block_start, block_end, f, commit, n_commit)


def fdllm_select_factor(conf, eps, mask, block_start, block_end, f, commit, n_commit=None):
    _select("fdllm_select_factor", conf, eps, mask, block_start, block_end, f, commit, n_commit)


def fdllm_select_threshold(conf, eps, mask, block_start, block_end, tau, commit, n_commit=None):
    _select("fdllm_select_threshold", conf, eps, mask, block_start, block_end, tau, commit, n_commit)


def fdllm_select_robust(conf, eps, mask, block_start, block_end, f, commit, n_commit=None,
                        eta=None, eta_uniform: float = 0.0):
    """Calibration-robust profile rule; eta [B,L] or a uniform allowance (see fdllm.h)."""
    B, L = conf.shape
    st = load().fdllm_select_robust(
        _ptr(conf, torch.float32, (B, L), "conf"), _ptr(eps, torch.float32, (B, L), "eps"),
        _ptr(eta, torch.float32, (B, L), "eta"), float(eta_uniform),
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), B, L, float(f),
        _ptr(commit, torch.uint8, (B, L), "commit"), _ptr(n_commit, torch.int32, (B,), "n_commit"),
        _stream(conf.device))
    _check(st, "fdllm_select_robust")


def fdllm_reveal(commit, tokens, x, mask):
    B, L = commit.shape
    st = load().fdllm_reveal(
        _ptr(commit, torch.uint8, (B, L), "commit"), _ptr(tokens, torch.int32, (B, L), "tokens"),
        _ptr(x, torch.int32, (B, L), "x"), _ptr(mask, torch.uint8, (B, L), "mask"), B, L,
        _stream(commit.device))
    _check(st, "fdllm_reveal")


def fdllm_workspace_size(B: int, L: int, V: int, dtype: torch.dtype) -> int:
    n = ctypes.c_size_t(0)
    code = BF16 if dtype == torch.bfloat16 else F32 if dtype == torch.float32 else -1
    _check(load().fdllm_workspace_size(B, L, V, code, ctypes.byref(n)), "fdllm_workspace_size")
    return int(n.value)


def fdllm_decode_step(logits, mask, block_start, block_end, x, selector: str, param: float,
                      tokens=None, conf=None, eps=None, lse=None, commit=None, n_commit=None,
                      workspace: Optional[torch.Tensor] = None, eta=None, eta_uniform: float = 0.0):
    """One fused decoding step; mask and x are updated in place (see fdllm.h)."""
    B, L, V = logits.shape
    if selector not in SELECTORS:
        raise ValueError(f"selector must be one of {sorted(SELECTORS)}")
    need = fdllm_workspace_size(B, L, V, logits.dtype)
    ws_ptr, ws_bytes = None, 0
    if workspace is not None:
        ws_ptr, ws_bytes = _ptr(workspace, name="workspace"), workspace.numel() * workspace.element_size()
    elif need:
        workspace = torch.empty(need, dtype=torch.uint8, device=logits.device)
        ws_ptr, ws_bytes = _ptr(workspace), need
    st = load().fdllm_decode_step(
        _ptr(logits, name="logits"), _dtype_code(logits), B, L, V,
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), _ptr(x, torch.int32, (B, L), "x"),
        SELECTORS[selector], float(param), _ptr(eta, torch.float32, (B, L), "eta"), float(eta_uniform),
        _ptr(tokens, torch.int32, (B, L), "tokens"), _ptr(conf, torch.float32, (B, L), "conf"),
        _ptr(eps, torch.float32, (B, L), "eps"), _ptr(lse, torch.float32, (B, L), "lse"),
        _ptr(commit, torch.uint8, (B, L), "commit"), _ptr(n_commit, torch.int32, (B,), "n_commit"),
        ws_ptr, ws_bytes, _stream(logits.device))
    _check(st, "fdllm_decode_step")
    return workspace


def fdllm_decode_step_static(logits, mask, block_start, block_end, x, selector: str, param: float,
                             tokens=None, conf=None, eps=None, lse=None, commit=None, n_commit=None,
                             eta=None, eta_uniform: float = 0.0):
    """fdllm_decode_step with the library's static scratch (no workspace)."""
    B, L, V = logits.shape
    if selector not in SELECTORS:
        raise ValueError(f"selector must be one of {sorted(SELECTORS)}")
    st = load().fdllm_decode_step_static(
        _ptr(logits, name="logits"), _dtype_code(logits), B, L, V,
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), _ptr(x, torch.int32, (B, L), "x"),
        SELECTORS[selector], float(param), _ptr(eta, torch.float32, (B, L), "eta"), float(eta_uniform),
        _ptr(tokens, torch.int32, (B, L), "tokens"), _ptr(conf, torch.float32, (B, L), "conf"),
        _ptr(eps, torch.float32, (B, L), "eps"), _ptr(lse, torch.float32, (B, L), "lse"),
        _ptr(commit, torch.uint8, (B, L), "commit"), _ptr(n_commit, torch.int32, (B,), "n_commit"),
        _stream(logits.device))
    _check(st, "fdllm_decode_step_static")


def fdllm_check_inputs(logits, mask, block_start, block_end, counts=None):
    """Opt-in input check (synchronises the stream).  Returns (status, counts
    [3]: windows outside the span, windows longer than the block limit,
    candidate rows with a NaN / inf / out-of-range logit)."""
    B, L, V = logits.shape
    if counts is None:
        counts = torch.empty(3, dtype=torch.int32, device=logits.device)
    st = load().fdllm_check_inputs(
        _ptr(logits, name="logits"), _dtype_code(logits), B, L, V,
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), _ptr(counts, torch.int32, (3,), "counts"),
        _stream(logits.device))
    if st not in (OK, ERR_BOUNDS, ERR_BLOCK_TOO_LARGE, ERR_NONFINITE):
        _check(st, "fdllm_check_inputs")
    return st, [int(v) for v in counts.cpu()]


def fdllm_lmhead_workspace_size(B: int, L: int, d: int, V: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().fdllm_lmhead_workspace_size(B, L, d, V, ctypes.byref(n)), "fdllm_lmhead_workspace_size")
    return int(n.value)


def _lm_args(hidden, weight):
    B, L, d = hidden.shape
    V, d2 = weight.shape
    if d2 != d:
        raise ValueError(f"weight must be [V, {d}], got {tuple(weight.shape)}")
    if hidden.dtype != torch.bfloat16 or weight.dtype != torch.bfloat16:
        raise ValueError("hidden and weight must be bfloat16")
    return B, L, d, V


def _lm_workspace(workspace, B, L, d, V, device):
    if workspace is None:
        workspace = torch.empty(fdllm_lmhead_workspace_size(B, L, d, V), dtype=torch.uint8, device=device)
    return workspace, _ptr(workspace, name="workspace"), workspace.numel() * workspace.element_size()


def fdllm_lmhead_confidence(hidden, weight, mask, block_start, block_end, tokens, conf, eps=None,
                            lse=None, workspace=None):
    """Greedy token / confidence / eps / lse from hidden states (see fdllm.h)."""
    B, L, d, V = _lm_args(hidden, weight)
    workspace, wp, wb = _lm_workspace(workspace, B, L, d, V, hidden.device)
    st = load().fdllm_lmhead_confidence(
        _ptr(hidden, name="hidden"), _ptr(weight, name="weight"), B, L, d, V,
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), _ptr(tokens, torch.int32, (B, L), "tokens"),
        _ptr(conf, torch.float32, (B, L), "conf"), _ptr(eps, torch.float32, (B, L), "eps"),
        _ptr(lse, torch.float32, (B, L), "lse"), wp, wb, _stream(hidden.device))
    _check(st, "fdllm_lmhead_confidence")
    return workspace


def fdllm_lmhead_decode_step(hidden, weight, mask, block_start, block_end, x, selector: str,
                             param: float, tokens=None, conf=None, eps=None, lse=None, commit=None,
                             n_commit=None, workspace=None, eta=None, eta_uniform: float = 0.0):
    """One decoding step from hidden states; mask and x updated in place (see fdllm.h)."""
    B, L, d, V = _lm_args(hidden, weight)
    if selector not in SELECTORS:
        raise ValueError(f"selector must be one of {sorted(SELECTORS)}")
    workspace, wp, wb = _lm_workspace(workspace, B, L, d, V, hidden.device)
    st = load().fdllm_lmhead_decode_step(
        _ptr(hidden, name="hidden"), _ptr(weight, name="weight"), B, L, d, V,
        _ptr(mask, torch.uint8, (B, L), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), _ptr(x, torch.int32, (B, L), "x"),
        SELECTORS[selector], float(param), _ptr(eta, torch.float32, (B, L), "eta"), float(eta_uniform),
        _ptr(tokens, torch.int32, (B, L), "tokens"), _ptr(conf, torch.float32, (B, L), "conf"),
        _ptr(eps, torch.float32, (B, L), "eps"), _ptr(lse, torch.float32, (B, L), "lse"),
        _ptr(commit, torch.uint8, (B, L), "commit"), _ptr(n_commit, torch.int32, (B,), "n_commit"),
        wp, wb, _stream(hidden.device))
    _check(st, "fdllm_lmhead_decode_step")
    return workspace


def fdllm_synth_logits(logits, block_start, block_end, blk: int, seed: int, step: int):
    """Synthetic logits of every active block at `step` (recipe in fdllm.h)."""
    B, L, V = logits.shape
    if logits.dtype != torch.bfloat16:
        raise ValueError("synthetic logits are bfloat16")
    st = load().fdllm_synth_logits(
        _ptr(logits, name="logits"), B, L, V, int(blk),
        _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), int(seed) & ((1 << 64) - 1), int(step),
        _stream(logits.device))
    _check(st, "fdllm_synth_logits")


def fdllm_advance_blocks(mask, block_start, block_end, blk: int, n_active=None):
    """Move every window to its next block with a masked position (see fdllm.h)."""
    B, G = mask.shape
    st = load().fdllm_advance_blocks(
        _ptr(mask, torch.uint8, (B, G), "mask"), _ptr(block_start, torch.int32, (B,), "block_start"),
        _ptr(block_end, torch.int32, (B,), "block_end"), B, G, int(blk),
        _ptr(n_active, torch.int32, (1,), "n_active"), _stream(mask.device))
    _check(st, "fdllm_advance_blocks")


class Generation:
    """A device-resident generation (fdllm_generation_*): owns its torch buffers.

    After run(): .x and .mask hold the result, .hist[t, b] the n_commit of
    sequence b at step t (when record_history), and run() returns the steps.
    """

    def __init__(self, B: int, G: int, blk: int, V: int, seed: int, selector: str, param: float,
                 eta=None, eta_uniform: float = 0.0, max_steps: Optional[int] = None,
                 chunk: int = 8, use_graph: bool = True, record_history: bool = True,
                 device=None):
        if selector not in SELECTORS:
            raise ValueError(f"selector must be one of {sorted(SELECTORS)}")
        dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.lib = load()
        self.device = dev
        self.max_steps = int(max_steps or G)
        self.logits = torch.empty((B, G, V), dtype=torch.bfloat16, device=dev)
        self.mask = torch.empty((B, G), dtype=torch.uint8, device=dev)
        self.x = torch.empty((B, G), dtype=torch.int32, device=dev)
        self.start = torch.empty((B,), dtype=torch.int32, device=dev)
        self.end = torch.empty((B,), dtype=torch.int32, device=dev)
        self.hist = (torch.zeros((self.max_steps, B), dtype=torch.int32, device=dev)
                     if record_history else None)
        self.eta = eta
        d = GenerationDesc()
        d.B, d.G, d.blk, d.V = B, G, blk, V
        d.seed, d.sel, d.param = int(seed) & ((1 << 64) - 1), SELECTORS[selector], float(param)
        d.eta = _ptr(eta, torch.float32, (B, G), "eta")
        d.eta_uniform = float(eta_uniform)
        d.max_steps, d.chunk, d.use_graph = self.max_steps, int(chunk), int(bool(use_graph))
        d.logits, d.mask, d.x = _ptr(self.logits), _ptr(self.mask), _ptr(self.x)
        d.block_start, d.block_end = _ptr(self.start), _ptr(self.end)
        d.n_commit_hist = _ptr(self.hist) if self.hist is not None else None
        need = ctypes.c_size_t(0)
        _check(self.lib.fdllm_generation_workspace_size(ctypes.byref(d), ctypes.byref(need)),
               "fdllm_generation_workspace_size")
        self.workspace = torch.empty(max(int(need.value), 1), dtype=torch.uint8, device=dev)
        d.workspace, d.workspace_bytes = _ptr(self.workspace), int(need.value)
        self.desc = d
        h = ctypes.c_void_p(0)
        _check(self.lib.fdllm_generation_create(ctypes.byref(d), ctypes.byref(h)),
               "fdllm_generation_create")
        self.handle = h

    def run(self) -> int:
        steps = ctypes.c_int32(0)
        _check(self.lib.fdllm_generation_run(self.handle, _stream(self.device), ctypes.byref(steps)),
               "fdllm_generation_run")
        return int(steps.value)

    def close(self):
        if getattr(self, "handle", None) and self.handle.value:
            h, self.handle = self.handle, ctypes.c_void_p(0)
            _check(self.lib.fdllm_generation_destroy(h), "fdllm_generation_destroy")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def select(selector: str, conf, eps, mask, block_start, block_end, param, commit, n_commit=None,
           eta=None, eta_uniform: float = 0.0):
    """Dispatch to fdllm_select_<selector>."""
    if selector == "robust":
        fdllm_select_robust(conf, eps, mask, block_start, block_end, param, commit, n_commit,
                            eta=eta, eta_uniform=eta_uniform)
        return
    {"profile": fdllm_select_profile, "factor": fdllm_select_factor,
     "threshold": fdllm_select_threshold}[selector](conf, eps, mask, block_start, block_end,
                                                    param, commit, n_commit)


def load_bench(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libfdllm_bench.so (the read-only stream reference); raises if absent."""
    global _bench_lib
    if _bench_lib is not None and path is None:
        return _bench_lib
    p = path or BENCH_LIB_PATH
    if not os.path.exists(p):
        raise FileNotFoundError(
            f"{p} is missing: build it first (python -m paper_2606_02955_amd.build)")
    lib = ctypes.CDLL(p)
    lib.fdllm_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                      ctypes.c_void_p]
    lib.fdllm_stream_read.restype = ctypes.c_int
    if path is None:
        _bench_lib = lib
    return lib


def fdllm_stream_read(buf: torch.Tensor, sink: torch.Tensor):
    """Read every byte of `buf` once (bandwidth reference; see fdllm_bench.h)."""
    nbytes = buf.numel() * buf.element_size()
    st = load_bench().fdllm_stream_read(_ptr(buf, name="buf"), nbytes,
                                        _ptr(sink, torch.int32, (1,), "sink"), _stream(buf.device))
    if st != 0:
        raise RuntimeError(f"fdllm_stream_read: status {st}")
