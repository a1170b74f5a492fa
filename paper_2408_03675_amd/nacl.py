"""Python binding of libnacl.so (the C ABI declared in include/nacl.h).

Argument marshalling only: every step of the eviction runs in the library's
HIP kernels.  torch tensors provide device memory and the stream.  If the
built library is missing, importing works but every call raises; there is no
CPU fallback.
"""

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libnacl.so")

NACL_OK = 0
NACL_ERR_INVALID_ARG = 1
NACL_ERR_UNSUPPORTED = 2
NACL_ERR_WORKSPACE = 3
NACL_ERR_HIP = 4

NACL_F32 = 0
NACL_BF16 = 1

SAMPLE_SOFTMAX = 0
SAMPLE_PROPORTIONAL = 1
SAMPLE_UNIFORM = 2

EXPORTED = ("nacl_workspace_bytes", "nacl_score", "nacl_select", "nacl_compact", "nacl_compact_slots",
            "nacl_append", "nacl_evict", "nacl_evict_slots", "nacl_evict_noalloc", "nacl_attention",
            "nacl_status_string",
            "nacl_last_error_detail", "nacl_version")


class NaclError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"nacl status {status}: {detail}")
        self.status = status
        self.detail = detail


class _Problem(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("L", ctypes.c_int32), ("D", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("P", ctypes.c_int32), ("n_protect", ctypes.c_int32),
        ("sm_scale", ctypes.c_float),
        ("q_stride", ctypes.c_int64 * 3), ("k_stride", ctypes.c_int64 * 3),
        ("v_stride", ctypes.c_int64 * 3),
        ("proxy_pos", ctypes.POINTER(ctypes.c_int32)),
        ("proxy_pos_dev", ctypes.c_void_p),
        ("q_group", ctypes.c_int32),
    ]


_lib = None


def load_library(path=LIB_PATH):
    """Loads libnacl.so once and declares the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2408_03675_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(_Problem)
    vp, sz, i32, u32, u64 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64
    lib.nacl_workspace_bytes.argtypes = [P]
    lib.nacl_workspace_bytes.restype = sz
    lib.nacl_score.argtypes = [P, vp, vp, vp, vp, vp, sz, vp]
    lib.nacl_score.restype = ctypes.c_int
    lib.nacl_select.argtypes = [P, vp, i32, i32, i32, u64, u32, vp, vp, sz, vp]
    lib.nacl_select.restype = ctypes.c_int
    lib.nacl_compact.argtypes = [P, vp, vp, vp, i32, vp, vp, vp]
    lib.nacl_compact.restype = ctypes.c_int
    lib.nacl_compact_slots.argtypes = [P, vp, vp, vp, i32, vp, vp]
    lib.nacl_compact_slots.restype = ctypes.c_int
    lib.nacl_evict_slots.argtypes = [P, vp, vp, vp, i32, i32, i32, u64, u32, vp, vp, vp, vp, sz, vp]
    lib.nacl_evict_slots.restype = ctypes.c_int
    lib.nacl_append.argtypes = [P, vp, vp, i32, vp, vp, i32, vp]
    lib.nacl_append.restype = ctypes.c_int
    lib.nacl_evict.argtypes = [P, vp, vp, vp, i32, i32, i32, u64, u32, vp, vp, vp, vp, vp, sz, vp]
    lib.nacl_evict.restype = ctypes.c_int
    lib.nacl_evict_noalloc.argtypes = [P, vp, vp, vp, i32, i32, i32, u64, u32, vp, vp, vp, vp, vp, vp]
    lib.nacl_evict_noalloc.restype = ctypes.c_int
    lib.nacl_attention.argtypes = [P, vp, vp, vp, vp, vp, vp, vp]
    lib.nacl_attention.restype = ctypes.c_int
    lib.nacl_status_string.argtypes = [ctypes.c_int]
    lib.nacl_status_string.restype = ctypes.c_char_p
    lib.nacl_last_error_detail.argtypes = []
    lib.nacl_last_error_detail.restype = ctypes.c_char_p
    lib.nacl_version.argtypes = []
    lib.nacl_version.restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status):
    if status != NACL_OK:
        lib = load_library()
        raise NaclError(status, lib.nacl_last_error_detail().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _gpu(t, name, dev, shape=None, dtype=None, strides=None, contiguous=False):
    """Checks a tensor argument before its address reaches the kernels: on the
    call's GPU, of the expected shape and dtype, with the problem's strides (Q,
    K, V) or contiguous (scores, indices, outputs, workspace)."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a tensor on the GPU")
    if t.device != dev:
        raise ValueError(f"{name} is on {t.device}, the call runs on {dev}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if strides is not None and (t.dim() != 4 or t.stride(3) != 1 or tuple(t.stride()[:3]) != tuple(strides)):
        raise ValueError(f"{name} has strides {tuple(t.stride())}, the problem has {tuple(strides)} (+ 1)")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _strides(t):
    if t.dim() != 4 or t.stride(3) != 1:
        raise ValueError("Q/K/V must be [B, H, L, D] with a contiguous last dimension")
    return tuple(int(s) for s in t.stride()[:3])


class Problem:
    """nacl_problem for one layer, with its host proxy-position array kept
    alive.  `dtype` is "bf16" or "f32"."""

    def __init__(self, B, H, L, D, dtype, proxy_pos, n_protect=None, sm_scale=None,
                 q_stride=None, k_stride=None, v_stride=None, proxy_pos_dev=None, q_group=1):
        pos = [int(x) for x in proxy_pos]
        self._pos = (ctypes.c_int32 * max(1, len(pos)))(*pos)
        self.proxy_pos = pos
        self.q_group = int(q_group)
        dense = (H * L * D, L * D, D)
        dense_q = (H * self.q_group * L * D, L * D, D)
        s = _Problem()
        s.B, s.H, s.L, s.D = B, H, L, D
        s.dtype = NACL_F32 if dtype in ("f32", torch.float32) else NACL_BF16
        s.P = len(pos)
        s.n_protect = len(pos) if n_protect is None else int(n_protect)
        s.sm_scale = float(sm_scale) if sm_scale else 1.0 / (D ** 0.5)
        s.q_stride[:] = q_stride or dense_q
        s.k_stride[:] = k_stride or dense
        s.v_stride[:] = v_stride or dense
        s.proxy_pos = ctypes.cast(self._pos, ctypes.POINTER(ctypes.c_int32))
        if proxy_pos_dev is not None:
            if not (isinstance(proxy_pos_dev, torch.Tensor) and proxy_pos_dev.is_cuda and
                    proxy_pos_dev.dtype == torch.int32 and proxy_pos_dev.is_contiguous() and
                    proxy_pos_dev.numel() == len(pos)):
                raise ValueError("proxy_pos_dev must be a contiguous int32 GPU tensor with one entry per proxy")
        self._pos_dev = proxy_pos_dev
        s.proxy_pos_dev = None if proxy_pos_dev is None else proxy_pos_dev.data_ptr()
        s.q_group = self.q_group
        self.c = s

    @classmethod
    def from_tensors(cls, q, k, v, proxy_pos, n_protect=None, sm_scale=None, proxy_pos_dev=None):
        """q may have a multiple of k's heads (grouped-query attention)."""
        B, H, L, D = k.shape
        if q.dim() != 4 or q.shape[1] % H:
            raise ValueError("q must be [B, H * q_group, L, D] for k of [B, H, L, D]")
        return cls(B, H, L, D, k.dtype, proxy_pos, n_protect, sm_scale,
                   _strides(q), _strides(k), _strides(v), proxy_pos_dev, q_group=q.shape[1] // H)

    @property
    def B(self):
        return self.c.B

    @property
    def H(self):
        return self.c.H

    @property
    def L(self):
        return self.c.L

    @property
    def D(self):
        return self.c.D

    @property
    def torch_dtype(self):
        return torch.float32 if self.c.dtype == NACL_F32 else torch.bfloat16

    def ref(self):
        return ctypes.byref(self.c)

    # Shapes the entry points expect.
    def qkv(self, t, name, dev, which):
        st = {"q": self.c.q_stride, "k": self.c.k_stride, "v": self.c.v_stride}[which]
        heads = self.H * self.q_group if which == "q" else self.H
        return _gpu(t, name, dev, (self.B, heads, self.L, self.D), self.torch_dtype, tuple(st))


def workspace_bytes(prob):
    return int(load_library().nacl_workspace_bytes(prob.ref()))


def workspace(prob, device="cuda"):
    """A workspace for prob, zeroed so that its sticky health word starts
    clean (the library itself needs no initialised contents)."""
    n = workspace_bytes(prob)
    if n == 0:
        lib = load_library()
        raise NaclError(NACL_ERR_INVALID_ARG, lib.nacl_last_error_detail().decode())
    return torch.zeros(n, dtype=torch.uint8, device=device)


def health(ws):
    """(this call's, sticky) health words of a workspace (include/nacl.h);
    reading them waits for the stream."""
    w = ws[4:12].view(torch.int32).cpu()
    return int(w[0]), int(w[1])


def score(prob, q, k, ws, lse=None, out=None):
    """F [B, H, L] fp32 (Section 5.1).  lse: optional [B, H, P] natural
    log-sum-exp from the caller."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    prob.qkv(q, "q", dev, "q")
    prob.qkv(k, "k", dev, "k")
    if lse is not None:
        _gpu(lse, "lse", dev, (prob.B, prob.H * prob.q_group, prob.c.P), torch.float32, contiguous=True)
    _gpu(ws, "ws", dev, dtype=torch.uint8, contiguous=True)
    if out is None:
        out = torch.empty((prob.B, prob.H, prob.L), dtype=torch.float32, device=k.device)
    _gpu(out, "out", dev, (prob.B, prob.H, prob.L), torch.float32, contiguous=True)
    _check(lib.nacl_score(prob.ref(), _ptr(q), _ptr(k), _ptr(lse), _ptr(out), _ptr(ws),
                          ws.numel(), _stream(k.device)))
    return out


def select(prob, scores, C, Cr, sampling=SAMPLE_SOFTMAX, seed=0, layer=0, ws=None, out=None):
    """keep_idx [B, H, C] int32, ascending (Sections 5.1-5.2, Algorithm 1)."""
    lib = load_library()
    dev = _gpu(scores, "scores", scores.device, (prob.B, prob.H, prob.L), torch.float32, contiguous=True).device
    if ws is not None:
        _gpu(ws, "ws", dev, dtype=torch.uint8, contiguous=True)
    if out is None:
        out = torch.empty((prob.B, prob.H, C), dtype=torch.int32, device=scores.device)
    _gpu(out, "out", dev, (prob.B, prob.H, int(C)), torch.int32, contiguous=True)
    _check(lib.nacl_select(prob.ref(), _ptr(scores), int(C), int(Cr), int(sampling), int(seed),
                           int(layer), _ptr(out), _ptr(ws), 0 if ws is None else ws.numel(),
                           _stream(scores.device)))
    return out


def compact(prob, k, v, keep_idx, k_out=None, v_out=None, in_place=False):
    """K', V' [B, H, C, D] (Section 3).  in_place: the kept rows move to rows
    0..C-1 of each head of k and v themselves (generation-phase cache)."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    prob.qkv(k, "k", dev, "k")
    prob.qkv(v, "v", dev, "v")
    C = keep_idx.shape[-1]
    _gpu(keep_idx, "keep_idx", dev, (prob.B, prob.H, C), torch.int32, contiguous=True)
    if in_place:
        k_out, v_out = k, v
    else:
        if k_out is None:
            k_out = torch.empty((prob.B, prob.H, C, prob.D), dtype=k.dtype, device=k.device)
        if v_out is None:
            v_out = torch.empty((prob.B, prob.H, C, prob.D), dtype=v.dtype, device=v.device)
        for t, name in ((k_out, "k_out"), (v_out, "v_out")):
            _gpu(t, name, dev, (prob.B, prob.H, C, prob.D), prob.torch_dtype, contiguous=True)
    _check(lib.nacl_compact(prob.ref(), _ptr(k), _ptr(v), _ptr(keep_idx), int(C), _ptr(k_out),
                            _ptr(v_out), _stream(k.device)))
    return k_out, v_out


def attention(prob, q, k, v, out=None, lse=None, lse_proxy=False):
    """Causal attention of the prefill and each row's log-sum-exp (the
    forward pass whose log-sum-exp Appendix A.7 hands to the score).
    Returns (out [B, H*q_group, L, D] bf16, lse [B, H*q_group, L] fp32,
    lse_proxy [B, H*q_group, P] fp32 or None).  lse_proxy=True needs the
    problem's proxy_pos_dev; the result is nacl_score's lse argument."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    prob.qkv(q, "q", dev, "q")
    prob.qkv(k, "k", dev, "k")
    prob.qkv(v, "v", dev, "v")
    Hq = prob.H * prob.q_group
    if out is None:
        out = torch.empty((prob.B, Hq, prob.L, prob.D), dtype=prob.torch_dtype, device=dev)
    _gpu(out, "out", dev, (prob.B, Hq, prob.L, prob.D), prob.torch_dtype, contiguous=True)
    if lse is None:
        lse = torch.empty((prob.B, Hq, prob.L), dtype=torch.float32, device=dev)
    _gpu(lse, "lse", dev, (prob.B, Hq, prob.L), torch.float32, contiguous=True)
    lp = None
    if lse_proxy is True:
        lp = torch.empty((prob.B, Hq, prob.c.P), dtype=torch.float32, device=dev)
    elif lse_proxy is not False and lse_proxy is not None:
        lp = _gpu(lse_proxy, "lse_proxy", dev, (prob.B, Hq, prob.c.P), torch.float32, contiguous=True)
    _check(lib.nacl_attention(prob.ref(), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(lp),
                              _stream(k.device)))
    return out, lse, lp


def compact_slots(prob, k, v, keep_idx, slot_idx=None):
    """Slot form of the in-place cache update (Section 3, generation phase):
    kept rows below C stay, kept rows at or past C fill the other slots below
    C, in ascending order.  keep_idx [B, H, C] is the ascending keep set.
    Returns slot_idx [B, H, C]: the old row each slot holds afterwards."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    prob.qkv(k, "k", dev, "k")
    prob.qkv(v, "v", dev, "v")
    C = keep_idx.shape[-1]
    _gpu(keep_idx, "keep_idx", dev, (prob.B, prob.H, C), torch.int32, contiguous=True)
    if slot_idx is None:
        slot_idx = torch.empty((prob.B, prob.H, C), dtype=torch.int32, device=dev)
    _gpu(slot_idx, "slot_idx", dev, (prob.B, prob.H, C), torch.int32, contiguous=True)
    _check(lib.nacl_compact_slots(prob.ref(), _ptr(k), _ptr(v), _ptr(keep_idx), int(C), _ptr(slot_idx),
                                  _stream(k.device)))
    return slot_idx


def append(prob, k, v, row0, k_new, v_new):
    """Rows [row0, row0 + m) of every head of the cache k, v take k_new, v_new
    [B, H, m, D] (Algorithm 1, generation phase)."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    prob.qkv(k, "k", dev, "k")
    prob.qkv(v, "v", dev, "v")
    m = k_new.shape[2]
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        _gpu(t, name, dev, (prob.B, prob.H, m, prob.D), prob.torch_dtype, contiguous=True)
    _check(lib.nacl_append(prob.ref(), _ptr(k), _ptr(v), int(row0), _ptr(k_new), _ptr(v_new), int(m),
                           _stream(k.device)))


def evict(prob, q, k, v, C, Cr, sampling=SAMPLE_SOFTMAX, seed=0, layer=0, ws=None,
          scores=None, keep_idx=None, k_out=None, v_out=None, in_place=False):
    """score -> select -> compact on the current stream.  Returns
    (scores, keep_idx, k_out, v_out); with in_place the kept rows move to rows
    0..C-1 of each head of k and v, which are returned as k_out and v_out."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        prob.qkv(t, name, dev, name)
    if ws is None:
        ws = workspace(prob, dev)
    if scores is None:
        scores = torch.empty((prob.B, prob.H, prob.L), dtype=torch.float32, device=dev)
    if keep_idx is None:
        keep_idx = torch.empty((prob.B, prob.H, C), dtype=torch.int32, device=dev)
    if in_place:
        k_out, v_out = k, v
    else:
        if k_out is None:
            k_out = torch.empty((prob.B, prob.H, C, prob.D), dtype=k.dtype, device=dev)
        if v_out is None:
            v_out = torch.empty((prob.B, prob.H, C, prob.D), dtype=v.dtype, device=dev)
        for t, name in ((k_out, "k_out"), (v_out, "v_out")):
            _gpu(t, name, dev, (prob.B, prob.H, int(C), prob.D), prob.torch_dtype, contiguous=True)
    _gpu(ws, "ws", dev, dtype=torch.uint8, contiguous=True)
    _gpu(scores, "scores", dev, (prob.B, prob.H, prob.L), torch.float32, contiguous=True)
    _gpu(keep_idx, "keep_idx", dev, (prob.B, prob.H, int(C)), torch.int32, contiguous=True)
    _check(lib.nacl_evict(prob.ref(), _ptr(q), _ptr(k), _ptr(v), int(C), int(Cr), int(sampling),
                          int(seed), int(layer), _ptr(scores), _ptr(keep_idx), _ptr(k_out),
                          _ptr(v_out), _ptr(ws), ws.numel(), _stream(dev)))
    return scores, keep_idx, k_out, v_out


def evict_slots(prob, q, k, v, C, Cr, sampling=SAMPLE_SOFTMAX, seed=0, layer=0, ws=None,
                scores=None, keep_idx=None, slot_idx=None):
    """score -> select -> slot-form in-place update of k, v on the current
    stream (generation-phase eviction, Section 3).  Returns (scores, keep_idx,
    slot_idx): the ascending keep set and the old row each slot below C
    holds afterwards."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        prob.qkv(t, name, dev, name)
    if ws is None:
        ws = workspace(prob, dev)
    if scores is None:
        scores = torch.empty((prob.B, prob.H, prob.L), dtype=torch.float32, device=dev)
    if keep_idx is None:
        keep_idx = torch.empty((prob.B, prob.H, C), dtype=torch.int32, device=dev)
    if slot_idx is None:
        slot_idx = torch.empty((prob.B, prob.H, C), dtype=torch.int32, device=dev)
    _gpu(ws, "ws", dev, dtype=torch.uint8, contiguous=True)
    _gpu(scores, "scores", dev, (prob.B, prob.H, prob.L), torch.float32, contiguous=True)
    for t, name in ((keep_idx, "keep_idx"), (slot_idx, "slot_idx")):
        _gpu(t, name, dev, (prob.B, prob.H, int(C)), torch.int32, contiguous=True)
    _check(lib.nacl_evict_slots(prob.ref(), _ptr(q), _ptr(k), _ptr(v), int(C), int(Cr), int(sampling),
                                int(seed), int(layer), _ptr(scores), _ptr(keep_idx), _ptr(slot_idx),
                                _ptr(ws), ws.numel(), _stream(dev)))
    return scores, keep_idx, slot_idx


NOALLOC_WORKSPACE_MAX = 64 << 20


def evict_noalloc(prob, q, k, v, C, Cr, sampling=SAMPLE_SOFTMAX, seed=0, layer=0,
                  scores=None, keep_idx=None, k_out=None, v_out=None, health=None):
    """nacl_evict_noalloc: the same step with the library's built-in device
    scratch as workspace (no workspace argument).  prob must carry a device
    copy of the proxy positions.  health: optional int32 [2] GPU tensor that
    receives the call's health words.  Outputs must be given or are
    allocated here by torch before the call (the library allocates
    nothing)."""
    lib = load_library()
    dev = _gpu(k, "k", k.device).device
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        prob.qkv(t, name, dev, name)
    if scores is None:
        scores = torch.empty((prob.B, prob.H, prob.L), dtype=torch.float32, device=dev)
    if keep_idx is None:
        keep_idx = torch.empty((prob.B, prob.H, C), dtype=torch.int32, device=dev)
    if k_out is None:
        k_out = torch.empty((prob.B, prob.H, C, prob.D), dtype=k.dtype, device=dev)
    if v_out is None:
        v_out = torch.empty((prob.B, prob.H, C, prob.D), dtype=v.dtype, device=dev)
    _gpu(scores, "scores", dev, (prob.B, prob.H, prob.L), torch.float32, contiguous=True)
    _gpu(keep_idx, "keep_idx", dev, (prob.B, prob.H, int(C)), torch.int32, contiguous=True)
    if k_out is not k:
        for t, name in ((k_out, "k_out"), (v_out, "v_out")):
            _gpu(t, name, dev, (prob.B, prob.H, int(C), prob.D), prob.torch_dtype, contiguous=True)
    if health is not None:
        _gpu(health, "health", dev, (2,), torch.int32, contiguous=True)
    _check(lib.nacl_evict_noalloc(prob.ref(), _ptr(q), _ptr(k), _ptr(v), int(C), int(Cr), int(sampling),
                                  int(seed), int(layer), _ptr(scores), _ptr(keep_idx), _ptr(k_out),
                                  _ptr(v_out), _ptr(health), _stream(dev)))
    return scores, keep_idx, k_out, v_out
