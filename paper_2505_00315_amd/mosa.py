"""Python binding of libmosa.so (ctypes): argument marshalling only.

Every step of the layer runs in the HIP kernels behind the C ABI declared in
``include/mosa.h``; PyTorch provides device memory and the current stream.
There is no fallback: if the library is not built, loading fails loudly.
"""
import ctypes
import os

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmosa.so")

MOSA_OK = 0
MOSA_ERR_INVALID_ARG = -1
MOSA_ERR_UNSUPPORTED = -2
MOSA_ERR_WORKSPACE = -3
MOSA_ERR_HIP = -4
MOSA_F32 = 0
MOSA_BF16 = 1

SYMBOLS = ("mosa_workspace_size", "mosa_saved_offsets", "mosa_forward", "mosa_backward",
           "mosa_forward_timed", "mosa_backward_timed", "mosa_status_string", "mosa_adaptive_k",
           "mosa_forward_noalloc")
NOALLOC_SCRATCH_MAX = 64 << 20  # MOSA_NOALLOC_SCRATCH_MAX
MAX_STAGES = 32

WEIGHT_NAMES = ("Wr", "Wq", "Wk", "Wv", "Wo", "Wq_d", "Wk_d", "Wv_d", "Wo_d")
GRAD_NAMES = tuple("d" + n for n in WEIGHT_NAMES)
SAVED_NAMES = ("I", "r", "slot", "QKV", "A", "lse", "QKVd", "Ad", "lsed", "rope", "status")


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("batch", "seq_len", "d_model", "heads", "d_head", "k", "causal", "dense_heads", "dtype",
                 "first_token", "fixed_stride", "rope")] + [("rope_base", ctypes.c_float), ("window", ctypes.c_int32)]


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_NAMES]


class Grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in GRAD_NAMES]


class SavedLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in SAVED_NAMES + ("total",)]


class StageEvents(ctypes.Structure):
    _fields_ = [("events", ctypes.c_void_p * MAX_STAGES), ("names", ctypes.c_char_p * MAX_STAGES),
                ("count", ctypes.c_int)]


class MosaError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(paper_2505_00315_amd/build.py); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.mosa_workspace_size.argtypes = [P(Shape), P(ctypes.c_size_t), P(ctypes.c_size_t)]
        L.mosa_saved_offsets.argtypes = [P(Shape), P(SavedLayout)]
        L.mosa_forward.argtypes = [P(Shape), ctypes.c_void_p, P(Weights), ctypes.c_void_p, ctypes.c_int,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
        L.mosa_backward.argtypes = [P(Shape), ctypes.c_void_p, P(Weights), ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, P(Grads), ctypes.c_void_p,
                                    ctypes.c_size_t, ctypes.c_void_p]
        L.mosa_forward_timed.argtypes = L.mosa_forward.argtypes + [P(StageEvents)]
        L.mosa_forward_noalloc.argtypes = [P(Shape), ctypes.c_void_p, P(Weights), ctypes.c_void_p, ctypes.c_int,
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                           ctypes.c_void_p]
        L.mosa_backward_timed.argtypes = L.mosa_backward.argtypes + [P(StageEvents)]
        L.mosa_status_string.argtypes = [ctypes.c_int]
        L.mosa_status_string.restype = ctypes.c_char_p
        L.mosa_adaptive_k.argtypes = [ctypes.c_int, ctypes.c_int]
        L.mosa_adaptive_k.restype = ctypes.c_int
        for n in ("mosa_workspace_size", "mosa_saved_offsets", "mosa_forward", "mosa_backward",
                  "mosa_forward_timed", "mosa_backward_timed", "mosa_forward_noalloc"):
            getattr(L, n).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().mosa_status_string(int(status)).decode()


def _check(status, what):
    if status != MOSA_OK:
        raise MosaError(status, what)


def make_shape(batch, seq_len, d_model, heads, d_head, k, causal=True, dense_heads=0, dtype="bf16",
               first_token=False, fixed_stride=0, rope=False, rope_base=10000.0, window=0):
    code = {"bf16": MOSA_BF16, "f32": MOSA_F32, torch.bfloat16: MOSA_BF16, torch.float32: MOSA_F32}[dtype]
    return Shape(batch, seq_len, d_model, heads, d_head, k if heads > 0 else 0, int(bool(causal)),
                 dense_heads, code, int(bool(first_token)), int(fixed_stride), int(bool(rope)),
                 float(rope_base), int(window))


def adaptive_k(seq_len, rho):
    """The paper's k for short inputs, max(floor(T / rho), 2) (Section 3.5)."""
    k = lib().mosa_adaptive_k(int(seq_len), int(rho))
    if k <= 0:
        raise ValueError(f"adaptive_k: invalid seq_len={seq_len} or rho={rho}")
    return k


def torch_dtype(shape: Shape):
    return torch.bfloat16 if shape.dtype == MOSA_BF16 else torch.float32


def workspace_size(shape: Shape):
    saved, scratch = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().mosa_workspace_size(ctypes.byref(shape), ctypes.byref(saved), ctypes.byref(scratch)),
           "mosa_workspace_size")
    return saved.value, scratch.value


def saved_offsets(shape: Shape):
    out = SavedLayout()
    _check(lib().mosa_saved_offsets(ctypes.byref(shape), ctypes.byref(out)), "mosa_saved_offsets")
    return {n: getattr(out, n) for n in SAVED_NAMES + ("total",)}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def alloc_workspace(shape: Shape, device="cuda"):
    saved, scratch = workspace_size(shape)
    return (torch.empty(max(saved, 256), dtype=torch.uint8, device=device),
            torch.empty(max(scratch, 256), dtype=torch.uint8, device=device))


def _weights(w):
    return Weights(*[_ptr(w.get(n)) for n in WEIGHT_NAMES])


def _weight_numel(shape: Shape):
    """Element counts of the parameters (Wr [H,d]; Wq/Wk/Wv [H,d,dh]; Wo [H,dh,d];
    dense heads the same with Hd)."""
    H, Hd, d, dh = shape.heads, shape.dense_heads, shape.d_model, shape.d_head
    return {"Wr": H * d, "Wq": H * d * dh, "Wk": H * d * dh, "Wv": H * d * dh, "Wo": H * dh * d,
            "Wq_d": Hd * d * dh, "Wk_d": Hd * d * dh, "Wv_d": Hd * d * dh, "Wo_d": Hd * dh * d}


def _check_tensor(t, what, dtype, numel, device):
    """A tensor handed to the library must have the storage type, element
    count and device the shape implies and be contiguous: the kernels index
    it by the shape alone, so anything else would read or write out of bounds."""
    if t is None:
        raise ValueError(f"{what}: missing")
    if t.dtype != dtype:
        raise TypeError(f"{what}: dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what}: not contiguous")
    if t.numel() != numel:
        raise ValueError(f"{what}: {t.numel()} elements, expected {numel}")
    if t.device != device:
        raise ValueError(f"{what}: on {t.device}, expected {device}")


def _check_params(shape: Shape, params, names, device, optional=()):
    st = torch_dtype(shape)
    for n, numel in zip(names, _weight_numel(shape).values()):
        t = params.get(n)
        if numel == 0 or (t is None and n in optional):
            continue
        _check_tensor(t, n, st, numel, device)


def _check_buffers(shape: Shape, saved, scratch, device):
    need_saved, need_scratch = workspace_size(shape)
    for t, what, need in ((saved, "saved", need_saved), (scratch, "scratch", need_scratch)):
        if t is None or t.dtype != torch.uint8 or not t.is_contiguous() or t.device != device:
            raise ValueError(f"{what}: a contiguous uint8 tensor on {device} is required")
        if t.numel() < need:
            raise ValueError(f"{what}: {t.numel()} bytes, at least {need} required")


def forward(shape: Shape, X, w, Y=None, accumulate=False, saved=None, scratch=None, I_out=None, r_out=None,
            stream=None, events=None):
    """Run mosa_forward (mosa_forward_timed when ``events`` is a StageEvents).
    ``w`` maps weight names (see WEIGHT_NAMES) to device tensors.
    Returns (Y, saved, scratch)."""
    st = torch_dtype(shape)
    dev = X.device
    act = shape.batch * shape.seq_len * shape.d_model
    _check_tensor(X, "X", st, act, dev)
    if dev.type != "cuda":
        raise ValueError("X: the layer runs on the GPU only")
    _check_params(shape, w, WEIGHT_NAMES, dev, optional=("Wr",) if shape.fixed_stride else ())
    if Y is None:
        Y = torch.empty_like(X)
    _check_tensor(Y, "Y", st, act, dev)
    if saved is None or scratch is None:
        saved, scratch = alloc_workspace(shape, dev)
    _check_buffers(shape, saved, scratch, dev)
    sel = shape.batch * shape.heads * shape.k
    if I_out is not None:
        _check_tensor(I_out, "I_out", torch.int32, sel, dev)
    if r_out is not None:
        _check_tensor(r_out, "r_out", torch.float32, sel, dev)
    args = [ctypes.byref(shape), _ptr(X), ctypes.byref(_weights(w)), _ptr(Y), int(accumulate), _ptr(I_out),
            _ptr(r_out), _ptr(saved), saved.numel(), _ptr(scratch), scratch.numel(), _stream(stream)]
    if events is None:
        _check(lib().mosa_forward(*args), "mosa_forward")
    else:
        _check(lib().mosa_forward_timed(*args, ctypes.byref(events)), "mosa_forward_timed")
    return Y, saved, scratch


def forward_noalloc(shape: Shape, X, w, Y=None, accumulate=False, saved=None, I_out=None, r_out=None,
                    stream=None):
    """Run mosa_forward_noalloc (scratch from the library's static buffer).
    Returns (Y, saved)."""
    st = torch_dtype(shape)
    dev = X.device
    act = shape.batch * shape.seq_len * shape.d_model
    _check_tensor(X, "X", st, act, dev)
    if dev.type != "cuda":
        raise ValueError("X: the layer runs on the GPU only")
    _check_params(shape, w, WEIGHT_NAMES, dev, optional=("Wr",) if shape.fixed_stride else ())
    if Y is None:
        Y = torch.empty_like(X)
    _check_tensor(Y, "Y", st, act, dev)
    need_saved, _ = workspace_size(shape)
    if saved is None:
        saved = torch.empty(max(need_saved, 256), dtype=torch.uint8, device=dev)
    if saved.dtype != torch.uint8 or not saved.is_contiguous() or saved.device != dev or saved.numel() < need_saved:
        raise ValueError(f"saved: a contiguous uint8 tensor on {dev} of at least {need_saved} bytes is required")
    sel = shape.batch * shape.heads * shape.k
    if I_out is not None:
        _check_tensor(I_out, "I_out", torch.int32, sel, dev)
    if r_out is not None:
        _check_tensor(r_out, "r_out", torch.float32, sel, dev)
    _check(lib().mosa_forward_noalloc(ctypes.byref(shape), _ptr(X), ctypes.byref(_weights(w)), _ptr(Y),
                                      int(accumulate), _ptr(I_out), _ptr(r_out), _ptr(saved), saved.numel(),
                                      _stream(stream)), "mosa_forward_noalloc")
    return Y, saved


def backward(shape: Shape, X, w, dY, saved, grads, dX=None, accumulate_dX=False, scratch=None, stream=None,
             events=None):
    """Run mosa_backward (mosa_backward_timed when ``events`` is given).
    ``grads`` maps gradient names (see GRAD_NAMES) to device tensors that are
    written.  Returns dX."""
    st = torch_dtype(shape)
    dev = X.device
    act = shape.batch * shape.seq_len * shape.d_model
    _check_tensor(X, "X", st, act, dev)
    if dev.type != "cuda":
        raise ValueError("X: the layer runs on the GPU only")
    _check_tensor(dY, "dY", st, act, dev)
    _check_params(shape, w, WEIGHT_NAMES, dev, optional=("Wr",) if shape.fixed_stride else ())
    _check_params(shape, grads, GRAD_NAMES, dev, optional=("dWr",) if shape.fixed_stride else ())
    if dX is None:
        dX = torch.empty_like(X)
    _check_tensor(dX, "dX", st, act, dev)
    if scratch is None:
        _, scratch = alloc_workspace(shape, dev)
    _check_buffers(shape, saved, scratch, dev)
    g = Grads(*[_ptr(grads.get(n)) for n in GRAD_NAMES])
    args = [ctypes.byref(shape), _ptr(X), ctypes.byref(_weights(w)), _ptr(dY), _ptr(saved), saved.numel(), _ptr(dX),
            int(accumulate_dX), ctypes.byref(g), _ptr(scratch), scratch.numel(), _stream(stream)]
    if events is None:
        _check(lib().mosa_backward(*args), "mosa_backward")
    else:
        _check(lib().mosa_backward_timed(*args, ctypes.byref(events)), "mosa_backward_timed")
    return dX


class SelectionError(RuntimeError):
    """The certified selection of some (b, h) rows did not hold exactly k tokens."""


def check_selection(shape: Shape, saved):
    """Raise SelectionError when the forward flagged a row whose selection is
    not certified (the router's logit error bound failed); waits for the
    forward to finish."""
    if shape.heads == 0:
        return
    bad = saved_view(shape, saved, "status")
    n = int((bad != 0).sum().item())
    if n:
        rows = (bad != 0).nonzero()[:8].tolist()
        raise SelectionError(f"{n} (b, h) rows without a certified top-{shape.k} selection, e.g. {rows}")


class StageTimer:
    """hipEvent_t handles for the timed entry points: ``sets`` StageEvents
    objects, each with MAX_STAGES events (created through the HIP runtime the
    library links against)."""

    def __init__(self, sets=1):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.handles = []
        self.sets = []
        for _ in range(sets):
            ev = StageEvents()
            for i in range(MAX_STAGES):
                h = ctypes.c_void_p()
                if self.hip.hipEventCreate(ctypes.byref(h)) != 0:
                    raise RuntimeError("hipEventCreate failed")
                self.handles.append(h.value)
                ev.events[i] = h.value
            self.sets.append(ev)

    def elapsed_ms(self, a, b):
        out = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(out), ctypes.c_void_p(a), ctypes.c_void_p(b)) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return out.value

    def stages(self, ev):
        """[(stage name, ms)] of one recorded StageEvents, in launch order."""
        return [(ev.names[j].decode(), self.elapsed_ms(ev.events[j - 1], ev.events[j])) for j in range(1, ev.count)]

    def close(self):
        for h in self.handles:
            self.hip.hipEventDestroy(ctypes.c_void_p(h))
        self.handles = []


def saved_view(shape: Shape, saved, name):
    """Typed view of one tensor the forward keeps in ``saved`` (for inspection).
    "Q", "K", "V" (and "Qd", "Kd", "Vd") are slices of the packed QKV rows."""
    part = {"Q": 0, "K": 1, "V": 2, "Qd": 0, "Kd": 1, "Vd": 2}
    if name in part:
        whole = saved_view(shape, saved, "QKV" if len(name) == 1 else "QKVd")
        return whole[..., part[name], :]
    off = saved_offsets(shape)
    B, T, H, Hd, k, dh = shape.batch, shape.seq_len, shape.heads, shape.dense_heads, shape.k, shape.d_head
    st = torch_dtype(shape)
    spec = {"I": (torch.int32, (B, H, k)), "r": (torch.float32, (B, H, k)), "slot": (torch.int16, (B, H, T)),
            "QKV": (st, (B, H, k, 3, dh)), "A": (st, (B, H, k, dh)), "lse": (torch.float32, (B, H, k)),
            "QKVd": (st, (B, Hd, T, 3, dh)), "Ad": (st, (B, Hd, T, dh)), "lsed": (torch.float32, (B, Hd, T)),
            "status": (torch.int32, (B, H))}[name]
    dt, shp = spec
    n = 1
    for s in shp:
        n *= s
    nbytes = n * torch.tensor([], dtype=dt).element_size()
    return saved[off[name]: off[name] + nbytes].view(dt).view(shp)
