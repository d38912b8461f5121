"""ctypes binding of liblst (include/lst.h): argument marshalling only.

Every step of the method runs in the HIP kernels of liblst.so.  PyTorch
provides device memory and the stream; tensors are passed as raw device
pointers.  There is no fallback: if the library is not built, or no GPU is
visible, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch  # loaded before liblst so both share one HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblst.so")

LST_LOSS_SQUARED = 0
LST_LOSS_SPHERICAL_SOFTMAX = 1
LST_LOSS_TAYLOR_SOFTMAX = 2
LOSSES = {"squared": LST_LOSS_SQUARED, "spherical_softmax": LST_LOSS_SPHERICAL_SOFTMAX,
          "taylor_softmax": LST_LOSS_TAYLOR_SOFTMAX}

LST_OK = 0
LST_E_ARG = -1
LST_E_SHAPE = -2
LST_E_INDEX = -3
LST_E_NOT_SPD = -4
LST_E_NONFINITE = -5
LST_E_HIP = -6
LST_E_STATE = -7
LST_E_SYNC = -8

# Exported C symbols and their signatures (kept in step with include/lst.h).
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_F = ctypes.c_float
SIGNATURES = {
    "lst_workspace_bytes": (ctypes.c_size_t, [_I64, _I32, _I32, _I32, _I32]),
    "lst_naive_workspace_bytes": (ctypes.c_size_t, [_I64, _I32, _I32, _I32, _I32]),
    "lst_create": (_I32, [ctypes.POINTER(_P), _I64, _I32, _I32, _I32, _I32, _F, _P, _I64, _P, _P,
                          _P, _P, _I32, _P, ctypes.c_size_t, _P]),
    "lst_set_option": (_I32, [_P, _I32, _I64]),
    "lst_init_factored": (_I32, [_P, _P, _I64, _P, _I32]),
    "lst_step": (_I32, [_P, _P, _I32, _P, _P, _I32, _F, _P, _P]),
    "lst_materialize_W": (_I32, [_P, _P, _I64]),
    "lst_sync_status": (_I32, [_P]),
    "lst_status_string": (ctypes.c_char_p, [_I32]),
    "lst_destroy": (None, [_P]),
    "lst_naive_create": (_I32, [ctypes.POINTER(_P), _I64, _I32, _I32, _I32, _I32, _F, _P, _I64,
                                _P, ctypes.c_size_t, _P]),
    "lst_naive_step": (_I32, [_P, _P, _I32, _P, _P, _I32, _F, _P, _P]),
    "lst_use_graphs": (_I32, [_P, _I32]),
    "lst_profile_enable": (_I32, [_P, _I32]),
    "lst_profile_read": (_I32, [_P, ctypes.POINTER(_I32), ctypes.POINTER(ctypes.c_double), _I32]),
    "lst_input_forward": (_I32, [_P, _I64, _I64, _I32, _P, _P, _I32, _I32, _P, _P, _P]),
    "lst_input_update": (_I32, [_P, _I64, _I64, _I32, _P, _P, _I32, _I32, _P, _F, _P, _P]),
    "lst_step_noalloc": (_I32, [_I64, _I32, _I32, _F, _P, _I64, _P, _P, _P, _P, _I32, _P, _I32, _P,
                                _P, _I32, _F, _P, _P, _P, _P]),
    "lst_restore_pristine": (_I32, [_P]),
    "lst_refresh_uinvt": (_I32, [_P, _I32, _I32, _P]),
    "lst_power_iteration": (_I32, [_P, _I32, _I32, _P, _P, _P]),
    "lst_fix_singular_value": (_I32, [_P, _P, _P, _F]),
    "lst_singular_stabilize": (_I32, [_P, _F, _F, _I32, _P, _I32, ctypes.POINTER(_I32),
                                      ctypes.POINTER(_F)]),
}

PHASES = ["contract", "gather", "zgrad", "mid", "update", "naive_fwd", "naive_loss", "naive_grad",
          "naive_update", "online"]

LST_OPT_ONLINE_KERNEL = 0
LST_OPT_SPIN_LIMIT = 1

_lib = None
_lock = threading.Lock()


def library_path() -> str:
    return LIB_PATH


def lib() -> ctypes.CDLL:
    """Load liblst.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with paper_1606_08061_amd.build.build()")
            L = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(L, name)
                fn.restype = res
                fn.argtypes = args
            _lib = L
        return _lib


class LstError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} ({status})")


def status_string(status: int) -> str:
    return lib().lst_status_string(status).decode()


def _check(status: int, where: str) -> None:
    if status != LST_OK:
        raise LstError(status, where)


def _ptr(t) -> int:
    return 0 if t is None else t.data_ptr()


def _stream_handle(stream) -> int:
    return stream.cuda_stream if stream is not None else torch.cuda.current_stream().cuda_stream


# ---- C entry points under their own names (raw pointers and sizes) ----

def lst_workspace_bytes(D, d, m_max, K_max, loss) -> int:
    return int(lib().lst_workspace_bytes(D, d, m_max, K_max, loss))


def lst_naive_workspace_bytes(D, d, m_max, K_max, loss) -> int:
    return int(lib().lst_naive_workspace_bytes(D, d, m_max, K_max, loss))


def lst_create(D, d, m_max, K_max, loss, eps, V, ldv, U, UinvT, Q, WO, ldd, ws, ws_bytes,
               stream) -> tuple[int, int]:
    ctx = _P()
    st = lib().lst_create(ctypes.byref(ctx), D, d, m_max, K_max, loss, eps, V, ldv, U, UinvT, Q,
                          WO, ldd, ws, ws_bytes, stream)
    return st, (ctx.value or 0)


def lst_naive_create(D, d, m_max, K_max, loss, eps, W, ldw, ws, ws_bytes,
                     stream) -> tuple[int, int]:
    ctx = _P()
    st = lib().lst_naive_create(ctypes.byref(ctx), D, d, m_max, K_max, loss, eps, W, ldw, ws,
                                ws_bytes, stream)
    return st, (ctx.value or 0)


def lst_set_option(ctx, option, value) -> int:
    return lib().lst_set_option(ctx, option, value)


def lst_init_factored(ctx, V0, ldv0, U0, ldu0) -> int:
    return lib().lst_init_factored(ctx, V0, ldv0, U0, ldu0)


def lst_step(ctx, H, m, idx, val, K, lr, loss_dev, grad_H) -> int:
    return lib().lst_step(ctx, H, m, idx, val, K, lr, loss_dev, grad_H)


def lst_naive_step(ctx, H, m, idx, val, K, lr, loss_dev, grad_H) -> int:
    return lib().lst_naive_step(ctx, H, m, idx, val, K, lr, loss_dev, grad_H)


def lst_materialize_W(ctx, W, ldw) -> int:
    return lib().lst_materialize_W(ctx, W, ldw)


def lst_sync_status(ctx) -> int:
    return lib().lst_sync_status(ctx)


def lst_destroy(ctx) -> None:
    lib().lst_destroy(ctx)


def lst_use_graphs(ctx, on) -> int:
    return lib().lst_use_graphs(ctx, on)


def lst_profile_enable(ctx, on) -> int:
    return lib().lst_profile_enable(ctx, on)


def lst_profile_read(ctx) -> tuple[int, dict]:
    n = len(PHASES)
    counts = (_I32 * n)()
    ms = (ctypes.c_double * n)()
    st = lib().lst_profile_read(ctx, counts, ms, n)
    return st, {PHASES[p]: (int(counts[p]), float(ms[p])) for p in range(n)}


def lst_input_forward(W1, ldw, D_in, d, idx, val, m, K, A, status, stream) -> int:
    return lib().lst_input_forward(W1, ldw, D_in, d, idx, val, m, K, A, status, stream)


def lst_input_update(W1, ldw, D_in, d, idx, val, m, K, grad_A, lr, status, stream) -> int:
    return lib().lst_input_update(W1, ldw, D_in, d, idx, val, m, K, grad_A, lr, status, stream)


def lst_step_noalloc(D, d, loss, eps, V, ldv, U, UinvT, Q, WO, ldd, H, m, idx, val, K, lr,
                     loss_dev, grad_H, status, stream) -> int:
    return lib().lst_step_noalloc(D, d, loss, eps, V, ldv, U, UinvT, Q, WO, ldd, H, m, idx, val, K,
                                  lr, loss_dev, grad_H, status, stream)


class SparseInput:
    """The sparse input layer of section 2.2 over a D_in x d device tensor W1."""

    def __init__(self, W1, stream=None):
        _need(W1, torch.float32, tuple(W1.shape), "W1")
        if W1.dim() != 2:
            raise ValueError("W1 must be D_in x d")
        self.W1 = W1
        self.D_in, self.d = int(W1.shape[0]), int(W1.shape[1])
        self.stream = stream if stream is not None else torch.cuda.current_stream(W1.device)
        self.status = torch.zeros((), dtype=torch.int32, device=W1.device)

    def _slots(self, idx, val):
        m, K = int(idx.shape[0]), int(idx.shape[1])
        _need(idx, torch.int32, (m, K), "idx")
        _need(val, torch.float32, (m, K), "val")
        return m, K

    def forward(self, idx, val, out=None):
        m, K = self._slots(idx, val)
        if out is None:
            out = torch.empty((m, self.d), dtype=torch.float32, device=self.W1.device)
        _need(out, torch.float32, (m, self.d), "A")
        _check(lst_input_forward(_ptr(self.W1), self.d, self.D_in, self.d, _ptr(idx), _ptr(val), m,
                                 K, _ptr(out), _ptr(self.status), _stream_handle(self.stream)),
               "lst_input_forward")
        return out

    def update(self, idx, val, grad_A, lr) -> None:
        m, K = self._slots(idx, val)
        _need(grad_A, torch.float32, (m, self.d), "grad_A")
        _check(lst_input_update(_ptr(self.W1), self.d, self.D_in, self.d, _ptr(idx), _ptr(val), m,
                                K, _ptr(grad_A), float(lr), _ptr(self.status),
                                _stream_handle(self.stream)), "lst_input_update")

    def check(self) -> None:
        """Raises LstError(LST_E_INDEX) if an index was out of range (and clears the status)."""
        st = int(self.status.item())
        if st:
            self.status.zero_()
            raise LstError(LST_E_INDEX, "sparse input layer")


def lst_restore_pristine(ctx) -> int:
    return lib().lst_restore_pristine(ctx)


def lst_refresh_uinvt(ctx, iters, from_scratch, resid_dev) -> int:
    return lib().lst_refresh_uinvt(ctx, iters, from_scratch, resid_dev)


def lst_power_iteration(ctx, which, log2_iters, u0, u_out, sigma_out) -> int:
    return lib().lst_power_iteration(ctx, which, log2_iters, u0, u_out, sigma_out)


def lst_fix_singular_value(ctx, u, sigma_dev, target) -> int:
    return lib().lst_fix_singular_value(ctx, u, sigma_dev, target)


def lst_singular_stabilize(ctx, lo, hi, log2_iters, u0, max_fixes) -> tuple[int, tuple, tuple]:
    n = (_I32 * 2)()
    sig = (_F * 2)()
    st = lib().lst_singular_stabilize(ctx, lo, hi, log2_iters, u0, max_fixes, n, sig)
    return st, (int(n[0]), int(n[1])), (float(sig[0]), float(sig[1]))


# ---- tensor-level wrappers ----

def _need(t, dtype, shape, name):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _workspace(nbytes: int, device) -> torch.Tensor:
    """A device workspace of nbytes (torch's allocator returns 256-byte aligned blocks)."""
    ws = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise RuntimeError("workspace is not 256-byte aligned")
    return ws


class _Ctx:
    def __init__(self, D, d, m_max, K_max, loss, eps, device, stream):
        if not torch.cuda.is_available():
            raise RuntimeError("liblst needs a GPU; none is visible")
        self.D, self.d, self.m_max, self.K_max = int(D), int(d), int(m_max), int(K_max)
        self.loss_name = loss
        self.loss = LOSSES[loss]
        self.eps = float(eps)
        self.device = torch.device(device) if device is not None else torch.device("cuda")
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.ctx = 0
        self.loss_buf = torch.zeros((), dtype=torch.float32, device=self.device)

    def _batch(self, H, idx, val):
        # one cheap combined check on the hot path; the detailed one only to report what failed
        m = H.shape[0]
        K = idx.shape[1] if idx.dim() == 2 else -1
        if not (H.is_cuda and idx.is_cuda and val.is_cuda and H.dtype is torch.float32
                and idx.dtype is torch.int32 and val.dtype is torch.float32
                and H.dim() == 2 and H.shape[1] == self.d and idx.shape[0] == m
                and val.shape == idx.shape and H.is_contiguous() and idx.is_contiguous()
                and val.is_contiguous()):
            _need(H, torch.float32, (m, self.d), "H")
            _need(idx, torch.int32, (m, max(K, 0)), "idx")
            _need(val, torch.float32, (m, max(K, 0)), "val")
        return m, K

    def sync_status(self) -> int:
        return lst_sync_status(self.ctx)

    def check(self, where="lst_sync_status") -> None:
        _check(self.sync_status(), where)

    def profile(self, on: bool = True) -> None:
        _check(lst_profile_enable(self.ctx, 1 if on else 0), "lst_profile_enable")

    def profile_read(self) -> dict:
        """{phase: (launches, total ms)} since the last enable / read."""
        st, res = lst_profile_read(self.ctx)
        _check(st, "lst_profile_read")
        return res

    def close(self) -> None:
        if self.ctx:
            lst_destroy(self.ctx)
            self.ctx = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Factored(_Ctx):
    """The factored output layer W = V U with Q and U^{-T} (device tensors V, U, UinvT, Q)."""

    def __init__(self, D, d, m_max, K_max, loss="squared", eps=1e-3, device=None, stream=None):
        super().__init__(D, d, m_max, K_max, loss, eps, device, stream)
        kw = dict(dtype=torch.float32, device=self.device)
        self.V = torch.zeros((self.D, self.d), **kw)
        self.U = torch.zeros((self.d, self.d), **kw)
        self.UinvT = torch.zeros((self.d, self.d), **kw)
        self.Q = torch.zeros((self.d, self.d), **kw)
        # w_bar (row 0) and omega (row 1) of W = V U + 1_D omega^T; used by the Taylor softmax
        self.WO = torch.zeros((2, self.d), **kw)
        nb = lst_workspace_bytes(self.D, self.d, self.m_max, self.K_max, self.loss)
        if nb == 0:
            raise LstError(LST_E_SHAPE, "lst_workspace_bytes")
        self.ws = _workspace(nb, self.device)
        st, self.ctx = lst_create(self.D, self.d, self.m_max, self.K_max, self.loss, self.eps,
                                  _ptr(self.V), self.d, _ptr(self.U), _ptr(self.UinvT),
                                  _ptr(self.Q), _ptr(self.WO), self.d, _ptr(self.ws), nb,
                                  _stream_handle(self.stream))
        _check(st, "lst_create")
        self._step_fn = lib().lst_step

    @property
    def wbar(self):
        return self.WO[0]

    @property
    def omega(self):
        return self.WO[1]

    def init(self, V0=None, U0=None) -> None:
        """Algorithm 1: V = V0, U = U0 (or I), then U^{-T}, Q and w_bar from them (omega as
        it stands in WO[1]: zero unless the caller set it)."""
        if V0 is not None:
            _need(V0, torch.float32, (self.D, self.d), "V0")
        if U0 is not None:
            _need(U0, torch.float32, (self.d, self.d), "U0")
        _check(lst_init_factored(self.ctx, _ptr(V0), self.d, _ptr(U0), self.d),
               "lst_init_factored")

    def step(self, H, idx, val, lr, grad_H=None, loss_out=None, want_grad=True):
        m, K = self._batch(H, idx, val)
        if grad_H is None and want_grad:
            grad_H = torch.empty((m, self.d), dtype=torch.float32, device=self.device)
        if grad_H is not None and not (grad_H.is_cuda and grad_H.dtype is torch.float32
                                       and grad_H.shape == H.shape and grad_H.is_contiguous()):
            _need(grad_H, torch.float32, (m, self.d), "grad_H")
        loss_out = self.loss_buf if loss_out is None else loss_out
        st = self._step_fn(self.ctx, H.data_ptr(), m, idx.data_ptr(), val.data_ptr(), K, lr,
                           loss_out.data_ptr(), 0 if grad_H is None else grad_H.data_ptr())
        if st:
            _check(st, "lst_step")
        return loss_out, grad_H

    def materialize_W(self, out=None):
        if out is None:
            out = torch.empty((self.D, self.d), dtype=torch.float32, device=self.device)
        _need(out, torch.float32, (self.D, self.d), "W")
        _check(lst_materialize_W(self.ctx, _ptr(out), self.d), "lst_materialize_W")
        return out

    def use_graphs(self, on: bool = True) -> None:
        _check(lst_use_graphs(self.ctx, 1 if on else 0), "lst_use_graphs")

    def set_option(self, option: int, value: int) -> None:
        _check(lst_set_option(self.ctx, int(option), int(value)), "lst_set_option")

    # ---- section 5: numerical stabilisation between steps ----

    def restore_pristine(self) -> None:
        """V <- V U, U <- I, U^{-T} <- I (in place; d <= 1024)."""
        _check(lst_restore_pristine(self.ctx), "lst_restore_pristine")

    def refresh_uinvt(self, iters=2, from_scratch=False, resid=None):
        """Recompute U^{-T} from U (Newton-Schulz rounds); resid: optional 0-d device tensor
        receiving max |I - U^{-T} U^T|."""
        if resid is not None:
            _need(resid, torch.float32, (), "resid")
        _check(lst_refresh_uinvt(self.ctx, int(iters), 1 if from_scratch else 0, _ptr(resid)),
               "lst_refresh_uinvt")
        return resid

    def power_iteration(self, which, log2_iters, u0, u_out=None, sigma_out=None):
        """which = "largest" or "smallest" singular value of U; returns (u, sigma) device tensors."""
        w = {"largest": 0, "smallest": 1}[which]
        _need(u0, torch.float32, (self.d,), "u0")
        if u_out is None:
            u_out = torch.empty(self.d, dtype=torch.float32, device=self.device)
        if sigma_out is None:
            sigma_out = torch.empty((), dtype=torch.float32, device=self.device)
        _need(u_out, torch.float32, (self.d,), "u_out")
        _need(sigma_out, torch.float32, (), "sigma_out")
        _check(lst_power_iteration(self.ctx, w, int(log2_iters), _ptr(u0), _ptr(u_out),
                                   _ptr(sigma_out)), "lst_power_iteration")
        return u_out, sigma_out

    def fix_singular_value(self, u, sigma, target=1.0) -> None:
        """Algorithm 5 fix-singular-value with device tensors u (d) and sigma (0-d)."""
        _need(u, torch.float32, (self.d,), "u")
        _need(sigma, torch.float32, (), "sigma")
        _check(lst_fix_singular_value(self.ctx, _ptr(u), _ptr(sigma), float(target)),
               "lst_fix_singular_value")

    def singular_stabilize(self, u0, lo=1e-3, hi=100.0, log2_iters=7, max_fixes=8):
        """Section 5.3's loop; returns ((fixes of the smallest, of the largest),
        (last smallest, last largest singular value))."""
        _need(u0, torch.float32, (self.d,), "u0")
        st, n, sig = lst_singular_stabilize(self.ctx, float(lo), float(hi), int(log2_iters),
                                            _ptr(u0), int(max_fixes))
        _check(st, "lst_singular_stabilize")
        return n, sig


class Naive(_Ctx):
    """The naive O(D d) output layer with an explicit W (device tensor)."""

    def __init__(self, D, d, m_max, K_max, loss="squared", eps=1e-3, device=None, stream=None):
        super().__init__(D, d, m_max, K_max, loss, eps, device, stream)
        self.W = torch.zeros((self.D, self.d), dtype=torch.float32, device=self.device)
        nb = lst_naive_workspace_bytes(self.D, self.d, self.m_max, self.K_max, self.loss)
        if nb == 0:
            raise LstError(LST_E_SHAPE, "lst_naive_workspace_bytes")
        self.ws = _workspace(nb, self.device)
        st, self.ctx = lst_naive_create(self.D, self.d, self.m_max, self.K_max, self.loss,
                                        self.eps, _ptr(self.W), self.d, _ptr(self.ws), nb,
                                        _stream_handle(self.stream))
        _check(st, "lst_naive_create")
        self._step_fn = lib().lst_naive_step

    def init(self, W0) -> None:
        _need(W0, torch.float32, (self.D, self.d), "W0")
        with torch.cuda.stream(self.stream):
            self.W.copy_(W0)

    def step(self, H, idx, val, lr, grad_H=None, loss_out=None, want_grad=True):
        m, K = self._batch(H, idx, val)
        if grad_H is None and want_grad:
            grad_H = torch.empty((m, self.d), dtype=torch.float32, device=self.device)
        if grad_H is not None:
            _need(grad_H, torch.float32, (m, self.d), "grad_H")
        loss_out = self.loss_buf if loss_out is None else loss_out
        _check(self._step_fn(self.ctx, _ptr(H), m, _ptr(idx), _ptr(val), K, float(lr),
                             _ptr(loss_out), _ptr(grad_H)), "lst_naive_step")
        return loss_out, grad_H

    def materialize_W(self, out=None):
        if out is None:
            out = torch.empty((self.D, self.d), dtype=torch.float32, device=self.device)
        _need(out, torch.float32, (self.D, self.d), "W")
        _check(lst_materialize_W(self.ctx, _ptr(out), self.d), "lst_materialize_W")
        return out
