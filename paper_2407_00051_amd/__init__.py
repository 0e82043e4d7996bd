"""Python binding of libsagips.so, the MI355X (gfx950) implementation of one
rank's SAGIPS sample -> discriminate -> backward step (arXiv 2407.00051).

The binding only marshals arguments: every step runs in the library's HIP
kernels.  PyTorch supplies device memory and the stream (the context runs on
torch's current stream of its device unless another is set).  There is no
CPU fallback: if the library is missing or fails to load, importing the
calls raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsagips.so")
MAX_LAYERS = 8
MAX_TENSORS = 16

OK, E_INVAL, E_ARCH, E_NOMEM, E_HIP, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
FEAT_IDENTITY, FEAT_HD8, FEAT_PROXY2 = 0, 1, 2
CRITIC_BUFFER, CRITIC_QUADRATIC = 0, 1

EXPORTED = ("sagips_create", "sagips_destroy", "sagips_set_stream", "sagips_set_bf16_chunk_rows",
            "sagips_last_error", "sagips_set_timing",
            "sagips_kernel_times", "sagips_sample_events", "sagips_disc_fwd_bwd", "sagips_param_grad",
            "sagips_bootstrap", "sagips_bootstrap_rows", "sagips_gen_forward", "sagips_gen_backward", "sagips_ensemble_response",
            "sagips_adam_step", "sagips_disc_fwd_bwd_noalloc", "sagips_noalloc_scratch_bytes")


class SagipsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"sagips status {status}: {message}")
        self.status = status


class Source(ctypes.Structure):
    _fields_ = [("theta", ctypes.c_void_p), ("n_theta", ctypes.c_int32), ("d", ctypes.c_int32),
                ("events_per_theta", ctypes.c_int64), ("seed", ctypes.c_uint64),
                ("counter_base", ctypes.c_uint64), ("stream", ctypes.c_uint32)]


class Mlp(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("width", ctypes.c_int32 * (MAX_LAYERS + 1)),
                ("W", ctypes.c_void_p * MAX_LAYERS), ("b", ctypes.c_void_p * MAX_LAYERS),
                ("leaky_slope", ctypes.c_float), ("precision", ctypes.c_int32), ("features", ctypes.c_int32)]


class GenStack(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("width", ctypes.c_int32 * (MAX_LAYERS + 1)),
                ("W", ctypes.c_void_p * MAX_LAYERS), ("b", ctypes.c_void_p * MAX_LAYERS),
                ("n_members", ctypes.c_int32), ("leaky_slope", ctypes.c_float)]


class ParamSet(ctypes.Structure):
    _fields_ = [("n_tensors", ctypes.c_int32), ("param", ctypes.c_void_p * MAX_TENSORS),
                ("grad", ctypes.c_void_p * MAX_TENSORS), ("m", ctypes.c_void_p * MAX_TENSORS),
                ("v", ctypes.c_void_p * MAX_TENSORS), ("size", ctypes.c_int64 * MAX_TENSORS)]


class DiscOut(ctypes.Structure):
    _fields_ = [("logits_fake", ctypes.c_void_p), ("logits_real", ctypes.c_void_p),
                ("loss_d", ctypes.c_void_p), ("loss_g", ctypes.c_void_p),
                ("dW", ctypes.c_void_p * MAX_LAYERS), ("db", ctypes.c_void_p * MAX_LAYERS),
                ("dLg_dx", ctypes.c_void_p), ("dLg_dtheta", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsagips.so (once) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run python -m paper_2407_00051_amd.build")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.sagips_create.argtypes = [ctypes.POINTER(vp), i32, vp]
    lib.sagips_destroy.argtypes = [vp]
    lib.sagips_set_stream.argtypes = [vp, vp]
    lib.sagips_set_bf16_chunk_rows.argtypes = [vp, i64]
    lib.sagips_last_error.argtypes = [vp]
    lib.sagips_last_error.restype = ctypes.c_char_p
    lib.sagips_set_timing.argtypes = [vp, i32]
    lib.sagips_kernel_times.argtypes = [vp, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(i64),
                                        ctypes.POINTER(ctypes.c_double), i32]
    lib.sagips_sample_events.argtypes = [vp, ctypes.POINTER(Source), vp, vp]
    lib.sagips_disc_fwd_bwd.argtypes = [vp, ctypes.POINTER(Mlp), vp, ctypes.POINTER(Source), i64, vp, i64,
                                        ctypes.POINTER(DiscOut)]
    lib.sagips_disc_fwd_bwd_noalloc.argtypes = lib.sagips_disc_fwd_bwd.argtypes
    lib.sagips_noalloc_scratch_bytes.argtypes = []
    lib.sagips_noalloc_scratch_bytes.restype = ctypes.c_size_t
    lib.sagips_param_grad.argtypes = [vp, ctypes.POINTER(Source), i32, vp, vp, vp]
    lib.sagips_bootstrap.argtypes = [vp, vp, i64, i32, ctypes.c_uint64, ctypes.c_uint32, i64, vp, vp]
    lib.sagips_bootstrap_rows.argtypes = lib.sagips_bootstrap.argtypes
    lib.sagips_gen_forward.argtypes = [vp, ctypes.POINTER(GenStack), vp, i64, vp]
    lib.sagips_gen_backward.argtypes = [vp, ctypes.POINTER(GenStack), vp, i64, vp, ctypes.POINTER(vp),
                                        ctypes.POINTER(vp)]
    lib.sagips_ensemble_response.argtypes = [vp, ctypes.POINTER(GenStack), vp, i64, vp, vp, vp, vp]
    lib.sagips_adam_step.argtypes = [vp, ctypes.POINTER(ParamSet), i32, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_double]
    for name in ("sagips_create", "sagips_destroy", "sagips_set_stream", "sagips_set_bf16_chunk_rows",
                 "sagips_set_timing",
                 "sagips_kernel_times", "sagips_sample_events", "sagips_disc_fwd_bwd", "sagips_param_grad",
                 "sagips_bootstrap", "sagips_bootstrap_rows", "sagips_gen_forward", "sagips_gen_backward", "sagips_ensemble_response",
                 "sagips_adam_step", "sagips_disc_fwd_bwd_noalloc"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _check_tensor(t, name, dtype=None, shape=None, device=None):
    import torch
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a GPU device")
    if device is not None and t.device.index != device:
        raise ValueError(f"{name} is on cuda:{t.device.index}, the context on cuda:{device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


class Context:
    """A library context on one GPU.

    Without a stream it follows torch: every call runs on torch's current stream
    of the device at the time of the call, the stream on which the binding also
    allocates the outputs it returns.  With an explicit stream every call runs
    there, and outputs the binding allocates are marked as used by that stream
    (record_stream), so that torch's caching allocator does not hand their memory
    out again before the library's kernels are done with it."""

    def __init__(self, device: int = 0, stream=None):
        import torch
        self.lib = load_library()
        self.device = device
        self._follow = stream is None
        if stream is None:
            stream = torch.cuda.current_stream(device)
        self._stream = stream
        h = ctypes.c_void_p()
        st = self.lib.sagips_create(ctypes.byref(h), device, ctypes.c_void_p(stream.cuda_stream))
        if st != OK:
            raise SagipsError(st, self.lib.sagips_last_error(None).decode())
        self.h = h

    # -- plumbing -------------------------------------------------------------
    def _check(self, st: int):
        if st != OK:
            raise SagipsError(st, self.lib.sagips_last_error(self.h).decode())

    def close(self):
        if getattr(self, "h", None):
            self.lib.sagips_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def stream(self):
        return self._stream

    def set_stream(self, stream):
        """Run later calls on `stream` (and stop following torch's current stream)."""
        self._check(self.lib.sagips_set_stream(self.h, ctypes.c_void_p(stream.cuda_stream)))
        self._stream = stream
        self._follow = False

    def _enter(self):
        """Before a call: in follow mode, switch to torch's current stream if it changed."""
        if self._follow:
            import torch
            cur = torch.cuda.current_stream(self.device)
            if cur.cuda_stream != self._stream.cuda_stream:
                self._check(self.lib.sagips_set_stream(self.h, ctypes.c_void_p(cur.cuda_stream)))
                self._stream = cur

    def _owned(self, *tensors):
        """Outputs the binding allocated on torch's current stream, used by the library's stream."""
        if self._follow:
            return
        import torch
        if torch.cuda.current_stream(self.device).cuda_stream == self._stream.cuda_stream:
            return
        for t in tensors:
            if isinstance(t, (list, tuple)):
                self._owned(*t)
            elif t is not None:
                t.record_stream(self._stream)

    def set_bf16_chunk_rows(self, rows: int = 0):
        """Rows per chunk of the bf16 discriminator (0: the default, 4,194,304)."""
        self._check(self.lib.sagips_set_bf16_chunk_rows(self.h, int(rows)))

    def set_timing(self, enable: bool):
        self._check(self.lib.sagips_set_timing(self.h, 1 if enable else 0))

    def kernel_times(self) -> Dict[str, tuple]:
        """{kernel name: (launches, total ms)} since the last call; syncs the stream."""
        cap = 64
        names = (ctypes.c_char_p * cap)()
        launches = (ctypes.c_int64 * cap)()
        ms = (ctypes.c_double * cap)()
        n = self.lib.sagips_kernel_times(self.h, names, launches, ms, cap)
        if n < 0:
            self._check(n)
        return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(min(n, cap))}

    def source(self, theta, events_per_theta: int, seed: int, counter_base: int = 0, stream: int = 0) -> Source:
        import torch
        _check_tensor(theta, "theta", torch.float32, device=self.device)
        if theta.dim() != 2 or theta.shape[1] not in (4, 6):
            raise ValueError("theta must be [n_theta][4] or [n_theta][6]")
        return Source(theta.data_ptr(), theta.shape[0], theta.shape[1] // 2, int(events_per_theta), int(seed),
                      int(counter_base), int(stream))

    # -- 1. parameters -> events ---------------------------------------------------
    def sample_events(self, theta, events_per_theta: int, seed: int, counter_base: int = 0, stream: int = 0,
                      want_x: bool = True, want_words: bool = False, out=None, words_out=None):
        """Events [N][d] fp32 (and optionally the raw Philox words [N][4] int32)."""
        import torch
        self._enter()
        src = self.source(theta, events_per_theta, seed, counter_base, stream)
        N = src.n_theta * src.events_per_theta
        x = None
        w = None
        if want_x:
            x = out if out is not None else torch.empty((N, src.d), dtype=torch.float32, device=theta.device)
            _check_tensor(x, "out", torch.float32, (N, src.d), self.device)
        if want_words:
            w = words_out if words_out is not None else torch.empty((N, 4), dtype=torch.int32, device=theta.device)
            _check_tensor(w, "words_out", torch.int32, (N, 4), self.device)
        self._owned(x if out is None else None, w if words_out is None else None)
        self._check(self.lib.sagips_sample_events(self.h, ctypes.byref(src), _ptr(x), _ptr(w)))
        self._keep = (theta,)
        if want_words and want_x:
            return x, w
        return x if want_x else w

    # -- 4. reference data -> bootstrapped sub-sample --------------------------------
    def bootstrap(self, data, n_out: int, seed: int, step: int, want_idx: bool = False, out=None, idx_out=None,
                  row_order: bool = False):
        """The step's sub-sample [n_out][d] of the rows of data (drawn with replacement), and
        optionally the drawn row indices [n_out] int64; with row_order the same multiset in
        ascending row order."""
        import torch
        self._enter()
        _check_tensor(data, "data", torch.float32, None, self.device)
        if data.dim() != 2 or data.shape[1] not in (2, 3):
            raise ValueError("data must be [n_data][d] with d in {2, 3}")
        d = data.shape[1]
        x = out if out is not None else torch.empty((n_out, d), dtype=torch.float32, device=data.device)
        _check_tensor(x, "out", torch.float32, (n_out, d), self.device)
        idx = None
        if want_idx:
            idx = idx_out if idx_out is not None else torch.empty(n_out, dtype=torch.int64, device=data.device)
            _check_tensor(idx, "idx_out", torch.int64, (n_out,), self.device)
        self._owned(x if out is None else None, idx if idx_out is None else None)
        fn = self.lib.sagips_bootstrap_rows if row_order else self.lib.sagips_bootstrap
        self._check(fn(self.h, _ptr(data), data.shape[0], d, seed & (2**64 - 1), step & 0xFFFFFFFF, n_out, _ptr(x),
                       _ptr(idx)))
        self._keep = (data,)
        return (x, idx) if want_idx else x

    # -- generator (noise -> parameters) and the ensemble response -------------------
    def _gen(self, W: Sequence, b: Sequence, slope: float):
        """GenStack for stacked members: W[l] is [M][out][in] (or [out][in] for one member),
        b[l] is [M][out] (or [out])."""
        import torch
        n_layers = len(W)
        if n_layers != len(b) or not 2 <= n_layers <= MAX_LAYERS:
            raise ValueError("W and b must have the same length, 2..8")
        W3 = [w if w.dim() == 3 else w.unsqueeze(0) for w in W]
        b2 = [v if v.dim() == 2 else v.unsqueeze(0) for v in b]
        M = W3[0].shape[0]
        g = GenStack()
        g.n_layers = n_layers
        g.n_members = M
        g.leaky_slope = float(slope)
        g.width[0] = W3[0].shape[2]
        for l in range(n_layers):
            _check_tensor(W3[l], f"W[{l}]", torch.float32, (M, W3[l].shape[1], g.width[l]), self.device)
            g.width[l + 1] = W3[l].shape[1]
            _check_tensor(b2[l], f"b[{l}]", torch.float32, (M, g.width[l + 1]), self.device)
            g.W[l] = W3[l].data_ptr()
            g.b[l] = b2[l].data_ptr()
        return g, M

    def gen_forward(self, W: Sequence, b: Sequence, noise, slope: float = 0.2, out=None):
        """theta [M][k][out] = 1 + softplus(G_m(noise)) for every member m."""
        import torch
        self._enter()
        g, M = self._gen(W, b, slope)
        _check_tensor(noise, "noise", torch.float32, (noise.shape[0], g.width[0]), self.device)
        k = noise.shape[0]
        th = out if out is not None else torch.empty((M, k, g.width[g.n_layers]), dtype=torch.float32,
                                                     device=noise.device)
        _check_tensor(th, "out", torch.float32, (M, k, g.width[g.n_layers]), self.device)
        self._owned(th if out is None else None)
        self._check(self.lib.sagips_gen_forward(self.h, ctypes.byref(g), noise.data_ptr(), k, th.data_ptr()))
        return th

    def gen_backward(self, W: Sequence, b: Sequence, noise, dL_dtheta, slope: float = 0.2, dW=None, db=None):
        """Gradients (dW, db), shaped like W and b, of sum <dL/dtheta, theta> per member."""
        import torch
        self._enter()
        g, M = self._gen(W, b, slope)
        _check_tensor(noise, "noise", torch.float32, (noise.shape[0], g.width[0]), self.device)
        k = noise.shape[0]
        n_out = g.width[g.n_layers]
        if M > 1 or dL_dtheta.dim() == 3:
            _check_tensor(dL_dtheta, "dL_dtheta", torch.float32, (M, k, n_out), self.device)
        else:
            _check_tensor(dL_dtheta, "dL_dtheta", torch.float32, (k, n_out), self.device)
        new_dW, new_db = dW is None, db is None
        dW = dW if dW is not None else [torch.empty_like(w) for w in W]
        db = db if db is not None else [torch.empty_like(v) for v in b]
        self._owned(dW if new_dW else None, db if new_db else None)
        for l in range(g.n_layers):
            _check_tensor(dW[l], f"dW[{l}]", torch.float32, tuple(W[l].shape), self.device)
            _check_tensor(db[l], f"db[{l}]", torch.float32, tuple(b[l].shape), self.device)
        pw = (ctypes.c_void_p * MAX_LAYERS)(*[t.data_ptr() for t in dW])
        pb = (ctypes.c_void_p * MAX_LAYERS)(*[t.data_ptr() for t in db])
        self._check(self.lib.sagips_gen_backward(self.h, ctypes.byref(g), noise.data_ptr(), k,
                                                 dL_dtheta.data_ptr(), pw, pb))
        return dW, db

    def ensemble_response(self, W: Sequence, b: Sequence, noise, p_true=None, slope: float = 0.2) -> dict:
        """p_hat and sigma [out] averaged over the noise batch, and r_hat = (p_true - p_hat) / p_true."""
        import torch
        self._enter()
        g, M = self._gen(W, b, slope)
        _check_tensor(noise, "noise", torch.float32, (noise.shape[0], g.width[0]), self.device)
        n_out = g.width[g.n_layers]
        f32 = dict(dtype=torch.float32, device=noise.device)
        o = {"p_hat": torch.empty(n_out, **f32), "sigma": torch.empty(n_out, **f32), "r_hat": None}
        if p_true is not None:
            _check_tensor(p_true, "p_true", torch.float32, (n_out,), self.device)
            o["r_hat"] = torch.empty(n_out, **f32)
        self._owned(o["p_hat"], o["sigma"], o["r_hat"])
        self._check(self.lib.sagips_ensemble_response(self.h, ctypes.byref(g), noise.data_ptr(), noise.shape[0],
                                                      _ptr(p_true), o["p_hat"].data_ptr(), o["sigma"].data_ptr(),
                                                      _ptr(o["r_hat"])))
        return o

    # -- optimiser ------------------------------------------------------------------
    def adam_step(self, params: Sequence, grads: Sequence, m: Sequence, v: Sequence, step: int, lr: float,
                  beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8) -> None:
        """In-place Adam step on up to 16 fp32 tensors (m, v start at zero; step counts from 1)."""
        import torch
        self._enter()
        n = len(params)
        if not (n == len(grads) == len(m) == len(v)) or not 1 <= n <= MAX_TENSORS:
            raise ValueError("params, grads, m, v must have the same length, 1..16")
        ps = ParamSet()
        ps.n_tensors = n
        for i in range(n):
            for t, name in ((params[i], "param"), (grads[i], "grad"), (m[i], "m"), (v[i], "v")):
                _check_tensor(t, f"{name}[{i}]", torch.float32, tuple(params[i].shape), self.device)
            ps.param[i], ps.grad[i] = params[i].data_ptr(), grads[i].data_ptr()
            ps.m[i], ps.v[i] = m[i].data_ptr(), v[i].data_ptr()
            ps.size[i] = params[i].numel()
        self._check(self.lib.sagips_adam_step(self.h, ctypes.byref(ps), int(step), lr, beta1, beta2, eps))

    # -- 2. events -> discriminator -> BCE -> backward -------------------------------
    def disc_fwd_bwd(self, W: Sequence, b: Sequence, real_x, fake_x=None, fake_source: Optional[dict] = None,
                     precision: int = F32, features: int = FEAT_IDENTITY, slope: float = 0.2,
                     want_logits: bool = True, want_grads: bool = True, want_dx: bool = True,
                     want_dtheta: bool = True, outputs: Optional[dict] = None, no_alloc: bool = False) -> dict:
        """One discriminator step.  fake_source = dict(theta=, events_per_theta=, seed=[, counter_base=, stream=])
        samples the fake events inside the kernel and also returns dLg_dtheta.  With no_alloc the
        library takes its workspace from its fixed per-device scratch (sagips_disc_fwd_bwd_noalloc)
        instead of allocating; pass every output in `outputs` so that the binding allocates nothing
        either."""
        import torch
        self._enter()
        n_layers = len(W)
        if n_layers != len(b) or not 1 <= n_layers <= MAX_LAYERS:
            raise ValueError("W and b must have the same length, 1..8")
        widths = [W[0].shape[1]] + [w.shape[0] for w in W]
        mlp = Mlp()
        mlp.n_layers = n_layers
        for i, wd in enumerate(widths):
            mlp.width[i] = wd
        for l in range(n_layers):
            _check_tensor(W[l], f"W[{l}]", torch.float32, (widths[l + 1], widths[l]), self.device)
            _check_tensor(b[l], f"b[{l}]", torch.float32, (widths[l + 1],), self.device)
            mlp.W[l] = W[l].data_ptr()
            mlp.b[l] = b[l].data_ptr()
        mlp.leaky_slope = float(slope)
        mlp.precision = int(precision)
        mlp.features = int(features)
        dev = real_x.device
        _check_tensor(real_x, "real_x", torch.float32, device=self.device)
        src = None
        if fake_source is not None:
            fs = dict(fake_source)
            src = self.source(fs.pop("theta"), fs.pop("events_per_theta"), fs.pop("seed"), **fs)
            n_fake = src.n_theta * src.events_per_theta
            d = src.d
        elif fake_x is not None:
            _check_tensor(fake_x, "fake_x", torch.float32, device=self.device)
            n_fake = fake_x.shape[0]
            d = fake_x.shape[1]
        else:                       # no fake input: the library rejects the call
            n_fake, d = 0, widths[0]
        n_real = real_x.shape[0]
        d_in = widths[0] if features == FEAT_IDENTITY else 3
        if (fake_x is not None and d != d_in) or real_x.dim() != 2 or real_x.shape[1] != d_in:
            raise ValueError(f"events must be [n][{d_in}] for this network and feature map")
        o = dict(outputs or {})
        given = set(o)
        f32 = dict(dtype=torch.float32, device=dev)
        if want_logits:
            o.setdefault("logits_fake", torch.empty(max(n_fake, 1), **f32))
            o.setdefault("logits_real", torch.empty(n_real, **f32))
        o.setdefault("loss_d", torch.empty(1, **f32))
        o.setdefault("loss_g", torch.empty(1, **f32))
        if want_grads:
            o.setdefault("dW", [torch.empty_like(w) for w in W])
            o.setdefault("db", [torch.empty_like(v) for v in b])
        if want_dx:
            o.setdefault("dLg_dx", torch.empty((max(n_fake, 1), d), **f32))
        if want_dtheta and src is not None:
            o.setdefault("dLg_dtheta", torch.empty((src.n_theta, 2 * src.d), **f32))
        self._owned(*[v for k, v in o.items() if k not in given])
        out = DiscOut()
        for k in ("logits_fake", "logits_real", "loss_d", "loss_g", "dLg_dx", "dLg_dtheta"):
            if o.get(k) is not None:
                _check_tensor(o[k], k, torch.float32, device=self.device)
                setattr(out, k, o[k].data_ptr())
        if "dW" in o:
            for l in range(n_layers):
                out.dW[l] = o["dW"][l].data_ptr()
                out.db[l] = o["db"][l].data_ptr()
        fn = self.lib.sagips_disc_fwd_bwd_noalloc if no_alloc else self.lib.sagips_disc_fwd_bwd
        st = fn(self.h, ctypes.byref(mlp), _ptr(fake_x),
                                          ctypes.byref(src) if src is not None else None, n_fake,
                                          real_x.data_ptr(), n_real, ctypes.byref(out))
        self._check(st)
        return o

    # -- 3. dL/dx -> pathwise dx/dtheta -> per-parameter reduction ---------------------------
    def param_grad(self, theta, events_per_theta: int, seed: int, dL_dx=None, counter_base: int = 0,
                   stream: int = 0, out=None, loss_out=None, want_loss: bool = True):
        """dL/dtheta [n_theta][2d]; with dL_dx None the quadratic critic is used and its loss returned too."""
        import torch
        self._enter()
        src = self.source(theta, events_per_theta, seed, counter_base, stream)
        g = out if out is not None else torch.empty((src.n_theta, 2 * src.d), dtype=torch.float32, device=theta.device)
        _check_tensor(g, "out", torch.float32, (src.n_theta, 2 * src.d), self.device)
        loss = None
        if dL_dx is None:
            critic = CRITIC_QUADRATIC
            if want_loss:
                loss = loss_out if loss_out is not None else torch.empty(1, dtype=torch.float32, device=theta.device)
        else:
            critic = CRITIC_BUFFER
            _check_tensor(dL_dx, "dL_dx", torch.float32, (src.n_theta * src.events_per_theta, src.d), self.device)
        self._owned(g if out is None else None, loss if loss_out is None else None)
        self._check(self.lib.sagips_param_grad(self.h, ctypes.byref(src), critic, _ptr(dL_dx), g.data_ptr(),
                                               _ptr(loss)))
        return (g, loss) if critic == CRITIC_QUADRATIC else g


_default: Dict[int, Context] = {}


def default_context(device: int = 0) -> Context:
    if device not in _default:
        _default[device] = Context(device)
    return _default[device]


def sample_events(theta, events_per_theta: int, seed: int, **kw):
    return default_context(theta.device.index).sample_events(theta, events_per_theta, seed, **kw)


def disc_fwd_bwd(W, b, real_x, **kw):
    return default_context(real_x.device.index).disc_fwd_bwd(W, b, real_x, **kw)


def param_grad(theta, events_per_theta: int, seed: int, **kw):
    return default_context(theta.device.index).param_grad(theta, events_per_theta, seed, **kw)
