"""ctypes binding of librn18.so: the C ABI of include/rn18.h and
include/rn18_ops.h under the same names.

Argument marshalling only: torch tensors provide device memory
(``data_ptr()``) and the HIP stream (``torch.cuda.current_stream()``); every
step of the computation runs in the library's HIP kernels. If the library is
not built, importing a function raises instead of falling back to anything.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librn18.so")

RN18_OK, RN18_EINVAL, RN18_ELABEL, RN18_ENOMEM, RN18_EHIP, RN18_ENONFINITE = 0, -1, -2, -3, -4, -5
RN18_TINY, RN18_CIFAR, RN18_IMAGENET = 0, 1, 2
RN18_FP32, RN18_BF16, RN18_FP16 = 0, 1, 2
ARCH_IDS = {"tiny": RN18_TINY, "cifar": RN18_CIFAR, "imagenet": RN18_IMAGENET}
PREC_IDS = {"fp32": RN18_FP32, "bf16": RN18_BF16, "fp16": RN18_FP16}

# Every symbol the headers declare (checked by the CPU test suite).
EXPORTED = [
    "rn18_state_floats", "rn18_init", "rn18_workspace_bytes", "rn18_set_workspace", "rn18_train_step",
    "rn18_eval_logits", "ps_dual_merge", "ps_worker_delta", "rn18_sync_status", "rn18_get_momentum",
    "rn18_set_momentum", "rn18_set_dropout", "rn18_set_loss_scale", "rn18_get_loss_scale", "rn18_destroy",
    "rn18_last_error", "rn18_profile_enable",
    "rn18_profile_read",
    "rn18op_conv2d_fwd", "rn18op_conv2d_dgrad", "rn18op_conv2d_wgrad_workspace", "rn18op_conv2d_wgrad",
    "rn18op_maxpool_fwd", "rn18op_maxpool_bwd", "rn18_debug_set", "rn18_debug_copy",
    "rn18_debug_capture", "rn18op_round_bf16", "rn18op_conv2d_wgrad_noalloc_limit", "rn18op_conv2d_wgrad_noalloc",
]


class Rn18Error(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("rn18 error %d: %s" % (code, msg))
        self.code = code


class rn18_prof_rec(ctypes.Structure):
    _fields_ = [("cls", ctypes.c_int), ("layer", ctypes.c_int), ("tile", ctypes.c_int), ("pad_", ctypes.c_int),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double), ("ms", ctypes.c_double),
                ("kernel", ctypes.c_char * 104)]


K_NAMES = ["conv_fwd", "conv_dgrad", "conv_wgrad", "wgrad_reduce", "bn_stats", "bn_apply", "bn_bwd_reduce",
           "bn_bwd_apply", "maxpool", "avgpool", "head", "sgd", "prep"]


class rn18_config(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_int), ("num_classes", ctypes.c_int), ("prec", ctypes.c_int),
                ("momentum", ctypes.c_float), ("weight_decay", ctypes.c_float), ("bn_eps", ctypes.c_float),
                ("bn_momentum", ctypes.c_float)]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int
_Z = ctypes.c_size_t
_F = ctypes.c_float


def lib():
    """Load the HIP library; raise if it is not built (no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("librn18.so is not built (run __graft_entry__.build()); there is no fallback path")
    L = ctypes.CDLL(LIB_PATH)
    sig = {
        "rn18_state_floats": (_Z, [ctypes.POINTER(rn18_config), ctypes.POINTER(_Z)]),
        "rn18_init": (_I, [ctypes.POINTER(rn18_config), ctypes.c_uint64, _P, _P, ctypes.POINTER(_P)]),
        "rn18_workspace_bytes": (_Z, [_P, _I, _I, _I]),
        "rn18_set_workspace": (_I, [_P, _P, _Z]),
        "rn18_train_step": (_I, [_P, _P, _P, _P, _I, _I, _I, _F, _P]),
        "rn18_eval_logits": (_I, [_P, _P, _P, _I, _I, _I, _P]),
        "ps_dual_merge": (_I, [_P, _P, _P, _Z, _F, _P]),
        "ps_worker_delta": (_I, [_P, _P, _P, _Z, _P]),
        "rn18_sync_status": (_I, [_P]),
        "rn18_get_momentum": (_I, [_P, _P]),
        "rn18_set_momentum": (_I, [_P, _P]),
        "rn18_set_dropout": (_I, [_P, _F, ctypes.c_uint64, ctypes.c_uint64]),
        "rn18_set_loss_scale": (_I, [_P, _F, ctypes.c_uint]),
        "rn18_get_loss_scale": (_I, [_P, ctypes.POINTER(_F), ctypes.POINTER(ctypes.c_uint64)]),
        "rn18_destroy": (None, [_P]),
        "rn18_last_error": (ctypes.c_char_p, []),
        "rn18op_conv2d_fwd": (_I, [_I, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P]),
        "rn18op_conv2d_dgrad": (_I, [_I, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P]),
        "rn18op_conv2d_wgrad_workspace": (_Z, [_I, _I, _I, _I, _I, _I, _I, _I, _I]),
        "rn18op_conv2d_wgrad": (_I, [_I, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P, _Z, _P]),
        "rn18op_conv2d_wgrad_noalloc_limit": (_Z, []),
        "rn18op_conv2d_wgrad_noalloc": (_I, [_I, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _I, _P]),
        "rn18op_maxpool_fwd": (_I, [_I, _P, _P, _P, _I, _I, _I, _I, _P]),
        "rn18op_maxpool_bwd": (_I, [_I, _P, _P, _P, _I, _I, _I, _I, _P]),
        "rn18op_round_bf16": (_I, [_P, _P, _Z, _P]),
        "rn18_debug_set": (_I, [_P, _I, ctypes.c_long]),
        "rn18_profile_enable": (_I, [_P, _I]),
        "rn18_profile_read": (_I, [_P, ctypes.POINTER(rn18_prof_rec), _I, ctypes.POINTER(_I)]),
        "rn18_debug_copy": (_I, [_P, _I, _I, _I, _I, _I, _P, _Z]),
        "rn18_debug_capture": (_I, [_P, _I, _I, _P, _Z]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(code):
    if code != RN18_OK:
        raise Rn18Error(code, lib().rn18_last_error().decode())
    return code


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def make_config(arch, num_classes, prec="fp32", momentum=0.9, weight_decay=5e-4, bn_eps=1e-5, bn_momentum=0.1):
    return rn18_config(ARCH_IDS[arch] if isinstance(arch, str) else arch, num_classes,
                       PREC_IDS[prec] if isinstance(prec, str) else prec, momentum, weight_decay, bn_eps,
                       bn_momentum)


# ------------------------------------------------------------------ C ABI, same names
def rn18_state_floats(cfg):
    p = _Z(0)
    total = lib().rn18_state_floats(ctypes.byref(cfg), ctypes.byref(p))
    if total == 0:
        raise Rn18Error(RN18_EINVAL, "invalid config")
    return total, p.value


def rn18_init(cfg, seed, state_out=None, stream=None):
    h = _P()
    _check(lib().rn18_init(ctypes.byref(cfg), ctypes.c_uint64(seed), _stream(stream), _ptr(state_out), ctypes.byref(h)))
    return h


def rn18_workspace_bytes(ctx, N, H, W):
    return lib().rn18_workspace_bytes(ctx, N, H, W)


def rn18_set_workspace(ctx, ws):
    _check(lib().rn18_set_workspace(ctx, _ptr(ws), ws.numel() * ws.element_size()))


def rn18_train_step(ctx, state, images, labels, N, H, W, lr, loss=None):
    return _check(lib().rn18_train_step(ctx, _ptr(state), _ptr(images), _ptr(labels), N, H, W, lr, _ptr(loss)))


def rn18_eval_logits(ctx, state, images, N, H, W, logits):
    return _check(lib().rn18_eval_logits(ctx, _ptr(state), _ptr(images), N, H, W, _ptr(logits)))


def ps_dual_merge(state, g_small, g_large, n, factor, stream=None):
    return _check(lib().ps_dual_merge(_ptr(state), _ptr(g_small), _ptr(g_large), n, factor, _stream(stream)))


def ps_worker_delta(pulled, local, delta, n, stream=None):
    return _check(lib().ps_worker_delta(_ptr(pulled), _ptr(local), _ptr(delta), n, _stream(stream)))


def rn18_sync_status(ctx):
    return lib().rn18_sync_status(ctx)


def rn18_set_dropout(ctx, p, seed, step):
    return _check(lib().rn18_set_dropout(ctx, ctypes.c_float(p), ctypes.c_uint64(seed), ctypes.c_uint64(step)))


def rn18_set_loss_scale(ctx, scale, growth_interval=2000):
    return _check(lib().rn18_set_loss_scale(ctx, ctypes.c_float(scale), ctypes.c_uint(growth_interval)))


def rn18_get_loss_scale(ctx):
    """(scale, skipped steps) of an fp16 context."""
    sc, sk = _F(0.0), ctypes.c_uint64(0)
    _check(lib().rn18_get_loss_scale(ctx, ctypes.byref(sc), ctypes.byref(sk)))
    return sc.value, sk.value


def rn18_get_momentum(ctx, dst):
    return _check(lib().rn18_get_momentum(ctx, _ptr(dst)))


def rn18_set_momentum(ctx, src):
    return _check(lib().rn18_set_momentum(ctx, _ptr(src)))


def rn18_destroy(ctx):
    lib().rn18_destroy(ctx)


def rn18_profile_enable(ctx, on):
    return _check(lib().rn18_profile_enable(ctx, 1 if on else 0))


def rn18_profile_read(ctx, max_records=4096):
    """Profile records (kernel class, layer, tile, kernel name, flops, bytes, ms) in launch order."""
    buf = (rn18_prof_rec * max_records)()
    n = _I(0)
    _check(lib().rn18_profile_read(ctx, buf, max_records, ctypes.byref(n)))
    return [dict(cls=K_NAMES[r.cls], layer=r.layer, tile=r.tile, kernel=r.kernel.decode(), flops=r.flops,
                 bytes=r.bytes, ms=r.ms)
            for r in buf[:min(n.value, max_records)]]


def rn18_last_error():
    return lib().rn18_last_error().decode()


def rn18op_conv2d_fwd(prec, x, w, y, N, H, W, Cin, Cout, k, s, p, stream=None):
    return _check(lib().rn18op_conv2d_fwd(prec, _ptr(x), _ptr(w), _ptr(y), N, H, W, Cin, Cout, k, s, p, _stream(stream)))


def rn18op_conv2d_dgrad(prec, dy, w, dx, N, H, W, Cin, Cout, k, s, p, stream=None):
    return _check(lib().rn18op_conv2d_dgrad(prec, _ptr(dy), _ptr(w), _ptr(dx), N, H, W, Cin, Cout, k, s, p,
                                            _stream(stream)))


def rn18op_conv2d_wgrad_workspace(prec, N, H, W, Cin, Cout, k, s, p):
    return lib().rn18op_conv2d_wgrad_workspace(prec, N, H, W, Cin, Cout, k, s, p)


def rn18op_conv2d_wgrad(prec, dy, x, dw, N, H, W, Cin, cin_real, Cout, k, s, p, ws, stream=None):
    return _check(lib().rn18op_conv2d_wgrad(prec, _ptr(dy), _ptr(x), _ptr(dw), N, H, W, Cin, cin_real, Cout, k, s, p,
                                            _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def rn18op_conv2d_wgrad_noalloc_limit():
    return lib().rn18op_conv2d_wgrad_noalloc_limit()


def rn18op_conv2d_wgrad_noalloc(prec, dy, x, dw, N, H, W, Cin, cin_real, Cout, k, s, p, stream=None):
    return _check(lib().rn18op_conv2d_wgrad_noalloc(prec, _ptr(dy), _ptr(x), _ptr(dw), N, H, W, Cin, cin_real, Cout,
                                                    k, s, p, _stream(stream)))


def rn18op_maxpool_fwd(prec, x, y, arg, N, H, W, C, stream=None):
    return _check(lib().rn18op_maxpool_fwd(prec, _ptr(x), _ptr(y), _ptr(arg), N, H, W, C, _stream(stream)))


def rn18op_maxpool_bwd(prec, dy, arg, dx, N, H, W, C, stream=None):
    return _check(lib().rn18op_maxpool_bwd(prec, _ptr(dy), _ptr(arg), _ptr(dx), N, H, W, C, _stream(stream)))


def rn18op_round_bf16(x, y, n, stream=None):
    return _check(lib().rn18op_round_bf16(_ptr(x), _ptr(y), n, _stream(stream)))


DBG = dict(y=0, z1=1, out=2, gA=3, gB=4, gz=5, gy=6, gyd=7, grad=8, wf=9, wd=10, mean=11, rstd=12, zstem=13,
           parg=14)


RN18_DBG_STOP_BLOCKS, RN18_DBG_GATHER_CONFIG, RN18_DBG_WGRAD_CONFIG, RN18_DBG_CONV_CHUNK, RN18_DBG_SERIAL = 0, 1, 2, 3, 4
RN18_DBG_GATHER_SPLIT = 5


def rn18_debug_set(ctx, key, value):
    return _check(lib().rn18_debug_set(ctx, key, value))


CAP = dict(dy=0, dz1=1, dx=3, da_avg=4, da_pool=5)


def rn18_debug_capture(ctx, kind, index, dst):
    if dst is None:
        return _check(lib().rn18_debug_capture(ctx, 0, 0, None, 0))
    return _check(lib().rn18_debug_capture(ctx, CAP[kind] if isinstance(kind, str) else kind, index, _ptr(dst),
                                           dst.numel() * dst.element_size()))


def rn18_debug_copy(ctx, N, H, W, which, index, dst):
    return _check(lib().rn18_debug_copy(ctx, N, H, W, DBG[which] if isinstance(which, str) else which, index,
                                        _ptr(dst), dst.numel() * dst.element_size()))


# ------------------------------------------------------------------ thin owner of a context
class Worker:
    """One training context (a parameter-server worker): the library context
    plus a torch-allocated device workspace sized for the largest shape seen.
    Holds no state of its own beyond memory ownership.

    The context is bound to `stream` (torch's current stream at construction
    by default); the workspace is allocated on that stream, so torch's
    allocator hands a replaced workspace to later allocations only in that
    stream's order, after every step that used it."""

    def __init__(self, arch, num_classes, prec="fp32", seed=0, state=None, stream=None, **hyper):
        import torch
        self.cfg = make_config(arch, num_classes, prec, **hyper)
        self.n_state, self.n_trainable = rn18_state_floats(self.cfg)
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.ctx = rn18_init(self.cfg, seed, state, stream=self.stream)
        self.ws = None
        self.torch = torch

    def _ensure(self, N, H, W):
        need = rn18_workspace_bytes(self.ctx, N, H, W)
        if need == 0:
            raise Rn18Error(RN18_EINVAL, rn18_last_error())
        if self.ws is None or self.ws.numel() < need:
            with self.torch.cuda.stream(self.stream):
                ws = self.torch.empty(need, dtype=self.torch.uint8, device="cuda")
            rn18_set_workspace(self.ctx, ws)
            self.ws = ws

    def train_step(self, state, images, labels, lr, loss=None):
        N, _, H, W = images.shape
        self._ensure(N, H, W)
        return rn18_train_step(self.ctx, state, images, labels, N, H, W, lr, loss)

    def eval_logits(self, state, images, logits):
        N, _, H, W = images.shape
        self._ensure(N, H, W)
        return rn18_eval_logits(self.ctx, state, images, N, H, W, logits)

    def sync_status(self):
        return rn18_sync_status(self.ctx)

    def close(self):
        if self.ctx:
            rn18_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
