"""ctypes binding of libhs (the C ABI in include/hs.h).

Argument marshalling only: every function forwards to the library of the
same name.  Device pointers are passed as integers (e.g. a torch tensor's
data_ptr()), streams as the integer handle of a hipStream_t (0 = default).
The library must have been built (``python -m paper_2110_08941_amd.build``);
importing this module without it raises immediately -- there is no fallback.
"""
import ctypes
import os
import re

# The process must hold ONE HIP runtime.  PyTorch ships its own copy of
# libamdhip64 (same soname as the system one); loading torch first makes the
# library's dependency resolve to that copy instead of mapping a second one.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhs.so")

HS_OK, HS_ERR_INVALID, HS_ERR_HIP, HS_ERR_OOM, HS_ERR_UNSUPPORTED = 0, -1, -2, -3, -4
ARCH = {"mlp": 0, "small_cnn": 1, "resnet18": 2, "vgg16": 3, "resnet50": 4}
DTYPE = {"fp32": 0, "bf16": 1}
KIND = {0: "conv_w", 1: "lin_w", 2: "bias", 3: "bn_gamma", 4: "bn_beta"}


class HSError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("libhs status %d: %s" % (status, msg))
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libhs.so not built at %s (python -m paper_2110_08941_amd.build)" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, D, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_float
    PP = ctypes.POINTER(ctypes.c_void_p)
    PI32 = ctypes.POINTER(ctypes.c_int32)
    PI64 = ctypes.POINTER(ctypes.c_int64)
    PD = ctypes.POINTER(ctypes.c_double)
    sigs = {
        "hs_model_create": (I32, [I32, I32, PP]),
        "hs_model_destroy": (I32, [P]),
        "hs_num_params": (I64, [P]),
        "hs_num_true_params": (I64, [P]),
        "hs_num_param_tensors": (I32, [P]),
        "hs_param_tensor": (I32, [P, I32, PI64, PI64, PI32, PI64, PI32,
                                  ctypes.POINTER(ctypes.c_char_p)]),
        "hs_input_numel": (I64, [P]),
        "hs_forward_macs": (I64, [P]),
        "hs_workspace_create": (I32, [P, I32, PP]),
        "hs_workspace_destroy": (I32, [P]),
        "hs_workspace_bytes": (I64, [P]),
        "hs_workspace_set_streams": (I32, [P, I32]),
        "hs_worker_grad": (I32, [P, P, P, P, P, P, I32, P, P, P]),
        "hs_workers_grad": (I32, [P, P, P, P, P, P, PI32, I32, PP, P, P]),
        "hs_workers_grad_static": (I32, [P, P, P, P, P, PI32, I32, PP, P, P]),
        "hs_workers_grad_wavg": (I32, [P, P, P, P, P, P, PI32, I32, P, P, P]),
        "hs_workers_grad_static_bytes": (I64, [P, I32]),
        "hs_weighted_average": (I32, [PP, PI32, I32, I64, P, P]),
        "hs_sgd_step": (I32, [P, P, P, I64, F, F, F, P, P]),
        "hs_wavg_sgd": (I32, [PP, PI32, I32, P, P, I64, F, F, F, P, P]),
        "hs_params_to_bf16": (I32, [P, P, I64, P]),
        "hs_estimate_cp": (I32, [PI32, PD, I32, PD]),
        "hs_repartition": (I32, [PD, I32, I32, PI32]),
        "hs_partitioner_create": (I32, [I32, I32, I32, PP]),
        "hs_partitioner_destroy": (I32, [P]),
        "hs_partitioner_partition": (I32, [P, PI32]),
        "hs_partitioner_set_partition": (I32, [P, PI32]),
        "hs_partitioner_observe": (I32, [P, PI32, PD, PD, PI32, PD]),
        "hs_partitioner_set_estimator": (I32, [P, I32, ctypes.c_double, I32]),
        "hs_layer_gemm": (I32, [I32, I32, I32, I32, I32, I32, I32, I32, I32, I32, P, P, P, P, I32,
                                I32, P, I64, P]),
        "hs_probe_enable": (I32, [P, I32, I32, I32, I32]),
        "hs_probe_read": (I32, [P, PD, PI64, PD]),
        "hs_probe_mfma_loop": (I32, [I32, I32, P, P]),
        "hs_probe_copy": (I32, [P, P, I64, P]),
        "hs_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    try:
        maps = open("/proc/self/maps").read()
    except OSError:
        maps = ""
    runtimes = set(re.findall(r"(/\S*libamdhip64[^/\s]*)", maps))
    if len(runtimes) > 1:
        raise ImportError("two HIP runtimes are mapped in this process: %s" % sorted(runtimes))
    return lib


_lib = _load()
EXPORTED = (
    "hs_model_create", "hs_model_destroy", "hs_num_params", "hs_num_true_params",
    "hs_num_param_tensors", "hs_param_tensor", "hs_input_numel", "hs_forward_macs",
    "hs_workspace_create", "hs_workspace_destroy", "hs_workspace_bytes",
    "hs_workspace_set_streams", "hs_worker_grad",
    "hs_workers_grad", "hs_workers_grad_static", "hs_workers_grad_static_bytes",
    "hs_workers_grad_wavg",
    "hs_weighted_average", "hs_sgd_step", "hs_wavg_sgd", "hs_params_to_bf16", "hs_estimate_cp",
    "hs_repartition", "hs_partitioner_create", "hs_partitioner_destroy",
    "hs_partitioner_partition", "hs_partitioner_set_partition", "hs_partitioner_observe",
    "hs_partitioner_set_estimator",
    "hs_layer_gemm", "hs_probe_enable", "hs_probe_read", "hs_probe_mfma_loop", "hs_probe_copy",
    "hs_last_error")


def lib():
    return _lib


def last_error():
    return _lib.hs_last_error().decode()


def _check(st):
    if st != HS_OK:
        raise HSError(st, last_error())


def _ptrs(seq):
    return (ctypes.c_void_p * len(seq))(*[int(p) for p in seq])


def _i32(seq):
    return (ctypes.c_int32 * len(seq))(*[int(v) for v in seq])


def _f64(seq):
    return (ctypes.c_double * len(seq))(*[float(v) for v in seq])


# ---------------------------------------------------------------- models --
def model_create(arch, dtype):
    h = ctypes.c_void_p()
    _check(_lib.hs_model_create(ARCH.get(arch, arch), DTYPE.get(dtype, dtype), ctypes.byref(h)))
    return h.value


def model_destroy(model):
    _check(_lib.hs_model_destroy(model))


def num_params(model):
    return int(_lib.hs_num_params(model))


def num_true_params(model):
    return int(_lib.hs_num_true_params(model))


def input_numel(model):
    return int(_lib.hs_input_numel(model))


def forward_macs(model):
    return int(_lib.hs_forward_macs(model))


def param_table(model):
    """[(name, kind, shape, offset)] in layout order."""
    out = []
    for i in range(_lib.hs_num_param_tensors(model)):
        off, numel, ndim, kind = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
        dims = (ctypes.c_int64 * 4)()
        name = ctypes.c_char_p()
        _check(_lib.hs_param_tensor(model, i, ctypes.byref(off), ctypes.byref(numel),
                                    ctypes.byref(ndim), dims, ctypes.byref(kind), ctypes.byref(name)))
        out.append((name.value.decode(), KIND[kind.value], tuple(dims[:ndim.value]), off.value))
    return out


def workspace_create(model, max_n):
    h = ctypes.c_void_p()
    _check(_lib.hs_workspace_create(model, int(max_n), ctypes.byref(h)))
    return h.value


def workspace_destroy(ws):
    _check(_lib.hs_workspace_destroy(ws))


def workspace_bytes(ws):
    return int(_lib.hs_workspace_bytes(ws))


def workspace_set_streams(ws, streams):
    _check(_lib.hs_workspace_set_streams(ws, int(streams)))


# ---------------------------------------------------------------- step --
def worker_grad(model, ws, theta, theta_bf16, x_m, y_m, n_m, g_m, loss_m=0, stream=0):
    _check(_lib.hs_worker_grad(model, ws, theta, theta_bf16 or None, x_m, y_m, int(n_m), g_m,
                               loss_m or None, stream or None))


def workers_grad(model, ws, theta, theta_bf16, x, y, n, g, loss=0, stream=0):
    """All len(n) workers' gradients in one pass; g: device pointers, one per
    worker; loss: device fp32 [M] or 0."""
    if len(g) != len(n):
        raise ValueError("workers_grad: one gradient buffer per worker")
    _check(_lib.hs_workers_grad(model, ws, theta, theta_bf16 or None, x, y, _i32(n), len(n),
                                _ptrs(g), loss or None, stream or None))


def workers_grad_wavg(model, ws, theta, theta_bf16, x, y, n, g_bar, loss=0, stream=0):
    """The partition-weighted gradient sum_m (n_m / sum n) g_m of all workers in
    one pass, into g_bar (device pointer)."""
    _check(_lib.hs_workers_grad_wavg(model, ws, theta, theta_bf16 or None, x, y, _i32(n), len(n),
                                     g_bar, loss or None, stream or None))


def workers_grad_static(model, theta, theta_bf16, x, y, n, g, loss=0, stream=0):
    """workers_grad without a workspace (the library's static device buffer)."""
    if len(g) != len(n):
        raise ValueError("workers_grad_static: one gradient buffer per worker")
    _check(_lib.hs_workers_grad_static(model, theta, theta_bf16 or None, x, y, _i32(n), len(n),
                                       _ptrs(g), loss or None, stream or None))


def workers_grad_static_bytes(model, total_n):
    return int(_lib.hs_workers_grad_static_bytes(model, int(total_n)))


def weighted_average(g, n, P, g_out, stream=0):
    _check(_lib.hs_weighted_average(_ptrs(g), _i32(n), len(g), int(P), g_out, stream or None))


def sgd_step(theta, g, mom, P, lr, mu, wd, theta_bf16=0, stream=0):
    _check(_lib.hs_sgd_step(theta, g, mom or None, int(P), lr, mu, wd, theta_bf16 or None,
                            stream or None))


def wavg_sgd(g, n, theta, mom, P, lr, mu, wd, theta_bf16=0, stream=0):
    _check(_lib.hs_wavg_sgd(_ptrs(g), _i32(n), len(g), theta, mom or None, int(P), lr, mu, wd,
                            theta_bf16 or None, stream or None))


def params_to_bf16(theta, theta_bf16, P, stream=0):
    _check(_lib.hs_params_to_bf16(theta, theta_bf16, int(P), stream or None))


def probe_enable(ws, mode, bm, bn, capacity=4096):
    _check(_lib.hs_probe_enable(ws, int(mode), int(bm), int(bn), int(capacity)))


def probe_read(ws):
    """(total_ms, launches, flops) of the probed launches since the last read."""
    t, n, f = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
    _check(_lib.hs_probe_read(ws, ctypes.byref(t), ctypes.byref(n), ctypes.byref(f)))
    return t.value, n.value, f.value


def probe_mfma_loop(blocks, iters, out, stream=0):
    """Asynchronous launch of the MFMA loop (hs_probe_mfma_loop); out: device
    pointer to blocks x 512 floats.  FLOPs: blocks x 8 x iters x 8 x 32768."""
    _check(_lib.hs_probe_mfma_loop(int(blocks), int(iters), out, stream or None))


def probe_copy(src, dst, nbytes, stream=0):
    """Asynchronous plain device copy (hs_probe_copy) of nbytes."""
    _check(_lib.hs_probe_copy(src, dst, int(nbytes), stream or None))


def layer_gemm(mode, dtype, n, H, W, C, K, R, stride, pad, a, b, out, bias=0, relu=False,
               out_f32=False, scratch=0, scratch_floats=0, stream=0):
    _check(_lib.hs_layer_gemm(int(mode), DTYPE.get(dtype, dtype), n, H, W, C, K, R, stride, pad,
                              a, b, out, bias or None, int(bool(relu)), int(bool(out_f32)),
                              scratch or None, int(scratch_floats), stream or None))


# ------------------------------------------------- compute power, partition --
def estimate_cp(n, mean_time):
    out = (ctypes.c_double * len(n))()
    _check(_lib.hs_estimate_cp(_i32(n), _f64(mean_time), len(n), out))
    return list(out)


def repartition(throughput, N):
    out = (ctypes.c_int32 * len(throughput))()
    _check(_lib.hs_repartition(_f64(throughput), len(throughput), int(N), out))
    return list(out)


class Partitioner:
    """Dynamic Partitioning state (hs_partitioner_*)."""

    def __init__(self, M, N, window):
        h = ctypes.c_void_p()
        _check(_lib.hs_partitioner_create(int(M), int(N), int(window), ctypes.byref(h)))
        self.h, self.M = h.value, int(M)

    def partition(self):
        out = (ctypes.c_int32 * self.M)()
        _check(_lib.hs_partitioner_partition(self.h, out))
        return list(out)

    def set_partition(self, n):
        _check(_lib.hs_partitioner_set_partition(self.h, _i32(n)))

    def set_estimator(self, kind, alpha=1.0, history=1):
        """Compute-power estimator across windows: "window" (Eq. (2) on the
        last window), "ema" (factor alpha) or "history" (mean of the last
        `history` windows' estimates); see hs_partitioner_set_estimator."""
        k = {"window": 0, "ema": 1, "history": 2}[kind]
        _check(_lib.hs_partitioner_set_estimator(self.h, k, float(alpha), int(history)))

    def observe(self, n_used, tau, speed):
        """Reports one step run with partition n_used; returns the CP vector if
        this step closed a window, else None."""
        rep = ctypes.c_int32()
        cp = (ctypes.c_double * self.M)()
        _check(_lib.hs_partitioner_observe(self.h, _i32(n_used), _f64(tau), _f64(speed),
                                           ctypes.byref(rep), cp))
        return list(cp) if rep.value else None

    def close(self):
        if self.h:
            _lib.hs_partitioner_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
