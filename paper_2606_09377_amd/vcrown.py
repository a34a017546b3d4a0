"""ctypes binding of libvcrown (include/vcrown.h).

Argument marshalling only: tensors are torch CUDA tensors (PyTorch provides device memory
and streams); every step of the bound computation runs in the library's HIP kernels.
There is no fallback: if the library is not built, or no GPU is present, calls fail.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "lib", "libvcrown.so")
ABI_VERSION = 3   # VCR_ABI_VERSION of include/vcrown.h this binding is written for
HEADER = os.path.join(os.path.dirname(HERE), "include", "vcrown.h")

VCR_OK, VCR_ERR_ARG, VCR_ERR_SHAPE, VCR_ERR_STATE, VCR_ERR_OOM, VCR_ERR_DEVICE, VCR_ERR_UNSUPPORTED = range(7)
STATUS_NAMES = ["OK", "ERR_ARG", "ERR_SHAPE", "ERR_STATE", "ERR_OOM", "ERR_DEVICE", "ERR_UNSUPPORTED"]
OPS = {"dense": 0, "conv2d": 1, "relu": 2, "add": 3, "flatten": 4}
(OPT_CLIP_ENABLE, OPT_CLIP_LO, OPT_CLIP_HI, OPT_INTERSECT_IBP, OPT_WORKSPACE_CAP_BYTES, OPT_SYNC_CHECK,
 OPT_TIME_GEMM, OPT_GRAPH, OPT_CHECK_FINITE, OPT_LAMBDA_RULE) = range(1, 11)
# values of OPT_LAMBDA_RULE (the lower slope of unstable ReLU neurons)
LAMBDA_RULES = {"adaptive": 0, "zero": 1, "one": 2, "same_slope": 3}
MAX_SPLITS = 64   # VCR_MAX_SPLITS


class VcrNode(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("in0", ctypes.c_int32), ("in1", ctypes.c_int32),
                ("out_features", ctypes.c_int32), ("out_ch", ctypes.c_int32), ("kh", ctypes.c_int32),
                ("kw", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("W", ctypes.c_void_p), ("b", ctypes.c_void_p)]


class VcrSplits(ctypes.Structure):
    _fields_ = [("n_domains", ctypes.c_int32), ("per_domain", ctypes.c_int32),
                ("relu_id", ctypes.c_void_p), ("neuron", ctypes.c_void_p), ("sign", ctypes.c_void_p)]


class VcrStats(ctypes.Structure):
    _fields_ = [("ms_last_call", ctypes.c_double), ("gemm_flops_last_call", ctypes.c_uint64),
                ("peak_workspace_bytes", ctypes.c_uint64), ("workspace_bytes", ctypes.c_uint64),
                ("n_chunks_last_call", ctypes.c_int32), ("invalid_domains", ctypes.c_int32),
                ("n_relu", ctypes.c_int32), ("unstable", ctypes.c_int32 * 64),
                ("timed_gemm_launches", ctypes.c_uint64), ("timed_gemm_ms", ctypes.c_double),
                ("timed_gemm_flops", ctypes.c_uint64), ("timed_conv_launches", ctypes.c_uint64),
                ("timed_conv_ms", ctypes.c_double), ("timed_conv_flops", ctypes.c_uint64),
                ("net_bytes", ctypes.c_uint64), ("timed_small_launches", ctypes.c_uint64),
                ("timed_small_ms", ctypes.c_double), ("timed_small_flops", ctypes.c_uint64),
                ("timed_mid_launches", ctypes.c_uint64), ("timed_mid_ms", ctypes.c_double),
                ("timed_mid_flops", ctypes.c_uint64)]


class VcrAlphaOpts(ctypes.Structure):
    _fields_ = [("iters", ctypes.c_int32), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("adam_eps", ctypes.c_float), ("alpha_init", ctypes.c_void_p),
                ("alpha_out", ctypes.c_void_p), ("grad_out", ctypes.c_void_p), ("lb_hist", ctypes.c_void_p),
                ("ub_hist", ctypes.c_void_p)]


class VcrBetaOpts(ctypes.Structure):
    _fields_ = [("iters", ctypes.c_int32), ("lr_alpha", ctypes.c_float), ("lr_beta", ctypes.c_float),
                ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("adam_eps", ctypes.c_float),
                ("lb_hist", ctypes.c_void_p), ("ub_hist", ctypes.c_void_p)]


class VcrBabOpts(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("max_rounds", ctypes.c_int32), ("bound", VcrBetaOpts),
                ("order_relu", ctypes.c_void_p), ("order_neuron", ctypes.c_void_p), ("order_len", ctypes.c_int32)]


class VcrBabResult(ctypes.Structure):
    _fields_ = [("verified", ctypes.c_int32), ("rounds", ctypes.c_int32), ("evaluated", ctypes.c_int64),
                ("remaining", ctypes.c_int64), ("root_min_lb", ctypes.c_float), ("worst_lb", ctypes.c_float)]


class VcrError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES[status] if 0 <= status < 7 else status}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libvcrown.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run paper_2606_09377_amd.build.build()")
    lib = ctypes.CDLL(path)
    P, I32, F32, D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_double
    sig = {
        "vcr_abi_version": ([], I32),
        "vcr_create": ([I32, ctypes.POINTER(P)], I32),
        "vcr_destroy": ([P], None),
        "vcr_last_error": ([P], ctypes.c_char_p),
        "vcr_set_stream": ([P, P], I32),
        "vcr_set_option": ([P, I32, D], I32),
        "vcr_load_net": ([P, ctypes.POINTER(VcrNode), I32, ctypes.POINTER(I32)], I32),
        "vcr_ibp_bounds": ([P, P, I32, F32, P, I32, P, P], I32),
        "vcr_crown_bounds": ([P, P, I32, F32, P, I32, ctypes.POINTER(VcrSplits), P, P], I32),
        "vcr_get_layer_bounds": ([P, I32, P, P], I32),
        "vcr_workspace_bytes": ([P, I32, I32, I32, ctypes.POINTER(ctypes.c_uint64)], I32),
        "vcr_get_stats": ([P, ctypes.POINTER(VcrStats)], I32),
        "vcr_alpha_crown_bounds": ([P, P, I32, F32, P, I32, ctypes.POINTER(VcrAlphaOpts), P, P], I32),
        "vcr_relu_neurons": ([P], ctypes.c_int64),
        "vcr_beta_crown_bounds": ([P, P, F32, P, I32, ctypes.POINTER(VcrSplits), ctypes.POINTER(VcrBetaOpts), P, P],
                                  I32),
        "vcr_bab_verify": ([P, P, F32, P, I32, ctypes.POINTER(VcrBabOpts), ctypes.POINTER(VcrBabResult), P], I32),
        "vcr_crown_bounds_noalloc": ([P, P, I32, F32, P, I32, P, P], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    if lib.vcr_abi_version() != ABI_VERSION:
        raise RuntimeError(f"{path} has ABI version {lib.vcr_abi_version()}, this binding expects {ABI_VERSION}: "
                           "rebuild the library")
    _lib = lib
    return lib


def header_symbols(path: str = HEADER):
    """Names of the functions include/vcrown.h declares."""
    txt = open(path).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(vcr_[a-z_]+)\s*\(", txt)))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _net_nodes(net):
    """(ctypes node array, keep-alive list, in_chw) from a workloads.Net-like object."""
    keep = []
    arr = (VcrNode * len(net.nodes))()
    for i, nd in enumerate(net.nodes):
        x = arr[i]
        x.op = OPS[nd.op]
        x.in0 = nd.in0
        x.in1 = nd.in1 if nd.op == "add" else -1
        if nd.W is not None:
            W = np.ascontiguousarray(nd.W, dtype=np.float32)
            b = np.ascontiguousarray(nd.b, dtype=np.float32)
            keep += [W, b]
            x.W = W.ctypes.data
            x.b = b.ctypes.data
            if nd.op == "dense":
                x.out_features = W.shape[0]
            else:
                x.out_ch, x.kh, x.kw = W.shape[0], W.shape[2], W.shape[3]
                x.stride, x.pad = nd.stride, nd.pad
    shp = tuple(net.in_shape)
    chw = (ctypes.c_int32 * 3)(*(shp + (1,) * (3 - len(shp))))
    return arr, keep, chw


class Ctx:
    """A vcrown context on one HIP device (device=-1: validation only, no GPU work)."""

    def __init__(self, device: int = 0):
        self.lib = load_library()
        h = ctypes.c_void_p()
        st = self.lib.vcr_create(device, ctypes.byref(h))
        if st != VCR_OK:
            raise VcrError(st, f"vcr_create({device}) failed")
        self.h = h
        self.device = device
        self.n_relu = 0
        self.relu_sizes = []

    def close(self):
        if getattr(self, "h", None):
            self.lib.vcr_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, st):
        if st != VCR_OK:
            raise VcrError(st, self.lib.vcr_last_error(self.h).decode())

    def set_option(self, key: int, value: float):
        self._check(self.lib.vcr_set_option(self.h, key, float(value)))

    def set_stream(self, stream=None):
        """Queue work on a torch stream (default: torch's current stream)."""
        import torch
        s = torch.cuda.current_stream() if stream is None else stream
        self._check(self.lib.vcr_set_stream(self.h, ctypes.c_void_p(s.cuda_stream)))

    def load_net(self, net):
        arr, keep, chw = _net_nodes(net)
        self._check(self.lib.vcr_load_net(self.h, arr, len(net.nodes), chw))
        del keep
        self.relu_sizes = _relu_sizes(net)
        self.n_relu = len(self.relu_sizes)
        self.n_out = _out_size(net)

    def _stream_sync(self):
        if self.device >= 0:
            self.set_stream()

    def crown_bounds(self, x0, eps, C, splits=None, out=None):
        """CROWN bounds on C f(x).  x0 (B, n0), C (B, m, n_out) float32 CUDA tensors.
        splits: optional (relu_id, neuron, sign) CUDA tensors of shape (D, S), B must be 1."""
        import torch
        B, m = C.shape[0], C.shape[1]
        rows = splits[0].shape[0] if splits is not None else B
        if out is None:
            lb = torch.empty((rows, m), dtype=torch.float32, device=x0.device)
            ub = torch.empty((rows, m), dtype=torch.float32, device=x0.device)
        else:
            lb, ub = out
        _check_tensor(x0, (B, None))
        _check_tensor(C, (B, m, None))
        self._stream_sync()
        sp = None
        if splits is not None:
            rid, neu, sgn = splits
            for t, dt in ((rid, torch.int32), (neu, torch.int32), (sgn, torch.int8)):
                if t.dtype != dt or not t.is_contiguous() or t.shape != rid.shape:
                    raise ValueError("splits must be contiguous (D, S) int32, int32, int8 tensors")
            sp = VcrSplits(rid.shape[0], rid.shape[1], rid.data_ptr(), neu.data_ptr(), sgn.data_ptr())
            sp = ctypes.byref(sp)
        self._check(self.lib.vcr_crown_bounds(self.h, _ptr(x0), B, ctypes.c_float(float(eps)), _ptr(C), m, sp,
                                              _ptr(lb), _ptr(ub)))
        return lb, ub

    def crown_bounds_noalloc(self, x0, eps, C, out):
        """CROWN bounds on C f(x) (no splits) through the allocation-free entry point: the
        call runs in the library's fixed per-GPU scratch.  out = (lb, ub), caller-allocated
        (B, m) float32 CUDA tensors."""
        B, m = C.shape[0], C.shape[1]
        lb, ub = out
        _check_tensor(x0, (B, None))
        _check_tensor(C, (B, m, None))
        _check_tensor(lb, (B, m))
        _check_tensor(ub, (B, m))
        self._stream_sync()
        self._check(self.lib.vcr_crown_bounds_noalloc(self.h, _ptr(x0), B, ctypes.c_float(float(eps)), _ptr(C), m,
                                                      _ptr(lb), _ptr(ub)))
        return lb, ub

    def alpha_crown_bounds(self, x0, eps, C, iters=20, lr=0.1, beta1=0.9, beta2=0.999, adam_eps=1e-8,
                           alpha_init=None, want_alpha=False, want_grad=False, want_hist=False, out=None):
        """alpha-CROWN bounds on C f(x) (x0 (B, n0), C (B, m, n_out) float32 CUDA tensors).

        Returns (lb, ub, extra): extra holds "alpha" and "grad" ((B, 2m, n_total): rows q < m
        the lower bound of spec row q, m + q its upper bound; columns the ReLU neurons in node
        order) and "lb_hist", "ub_hist" ((iters + 1, B, m)) when asked for."""
        import torch
        B, m = C.shape[0], C.shape[1]
        _check_tensor(x0, (B, None))
        _check_tensor(C, (B, m, None))
        n_total = int(self.lib.vcr_relu_neurons(self.h))
        dev = x0.device
        if out is None:
            lb = torch.empty((B, m), dtype=torch.float32, device=dev)
            ub = torch.empty((B, m), dtype=torch.float32, device=dev)
        else:
            lb, ub = out
            _check_tensor(lb, (B, m))
            _check_tensor(ub, (B, m))
        extra = {}
        o = VcrAlphaOpts(int(iters), float(lr), float(beta1), float(beta2), float(adam_eps), None, None, None, None, None)
        if alpha_init is not None:
            _check_tensor(alpha_init, (B, 2 * m, n_total))
            o.alpha_init = alpha_init.data_ptr()
        if want_alpha:
            extra["alpha"] = torch.empty((B, 2 * m, n_total), dtype=torch.float32, device=dev)
            o.alpha_out = extra["alpha"].data_ptr()
        if want_grad:
            extra["grad"] = torch.empty((B, 2 * m, n_total), dtype=torch.float32, device=dev)
            o.grad_out = extra["grad"].data_ptr()
        if want_hist:
            extra["lb_hist"] = torch.empty((iters + 1, B, m), dtype=torch.float32, device=dev)
            extra["ub_hist"] = torch.empty((iters + 1, B, m), dtype=torch.float32, device=dev)
            o.lb_hist = extra["lb_hist"].data_ptr()
            o.ub_hist = extra["ub_hist"].data_ptr()
        self._stream_sync()
        self._check(self.lib.vcr_alpha_crown_bounds(self.h, _ptr(x0), B, ctypes.c_float(float(eps)), _ptr(C), m,
                                                    ctypes.byref(o), _ptr(lb), _ptr(ub)))
        return lb, ub, extra

    def beta_crown_bounds(self, x0, eps, C, splits, iters=20, lr_alpha=0.1, lr_beta=0.05, beta1=0.9, beta2=0.999,
                          adam_eps=1e-8, want_hist=False):
        """beta-CROWN bounds of subdomains of one input: x0 (1, n0), C (1, m, n_out) CUDA
        tensors, splits (relu_id, neuron, sign) (D, S) CUDA tensors (relu_id -1: unused slot).
        Returns (lb, ub, extra) with lb, ub (D, m); extra "lb_hist", "ub_hist" (iters + 1, D, m)."""
        import torch
        m = C.shape[1]
        _check_tensor(x0, (1, None))
        _check_tensor(C, (1, m, None))
        rid, neu, sgn = splits
        for t, dt in ((rid, torch.int32), (neu, torch.int32), (sgn, torch.int8)):
            if t.dtype != dt or not t.is_contiguous() or t.shape != rid.shape:
                raise ValueError("splits must be contiguous (D, S) int32, int32, int8 tensors")
        D = rid.shape[0]
        dev = x0.device
        lb = torch.empty((D, m), dtype=torch.float32, device=dev)
        ub = torch.empty((D, m), dtype=torch.float32, device=dev)
        o = VcrBetaOpts(int(iters), float(lr_alpha), float(lr_beta), float(beta1), float(beta2), float(adam_eps),
                        None, None)
        extra = {}
        if want_hist:
            extra["lb_hist"] = torch.empty((iters + 1, D, m), dtype=torch.float32, device=dev)
            extra["ub_hist"] = torch.empty((iters + 1, D, m), dtype=torch.float32, device=dev)
            o.lb_hist, o.ub_hist = extra["lb_hist"].data_ptr(), extra["ub_hist"].data_ptr()
        sp = VcrSplits(D, rid.shape[1], rid.data_ptr(), neu.data_ptr(), sgn.data_ptr())
        self._stream_sync()
        self._check(self.lib.vcr_beta_crown_bounds(self.h, _ptr(x0), ctypes.c_float(float(eps)), _ptr(C), m,
                                                   ctypes.byref(sp), ctypes.byref(o), _ptr(lb), _ptr(ub)))
        return lb, ub, extra

    def bab_verify(self, x0, eps, C, batch=512, max_rounds=10, iters=20, lr_alpha=0.1, lr_beta=0.05, beta1=0.9,
                   beta2=0.999, adam_eps=1e-8, order=None):
        """Fixed-batch branch and bound on C f(x) > 0 (x0 (1, n0), C (1, m, n_out) CUDA tensors).
        order: optional [(relu position, neuron), ...] split priority.  Returns a dict with the
        result fields and "log": per round (taken, bounded, verified, left)."""
        m = C.shape[1]
        _check_tensor(x0, (1, None))
        _check_tensor(C, (1, m, None))
        bo = VcrBetaOpts(int(iters), float(lr_alpha), float(lr_beta), float(beta1), float(beta2), float(adam_eps),
                         None, None)
        keep = []
        o = VcrBabOpts(int(batch), int(max_rounds), bo, None, None, 0)
        if order is not None:
            orr = np.ascontiguousarray([int(a) for a, _ in order], dtype=np.int32)
            orn = np.ascontiguousarray([int(b) for _, b in order], dtype=np.int32)
            keep += [orr, orn]
            o.order_relu, o.order_neuron, o.order_len = orr.ctypes.data, orn.ctypes.data, len(orr)
        log = np.zeros((max(int(max_rounds), 1), 4), dtype=np.int64)
        res = VcrBabResult()
        self._stream_sync()
        self._check(self.lib.vcr_bab_verify(self.h, _ptr(x0), ctypes.c_float(float(eps)), _ptr(C), m, ctypes.byref(o),
                                            ctypes.byref(res), log.ctypes.data))
        return {"verified": bool(res.verified), "rounds": res.rounds, "evaluated": int(res.evaluated),
                "remaining": int(res.remaining), "root_min_lb": res.root_min_lb, "worst_lb": res.worst_lb,
                "log": [tuple(int(v) for v in r) for r in log[:res.rounds]]}

    def ibp_bounds(self, x0, eps, C):
        import torch
        B, m = C.shape[0], C.shape[1]
        _check_tensor(x0, (B, None))
        _check_tensor(C, (B, m, None))
        lb = torch.empty((B, m), dtype=torch.float32, device=x0.device)
        ub = torch.empty((B, m), dtype=torch.float32, device=x0.device)
        self._stream_sync()
        self._check(self.lib.vcr_ibp_bounds(self.h, _ptr(x0), B, ctypes.c_float(float(eps)), _ptr(C), m,
                                            _ptr(lb), _ptr(ub)))
        return lb, ub

    def layer_bounds(self, relu_id, B):
        import torch
        n = self.relu_sizes[relu_id]
        l = torch.empty((B, n), dtype=torch.float32, device="cuda")
        u = torch.empty((B, n), dtype=torch.float32, device="cuda")
        self._stream_sync()
        self._check(self.lib.vcr_get_layer_bounds(self.h, relu_id, _ptr(l), _ptr(u)))
        return l, u

    def workspace_bytes(self, B, m, n_domains=0):
        v = ctypes.c_uint64()
        self._check(self.lib.vcr_workspace_bytes(self.h, B, m, n_domains, ctypes.byref(v)))
        return int(v.value)

    def stats(self):
        s = VcrStats()
        self._check(self.lib.vcr_get_stats(self.h, ctypes.byref(s)))
        return {"ms_last_call": s.ms_last_call, "gemm_flops_last_call": int(s.gemm_flops_last_call),
                "peak_workspace_bytes": int(s.peak_workspace_bytes), "workspace_bytes": int(s.workspace_bytes),
                "n_chunks_last_call": s.n_chunks_last_call, "invalid_domains": s.invalid_domains,
                "n_relu": s.n_relu, "unstable": list(s.unstable[:min(s.n_relu, 64)]),
                "timed_gemm_launches": int(s.timed_gemm_launches), "timed_gemm_ms": s.timed_gemm_ms,
                "timed_gemm_flops": int(s.timed_gemm_flops), "timed_conv_launches": int(s.timed_conv_launches),
                "timed_conv_ms": s.timed_conv_ms, "timed_conv_flops": int(s.timed_conv_flops),
                "net_bytes": int(s.net_bytes), "timed_small_launches": int(s.timed_small_launches),
                "timed_small_ms": s.timed_small_ms, "timed_small_flops": int(s.timed_small_flops),
                "timed_mid_launches": int(s.timed_mid_launches), "timed_mid_ms": s.timed_mid_ms,
                "timed_mid_flops": int(s.timed_mid_flops)}


def _relu_sizes(net):
    sizes, shapes = [], []
    for nd in net.nodes:
        s = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
        if nd.op == "dense":
            shapes.append((nd.W.shape[0],))
        elif nd.op == "conv2d":
            kh, kw = nd.W.shape[2:]
            shapes.append((nd.W.shape[0], (s[1] + 2 * nd.pad - kh) // nd.stride + 1,
                           (s[2] + 2 * nd.pad - kw) // nd.stride + 1))
        elif nd.op == "flatten":
            shapes.append((int(np.prod(s)),))
        else:
            shapes.append(s)
        if nd.op == "relu":
            sizes.append(int(np.prod(s)))
    return sizes


def _out_size(net):
    return int(net.nodes[-1].W.shape[0])


def _check_tensor(t, shape):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous float32 CUDA tensor")
    if t.dim() != len(shape) or any(s is not None and s != d for s, d in zip(shape, t.shape)):
        raise ValueError(f"expected shape {shape}, got {tuple(t.shape)}")
