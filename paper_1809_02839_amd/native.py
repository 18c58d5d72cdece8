"""ctypes binding of libspectrain.so: one Python function per C ABI entry point
(argument marshalling only; every step of the stage runs in the library).

Device buffers are passed as torch tensors (their data pointers) and streams
as torch.cuda.Stream objects; host arrays as float32 NumPy arrays.
"""
import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspectrain.so")

ABI_VERSION = 3
OK, EINVAL, ENOMEM, EHIP, ESTATE, ENONFINITE = range(6)
STATUS_NAMES = {OK: "OK", EINVAL: "EINVAL", ENOMEM: "ENOMEM", EHIP: "EHIP", ESTATE: "ESTATE",
                ENONFINITE: "ENONFINITE"}
FP32, BF16 = 0, 1
KIND_FC, KIND_CONV3X3, KIND_BOTTLENECK, KIND_TRANSFORMER, KIND_RESLSTM = range(5)
HEAD_NONE, HEAD_CE = 0, 1
POLICY_PREDICT, POLICY_STASH = 0, 1
POLICIES = ("spectrain", "vanilla", "stash")
KIND_BY_NAME = {"fc": KIND_FC, "conv3x3": KIND_CONV3X3, "bottleneck": KIND_BOTTLENECK,
                "transformer": KIND_TRANSFORMER, "reslstm": KIND_RESLSTM}

EXPORTED = ("spectrain_version_difference", "spectrain_stage_create", "spectrain_stage_num_params",
            "spectrain_stage_predict", "spectrain_stage_forward", "spectrain_stage_backward",
            "spectrain_stage_backward_noalloc", "spectrain_stage_forward_backward",
            "spectrain_stage_update", "spectrain_stage_get_state", "spectrain_stage_set_state",
            "spectrain_stage_get_predicted", "spectrain_stage_profile", "spectrain_stage_profile_read",
            "spectrain_stage_read_stash", "spectrain_stage_destroy", "spectrain_last_error")


class StageDesc(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("kind", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("head", ctypes.c_int32), ("stage_index", ctypes.c_int32), ("num_stages", ctypes.c_int32),
                ("batch", ctypes.c_int32), ("num_layers", ctypes.c_int32), ("dims", ctypes.c_int32 * 8),
                ("lr", ctypes.c_float), ("momentum", ctypes.c_float), ("weight_policy", ctypes.c_int32)]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64), ("ms_total", ctypes.c_double),
                ("flops_total", ctypes.c_double), ("bytes_total", ctypes.c_double),
                ("extra_bytes_total", ctypes.c_double)]


class SpecTrainError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


_lib = None


def lib():
    """Open libspectrain.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_1809_02839_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        fp = ctypes.POINTER(ctypes.c_float)
        sig = {
            "spectrain_version_difference": (i32, [i32, i32, i32]),
            "spectrain_stage_create": (ctypes.c_int, [ctypes.POINTER(StageDesc), fp, sz, vp, ctypes.POINTER(vp)]),
            "spectrain_stage_num_params": (ctypes.c_int, [vp, ctypes.POINTER(sz)]),
            "spectrain_stage_predict": (ctypes.c_int, [vp, i32, i32]),
            "spectrain_stage_forward": (ctypes.c_int, [vp, i64, vp, vp, vp, vp]),
            "spectrain_stage_backward": (ctypes.c_int, [vp, i64, vp, vp]),
            "spectrain_stage_backward_noalloc": (ctypes.c_int, [vp, i64, vp, vp]),
            "spectrain_stage_forward_backward": (ctypes.c_int, [vp, i64, vp, vp, vp, vp, i64, vp, vp]),
            "spectrain_stage_update": (ctypes.c_int, [vp, i32, i32]),
            "spectrain_stage_get_state": (ctypes.c_int, [vp, fp, fp]),
            "spectrain_stage_set_state": (ctypes.c_int, [vp, fp, fp]),
            "spectrain_stage_get_predicted": (ctypes.c_int, [vp, i32, fp]),
            "spectrain_stage_profile": (ctypes.c_int, [vp, i32]),
            "spectrain_stage_profile_read": (ctypes.c_int, [vp, ctypes.POINTER(KernelStat), i32,
                                                            ctypes.POINTER(i32)]),
            "spectrain_stage_read_stash": (ctypes.c_int, [vp, i64, i32, vp, sz, ctypes.POINTER(sz)]),
            "spectrain_stage_destroy": (ctypes.c_int, [vp]),
            "spectrain_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _check(code):
    if code != OK:
        raise SpecTrainError(code, lib().spectrain_last_error().decode())


def _fptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def _dptr(t, dtype=None, what="tensor"):
    """Device pointer of a torch tensor. The library reads raw pointers, so a
    host tensor, a strided view or the wrong element type is refused here
    rather than reaching a kernel."""
    if t is None:
        return None
    if not getattr(t, "is_cuda", False):
        raise ValueError(f"{what} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and str(t.dtype) != dtype:
        raise ValueError(f"{what} must be {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def version_difference(k: int, N: int, forward: bool) -> int:
    return int(lib().spectrain_version_difference(k, N, 1 if forward else 0))


def policy_versions(policy: str, k: int, N: int):
    """(s before a forward, s before a backward) of stage k of N: Eq. 5 and
    Eq. 6 for SpecTrain; 0 for both under the Vanilla and stashing policies
    (every pass starts from the latest weights; with stashing the backward
    then reads the copy its forward used)."""
    if policy == "spectrain":
        return version_difference(k, N, True), version_difference(k, N, False)
    if policy in ("vanilla", "stash"):
        return 0, 0
    raise ValueError(f"unknown policy {policy!r}")


def make_desc(kind, dtype, head, stage_index, num_stages, batch, num_layers, dims, lr, momentum,
              weight_policy=POLICY_PREDICT) -> StageDesc:
    d = StageDesc()
    d.abi_version = ABI_VERSION
    d.kind = KIND_BY_NAME[kind] if isinstance(kind, str) else int(kind)
    d.dtype = {"fp32": FP32, "bf16": BF16}[dtype] if isinstance(dtype, str) else int(dtype)
    d.head = {"none": HEAD_NONE, "ce": HEAD_CE}[head] if isinstance(head, str) else int(head)
    d.stage_index, d.num_stages, d.batch, d.num_layers = stage_index, num_stages, batch, num_layers
    for i, v in enumerate(dims):
        d.dims[i] = int(v)
    d.lr, d.momentum = lr, momentum
    d.weight_policy = int(weight_policy)
    return d


def desc_from_spec(spec) -> StageDesc:
    policy = getattr(spec, "policy", "spectrain")
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy!r}")
    return make_desc(spec.kind, spec.dtype, spec.head, spec.stage_index, spec.num_stages, spec.batch,
                     spec.num_layers, spec.dims, spec.lr, spec.momentum,
                     POLICY_STASH if policy == "stash" else POLICY_PREDICT)


class Stage:
    """Owner of one spectrain_stage_t; methods map 1:1 to the C entry points."""

    def __init__(self, desc: StageDesc, W0: np.ndarray, stream=None):
        W0 = np.ascontiguousarray(W0, dtype=np.float32)
        self._stream = stream
        handle = ctypes.c_void_p()
        sptr = ctypes.c_void_p(stream.cuda_stream) if stream is not None else None
        _check(lib().spectrain_stage_create(ctypes.byref(desc), _fptr(W0), W0.size, sptr, ctypes.byref(handle)))
        self.h = handle
        self.desc = desc
        n = ctypes.c_size_t()
        _check(lib().spectrain_stage_num_params(self.h, ctypes.byref(n)))
        self.n_params = n.value

    def predict(self, s: int, slot: int):
        _check(lib().spectrain_stage_predict(self.h, s, slot))

    @property
    def _act(self):
        return "torch.bfloat16" if self.desc.dtype == BF16 else "torch.float32"

    def forward(self, mb: int, x, y=None, labels=None, loss=None):
        a = self._act
        _check(lib().spectrain_stage_forward(self.h, mb, _dptr(x, a, "x"), _dptr(y, a, "y"),
                                             _dptr(labels, "torch.int32", "labels"),
                                             _dptr(loss, "torch.float32", "loss")))

    def backward(self, mb: int, dy=None, dx=None):
        a = self._act
        _check(lib().spectrain_stage_backward(self.h, mb, _dptr(dy, a, "dy"), _dptr(dx, a, "dx")))

    def backward_noalloc(self, mb: int, dy=None, dx=None):
        a = self._act
        _check(lib().spectrain_stage_backward_noalloc(self.h, mb, _dptr(dy, a, "dy"), _dptr(dx, a, "dx")))

    def forward_backward(self, mb_fwd: int, x, y, mb_bwd: int, dy=None, dx=None, labels=None, loss=None):
        """forward(mb_fwd) then backward(mb_bwd), the two passes running concurrently."""
        a = self._act
        _check(lib().spectrain_stage_forward_backward(self.h, mb_fwd, _dptr(x, a, "x"), _dptr(y, a, "y"),
                                                      _dptr(labels, "torch.int32", "labels"),
                                                      _dptr(loss, "torch.float32", "loss"), mb_bwd,
                                                      _dptr(dy, a, "dy"), _dptr(dx, a, "dx")))

    def update(self, s_next_fwd: int, s_next_bwd: int):
        _check(lib().spectrain_stage_update(self.h, s_next_fwd, s_next_bwd))

    def get_state(self):
        W = np.empty(self.n_params, np.float32)
        v = np.empty(self.n_params, np.float32)
        _check(lib().spectrain_stage_get_state(self.h, _fptr(W), _fptr(v)))
        return W, v

    def set_state(self, W: np.ndarray, v=None):
        W = np.ascontiguousarray(W, dtype=np.float32)
        v = None if v is None else np.ascontiguousarray(v, dtype=np.float32)
        _check(lib().spectrain_stage_set_state(self.h, _fptr(W), _fptr(v)))

    def get_predicted(self, slot: int):
        out = np.empty(self.n_params, np.float32)
        _check(lib().spectrain_stage_get_predicted(self.h, slot, _fptr(out)))
        return out

    def read_stash(self, mb: int, index: int) -> np.ndarray:
        """Stash buffer `index` of mini-batch mb (in flight) as raw bytes
        (uint8; empty when the stage does not use that index)."""
        n = ctypes.c_size_t()
        _check(lib().spectrain_stage_read_stash(self.h, mb, index, None, 0, ctypes.byref(n)))
        out = np.empty(n.value, np.uint8)
        if n.value:
            _check(lib().spectrain_stage_read_stash(self.h, mb, index, ctypes.c_void_p(out.ctypes.data), out.size,
                                                    ctypes.byref(n)))
        return out

    def profile(self, enable: bool, serial: bool = False):
        """Time every launch (serial: each on the stage stream, one at a time)."""
        _check(lib().spectrain_stage_profile(self.h, (2 if serial else 1) if enable else 0))

    def profile_read(self):
        """{family: dict(launches, ms_total, flops_total, bytes_total, extra_bytes_total)} in first-launch order."""
        cap = 64
        arr = (KernelStat * cap)()
        n = ctypes.c_int32()
        _check(lib().spectrain_stage_profile_read(self.h, arr, cap, ctypes.byref(n)))
        return {arr[i].name.decode(): dict(launches=arr[i].launches, ms_total=arr[i].ms_total,
                                           flops_total=arr[i].flops_total, bytes_total=arr[i].bytes_total,
                                           extra_bytes_total=arr[i].extra_bytes_total)
                for i in range(min(n.value, cap))}

    def destroy(self):
        if self.h is not None and self.h.value:
            _check(lib().spectrain_stage_destroy(self.h))
        self.h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass
