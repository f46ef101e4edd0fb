"""Python binding of libzo, the 1.5-SPSA probe regenerate-and-apply sweep for MI355X (gfx950).

Argument marshalling only: every step of the sweep runs in the library's HIP kernels (or,
for zo_probe_coeffs, its host C code). PyTorch supplies device memory (a tensor's
data_ptr) and the stream (torch's current stream unless one is given). The functions keep
the C names of include/zo.h:

  zo_perturb(theta, k, eps, seed, step, offset=0)       theta <- theta + eps z_k
  zo_probe_coeffs(L_plus, L_minus, L_clean, eps)        c_k from the losses (host)
  zo_probe_coeffs_ex(..., alpha, lambda_reg)            also c64, curvature, weight
  zo_update(theta, c, lr, seed, step)                   theta <- theta - lr sum_k c_k z_k
  zo_update_ex(theta, c, lr, seed, step, offset, k_base)
  zo_perturb2(theta, k_a, eps_a, k_b, eps_b, seed, step) theta + eps_a z_a + eps_b z_b (one pass)
  zo_update_restore(theta, c, lr, seed, step, k_restore, eps_restore)
                                                        restore of one probe fused with the update
  zo_perturb_segments(tensors, offsets, k_a, eps_a, k_b, eps_b, seed, step)
  zo_update_segments(tensors, offsets, c, lr, seed, step, k_restore=0, eps_restore=0.0)
                                                        the same over a list of separate tensors
  zo_gen_bits(out, tile_begin, seed, step, group)       raw probe blocks (uint8 tensor)

If libzo.so has not been built the import succeeds but every call raises ZoLibraryMissing:
there is no fallback implementation.
"""

import ctypes
import os

import numpy as np

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libzo.so")

ZO_F32, ZO_BF16 = 0, 1
ZO_OK, ZO_ERR_NULL, ZO_ERR_ARG, ZO_ERR_NONFINITE, ZO_ERR_HIP = 0, -1, -2, -3, -4
ZO_K_MAX = 1024
ZO_N_MAX = 1 << 40
TILE = 16

EXPORTS = ("zo_perturb", "zo_perturb2", "zo_probe_coeffs", "zo_probe_coeffs_ex", "zo_update", "zo_update_ex",
           "zo_update_restore", "zo_perturb_segments", "zo_update_segments", "zo_gen_bits", "zo_strerror",
           "zo_set_max_blocks", "zo_version")


class ZoSegment(ctypes.Structure):
    _fields_ = [("params", ctypes.c_void_p), ("offset", ctypes.c_uint64), ("n", ctypes.c_uint64)]


class ZoLibraryMissing(RuntimeError):
    pass


class ZoError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {_lib().zo_strerror(status).decode()} (status {status})")


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ZoLibraryMissing(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        u64, u32, f32, f64, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float, ctypes.c_double, ctypes.c_void_p
        pd, pf = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_float)
        lib.zo_perturb.argtypes = [vp, ctypes.c_int, u64, u64, u64, u32, u32, f32, vp]
        lib.zo_probe_coeffs.argtypes = [pd, pd, u32, f64, f64, pf]
        lib.zo_probe_coeffs_ex.argtypes = [pd, pd, u32, f64, f64, f64, f64, pf, pd, pd, pd]
        lib.zo_update.argtypes = [vp, ctypes.c_int, u64, u64, u32, u32, pf, f32, vp]
        lib.zo_update_ex.argtypes = [vp, ctypes.c_int, u64, u64, u64, u32, u32, u32, pf, f32, vp]
        lib.zo_perturb2.argtypes = [vp, ctypes.c_int, u64, u64, u64, u32, u32, f32, u32, f32, vp]
        lib.zo_update_restore.argtypes = [vp, ctypes.c_int, u64, u64, u64, u32, u32, u32, pf, f32, u32, f32, vp]
        ps = ctypes.POINTER(ZoSegment)
        lib.zo_perturb_segments.argtypes = [ps, u32, ctypes.c_int, u64, u32, u32, f32, u32, f32, vp]
        lib.zo_update_segments.argtypes = [ps, u32, ctypes.c_int, u64, u32, u32, u32, pf, f32, u32, f32, vp]
        lib.zo_gen_bits.argtypes = [vp, u64, u64, u64, u32, u32, vp]
        lib.zo_strerror.argtypes = [ctypes.c_int]
        lib.zo_strerror.restype = ctypes.c_char_p
        lib.zo_set_max_blocks.argtypes = [u32]
        lib.zo_set_max_blocks.restype = None
        lib.zo_version.restype = ctypes.c_char_p
        for name in ("zo_perturb", "zo_perturb2", "zo_probe_coeffs", "zo_probe_coeffs_ex", "zo_update",
                     "zo_update_ex", "zo_update_restore", "zo_perturb_segments", "zo_update_segments",
                     "zo_gen_bits"):
            getattr(lib, name).restype = ctypes.c_int
        _LIB = lib
    return _LIB


def library():
    """The loaded ctypes library (raises ZoLibraryMissing if it is not built)."""
    return _lib()


def _check(status, what):
    if status != ZO_OK:
        raise ZoError(status, what)


def _stream(theta_or_device, stream):
    """The hipStream_t to launch on: torch's current stream of the tensor's device, or the
    given stream (a torch stream, which must belong to that device, or a raw handle). The
    library launches on the current device, so the tensors must live there."""
    import torch
    dev = theta_or_device.device if hasattr(theta_or_device, "device") else theta_or_device  # None: no tensors
    if dev is not None and torch.device(dev).index not in (None, torch.cuda.current_device()):
        raise ValueError(f"the tensors live on {dev}, the current device is cuda:{torch.cuda.current_device()}")
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    if hasattr(stream, "cuda_stream"):
        sdev = getattr(stream, "device", None)
        if dev is not None and sdev is not None and torch.device(sdev) != torch.device(dev):
            raise ValueError(f"the stream belongs to {sdev}, the tensors to {dev}")
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _theta_args(theta):
    import torch
    if not isinstance(theta, torch.Tensor) or not theta.is_cuda:
        raise TypeError("theta must be a CUDA (HIP) torch tensor")
    if not theta.is_contiguous():
        raise ValueError("theta must be contiguous")
    if theta.dtype == torch.float32:
        dt = ZO_F32
    elif theta.dtype == torch.bfloat16:
        dt = ZO_BF16
    else:
        raise TypeError("theta must be float32 or bfloat16")
    return ctypes.c_void_p(theta.data_ptr()), dt, theta.numel()


def zo_perturb(theta, k, eps, seed, step, offset=0, stream=None):
    """theta[i] <- theta[i] + eps * z_k[offset + i], in place, asynchronously on the stream."""
    p, dt, n = _theta_args(theta)
    _check(_lib().zo_perturb(p, dt, offset, n, seed, step, k, eps, _stream(theta, stream)), "zo_perturb")


def zo_perturb2(theta, k_a, eps_a, k_b, eps_b, seed, step, offset=0, stream=None):
    """theta[i] <- theta[i] + (eps_a z_{k_a} + eps_b z_{k_b})[offset + i], one pass, in place."""
    p, dt, n = _theta_args(theta)
    _check(_lib().zo_perturb2(p, dt, offset, n, seed, step, k_a, eps_a, k_b, eps_b, _stream(theta, stream)),
           "zo_perturb2")


def zo_update_restore(theta, c, lr, seed, step, k_restore, eps_restore, offset=0, k_base=0, stream=None):
    """theta <- theta + eps_restore z_{k_restore} - lr * sum_j c[j] z_{k_base+j}, one pass, in place."""
    p, dt, n = _theta_args(theta)
    c = np.ascontiguousarray(np.asarray(c, dtype=np.float32))
    cp = c.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if c.size else None
    _check(_lib().zo_update_restore(p, dt, offset, n, seed, step, k_base, c.size, cp, lr, k_restore, eps_restore,
                                    _stream(theta, stream)), "zo_update_restore")


def _segments(tensors, offsets):
    tensors = list(tensors)
    if len(tensors) != len(offsets):
        raise ValueError("one global offset per tensor")
    dts = {t.dtype for t in tensors}
    if len(dts) > 1:
        raise TypeError("all tensors must share one dtype")
    devs = {t.device for t in tensors}
    if len(devs) > 1:
        raise ValueError("all tensors must be on one device (the stream's)")
    arr = (ZoSegment * max(len(tensors), 1))()
    dt = ZO_F32
    for i, (t, o) in enumerate(zip(tensors, offsets)):
        p, dt, n = _theta_args(t)
        arr[i] = ZoSegment(p, int(o), n)
    return arr, len(tensors), dt, (tensors[0] if tensors else None)


def zo_perturb_segments(tensors, offsets, k_a, eps_a, k_b, eps_b, seed, step, stream=None):
    """For each tensor t_s with global offset o_s: t_s <- t_s + (eps_a z_{k_a} + eps_b z_{k_b})[o_s + i]."""
    arr, n, dt, ref = _segments(tensors, offsets)
    _check(_lib().zo_perturb_segments(arr, n, dt, seed, step, k_a, eps_a, k_b, eps_b, _stream(ref, stream)),
           "zo_perturb_segments")


def zo_update_segments(tensors, offsets, c, lr, seed, step, k_restore=0, eps_restore=0.0, k_base=0, stream=None):
    """For each tensor: t_s <- t_s + eps_restore z_{k_restore} - lr * sum_j c[j] z_{k_base+j} (global indices)."""
    arr, n, dt, ref = _segments(tensors, offsets)
    c = np.ascontiguousarray(np.asarray(c, dtype=np.float32))
    cp = c.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if c.size else None
    _check(_lib().zo_update_segments(arr, n, dt, seed, step, k_base, c.size, cp, lr, k_restore, eps_restore,
                                     _stream(ref, stream)), "zo_update_segments")


def zo_update_ex(theta, c, lr, seed, step, offset=0, k_base=0, stream=None):
    """theta[i] <- theta[i] - lr * sum_j c[j] z_{k_base+j}[offset + i], in place."""
    p, dt, n = _theta_args(theta)
    c = np.ascontiguousarray(np.asarray(c, dtype=np.float32))
    cp = c.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if c.size else None
    _check(_lib().zo_update_ex(p, dt, offset, n, seed, step, k_base, c.size, cp, lr, _stream(theta, stream)),
           "zo_update_ex")


def zo_update(theta, c, lr, seed, step, stream=None):
    """theta[i] <- theta[i] - lr * sum_k c[k] z_k[i] over the whole vector (offset 0, k_base 0)."""
    p, dt, n = _theta_args(theta)
    c = np.ascontiguousarray(np.asarray(c, dtype=np.float32))
    cp = c.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) if c.size else None
    _check(_lib().zo_update(p, dt, n, seed, step, c.size, cp, lr, _stream(theta, stream)), "zo_update")


def _doubles(x):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def zo_probe_coeffs_ex(L_plus, L_minus, L_clean, eps, alpha=0.1, lambda_reg=1.0):
    """Returns dict(c=float32[K], c64, curv, w) computed by the library's host function."""
    lp, lpp = _doubles(L_plus)
    lm, lmp = _doubles(L_minus)
    if lp.size != lm.size:
        raise ValueError("L_plus and L_minus differ in length")
    K = lp.size
    c = np.zeros(K, np.float32)
    c64, curv, w = np.zeros(K), np.zeros(K), np.zeros(K)
    pd = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    _check(_lib().zo_probe_coeffs_ex(lpp, lmp, K, L_clean, eps, alpha, lambda_reg,
                                     c.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), pd(c64), pd(curv), pd(w)),
           "zo_probe_coeffs_ex")
    return {"c": c, "c64": c64, "curv": curv, "w": w}


def zo_probe_coeffs(L_plus, L_minus, L_clean, eps):
    """float32 coefficients with the paper's alpha = 0.1 and lambda_reg = 1."""
    lp, lpp = _doubles(L_plus)
    lm, lmp = _doubles(L_minus)
    if lp.size != lm.size:
        raise ValueError("L_plus and L_minus differ in length")
    c = np.zeros(lp.size, np.float32)
    _check(_lib().zo_probe_coeffs(lpp, lmp, lp.size, L_clean, eps, c.ctypes.data_as(ctypes.POINTER(ctypes.c_float))),
           "zo_probe_coeffs")
    return c


def zo_gen_bits(out, tile_begin, seed, step, group, stream=None):
    """Write the 16-byte probe block of tiles tile_begin .. tile_begin + out.numel()/16 - 1."""
    import torch
    if not isinstance(out, torch.Tensor) or not out.is_cuda or out.dtype != torch.uint8 or not out.is_contiguous():
        raise TypeError("out must be a contiguous uint8 CUDA tensor")
    if out.numel() % TILE:
        raise ValueError("out must hold a whole number of 16-byte blocks")
    _check(_lib().zo_gen_bits(ctypes.c_void_p(out.data_ptr()), tile_begin, out.numel() // TILE, seed, step, group,
                              _stream(out, stream)), "zo_gen_bits")


def zo_set_max_blocks(max_blocks):
    _lib().zo_set_max_blocks(int(max_blocks))


def zo_version():
    return _lib().zo_version().decode()
