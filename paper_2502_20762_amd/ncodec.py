"""ctypes binding of libncodec.so (the C ABI declared in include/ncodec.h).

The ``ncodec_*`` functions mirror the C entry points one to one and only
marshal arguments: device buffers are passed as integer addresses, host
weights as a float32 NumPy array.  :class:`Codec` is a thin convenience layer
that uses PyTorch for device memory and the stream; every step of the
transform runs in the HIP kernels of the library.  There is no fallback: if
the library is not built, importing the binding raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libncodec.so")

NCODEC_OK = 0
NCODEC_EINVAL = -1
NCODEC_ESHAPE = -2
NCODEC_EHIP = -3
NCODEC_ESTATE = -4
NCODEC_EOVERFLOW = -5
NCODEC_ENOMEM = -6
NCODEC_PATH_FP16 = 0
NCODEC_PATH_INT16 = 1

PATHS = {"fp16": NCODEC_PATH_FP16, "int16": NCODEC_PATH_INT16}
NCODEC_BLOCK_LRELU, NCODEC_BLOCK_GATED = 0, 1
BLOCKS = {"lrelu": NCODEC_BLOCK_LRELU, "gated": NCODEC_BLOCK_GATED}


class ncodec_config(ctypes.Structure):
    _fields_ = [
        ("height", ctypes.c_int32),
        ("width", ctypes.c_int32),
        ("channels", ctypes.c_int32),
        ("n_enc_blocks", ctypes.c_int32),
        ("n_dec_blocks", ctypes.c_int32),
        ("path", ctypes.c_int32),
        ("block", ctypes.c_int32),
        ("n_fe_blocks", ctypes.c_int32),
        ("n_rg_blocks", ctypes.c_int32),
        ("qp_banks", ctypes.c_int32),
        ("hyperprior", ctypes.c_int32),
    ]


class ncodec_kernel_timing(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_char * 16), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


class NcodecError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"ncodec status {status}: {message}")
        self.status = status


_P = ctypes.c_void_p
_SIGNATURES = {
    "ncodec_weight_count": (ctypes.c_size_t, [ctypes.POINTER(ncodec_config)]),
    "ncodec_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ncodec_config)]),
    "ncodec_symbol_count": (ctypes.c_size_t, [ctypes.POINTER(ncodec_config)]),
    "ncodec_create": (ctypes.c_int, [ctypes.POINTER(ncodec_config), _P, ctypes.c_size_t, _P, ctypes.c_size_t, _P,
                                     ctypes.POINTER(_P)]),
    "ncodec_reset": (ctypes.c_int, [_P]),
    "ncodec_set_qp": (ctypes.c_int, [_P, ctypes.c_int32]),
    "ncodec_set_rate": (ctypes.c_int, [_P, ctypes.c_double]),
    "ncodec_encode_frame": (ctypes.c_int, [_P, _P, _P, _P]),
    "ncodec_decode_frame": (ctypes.c_int, [_P, _P, _P]),
    "ncodec_estimate_bits": (ctypes.c_int, [_P, _P, _P, ctypes.c_int64, _P]),
    "ncodec_estimate_bits_noalloc": (ctypes.c_int, [_P, _P, ctypes.c_int64, _P, _P]),
    "ncodec_stream_capacity": (ctypes.c_size_t, [ctypes.POINTER(ncodec_config)]),
    "ncodec_scale_indices": (ctypes.c_int, [_P, _P]),
    "ncodec_rans_encode": (ctypes.c_int, [_P, _P, _P, ctypes.c_int64, _P, ctypes.c_size_t, _P]),
    "ncodec_rans_decode": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P, ctypes.c_int64, _P, _P]),
    "ncodec_encode_frame_coded": (ctypes.c_int, [_P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "ncodec_decode_frame_coded": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P, _P]),
    "ncodec_parallel_coding": (ctypes.c_int, [_P, ctypes.c_int32]),
    "ncodec_get_state": (ctypes.c_int, [_P, _P, _P]),
    "ncodec_set_state": (ctypes.c_int, [_P, _P, _P]),
    "ncodec_kernels_per_frame": (ctypes.c_int32, [_P, ctypes.c_int32]),
    "ncodec_timing_enable": (ctypes.c_int, [_P, ctypes.c_int32]),
    "ncodec_graph_enable": (ctypes.c_int, [_P, ctypes.c_int32]),
    "ncodec_block_chains": (ctypes.c_int, [_P, ctypes.c_int32]),
    "ncodec_block_chain_status": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
    "ncodec_timing_read": (ctypes.c_int, [_P, ctypes.POINTER(ncodec_kernel_timing), ctypes.c_int32,
                                          ctypes.POINTER(ctypes.c_int32)]),
    "ncodec_last_error": (ctypes.c_char_p, [_P]),
    "ncodec_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "ncodec_destroy": (None, [_P]),
}

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2502_20762_amd.build` "
                          "(there is no CPU fallback)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def make_config(height, width, channels, n_enc_blocks, n_dec_blocks, path, block="lrelu", n_fe_blocks=0,
                n_rg_blocks=0, qp_banks=False, hyperprior=False) -> ncodec_config:
    if isinstance(path, str):
        path = PATHS[path]
    if isinstance(block, str):
        block = BLOCKS[block]
    return ncodec_config(height, width, channels, n_enc_blocks, n_dec_blocks, path, block, n_fe_blocks,
                         n_rg_blocks, int(bool(qp_banks)), int(bool(hyperprior)))


def _p(v: int):
    """Device address for a pointer argument (0 -> NULL)."""
    return v or None


def _check(st: int, ctx=None) -> None:
    if st != NCODEC_OK:
        msg = load_library().ncodec_last_error(ctx)
        raise NcodecError(st, (msg or b"").decode() or load_library().ncodec_status_string(st).decode())


# ---------------------------------------------------------------- C entry points
def ncodec_weight_count(cfg: ncodec_config) -> int:
    return int(load_library().ncodec_weight_count(ctypes.byref(cfg)))


def ncodec_workspace_bytes(cfg: ncodec_config) -> int:
    return int(load_library().ncodec_workspace_bytes(ctypes.byref(cfg)))


def ncodec_symbol_count(cfg: ncodec_config) -> int:
    return int(load_library().ncodec_symbol_count(ctypes.byref(cfg)))


def ncodec_create(cfg: ncodec_config, host_weights: np.ndarray, d_workspace: int, ws_bytes: int,
                  hip_stream: int = 0):
    w = np.ascontiguousarray(host_weights, dtype=np.float32)
    out = _P()
    st = load_library().ncodec_create(ctypes.byref(cfg), w.ctypes.data, w.size, d_workspace, ws_bytes,
                                      hip_stream or None, ctypes.byref(out))
    _check(st, None)
    return out


def ncodec_reset(ctx) -> None:
    _check(load_library().ncodec_reset(ctx), ctx)


def ncodec_set_qp(ctx, qp: int) -> None:
    _check(load_library().ncodec_set_qp(ctx, int(qp)), ctx)


def ncodec_set_rate(ctx, qp: float) -> None:
    _check(load_library().ncodec_set_rate(ctx, float(qp)), ctx)


def ncodec_encode_frame(ctx, d_frame: int, d_q: int, d_bits: int = 0) -> None:
    _check(load_library().ncodec_encode_frame(ctx, d_frame, d_q, d_bits or None), ctx)


def ncodec_decode_frame(ctx, d_q: int, d_frame_out: int) -> None:
    _check(load_library().ncodec_decode_frame(ctx, d_q, d_frame_out), ctx)


def ncodec_estimate_bits(ctx, d_q: int, d_scale: int, n: int, d_bits: int) -> None:
    _check(load_library().ncodec_estimate_bits(ctx, d_q or None, d_scale or None, n, d_bits), ctx)


def ncodec_estimate_bits_noalloc(d_q: int, d_sigma: int, n: int, d_bits: int, stream: int = 0) -> None:
    _check(load_library().ncodec_estimate_bits_noalloc(d_q or None, d_sigma or None, n, d_bits or None,
                                                       stream or None), None)


def ncodec_stream_capacity(cfg: ncodec_config) -> int:
    return int(load_library().ncodec_stream_capacity(ctypes.byref(cfg)))


def ncodec_scale_indices(ctx, d_k: int) -> None:
    _check(load_library().ncodec_scale_indices(ctx, _p(d_k)), ctx)


def ncodec_rans_encode(ctx, d_q: int, d_k: int, n: int, d_stream: int, capacity: int, d_stream_bytes: int) -> None:
    _check(load_library().ncodec_rans_encode(ctx, _p(d_q), _p(d_k), n, _p(d_stream), capacity, _p(d_stream_bytes)), ctx)


def ncodec_rans_decode(ctx, d_stream: int, stream_bytes: int, d_k: int, n: int, d_q: int, d_status: int = 0) -> None:
    _check(load_library().ncodec_rans_decode(ctx, _p(d_stream), stream_bytes, _p(d_k), n, _p(d_q), _p(d_status)), ctx)


def ncodec_encode_frame_coded(ctx, d_frame: int, d_q: int, d_bits: int, d_stream: int, capacity: int,
                              d_stream_bytes: int) -> None:
    _check(load_library().ncodec_encode_frame_coded(ctx, _p(d_frame), _p(d_q), _p(d_bits), _p(d_stream), capacity,
                                                    _p(d_stream_bytes)), ctx)


def ncodec_decode_frame_coded(ctx, d_stream: int, stream_bytes: int, d_frame_out: int, d_status: int = 0) -> None:
    _check(load_library().ncodec_decode_frame_coded(ctx, _p(d_stream), stream_bytes, _p(d_frame_out), _p(d_status)),
           ctx)


def ncodec_parallel_coding(ctx, enable: bool) -> None:
    _check(load_library().ncodec_parallel_coding(ctx, 1 if enable else 0), ctx)


def ncodec_get_state(ctx, d_feat: int, d_yhat: int) -> None:
    _check(load_library().ncodec_get_state(ctx, d_feat or None, d_yhat or None), ctx)


def ncodec_set_state(ctx, d_feat: int, d_yhat: int) -> None:
    _check(load_library().ncodec_set_state(ctx, d_feat or None, d_yhat or None), ctx)


def ncodec_kernels_per_frame(ctx, decode: bool) -> int:
    return int(load_library().ncodec_kernels_per_frame(ctx, 1 if decode else 0))


def ncodec_timing_enable(ctx, enable: bool) -> None:
    _check(load_library().ncodec_timing_enable(ctx, 1 if enable else 0), ctx)


def ncodec_graph_enable(ctx, enable: bool) -> None:
    _check(load_library().ncodec_graph_enable(ctx, 1 if enable else 0), ctx)


def ncodec_block_chains(ctx, enable: bool) -> None:
    _check(load_library().ncodec_block_chains(ctx, 1 if enable else 0), ctx)


def ncodec_block_chain_status(ctx) -> tuple:
    """(in_use, timeouts) of the context's block chains."""
    u, v = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(load_library().ncodec_block_chain_status(ctx, ctypes.byref(u), ctypes.byref(v)), ctx)
    return int(u.value), int(v.value)


def ncodec_timing_read(ctx) -> dict:
    """{kind: (launches, total_ms)} for the kernels enqueued since timing was enabled."""
    buf = (ncodec_kernel_timing * 32)()
    n = ctypes.c_int32(0)
    _check(load_library().ncodec_timing_read(ctx, buf, 32, ctypes.byref(n)), ctx)
    return {buf[i].kind.decode(): (int(buf[i].launches), float(buf[i].total_ms)) for i in range(min(n.value, 32))}


def ncodec_last_error(ctx=None) -> str:
    return (load_library().ncodec_last_error(ctx) or b"").decode()


def ncodec_status_string(st: int) -> str:
    return load_library().ncodec_status_string(st).decode()


def ncodec_destroy(ctx) -> None:
    load_library().ncodec_destroy(ctx)


def _capacity(n: int) -> int:
    """Worst-case container bytes for n symbols (the ABI's bound)."""
    ns = (n + 8191) // 8192
    return 20 + 4 * ((ns + 1) // 2) + ns * (128 + 2 * 8192) * 2


# ---------------------------------------------------------------- convenience
class Codec:
    """One encoder or decoder context with a torch-allocated workspace.

    Frames are (3, H, W) fp16 CUDA tensors; symbols are (C, H/16, W/16) int16.
    """

    def __init__(self, height, width, channels, n_enc_blocks, n_dec_blocks, path, weights,
                 device="cuda:0", stream=None, block="lrelu", n_fe_blocks=0, n_rg_blocks=0, qp_banks=False,
                 hyperprior=False):
        import torch

        self.torch = torch
        self.cfg = make_config(height, width, channels, n_enc_blocks, n_dec_blocks, path, block, n_fe_blocks,
                               n_rg_blocks, qp_banks, hyperprior)
        self.hyperprior = bool(hyperprior)
        self.device = torch.device(device)
        self.path = self.cfg.path
        nbytes = ncodec_workspace_bytes(self.cfg)
        if nbytes == 0:
            raise NcodecError(NCODEC_ESHAPE, "invalid configuration")
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            self.ctx = ncodec_create(self.cfg, weights, self.workspace.data_ptr(), nbytes, self.stream.cuda_stream)
        H, W, C = height, width, channels
        self.frame_shape = (3, H, W)
        # the frame's symbols: y (C x H/16 x W/16), then, with the two-step
        # entropy model, z (64 x H/32 x W/32), as one flat array
        self.y_shape = (C, H // 16, W // 16)
        self.z_shape = (64, H // 32, W // 32)
        self.q_shape = (ncodec_symbol_count(self.cfg),) if self.hyperprior else self.y_shape
        self.feat_shape = (C, H // 8, W // 8)
        self.state_dtype = torch.int16 if self.path == NCODEC_PATH_INT16 else torch.float16

    def _empty(self, shape, dtype):
        return self.torch.empty(shape, dtype=dtype, device=self.device)

    def encode(self, frame, q_out=None, bits_out=None, want_bits=True):
        torch = self.torch
        assert frame.dtype == torch.float16 and tuple(frame.shape) == self.frame_shape and frame.is_contiguous()
        q = q_out if q_out is not None else self._empty(self.q_shape, torch.int16)
        bits = bits_out if bits_out is not None else (self._empty((), torch.float64) if want_bits else None)
        ncodec_encode_frame(self.ctx, frame.data_ptr(), q.data_ptr(), bits.data_ptr() if bits is not None else 0)
        return q, bits

    def decode(self, q, out=None):
        torch = self.torch
        assert q.dtype == torch.int16 and tuple(q.shape) == self.q_shape and q.is_contiguous()
        odt = torch.int16 if self.path == NCODEC_PATH_INT16 else torch.float16
        x = out if out is not None else self._empty(self.frame_shape, odt)
        ncodec_decode_frame(self.ctx, q.data_ptr(), x.data_ptr())
        return x

    def estimate_bits(self, q, scale, bits_out=None):
        """Bits of q under scales `scale`: float32 sigma on an fp16 context, the
        prior's int16 scale outputs s_i on an int16 context."""
        torch = self.torch
        sdt = torch.int16 if self.path == NCODEC_PATH_INT16 else torch.float32
        assert q.dtype == torch.int16 and scale.dtype == sdt and q.numel() == scale.numel()
        assert q.is_contiguous() and scale.is_contiguous()
        bits = bits_out if bits_out is not None else self._empty((), torch.float64)
        ncodec_estimate_bits(self.ctx, q.data_ptr(), scale.data_ptr(), q.numel(), bits.data_ptr())
        return bits

    # ---- entropy coding
    def stream_capacity(self) -> int:
        return ncodec_stream_capacity(self.cfg)

    def scale_indices(self, out=None):
        k = out if out is not None else self._empty(self.q_shape, self.torch.uint8)
        ncodec_scale_indices(self.ctx, k.data_ptr())
        return k

    def rans_encode(self, q, k, stream=None, nbytes_out=None):
        """Container of the symbols q under scale indices k (flattened): returns
        (stream buffer, device byte count)."""
        torch = self.torch
        assert q.dtype == torch.int16 and k.dtype == torch.uint8 and q.numel() == k.numel()
        assert q.is_contiguous() and k.is_contiguous()
        n = q.numel()
        cap = _capacity(n)
        buf = stream if stream is not None else self._empty((cap,), torch.uint8)
        nb = nbytes_out if nbytes_out is not None else self._empty((), torch.int64)
        ncodec_rans_encode(self.ctx, q.data_ptr(), k.data_ptr(), n, buf.data_ptr(), buf.numel(), nb.data_ptr())
        return buf, nb

    def rans_decode(self, stream, nbytes, k, out=None, status_out=None):
        torch = self.torch
        assert stream.dtype == torch.uint8 and k.dtype == torch.uint8 and k.is_contiguous()
        q = out if out is not None else self._empty(tuple(k.shape), torch.int16)
        st = status_out if status_out is not None else self._empty((), torch.int32)
        ncodec_rans_decode(self.ctx, stream.data_ptr(), int(nbytes), k.data_ptr(), k.numel(), q.data_ptr(),
                           st.data_ptr())
        return q, st

    def encode_coded(self, frame, stream=None, nbytes_out=None, q_out=None, bits_out=None):
        torch = self.torch
        assert frame.dtype == torch.float16 and tuple(frame.shape) == self.frame_shape and frame.is_contiguous()
        buf = stream if stream is not None else self._empty((self.stream_capacity(),), torch.uint8)
        nb = nbytes_out if nbytes_out is not None else self._empty((3,) if self.hyperprior else (), torch.int64)
        ncodec_encode_frame_coded(self.ctx, frame.data_ptr(), q_out.data_ptr() if q_out is not None else 0,
                                  bits_out.data_ptr() if bits_out is not None else 0, buf.data_ptr(), buf.numel(),
                                  nb.data_ptr())
        return buf, nb

    def decode_coded(self, stream, nbytes, out=None, status_out=None):
        torch = self.torch
        odt = torch.int16 if self.path == NCODEC_PATH_INT16 else torch.float16
        x = out if out is not None else self._empty(self.frame_shape, odt)
        st = status_out if status_out is not None else self._empty((3,) if self.hyperprior else (), torch.int32)
        ncodec_decode_frame_coded(self.ctx, stream.data_ptr(), int(nbytes), x.data_ptr(), st.data_ptr())
        return x, st

    def get_state(self):
        feat = self._empty(self.feat_shape, self.state_dtype)
        yhat = self._empty(self.y_shape, self.state_dtype)
        ncodec_get_state(self.ctx, feat.data_ptr(), yhat.data_ptr())
        return feat, yhat

    def set_state(self, feat, yhat):
        assert feat.dtype == self.state_dtype and yhat.dtype == self.state_dtype
        assert feat.is_contiguous() and yhat.is_contiguous()
        ncodec_set_state(self.ctx, feat.data_ptr(), yhat.data_ptr())

    def reset(self):
        ncodec_reset(self.ctx)

    def set_qp(self, qp: int):
        ncodec_set_qp(self.ctx, qp)

    def set_rate(self, qp: float):
        ncodec_set_rate(self.ctx, qp)

    def parallel_coding(self, enable: bool):
        ncodec_parallel_coding(self.ctx, enable)

    def kernels_per_frame(self, decode=False):
        return ncodec_kernels_per_frame(self.ctx, decode)

    def timing(self, enable: bool):
        ncodec_timing_enable(self.ctx, enable)

    def graphs(self, enable: bool):
        ncodec_graph_enable(self.ctx, enable)

    def block_chains(self, enable: bool):
        ncodec_block_chains(self.ctx, enable)

    def block_chain_status(self) -> tuple:
        return ncodec_block_chain_status(self.ctx)

    def timing_read(self) -> dict:
        return ncodec_timing_read(self.ctx)

    def close(self):
        if getattr(self, "ctx", None):
            ncodec_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
