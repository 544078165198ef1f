"""The context-free, allocation-free rate estimate (ncodec_estimate_bits_noalloc),
called through the C ABI, against ncodec_estimate_bits on an fp16 context: the
same kernels and summation order, so the totals must be equal bit for bit; and
against the oracle's rate (Supp. B.2) to 1e-5.  Two calls in a row, the second
with fewer symbols, on the library's static per-GPU scratch."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2502_20762_amd import ncodec as nc
from paper_2502_20762_amd.ncodec import Codec

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def say(*a):
    print("[gpu-noalloc]", *a, flush=True)


def test_noalloc_rate_matches_context_entry_point():
    lib = nc.load_library()
    flat = synth.make_weights(64, 1, 1)
    c = Codec(16, 16, 64, 1, 1, "fp16", flat, device=DEV)
    stream = torch.cuda.current_stream().cuda_stream
    rng = np.random.default_rng(21)
    for n in (2088960, 4099, 0):
        say("noalloc estimate_bits n =", n)
        q = rng.integers(-40, 41, size=n).astype(np.int16)
        sg = rng.uniform(0.11, 30.0, size=n).astype(np.float32)
        dq, ds = torch.from_numpy(q).to(DEV), torch.from_numpy(sg).to(DEV)
        out = torch.full((2,), -1.0, dtype=torch.float64, device=DEV)
        st = lib.ncodec_estimate_bits_noalloc(ctypes.c_void_p(dq.data_ptr()), ctypes.c_void_p(ds.data_ptr()),
                                              n, ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stream))
        assert st == nc.NCODEC_OK, nc.ncodec_last_error(None)
        ref_ctx = c.estimate_bits(dq, ds)
        torch.cuda.synchronize()
        got = float(out[0].cpu())
        assert float(out[1].cpu()) == -1.0  # nothing written past the output
        assert got == float(ref_ctx.cpu()), (n, got, float(ref_ctx.cpu()))
        ref = oracle.estimate_bits(q, sg.astype(np.float64))
        assert abs(got - ref) <= 1e-5 * max(ref, 1e-30), (n, got, ref)


def test_noalloc_rejects_bad_arguments():
    lib = nc.load_library()
    d = torch.zeros(4, dtype=torch.float64, device=DEV)
    p = ctypes.c_void_p(d.data_ptr())
    assert lib.ncodec_estimate_bits_noalloc(p, p, 1 << 31, p, None) == nc.NCODEC_EINVAL
    assert "2^31" in nc.ncodec_last_error(None)
    assert lib.ncodec_estimate_bits_noalloc(p, p, -1, p, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_estimate_bits_noalloc(p, p, 4, None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_estimate_bits_noalloc(None, None, 4, p, None) == nc.NCODEC_EINVAL
