"""CPU oracle for the DCVC-RT single-scale conditional transform.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with
the HIP library (``paper_2502_20762_amd``) and never imports it.

It is a plain, slow, obviously-correct NumPy float64 program written from the
paper (Jia et al., "Towards Practical Real-Time Neural Video Compression",
CVPR 2025):

* ``codec_float``  -- the floating-point transform (Sec. 4.1-4.3, Fig. 4).
* ``codec_int``    -- the integerised transform (Sec. 4.5, Eq. 3; Supp. B.4,
                      Alg. 1).
* ``bits``         -- the Gaussian likelihood / bit estimate.
* ``entropy``      -- the coder: quantised-scale Gaussian tables and
                      interleaved rANS streams (Fig. 4 "AE"/"AD", Fig. 6).
* ``hyperprior``   -- the two-step entropy model with the hyper latent z
                      (Sec. 4.4; supplementary "Entropy model").
* ``params``       -- its own reading of the canonical flat parameter list.

Parity status of each function is stated in its docstring; every function is
pinned by ``tests/test_oracle_*.py`` against closed forms, brute force or
library routines (none is "parity unpinned").
"""
from . import bits, codec_float, codec_int, entropy, hyperprior, ops, params  # noqa: F401
from .bits import estimate_bits, likelihood, sigma_from_s  # noqa: F401
from .params import Params, unpack  # noqa: F401
