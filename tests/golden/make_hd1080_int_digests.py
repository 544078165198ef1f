"""Write the expected per-frame digests of the integerised 1080p sequence.

Free-running run of the CPU oracle (``oracle.codec_int``) over the 32-frame
1920x1088 workload (C = 256, 8 + 8 DC blocks, the frames of ``synth``), as the
encoder and decoder of a low-delay P-frame codec run it: every frame is coded
from the oracle's own previous state.  For each frame it records the SHA-256
of the symbols q, the new latent state yhat_t, the new context f_t and the
reconstruction xhat (each as planar little-endian int16 bytes), the estimated
bits, and the largest magnitudes of f_t and yhat_t.

Integer results are exact and identical on every device (Sec. 4.5; Supp. B.4,
Alg. 1), so the GPU's free-running sequence must reproduce every digest.

The decoder's context equals the encoder's (both run the same decoder
transform on the same yhat), so xhat is the reconstruction of the encoder's
f_t; frames 0 and 1 are also decoded through ``decode_frame`` as a check.

Calls only ``oracle`` and ``synth``.  Run from the repository root:
    python tests/golden/make_hd1080_int_digests.py
It takes about 40 minutes on 8 CPU cores.
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402
from oracle import codec_int as ci  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "hd1080_int_digests.json")


def digest(a: np.ndarray) -> str:
    a = np.asarray(a)
    assert a.min() >= -32768 and a.max() <= 32767
    return hashlib.sha256(np.ascontiguousarray(a.astype("<i2")).tobytes()).hexdigest()


def main(n_frames: int | None = None) -> None:
    pre = synth.PRESETS["hd1080_int"]
    n = pre.n_frames if n_frames is None else n_frames
    flat = synth.make_weights(pre.channels, pre.n_enc, pre.n_dec)
    ip = ci.integerize(oracle.unpack(flat, pre.channels, pre.n_enc, pre.n_dec))
    st = ci.zero_state(ip, pre.height, pre.width)
    rows = []
    for t, x in enumerate(synth.frame_sequence(pre, n)):
        t0 = time.time()
        r = ci.encode_frame(ip, x, st)
        if t < 2:
            xhat, dst = ci.decode_frame(ip, r.q, st)
            assert np.array_equal(dst.feat, r.state.feat) and np.array_equal(dst.yhat, r.state.yhat)
        else:
            xhat = ci.reconstruct(ip, r.state.feat)
        rows.append({
            "frame": t,
            "q": digest(r.q),
            "yhat": digest(r.state.yhat),
            "feat": digest(r.state.feat),
            "xhat": digest(xhat),
            "bits": r.bits,
            "max_abs_feat": int(np.abs(r.state.feat).max()),
            "max_abs_yhat": int(np.abs(r.state.yhat).max()),
        })
        st = r.state
        print(f"frame {t}: {time.time() - t0:.1f} s, bits {r.bits:.1f}, max|f| {rows[-1]['max_abs_feat']}",
              flush=True)
    doc = {
        "what": "free-running integerised 1080p sequence: per-frame SHA-256 of planar little-endian int16 "
                "q, yhat_t, f_t, xhat; estimated bits; max |f_t|, |yhat_t| (K1 = 512 units)",
        "preset": pre.name, "height": pre.height, "width": pre.width, "channels": pre.channels,
        "n_enc": pre.n_enc, "n_dec": pre.n_dec, "seed_weights": synth.SEED_W, "seed_frames": synth.SEED_X,
        "writer": "tests/golden/make_hd1080_int_digests.py (oracle.codec_int only)",
        "frames": rows,
    }
    with open(OUT, "w") as f:
        json.dump(doc, f, indent=1)
    print("wrote", OUT)


if __name__ == "__main__":
    main(int(sys.argv[1]) if len(sys.argv) > 1 else None)
