"""Host-side checks of the C ABI: the library loads, exports every declared
entry point, and validates arguments before touching the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import synth
from paper_2502_20762_amd import ncodec as nc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ncodec.h")


@pytest.fixture(scope="module")
def lib():
    return nc.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ncodec_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(nc._SIGNATURES), "binding and header disagree"


def test_config_struct_matches_header():
    text = open(HEADER).read()
    block = re.search(r"typedef struct \{(.*?)\} ncodec_config;", text, re.S).group(1)
    fields = re.findall(r"int32_t\s+([a-z_]+(?:\s*,\s*[a-z_]+)*)\s*;", block)
    names = [f.strip() for grp in fields for f in grp.split(",")]
    assert names == [f for f, _ in nc.ncodec_config._fields_]


@pytest.mark.parametrize("C,ne,nd", [(64, 2, 2), (128, 6, 6), (256, 8, 8), (64, 0, 0), (384, 2, 2), (512, 8, 8)])
def test_weight_count_matches_oracle(C, ne, nd):
    cfg = nc.make_config(64, 64, C, ne, nd, "fp16")
    assert nc.ncodec_weight_count(cfg) == oracle.params.count(C, ne, nd)
    assert nc.ncodec_weight_count(cfg) == sum(int(np.prod(s)) for _, s, _, _ in synth.param_list(C, ne, nd))


@pytest.mark.parametrize("bad", [
    dict(height=1080), dict(width=8), dict(height=0), dict(width=8208), dict(channels=96), dict(channels=320),
    dict(channels=768), dict(n_enc_blocks=-1), dict(n_dec_blocks=33), dict(path=2), dict(block=2),
])
def test_invalid_configs_rejected(bad):
    kw = dict(height=64, width=64, channels=64, n_enc_blocks=2, n_dec_blocks=2, path=0)
    kw.update(bad)
    cfg = nc.ncodec_config(**kw)
    assert nc.ncodec_weight_count(cfg) == 0
    assert nc.ncodec_workspace_bytes(cfg) == 0
    with pytest.raises(nc.NcodecError) as e:
        nc.ncodec_create(cfg, np.zeros(10, np.float32), 0x10000, 1 << 30)
    assert e.value.status == nc.NCODEC_ESHAPE


def test_wide_configs_accepted_with_block_buffers():
    # above C = 256 a DC block runs as three launches through two extra 1/8-scale buffers
    narrow = nc.ncodec_workspace_bytes(nc.make_config(64, 64, 256, 2, 2, "fp16"))
    wide = nc.ncodec_workspace_bytes(nc.make_config(64, 64, 512, 2, 2, "fp16"))
    # the wide context also holds the depthwise output (C) and the hidden layer (2C) at 1/8 scale
    assert wide > 2 * narrow
    assert nc.ncodec_workspace_bytes(nc.make_config(64, 64, 384, 2, 2, "int16")) > 0


def test_workspace_bytes_grow_with_size():
    a = nc.ncodec_workspace_bytes(nc.make_config(64, 64, 64, 2, 2, "fp16"))
    b = nc.ncodec_workspace_bytes(nc.make_config(1088, 1920, 256, 8, 8, "fp16"))
    c = nc.ncodec_workspace_bytes(nc.make_config(1088, 1920, 256, 8, 8, "int16"))
    assert 0 < a < b and c > 0
    # five 1/8-scale feature maps + three latents dominate at 1080p (plus ~10 MB of weights)
    assert 5 * 32640 * 256 * 2 < b < 5 * 32640 * 256 * 2 + (64 << 20)


FAKE_WS = 0x7F0000000000  # never dereferenced: every case below fails validation first


def create_status(cfg, w, ws=FAKE_WS, nbytes=1 << 40):
    try:
        nc.ncodec_create(cfg, w, ws, nbytes)
    except nc.NcodecError as e:
        return e.status, nc.ncodec_last_error(None)
    return nc.NCODEC_OK, ""


def test_create_argument_validation():
    cfg = nc.make_config(64, 64, 64, 2, 2, "fp16")
    w = synth.make_weights(64, 2, 2)
    assert create_status(cfg, w[:-1])[0] == nc.NCODEC_EINVAL
    assert create_status(cfg, w, ws=0)[0] == nc.NCODEC_EINVAL
    assert create_status(cfg, w, ws=FAKE_WS + 16)[0] == nc.NCODEC_ENOMEM
    st, msg = create_status(cfg, w, nbytes=1024)
    assert st == nc.NCODEC_ENOMEM and "needs" in msg
    bad = w.copy()
    bad[5] = np.nan
    assert create_status(cfg, bad)[0] == nc.NCODEC_EINVAL
    # int path: a pointwise weight whose int16 value exceeds the int8-digit range
    cfgi = nc.make_config(64, 64, 64, 2, 2, "int16")
    big = w.copy()
    big[0] = 3.99   # round(8192 * 3.99) = 32686 > 32639
    st, msg = create_status(cfgi, big)
    assert st == nc.NCODEC_EINVAL and "32639" in msg


def test_null_context_calls(lib):
    assert lib.ncodec_reset(None) == nc.NCODEC_EINVAL
    assert lib.ncodec_encode_frame(None, None, None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_decode_frame(None, None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_estimate_bits(None, None, None, 0, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_get_state(None, None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_kernels_per_frame(None, 0) == 0
    assert lib.ncodec_scale_indices(None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_rans_encode(None, None, None, 1, None, 0, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_rans_decode(None, None, 0, None, 1, None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_encode_frame_coded(None, None, None, None, None, 0, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_decode_frame_coded(None, None, 0, None, None) == nc.NCODEC_EINVAL
    assert lib.ncodec_block_chains(None, 1) == nc.NCODEC_EINVAL
    assert lib.ncodec_block_chain_status(None, None, None) == nc.NCODEC_EINVAL
    lib.ncodec_destroy(None)


def test_stream_capacity_is_the_worst_case_bound():
    # 20-byte header, 2 bytes per stream length (padded to 4), and per stream of
    # 8192 symbols 64 two-word final states plus at most 2 words per symbol (one
    # per sub-symbol: the table entry and, for an escape, the 16-bit field)
    for H, W, C in [(64, 64, 64), (480, 832, 128), (1088, 1920, 256)]:
        n = (H // 16) * (W // 16) * C
        ns = -(-n // 8192)
        want = 20 + 4 * ((ns + 1) // 2) + ns * (128 + 2 * 8192) * 2
        assert nc.ncodec_stream_capacity(nc.make_config(H, W, C, 1, 1, "fp16")) == want
        assert nc._capacity(n) == want
    assert nc.ncodec_stream_capacity(nc.make_config(63, 64, 64, 1, 1, "fp16")) == 0


def test_status_strings():
    for st in range(-6, 1):
        assert nc.ncodec_status_string(st) not in ("", "unknown status")
    assert nc.ncodec_status_string(-42) == "unknown status"
