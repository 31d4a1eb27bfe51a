"""Host-side checks of libmapl that need no GPU: the library loads, exports
every entry point include/mapl.h declares, and rejects bad arguments before
enqueuing anything.  Pointers below are fake and are never dereferenced:
validation runs first and fails."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_05484_amd import mapl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mapl.h")
FAKE = 0x7f0000000000  # 256-aligned, never dereferenced


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(mapl_\w+)\s*\(", src, re.M)))


def test_exports_every_declared_symbol():
    L = mapl.lib()
    declared = _declared()
    assert set(declared) == set(mapl.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name
    assert L.mapl_version() == 2


def test_desc_layout_matches_header():
    # five int64 then seven int32: 5*8 + 7*4 = 68 bytes, padded to 72 (int64 alignment)
    assert ctypes.sizeof(mapl.CodecDesc) == 72


def _enc(D, **kw):
    args = dict(X=FAKE, ids=FAKE + 0x10000000, U=FAKE + 0x20000000, A_s=FAKE + 0x30000000,
                B_s=FAKE + 0x40000000, C=FAKE + 0x50000000, payload=FAKE + 0x60000000,
                ws=FAKE + 0x70000000, ws_bytes=1 << 40)
    args.update(kw)
    return mapl.lib().mapl_encode(ctypes.byref(D), args["X"], args["ids"], args["U"], args["A_s"], args["B_s"],
                                  args["C"], args["payload"], args["ws"], args["ws_bytes"], None)


@pytest.mark.parametrize("field,value,status", [
    ("d", 100, -2), ("d", 32, -2), ("r", 48, -2), ("r", 2048, -2), ("k", 8, -2), ("L", 9, -2),
    ("K", 100, -2), ("x_dtype", 7, -3), ("ab_dtype", 0, -3), ("anchor_space", 5, -2), ("T", -1, -2),
])
def test_encode_rejects_bad_descriptors(field, value, status):
    D = mapl.desc(T=64, d=256, r=64, V=100, k=16, L=2, K=64)
    setattr(D, field, value)
    assert _enc(D) == status
    assert mapl.last_error() != ""


def test_code_dtype_too_small_is_range_error():
    D = mapl.desc(T=64, d=256, r=64, V=100, k=16, L=2, K=1024, code_dtype="u8")
    assert _enc(D) == -4


def test_rvq_above_r256_on_bf16_unsupported():
    D = mapl.desc(T=64, d=1024, r=512, V=100, k=16, L=1, K=64)
    assert _enc(D) == -8


@pytest.mark.parametrize("L", [0, 2])
def test_bf16_rank_not_multiple_of_64_unsupported(L):
    """The bf16 GEMM and weight-gradient tiles need r % 64 == 0; r = 32 and
    r = 96 are refused up front (the fp32 path takes r = 32)."""
    for r in (32, 96):
        D = mapl.desc(T=64, d=256, r=r, V=100, k=16, L=L, K=64)
        assert _enc(D) == -8
        assert "r % 64" in mapl.last_error()


def test_null_and_alignment_and_alias_and_workspace():
    D = mapl.desc(T=64, d=256, r=64, V=100, k=16, L=0)
    assert _enc(D, X=None) == -1
    assert _enc(D, U=FAKE + 0x20000004) == -5
    # payload [64,64] bf16 overlapping X
    assert _enc(D, payload=FAKE + 64) == -6
    assert _enc(D, ws=None, ws_bytes=0) == -7
    assert _enc(D, ws_bytes=16) == -7
    assert _enc(D, ws=FAKE + 0x70000010) == -5
    # no anchor: ids/A_s/B_s may be NULL
    D0 = mapl.desc(T=64, d=256, r=64, V=0, k=0, L=0)
    need = mapl.workspace_bytes(D0, mapl.CALL_ENCODE)
    assert need > 0
    assert _enc(D0, ids=None, A_s=None, B_s=None, ws_bytes=need - 1) == -7


def test_workspace_bytes_monotone_and_errors():
    a = mapl.workspace_bytes(mapl.desc(T=1024, d=1024, r=128, V=32000, k=16, L=4, K=256), mapl.CALL_ENCODE)
    b = mapl.workspace_bytes(mapl.desc(T=8192, d=1024, r=128, V=32000, k=16, L=4, K=256), mapl.CALL_ENCODE)
    assert 0 < a < b
    with pytest.raises(mapl.MaplError):
        mapl.workspace_bytes(mapl.desc(T=8, d=100, r=64), mapl.CALL_ENCODE)
    s = mapl.workspace_bytes(None, mapl.CALL_STIEFEL, 16, 2048, 512)
    assert s >= 2 * 16 * 2048 * 512 * 4


def test_stiefel_rejects_bad_arguments():
    L = mapl.lib()
    f = lambda **kw: L.mapl_stiefel_step(kw.get("P", 2), kw.get("d", 256), kw.get("r", 32), kw.get("U", FAKE),
                                         kw.get("G", FAKE + 0x10000000), kw.get("M", FAKE + 0x20000000),
                                         kw.get("lr", 1e-2), kw.get("beta", 0.95), kw.get("lmo", 5),
                                         kw.get("ret", 7), kw.get("ws", FAKE + 0x30000000),
                                         kw.get("wsb", 1 << 40), None)
    assert f(r=48) == -2
    assert f(r=512, d=256) == -2
    assert f(lmo=0) == -2 and f(ret=17) == -2
    assert f(beta=1.0) == -4 and f(lr=-1.0) == -4
    assert f(M=FAKE + 64) == -6      # M overlaps U
    assert f(G=None) == -1
    assert f(wsb=100) == -7


def test_payload_bytes_against_paper(tmp_path):
    """Fig. 1 caption and Table 1: a bf16 payload of rank r costs 2r bytes per
    token (64 -> 128 ... 512 -> 1024); the uncompressed boundary 2d bytes."""
    import json
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "paper_bytes_per_token.json")))
    for row in g["mapl_bf16"]:
        D = mapl.desc(T=1, d=2048, r=row["r"], L=0)
        assert mapl.payload_bytes_per_token(D) == row["bytes"]
    for row in g["uncompressed_bf16"]:
        D = mapl.desc(T=1, d=row["d"], r=row["d"] if row["d"] <= 1024 else 1024, L=0)
        assert 2 * row["d"] == row["bytes"]
    # the paper's VQ setting (Table 1's MAPL+VQ rows, App. E): 256 bytes per token
    for row in g["mapl_vq"]:
        D = mapl.desc(T=1, d=row["d"], r=row["r"], L=row["R"], K=row["K"], group_dim=row["group_dim"])
        assert mapl.payload_bytes_per_token(D) == row["bytes"]
    # the build's RVQ payloads: L stages of u8 / u16 codes
    assert mapl.payload_bytes_per_token(mapl.desc(T=1, d=1024, r=128, L=4, K=256)) == 4
    assert mapl.payload_bytes_per_token(mapl.desc(T=1, d=2048, r=256, L=2, K=1024)) == 4


def test_polar_table_matches_oracle_schedule():
    """The library's PolarExpress table (its own LP + Newton generator) equals
    the oracle's Remez-derived greedy schedule."""
    from oracle import polar_schedule as ps
    src = open(os.path.join(ROOT, "paper_2606_05484_amd", "csrc", "polar_coeffs.h")).read()
    for name, lo in (("kLmoCoef", 1e-3), ("kRetractCoef", 0.5)):
        blk = src[src.index(name + "["):]
        blk = blk[:blk.index("};")]
        rows = np.array([[float(v) for v in r.split(",") if v.strip()] for r in re.findall(r"\{([^{}]*)\}", blk)])
        ref = np.array(ps.greedy_schedule(lo, rows.shape[0])[0])
        assert np.abs(rows - ref).max() <= 1e-12 * np.abs(ref).max()


def test_noalloc_rejects_requests_beyond_its_scratch():
    """mapl_encode_noalloc refuses, before touching any pointer or device,
    a request whose workspace exceeds the static scratch (here the fp32 Z0 of
    2^22 tokens at r = 128: 2 GiB)."""
    D = mapl.desc(T=1 << 22, d=1024, r=128, V=100, k=16, L=2, K=256)
    assert mapl.workspace_bytes(D, mapl.CALL_ENCODE) > mapl.NOALLOC_SCRATCH_BYTES
    with pytest.raises(mapl.MaplError) as e:
        mapl.encode_noalloc(D, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, stream=0)
    assert e.value.status == -7 and "scratch" in str(e.value)
