"""Kernel fingerprints read from the built library's code objects
(paper_2506_11209_amd/kernel_code.py), which tie the committed counter
records to the machine code they were measured on."""
import json
import os

import pytest

from paper_2506_11209_amd import kernel_code as kc
from paper_2506_11209_amd.build import MODE_GEMM, instances

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2506_11209_amd", "libwsgemm.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")


def test_every_compiled_gemm_kernel_has_a_fingerprint():
    seen = {}
    for (tm, tn, tk, nc, np_, split, bf16, trace, mode, general) in instances():
        if np_ == 0:
            continue  # the synchronous kernel is another template
        sym = kc.gemm_symbol(tm, tn, tk, nc, np_, split, bool(bf16), bool(trace), mode, bool(general))
        fp = kc.kernel_fingerprint(sym, LIB)
        assert len(fp) == 16
        seen[sym] = fp
    # distinct kernels have distinct code
    assert len(set(seen.values())) == len(seen)


def test_fingerprint_is_repeatable_and_unknown_kernels_raise():
    sym = kc.gemm_symbol(256, 128, 64, 4, 4, 1)
    assert kc.kernel_fingerprint(sym, LIB) == kc.kernel_fingerprint(sym, LIB)
    with pytest.raises(LookupError):
        kc.kernel_fingerprint(kc.gemm_symbol(256, 128, 64, 4, 4, 1, mode=MODE_GEMM + 99), LIB)


def test_traffic_record_matches_only_its_own_kernel(tmp_path, monkeypatch):
    import bench
    point = (256, 128, 64, 3, 4, 4)
    rec = {"point": "256x128x64x3x4x4/registers", "kernel_fingerprint": bench.kernel_fingerprint(point),
           "workload": bench.WORKLOAD, "traffic_bytes_per_launch": 123.0}
    (tmp_path / "x_hbm_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.traffic_for("256x128x64x3x4x4/registers", point) == 123.0
    assert bench.traffic_for("256x128x64x3x4x4/dma", point) is None
    assert bench.traffic_for("256x128x64x3x4x4/registers", point, workload="gemm_4096x4096x4096_bf16_normal") is None
    rec["kernel_fingerprint"] = "0" * 16
    (tmp_path / "x_hbm_traffic.json").write_text(json.dumps(rec))
    assert bench.traffic_for("256x128x64x3x4x4/registers", point) is None
