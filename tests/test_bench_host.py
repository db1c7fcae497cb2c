"""Host-side pieces of bench.py that need no GPU: the least-squares fit of peak HBM against
S, and the lookup of a recorded HBM-traffic measurement, which applies only while the hash
of the kernel's sources and compile flags matches the one recorded."""
import os

import bench


def test_linear_fit_exact_line():
    xs = [8192, 16384, 32768, 65536]
    ys = [3.5e9 + 246252.0 * x for x in xs]
    a, b, r2 = bench.linear_fit(xs, ys)
    assert abs(a - 3.5e9) < 1e-3 * 3.5e9 and abs(b - 246252.0) < 1e-6 * 246252.0 and r2 > 1 - 1e-12


def test_linear_fit_noisy_line():
    xs = [1.0, 2.0, 3.0, 4.0]
    ys = [1.0, 2.1, 2.9, 4.0]
    a, b, r2 = bench.linear_fit(xs, ys)
    assert abs(b - 0.98) < 1e-12 and abs(a - 0.05) < 1e-12 and 0.99 < r2 < 1.0


def test_source_hash_is_stable_and_path_free():
    h1 = bench.source_hash("attn.bwd_dkdv")
    h2 = bench.source_hash("attn.bwd_dkdv")
    assert h1 == h2 and len(h1) == 16
    assert bench.source_hash("gemm.ffn1") is None          # no traffic record kept for GEMMs
    assert len({bench.source_hash(c) for c in bench.TRAFFIC_SOURCES}) == len(bench.TRAFFIC_SOURCES)


def test_recorded_traffic_applies_only_to_matching_hash(tmp_path, monkeypatch):
    h = bench.source_hash("attn.fwd")
    rec = tmp_path / "record.md"
    rec.write_text("| class | workload | source hash | fetch bytes | write bytes | total bytes |\n"
                   "|---|---|---|---|---|---|\n"
                   f"| attn.fwd | bf16_7b_s32768 | {h} | 100 | 20 | 120 |\n"
                   "| attn.bwd_dq | bf16_7b_s32768 | 0123456789abcdef | 1 | 1 | 2 |\n")
    monkeypatch.setattr(bench, "TRAFFIC_RECORD", str(rec))
    assert bench.recorded_traffic("attn.fwd", "bf16_7b_s32768") == 120
    assert bench.recorded_traffic("attn.fwd", "bf16_13b_s65536") is None      # other workload
    assert bench.recorded_traffic("attn.bwd_dq", "bf16_7b_s32768") is None    # stale hash
    assert bench.recorded_traffic("gemm.qkv", "bf16_7b_s32768") is None       # no record kept
    monkeypatch.setattr(bench, "TRAFFIC_RECORD", os.path.join(str(tmp_path), "missing.md"))
    assert bench.recorded_traffic("attn.fwd", "bf16_7b_s32768") is None


def test_peak_hbm_fit_uses_lengths_with_full_groups():
    pts = [{"S": S, "group_rows": min(S, 16384), "peak_hbm_bytes": (1e9 if S < 16384 else 5e9) + 2.5e5 * S}
           for S in (8192, 16384, 32768, 65536)]
    fit = bench.peak_hbm_fit(pts)
    assert fit["lengths"] == [16384, 32768, 65536]
    assert abs(fit["bytes_per_token"] - 2.5e5) < 1e-3 and abs(fit["intercept_bytes"] - 5e9) < 1.0
    one = bench.peak_hbm_fit([{"S": 524288, "group_rows": 16384, "peak_hbm_bytes": 1.3e11}])
    assert one["bytes_per_token"] is None and one["lengths"] == [524288]
