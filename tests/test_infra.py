"""CPU checks of the test and bench infrastructure: the oracle's process pool (used by the full-size
GPU parity samples) gives the same unit results as a direct oracle call, and the bench reports the
counter-measured HBM traffic only while the decode sources match the ones it was measured on."""

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

import oracle  # noqa: E402


def test_oracle_pool_matches_direct_units():
    """Margins and Eq. 5 head terms of prefill units evaluated on the pool's memory-mapped copies equal the
    direct oracle's; a planted error in one unit's output shows up as a positive margin of that unit only."""
    from oracle_pool import OraclePool
    rng = np.random.default_rng(5)
    B, N, C, Lq, Lm, H, d = 2, 3, 20, 4, 3, 2, 16
    r = lambda *s: rng.standard_normal(s).astype(np.float32)
    x = {"q_pre": r(B, N, C + 1, H, d), "k_pre": r(B, N, C + 1, H, d), "v_pre": r(B, N, C + 1, H, d),
         "q_qm": r(B, Lq + Lm, H, d), "k_qm": r(B, Lq + Lm, H, d), "v_qm": r(B, Lq + Lm, H, d)}
    Sc = 1 + C + Lq + Lm
    o = np.zeros((B, N, Sc, H, d), dtype=np.float32)
    want = {}
    for b in range(B):
        for n in range(N):
            for h in range(H):
                u = oracle.prefill_unit_ref(*(x[k].astype(np.float64) for k in
                                              ("q_pre", "k_pre", "v_pre", "q_qm", "k_qm", "v_qm")), b, n, h, Lq)
                o[b, n, :, h] = u["o"]
                want[(b, n, h)] = u["e_head"]
    o[1, 2, 5, 1, 3] += 0.5   # planted error in unit (1, 2, 1)
    units = [(b, n, h) for b in range(B) for n in range(N) for h in range(H)]
    with OraclePool({**x, "o": o}) as pool:
        res = pool.prefill_units(units, Lq, 1e-2, 0.0)
    for b, n, h, margin, e_head in res:
        np.testing.assert_allclose(e_head, want[(b, n, h)], rtol=1e-12, atol=1e-12)
        if (b, n, h) == (1, 2, 1):
            assert abs(margin - (0.5 - 1e-2)) < 1e-5, margin
        else:
            assert margin <= 0, (b, n, h, margin)


def test_traffic_reported_only_for_the_measured_sources(tmp_path, monkeypatch):
    import bench
    src = tmp_path / "kernel.hip"
    src.write_text("// decode kernel, version 1\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCES", [str(src)])
    summary = tmp_path / "traffic.md"
    summary.write_text("# counters\n\nkernel_source_sha256: %s\ntraffic_bytes_per_launch: 286195760\n"
                       % bench.kernel_source_digest())
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(summary))
    assert bench.measured_traffic() == 286195760
    src.write_text("// decode kernel, version 2\n")
    assert bench.measured_traffic() is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "absent.md"))
    assert bench.measured_traffic() is None

