"""Pin the FLOP model used for MFMA utilisation to the paper's printed FLOPs.

Tables 1 and 2 print the per-image FLOPs of dense FLUX.1-dev (1024^2) and
FLUX.1-Kontext-dev sampling; 57 blocks x (24 D^2 S + 4 S^2 D) x NFE must
reproduce them to within the share of the non-block layers (embedders, final
layer), which the model leaves out.
"""
import json
import os

import pytest

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_flops.json")


def _cases():
    return json.load(open(GOLDEN))["cases"]


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c["source"])
def test_block_flop_model_matches_paper(case):
    model = bench.dense_model_flops(case["tokens"]) * case["nfe"] / 1e12
    assert abs(model - case["tflops"]) / case["tflops"] < 5e-3, (model, case["tflops"])
    assert model <= case["tflops"]  # the model omits the non-block layers


def test_block_flops_split():
    f = bench.block_flops(1741, 3072)
    assert f["gemm"] == 24 * 3072 ** 2 * 1741
    assert f["attention"] == 4 * 1741 ** 2 * 3072
    assert abs(f["total"] / 1e9 - 431.57) < 0.01
    assert bench.dense_model_flops(4608, blocks=1) == f["total"] - f["gemm"] - f["attention"] + \
        24 * 3072 ** 2 * 4608 + 4 * 4608 ** 2 * 3072


def test_stage_bytes_flux_1024():
    from synth import configs as C
    b = bench.stage_bytes(C.FLUX_1024)
    assert abs(b["score"] / 1e6 - 79.1) < 0.1
    assert abs(b["gather_upsample"] / 1e6 - 56.0) < 0.1   # 45.3 MB of relayout + the block's first stage (10.7 MB)
    assert b["select"] == 0            # N = 4096: the selection runs inside the scoring call
    assert b["scatter"] == 0           # the scatter is the last projection's second store


def test_gemm_compulsory_bytes():
    # both streams' weights (2 x 36864 x 3072 bf16) plus each activation read or written once
    b = bench.gemm_min_bytes(1741, 3072, 12288)
    weights = 2 * 2 * (3 + 1 + 4 + 4) * 3072 * 3072
    acts = 2 * 1741 * ((4 + 3 + 1 + 2) * 3072 + 2 * 12288)   # QKV, O, MLP in, MLP out
    assert b == weights + acts
    assert abs(b / 4 / 1e6 - 161.38) < 0.01


def test_traffic_record_tracks_gemm_sources(monkeypatch, tmp_path):
    rec = bench.measured_traffic()
    if rec is not None:   # recorded for exactly the current GEMM sources
        assert rec["sources_sha256"] == bench.gemm_sources_sha256() and rec["bytes_per_launch"] > 0
    stale = tmp_path / "t.md"
    stale.write_text('traffic_json: {"sources_sha256": "0", "bytes_per_launch": 1}\n')
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(stale))
    assert bench.measured_traffic() is None
