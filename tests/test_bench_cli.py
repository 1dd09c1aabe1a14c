"""Host-side checks of bench.py's workload grammar (no GPU): each spec builds the workload it
names, with its block shape, density, token count and dtype, and specs a workload cannot honour
are refused instead of silently measuring something else."""
import pytest

import bench


def _shape(wl):
    p = wl.projections[0]
    return p.R, p.C, p.W.shape


def test_fused_qkv_spec():
    wl = bench.build_workload("fused_qkv:16x16:0.2:bf16")
    assert wl.bf16 and wl.tokens == 4096
    assert _shape(wl) == (16, 16, (2304, 768))
    assert wl.projections[0].density == pytest.approx(0.2)


def test_ffn_spec_density_tokens_dtype():
    wl = bench.build_workload("ffn:32x1:0.05:256")
    assert not wl.bf16 and wl.tokens == 256
    assert [p.W.shape for p in wl.projections] == [(3072, 768), (768, 3072)]
    assert all(p.density == pytest.approx(0.05) for p in wl.projections)
    assert bench.build_workload("ffn:32x32:bf16").bf16


def test_reblock_spec():
    wl = bench.build_workload("sweep:64x64@32x32")
    assert wl.notes["reblock"] == (32, 32)
    assert _shape(wl)[:2] == (64, 64)


@pytest.mark.parametrize("spec", ["sweep:32x1:bf16", "bert_large:32x32:bf16", "nonsense:32x1"])
def test_refused_specs(spec):
    with pytest.raises(SystemExit):
        bench.build_workload(spec)
