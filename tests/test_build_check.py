"""The build's kernel-resource check (no GPU needed): it must flag scratch,
vector register spills and an FFN kernel held to one wave a SIMD, and let
scalar spills and other kernels' occupancy pass."""
from paper_2607_00466_amd import build


def _remarks(name, scratch=0, vspill=0, sspill=0, occ=2):
    return "\n".join(f"x.hip:1:1: remark: {k}: {v} [-Rpass-analysis=kernel-resource-usage]" for k, v in [
        ("Function Name", name), ("VGPRs", 100), ("ScratchSize [bytes/lane]", scratch),
        ("Occupancy [waves/SIMD]", occ), ("SGPRs Spill", sspill), ("VGPRs Spill", vspill)])


def test_clean_kernels_pass():
    err = _remarks("_ZN4eldr10ffn_kernelILi0E", sspill=27) + "\n" + _remarks("_ZN4eldr14combine_kernelE", occ=1)
    assert build._resource_problems(err) == []


def test_scratch_spills_and_low_ffn_occupancy_fail():
    assert build._resource_problems(_remarks("_ZN4eldr10ffn_kernelILi1E", scratch=208))
    assert build._resource_problems(_remarks("_ZN4eldr13gate_kernelE", vspill=4))
    p = build._resource_problems(_remarks("_ZN4eldr16ffn_fused_kernelILi4E", occ=1))
    assert p and "occupancy 1" in p[0]
