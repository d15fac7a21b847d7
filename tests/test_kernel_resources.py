"""Register-allocation contract of the built kernels (our own gfx950 code objects, read with
the ROCm LLVM tools on the CPU): no kernel spills registers to scratch memory, except the
instantiations listed in ALLOWED, which are measured, documented and not on any automatic
path's hot loop.  A compiler or source change that starts spilling in a hot kernel (a slow
and easily missed regression: results stay correct) fails here before any GPU run.
"""
import pytest

from _codeobj import kernel_resources, template_args

SOURCES = ["prefill_bf16.hip", "decode_bf16.hip", "f32.hip", "fold.hip", "mla.hip", "baseline.hip"]

# Epilogue kinds (csrc/fn_device.h).
EPI_REGLU, EPI_BILINEAR, EPI_RELU_DEFER = 5, 6, 8


def allowed(source, args, fields):
    """True for the known spilling instantiations of the prefill kernel.  Template arguments:
    BM, BN, WM, WN, STAGES, PF, EPI, SPREAD, GS, KCHK, KD."""
    if source != "prefill_bf16.hip" or len(args) != 11:
        return False
    bm, bn, wm, wn, stages, pf, epi, spread, gs, kchk, kd = args
    if (bm, bn, wm, wn) != (256, 256, 2, 4):
        return False
    if stages == 5 or not pf:
        return True  # forced tuning tiles (5-stage ring, no register prefetch); never chosen automatically
    # The automatic 256 x 256 tile of three epilogue-family kinds with the lane-checked
    # activation transfers (K not a multiple of 64) keeps one value in scratch across the
    # k loop (stored once before it, reloaded after it).
    return epi in (EPI_REGLU, EPI_BILINEAR, EPI_RELU_DEFER) and kchk == 1 and fields["vgpr_spill_count"] <= 1


@pytest.mark.parametrize("source", SOURCES)
def test_no_unexpected_spills(source, tmp_path):
    res = kernel_resources(source, tmp_path)
    assert res, "no kernels found"
    bad = []
    for name, f in res.items():
        spills = f.get("private_segment_fixed_size", 0) or f.get("vgpr_spill_count", 0) or f.get("sgpr_spill_count", 0)
        if spills and not allowed(source, template_args(name), f):
            bad.append((name, f.get("private_segment_fixed_size"), f.get("vgpr_spill_count"), f.get("sgpr_spill_count")))
    assert not bad, bad


def test_hot_prefill_kernels_hold_everything_in_registers(tmp_path):
    # The 256 x 256 tiles of the large-shape workloads (8 waves: RMS kinds and LayerNorm, lean
    # and lane-checked; 4 waves with the asm k blocks: RMS, SwiGLU and the plain GEMM) and the
    # 128-row tiles with 64-deep steps.
    res = {tuple(template_args(n)): f for n, f in kernel_resources("prefill_bf16.hip", tmp_path).items()}
    hot = [(256, 256, 2, 4, 4, 1, epi, 1, 0, kchk, 1) for epi in (0, 1, 2) for kchk in (0, 1)]
    hot += [(256, 256, 2, 2, 4, 1, epi, 0, 0, 0, 1) for epi in (0, 1, 3)]  # 4 waves, hand-scheduled k blocks
    hot += [(128, 96, 4, 2, 4, 1, 0, 0, 0, kchk, 2) for kchk in (0, 1)]
    for h in hot:
        assert h in res, h
        assert res[h]["private_segment_fixed_size"] == 0 and res[h]["vgpr_spill_count"] == 0, (h, res[h])


def test_checker_parses_template_arguments():
    assert template_args("_ZN2fn19prefill_bf16_kernelILi256ELi256ELi2ELi4ELi4ELb1ELi0ELb1ELb0ELb0ELi1EEEvPKDF16b") == \
        [256, 256, 2, 4, 4, 1, 0, 1, 0, 0, 1]
    assert allowed("prefill_bf16.hip", [256, 256, 2, 4, 5, 1, 0, 0, 0, 1, 1], {"vgpr_spill_count": 3})
    assert not allowed("prefill_bf16.hip", [256, 256, 2, 4, 4, 1, 0, 1, 0, 1, 1], {"vgpr_spill_count": 1})
    assert not allowed("prefill_bf16.hip", [256, 256, 2, 4, 4, 1, EPI_REGLU, 1, 0, 1, 1], {"vgpr_spill_count": 2})


def test_asm_step_include_matches_its_generator():
    # prefill_w4_step.inc is generated; the committed file must be what the generator writes.
    import importlib.util
    import os
    here = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2407_09577_amd", "csrc")
    spec = importlib.util.spec_from_file_location("gen_prefill_w4_step", os.path.join(here, "gen_prefill_w4_step.py"))
    gen = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(gen)
    assert open(os.path.join(here, "prefill_w4_step.inc")).read() == gen.generate()


def test_asm_step_keeps_m0_next_to_its_transfers():
    # In the generated sequence every M0 write is the s_mov right before its LDS-DMA transfer
    # (the contract test_lds_dma_m0 checks on the built code), and the transfers of one
    # block are the eight of the wave, activation fragments first.
    import importlib.util
    import os
    import re
    here = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2407_09577_amd", "csrc")
    spec = importlib.util.spec_from_file_location("gen_prefill_w4_step", os.path.join(here, "gen_prefill_w4_step.py"))
    gen = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(gen)
    for gram in (True, False):
        o = gen.Ops(gram, True)
        ins = gen.body(o, 0, gram, True).split("\\n\\t")
        movs = [k for k, t in enumerate(ins) if "m0" in t.split()[1:2] or t.startswith("s_mov_b32 m0")]
        assert len(movs) == gen.NL
        for k in movs:
            assert ins[k].startswith("s_mov_b32 m0,") and ins[k + 1].startswith("buffer_load_dwordx4") and \
                ins[k + 1].endswith(" lds")
        assert sum(t.startswith("v_mfma") for t in ins) == 64 + (gen.TW if gram else 0)
        assert sum(t.startswith("ds_read_b128") for t in ins) == 16
        assert ins[-1] == "s_waitcnt lgkmcnt(0)"
        rs = [re.search(r", (%\d+), 0 offen lds", t).group(1) for t in ins if t.endswith(" lds")]
        assert rs[:gen.NA] == [o["rsa"]] * gen.NA and rs[gen.NA:] == [o["rsw"]] * (gen.NL - gen.NA)
