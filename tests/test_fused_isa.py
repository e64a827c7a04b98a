"""The fused top-1 kernel's counted waits against its built ISA (CPU only).

The kernel waits for its inline-assembly loads with hand-counted vmcnt
values; the compiler does not see those loads.  Two properties of the built
code keep those counts valid, and both are checked here on the gfx950
assembly of the three translation units that instantiate the kernel:
  * no instruction touches a register that an inline load is still filling
    (every control-flow path from the load to a covering wait);
  * the register allocation is the validated one: the spill slots (the
    hidden-split variant with five [t|u] tiles keeps two values in scratch,
    outside its hidden loop) are exactly those of the build that was run on
    the GPU.  A source change that moves a spill into the hand-scheduled
    loop puts a scratch access among the counted loads; it showed as wrong
    results at 129 tokens, D = 384, H = 3072, so any change of these figures
    needs a new GPU validation before the table below is updated.
"""
import os
import re

import pytest

import isa_check


# (translation unit, NFT, split) -> (spilled registers, private bytes)
VALIDATED = {("fused.hip", n, 0): (0, 0) for n in range(1, 6)}
VALIDATED.update({("fused_split.hip", n, 1): (0, 0) for n in range(1, 5)})
VALIDATED[("fused_split.hip", 5, 1)] = (2, 12)
# the variants with the class rows' workgroups (k_fused_top1_cls; "split"
# 2 marks them): the same body after a branch on the workgroup index
VALIDATED.update({("fused_cls.hip", n, 2): (0, 0) for n in range(1, 6)})


@pytest.fixture(scope="module")
def asm():
    """The device assembly the library build kept for the translation
    units (built from the sources in the tree)."""
    from paper_2606_28516_amd import build as hb
    out = {}
    for src in hb.KEEP_ASM:
        path = hb.device_asm(src)
        if not os.path.exists(path) or not os.path.exists(path + ".digest"):
            pytest.skip("no kept assembly: run the library build first")
        if open(path + ".digest").read().strip() != hb.source_digest():
            pytest.skip("kept assembly is older than the sources: run the library build first")
        out[src] = open(path).read()
    return out


def _meta(text, name):
    md = text[text.index("amdhsa.kernels:"):]
    for ent in md.split("\n  - ")[1:]:
        if re.search(rf"\.name:\s+{re.escape(name)}\s", ent):
            get = lambda k: int(re.search(k + r":\s+(\d+)", ent).group(1))  # noqa: E731
            return get(r"\.vgpr_spill_count"), get(r"\.private_segment_fixed_size")
    raise KeyError(name)


@pytest.mark.parametrize("src,nft,split", sorted(VALIDATED))
def test_fused_kernel_isa(asm, src, nft, split):
    if split == 2:
        name = f"_ZN8clearmoe12_GLOBAL__N_116k_fused_top1_clsILi{nft}EEEvNS_9FusedArgsENS_9ClassArgsE"
    else:
        name = f"_ZN8clearmoe12_GLOBAL__N_112k_fused_top1ILi{nft}ELb{split}EEEvNS_9FusedArgsE"
    text = asm[src]
    assert _meta(text, name) == VALIDATED[(src, nft, split)], _meta(text, name)
    insts, labels = isa_check.kernel_body(text, name)
    loads, found = isa_check.hazards(insts, labels)
    reg = [f for f in found if "registers touched" in f]
    assert loads > 0
    assert not reg, reg[:3]
