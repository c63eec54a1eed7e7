"""The measurement kernels (include/pearl_bench.h) through the C ABI (needs an MI355X): the copy
and the fill write exactly their byte range (bit-exact, ragged sizes that end mid-workgroup, a
guard region after the range untouched); the read-only probe leaves its sink alone on random data."""
import numpy as np
import pytest
import torch

from paper_2609_35158_amd import binding as bd
from gpu_helpers import say

pytestmark = pytest.mark.gpu

SIZES = [16, 4096, 16 * 2047, 16 * 2048, 16 * 2049, 16 * 123457, 1 << 24]
GUARD = 4096


@pytest.mark.parametrize("nbytes", SIZES)
def test_copy_and_fill_are_exact(nbytes):
    say("hbm probe copy/fill nbytes=%d" % nbytes)
    g = torch.Generator(device="cpu").manual_seed(nbytes)
    src = torch.randint(0, 256, (nbytes + GUARD,), dtype=torch.uint8, generator=g).cuda()
    dst = torch.full((nbytes + GUARD,), 0xA5, dtype=torch.uint8, device="cuda")
    bd.hbm_copy(src[:nbytes], dst[:nbytes])
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src[:nbytes])
    assert bool((dst[nbytes:] == 0xA5).all())
    bd.hbm_fill(dst[:nbytes], 0x01020304)
    torch.cuda.synchronize()
    words = dst[:nbytes].cpu().numpy().view(np.uint32)
    assert bool((words == 0x01020304).all())
    assert bool((dst[nbytes:] == 0xA5).all())


@pytest.mark.parametrize("nontemporal", [False, True])
def test_read_probe_leaves_sink(nontemporal):
    say("hbm probe read nontemporal=%s" % nontemporal)
    g = torch.Generator(device="cpu").manual_seed(5)
    src = torch.randint(0, 256, (1 << 24,), dtype=torch.uint8, generator=g).cuda()
    sink = torch.zeros(16, dtype=torch.uint8, device="cuda")
    bd.hbm_read(src, sink, nontemporal=nontemporal)
    torch.cuda.synchronize()
    assert bool((sink == 0).all())
