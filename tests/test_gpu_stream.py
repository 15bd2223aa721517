"""The streaming probe (smol_stream_probe) on the GPU: every granule of the
written buffer is written, in every read/write mix, load/store form and wave
count the benchmark uses, including ragged sizes whose last wave ends
mid-step; pure reads write nothing. The VALU probe (smol_valu_probe) times
every wave of a launch, for every instruction kind."""
from __future__ import annotations

import pytest

from paper_2007_13005_amd import smol
from tests.gpu_util import note

pytestmark = pytest.mark.gpu

SENTINEL = 0xAB


@pytest.mark.parametrize("read_bytes, write_bytes", [
    (0, 16 * 1000), (16 * 777, 16 * 131), (1 << 20, 1 << 20), (92_735_232, 19_267_584),
    (16 * 3, 16 * 5000), (16 * 70_001, 16)])
@pytest.mark.parametrize("flags", [0, 1, 3, 5, 7])
@pytest.mark.parametrize("waves", [1, 7, 2048])
def test_probe_writes_every_granule(read_bytes, write_bytes, flags, waves):
    import torch
    note(f"stream probe r={read_bytes} w={write_bytes} flags={flags} waves={waves}")
    src = torch.ones(max(read_bytes, 16), dtype=torch.uint8, device="cuda:0")
    dst = torch.full((write_bytes + 64,), SENTINEL, dtype=torch.uint8, device="cuda:0")
    smol.stream_probe(src.data_ptr() if read_bytes else 0, read_bytes, dst.data_ptr(),
                      write_bytes, waves, flags, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    g = dst[:write_bytes].view(-1, 16)
    untouched = (g == SENTINEL).all(dim=1)
    assert not bool(untouched.any()), int(untouched.sum())
    # nothing past the buffer
    assert bool((dst[write_bytes:] == SENTINEL).all())


def test_pure_read_writes_nothing():
    import torch
    src = torch.ones(1 << 20, dtype=torch.uint8, device="cuda:0")
    dst = torch.full((4096,), SENTINEL, dtype=torch.uint8, device="cuda:0")
    smol.stream_probe(src.data_ptr(), 1 << 20, dst.data_ptr(), 0, 512, 3,
                      torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert bool((dst == SENTINEL).all())


@pytest.mark.parametrize("kind", range(len(smol.VALU_KINDS)))
def test_valu_probe_times_every_wave(kind):
    import torch
    note(f"valu probe kind={kind}")
    ticks = torch.zeros(2048, dtype=torch.int64, device="cuda:0")
    smol.valu_probe(kind, 2048, 64, ticks.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert bool((ticks > 0).all())
