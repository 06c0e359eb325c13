"""The measurement aids of include/saf_measure.h on the GPU: they run to
completion through the C ABI, report a plausible shader clock, and leave
their sinks untouched (the sinks are written only under conditions the
probes never meet)."""

import pytest

from gpu_helpers import announce, torch_cuda

pytestmark = pytest.mark.gpu


def test_lds_pattern_probe_every_pattern():
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    sink = torch.zeros(65536, dtype=torch.int32, device="cuda")
    for pat in range(len(binding.LDS_PATTERNS)):
        announce(f"lds pattern probe {pat}")
        binding.saf_lds_pattern_probe(pat, 16, sink)
    torch.cuda.synchronize()
    assert not sink.any()


@pytest.mark.parametrize("shape,waves", [(0, 1), (0, 2), (1, 1), (1, 2)])
def test_mfma_rate_probe(shape, waves):
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    announce(f"mfma rate probe shape {shape} waves {waves}")
    clk = torch.zeros(2, dtype=torch.int64, device="cuda")
    sink = torch.zeros(16384, dtype=torch.float32, device="cuda")
    binding.saf_mfma_rate_probe(shape, waves, 64, clk, sink)
    torch.cuda.synchronize()
    cycles, ticks = clk.cpu().tolist()
    assert cycles > 0 and ticks > 0
    assert 100.0 < cycles / ticks * 100.0 < 3000.0  # MHz
    assert not sink.any()


def test_clock_probe():
    torch = torch_cuda()
    from paper_2609_34650_amd import binding
    announce("clock probe")
    out = torch.zeros(2, dtype=torch.int64, device="cuda")
    binding.saf_clock_probe(out, 2000)
    torch.cuda.synchronize()
    cycles, ticks = out.cpu().tolist()
    assert ticks >= 200000  # 2 ms of the 100 MHz reference clock
    assert 100.0 < cycles / ticks * 100.0 < 3000.0
