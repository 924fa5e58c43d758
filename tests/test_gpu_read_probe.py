"""The read-ceiling probe reads every byte of both buffers once: its
per-thread sums add up to the buffers' sum (small integers, so exactly)."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("na,nb,grid", [(1 << 20, 3 << 18, 256), (4, 0, 7), (12, 1000, 3)])
def test_read_probe_reads_everything_once(cuda_device, na, nb, grid):
    from paper_2607_19456_amd import hbm_probe
    g = torch.Generator(device=cuda_device)
    g.manual_seed(5)
    a = torch.randint(0, 4, (na,), generator=g, device=cuda_device).float()
    b = torch.randint(0, 4, (nb,), generator=g, device=cuda_device).float()
    partial = hbm_probe.read(a, b, grid=grid)
    torch.cuda.synchronize()
    assert partial.numel() == grid * hbm_probe.THREADS
    total = float(partial.double().sum())
    assert total == float(a.double().sum() + b.double().sum())
