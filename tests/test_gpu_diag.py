"""The streaming-read probe reads every word exactly once: the workgroup partial sums add up
to the sum of the buffer (small integers, so every fp32 sum is exact)."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_floats,n_parts", [(4, 1), (1 << 20, 64), ((1 << 20) + 12, 2048),
                                              (4096 * 3 + 8, 7), (64, 4096)])
def test_read_probe_covers_the_buffer_once(n_floats, n_parts):
    from paper_2608_05448_amd import dblast as D
    print(f"[diag] read probe {n_floats} floats, {n_parts} workgroups", flush=True)
    g = torch.Generator().manual_seed(n_floats)
    buf = torch.randint(0, 4, (n_floats,), generator=g).to(torch.float32).cuda()
    parts = torch.full((n_parts,), float("nan"), dtype=torch.float32, device="cuda")
    D.dbl_stream_read_probe(buf, parts)
    torch.cuda.synchronize()
    assert torch.isfinite(parts).all().item()
    assert parts.double().sum().item() == buf.double().sum().item()
