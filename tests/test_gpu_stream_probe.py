"""The stream probe (the measurement aid the roofline ceilings come from)
computes what its declaration says, on ragged sizes, and rejects overlapping
arguments (needs an MI355X)."""
import pytest
import torch

from paper_2008_05823_amd import saef

pytestmark = pytest.mark.gpu

N = 3 * 2048 + 37  # several tiles and a ragged tail


def _inputs(n):
    g = torch.Generator().manual_seed(5)
    a = torch.randn(n, generator=g).cuda()
    b = torch.randn(n, generator=g).cuda()
    return a, b


def test_probe_sum():
    print("[case] stream probe c = a + b", flush=True)
    a, b = _inputs(N)
    c = torch.full_like(a, float("nan"))
    saef.saef_stream_probe(a, b, c)
    torch.cuda.synchronize()
    assert torch.equal(c, a + b)


def test_probe_copy_and_in_place():
    print("[case] stream probe copy, in place", flush=True)
    a, _ = _inputs(N)
    keep = a.clone()
    c = torch.full_like(a, float("nan"))
    saef.saef_stream_probe(a, None, c)
    saef.saef_stream_probe(a, None, a)
    torch.cuda.synchronize()
    assert torch.equal(c, keep) and torch.equal(a, keep)


def test_probe_rejects_overlap():
    print("[case] stream probe overlap checks", flush=True)
    buf = torch.zeros(2 * N, device="cuda")
    a, b = buf[:N], torch.zeros(N, device="cuda")
    with pytest.raises(saef.SaefError):
        saef.saef_stream_probe(a, b, buf[1:N + 1])       # c overlaps a
    with pytest.raises(saef.SaefError):
        saef.saef_stream_probe(a, b, a)                  # c is a, with b
    with pytest.raises(saef.SaefError):
        saef.saef_stream_probe(a, None, buf[7:N + 7])    # partial overlap, copy
