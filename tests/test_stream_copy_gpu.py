"""The HBM reference copy (muon_stream_copy): exact bytes, a ragged tail,
and the argument checks."""
import pytest

from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


@pytest.mark.parametrize("nbytes", [16, 4096 * 16 + 16, (16384 * 16) * 3 + 48, 1000003])
def test_stream_copy_is_exact(muon, nbytes):
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(nbytes)
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda", generator=g)
    dst = torch.zeros_like(src)
    muon.stream_copy(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)


def test_stream_copy_refuses_overlap_and_misalignment(muon):
    import torch
    from paper_2609_21594_amd.binding import MuonError
    buf = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(MuonError, match="overlap"):
        muon.stream_copy(buf[1024:33792], buf[0:32768])
    with pytest.raises(MuonError, match="aligned"):
        muon.stream_copy(buf[40000:40100], buf[1:101])
