"""e2s_read_probe, the benchmark's streaming-read measurement helper: it reads its
buffer and writes nothing (its sink only when the XOR of all words equals a fixed
value, which these inputs avoid)."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
pytest.importorskip("paper_2608_23253_amd")
from paper_2608_23253_amd import _lib as L  # noqa: E402


@pytest.mark.parametrize("nbytes,wgs", [(16, 1), (4096, 7), (1 << 22, 512), ((1 << 20) + 48, 1000)])
def test_read_probe_reads_and_writes_nothing(nbytes, wgs):
    buf = torch.full((nbytes // 4,), 0x01010101, device="cuda", dtype=torch.int32)
    guard = buf.clone()
    sink = torch.zeros(1, device="cuda", dtype=torch.int32)
    L.read_probe(buf, wgs, sink)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
    assert torch.equal(buf, guard)
