"""The HBM read-bandwidth probe through the C ABI: it launches, reads the whole buffer without
writing anything (its sink stays untouched for a buffer whose words fold to zero), and refuses a
misaligned buffer on the device path too."""
import pytest

torch = pytest.importorskip("torch")

from paper_2609_24298_amd import kvc

pytestmark = pytest.mark.gpu


def test_read_probe_runs_and_leaves_sink():
    buf = torch.zeros(64 << 20, dtype=torch.uint8, device="cuda:0")
    sink = torch.full((1,), 7, dtype=torch.int32, device="cuda:0")
    kvc.kvc_read_probe(buf, sink)
    kvc.kvc_read_probe(buf[: 16 * 1000 + 16], sink)  # ragged grid: fewer words than one block per CU
    torch.cuda.synchronize()
    assert sink.item() == 7
    with pytest.raises(kvc.KvcError):
        kvc.kvc_read_probe(buf[8:8 + 1024], sink)
