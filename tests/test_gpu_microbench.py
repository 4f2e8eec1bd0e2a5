"""The MAC microbenchmark entry point (a measurement helper): it runs, writes
its sink and reports the words it multiplies; bad arguments are rejected."""
import pytest

import paper_2609_35352_amd as fiona

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def test_mac_microbench_runs():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sink = torch.full((4 * 256,), -1, dtype=torch.int64, device="cuda:0")
    words = fiona.mac_microbench(4, 3, sink)
    torch.cuda.synchronize()
    assert words == 4 * 256 * 3 * 56
    assert int((sink == -1).sum()) < 4   # every thread wrote its word (an xor could be -1 by chance)
    with pytest.raises(fiona.FionaError) as e:
        fiona.mac_microbench(0, 3, sink)
    assert e.value.status == -1
