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


def test_stream_probes_move_their_bytes():
    """The HBM ceiling probes: the read writes its sink, the copy copies, and
    the write fills every 16-byte slot with its index; bad arguments are
    rejected."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    n = 1 << 20   # 8 MiB of int64
    src = torch.arange(n, dtype=torch.int64, device="cuda:0")
    dst = torch.full((n,), -1, dtype=torch.int64, device="cuda:0")
    sink = torch.full((64,), -1, dtype=torch.int64, device="cuda:0")
    assert fiona.stream_read(src, 64, sink) == n * 8
    assert fiona.stream_copy(src, dst, 64) == 2 * n * 8
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    assert fiona.stream_write(dst, 64) == n * 8
    torch.cuda.synchronize()
    w = dst.view(torch.int32).view(-1, 4).cpu()
    slots = torch.arange(n // 2, dtype=torch.int64)
    assert torch.equal(w[:, 1].to(torch.int64) & 0xFFFFFFFF, slots) and int(w[:, 2].abs().sum()) == 0
    with pytest.raises(fiona.FionaError) as e:
        fiona.stream_write(dst[1:n - 1], 64)   # 8-byte offset: not 16-byte aligned
    assert e.value.status == -4
