"""The streaming-read ceiling kernel (dv_stream_read): it reads every byte it is given,
whole 1 KB slots and the chunks after the last one, and writes nothing."""
import pytest
import torch

from paper_2310_17157_amd import binding as Bd

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 1008, 1024, 1024 * 1024 + 48, 64 << 20])
def test_stream_read_sizes_leave_the_sink_untouched(nbytes):
    buf = torch.randint(0, 255, (nbytes,), dtype=torch.uint8, device="cuda")
    sink = torch.full((1,), 1.5, dtype=torch.float32, device="cuda")
    Bd.dv_stream_read(buf, sink, nbytes)
    torch.cuda.synchronize()
    assert sink.item() == 1.5


def test_stream_read_rejects_a_partial_chunk():
    buf = torch.zeros(64, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    with pytest.raises(Exception):
        Bd.dv_stream_read(buf, sink, 40)
