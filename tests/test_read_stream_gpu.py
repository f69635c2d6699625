"""The plain read used as the streaming-rate reference (graft_read_stream):
every 32-bit word of the buffer is read exactly once (the sink's xor equals
the buffer's), at sizes below one workgroup's share, across the grid cap and
with a ragged tail; bad arguments are rejected."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.mark.parametrize("n_words", [4, 4 * 255, 4 * 1024 * 256 + 4 * 37, 4 * 4096 * 256 * 5 + 4 * 3])
def test_every_word_read_once(n_words):
    import paper_2608_20375_amd as G
    rng = np.random.default_rng(n_words)
    host = rng.integers(0, 2 ** 32, size=n_words, dtype=np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.full((G.READ_STREAM_SINK_WORDS,), -1, dtype=torch.int32, device="cuda")
    G.read_stream(src, sink)
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


def test_argument_errors():
    import paper_2608_20375_amd as G
    buf = torch.zeros(64, dtype=torch.int32, device="cuda")
    with pytest.raises(G.GraftError):
        G.read_stream(torch.zeros(15, dtype=torch.uint8, device="cuda"))    # not a multiple of 16
    with pytest.raises(G.GraftError):
        G.read_stream(buf[1:5])                                               # src not 16-byte aligned
    with pytest.raises(ValueError):
        G.read_stream(buf, torch.zeros(16, dtype=torch.int32, device="cuda"))  # sink too small
