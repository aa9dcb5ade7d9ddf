"""The library's measurement helpers on the GPU: the read-stream kernel reads every word
once (the XOR of its per-workgroup words equals the XOR of the buffer), the empty
launch runs for the fused grid's shape, and the chains of dependencies between two
streams complete in every mode."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "no GPU visible"
    import paper_2606_30389_amd  # noqa: F401  (fails loudly when libprr.so is missing)
    return _t


@pytest.mark.parametrize("words,grid", [(4, 1), (4 * 1000 + 4, 3), (4 * 256 * 8 * 5 + 12, 5), (1 << 20, 64)])
def test_read_stream_reads_every_word_once(torch, words, grid):
    from paper_2606_30389_amd import _lib as L
    rng = np.random.default_rng(words + grid)
    host = rng.integers(0, 2**32, size=words, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.full((grid,), -1, dtype=torch.int32, device="cuda")
    L.prr_read_stream(buf, words * 4, sink, grid, torch.cuda.current_stream())
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


def test_read_stream_rejects_bad_sizes(torch):
    from paper_2606_30389_amd import _lib as L
    buf = torch.zeros(64, dtype=torch.int32, device="cuda")
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    for nbytes, grid in ((0, 1), (20, 1), (256, 0)):
        with pytest.raises(L.PrrError):
            L.prr_read_stream(buf, nbytes, sink, grid)


def test_empty_launch_of_the_fused_grid(torch):
    from paper_2606_30389_amd import _lib as L
    L.prr_empty_launch(356, 512, torch.cuda.current_stream())
    torch.cuda.synchronize()
    with pytest.raises(L.PrrError):
        L.prr_empty_launch(0, 512)


@pytest.mark.parametrize("mode", [0, 1, 2])
def test_stream_chain_completes(torch, mode):
    from paper_2606_30389_amd import _lib as L
    s, p2 = torch.cuda.current_stream(), torch.cuda.Stream()
    for n in (2, 40, 256):  # (repeated calls reuse the events and the growing stream-memory values)
        L.prr_stream_chain(n, mode, s, p2)
    torch.cuda.synchronize()
