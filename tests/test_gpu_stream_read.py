"""ppas_stream_read, the streaming read that measures the device's HBM read ceiling:
its output is the XOR of every 16-byte word of the buffer, so the test checks that
every word was read exactly once (a word read twice or skipped changes the XOR for
almost every buffer) against NumPy on the host."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
ppas = pytest.importorskip("paper_2608_15171_amd.ppas", reason="libppas.so not built")


def xor_words(host: np.ndarray) -> np.ndarray:
    return np.bitwise_xor.reduce(host.view(np.uint32).reshape(-1, 4), axis=0)


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, 1 << 20, (64 << 20) + 16 * 12345, 300 << 20])
def test_xor_of_every_word(nbytes):
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 2 ** 32, size=nbytes // 4, dtype=np.uint32).view(np.uint8)
    buf = torch.from_numpy(host).cuda()
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    ppas.stream_read(buf, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, xor_words(host))


def test_xor_accumulates_into_the_sink_and_a_second_pass_cancels():
    host = np.random.default_rng(1).integers(0, 2 ** 32, size=(8 << 20) // 4, dtype=np.uint32).view(np.uint8)
    buf = torch.from_numpy(host).cuda()
    seed = np.array([0x12345678, 0x9ABCDEF0, 0x0F0F0F0F, 0xFFFFFFFF], dtype=np.uint32)
    sink = torch.from_numpy(seed.view(np.int32).copy()).cuda()
    ppas.stream_read(buf, sink)
    torch.cuda.synchronize()
    assert np.array_equal(sink.cpu().numpy().view(np.uint32), seed ^ xor_words(host))
    ppas.stream_read(buf, sink)
    torch.cuda.synchronize()
    assert np.array_equal(sink.cpu().numpy().view(np.uint32), seed)


def test_a_view_at_an_offset_reads_only_its_words():
    host = np.random.default_rng(2).integers(0, 2 ** 32, size=(1 << 20) // 4, dtype=np.uint32).view(np.uint8)
    buf = torch.from_numpy(host).cuda()
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    ppas.stream_read(buf[4096:4096 + 16 * 1000], sink)
    torch.cuda.synchronize()
    assert np.array_equal(sink.cpu().numpy().view(np.uint32), xor_words(host[4096:4096 + 16 * 1000]))


def test_refusals():
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    buf = torch.zeros(64, dtype=torch.uint8, device="cuda")
    with pytest.raises(ppas.PPASError):
        ppas.stream_read(buf[:24], sink)            # not whole 16-byte words
    with pytest.raises(ppas.PPASError):
        ppas.stream_read(buf[8:24], sink)           # misaligned start
    with pytest.raises(ValueError):
        ppas.stream_read(buf, torch.zeros(2, dtype=torch.int32, device="cuda"))
