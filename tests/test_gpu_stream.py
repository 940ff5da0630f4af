"""The streaming diagnostic dsm_test_stream: a pure read (one XOR word per
1024-element piece) and a pure write (a fill), the access shape of the
optimizer kernels without their arithmetic.  Checked against numpy on the
host: every word, every written element, and that nothing past the range is
touched."""
import numpy as np
import pytest
import torch

from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

P = dsm.DSM_PIECE_ELEMS
GUARD = 4096           # floats of sentinel after the range
OFFSET = 64            # the range starts 256 bytes into the allocation


def stream():
    return torch.cuda.current_stream().cuda_stream


@pytest.mark.parametrize("n_pieces", [0, 1, 7, 8, 43, 1000, 8 * 300 + 5])
def test_stream_read_words_match_host_xor(n_pieces):
    gen = torch.Generator(device="cuda").manual_seed(1000 + n_pieces)
    buf = torch.randn(OFFSET + n_pieces * P + GUARD, generator=gen, device="cuda")
    words = torch.full((n_pieces + 1,), 0x7A7A7A7A, dtype=torch.int32, device="cuda")
    dsm.dsm_test_stream(dsm.DSM_STREAM_READ, buf.data_ptr() + 4 * OFFSET, n_pieces * P,
                        words.data_ptr(), 0.0, stream())
    torch.cuda.synchronize()
    host = buf.cpu().numpy().view(np.uint32)[OFFSET:OFFSET + n_pieces * P]
    want = np.bitwise_xor.reduce(host.reshape(n_pieces, P), axis=1) if n_pieces else \
        np.zeros(0, dtype=np.uint32)
    got = words.cpu().numpy().view(np.uint32)
    np.testing.assert_array_equal(got[:n_pieces], want)
    assert got[n_pieces] == 0x7A7A7A7A, "word past the last piece was written"


@pytest.mark.parametrize("n_pieces,value", [(0, 1.0), (1, -0.0), (9, 3.25), (1000, 1e-30),
                                            (8 * 300 + 5, float("inf"))])
def test_stream_write_fills_only_the_range(n_pieces, value):
    buf = torch.full((OFFSET + n_pieces * P + GUARD,), 7.5, device="cuda")
    dsm.dsm_test_stream(dsm.DSM_STREAM_WRITE, buf.data_ptr() + 4 * OFFSET, n_pieces * P,
                        None, value, stream())
    torch.cuda.synchronize()
    host = buf.cpu().numpy()
    bits = host.view(np.uint32)
    want_bits = np.array([value], dtype=np.float32).view(np.uint32)[0]
    assert (bits[OFFSET:OFFSET + n_pieces * P] == want_bits).all()
    assert (host[:OFFSET] == 7.5).all() and (host[OFFSET + n_pieces * P:] == 7.5).all()


def test_stream_read_after_write_round_trips():
    n_pieces = 8 * 64 + 3
    buf = torch.empty(n_pieces * P, device="cuda")
    words = torch.empty(n_pieces, dtype=torch.int32, device="cuda")
    dsm.dsm_test_stream(dsm.DSM_STREAM_WRITE, buf.data_ptr(), buf.numel(), None, 2.0, stream())
    dsm.dsm_test_stream(dsm.DSM_STREAM_READ, buf.data_ptr(), buf.numel(), words.data_ptr(), 0.0,
                        stream())
    torch.cuda.synchronize()
    # An even count of equal words XORs to zero.
    assert not words.any()
