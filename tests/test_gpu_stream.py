"""The streaming diagnostic dsm_test_stream: a pure read (a word is written
only for a 1024-element piece whose XOR of 32-bit patterns matches the given
pattern) and a pure write (a fill with the given bit pattern), the access
shape of the optimizer kernels without their arithmetic.  Checked against
numpy on the host: every word, every written element, and that nothing past
the range is touched."""
import numpy as np
import pytest
import torch

from paper_2411_17866_amd import dsm

pytestmark = pytest.mark.gpu

P = dsm.DSM_PIECE_ELEMS
GUARD = 4096           # floats of sentinel after the range
OFFSET = 64            # the range starts 256 bytes into the allocation
SENTINEL = 0x7A7A7A7A


def stream():
    return torch.cuda.current_stream().cuda_stream


def host_xor(buf, n_pieces):
    host = buf.cpu().numpy().view(np.uint32)[OFFSET:OFFSET + n_pieces * P]
    if n_pieces == 0:
        return np.zeros(0, dtype=np.uint32)
    return np.bitwise_xor.reduce(host.reshape(n_pieces, P), axis=1)


@pytest.mark.parametrize("n_pieces", [1, 7, 8, 43, 1000, 8 * 300 + 5])
def test_stream_read_marks_exactly_the_matching_pieces(n_pieces):
    gen = torch.Generator(device="cuda").manual_seed(1000 + n_pieces)
    buf = torch.randn(OFFSET + n_pieces * P + GUARD, generator=gen, device="cuda")
    # Make a few pieces share one checksum: copies of piece 0.
    for k in range(3, n_pieces, 5):
        buf[OFFSET + k * P:OFFSET + (k + 1) * P] = buf[OFFSET:OFFSET + P]
    xor = host_xor(buf, n_pieces)
    for pattern in (int(xor[0]), int(xor[-1]), int(xor[n_pieces // 2])):
        words = torch.full((n_pieces + 1,), SENTINEL, dtype=torch.int32, device="cuda")
        dsm.dsm_test_stream(dsm.DSM_STREAM_READ, buf.data_ptr() + 4 * OFFSET, n_pieces * P,
                            words.data_ptr(), pattern, stream())
        torch.cuda.synchronize()
        got = words.cpu().numpy().view(np.uint32)
        want = np.where(xor == pattern, np.uint32(1), np.uint32(SENTINEL))
        np.testing.assert_array_equal(got[:n_pieces], want)
        assert got[n_pieces] == SENTINEL, "word past the last piece was written"


@pytest.mark.parametrize("n_pieces", [0, 1, 9, 8 * 300 + 5])
def test_stream_read_without_a_match_writes_nothing(n_pieces):
    buf = torch.full((OFFSET + n_pieces * P + GUARD,), 1.25, device="cuda")
    words = torch.full((n_pieces + 1,), SENTINEL, dtype=torch.int32, device="cuda")
    # 1024 equal floats XOR to 0, so any non-zero pattern matches no piece.
    dsm.dsm_test_stream(dsm.DSM_STREAM_READ, buf.data_ptr() + 4 * OFFSET, n_pieces * P,
                        words.data_ptr(), 0x5A5A5A5A, stream())
    torch.cuda.synchronize()
    assert (words.cpu().numpy().view(np.uint32) == SENTINEL).all()


@pytest.mark.parametrize("n_pieces,pattern", [(0, 0x3F800000), (1, 0x80000000), (9, 0x40500000),
                                              (1000, 0x0DA24260), (8 * 300 + 5, 0x7F800000),
                                              (17, 0x7FC01234)])
def test_stream_write_fills_only_the_range(n_pieces, pattern):
    buf = torch.full((OFFSET + n_pieces * P + GUARD,), 7.5, device="cuda")
    dsm.dsm_test_stream(dsm.DSM_STREAM_WRITE, buf.data_ptr() + 4 * OFFSET, n_pieces * P,
                        None, pattern, stream())
    torch.cuda.synchronize()
    host = buf.cpu().numpy()
    bits = host.view(np.uint32)
    assert (bits[OFFSET:OFFSET + n_pieces * P] == pattern).all()
    assert (host[:OFFSET] == 7.5).all() and (host[OFFSET + n_pieces * P:] == 7.5).all()


def test_stream_read_after_write_round_trips():
    n_pieces = 8 * 64 + 3
    buf = torch.empty(n_pieces * P, device="cuda")
    words = torch.zeros(n_pieces, dtype=torch.int32, device="cuda")
    dsm.dsm_test_stream(dsm.DSM_STREAM_WRITE, buf.data_ptr(), buf.numel(), None, 0x40000000,
                        stream())
    # An even count of equal words XORs to zero: every piece matches pattern 0.
    dsm.dsm_test_stream(dsm.DSM_STREAM_READ, buf.data_ptr(), buf.numel(), words.data_ptr(), 0,
                        stream())
    torch.cuda.synchronize()
    assert (words == 1).all()


def test_stream_at_the_largest_grid():
    """2^24 - 1 pieces (64 GiB), the most one grid dimension takes: 64-bit
    addressing to the last piece, written then read back."""
    n_pieces = (1 << 24) - 1
    buf = torch.empty(n_pieces * P + 64, device="cuda")
    buf[-64:] = 9.0
    words = torch.zeros(n_pieces + 1, dtype=torch.int32, device="cuda")
    try:
        dsm.dsm_test_stream(dsm.DSM_STREAM_WRITE, buf.data_ptr(), n_pieces * P, None, 0x3FC00000,
                            stream())
        # 1024 equal floats XOR to 0: pattern 0 marks every piece.
        dsm.dsm_test_stream(dsm.DSM_STREAM_READ, buf.data_ptr(), n_pieces * P, words.data_ptr(), 0,
                            stream())
        torch.cuda.synchronize()
        assert int(words[:n_pieces].sum()) == n_pieces and int(words[n_pieces]) == 0
        assert float(buf[0]) == 1.5 and float(buf[n_pieces * P - 1]) == 1.5
        assert (buf[-64:] == 9.0).all(), "wrote past the last piece"
    finally:
        del buf, words
        torch.cuda.empty_cache()
