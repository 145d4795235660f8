"""The plain-read calibration kernel (sf_read_xor) against numpy's XOR
reduction of the same 64-bit words, piece by piece: empty and one-word
buffers, odd word counts (the lone tail word), sizes around the 256 KB piece,
a buffer of thousands of pieces, byte tensors and a side stream."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
CHUNK = 256 * 1024


@pytest.fixture(scope="module")
def sf():
    from paper_2606_06751_amd import stagefrontier
    return stagefrontier


def host_pieces(words: np.ndarray) -> np.ndarray:
    """XOR of each CHUNK-byte piece of the words, as uint64."""
    w = words.view(np.uint64)
    per = CHUNK // 8
    return np.array([np.bitwise_xor.reduce(w[i:i + per]) for i in range(0, w.size, per)],
                    dtype=np.uint64)


def as_u64(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint64)


@pytest.mark.parametrize("nbytes", [0, 8, 16, 24, 4088, 4096, CHUNK - 8, CHUNK, CHUNK + 8,
                                    3 * CHUNK + 24, 4 << 20, (4 << 20) + 8])
def test_read_xor_sizes(sf, nbytes):
    rng = np.random.Generator(np.random.PCG64(nbytes))
    words = rng.integers(0, np.iinfo(np.int64).max, size=nbytes // 8, dtype=np.int64)
    words ^= rng.integers(0, 2, size=words.size, dtype=np.int64) << 63   # set the top bit too
    print("case nbytes=%d" % nbytes, flush=True)
    x = torch.from_numpy(words).to(DEV)
    out = sf.sf_read_xor(x)
    assert out.shape == (sf.sf_read_xor_pieces(nbytes),)
    np.testing.assert_array_equal(as_u64(out), host_pieces(words))


def test_read_xor_many_pieces(sf):
    """Thousands of pieces, the last one partial with a lone tail word; the
    XOR of all words equals the XOR of the whole buffer."""
    n = (300 << 20) // 8 + 3
    g = torch.Generator(device=DEV)
    g.manual_seed(7)
    x = torch.randint(-(1 << 62), 1 << 62, (n,), dtype=torch.int64, device=DEV, generator=g)
    out = sf.sf_read_xor(x)
    host = x.cpu().numpy()
    want = np.bitwise_xor.reduce(host.view(np.uint64).reshape(-1)[: (n // (CHUNK // 8)) * (CHUNK // 8)]
                                 .reshape(-1, CHUNK // 8), axis=1)
    got = as_u64(out)
    np.testing.assert_array_equal(got[:want.size], want)
    assert got[-1] == np.bitwise_xor.reduce(host.view(np.uint64)[want.size * (CHUNK // 8):])
    assert np.bitwise_xor.reduce(got) == np.bitwise_xor.reduce(host.view(np.uint64))


def test_read_xor_byte_tensor_and_reuse(sf):
    """A uint8 tensor is read as its little-endian 64-bit words; reused
    result words are overwritten."""
    rng = np.random.Generator(np.random.PCG64(3))
    raw = rng.integers(0, 256, size=5 * CHUNK + 40, dtype=np.uint8)
    x = torch.from_numpy(raw).to(DEV)
    out = torch.full((6,), -1, dtype=torch.int64, device=DEV)
    sf.sf_read_xor(x, out)
    np.testing.assert_array_equal(as_u64(out), host_pieces(raw.view(np.int64)))
    one = out[:1]
    sf.sf_read_xor(x[:16], one)
    np.testing.assert_array_equal(as_u64(one), host_pieces(raw[:16].view(np.int64)))


def test_read_xor_offset_view_and_side_stream(sf):
    rng = np.random.Generator(np.random.PCG64(4))
    words = rng.integers(-(1 << 40), 1 << 40, size=100003, dtype=np.int64)
    x = torch.from_numpy(words).to(DEV)
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        out = sf.sf_read_xor(x[2:], stream=side)     # 16-byte aligned view
    side.synchronize()
    np.testing.assert_array_equal(as_u64(out), host_pieces(words[2:]))
    with pytest.raises(sf.StageFrontierError):
        sf.sf_read_xor(x[1:])                         # 8-byte aligned only: rejected


def test_read_xor_rejects_result_inside_buffer(sf):
    x = torch.zeros(1024, dtype=torch.int64, device=DEV)
    with pytest.raises(sf.StageFrontierError):
        sf.sf_read_xor(x, x[4:5])
    with pytest.raises(ValueError):
        sf.sf_read_xor(x, torch.empty((2,), dtype=torch.int64, device=DEV))   # wrong length
