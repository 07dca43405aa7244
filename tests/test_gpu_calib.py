"""The measurement kernels read exactly the bytes they are given: every 16-byte
chunk once (the XOR of the per-workgroup checksum words equals the XOR of all
32-bit words of the buffer), and for the contiguous patterns each word covers
its own region."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
S = pytest.importorskip("paper_2606_15453_amd.stmoe")

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
REGION = {1: 256 << 10, 2: 32 << 10}


@pytest.mark.parametrize("pattern", [0, 1, 2])
@pytest.mark.parametrize("nbytes", [16, 32 << 10, (32 << 10) + 16, (3 << 20) + 48, 9 << 20])
def test_calib_read_checksums(pattern, nbytes):
    rng = np.random.default_rng(nbytes + pattern)
    host = rng.integers(0, 256, nbytes, dtype=np.uint8)
    src = torch.from_numpy(host).to(DEV)
    n_out = S.calib_read_out_words(nbytes, pattern)
    out = torch.full((n_out,), -1, dtype=torch.int32, device=DEV)
    S.calib_read(src, nbytes, out, pattern=pattern)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32)
    words = host.view(np.uint32)
    assert np.bitwise_xor.reduce(got) == np.bitwise_xor.reduce(words)
    if pattern in REGION:
        r = REGION[pattern] // 4
        assert n_out == -(-nbytes // REGION[pattern])
        for w in range(n_out):
            assert got[w] == np.bitwise_xor.reduce(words[w * r:(w + 1) * r]), w


@pytest.mark.parametrize("workgroups", [1, 3, 64, 1024])
@pytest.mark.parametrize("nbytes", [16, (1 << 20) + 48, 9 << 20])
def test_calib_copy_grid_copies_every_byte(workgroups, nbytes):
    rng = np.random.default_rng(workgroups + nbytes)
    src = torch.from_numpy(rng.integers(0, 256, nbytes, dtype=np.uint8)).to(DEV)
    dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device=DEV)
    S.calib_copy_grid(src.data_ptr(), dst.data_ptr(), nbytes, workgroups)
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src)
    assert int(dst[nbytes:].sum()) == 0          # nothing written past the end
