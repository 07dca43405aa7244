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


@pytest.mark.parametrize("producers,consumers,chunk1,chunk2", [(64, 32, 4096, 8192), (7, 300, 16 << 10, 24 << 10),
                                                               (260, 5, 48, 32 << 10)])
def test_calib_handoff_modes_agree(producers, consumers, chunk1, chunk2):
    """Every mode gives each consumer the wrapping sum of its own chunk's
    words plus every producer's published word; the in-launch waits end
    without the error word, and the counter advances by the producers of
    every one-launch call."""
    rng = np.random.default_rng(producers + consumers)
    w1h = rng.integers(0, 2 ** 32, producers * chunk1 // 4, dtype=np.uint64).astype(np.uint32)
    w2h = rng.integers(0, 2 ** 32, consumers * chunk2 // 4, dtype=np.uint64).astype(np.uint32)
    w1 = torch.from_numpy(w1h.view(np.int32)).to(DEV)
    w2 = torch.from_numpy(w2h.view(np.int32)).to(DEV)
    act = torch.zeros(producers, dtype=torch.int32, device=DEV)
    sync = torch.zeros(S.HANDOFF_SYNC_WORDS, dtype=torch.int32, device=DEV)
    total = int(w1h.astype(np.uint64).sum() % 2 ** 32)
    want = (w2h.reshape(consumers, -1).astype(np.uint64).sum(axis=1) + total) % 2 ** 32
    target = 0
    for mode in (0, 1, 2, 3, 4, 1, 2, 3, 4, 4):
        out = torch.full((consumers,), -1, dtype=torch.int32, device=DEV)
        if mode:
            target += producers
        S.calib_handoff(w1, chunk1, producers, w2, chunk2, consumers, mode, act, out, sync, target)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().view(np.uint32), want.astype(np.uint32)), mode
        assert int(sync[1].item()) == 0
        assert int(sync[0].item()) == target
