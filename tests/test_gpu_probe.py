"""libpsc_probe.so on the device: every workgroup's chain of dependent loads
ends at the row the same chain reaches on the host, its stores cover exactly
the 16 KiB of `out` it owns, and nothing past the grid's share is written."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_03065_amd import probe  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _last_row(tab, n_rows, wg, seed, k, mode):
    x = ((wg * 2654435761 + seed * 40503) & 0xFFFFFFFF) % n_rows
    for i in range(k):
        row = tab[x * 256:(x + 1) * 256].astype(np.int64)
        if mode == probe.WAVE_LOAD:
            lane = (i * 5) & 63
            v = row[4 * lane] ^ row[4 * lane + 1] ^ row[4 * lane + 2] ^ row[4 * lane + 3]
        else:
            v = row[2 * (i & 63)] ^ row[2 * (i & 63) + 1]
        x = abs(int(np.int32(v))) % n_rows      # the magnitude of the 32-bit value, modulo n_rows
    return x


@pytest.mark.parametrize("mode", [probe.WAVE_LOAD, probe.SCALAR_LOAD])
def test_chase_reaches_the_host_chain_and_stores_its_share(mode):
    gx, gy, n_rows, k, seed = 3, 5, 37, 11, 1234
    rng = np.random.default_rng(7 + mode)
    tab_h = rng.integers(-2**31, 2**31, size=n_rows * 256, dtype=np.int64).astype(np.int32)
    tab = torch.from_numpy(tab_h).to(DEV)
    share = gx * gy * 16384
    out = torch.zeros(share + 4096, dtype=torch.uint8, device=DEV)
    out[share:] = 0xA5
    stream = torch.cuda.Stream(device=DEV)
    probe.chase(mode, out, tab, n_rows, k, 1, (gx, gy), seed, stream)
    torch.cuda.synchronize()
    words = out[:share].cpu().numpy().view(np.uint32).reshape(gx * gy, 4, 256, 4)   # [wg][wave][vector][word]
    assert (out[share:].cpu().numpy() == 0xA5).all()
    for wg in range(gx * gy):
        last = _last_row(tab_h, n_rows, wg, seed, k, mode)
        w = words[wg]
        assert (w[..., :3] == 0xFF80FF80).all()
        assert (w[..., 3] == (0xFF800000 | last)).all(), (wg, last, hex(int(w[0, 0, 3])))


def test_chase_without_stores_leaves_out_alone():
    tab = torch.zeros(4 * 256, dtype=torch.int32, device=DEV)
    out = torch.full((2 * 16384,), 0x5A, dtype=torch.uint8, device=DEV)
    stream = torch.cuda.Stream(device=DEV)
    probe.chase(probe.WAVE_LOAD, out, tab, 4, 3, 0, (2, 1), 0, stream)
    torch.cuda.synchronize()
    assert (out.cpu().numpy() == 0x5A).all()
