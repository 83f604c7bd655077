"""Host-side checks of the encode kernels' workgroup-to-tile maps.

The launch grids and the slot -> (latent tile, token tile) maps below are
the ones the encode kernels compute from blockIdx; every tile of the
problem must be visited exactly once and no slot may land outside it."""
import numpy as np
import pytest


def decode_map(n_mt, n_nt, fast_tiles=4, bt_=8, bl_=4):
    """sae_stream_kernel: 256 latents x 128 tokens per tile."""
    if n_nt <= fast_tiles:
        grid = n_mt * n_nt
        for L in range(grid):
            nt, mt = L // n_mt, L % n_mt
            if nt < n_nt:
                yield mt, nt
        return
    m8 = (n_mt + 7) // 8
    nbt = (n_nt + bt_ - 1) // bt_
    nbl = (m8 + bl_ - 1) // bl_
    for L in range(8 * nbt * nbl * bt_ * bl_):
        xcd, slot = L % 8, L // 8
        b, p = slot // (bt_ * bl_), slot % (bt_ * bl_)
        bt, bl = b % nbt, b // nbt
        lt, nt = bl_ * bl + p // bt_, bt_ * bt + p % bt_
        if nt >= n_nt or lt >= m8:
            continue
        mt = xcd * m8 + lt
        if mt < n_mt:
            yield mt, nt


def prefill_map(n_mt, n_nt):
    """sae_gemm_kernel: 256 latents x 256 tokens per tile, same XCD blocks."""
    yield from decode_map(n_mt, n_nt, fast_tiles=0)


def _cover(gen, n_mt, n_nt):
    seen = np.zeros((n_mt, n_nt), np.int32)
    for mt, nt in gen:
        assert 0 <= mt < n_mt and 0 <= nt < n_nt
        seen[mt, nt] += 1
    return seen


@pytest.mark.parametrize("m,T", [(256, 1), (65536, 256), (65536, 512), (1024, 300), (768, 1000),
                                 (131072, 1024), (2560, 4000)])
def test_decode_map_covers_every_tile_once(m, T):
    n_mt, n_nt = m // 256, (T + 127) // 128
    assert (_cover(decode_map(n_mt, n_nt), n_mt, n_nt) == 1).all()


@pytest.mark.parametrize("m,T", [(256, 1025), (1024, 1500), (2048, 2100), (2560, 1025),
                                 (131072, 8192), (65536, 3000), (768, 1300)])
def test_prefill_map_covers_every_tile_once(m, T):
    n_mt, n_nt = m // 256, (T + 255) // 256
    assert (_cover(prefill_map(n_mt, n_nt), n_mt, n_nt) == 1).all()
