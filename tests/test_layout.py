"""The tiled expert-weight layout (molt_pack_weights): the numpy definition used by the GPU
tests is a permutation of the bytes that keeps every 32-row x 128-byte tile contiguous, and
the library's packer reproduces it bit-exactly."""
import numpy as np
import pytest
import torch

from tests.helpers import tiled_layout


def test_layout_is_a_tile_preserving_permutation():
    rows, rb = 64, 384
    idx = np.arange(rows * rb, dtype=np.int64)
    src = idx.reshape(rows, rb)
    # pack the byte index itself (as 8 bytes per entry is overkill: use four byte planes)
    planes = [tiled_layout(((src >> (8 * b)) & 0xFF).astype(np.uint8)) for b in range(3)]
    back = planes[0].astype(np.int64) | (planes[1].astype(np.int64) << 8) | (planes[2].astype(np.int64) << 16)
    assert np.array_equal(np.sort(back), idx)                       # a permutation
    for t in range(rows * rb // 4096):                              # each 4 KB = one tile
        tile = back[t * 4096:(t + 1) * 4096]
        r, j = tile // rb, tile % rb
        assert len(np.unique(r // 32)) == 1 and len(np.unique(j // 128)) == 1
    # lane l of quarter c holds row l % 32, bytes 64 (l / 32) + 16 c .. +16 of the slice
    first = back[:4096].reshape(4, 64, 16)
    for c in range(4):
        for l in (0, 5, 31, 32, 63):
            assert list(first[c, l] // rb) == [l % 32] * 16
            assert list(first[c, l] % rb) == list(range(64 * (l // 32) + 16 * c, 64 * (l // 32) + 16 * c + 16))


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,shape", [(torch.uint8, (2, 96, 256)), (torch.bfloat16, (4, 64, 320)),
                                         (torch.float32, (1, 32, 96)), (torch.bfloat16, (40, 192)),
                                         (torch.float32, (7, 64))])
def test_pack_weights_matches_definition(lib, dtype, shape):
    g = torch.Generator().manual_seed(7)
    raw = torch.randint(0, 256, (int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size(),),
                        dtype=torch.uint8, generator=g)
    w = raw.view(dtype).reshape(shape)
    packed = lib.pack_weights(w.cuda())
    torch.cuda.synchronize()
    rows = int(np.prod(shape[:-1]))
    want_shape = shape if rows % 32 == 0 else ((rows + 31) // 32 * 32, shape[-1])
    assert tuple(packed.shape) == tuple(want_shape) and packed.dtype == w.dtype
    rb = shape[-1] * w.element_size()
    want = tiled_layout(raw.numpy().reshape(-1, rb))
    got = packed.cpu().contiguous().view(torch.uint8).numpy().ravel()
    assert np.array_equal(got, want)
