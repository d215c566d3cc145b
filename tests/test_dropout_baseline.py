"""GPU parity of the conventional-dropout baseline kernels (Sec. II-C): the
element keep mask is bit-exact with the oracle's counter-based draws, the
masked values are exactly scale * y or 0, and the backward applies the same
mask. Through the C ABI."""
import numpy as np
import pytest
import torch

from gpu_util import ard_dtype, device
from oracle import prng as oprng
from paper_1805_08939_amd import api, synth

pytestmark = pytest.mark.gpu


def _bits(words, total):
    w = np.asarray(words, dtype=np.uint64)
    e = np.arange(total)
    return ((w[e // 32] >> (e % 32).astype(np.uint64)) & 1).astype(bool)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n,batch", [(37, 5), (10, 3), (513, 128), (1, 1)])
@pytest.mark.parametrize("p", [0.0, 0.3, 0.7])
def test_mask_and_values_against_oracle(dtype, n, batch, p):
    d = device()
    total = n * batch
    g = synth.generator(n * 1000 + batch)
    Y = synth.to_storage(synth.normal(g, (n, batch)), dtype)
    dY = synth.to_storage(synth.normal(g, (n, batch)), dtype)
    words = (total + 31) // 32
    mask = torch.full((words + 1,), 0x5A5A5A5A, dtype=torch.int32, device=d)  # one guard word
    Yd, dYd = Y.clone().to(d), dY.clone().to(d)
    scale = 1.0 / (1.0 - p)
    api.ard_dropout_fwd(ard_dtype(dtype), n, batch, p, scale, 8939, 3, 77, Yd, mask)
    api.ard_dropout_bwd(ard_dtype(dtype), n, batch, scale, mask, dYd)
    torch.cuda.synchronize()
    want = oprng.tile_bitmap_bernoulli(n, batch, p, 8939, 3, 77)
    got = [int(x) & 0xFFFFFFFF for x in mask[:words].cpu().tolist()]
    assert got == want
    assert int(mask[words]) == 0x5A5A5A5A  # nothing past the mask
    keep = torch.from_numpy(_bits(want, total).reshape(n, batch))
    sdt = synth.storage_dtype(dtype)
    zero = torch.zeros((), dtype=sdt)
    assert torch.equal(Yd.cpu(), torch.where(keep, (Y.float() * scale).to(sdt), zero))
    assert torch.equal(dYd.cpu(), torch.where(keep, (dY.float() * scale).to(sdt), zero))


def test_drop_rate():
    """Empirical drop rate of the element mask within 0.01 of p over 2^18 draws."""
    d = device()
    n, batch = 2048, 128
    for p in (0.3, 0.5, 0.7):
        Y = torch.ones(n, batch, device=d)
        mask = torch.zeros((n * batch + 31) // 32, dtype=torch.int32, device=d)
        api.ard_dropout_fwd(api.ARD_F32, n, batch, p, 1.0, 8939, 1, 5, Y, mask)
        torch.cuda.synchronize()
        assert abs(1.0 - float(Y.mean()) - p) < 0.01


def test_invalid_arguments():
    d = device()
    Y = torch.ones(4, 4, device=d)
    mask = torch.zeros(1, dtype=torch.int32, device=d)
    for args in [(api.ARD_F32, 4, 4, 1.0), (api.ARD_F32, 4, 4, -0.1), (api.ARD_F32, 0, 4, 0.5), (7, 4, 4, 0.5)]:
        with pytest.raises(api.ArdError):
            api.ard_dropout_fwd(*args, 1.0, 1, 0, 0, Y, mask)
    with pytest.raises(api.ArdError):
        api.ard_dropout_fwd(api.ARD_F32, 4, 4, 0.5, 1.0, 1, 1 << 24, 0, Y, mask)
    with pytest.raises(api.ArdError):
        api.ard_dropout_bwd(api.ARD_F32, 4, 4, 1.0, None, Y)
