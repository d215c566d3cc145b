"""ard_fc_fwd_noalloc (the FC forward with the library's static per-GPU
scratch instead of a workspace) against ard_fc_fwd with a workspace, through
the C ABI: two calls in a row, the second on a smaller layer, each bit for bit
the workspace call's result; a layer needing more than the static scratch is
rejected before any launch."""
import numpy as np
import pytest
import torch

from gpu_util import device, row_plan, to_dev, workspace
from paper_1805_08939_amd import api, synth

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 32 << 20


def layer(dtype, B, K, N, pin, pout, seed, layout=api.ARD_WEIGHTS_FULL):
    g = synth.generator(seed)
    X = synth.to_storage(synth.normal(g, (B, K)), dtype)
    W = synth.to_storage(synth.normal(g, (N, K), 0.05), dtype)
    b = synth.normal(g, (N,), 0.1)
    desc = api.fc_desc(api.ARD_F32 if dtype == "f32" else api.ARD_BF16, B, K, N,
                       row_plan(K, *pin, with_list=False), row_plan(N, *pout, with_list=False), 1.25,
                       api.ARD_ACT_RELU, api.ARD_DROPPED_ZERO, layout)
    if layout == api.ARD_WEIGHTS_INPUT_MAJOR:
        W = W.T.contiguous()
    return desc, to_dev(X.T), to_dev(W), to_dev(b), synth.storage_dtype(dtype)


def test_noalloc_forward_matches_workspace_forward():
    cases = [
        # full weights with a gathered input side: the compact weight copy
        # lives in the scratch (and the split partial sums, if any)
        ("bf16", 512, 3000, 1500, (3, 1), (2, 0)),
        # a smaller layer next: a tiny output grid whose contraction is split,
        # partial sums in the scratch
        ("f32", 8, 4096, 8, (1, 0), (1, 0)),
        # input-major weights (a last layer): the kept inputs are read in place
        ("bf16", 64, 4096, 1024, (2, 1), (1, 0), api.ARD_WEIGHTS_INPUT_MAJOR),
    ]
    for i, (dtype, B, K, N, pin, pout, *layout) in enumerate(cases):
        desc, Xt, W, b, sdt = layer(dtype, B, K, N, pin, pout, seed=100 + i, layout=layout[0] if layout else
                                    api.ARD_WEIGHTS_FULL)
        need = api.ard_fc_workspace_bytes(desc)
        assert need <= SCRATCH_BYTES and (need > 0 or layout)
        ref = torch.full((N, B), 3.0, dtype=sdt, device=device())
        got = torch.full((N, B), -3.0, dtype=sdt, device=device())
        api.ard_fc_fwd(desc, Xt, W, b, ref, workspace(need))
        api.ard_fc_fwd_noalloc(desc, Xt, W, b, got)
        torch.cuda.synchronize()
        assert torch.isfinite(ref.float()).all()
        assert torch.equal(got, ref), f"case {i}: noalloc result differs from the workspace call"


def test_noalloc_rejects_layers_beyond_the_scratch():
    # the wide MLP's hidden layer with full weights and half its inputs
    # dropped: the compact copy alone is 64 MiB
    desc, Xt, W, b, sdt = layer("bf16", 16, 8192, 8192, (2, 0), (1, 0), seed=7)
    assert api.ard_fc_workspace_bytes(desc) > SCRATCH_BYTES
    Y = torch.full((8192, 16), 5.0, dtype=sdt, device=device())
    with pytest.raises(api.ArdError) as e:
        api.ard_fc_fwd_noalloc(desc, Xt, W, b, Y)
    assert e.value.status == 5
    torch.cuda.synchronize()
    assert (Y.float() == 5.0).all()  # nothing was launched
