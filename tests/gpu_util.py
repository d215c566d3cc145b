"""Helpers for the GPU parity tests (imported only by tests marked gpu)."""
import numpy as np
import torch

from oracle import patterns as opat
from paper_1805_08939_amd import api, synth

F32_TOL = 1e-4   # max relative error, fp32 paths
BF16_TOL = 2e-2  # max relative error, bf16 paths (fp32 accumulation)


def device():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    return torch.device("cuda:0")


def tol(dtype_name):
    return F32_TOL if dtype_name == "f32" else BF16_TOL


def ard_dtype(dtype_name):
    return api.ARD_F32 if dtype_name == "f32" else api.ARD_BF16


def row_plan(n, period, offset, check=True, with_list=True):
    """Builds a row plan on the device; checks its list against the oracle.
    with_list=False: a list-free plan (no device list, nothing launched)."""
    kept = opat.row_kept_count(n, period, offset)
    if not with_list:
        plan = api.ard_plan_rows(n, period, offset, None)
        assert plan.kept == kept and not plan.d_idx
        return plan
    idx = torch.full((max(kept, 1),), -1, dtype=torch.int32, device=device())
    plan = api.ard_plan_rows(n, period, offset, idx)
    if check:
        torch.cuda.synchronize()
        assert plan.kept == kept
        assert idx[:kept].cpu().tolist() == opat.row_kept_list(n, period, offset)
    return plan


def to_dev(t):
    return t.contiguous().to(device())


def f64(t):
    return synth.as_f64(t).numpy()


def compare(got, want, norm, rel_tol, what):
    """Componentwise check |got - want| <= rel_tol * norm, where norm is the
    GEMM error normaliser (|A| |B| of the masked operands, plus |bias|). Where
    norm is 0 the result must be exactly 0. Also checks the normwise error
    max|got - want| / max|want|. Returns (componentwise, normwise) errors."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    norm = np.asarray(norm, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite values"
    diff = np.abs(got - want)
    zero = norm == 0.0
    assert not diff[zero].any(), f"{what}: nonzero where the exact result is 0"
    comp = float((diff[~zero] / norm[~zero]).max()) if (~zero).any() else 0.0
    scale = float(np.abs(want).max())
    normwise = float(diff.max() / scale) if scale > 0 else float(diff.max())
    assert comp <= rel_tol, f"{what}: componentwise error {comp:.3e} > {rel_tol}"
    assert normwise <= rel_tol, f"{what}: normwise error {normwise:.3e} > {rel_tol}"
    return comp, normwise


def workspace(nbytes):
    """A device workspace of at least nbytes (None when nothing is needed)."""
    if nbytes == 0:
        return None
    return torch.empty((nbytes + 15) // 16 * 4, dtype=torch.float32, device=device())


def full_weight_grad(mlp, l, pats, fill):
    """Layer l's weight gradient after a step of the benchmark's MLP, as a
    full [N][K] fp64 array: a layer whose inputs were dropped that step wrote
    the compact gradient dWc[kept_out][ldc] into its dW buffer; its entries are
    placed at [S_out][S_in] and every other entry gets fill. An input-major
    layer's buffer holds dW^T[K][N], returned transposed."""
    if getattr(mlp, "input_major", None) and mlp.input_major[l]:  # dW^T[K][N]
        return mlp.dW[l].t().double().cpu().numpy()
    dW = mlp.dW[l].double().cpu().numpy()
    if l not in mlp.step_compact:
        return dW
    N, K = dW.shape
    pin = pats[l - 1]
    pout = pats[l] if l < mlp.L - 1 else (1, 0)
    Sin, Sout = opat.row_kept_list(K, *pin), opat.row_kept_list(N, *pout)
    ldc = (len(Sin) + 7) // 8 * 8
    dWc = dW.reshape(-1)[:len(Sout) * ldc].reshape(len(Sout), ldc)[:, :len(Sin)]
    full = np.full((N, K), fill)
    full[np.ix_(Sout, Sin)] = dWc
    return full
