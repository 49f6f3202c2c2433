"""GPU parity of focus_fidelity against the float64 oracle.

Every position of small cases (vocab 1 .. 1024 across the one-thread,
half-wave and one-wave paths, logits and probabilities with exact zeros,
logits far enough below the rest that the clip acts, bf16 and f32, sequences
including empty ones) and sampled positions of the two full-size workloads (1 M positions of 4 nucleotides, 1 M positions of a 512-entry
vocabulary).  Tolerance (float32 arithmetic against float64 on the same
inputs): |got - ref| <= 2e-5 + 2e-5 |ref| per metric; identical inputs give
exact zeros.
"""

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce, to64
from oracle import fidelity as FD

pytestmark = pytest.mark.gpu

ATOL = RTOL = 2e-5


def _check(got, ref, what):
    err = np.abs(got - ref)
    bad = err > ATOL + RTOL * np.abs(ref)
    assert not bad.any(), f"{what}: worst {err.max():.3e} at {np.argwhere(bad)[:3].tolist()}"
    return float(err.max()) if err.size else 0.0


@pytest.mark.parametrize("vocab", [1, 2, 4, 7, 8, 9, 63, 64, 65, 512, 1000, 1024])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kind", ["logits", "probs"])
def test_small_all_positions(vocab, dtype, kind):
    announce(f"fidelity vocab={vocab} dtype={dtype} kind={kind}")
    n = 777
    p, q = fw.fidelity_logits(n, vocab, dtype, seed=vocab * 7 + (dtype == "bf16"), device=DEV)
    if kind == "probs":
        p = torch.softmax(p.float(), dim=1)
        q = torch.softmax(q.float() * 3, dim=1)
        p[::5, 0] = 0.0                      # exact zeros: the clip must act
        if dtype == "bf16":
            p, q = p.to(torch.bfloat16), q.to(torch.bfloat16)
    cu = [0, 100, 100, 500, n]
    out, mean = F.focus_fidelity(p.contiguous(), q.contiguous(),
                                 F.FOCUS_FID_LOGITS if kind == "logits" else F.FOCUS_FID_PROBS, cu_pos=cu)
    torch.cuda.synchronize()
    pp, qq = to64(p), to64(q)
    ref = FD.metrics_from_logits(pp, qq) if kind == "logits" else FD.metrics(pp, qq)
    _check(out.cpu().numpy().astype(np.float64), ref, f"per-position v{vocab}")
    _check(mean.cpu().numpy().astype(np.float64), FD.sequence_means(ref, cu), f"means v{vocab}")


@pytest.mark.parametrize("vocab", [4, 100, 256, 512])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_logits_that_clip(vocab, dtype):
    """Rows whose softmax puts some entries below the 1e-12 clip (logits 60
    below the rest) next to rows that clip nothing: the clip-and-renormalise
    path and the path that skips it, in one launch."""
    announce(f"fidelity clipped logits v{vocab} {dtype}")
    n = 513
    p, q = fw.fidelity_logits(n, vocab, "f32", seed=vocab + 11, device=DEV)
    p[::3, : max(1, vocab // 7)] -= 60.0       # every third row of p clips
    q[1::4, -1] -= 60.0                        # every fourth row of q clips one entry
    if dtype == "bf16":
        p, q = p.to(torch.bfloat16), q.to(torch.bfloat16)
    out, _ = F.focus_fidelity(p.contiguous(), q.contiguous())
    torch.cuda.synchronize()
    ref = FD.metrics_from_logits(to64(p), to64(q))
    _check(out.cpu().numpy().astype(np.float64), ref, f"clipped logits v{vocab} {dtype}")


@pytest.mark.parametrize("vocab", [4, 512])
def test_identical_inputs_give_exact_zeros(vocab):
    announce(f"fidelity identical v{vocab}")
    p, _ = fw.fidelity_logits(1000, vocab, "f32", seed=3, device=DEV)
    out, _ = F.focus_fidelity(p, p.clone())
    torch.cuda.synchronize()
    assert (out == 0).all()


def test_empty_and_bounds():
    announce("fidelity empty / bounds")
    p = torch.zeros(0, 4, device=DEV)
    out, mean = F.focus_fidelity(p, p, cu_pos=[0, 0])
    torch.cuda.synchronize()
    assert out.shape == (0, 5) and (mean == 0).all()
    x, y = fw.fidelity_logits(10, 4, "f32", seed=1, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out, mean = F.focus_fidelity(x, y, cu_pos=[0, 4, 11], err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & F.FOCUS_ERR_BOUNDS
    assert (mean[1] == 0).all()
    ref = FD.metrics_from_logits(to64(x), to64(y))
    _check(mean[0].cpu().numpy().astype(np.float64), ref[:4].mean(0), "mean of a valid sequence")


@pytest.mark.parametrize("name", list(fw.FIDELITY))
def test_workload_full_size_sampled(name):
    n, vocab, dtype = fw.FIDELITY[name]
    announce(f"fidelity workload {name}")
    p, q = fw.fidelity_logits(n, vocab, dtype, seed=fw.BASE_SEED, device=DEV)
    cu = np.linspace(0, n, 9).astype(np.int64)       # 8 sequences
    out, mean = F.focus_fidelity(p, q, cu_pos=cu)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, n - 1], np.random.default_rng(1).integers(0, n, 3000)]))
    idx = torch.as_tensor(rows, device=DEV)
    ref = FD.metrics_from_logits(to64(p[idx]), to64(q[idx]))
    worst = _check(out[idx].cpu().numpy().astype(np.float64), ref, name)
    # the means are over the device's own per-position values (the oracle mean
    # of all 1 M rows is a property check: within float32 summation error)
    o64 = out.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(mean.cpu().numpy(), FD.sequence_means(o64, cu), rtol=1e-5, atol=1e-7)
    print(f"[parity] fidelity {name}: worst abs {worst:.3e}", flush=True)
