"""The allocation-free decode entry point (focus_decode_step_noalloc) against
focus_decode_step with a caller workspace.

Both run the same kernels with the same split, so on identical state they
must agree bit for bit (stricter than the bf16 bar of the parity tests):
outputs, LSE, the updated lengths and the appended cache / window rows.  Two
calls in a row, the second with a smaller batch and shorter caches, check that
the shared per-device scratch array carries nothing from one call to the
next; a third descriptor whose partials exceed the array is refused before
any launch.
"""

import ctypes as C

import numpy as np
import pytest
import torch

import focus_workloads as fw
import paper_2511_14694_amd as F
from gpu_util import DEV, announce
from paper_2511_14694_amd import _abi

pytestmark = pytest.mark.gpu


def _state(B, H, Hkv, D, cap_c, cap_w, seed):
    g = seed
    st = {
        "q": fw.randn((B, H, D), "bf16", g + 1, DEV),
        "k_new": fw.randn((B, Hkv, D), "bf16", g + 2, DEV),
        "v_new": fw.randn((B, Hkv, D), "bf16", g + 3, DEV),
        "cache_k": fw.randn((B, cap_c, Hkv, D), "bf16", g + 4, DEV),
        "cache_v": fw.randn((B, cap_c, Hkv, D), "bf16", g + 5, DEV),
        "win_k": fw.randn((B, cap_w, Hkv, D), "bf16", g + 6, DEV),
        "win_v": fw.randn((B, cap_w, Hkv, D), "bf16", g + 7, DEV),
    }
    rng = np.random.default_rng(seed)
    st["cache_len"] = torch.as_tensor(rng.integers(cap_c // 2, cap_c - 1, B), dtype=torch.int32, device=DEV)
    st["win_len"] = torch.as_tensor(rng.integers(0, cap_w - 1, B), dtype=torch.int32, device=DEV)
    # summary steps (into the cache), base steps, and window ends
    st["kind"] = torch.as_tensor(rng.choice([0, 1, 3], B).astype(np.uint8), device=DEV)
    return st


def _run(st, noalloc):
    s = {k: v.clone() for k, v in st.items()}
    B, H, D = s["q"].shape
    o = torch.full((B, H, D), float("nan"), dtype=torch.bfloat16, device=DEV)
    lse = torch.full((B, H), float("nan"), dtype=torch.float32, device=DEV)
    args = (s["q"], s["k_new"], s["v_new"], s["kind"], s["cache_k"], s["cache_v"], s["cache_len"],
            s["win_k"], s["win_v"], s["win_len"])
    if noalloc:
        F.focus_decode_step_noalloc(*args, o=o, lse=lse)
    else:
        F.focus_decode_step(*args, o=o, lse=lse)
    torch.cuda.synchronize()
    return s, o, lse


@pytest.mark.parametrize("calls", [[(16, 32, 32, 128, 3000, 1000, 5), (3, 8, 4, 128, 700, 300, 6)],
                                   [(4, 4, 2, 64, 900, 200, 7), (2, 4, 2, 64, 120, 40, 8)]])
def test_noalloc_matches_workspace_step(calls):
    for B, H, Hkv, D, cap_c, cap_w, seed in calls:
        announce(f"decode noalloc B={B} H={H} Hkv={Hkv} D={D} cache {cap_c} window {cap_w} seed {seed}")
        st = _state(B, H, Hkv, D, cap_c, cap_w, seed)
        ref, o_ref, lse_ref = _run(st, noalloc=False)
        got, o_got, lse_got = _run(st, noalloc=True)
        assert torch.equal(o_got.view(torch.int16), o_ref.view(torch.int16)), "o differs"
        assert torch.equal(lse_got, lse_ref), "lse differs"
        for name in ("cache_len", "win_len", "cache_k", "cache_v", "win_k", "win_v"):
            assert torch.equal(got[name], ref[name]), name
        assert not torch.isnan(o_got.float()).any()


def test_noalloc_refuses_partials_beyond_the_scratch():
    st = _state(2, 4, 4, 128, 64, 32, 9)
    d = _abi.DecodeDesc()
    d.dtype, d.batch, d.n_heads, d.n_kv_heads, d.head_dim = 0, 2, 4, 4, 128
    d.split_keys = 16
    for f in ("q", "k_new", "v_new", "kind", "cache_k", "cache_v", "cache_len", "win_k", "win_v", "win_len"):
        setattr(d, f, st[f].data_ptr())
    o = torch.empty_like(st["q"])
    d.o = o.data_ptr()
    # a capacity whose partials (batch x ceil(cap / 16) x heads x (D + 2) floats)
    # exceed the scratch array; the call must return before any launch
    d.cache_cap = 1 << 22
    d.win_cap = 32
    need = _abi.lib().focus_decode_workspace(C.byref(d))
    assert need > (16 << 20)
    assert _abi.lib().focus_decode_step_noalloc(C.byref(d), None) == 6   # FOCUS_E_WORKSPACE
