"""The allocation-free entry point (ppd_verify_step_static) against
ppd_verify_step with a caller workspace: the same kernels on the same
inputs, so logits, greedy tokens and the cached keys / values must be equal
bit for bit -- on two calls in a row, the second with a smaller tree (the
static array keeps what the first call left)."""
import numpy as np
import pytest
import torch

import paper_2405_18628_amd as ppd
from gpu_cases import make_case, say, tree_tensors, tree_for, workspace
from synth import workload

pytestmark = pytest.mark.gpu


def _step(case, tree, static):
    tt = tree_tensors(tree)
    T = tree.T
    logits = torch.full((T, case.shape.vocab), float("nan"), device="cuda")
    pred = torch.full((T,), -1, dtype=torch.int32, device="cuda")
    kv = ppd.KVCache(case.k, case.v)
    if static:
        status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        ppd.ppd_verify_step_static(case.model, kv, case.L, T, tt["ids"], tt["depth"], tt["mask"],
                                   logits, pred, status)
    else:
        ws = workspace(case, T)
        ppd.ppd_verify_step(case.model, kv, case.L, T, tt["ids"], tt["depth"], tt["mask"], ws, logits,
                            pred)
    torch.cuda.synchronize()
    k = case.k[:, :, case.L:case.L + T].clone()
    v = case.v[:, :, :, case.L:case.L + T].clone()
    st = int(status.item()) if static else ppd.ppd_device_status(ws)
    return logits, pred, k, v, st


def test_static_workspace_equals_caller_workspace():
    case = make_case(workload("small", cache_len=700))
    for spec in ("total:100", "total:17"):   # the second call smaller than the first
        tree = tree_for(case, spec=spec)
        say(f"[no-alloc] T={tree.T} L={case.L}")
        ref = _step(case, tree, static=False)
        got = _step(case, tree, static=True)
        assert ref[4] == 0 and got[4] == 0
        for a, b, what in zip(got[:4], ref[:4], ("logits", "pred", "keys", "values")):
            assert torch.equal(a, b), what


def test_static_workspace_rejects_a_step_too_large():
    """A step whose workspace exceeds the static array is refused before
    anything is enqueued (a model description that is never executed: an
    ffn of 262144 makes the SwiGLU activations alone 128 MiB at T = 128)."""
    import ctypes as C
    n = 2
    fake = 0x1000
    arr = (C.c_void_p * n)(*([fake] * n))
    m = ppd.ppd_model(n, 512, 4, 4, 128, 262144, 1000, 3, 1e-6, 10000.0, ppd.PPD_BF16, fake, fake,
                      *[C.cast(arr, C.POINTER(C.c_void_p)) for _ in range(6)], fake, fake)
    kv = ppd.ppd_kv(0x2000, 0x3000, 256, None)
    assert ppd.lib().ppd_workspace_bytes(C.byref(m), 128, 256) > (64 << 20)
    st = ppd.lib().ppd_verify_step_static(C.byref(m), C.byref(kv), 0, 128, fake, fake, fake, None,
                                          fake, None, None)
    assert st == ppd.PPD_EWORKSPACE, ppd.ppd_last_error()
    assert "static" in ppd.ppd_last_error()
