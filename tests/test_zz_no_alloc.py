"""The allocation-free head-error entry point against the workspace one.

loca_error_targets_noalloc runs the kernels of loca_error_targets on the library's
fixed scratch array; on the same inputs its outputs (credit coordinates, ||Q||^2
records, dev_info) must be those of the workspace call, bit for bit.  Three calls in
a row share the array: a full-vocabulary product case, then two small label sets,
the last smaller than the one before, so stale contents of the array from a larger
call are present when a smaller one runs.
"""
import numpy as np
import pytest

from gpu_helpers import log

pytestmark = pytest.mark.gpu


def _case(C, n, nb, k, d, ldt, adt, seed):
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    zt = torch.bfloat16 if ldt == "bf16" else torch.float32
    at = torch.bfloat16 if adt == "bf16" else torch.float32
    ld = (C + 7) // 8 * 8
    zbuf = torch.zeros((n, ld), device="cuda", dtype=zt)
    zbuf[:, :C] = (torch.randn((n, C), generator=g, device="cuda") * 3).to(zt)
    y = torch.randint(0, C, (n,), generator=g, device="cuda", dtype=torch.int32)
    A = (torch.randn((nb, C, k), generator=g, device="cuda") / np.sqrt(k)).to(at)
    B = torch.randn((nb, k, d), generator=g, device="cuda") / np.sqrt(k)
    aw = torch.rand(n, generator=g, device="cuda") * 2
    return zbuf[:, :C], y, A, B, aw


@pytest.mark.parametrize("order", [0])
def test_error_targets_noalloc_matches_workspace_call(order):
    import torch
    from paper_2608_03020_amd import loca
    loca.load()
    cases = [(3001, 512, 2, 32, 256, "bf16", "bf16", 1),   # vocabulary product path
             (5, 8192, 6, 64, 1024, "f32", "f32", 2),       # small label set
             (4, 1000, 3, 16, 600, "f32", "f32", 3)]        # smaller, after the larger call
    for C, n, nb, k, d, ldt, adt, seed in cases:
        need = loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, nb, n, d, k, C)
        assert need <= loca.error_targets_noalloc_max_bytes()
        log(f"case noalloc C={C} n={n} nb={nb} k={k} d={d} (workspace {need} bytes)")
        z, y, A, B, aw = _case(C, n, nb, k, d, ldt, adt, seed)
        Y_ref = torch.full((nb, n, k), float("nan"), device="cuda")
        Y_na = torch.full((nb, n, k), float("nan"), device="cuda")
        mb_ref, mb_na = loca.new_mb(nb), loca.new_mb(nb)
        info_ref = torch.full((1,), 99, dtype=torch.int32, device="cuda")
        info_na = torch.full((1,), 77, dtype=torch.int32, device="cuda")
        ws = loca.alloc_workspace(need)
        ws.fill_(255)
        loca.loca_error_targets(z, y, A, B, Y_ref, mb_ref, info_ref, ws, a_w=aw)
        loca.loca_error_targets_noalloc(z, y, A, B, Y_na, mb_na, info_na, a_w=aw)
        torch.cuda.synchronize()
        assert int(info_ref.item()) == 0 and int(info_na.item()) == 0
        assert not bool(torch.isnan(Y_na).any())
        assert torch.equal(Y_na, Y_ref)
        assert torch.equal(mb_na, mb_ref)


def test_error_targets_noalloc_rejects_oversize():
    import torch
    from paper_2608_03020_amd import loca
    n, C, k, d = 4096, 151936, 64, 2048  # the full-vocabulary product needs ~34 MB of scratch
    assert loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, 1, n, d, k, C) > loca.error_targets_noalloc_max_bytes()
    z = torch.zeros((n, C), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros(n, dtype=torch.int32, device="cuda")
    A = torch.zeros((1, C, k), dtype=torch.bfloat16, device="cuda")
    B = torch.zeros((1, k, d), device="cuda")
    Y = torch.zeros((1, n, k), device="cuda")
    mb = loca.new_mb(1)
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(loca.LocaError) as ex:
        loca.loca_error_targets_noalloc(z, y, A, B, Y, mb, info)
    assert ex.value.status == loca.LOCA_E_UNSUPPORTED
