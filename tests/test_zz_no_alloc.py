"""rotor_solve_noalloc (the static-workspace variant of rotor_solve) through
the C ABI: on two calls in a row, the second with a smaller input, its
tables equal those rotor_solve writes with a caller workspace, bit for bit;
sizes beyond its workspace are refused."""
import ctypes

import numpy as np
import pytest

from paper_1911_13214_amd import chaingen

pytestmark = pytest.mark.gpu


def _tables_both_ways(params, M):
    import torch

    from paper_1911_13214_amd import rotor
    n, _, L = params.shape
    d_params = rotor.upload_params(params, M, "cuda")
    ref_cost, ref_dec = rotor.alloc_tables(n, L, M, "cuda")
    work = rotor.alloc_workspace(n, L, M, "cuda")
    rotor.rotor_solve(d_params, n, L, M, ref_cost, ref_dec, work)
    cost, dec = rotor.alloc_tables(n, L, M, "cuda")
    cost.fill_(-5)
    dec.fill_(-5)
    lib = rotor.lib()
    st = lib.rotor_solve_noalloc(d_params.data_ptr(), n, L, M, cost.data_ptr(), dec.data_ptr(),
                                 torch.cuda.current_stream().cuda_stream)
    assert st == rotor.ROTOR_OK, rotor.status_string(st)
    torch.cuda.synchronize()
    pitch = rotor.rotor_layout(n, L, M)[0]
    assert pitch == cost.shape[-1]
    return (cost[..., :M + 1].cpu().numpy(), dec[..., :M + 1].cpu().numpy(),
            ref_cost[..., :M + 1].cpu().numpy(), ref_dec[..., :M + 1].cpu().numpy())


def test_noalloc_equals_rotor_solve_on_two_calls():
    from paper_1911_13214_amd import rotor
    # 16 chains of L=64, M=640: the blocked fill order, about 90 MB of workspace;
    # then one chain of L=50, M=500: the streamed order, about 2 MB
    cases = [(chaingen.random_chains(16, 64, seed=901), 640), (chaingen.random_chains(1, 50, seed=902), 500)]
    for params, M in cases:
        n, _, L = params.shape
        need = rotor.rotor_workspace_bytes(n, L, M)
        print(f"noalloc n={n} L={L} M={M} workspace {need} bytes", flush=True)
        assert need <= rotor.NOALLOC_WORK_BYTES
        c, d, rc, rd = _tables_both_ways(params, M)
        assert np.array_equal(c, rc) and np.array_equal(d, rd)


def test_noalloc_refuses_sizes_beyond_its_workspace():
    import torch

    from paper_1911_13214_amd import rotor
    print("noalloc capacity", flush=True)
    L, M = 200, 2000  # about 330 MB of workspace
    assert rotor.rotor_workspace_bytes(1, L, M) > rotor.NOALLOC_WORK_BYTES
    fake = torch.empty(8, dtype=torch.int64, device="cuda")
    st = rotor.lib().rotor_solve_noalloc(fake.data_ptr(), 1, L, M, fake.data_ptr(), fake.data_ptr(), None)
    assert st == rotor.ROTOR_ECAPACITY
    assert rotor.lib().rotor_solve_noalloc(None, 1, L, M, fake.data_ptr(), fake.data_ptr(), None) == rotor.ROTOR_EINVAL
    assert ctypes.sizeof(ctypes.c_void_p) == 8
