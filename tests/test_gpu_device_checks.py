"""Device invariant checks of the debug build (libadt_debug.so): data the host cannot see
before a launch (device parent arrays, key counts, accepted paths) is tested by the kernels,
which record a violation and stay within their buffers; adt_device_check reports it as
ADT_E_DEVICE_INVARIANT and clears it.  The release build runs the same malformed calls
within bounds and records nothing.  The invariants: the BFS order of the tree arrays
(Sec. 4.2: a parent before its child), the keys of a forward inside the cache, the accepted
path inside the tree (Sec. 3.1)."""
import ctypes as C

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _p(t):
    return C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


@pytest.fixture(scope="module")
def libs():
    from paper_2512_21857_amd import abi
    assert torch.cuda.is_available()
    return abi, abi.lib(), abi.lib_debug()


def _masks(L, parent, n):
    B, n_max = parent.shape
    mask = torch.zeros(B, n_max, 2, dtype=torch.int64, device="cuda")
    dep = torch.zeros(B, n_max, dtype=torch.int32, device="cuda")
    assert L.adt_tree_masks(_p(parent), _p(n), B, n_max, _p(mask), _p(dep), _stream()) == 0
    return mask, dep


def test_parent_order(libs):
    abi, R, D = libs
    good = torch.tensor([[-1, 0, 0, 1, 2, 3]], dtype=torch.int32, device="cuda")
    bad = torch.tensor([[-1, 0, 4, 1, 2, 3]], dtype=torch.int32, device="cuda")   # parent[2] = 4 comes later
    n = torch.tensor([6], dtype=torch.int32, device="cuda")
    _masks(D, good, n)
    assert D.adt_device_check(_stream()) == abi.OK
    m_bad, _ = _masks(D, bad, n)
    assert D.adt_device_check(_stream()) == abi.E_DEVICE_INVARIANT
    assert "parent" in abi.last_error(D)
    assert D.adt_device_check(_stream()) == abi.OK          # the record was cleared
    # release: same masks (the bad parent is treated as a root), nothing recorded
    m_rel, _ = _masks(R, bad, n)
    assert R.adt_device_check(_stream()) == abi.OK
    assert torch.equal(m_bad, m_rel)
    assert int(m_rel[0, 2, 0]) == 1 << 2                     # node 2 sees only itself


def test_keys_past_the_cache(libs):
    abi, R, D = libs
    B, H, Dh, S_cap, nq = 1, 2, 64, 256, 4
    g = torch.Generator(device="cuda").manual_seed(5)
    q = torch.randn(B, nq, H, Dh, generator=g, device="cuda").to(torch.bfloat16)
    k = torch.randn(B, H, S_cap, Dh, generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn(B, H, S_cap, Dh, generator=g, device="cuda").to(torch.bfloat16)
    mask = torch.full((B, nq, 2), -1, dtype=torch.int64, device="cuda")
    n_q = torch.tensor([nq], dtype=torch.int32, device="cuda")
    out = torch.empty_like(q)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")

    def run(L, kv_len, kv_cap):
        kl = torch.tensor([kv_len], dtype=torch.int32, device="cuda")
        assert L.adt_tree_attn(_p(q), _p(k), _p(v), H * S_cap * Dh, S_cap * Dh, _p(kl), _p(n_q), _p(n_q), _p(mask), B,
                               H, Dh, nq, kv_cap, 0.125, abi.BF16, _p(out), _p(ws), ws.numel(), _stream()) == 0

    run(D, 100, S_cap)
    assert D.adt_device_check(_stream()) == abi.OK
    run(D, 100, 64)                                          # 104 keys, a capacity of 64
    assert D.adt_device_check(_stream()) == abi.E_DEVICE_INVARIANT
    assert "cache capacity" in abi.last_error(D)
    run(R, 100, 64)
    assert R.adt_device_check(_stream()) == abi.OK
    assert torch.isfinite(out.float()).all()


def test_accepted_path_outside_the_tree(libs):
    abi, R, D = libs
    B, slices, S_cap, Dh, L0 = 1, 2, 512, 64, 100
    k0 = torch.arange(B * slices * S_cap * Dh, dtype=torch.float32, device="cuda").view(B, slices, S_cap, Dh)
    kv_len = torch.tensor([L0], dtype=torch.int32, device="cuda")
    n_acc = torch.tensor([3], dtype=torch.int32, device="cuda")

    def run(L, path_list):
        k, v = k0.clone(), (k0 + 0.5).clone()
        path = torch.tensor([path_list], dtype=torch.int32, device="cuda")
        assert L.adt_kv_compact(_p(k), _p(v), B, slices, Dh, slices * S_cap * Dh, S_cap * Dh, _p(kv_len), _p(path),
                                path.shape[1], _p(n_acc), 3, abi.F32, _stream()) == 0
        return k

    k = run(D, [0, 1, 3, 7])
    assert D.adt_device_check(_stream()) == abi.OK
    assert torch.equal(k[0, :, L0 + 2], k0[0, :, L0 + 3]) and torch.equal(k[0, :, L0 + 3], k0[0, :, L0 + 7])
    k = run(D, [0, 1, 3, 999])                               # node 999 of a tree of at most 128
    assert D.adt_device_check(_stream()) == abi.E_DEVICE_INVARIANT
    assert "accepted-path" in abi.last_error(D)
    assert torch.equal(k[0, :, L0 + 3], k0[0, :, L0 + 3])    # that row left in place
    assert torch.equal(k[0, :, L0 + 2], k0[0, :, L0 + 3])    # the valid entries still moved
    k = run(R, [0, 1, 3, 999])
    assert R.adt_device_check(_stream()) == abi.OK
    assert torch.equal(k[0, :, L0 + 3], k0[0, :, L0 + 3])
