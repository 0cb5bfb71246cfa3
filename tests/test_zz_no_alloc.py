"""adt_tree_attn_noalloc (no workspace, the library's own per-device scratch) against
adt_tree_attn with a caller workspace, through the C ABI: two calls in a row on shapes that
split the keys across workgroups (and so use the scratch), the second smaller than the
first; outputs bit-identical (same kernels, fixed merge order) and, on sampled rows, within
the bf16 tolerance of the oracle's tree attention (Sec. 3.1)."""
import numpy as np
import pytest
import torch

import synth
from oracle.attention import attend_rows, tree_key_slots
from oracle.tree import ancestors_and_self

pytestmark = pytest.mark.gpu


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def _f(a):
    return synth.bf16_bits_to_f32(a).astype(np.float64)


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_workspace_entry_point(order):
    from paper_2512_21857_amd import runtime as rt
    from paper_2512_21857_amd import abi
    assert torch.cuda.is_available()
    L = abi.lib()
    cases = [(1, 32, 128, 61, 2300, 2400, 11), (2, 8, 64, 9, 2100, 2200, 12)]
    for B, H, Dh, n, l_lo, l_hi, seed in cases:
        ab = synth.attn_microbench(B, H, Dh, n, seed=seed, l_lo=l_lo, l_hi=l_hi)
        kv_cap = int((ab.kv_len + ab.n_nodes).max())
        print(f"case B={B} H={H} Dh={Dh} n={n} kv_cap={kv_cap}", flush=True)
        q, k, v = _dev(ab.q), _dev(ab.k), _dev(ab.v)
        kl = torch.from_numpy(ab.kv_len).cuda()
        nn = torch.from_numpy(ab.n_nodes).cuda()
        mask, _ = rt.tree_masks(torch.from_numpy(ab.parent).cuda(), nn)
        ws_need = L.adt_tree_attn_workspace_size(B, H, Dh, n, kv_cap)
        assert ws_need > 0
        ref = rt.tree_attn(q, k, v, kl, nn, nn, mask, kv_cap)
        got = rt.tree_attn_noalloc(q, k, v, kl, nn, nn, mask, kv_cap)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), "no-alloc output differs"
        out = got.float().cpu().numpy()
        for b in range(B):
            keys = tree_key_slots(int(ab.kv_len[b]), ancestors_and_self(ab.parent[b]))
            rows = sorted({0, n // 2, n - 1})
            o = attend_rows(_f(ab.q[b])[rows], _f(ab.k[b]), _f(ab.v[b]), [keys[r] for r in rows], 1 / np.sqrt(Dh))
            assert np.all(np.abs(out[b][rows] - o) <= 2e-2 + 1e-2 * np.abs(o))
