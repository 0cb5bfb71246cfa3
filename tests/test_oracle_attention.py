"""Tree attention (Sec. 3.1: each node sees the prefix and its root-to-node path) pinned
against dense causal attention computed by torch's scaled_dot_product_attention."""
import itertools

import numpy as np
import torch

from oracle.attention import attend_rows, tree_key_slots
from oracle.tree import ancestors_and_self, is_bfs_ordered, packed_mask


def all_parent_arrays(n):
    """Every tree on nodes 0..n-1 with parent[i] < i (root 0)."""
    for tail in itertools.product(*[range(i) for i in range(1, n)]):
        yield [-1] + list(tail)


def causal_sdpa_last_row(q_row, K, V, scale):
    """Last row of causal attention over keys K/V ([H][T][Dh]) with query q_row ([H][Dh])."""
    H, T, Dh = K.shape
    qq = torch.zeros(H, T, Dh, dtype=torch.float64)
    qq[:, -1] = torch.from_numpy(q_row)
    out = torch.nn.functional.scaled_dot_product_attention(
        qq[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None], is_causal=True, scale=scale)
    return out[0, :, -1].numpy()


def _check_tree(parent, rng, L=5, H=2, Dh=8):
    n = len(parent)
    kc = rng.standard_normal((H, L + n, Dh))
    vc = rng.standard_normal((H, L + n, Dh))
    q = rng.standard_normal((n, H, Dh))
    anc = ancestors_and_self(parent)
    o = attend_rows(q, kc, vc, tree_key_slots(L, anc), 0.3)
    for i in range(n):
        seq = list(range(L)) + [L + j for j in anc[i]]            # prefix + path root..i
        ref = causal_sdpa_last_row(q[i], kc[:, seq], vc[:, seq], 0.3)
        np.testing.assert_allclose(o[i], ref, rtol=1e-12, atol=1e-12)


def test_tree_attention_equals_path_causal_attention_all_small_trees():
    rng = np.random.default_rng(0)
    count = 0
    for n in range(1, 7):
        for parent in all_parent_arrays(n):
            _check_tree(parent, rng, L=int(rng.integers(0, 4)))
            count += 1
    assert count == 1 + 1 + 2 + 6 + 24 + 120


def test_tree_attention_random_large_trees():
    import synth
    rng = np.random.default_rng(1)
    for n in (17, 61, 128):
        parent = synth.random_parents(rng, n)
        assert is_bfs_ordered(parent)
        _check_tree(parent, rng, L=9)


def test_chain_tree_is_causal_attention():
    rng = np.random.default_rng(2)
    n, L, H, Dh = 9, 4, 3, 16
    kc = rng.standard_normal((H, L + n, Dh))
    vc = rng.standard_normal((H, L + n, Dh))
    q = rng.standard_normal((n, H, Dh))
    parent = [-1] + list(range(n - 1))
    o = attend_rows(q, kc, vc, tree_key_slots(L, ancestors_and_self(parent)), 0.25)
    qq = np.zeros((H, L + n, Dh))
    qq[:, L:] = q.transpose(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(qq)[None], torch.from_numpy(kc)[None], torch.from_numpy(vc)[None],
        is_causal=True, scale=0.25)[0].numpy()
    np.testing.assert_allclose(o, ref[:, L:].transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


def test_packed_mask_bits():
    parent = [-1, 0, 0, 1, 1, 2, 3]
    m = packed_mask(parent, 1)
    assert [int(x) for x in m[:, 0]] == [0b1, 0b11, 0b101, 0b1011, 0b10011, 0b100101, 0b1001011]
    big = [-1] + list(range(99))           # chain of 100 nodes: row 99 has bits 0..99
    m2 = packed_mask(big, 2)
    assert int(m2[99, 0]) == 2 ** 64 - 1 and int(m2[99, 1]) == 2 ** 36 - 1
