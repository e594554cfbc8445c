"""Input generators: the vectorised hash equals a plain-integer restatement of
lowbias32, values are device-independent by construction (integer ops + one
float32 multiply), and trees satisfy the interface contract."""
import numpy as np
import pytest
import torch

from synth import rng, workload
from synth.trees import make_tree


def _lowbias32(x):
    x ^= x >> 16
    x = (x * 0x7FEB352D) & 0xFFFFFFFF
    x ^= x >> 15
    x = (x * 0x846CA68B) & 0xFFFFFFFF
    x ^= x >> 16
    return x


def test_hash_matches_plain_integers():
    xs = [0, 1, 2, 0xFFFFFFFF, 0x12345678, 0x80000000, 77777777]
    got = rng.hash32(torch.tensor(xs, dtype=torch.int64)).tolist()
    assert got == [_lowbias32(x) for x in xs]


def test_normal_moments_and_offsets():
    a = rng.normal((1 << 18,), 3, "w", 0.02)
    assert abs(a.mean().item()) < 2e-4 and abs(a.std().item() - 0.02) < 2e-4
    assert a.abs().max().item() <= 0.02 * 3.47
    # offset addressing: a slice regenerated alone is identical
    b = torch.empty(1000)
    rng.normal_(b, 3, "w", 0.02, offset=5000)
    assert torch.equal(a[5000:6000], b)
    c = rng.normal((100,), 3, "w", 0.02, dtype=torch.bfloat16)
    assert torch.equal(c, a[:100].to(torch.bfloat16))


def test_randint_range():
    x = rng.randint(100000, 32000, 1, "t")
    assert x.min().item() >= 0 and x.max().item() < 32000
    assert abs(x.float().mean().item() - 16000) < 200


@pytest.mark.parametrize("spec,depth", [("candidates:10", 4), ("candidates:32", 4),
                                        ("total:64", 5), ("total:16", 5), ("total:128", 5)])
def test_tree_contract(spec, depth):
    V = 32000
    for seed in range(50):
        t = make_tree(spec, V, 3, depth, seed, 17)
        assert t.parent[0] == -1 and t.ids[0] == 17
        assert all(0 <= t.parent[i] < i for i in range(1, t.T))
        if spec.startswith("total"):
            assert t.T == int(spec.split(":")[1])
        else:
            assert t.n_candidates == int(spec.split(":")[1])
        cand = t.ids[:t.n_candidates]
        assert (cand < V).all() and (t.ids[t.n_candidates:] >= V).all()
        kids = {}
        for i in range(1, t.n_candidates):
            kids.setdefault(int(t.parent[i]), []).append(int(t.ids[i]))
        for p, ks in kids.items():
            assert len(set(ks)) == len(ks) and len(ks) <= 4
        # every leaf candidate carries a 3-long chain of prompt ids V, V+1, V+2
        leaves = [i for i in range(t.n_candidates) if i not in kids]
        assert t.T == t.n_candidates + 3 * len(leaves)
        for i in range(t.n_candidates, t.T):
            p = int(t.parent[i])
            j = 0 if p < t.n_candidates else int(t.ids[p]) - V + 1
            assert t.ids[i] == V + j
        dep = np.zeros(t.T, int)
        for i in range(1, t.T):
            dep[i] = dep[t.parent[i]] + 1
        assert dep[:t.n_candidates].max() <= depth
