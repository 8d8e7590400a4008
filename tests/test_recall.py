"""The recall metrics on hand-made selections (CPU tensors; the metrics are
plain torch)."""
import torch

from paper_2503_10571_amd import recall


def test_set_recall():
    ref = torch.tensor([[[3, 1, 7, -1], [0, 2, -1, -1], [-1, -1, -1, -1]]],
                       dtype=torch.int32)
    sel = torch.tensor([[[1, 7, 9, -1], [2, 0, -1, -1], [5, -1, -1, -1]]],
                       dtype=torch.int32)
    got = recall.set_recall(sel, ref)
    assert torch.allclose(got, torch.tensor([[2 / 3, 1.0, 1.0]]))
    # duplicates in sel do not count twice; -1 in sel matches nothing
    sel2 = torch.tensor([[[1, 1, 1, -1], [-1, -1, -1, -1], [-1] * 4]],
                        dtype=torch.int32)
    assert torch.allclose(recall.set_recall(sel2, ref),
                          torch.tensor([[1 / 3, 0.0, 1.0]]))


def test_mass_ratio():
    mass = torch.tensor([[[0.5, 0.2, 0.1, 0.05, 0.15]]])
    ref = torch.tensor([[[0, 1, 4]]], dtype=torch.int32)       # 0.85
    sel = torch.tensor([[[0, 2, -1]]], dtype=torch.int32)      # 0.6
    r = recall.mass_ratio(sel, ref, mass)
    assert torch.allclose(r, torch.tensor([[0.6 / 0.85]]))
    assert torch.allclose(recall.mass_ratio(ref, ref, mass), torch.ones(1, 1))


def test_segment_mass_sums_to_candidate_share():
    """Segment masses are softmax probabilities: with no window tail they
    sum to 1, and each equals the softmax summed over its keys."""
    g = torch.Generator().manual_seed(0)
    B, Hkv, G, d, c, ns = 2, 2, 2, 16, 5, 6
    t = c * ns
    K = torch.randn(B, Hkv, t + 3, d, generator=g)
    q = torch.randn(B, Hkv * G, d, generator=g)
    m = recall.segment_mass(q, K, t, c, ns)
    assert torch.allclose(m.sum(-1), torch.ones(B, Hkv * G), atol=1e-5)
    b, h = 1, 3
    p = torch.softmax(K[b, h // G, :t] @ q[b, h] / d ** 0.5, 0)
    assert torch.allclose(m[b, h], p.view(ns, c).sum(1), atol=1e-6)


def test_captured_mass_adds_the_window():
    mass = torch.tensor([[[0.4, 0.2, 0.1]]])              # window holds 0.3
    sel = torch.tensor([[[0, 2, -1]]], dtype=torch.int32)
    assert torch.allclose(recall.captured_mass(sel, mass),
                          torch.tensor([[0.8]]))
