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


def test_captured_mass_adds_the_window():
    mass = torch.tensor([[[0.4, 0.2, 0.1]]])              # window holds 0.3
    sel = torch.tensor([[[0, 2, -1]]], dtype=torch.int32)
    assert torch.allclose(recall.captured_mass(sel, mass),
                          torch.tensor([[0.8]]))
