"""Checkpoint files of the training loop on the CPU (no kernel runs): every tensor of the
training state round-trips exactly, the learning rate too, and a mismatched checkpoint is
rejected."""
import numpy as np
import pytest
import torch

from paper_1701_00485_amd.networks import LeNet, VGGSmall


@pytest.mark.parametrize("cls", [LeNet, VGGSmall])
def test_state_round_trip(cls, tmp_path):
    a = cls(device="cpu")
    a.lr = 0.01
    for t in a.named_state().values():
        t.add_(torch.arange(t.numel(), dtype=t.dtype).view(t.shape) * 1e-3)  # momenta non-zero too
    path = str(tmp_path / "c.npz")
    a.save(path)
    b = cls(device="cpu", stream=11)
    b.load(path)
    assert b.lr == 0.01 and b._codes_current is False
    sa, sb = a.named_state(), b.named_state()
    assert list(sa) == list(sb)
    for k in sa:
        assert torch.equal(sa[k], sb[k]), k


def test_state_names_cover_every_layer():
    names = list(VGGSmall(device="cpu").named_state())
    assert len([n for n in names if n.endswith(".w")]) == 7  # six convolutions and the classifier
    assert len([n for n in names if n.endswith(".gamma")]) == 6
    assert len(LeNet(device="cpu").named_state()) == 8


def test_mismatched_checkpoint_is_rejected(tmp_path):
    path = str(tmp_path / "c.npz")
    LeNet(device="cpu").save(path)
    with pytest.raises((KeyError, ValueError)):  # another network's checkpoint
        VGGSmall(device="cpu").load(path)
    data = dict(np.load(path))
    data["conv1.w"] = data["conv1.w"][:, :3]
    np.savez(path, **data)
    with pytest.raises(ValueError):
        LeNet(device="cpu").load(path)
