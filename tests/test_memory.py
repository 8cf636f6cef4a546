"""Model-size accounting (Sec. 4, Fig. 2) on the CPU."""
import pytest

from paper_1701_00485_amd import memory


def test_alexnet_matches_the_cited_size():
    # Sec. 1 cites AlexNet at 61M parameters performing 1.5B operations per image
    w, f, o, _ = memory.count(memory.alexnet())
    assert (w + o) == pytest.approx(61e6, rel=5e-3)
    # multiply-adds of the 227 x 227 forward pass (output sizes 55, 27, 13, 13, 13)
    macs = 0
    for (kind, cin, cout, k, groups, _), hw in zip(memory.alexnet(), (55, 27, 13, 13, 13, 1, 1, 1)):
        macs += hw * hw * cout * (cin // groups) * k * k
    assert 2 * macs == pytest.approx(1.5e9, rel=5e-2)


def test_resnet18_matches_the_network_that_runs():
    # the same architecture as the ResNet-18 workload (its layer list), counted independently
    from paper_1701_00485_amd.networks import ResNet18
    w, f, o, _ = memory.count(memory.resnet18())
    convs = [(7, 3, 64)]
    cin = 64
    for cout, stride in ResNet18.STAGES:
        for b in range(2):
            s = stride if b == 0 else 1
            convs += [(3, cin, cout), (3, cout, cout)] + ([(1, cin, cout)] if (s != 1 or cin != cout) else [])
            cin = cout
    assert w == sum(k * k * ci * co for k, ci, co in convs) + 512 * 1000
    assert f == sum(co for _, _, co in convs) + 1000
    # FLOP of the forward pass agree with the workload's own count (2 per multiply-add)
    assert ResNet18.flops(1) == pytest.approx(3.6e9, rel=2e-2)


def test_sizes_and_ratios():
    t = memory.memory_table()
    for name, r in t.items():
        w, f, o = r["filter_weights"], r["filters"], r["other_params"]
        # 2 bits per weight is 1/32 of 64 bits; the per-filter scales and fp32 leftovers cost the rest
        assert r["tbn_bytes"] >= w // 4
        assert 28 < r["fp64_over_tbn"] < 32
        assert r["tbn_packed_bytes"] >= r["tbn_bytes"] - 1
        assert r["fp64_bytes"] == 8 * (w + o)
    # the padded layout costs little on these networks except for the thin first layers
    assert t["ResNet-18"]["tbn_packed_bytes"] < 1.03 * t["ResNet-18"]["tbn_bytes"]


def test_packed_words_match_the_library():
    import paper_1701_00485_amd as tbn
    for k, n in ((96, 363), (1000, 4096), (64, 147), (1, 1), (65, 65)):
        assert memory._packed_words(k, n) == tbn.packed_words(k, n)
