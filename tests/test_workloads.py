"""The seeded input generator: determinism, distribution, and the paged layout."""

import math

import numpy as np
import torch

from workloads import configs, synth


def test_normal_is_deterministic_and_sliceable():
    a = synth.normal((1000,), seed=5, stream=2, dtype=torch.float32)
    b = synth.normal((1000,), seed=5, stream=2, dtype=torch.float32)
    c = synth.normal((1000,), seed=5, stream=3, dtype=torch.float32)
    assert torch.equal(a, b) and not torch.equal(a, c)
    # The first elements do not depend on the tensor size.
    assert torch.equal(synth.normal((10,), 5, 2, dtype=torch.float32), a[:10])


def test_normal_moments():
    z = synth.normal((1 << 20,), seed=0, stream=0, dtype=torch.float32).double()
    assert abs(z.mean().item()) < 5e-3
    assert abs(z.std().item() - 1.0) < 5e-3
    # Tail mass beyond 2 sigma of N(0,1) is 4.55 %.
    assert abs((z.abs() > 2).double().mean().item() - 0.0455) < 2e-3


def test_bf16_is_rne_of_fp32():
    z32 = synth.normal((4096,), 1, 1, dtype=torch.float32)
    z16 = synth.normal((4096,), 1, 1, dtype=torch.bfloat16)
    assert torch.equal(z32.to(torch.bfloat16), z16)


def test_uniform_int_and_permutation():
    v = synth.uniform_int(5000, 3, 9, seed=1, stream=0)
    assert int(v.min()) == 3 and int(v.max()) == 9
    p = synth.permutation(777, seed=1, stream=0)
    assert torch.equal(torch.sort(p).values, torch.arange(777))


def test_tiny_config_shapes_and_scales():
    c = configs.tiny_fp32()
    assert c["x"].shape == (1, 128, 256) and c["W_R"].shape == (4, 64, 64)
    assert abs(c["W_Q"].std().item() - 1 / 16) < 2e-3


def test_paged_layout_small():
    c = configs.paged_gqa_bf16(B=6, H=8, G=2, d_head=16, L_lo=3, L_hi=70)
    lengths, table, data = c["lengths"], c["block_table"], c["data"]
    bs, poison = c["block_size"], c["poison_block"]
    owned = []
    for b in range(6):
        n = math.ceil(int(lengths[b]) / bs)
        owned += table[b, :n].tolist()
        assert torch.all(table[b, n:] == poison)
        rem = int(lengths[b]) % bs
        last = int(table[b, n - 1])
        if rem:
            assert torch.isnan(data[last, :, rem:, :].float()).all()
        assert torch.isfinite(data[last, :, :rem or bs, :].float()).all()
    assert sorted(owned) == list(range(c["num_blocks"] - 1))
    assert torch.isnan(data[poison].float()).all()


def test_decode_config_new_value_is_last_row():
    c = configs.decode_bf16(B=2, H=3, L=10, d_head=8)
    assert torch.equal(c["v_new"][:, 0], c["V"][:, :, 9, :])
    assert np.all(c["lengths_before"].numpy() == 9)


def test_testbed_config_layers_copies_and_new_rows():
    c = configs.testbed_gqa_bf16(L=20, layers=3, copies=2, d_head=8)
    assert c["V"].shape == (6, 1, 2, 20, 8) and c["K"].shape == c["V"].shape
    assert c["q"].shape == (3, 1, 12, 8)
    assert torch.equal(c["v_new"], c["V"][:, :, :, 19, :])
    # Copies are independent draws; the first copy does not depend on how many follow.
    assert not torch.equal(c["V"][:3], c["V"][3:])
    assert torch.equal(c["V"][:3], configs.testbed_gqa_bf16(L=20, layers=3, d_head=8)["V"])
    assert int(c["lengths"][0]) == 20 and int(c["lengths_before"][0]) == 19
