"""The seeded input generator: determinism, shapes and the layout contract."""
import numpy as np
import pytest
import torch

from paper_2608_26806_amd import workloads as W


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 100,
                        np.array([1.0, -2.5, 3.0e-39, 65504.0, 1.00390625, 1.01171875], np.float32)])
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(W.bf16_bits_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def _check_layout(lay):
    assert lay.cu_seqlens[0] == 0 and lay.cu_img[0] == 0 and lay.cu_text[0] == 0
    covered = np.zeros(lay.N_tok, np.int32)
    for s, n in zip(lay.img_start, lay.img_len):
        covered[s:s + n] += 1
    covered[lay.text_pos] += 1
    assert np.all(covered == 1)                    # every token is text xor exactly one image
    for b in range(lay.B):
        for i in range(lay.cu_img[b], lay.cu_img[b + 1]):
            assert lay.cu_seqlens[b] <= lay.img_start[i]
            assert lay.img_start[i] + lay.img_len[i] <= lay.cu_seqlens[b + 1]
        tp = lay.text_pos[lay.cu_text[b]:lay.cu_text[b + 1]]
        assert np.all(np.diff(tp) > 0)
        assert tp[-1] == lay.cu_seqlens[b + 1] - 1   # a text row closes every sequence


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_small_configs(cfg):
    wl = W.make_workload(cfg, payload=True, variation=(cfg == 1))
    lay = wl.layout
    _check_layout(lay)
    assert wl.q_text.shape == (lay.T_tot, wl.Hq, wl.d)
    assert wl.k.shape == (lay.N_tok, wl.Hkv, wl.d)
    assert wl.hidden_states.shape == (lay.N_tok, wl.hidden)
    assert wl.pos.shape == (wl.pos_planes, lay.N_tok)
    again = W.make_workload(cfg, payload=False)
    np.testing.assert_array_equal(wl.k, again.k)
    np.testing.assert_array_equal(wl.q_text, again.q_text)


def test_layout_shapes_of_all_configs():
    """Layout-only draws for the large configurations (tensor draws are exercised by the GPU tests)."""
    expect_T = {1: 16, 2: 64, 3: 96, 4: 128, 5: 512}
    for cfg, c in W.CONFIGS.items():
        imgs = W._image_sizes(cfg, c["B"], W._rng(cfg, W._S_LAYOUT))
        lay = W.build_layout(imgs, c["pre"], c["tail"], c["keep"])
        _check_layout(lay)
        assert lay.B == c["B"]
        assert lay.T_tot == expect_T[cfg] * c["B"]
    lay = W.build_layout([[1024] * 32] * 4, 4, 384, 10)
    assert list(lay.keep_total) == [3277] * 4
    lay = W.build_layout([[729] * 4], 4, 48, 25)
    assert list(lay.keep_total) == [729]


def test_config1_salient_and_scale():
    wl = W.make_workload(1, payload=False)
    lay = wl.layout
    assert wl.salient[lay.img_start[0]:lay.img_start[0] + 64].sum() == 8
    assert wl.salient.sum() == 8
    assert wl.dtype == "fp32" and wl.softmax_scale == pytest.approx(1 / 8)
