"""CPU tests of the parity helpers: which parameters a flagged (ill-conditioned)
ReLU / max-pool unit reaches, including through residual skips."""
import numpy as np

from paper_2408_01331_amd import workloads as W
from _parity import flagged_masks, perturb_ulp

L, RELU, RB, RE, POOL, FLAT = (lambda n: ("linear", n)), ("relu",), ("res_begin",), ("res_end",), ("pool",), \
    ("flatten",)


def _marked(masks):
    return [set(map(tuple, np.argwhere(m).tolist())) for m in masks]


def test_plain_chain_marks_own_row_and_next_column():
    spec = {"layers": [L(6), RELU, L(5), RELU, L(4)], "num_classes": 4}
    params = W.init_params(spec, (3,), 0, 0)
    m = flagged_masks(spec, params, {0: {2}})
    assert m[0][2].all() and m[0].sum() == 3            # row 2 of W0 [6, 3]
    assert m[1][2] and m[1].sum() == 1
    assert m[2][:, 2].all() and m[2].sum() == 5         # column 2 of W1 [5, 6]
    assert not m[3].any() and not m[4].any() and not m[5].any()


def test_skip_carries_the_unit_to_the_block_sum_and_its_readers():
    # W0 -> relu -> [W1 relu W2] + skip -> relu -> W3
    spec = {"layers": [L(6), RELU, RB, L(4), RELU, L(6), RE, RELU, L(3)], "num_classes": 3}
    params = W.init_params(spec, (5,), 0, 0)
    m = flagged_masks(spec, params, {0: {1}})
    assert m[0][1].all() and m[1][1]                      # own row and bias
    assert m[2][:, 1].all()                               # the block's first layer reads unit 1
    assert m[4][1].all() and m[5][1]                      # the sum's unit 1: end layer row / bias
    assert m[6][:, 1].all() and m[6].sum() == 3           # the layer after the block reads the sum's unit 1
    assert m[2].sum() == 4 and m[4].sum() == 4            # nothing else in those tensors


def test_back_to_back_blocks_recurse():
    spec = {"layers": [L(5), RELU, RB, L(5), RE, RELU, RB, L(5), RE, L(2)], "num_classes": 2}
    params = W.init_params(spec, (4,), 0, 0)
    m = flagged_masks(spec, params, {0: {3}})
    for w in (0, 2, 4):
        assert m[w][3].all(), w                           # rows of unit 3 in all three layers
    for w in (2, 4, 6):
        assert m[w][:, 3].all(), w                        # every reader of unit 3
    # a unit flagged at the first block's sum reaches the second block only
    m2 = flagged_masks(spec, params, {2: {0}})
    assert not m2[0].any() and m2[2][0].all() and m2[4][0].all() and m2[4][:, 0].all() and m2[6][:, 0].all()


def test_conv_flatten_linear_marks_the_channels_feature_block():
    spec = {"layers": [("conv", 4, 3, 1), RELU, POOL, FLAT, L(3)], "num_classes": 3}
    params = W.init_params(spec, (2, 6, 6), 0, 0)
    m = flagged_masks(spec, params, {0: {2}})
    assert m[0][2].all() and m[0].sum() == 2 * 9
    S = 9                                                  # 3x3 pooled map per channel
    assert m[2][:, 2 * S:3 * S].all() and m[2].sum() == 3 * S


def test_residual_conv_block():
    spec = {"layers": [("conv", 4, 3, 1), RELU, RB, ("conv", 4, 3, 1), RE, RELU, ("conv", 2, 1, 0), FLAT, L(3)],
            "num_classes": 3}
    params = W.init_params(spec, (2, 5, 5), 0, 0)
    m = flagged_masks(spec, params, {0: {1}})
    assert m[2][:, 1].all() and m[2][1].all() and m[3][1]   # block conv: reads channel 1, and its sum row 1
    assert m[4][:, 1].all()                                  # the 1x1 conv after the block reads channel 1


U, A = (lambda t: ("unflatten", t)), ("attention",)


def test_flat_unit_read_as_a_token_feature_and_its_residual_attention():
    # W0 [8, 5] -> relu -> 2 tokens of 4 -> [attention] + skip -> relu -> flatten -> W
    spec = {"layers": [L(8), RELU, U(2), RB, A, RE, RELU, FLAT, L(3)], "num_classes": 3}
    params = W.init_params(spec, (5,), 0, 0)
    assert [np.shape(p) for p in params] == [(8, 5), (8,), (12, 4), (12,), (4, 4), (4,), (3, 8), (3,)]
    m = flagged_masks(spec, params, {0: {6}})                # flat unit 6 = token 1, feature 2
    assert m[0][6].all() and m[0].sum() == 5 and m[1][6] and m[1].sum() == 1
    assert m[2][:, 2].all() and m[2].sum() == 12             # the in-projection reads feature 2
    assert m[4][2].all() and m[5][2] and m[4].sum() == 4     # the sum's feature 2: out-projection row
    assert m[6][:, [2, 6]].all() and m[6].sum() == 6         # flattened: feature 2 of both tokens
    assert not m[3].any() and not m[7].any()


def test_token_feature_flagged_at_the_attention_output():
    spec = {"layers": [U(3), A, RELU, L(8), RELU, FLAT, L(2)], "num_classes": 2}
    params = W.init_params(spec, (3 * 8,), 0, 0)
    m = flagged_masks(spec, params, {2: {5}})                # out-projection unit 5
    assert m[2][5].all() and m[3][5] and m[2].sum() == 8 and not m[0].any()
    assert m[4][:, 5].all() and m[4].sum() == 8              # the token-wise Linear reads feature 5
    m2 = flagged_masks(spec, params, {4: {1}})                # token-wise Linear unit 1, 3 tokens
    assert m2[4][1].all() and m2[6][:, [1, 9, 17]].all() and m2[6].sum() == 6


def test_perturb_ulp_moves_half_the_elements_by_one_ulp():
    p = [np.linspace(-1, 1, 10001, dtype=np.float32)]
    q = perturb_ulp(p, 3)[0]
    moved = q != p[0]
    assert 0.45 < moved.mean() < 0.55
    gap = np.abs(np.nextafter(p[0], np.float32(np.inf)) - p[0])
    gap_dn = np.abs(p[0] - np.nextafter(p[0], np.float32(-np.inf)))
    d = np.abs(q.astype(np.float64) - p[0])
    assert np.all((d == 0) | (d == gap) | (d == gap_dn))
