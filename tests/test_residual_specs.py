"""Residual blocks in model specs: the planner's validation (un_plan_bytes runs
on the host, no device needed) of what is a well-formed block, with the status
each malformed one returns."""
import pytest

from paper_2408_01331_amd import unifiednn as U


def _need_lib():
    try:
        U.lib()
    except OSError as e:  # not built
        pytest.skip(f"library not built: {e}")


def _spec(*layers, classes=5):
    return {"layers": list(layers), "num_classes": classes}


L, RELU, RB, RE = (lambda n: ("linear", n)), ("relu",), ("res_begin",), ("res_end",)

GOOD = [
    _spec(L(8), RELU, RB, L(8), RE, RELU, L(5)),
    _spec(L(8), RB, L(3), RELU, L(8), RE, RB, L(8), RE, L(5)),       # two blocks, no ReLUs after them
    _spec(L(8), RELU, RB, L(8), RE, RELU, RB, L(8), RE, RELU, L(5)),
    _spec(RB, L(16), RE, RELU, L(5)),                                  # a skip from the flat 16-feature input
]

BAD = [
    (_spec(RB, L(8), RE, L(5)), U.UN_ERR_INVALID),                     # at the 16-feature input, width changes
    (_spec(L(8), RB, L(8), RELU, RE, L(5)), U.UN_ERR_UNSUPPORTED),     # ReLU inside, right before the end
    (_spec(L(8), RB, L(7), RE, L(5)), U.UN_ERR_INVALID),               # width changes
    (_spec(L(8), RB, RE, L(5)), U.UN_ERR_INVALID),                     # empty
    (_spec(L(8), RE, L(5)), U.UN_ERR_INVALID),                         # end without begin
    (_spec(L(8), RB, L(8), L(5)), U.UN_ERR_INVALID),                   # never closed
    (_spec(L(5), RB, L(5), RE), U.UN_ERR_UNSUPPORTED),                 # ends at the logits
    (_spec(L(8), RB, L(8), RB, L(8), RE, RE, L(5)), U.UN_ERR_UNSUPPORTED),  # nested
]


C = lambda o, k=3, pad=1: ("conv", o, k, pad)
POOL, FLAT = ("pool",), ("flatten",)

GOOD_CNN = [
    _spec(C(8), RELU, RB, C(8), RE, RELU, C(8), RELU, POOL, FLAT, L(5)),
    _spec(C(8), RELU, POOL, RB, C(4), RELU, C(8), RE, RELU, RB, C(8, 1, 0), RE, FLAT, L(5)),
]

BAD_CNN = [
    (_spec(C(8), RB, C(8), RE, RELU, POOL, FLAT, L(5)), U.UN_ERR_UNSUPPORTED),          # pool of the sum
    (_spec(C(8), RB, C(8), RELU, POOL, C(8), RE, FLAT, L(5)), U.UN_ERR_UNSUPPORTED),    # pool inside
    (_spec(C(8), RB, C(8, 3, 0), RE, FLAT, L(5)), U.UN_ERR_INVALID),                    # map shrinks
    (_spec(C(8), RB, C(6), RE, FLAT, L(5)), U.UN_ERR_INVALID),                          # channels change
    (_spec(C(8), FLAT, RB, L(5), RE, L(5)), U.UN_ERR_UNSUPPORTED),                      # after a flatten
    (_spec(RB, C(8), RE, FLAT, L(5)), U.UN_ERR_UNSUPPORTED),                            # at an image input
]


@pytest.mark.parametrize("precision", ["f32", "bf16"])
def test_residual_conv_specs(precision):
    _need_lib()
    for s in GOOD_CNN:
        assert U.un_plan_bytes([s], 4, (8, 8, 8), precision)[0] > 0
    for s, status in BAD_CNN:
        with pytest.raises(U.UnError) as e:
            U.un_plan_bytes([s], 4, (8, 8, 8), precision)
        assert e.value.status == status, s


@pytest.mark.parametrize("precision", ["f32", "bf16"])
def test_residual_specs_accepted(precision):
    _need_lib()
    base, _ = U.un_plan_bytes([_spec(L(8), RELU, L(8), RELU, L(5))], 16, (16,), precision)
    for s in GOOD:
        arena, _ = U.un_plan_bytes([s], 16, (16,), precision)
        assert arena > 0
    # the markers hold no parameters and no buffers of their own
    same, _ = U.un_plan_bytes([GOOD[0]], 16, (16,), precision)
    assert same == base


@pytest.mark.parametrize("case", range(len(BAD)))
def test_residual_specs_rejected(case):
    _need_lib()
    spec, status = BAD[case]
    with pytest.raises(U.UnError) as e:
        U.un_plan_bytes([spec], 16, (16,), "f32")
    assert e.value.status == status


@pytest.mark.parametrize("precision", ["f32", "bf16"])
def test_conv_tensor_size_limits(precision):
    """The conv kernels address every activation, gradient and weight tensor
    with 32-bit byte offsets and an output row of elements with 24-bit
    multiplies: the planner refuses larger conv layers before anything is
    allocated, and takes the largest ones below the limits."""
    _need_lib()
    es = 2 if precision == "bf16" else 4
    conv = _spec(C(8), RELU, FLAT, L(5))
    # the largest batch of 8-channel 64x64 maps whose conv output stays under 2^31 bytes
    ok_batch = ((1 << 31) - 1) // (8 * 64 * 64 * es)
    assert U.un_plan_bytes([conv], ok_batch, (8, 64, 64), precision)[0] > 0
    with pytest.raises(U.UnError) as e:
        U.un_plan_bytes([conv], ok_batch + 1, (8, 64, 64), precision)
    assert e.value.status == U.UN_ERR_UNSUPPORTED
    # an output row of 2^24 elements (8192 columns x 2048 channels)
    with pytest.raises(U.UnError) as e:
        U.un_plan_bytes([_spec(C(2048, 1, 0), FLAT, L(5))], 1, (8, 1, 8192), precision)
    assert e.value.status == U.UN_ERR_UNSUPPORTED
