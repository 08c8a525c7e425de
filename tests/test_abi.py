"""CPU tests of the C-ABI library and the host-side logic (no GPU compute).

* the library loads and exports every function include/unifiednn.h declares;
* invalid specs are rejected by un_create with the documented status and
  message, before any device call is made;
* the input generators are reproducible and shaped as the workloads say;
* the benchmark's algorithmic FLOP count matches hand-computed values.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2408_01331_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "unifiednn.h")


@pytest.fixture(scope="module")
def U():
    from paper_2408_01331_amd import unifiednn as U
    if not os.path.exists(U.LIB_PATH):
        from paper_2408_01331_amd.build import build
        build()
    U.lib()
    return U


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(un_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary_calls():
    names = _declared_functions()
    for n in ["un_create", "un_load_batch", "un_step", "un_get_params", "un_set_params", "un_destroy",
              "un_last_error"]:
        assert n in names


def test_library_exports_every_declared_symbol(U):
    lib = ctypes.CDLL(U.LIB_PATH)
    names = _declared_functions()
    assert set(names) == set(U.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def _create_status(U, specs, batch=4, in_shape=(8,), precision="f32"):
    try:
        ctx = U.un_create(specs, batch, in_shape, precision)
    except U.UnError as e:
        return e.status, str(e)
    U.un_destroy(ctx)
    return U.UN_OK, ""


MLP = {"layers": [("linear", 5), ("relu",), ("linear", 3)], "num_classes": 3}


@pytest.mark.parametrize("spec,status,fragment", [
    ({"layers": [("relu",), ("linear", 3)], "num_classes": 3}, 7, "ReLU/MaxPool2"),
    ({"layers": [("linear", 3), ("relu",)], "num_classes": 3}, 7, "ReLU on the logits"),
    ({"layers": [("linear", 4)], "num_classes": 3}, 1, "num_classes"),
    ({"layers": [("linear", 5), ("relu",), ("conv", 4, 3, 1), ("flatten",), ("linear", 3)], "num_classes": 3}, 1,
     "conv needs an image input"),
    ({"layers": [("linear", 0), ("linear", 3)], "num_classes": 3}, 1, "bad linear out"),
    ({"layers": [], "num_classes": 3}, 1, "no layers"),
    ({"layers": [("linear", 3)], "num_classes": 0}, 1, "num_classes must be positive"),
])
def test_invalid_specs_rejected_before_any_device_call(U, spec, status, fragment):
    st, msg = _create_status(U, [MLP, spec])
    assert st == status, msg
    assert fragment in msg
    assert "model 1" in msg


def test_conv_spec_errors(U):
    img = (1, 6, 6)
    st, msg = _create_status(U, [{"layers": [("linear", 3)], "num_classes": 3}], in_shape=img)
    assert st == U.UN_ERR_INVALID and "flatten" in msg
    st, msg = _create_status(U, [{"layers": [("conv", 2, 9, 0), ("flatten",), ("linear", 3)],
                                  "num_classes": 3}], in_shape=img)
    assert st == U.UN_ERR_INVALID and "kernel larger" in msg
    st, msg = _create_status(U, [{"layers": [("conv", 3, 3, 0), ("pool",), ("flatten",), ("linear", 3)],
                                  "num_classes": 3}], in_shape=img)
    assert st == U.UN_ERR_UNSUPPORTED and "multiple of 8" in msg


def test_invalid_input_spec(U):
    st, msg = _create_status(U, [MLP], batch=0)
    assert st == U.UN_ERR_INVALID
    ctx = ctypes.c_void_p()
    assert U.lib().un_create(None, 1, None, ctypes.byref(ctx)) == U.UN_ERR_INVALID
    assert not ctx.value
    assert U.lib().un_last_error(None)


def test_null_context_calls(U):
    L = U.lib()
    assert L.un_step(None, ctypes.c_float(0.1), None) == U.UN_ERR_INVALID
    assert L.un_sync(None) == U.UN_ERR_INVALID
    L.un_destroy(None)


# ---------------------------------------------------------------------------
# Input generators
# ---------------------------------------------------------------------------
def test_generators_are_seeded_and_shaped():
    wl = W.get("cifar16")
    x0, y0 = W.make_batch(wl, 0)
    x1, y1 = W.make_batch(wl, 0)
    assert x0.shape == (256, 3, 32, 32) and x0.dtype == np.float32
    assert np.array_equal(x0, x1) and np.array_equal(y0, y1)
    assert not np.array_equal(W.make_batch(wl, 1)[0], x0)
    assert y0.min() >= 0 and y0.max() < 10
    assert np.array_equal(W.init_params(wl.specs[2], wl.in_shape, 0, 2)[0],
                          W.init_params(wl.specs[2], wl.in_shape, 0, 2)[0])


def test_workload_architectures():
    wl = W.get("mlp64")
    assert wl.n_models == 64 and wl.batch == 512 and wl.precision == "bf16"
    for s in wl.specs:
        lin = [l for l in s["layers"] if l[0] == "linear"]
        assert 2 <= len(lin) <= 6 and lin[-1][1] == 100
        assert all(64 <= l[1] <= 2048 for l in lin[:-1])
    c = W.get("cifar16")
    for s in c.specs:
        convs = [l[1] for l in s["layers"] if l[0] == "conv"]
        assert convs[0] in (32, 48, 64) and convs[1] in (64, 96, 128) and convs[2] in (128, 192, 256)
    l4 = W.get("lenet4")
    assert all(s["layers"][0][1] in (6, 8, 12) for s in l4.specs)


def test_bench_flop_count_by_hand():
    import bench
    wl = W.get("mlp2")
    flops, nbytes, n_params = bench.algorithmic_work(wl)
    fwd = 2 * 64 * (784 * 128 + 128 * 10 + 784 * 64 + 64 * 10)
    assert flops["gemm_fwd"] == fwd
    assert flops["gemm_bwd"] == fwd + 2 * 64 * (128 * 10 + 64 * 10)   # wgrad all, dgrad not for layer 1
    assert n_params == 101770 + 50890
    # fp32: 4-byte tensors, update = read + write of the master (8 B per parameter)
    B = 64
    fwd_b = sum(B * 784 * 4 + h * 784 * 4 + h * 4 + B * h * 4 + B * h * 4 + 10 * h * 4 + 10 * 4 + B * 10 * 4
                for h in (128, 64))
    assert nbytes["gemm_fwd"] == fwd_b
    bwd_b = sum((B * h * 4 + B * 784 * 4) + (B * 10 * 4 + B * h * 4) + 8 * (784 * h + h + 10 * h + 10)
                + (B * 10 * 4 + 10 * h * 4 + B * h * 4) for h in (128, 64))
    assert nbytes["gemm_bwd"] == bwd_b
    assert nbytes["ce"] == 2 * (B * 10 * 4 + B * 10 * 4)


def test_bench_conv_bytes_by_hand():
    import bench
    wl = W.Workload(name="t", n_models=1, description="", specs=[{"layers": [("conv", 8, 3, 1), ("relu",), ("pool",), ("flatten",),
                                                                ("linear", 10)], "num_classes": 10}],
                    batch=2, in_shape=(3, 6, 6), precision="bf16", steps=1, lr=0.01, seed=0)
    flops, nbytes, _ = bench.algorithmic_work(wl)
    assert flops["conv_fwd"] == 2 * 2 * 36 * 8 * 27 and flops["conv_dgrad"] == 0
    pooled = 2 * 3 * 3 * 8
    assert nbytes["conv_fwd"] == 2 * 36 * 3 * 2 + 8 * 27 * 2 + pooled * 3
    assert nbytes["conv_wgrad"] == pooled * 3 + 2 * 36 * 3 * 2
    assert nbytes["other"] == (8 * 27 + 8) * 10
