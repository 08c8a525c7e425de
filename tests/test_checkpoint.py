"""Per-model checkpoint files (host side, no GPU): names and shapes of a
PyTorch nn.Sequential state_dict, optimizer state and update count round trip."""
import numpy as np
import pytest

from paper_2408_01331_amd import checkpoint as C
from paper_2408_01331_amd import workloads as W
from paper_2408_01331_amd.unifiednn import flatten_params

torch = pytest.importorskip("torch")


class _Residual(torch.nn.Module):
    """inner(x) + x"""

    def __init__(self, inner):
        super().__init__()
        self.inner = inner

    def forward(self, x):
        return self.inner(x) + x


def _sequential(spec, in_shape):
    layers, shape, outer = [], tuple(in_shape), None
    for l in spec["layers"]:
        if l[0] == "res_begin":
            outer, layers = layers, []
            continue
        if l[0] == "res_end":
            outer.append(_Residual(torch.nn.Sequential(*layers)))
            layers, outer = outer, None
            continue
        if l[0] == "linear":
            layers.append(torch.nn.Linear(int(np.prod(shape)), l[1]))
            shape = (l[1],)
        elif l[0] == "conv":
            layers.append(torch.nn.Conv2d(shape[0], l[1], l[2], padding=l[3]))
            shape = (l[1], shape[1] + 2 * l[3] - l[2] + 1, shape[2] + 2 * l[3] - l[2] + 1)
        elif l[0] == "relu":
            layers.append(torch.nn.ReLU())
        elif l[0] == "pool":
            layers.append(torch.nn.MaxPool2d(2))
            shape = (shape[0], shape[1] // 2, shape[2] // 2)
        elif l[0] == "flatten":
            layers.append(torch.nn.Flatten())
            shape = (int(np.prod(shape)),)
    return torch.nn.Sequential(*layers)


class _Host:
    """The part of Hybrid a checkpoint uses, on the host."""

    def __init__(self, wl):
        self.specs, self.in_shape, self.precision = wl.specs, tuple(wl.in_shape), wl.precision
        self.in_shape_of = lambda i: self.in_shape
        self.params = {i: flatten_params(W.init_params(s, wl.in_shape, 3, i)) for i, s in enumerate(wl.specs)}
        self.optimizers = {i: dict(kind="sgd", momentum=0.0, betas=[0.9, 0.999], eps=1e-8) for i in range(len(wl.specs))}
        self.state = {i: (np.zeros(0, np.float32), 0) for i in range(len(wl.specs))}

    def get_params(self, i):
        return self.params[i]

    def set_params(self, i, flat):
        assert flat.size == self.params[i].size
        self.params[i] = np.asarray(flat, np.float32).copy()

    def get_opt_state(self, i):
        return self.state[i]

    def set_opt_state(self, i, state, step):
        self.state[i] = (np.asarray(state, np.float32).copy(), step)

    def set_optimizer(self, i, kind, momentum, betas, eps):
        self.optimizers[i] = dict(kind=kind, momentum=momentum, betas=list(betas), eps=eps)
        k = {"sgd": 0, "momentum": 1, "adam": 2}[kind]
        self.state[i] = (np.zeros(k * self.params[i].size, np.float32), 0)


@pytest.mark.parametrize("name", ["lenet4", "mlp8", "resnet8"])
def test_checkpoint_names_load_into_torch_sequential(name, tmp_path):
    wl = W.get(name)
    h = _Host(wl)
    i = 1
    path = str(tmp_path / "m.safetensors")
    C.save(h, i, path)
    tensors, meta = C.read(path)
    mod = _sequential(wl.specs[i], wl.in_shape)
    sd = {k: torch.from_numpy(v) for k, v in tensors.items()}
    mod.load_state_dict(sd, strict=True)
    np.testing.assert_array_equal(flatten_params([p.detach().numpy() for p in mod.parameters()]), h.params[i])
    assert meta["optimizer"]["kind"] == "sgd" and meta["step"] == 0


@pytest.mark.parametrize("kind", ["momentum", "adam"])
def test_checkpoint_round_trip_with_optimizer_state(kind, tmp_path):
    wl = W.get("lenet4")
    src, dst = _Host(wl), _Host(wl)
    i = 2
    src.set_optimizer(i, kind, 0.8, (0.85, 0.99), 1e-7)
    rng = np.random.default_rng(0)
    k = 1 if kind == "momentum" else 2
    src.set_opt_state(i, rng.standard_normal(k * src.params[i].size).astype(np.float32), 17)
    path = str(tmp_path / "m.safetensors")
    C.save(src, i, path)
    tensors, meta = C.read(path)
    names = C.param_names(wl.specs[i])
    assert sorted(tensors) == sorted(names + [f"{s}.{n}" for s in C.STATE_NAMES[kind] for n in names])
    C.load(dst, i, path)
    assert dst.optimizers[i] == src.optimizers[i]
    np.testing.assert_array_equal(dst.params[i], src.params[i])
    np.testing.assert_array_equal(dst.state[i][0], src.state[i][0])
    assert dst.state[i][1] == 17
    # into another architecture: refused
    with pytest.raises(ValueError):
        C.load(_Host(W.get("mlp8")), 0, path)
