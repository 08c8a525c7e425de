"""Write the oracle's 5-step trajectory of sampled models of the 16-CNN
workload (16 CIFAR-shaped CNNs, batch 256, bf16 with fp32 master weights),
for the GPU parity test that cannot afford to run the oracle itself (about a
minute and a half per model-step on 8 host cores).

    python tests/golden/make_cifar16_k5.py --model 1 [--steps 5]

writes tests/golden/cifar16_k5_m<model>.npz with, for that model trained
alone from its seeded start: the loss of every step, the final parameters, the
last step's gradient, the units the oracle flagged as ill-conditioned, and the
spread between the oracle's two evaluation orders (fp64 and fp32
accumulation) over the same steps.
It calls only the oracle and the seeded input generators; nothing here comes
from the GPU path. The sampled models (1, 4, 6, 11) cover every drawn width:
first conv 32 / 48 / 64, second 64 / 96 / 128, third 128 / 192 / 256.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
for p in (ROOT, os.path.dirname(HERE)):
    if p not in sys.path:
        sys.path.insert(0, p)

import oracle  # noqa: E402
from paper_2408_01331_amd import workloads as W  # noqa: E402
from _parity import oracle_spread  # noqa: E402

MODELS = (1, 4, 6, 11)
SPREAD_KEYS = ("update", "grad", "update_fro", "grad_fro", "loss")


def sha(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def input_digest(wl, i, steps):
    """sha256 of everything the trajectory is computed from: the workload's
    description (specs, rate, seed, precision), model i's starting parameters
    and the batches of the steps."""
    h = hashlib.sha256(wl.to_json().encode())
    h.update(str(i).encode())
    for p in W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init):
        h.update(np.ascontiguousarray(p, np.float32).tobytes())
    for s in range(steps):
        x, y = W.make_batch(wl, s)
        h.update(np.ascontiguousarray(x).tobytes())
        h.update(np.ascontiguousarray(y).tobytes())
    return h.hexdigest()


def path_of(i):
    return os.path.join(HERE, f"cifar16_k5_m{i}.npz")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--model", type=int, required=True)
    ap.add_argument("--steps", type=int, default=5)
    a = ap.parse_args()
    wl = W.get("cifar16")
    i = a.model
    th0 = W.init_params(wl.specs[i], wl.in_shape, wl.seed, i, wl.init)
    batches = [W.make_batch(wl, s) for s in range(a.steps)]
    t0 = time.time()
    flags = {}
    losses, params, grads = oracle.train(wl.specs[i], th0, batches, wl.lr, wl.precision, flags)
    print(f"model {i}: trajectory in {time.time() - t0:.0f} s, losses {np.round(losses, 5).tolist()}", flush=True)
    spread = oracle_spread(wl.specs[i], th0, batches, wl.lr, wl.precision, flags, (losses, params, grads))
    print(f"model {i}: fp32-accumulation run done at {time.time() - t0:.0f} s", flush=True)
    out = {"losses": np.asarray(losses, np.float64)}
    for t, (p, g) in enumerate(zip(params, grads)):
        out[f"p{t}"] = np.asarray(p, np.float32)
        out[f"g{t}"] = np.asarray(g, np.float32)
    for wi, units in flags.items():
        out[f"flags{wi}"] = np.array(sorted(units), np.int64)
    for k in SPREAD_KEYS:
        out[f"spread_{k}"] = np.asarray(spread[k], np.float64)
    meta = dict(model=i, steps=a.steps, lr=wl.lr, seed=wl.seed, precision=wl.precision, workload=wl.name,
                inputs_sha256=input_digest(wl, i, a.steps),
                oracle_sha256=sha(os.path.join(ROOT, "oracle", "oracle.py")))
    out["meta"] = np.array(json.dumps(meta))
    np.savez_compressed(path_of(i), **out)
    print(f"wrote {path_of(i)}", flush=True)


def load(i):
    """(losses, params, grads, flags), spread dict, meta of model i."""
    z = np.load(path_of(i), allow_pickle=False)
    meta = json.loads(str(z["meta"]))
    n = len([k for k in z.files if k.startswith("p")])
    params = [z[f"p{t}"] for t in range(n)]
    grads = [z[f"g{t}"] for t in range(n)]
    flags = {int(k[5:]): set(z[k].tolist()) for k in z.files if k.startswith("flags")}
    spread = {k: z[f"spread_{k}"].tolist() for k in SPREAD_KEYS}
    return (z["losses"], params, grads, flags), spread, meta


if __name__ == "__main__":
    main()
