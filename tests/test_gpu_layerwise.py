"""Every op of the workloads on the GPU, fed the oracle's own tensors.

The end-to-end iteration of a deep ReLU / BatchNorm network is chaotic under
float32 rounding: float32 evaluations of it (torch's, or the oracle with its
conv / BN outputs nudged by one float32 rounding) scatter by up to 50% on some
gradient tensors, so the end-to-end parity test there can only hold the GPU
to that scatter.  This test removes the chaos instead of widening the bar:
each op's kernels, plain and as the model folds them, run on the oracle's
own tensors at kernel-level bars (tests/layerwise.py).  These are reduced
batches; tests/test_gpu_full_batch.py does the same at the benchmark
configurations' own batches.
"""
import pytest

import synth
from oracle import cnn as OC
from oracle import nets as ON
from tests import layerwise

pytestmark = pytest.mark.gpu

CASES = [("resnet50", 2), ("resnet152", 2), ("inception_v4", 1), ("googlenet", 2), ("vgg16", 1), ("resnet18", 8),
         ("alexnet", 2), ("tiny", 4)]


@pytest.mark.parametrize("name,batch", CASES, ids=[f"{n}-b{b}" for n, b in CASES])
def test_each_op_on_oracle_tensors(name, batch):
    spec = ON.get(name)
    net = OC.Net(spec, batch)
    x, y, params = synth.cnn_inputs(30 + batch, batch, spec["hwc"], spec["classes"], net.param_specs)
    print(f"layerwise {name} batch {batch}", flush=True)
    res = net.loss_and_grads(x, y, params, keep=True)
    worst = layerwise.check_ops(name, net, y, params, res)
    print(f"{name}: worst error / bar per op kind: "
          + ", ".join(f"{k} {v:.3f}" for k, v in sorted(worst.items())), flush=True)
