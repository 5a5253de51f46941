"""Helpers shared by the test modules (comparison metrics, config builders)."""
import numpy as np

from paper_2609_28568_amd import synth

# Acceptance bars for the GPU path against the fp32 oracle on identical inputs:
# loss within 1e-2 absolute; activations and gradients within 2e-2 relative L2.
LOSS_ATOL = 1e-2
REL_L2 = 2e-2


def rel_l2(x, ref):
    x = np.asarray(x, np.float64).ravel()
    ref = np.asarray(ref, np.float64).ravel()
    n = np.linalg.norm(ref)
    if n == 0.0:
        return 0.0 if np.all(x == 0.0) else np.inf
    return float(np.linalg.norm(x - ref) / n)


def workload(name, **over):
    w = dict(synth.WORKLOADS[name])
    w.update(over)
    return w


def oracle_config(w, **optim):
    import oracle
    o = dict(synth.OPTIM)
    o.update(optim)
    return oracle.Config.from_dict({**w, **o})
