"""Helpers shared by the GPU tests: device placement of the seeded inputs and
the comparison bar against the oracle."""
import contextlib
import sys

import numpy as np

# fp32 output tolerance: max|dy| <= 1e-3 * max|y_oracle(fp64)|
Y_TOL = 1e-3


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a visible MI355X")
    return torch


def dev(a: np.ndarray):
    torch = torch_cuda()
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def dev_weights(ws: dict) -> dict:
    out = {k: dev(v) for k, v in ws.items()}
    if ws["A"].shape[0] == 0:
        out["A"] = out["B"] = out["beta"] = None
    return out


def host(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def assert_y(y_gpu: np.ndarray, ref: dict, exact32: bool = True, what: str = ""):
    y64 = ref["y64"]
    scale = float(np.abs(y64).max()) if y64.size else 0.0
    err = float(np.abs(y_gpu.astype(np.float64) - y64).max()) if y64.size else 0.0
    assert err <= Y_TOL * scale + 1e-30, f"{what}: max|dy|={err} > {Y_TOL}*{scale}"
    if exact32:
        bad = np.flatnonzero(y_gpu.view(np.uint32) != ref["y32"].view(np.uint32))
        assert bad.size == 0, f"{what}: {bad.size} y differ from the fp32-ordered oracle, first {bad[:5]}"


@contextlib.contextmanager
def forced_switch(D, which: int, value: int):
    """Sets one of the library's test switches for the body, then restores
    the automatic choice."""
    D.test_switch(which, value)
    try:
        yield
    finally:
        D.test_switch(which, 0)
